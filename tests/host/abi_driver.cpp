// A plain C++ program that runs one GPipe mini-batch of a boundary (no-loss)
// fp32 encoder partition through the library's C ABI alone: device buffers
// from hipMalloc, the partition's calls in the order Sections 2.2-2.3 give
// (M forwards, M re-materialising backwards in reverse order, one update),
// no Python and no torch in the process.
//
// Usage: abi_driver IN OUT
//   IN  (little-endian): int32 layers, d_model, d_ff, heads, seq_len,
//       seqs_per_microbatch, num_microbatches, nrec; float32 ln_eps, lr;
//       nrec parameter records (int32 layer, int32 id, int64 count,
//       float32[count]); x then dY, float32 [M][n S D] each.
//   OUT: y and dX (float32 [M][n S D] each), then for every record of IN
//       in its order the fp32 gradient accumulator before the update, then
//       the fp32 master parameter after it.
// Exit status 0 on success; 2 with the library's message on a failed call;
// 3 on a file or HIP runtime error.
#include <hip/hip_runtime_api.h>

#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <vector>

#include "../../include/gp.h"

namespace {

struct Rec {
    int32_t layer, id;
    int64_t count;
    std::vector<float> v;
};

[[noreturn]] void die(int code, const char* what, const char* detail) {
    std::fprintf(stderr, "abi_driver: %s: %s\n", what, detail ? detail : "");
    std::exit(code);
}

void check(gp_status s, const char* call) {
    if (s != GP_OK) die(2, call, gp_last_error());
}

void hip(hipError_t e, const char* call) {
    if (e != hipSuccess) die(3, call, hipGetErrorString(e));
}

template <typename T>
void get(FILE* f, T* p, size_t n) {
    if (std::fread(p, sizeof(T), n, f) != n) die(3, "read", "input file too short");
}

template <typename T>
void put(FILE* f, const T* p, size_t n) {
    if (std::fwrite(p, sizeof(T), n, f) != n) die(3, "write", "output file");
}

} // namespace

int main(int argc, char** argv) {
    if (argc != 3) die(3, "usage", "abi_driver IN OUT");
    FILE* in = std::fopen(argv[1], "rb");
    if (!in) die(3, "open", argv[1]);
    int32_t h[8];
    float fl[2];
    get(in, h, 8);
    get(in, fl, 2);
    const int layers = h[0], D = h[1], F = h[2], H = h[3], S = h[4], n = h[5], M = h[6], nrec = h[7];
    std::vector<Rec> recs(nrec);
    for (Rec& r : recs) {
        get(in, &r.layer, 1);
        get(in, &r.id, 1);
        get(in, &r.count, 1);
        r.v.resize((size_t)r.count);
        get(in, r.v.data(), r.v.size());
    }
    const size_t T = (size_t)n * S, per = T * D, all = per * M;
    std::vector<float> x(all), dy(all), y(all), dx(all);
    get(in, x.data(), all);
    get(in, dy.data(), all);
    std::fclose(in);

    gp_partition* p = nullptr;
    check(gp_partition_create(layers, D, F, H, &p), "gp_partition_create");
    gp_config c{};
    c.seq_len = S;
    c.seqs_per_microbatch = n;
    c.num_microbatches = M;
    c.dtype = GP_F32;
    c.kind = GP_ENCODER;
    c.loss = GP_LOSS_NONE;
    c.ln_eps = fl[0];
    c.optimizer = GP_OPT_SGD;
    check(gp_partition_configure(p, &c), "gp_partition_configure");
    for (const Rec& r : recs) check(gp_set_param(p, r.layer, r.id, r.v.data(), r.v.size()), "gp_set_param");

    hipStream_t st;
    hip(hipStreamCreateWithFlags(&st, hipStreamNonBlocking), "hipStreamCreateWithFlags");
    float *dx_d = nullptr, *dy_d = nullptr, *x_d = nullptr, *y_d = nullptr;
    for (float** b : {&x_d, &y_d, &dy_d, &dx_d}) hip(hipMalloc((void**)b, all * sizeof(float)), "hipMalloc");
    hip(hipMemcpy(x_d, x.data(), all * sizeof(float), hipMemcpyHostToDevice), "hipMemcpy x");
    hip(hipMemcpy(dy_d, dy.data(), all * sizeof(float), hipMemcpyHostToDevice), "hipMemcpy dy");

    for (int m = 0; m < M; ++m)
        check(gp_forward_microbatch(p, m, x_d + m * per, nullptr, y_d + m * per, (gp_stream)st),
              "gp_forward_microbatch");
    for (int m = M - 1; m >= 0; --m)
        check(gp_backward_microbatch_remat(p, m, dy_d + m * per, dx_d + m * per, nullptr, (gp_stream)st),
              "gp_backward_microbatch_remat");
    hip(hipStreamSynchronize(st), "hipStreamSynchronize");
    std::vector<std::vector<float>> grads(recs.size());
    for (size_t i = 0; i < recs.size(); ++i) {
        grads[i].resize(recs[i].v.size());
        check(gp_get_grad(p, recs[i].layer, recs[i].id, grads[i].data(), grads[i].size()), "gp_get_grad");
    }
    check(gp_accumulate_and_step(p, fl[1], nullptr, (gp_stream)st), "gp_accumulate_and_step");
    hip(hipStreamSynchronize(st), "hipStreamSynchronize");
    hip(hipMemcpy(y.data(), y_d, all * sizeof(float), hipMemcpyDeviceToHost), "hipMemcpy y");
    hip(hipMemcpy(dx.data(), dx_d, all * sizeof(float), hipMemcpyDeviceToHost), "hipMemcpy dx");

    FILE* out = std::fopen(argv[2], "wb");
    if (!out) die(3, "open", argv[2]);
    put(out, y.data(), all);
    put(out, dx.data(), all);
    for (const auto& g : grads) put(out, g.data(), g.size());
    std::vector<float> w;
    for (const Rec& r : recs) {
        w.resize(r.v.size());
        check(gp_get_param(p, r.layer, r.id, w.data(), w.size()), "gp_get_param");
        put(out, w.data(), w.size());
    }
    std::fclose(out);
    check(gp_partition_destroy(p), "gp_partition_destroy");
    for (float* b : {x_d, y_d, dy_d, dx_d}) hip(hipFree(b), "hipFree");
    hip(hipStreamDestroy(st), "hipStreamDestroy");
    return 0;
}
