#include <algorithm>
// misc.hip -- boundary intake, casts, loss heads and the synchronous update.
//
// All reductions are two-stage with a fixed order (per-block partials, then
// one finalising block), so every result is reproducible bit for bit.
#include "common.hpp"
#include "kernels.hpp"

namespace gp {

namespace {

constexpr int EW_BLOCKS = 1024;   // grid of the grid-stride elementwise kernels
constexpr int LOSS_BLOCKS = 256;  // partials of the MSE loss

template <typename T>
__global__ void __launch_bounds__(256) intake_kernel(const T* __restrict__ src, T* __restrict__ stash,
                                                     float* __restrict__ x32, long count) {
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < count; i += (long)gridDim.x * 256) {
        const T v = src[i];
        if (stash) stash[i] = v;
        if (x32) x32[i] = to_f32(v);
    }
}

// 8 bf16 elements per thread with 16-byte accesses (count % 8 == 0, aligned pointers).
__global__ void __launch_bounds__(256) intake_bf16_v8(const bf16x8* __restrict__ src, bf16x8* __restrict__ stash,
                                                      f32x4* __restrict__ x32, long n8) {
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n8; i += (long)gridDim.x * 256) {
        const bf16x8 v = src[i];
        if (stash) stash[i] = v;
        if (x32) {
            x32[2 * i] = f32x4{(float)v[0], (float)v[1], (float)v[2], (float)v[3]};
            x32[2 * i + 1] = f32x4{(float)v[4], (float)v[5], (float)v[6], (float)v[7]};
        }
    }
}

template <typename T>
__global__ void __launch_bounds__(256) cast_kernel(const float* __restrict__ src, T* __restrict__ dst, long count) {
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < count; i += (long)gridDim.x * 256)
        dst[i] = to_elt<T>(src[i]);
}

template <typename T>
__global__ void __launch_bounds__(256) mse_kernel(const float* __restrict__ y, const T* __restrict__ t, long count,
                                                  double norm, float* __restrict__ d32, T* __restrict__ de,
                                                  double* __restrict__ partial) {
    __shared__ double red[4];
    double s = 0.0;
    const float scale = (float)(2.0 / norm);
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < count; i += (long)gridDim.x * 256) {
        const float d = y[i] - to_f32(t[i]);
        s += (double)d * (double)d;
        const float g = scale * d;
        d32[i] = g;
        de[i] = to_elt<T>(g);
    }
    s = wave_sum_d(s);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = s;
    __syncthreads();
    if (threadIdx.x == 0) partial[blockIdx.x] = (red[0] + red[1] + red[2] + red[3]) / norm;
}

__global__ void loss_finalize_kernel(const double* __restrict__ partial, int nblk, double* __restrict__ acc,
                                     int accumulate) {
    if (threadIdx.x != 0 || blockIdx.x != 0) return;
    double s = 0.0;
    for (int b = 0; b < nblk; ++b) s += partial[b];
    acc[0] = accumulate ? acc[0] + s : s;
}

// Label-smoothed cross-entropy over one row of V logits per block.
// q_v = ls / V + (1 - ls) [v == label];  loss_row = -sum_v q_v log p_v
//   = lse - ls / V sum_v z_v - (1 - ls) z_label,   lse = log sum_v exp z_v;
// dZ_v = (p_v - q_v) / norm.
// With clip > 0 every logit first becomes min(max(z, -clip), clip) and the
// gradient passes only where |z| <= clip (the clip's derivative).
// A label outside [0, V) is read as class 0 (so every access stays inside
// the row) and raises bad_label[0], which the host reports.
template <typename T>
__global__ void __launch_bounds__(256) xent_kernel(T* __restrict__ z, int V, const int* __restrict__ labels,
                                                   float ls, float clip, double norm, double* __restrict__ partial,
                                                   int* __restrict__ bad_label) {
    __shared__ float red[4];
    __shared__ float bc[2];
    const long row = blockIdx.x;
    T* zr = z + row * (long)V;
    const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const float lim = clip > 0.f ? clip : INFINITY;
    auto logit = [&](int v) { return fminf(fmaxf(to_f32(zr[v]), -lim), lim); };
    float m = -INFINITY, sz = 0.f;
    for (int v = tid; v < V; v += 256) {
        const float x = logit(v);
        m = fmaxf(m, x);
        sz += x;
    }
    m = wave_max(m);
    sz = wave_sum(sz);
    if (lane == 0) red[w] = m;
    __syncthreads();
    if (tid == 0) bc[0] = fmaxf(fmaxf(red[0], red[1]), fmaxf(red[2], red[3]));
    __syncthreads();
    m = bc[0];
    __syncthreads();
    if (lane == 0) red[w] = sz;
    __syncthreads();
    if (tid == 0) bc[1] = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
    sz = bc[1];
    float se = 0.f;
    for (int v = tid; v < V; v += 256) se += expf(logit(v) - m);
    se = wave_sum(se);
    __syncthreads();
    if (lane == 0) red[w] = se;
    __syncthreads();
    if (tid == 0) bc[0] = red[0] + red[1] + red[2] + red[3];
    __syncthreads();
    se = bc[0];
    const int raw = labels[row];
    const bool ok = raw >= 0 && raw < V;
    const int lab = ok ? raw : 0;
    if (!ok && tid == 0) bad_label[0] = 1;
    const float zl = logit(lab);
    __syncthreads();
    const float lse = m + logf(se);
    const float inv = 1.f / se, u = ls / V, gn = (float)(1.0 / norm);
    for (int v = tid; v < V; v += 256) {
        const float z = to_f32(zr[v]);
        const float p = expf(fminf(fmaxf(z, -lim), lim) - m) * inv;
        const float q = u + (v == lab ? 1.f - ls : 0.f);
        zr[v] = to_elt<T>(fabsf(z) <= lim ? (p - q) * gn : 0.f);
    }
    if (tid == 0) partial[row] = ((double)lse - (double)u * sz - (1.0 - ls) * zl) / norm;
}

__global__ void __launch_bounds__(256) sgd_kernel(float* __restrict__ w, const float* __restrict__ g, float lr,
                                                  long count) {
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < count; i += (long)gridDim.x * 256) w[i] -= lr * g[i];
}

// RMSProp: ms <- rho ms + (1 - rho) g^2;  w <- w - lr g / sqrt(ms + eps).
// Four parameters per thread with 16-byte accesses (count % 4 == 0: every
// parameter block of the plan is 64-float aligned).
__global__ void __launch_bounds__(256) rmsprop_kernel(f32x4* __restrict__ w, const f32x4* __restrict__ g,
                                                      f32x4* __restrict__ ms, float lr, float rho, float eps,
                                                      long n4) {
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < n4; i += (long)gridDim.x * 256) {
        const f32x4 gv = g[i];
        f32x4 m = ms[i], wv = w[i];
#pragma unroll
        for (int e = 0; e < 4; ++e) {
            m[e] = rho * m[e] + (1.f - rho) * (gv[e] * gv[e]);
            wv[e] -= lr * gv[e] / sqrtf(m[e] + eps);
        }
        ms[i] = m;
        w[i] = wv;
    }
}

// kn = W, nk = W^T through a 64 x 64 LDS tile (both writes coalesced).
template <typename T>
__global__ void __launch_bounds__(256) refresh_kernel(const float* __restrict__ w, int in, int out,
                                                      T* __restrict__ kn, T* __restrict__ nk) {
    __shared__ float tile[64][65];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int r = ty; r < 64; r += 4) {
        const int row = r0 + r, col = c0 + tx;
        if (row < in && col < out) {
            const float v = w[(long)row * out + col];
            tile[r][tx] = v;
            kn[(long)row * out + col] = to_elt<T>(v);
        }
    }
    __syncthreads();
    for (int c = ty; c < 64; c += 4) {
        const int col = c0 + c, row = r0 + tx;
        if (row < in && col < out) nk[(long)col * in + row] = to_elt<T>(tile[tx][c]);
    }
}

// Four consecutive elements of a 16-bit working copy, rounded from fp32.
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
template <typename E> struct Copy4;
template <> struct Copy4<bf16> {
    static __device__ __forceinline__ void store(bf16* p, float a, float b, float c, float d) {
        *reinterpret_cast<bf16x4*>(p) = {(bf16)a, (bf16)b, (bf16)c, (bf16)d};
    }
};
template <> struct Copy4<_Float16> {
    static __device__ __forceinline__ void store(_Float16* p, float a, float b, float c, float d) {
        *reinterpret_cast<f16x4*>(p) = {(_Float16)a, (_Float16)b, (_Float16)c, (_Float16)d};
    }
};

// The same for bf16 copies of whole 64 x 64 tiles (in, out multiples of 64):
// 16-byte reads of W, 8-byte writes of both copies.  NK: the element type of
// the transposed copy (bf16, or fp16 for a GEMM with fp16 operands).
template <typename NK>
__global__ void __launch_bounds__(256) refresh_bf16_tiles(const float* __restrict__ w, int in, int out,
                                                          bf16* __restrict__ kn, NK* __restrict__ nk) {
    __shared__ float tile[64][65];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64, t = threadIdx.x;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int idx = t + 256 * k, r = idx >> 4, c = (idx & 15) * 4;
        const long o = (long)(r0 + r) * out + c0 + c;
        const f32x4 v = *reinterpret_cast<const f32x4*>(w + o);
#pragma unroll
        for (int j = 0; j < 4; ++j) tile[r][c + j] = v[j];
        *reinterpret_cast<bf16x4*>(kn + o) = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int idx = t + 256 * k, c = idx >> 4, r = (idx & 15) * 4;
        Copy4<NK>::store(nk + (long)(c0 + c) * in + r0 + r, tile[r][c], tile[r + 1][c], tile[r + 2][c], tile[r + 3][c]);
    }
}

// The update of a linear's weights fused with the refresh of its bf16 working
// copies (in, out multiples of 64): W <- W - lr G (SGD) or the RMSProp step
// (rms: ms <- rho ms + (1 - rho) G^2; W <- W - lr G / sqrt(ms + eps)) on the
// fp32 master, then kn = W, nk = W^T from the updated values through a
// 64 x 64 LDS tile -- one pass over W and G instead of an update pass and a
// refresh pass.  Per element the same arithmetic as sgd_kernel and
// rmsprop_kernel.
template <typename NK>
__global__ void __launch_bounds__(256) update_refresh_tiles(float* __restrict__ w, const float* __restrict__ g,
                                                            float* __restrict__ ms, float lr, float rho, float eps,
                                                            int rms, int in, int out, bf16* __restrict__ kn,
                                                            NK* __restrict__ nk) {
    __shared__ float tile[64][65];
    const int r0 = blockIdx.y * 64, c0 = blockIdx.x * 64, t = threadIdx.x;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int idx = t + 256 * k, r = idx >> 4, c = (idx & 15) * 4;
        const long o = (long)(r0 + r) * out + c0 + c;
        f32x4 v = *reinterpret_cast<const f32x4*>(w + o);
        const f32x4 gv = *reinterpret_cast<const f32x4*>(g + o);
        if (rms) {
            f32x4 m = *reinterpret_cast<const f32x4*>(ms + o);
#pragma unroll
            for (int e = 0; e < 4; ++e) {
                m[e] = rho * m[e] + (1.f - rho) * (gv[e] * gv[e]);
                v[e] -= lr * gv[e] / sqrtf(m[e] + eps);
            }
            *reinterpret_cast<f32x4*>(ms + o) = m;
        } else {
#pragma unroll
            for (int e = 0; e < 4; ++e) v[e] -= lr * gv[e];
        }
        *reinterpret_cast<f32x4*>(w + o) = v;
#pragma unroll
        for (int j = 0; j < 4; ++j) tile[r][c + j] = v[j];
        *reinterpret_cast<bf16x4*>(kn + o) = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
    }
    __syncthreads();
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        const int idx = t + 256 * k, c = idx >> 4, r = (idx & 15) * 4;
        Copy4<NK>::store(nk + (long)(c0 + c) * in + r0 + r, tile[r][c], tile[r + 1][c], tile[r + 2][c], tile[r + 3][c]);
    }
}

// The same update over the parameters outside the linears' weight blocks
// (biases, LayerNorm gains and shifts): workgroup b takes the float range
// [ranges[2 b], ranges[2 b] + ranges[2 b + 1]).
__global__ void __launch_bounds__(256) update_ranges_kernel(float* __restrict__ w, const float* __restrict__ g,
                                                            float* __restrict__ ms, float lr, float rho, float eps,
                                                            int rms, const long* __restrict__ ranges) {
    const long off = ranges[2 * blockIdx.x], n = ranges[2 * blockIdx.x + 1];
    for (long i = off + threadIdx.x; i < off + n; i += 256) {
        const float gv = g[i];
        if (rms) {
            const float m = rho * ms[i] + (1.f - rho) * (gv * gv);
            ms[i] = m;
            w[i] -= lr * gv / sqrtf(m + eps);
        } else {
            w[i] -= lr * gv;
        }
    }
}

// fp4 copy of bf16 rows (the W^T working copy, rows of `in` values): one wave
// per row; 8 values per lane step; one E8M0 scale per row (see e2m1_code).
__global__ void __launch_bounds__(256) quant4_rows_kernel(const bf16* __restrict__ src, int rows, int in,
                                                          unsigned char* __restrict__ q4, unsigned char* __restrict__ sc) {
    const int lane = threadIdx.x & 63;
    const long row = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows) return;
    const bf16x8* r8 = reinterpret_cast<const bf16x8*>(src + row * in);
    const int n8 = in / 8;
    float amax = 0.f;
    for (int i = lane; i < n8; i += 64) {
        const bf16x8 v = r8[i];
#pragma unroll
        for (int e = 0; e < 8; ++e) amax = fmaxf(amax, fabsf((float)v[e]));
    }
    const unsigned s = e8m0_for_amax(wave_max(amax));
    const float inv = e8m0_inv(s);
    unsigned* o4 = reinterpret_cast<unsigned*>(q4 + row * (in / 2));
    for (int i = lane; i < n8; i += 64) {
        const bf16x8 v = r8[i];
        unsigned q = 0;
#pragma unroll
        for (int e = 0; e < 8; ++e) q |= e2m1_code((float)v[e] * inv) << (4 * e);
        o4[i] = q;
    }
    if (lane == 0) sc[row] = (unsigned char)s;
}

// MFMA-loop peak probe: 4 waves per workgroup, each with 8 independent
// 32x32 accumulators and two operand sets of pseudo-random bf16 (so that the
// multiplier inputs toggle as in a real GEMM); 16 MFMAs per trip.
__global__ void __launch_bounds__(256) mfma_peak_kernel(float* __restrict__ out, int iters) {
    typedef __bf16 b8 __attribute__((ext_vector_type(8)));
    typedef float f16v __attribute__((ext_vector_type(16)));
    unsigned h = (blockIdx.x * 256u + threadIdx.x) * 2654435761u + 12345u;
    b8 a[2], b[2];
#pragma unroll
    for (int k = 0; k < 2; ++k)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            h = h * 1664525u + 1013904223u;
            a[k][e] = (__bf16)(((int)(h >> 16) - 32768) * (1.f / 32768.f));
            h = h * 1664525u + 1013904223u;
            b[k][e] = (__bf16)(((int)(h >> 16) - 32768) * (1.f / 32768.f));
        }
    f16v c[8];
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) c[j][r] = 0.f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < 2; ++k)
#pragma unroll
            for (int j = 0; j < 8; ++j) c[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[k], b[k], c[j], 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j)
#pragma unroll
        for (int r = 0; r < 16; ++r) s += c[j][r];
    out[blockIdx.x * 256 + threadIdx.x] = s;
}

__global__ void __launch_bounds__(256) finite_kernel(const float* __restrict__ x, long count, int* __restrict__ flag) {
    bool bad = false;
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < count; i += (long)gridDim.x * 256)
        bad |= !isfinite(x[i]);
    if (__any(bad) && (threadIdx.x & 63) == 0) flag[0] = 1;
}

int ew_grid(long count) {
    long g = (count + 255) / 256;
    return (int)(g < EW_BLOCKS ? (g > 0 ? g : 1) : EW_BLOCKS);
}

} // namespace

int loss_blocks() { return LOSS_BLOCKS; }
int xent_partials(long rows) { return (int)rows; }

gp_status intake(int dtype, const void* src, void* stash, float* x32, long count, hipStream_t st) {
    auto a16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    if (dtype == GP_BF16 && count % 8 == 0 && a16(src) && a16(stash) && a16(x32)) {
        klaunch(intake_bf16_v8, ew_grid(count / 8), 256, 0, st, reinterpret_cast<const bf16x8*>(src),
                reinterpret_cast<bf16x8*>(stash), reinterpret_cast<f32x4*>(x32), count / 8);
    } else if (dtype == GP_BF16)
        klaunch(intake_kernel<bf16>, ew_grid(count), 256, 0, st, reinterpret_cast<const bf16*>(src),
                                                             reinterpret_cast<bf16*>(stash), x32, count);
    else
        klaunch(intake_kernel<float>, ew_grid(count), 256, 0, st, reinterpret_cast<const float*>(src),
                                                              reinterpret_cast<float*>(stash), x32, count);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status cast_out(int dtype, const float* src, void* dst, long count, hipStream_t st) {
    if (dtype == GP_BF16) klaunch(cast_kernel<bf16>, ew_grid(count), 256, 0, st, src, reinterpret_cast<bf16*>(dst), count);
    else klaunch(cast_kernel<float>, ew_grid(count), 256, 0, st, src, reinterpret_cast<float*>(dst), count);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status mse_grad(int dtype, const float* y, const void* target, long count, double norm, float* d32, void* delt,
                   double* partial, int* nblk, hipStream_t st) {
    *nblk = LOSS_BLOCKS;
    if (dtype == GP_BF16)
        klaunch(mse_kernel<bf16>, LOSS_BLOCKS, 256, 0, st, y, reinterpret_cast<const bf16*>(target), count, norm, d32,
                                                      reinterpret_cast<bf16*>(delt), partial);
    else
        klaunch(mse_kernel<float>, LOSS_BLOCKS, 256, 0, st, y, reinterpret_cast<const float*>(target), count, norm, d32,
                                                       reinterpret_cast<float*>(delt), partial);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status loss_finalize(const double* partial, int nblk, double* acc, int accumulate, hipStream_t st) {
    klaunch(loss_finalize_kernel, 1, 64, 0, st, partial, nblk, acc, accumulate);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status xent_ls(int dtype, void* z, long rows, int V, const int* labels, float ls, float clip, double norm,
                  double* partial, int* bad_label, hipStream_t st) {
    if (dtype == GP_BF16)
        klaunch(xent_kernel<bf16>, (unsigned)rows, 256, 0, st, reinterpret_cast<bf16*>(z), V, labels, ls, clip, norm,
                partial, bad_label);
    else
        klaunch(xent_kernel<float>, (unsigned)rows, 256, 0, st, reinterpret_cast<float*>(z), V, labels, ls, clip, norm,
                partial, bad_label);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status mfma_peak(hipStream_t st, double* tflops) {
    int dev = 0, cus = 0;
    GP_HIP(hipGetDevice(&dev));
    GP_HIP(hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev));
    const int grid = 2 * cus, iters = 2000;
    float* out = nullptr;
    GP_HIP(hipMalloc(reinterpret_cast<void**>(&out), (size_t)grid * 256 * sizeof(float)));
    hipEvent_t e0 = nullptr, e1 = nullptr;
    gp_status s = GP_OK;
    double best = 0.0;
    if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) s = set_error(GP_ERR_HIP, "mfma_peak: event");
    for (int rep = 0; rep < 4 && s == GP_OK; ++rep) {
        hipEventRecord(e0, st);
        klaunch(mfma_peak_kernel, grid, 256, 0, st, out, iters);
        const hipError_t le = take_launch_status();
        hipEventRecord(e1, st);
        float ms = 0.f;
        if (le != hipSuccess || hipEventSynchronize(e1) != hipSuccess || hipEventElapsedTime(&ms, e0, e1) != hipSuccess) {
            s = set_error(GP_ERR_HIP, "mfma_peak: launch or timing failed");
            break;
        }
        const double fl = (double)grid * 4 * iters * 16 * 32768.0;
        if (rep > 0 && ms > 0.f) best = std::max(best, fl / (ms * 1e-3) * 1e-12);  // the first run warms up
    }
    if (e0) hipEventDestroy(e0);
    if (e1) hipEventDestroy(e1);
    hipStreamSynchronize(st);
    hipFree(out);
    if (s == GP_OK && tflops) *tflops = best;
    return s;
}

gp_status sgd_update(float* w, const float* g, float lr, long count, hipStream_t st) {
    klaunch(sgd_kernel, ew_grid(count), 256, 0, st, w, g, lr, count);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status rmsprop_update(float* w, const float* g, float* ms, float lr, float rho, float eps, long count,
                         hipStream_t st) {
    if (count % 4) return set_error(GP_ERR_INVALID_ARG, "rmsprop: parameter count must be a multiple of 4");
    klaunch(rmsprop_kernel, ew_grid(count / 4), 256, 0, st, reinterpret_cast<f32x4*>(w),
            reinterpret_cast<const f32x4*>(g), reinterpret_cast<f32x4*>(ms), lr, rho, eps, count / 4);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status update_refresh_linear(float* w, const float* g, float* ms, float lr, float rho, float eps, int in,
                                int out, void* kn, void* nk, void* q4, void* q4s, hipStream_t st, bool nk16) {
    if (in % 64 || out % 64) return set_error(GP_ERR_INVALID_ARG, "update_refresh: in and out must be multiples of 64");
    if (nk16 && q4) return set_error(GP_ERR_INVALID_ARG, "update_refresh: an fp16 W^T has no fp4 copy");
    dim3 grid(out / 64, in / 64);
    if (nk16)
        klaunch(update_refresh_tiles<_Float16>, grid, 256, 0, st, w, g, ms, lr, rho, eps, ms ? 1 : 0, in, out,
                reinterpret_cast<bf16*>(kn), reinterpret_cast<_Float16*>(nk));
    else
        klaunch(update_refresh_tiles<bf16>, grid, 256, 0, st, w, g, ms, lr, rho, eps, ms ? 1 : 0, in, out,
                reinterpret_cast<bf16*>(kn), reinterpret_cast<bf16*>(nk));
    GP_LAUNCH_CHECK();
    if (q4) {
        if (in % 8) return set_error(GP_ERR_UNSUPPORTED, "refresh: fp4 copies are made from bf16 rows");
        klaunch(quant4_rows_kernel, (out + 3) / 4, 256, 0, st, reinterpret_cast<const bf16*>(nk), out, in,
                reinterpret_cast<unsigned char*>(q4), reinterpret_cast<unsigned char*>(q4s));
        GP_LAUNCH_CHECK();
    }
    return GP_OK;
}

gp_status update_ranges(float* w, const float* g, float* ms, float lr, float rho, float eps, const long* ranges,
                        int nranges, hipStream_t st) {
    if (nranges <= 0) return GP_OK;
    klaunch(update_ranges_kernel, nranges, 256, 0, st, w, g, ms, lr, rho, eps, ms ? 1 : 0, ranges);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status refresh_linear(int dtype, const float* w, int in, int out, void* kn, void* nk, void* q4, void* q4s,
                         hipStream_t st, bool nk16) {
    dim3 grid((out + 63) / 64, (in + 63) / 64);
    if (nk16 && (dtype != GP_BF16 || in % 64 || out % 64 || q4))
        return set_error(GP_ERR_INVALID_ARG, "refresh: an fp16 W^T needs bf16 whole 64 x 64 tiles and no fp4 copy");
    if (nk16)
        klaunch(refresh_bf16_tiles<_Float16>, grid, 256, 0, st, w, in, out, reinterpret_cast<bf16*>(kn),
                reinterpret_cast<_Float16*>(nk));
    else if (dtype == GP_BF16 && in % 64 == 0 && out % 64 == 0)
        klaunch(refresh_bf16_tiles<bf16>, grid, 256, 0, st, w, in, out, reinterpret_cast<bf16*>(kn),
                reinterpret_cast<bf16*>(nk));
    else if (dtype == GP_BF16)
        klaunch(refresh_kernel<bf16>, grid, 256, 0, st, w, in, out, reinterpret_cast<bf16*>(kn), reinterpret_cast<bf16*>(nk));
    else
        klaunch(refresh_kernel<float>, grid, 256, 0, st, w, in, out, reinterpret_cast<float*>(kn), reinterpret_cast<float*>(nk));
    GP_LAUNCH_CHECK();
    if (q4) {
        if (dtype != GP_BF16 || in % 8) return set_error(GP_ERR_UNSUPPORTED, "refresh: fp4 copies are made from bf16 rows");
        klaunch(quant4_rows_kernel, (out + 3) / 4, 256, 0, st, reinterpret_cast<const bf16*>(nk), out, in,
                static_cast<unsigned char*>(q4), static_cast<unsigned char*>(q4s));
        GP_LAUNCH_CHECK();
    }
    return GP_OK;
}

// All-ones bytes over [p, p + bytes): a NaN in every fp32, bf16 and fp64
// element.  16-byte stores over the aligned middle, byte stores at the edges.
__global__ void __launch_bounds__(256) poison_kernel(unsigned char* __restrict__ p, long head, long n16, long tail) {
    const long t = (long)blockIdx.x * 256 + threadIdx.x, stride = (long)gridDim.x * 256;
    if (t < head) p[t] = 0xFF;
    uint4* q = reinterpret_cast<uint4*>(p + head);
    for (long i = t; i < n16; i += stride) q[i] = make_uint4(~0u, ~0u, ~0u, ~0u);
    if (t < tail) p[head + 16 * n16 + t] = 0xFF;
}

gp_status poison_fill(void* p, size_t bytes, hipStream_t st) {
    if (!p || bytes == 0) return GP_OK;
    unsigned char* c = static_cast<unsigned char*>(p);
    const long head = (long)((16 - (reinterpret_cast<uintptr_t>(c) & 15)) & 15);
    const long h = head < (long)bytes ? head : (long)bytes;
    const long n16 = ((long)bytes - h) / 16, tail = (long)bytes - h - 16 * n16;
    klaunch(poison_kernel, ew_grid(n16 > 256 ? n16 : 256), 256, 0, st, c, h, n16, tail);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

// Empty kernel that delimits a timed launch in a profiler's dispatch list.
// Its grid encodes the label (role workgroups in x, edge + 1 in y), which a
// kernel trace records.
__global__ void role_marker_kernel() {}

gp_status role_marker(int role, int edge, hipStream_t st) {
    klaunch(role_marker_kernel, dim3(role, edge + 1), 64, 0, st);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status finite_check(const float* x, long count, int* flag, hipStream_t st) {
    klaunch(finite_kernel, ew_grid(count), 256, 0, st, x, count, flag);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

} // namespace gp
