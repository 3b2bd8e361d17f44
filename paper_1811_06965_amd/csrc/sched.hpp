// sched.hpp -- HIP-free host logic of one GPipe partition: argument
// validation, the parameter/working-copy layout plan, the workspace plan and
// the micro-batch state machine.  Compiles with any C++17 compiler so it can
// be unit-tested on a machine without a GPU.
//
// State machine (GPipe, Section 2.2): within a mini-batch every micro-batch
// is forwarded in order 0..M-1, then back-propagated in reverse order
// M-1..0 with the forward recomputed (Section 2.3), then one update is
// applied.  Parameters may only change between mini-batches, so every
// micro-batch's backward uses the parameters of its forward.
#pragma once

#include <cstddef>
#include <algorithm>
#include <cstdint>
#include <string>
#include <utility>
#include <vector>

#include "../../include/gp.h"

namespace gp {

struct Dims {
    int L = 0, D = 0, F = 0, H = 0;
};

// Geometry fixed by gp_partition_configure.
struct Geometry {
    int S = 0, n = 0, M = 0;
    int dtype = GP_BF16, kind = GP_ENCODER, Smem = 0, loss = GP_LOSS_NONE, V = 0;
    float ls = 0.f, eps = 1e-5f;
    int check_finite = 0;
    int keep_act = 0;     // stored-activation mode: no recompute, every micro-batch's intermediates kept
    int optimizer = GP_OPT_SGD;
    float rms_decay = 0.f, rms_eps = 0.f;
    float logit_clip = 0.f;
    int ffn_fp4 = 1;  // bf16: fp4 correction of the feed-forward input projection (see Linear::split)
    int ffn_f16 = 1;  // bf16: that projection with fp16 operands instead, where the widths allow (Linear::f16)
    long long T() const { return (long long)n * S; }     // token rows of one micro-batch
    long long Tm() const { return (long long)n * Smem; } // memory rows of one micro-batch
};

inline gp_status check_dims(int L, int D, int F, int H, std::string& msg) {
    if (L <= 0 || D <= 0 || F <= 0 || H <= 0) {
        msg = "layers, d_model, d_ff and heads must be positive";
        return GP_ERR_INVALID_ARG;
    }
    if (D % H != 0) {
        msg = "d_model must be a multiple of heads";
        return GP_ERR_INVALID_ARG;
    }
    return GP_OK;
}

// Shapes the kernels implement.  GEMM operands are read as 16-byte vectors,
// so every matrix width is a multiple of 8; attention keeps a whole key row
// of up to 256 keys in registers (bf16) or loops over keys (fp32).
inline gp_status check_config(const Dims& d, const gp_config& c, std::string& msg) {
    if (c.seq_len <= 0 || c.seqs_per_microbatch <= 0 || c.num_microbatches <= 0) {
        msg = "seq_len, seqs_per_microbatch and num_microbatches must be positive";
        return GP_ERR_INVALID_ARG;
    }
    if (c.dtype != GP_F32 && c.dtype != GP_BF16) { msg = "unknown dtype"; return GP_ERR_INVALID_ARG; }
    if (c.kind != GP_ENCODER && c.kind != GP_DECODER_CROSS) { msg = "unknown layer kind"; return GP_ERR_INVALID_ARG; }
    if (c.loss != GP_LOSS_NONE && c.loss != GP_LOSS_MSE && c.loss != GP_LOSS_XENT_LS) {
        msg = "unknown loss"; return GP_ERR_INVALID_ARG;
    }
    if (c.kind == GP_DECODER_CROSS && c.mem_seq_len <= 0) { msg = "decoder needs mem_seq_len > 0"; return GP_ERR_INVALID_ARG; }
    if (c.kind == GP_ENCODER && c.mem_seq_len != 0) { msg = "encoder takes no memory (mem_seq_len must be 0)"; return GP_ERR_INVALID_ARG; }
    if (c.loss == GP_LOSS_XENT_LS && c.vocab <= 1) { msg = "cross-entropy head needs vocab > 1"; return GP_ERR_INVALID_ARG; }
    if (c.loss != GP_LOSS_XENT_LS && c.vocab != 0) { msg = "vocab is only used by the cross-entropy head"; return GP_ERR_INVALID_ARG; }
    if (!(c.label_smoothing >= 0.f && c.label_smoothing < 1.f)) { msg = "label_smoothing must be in [0, 1)"; return GP_ERR_INVALID_ARG; }
    if (!(c.ln_eps > 0.f)) { msg = "ln_eps must be positive"; return GP_ERR_INVALID_ARG; }
    if (c.keep_activations != 0 && c.keep_activations != 1) { msg = "keep_activations must be 0 or 1"; return GP_ERR_INVALID_ARG; }
    if (c.optimizer != GP_OPT_SGD && c.optimizer != GP_OPT_RMSPROP) { msg = "unknown optimizer"; return GP_ERR_INVALID_ARG; }
    if (c.optimizer == GP_OPT_RMSPROP && !(c.rms_decay >= 0.f && c.rms_decay < 1.f && c.rms_eps > 0.f)) {
        msg = "RMSProp needs rms_decay in [0, 1) and rms_eps > 0"; return GP_ERR_INVALID_ARG;
    }
    if (c.optimizer == GP_OPT_SGD && (c.rms_decay != 0.f || c.rms_eps != 0.f)) {
        msg = "rms_decay and rms_eps are only used by RMSProp"; return GP_ERR_INVALID_ARG;
    }
    if (!(c.logit_clip >= 0.f) || (c.logit_clip > 0.f && c.loss != GP_LOSS_XENT_LS)) {
        msg = "logit_clip must be >= 0, and nonzero only with the cross-entropy head"; return GP_ERR_INVALID_ARG;
    }
    const int dh = d.D / d.H;
    if (d.D % 8 || d.F % 8 || (c.loss == GP_LOSS_XENT_LS && c.vocab % 8)) {
        msg = "d_model, d_ff and vocab must be multiples of 8"; return GP_ERR_UNSUPPORTED;
    }
    if (c.dtype == GP_BF16) {
        if (dh != 64) { msg = "bf16 attention kernels need d_model / heads == 64"; return GP_ERR_UNSUPPORTED; }
        auto ok_len = [](int s) { return s % 32 == 0 && s <= 256; };
        if (!ok_len(c.seq_len) || (c.kind == GP_DECODER_CROSS && !ok_len(c.mem_seq_len))) {
            msg = "bf16 attention kernels need sequence lengths that are multiples of 32 and <= 256";
            return GP_ERR_UNSUPPORTED;
        }
    } else {
        if (dh > 64 || dh % 4) { msg = "fp32 attention kernels need d_model / heads <= 64 and a multiple of 4"; return GP_ERR_UNSUPPORTED; }
        if (c.seq_len > 1024 || c.mem_seq_len > 1024) { msg = "fp32 attention kernels need sequence lengths <= 1024"; return GP_ERR_UNSUPPORTED; }
    }
    return GP_OK;
}

// ------------------------------------------------------------ parameter plan
// fp32 masters and gradients share one layout.  A linear layer stores W as
// [in, out] row-major immediately followed by its bias [out]; a LayerNorm
// stores gamma [D] then beta [D].  Each linear layer also has two working
// copies in the partition dtype: W as [in, out] ("kn", the B operand of
// dX = dY W^T) and W^T as [out, in] ("nk", the B operand of Y = X W), so
// that both GEMMs stream their weight operand along the reduction dimension.
struct Linear {
    size_t w = 0, b = 0;        // float offsets of W and bias in master/grad
    size_t kn = 0, nk = 0;      // element offsets of the working copies
    size_t q4 = 0, q4s = 0;     // split: element offsets of the fp4 copy of W^T and its row scales
    int in = 0, out = 0;
    int role = 0;               // gp_kernel_role of its forward GEMM; +1 input gradient, +2 weight gradient
    // bf16 feed-forward input projection: the forward adds the product of the
    // LayerNorm output's bf16 rounding residuals (fp4) with an fp4 copy of W,
    // so that the pre-activations, whose signs set the ReLU mask the backward
    // uses, carry almost none of the rounding error of its bf16 input
    bool split = false;
    // bf16 feed-forward input projection with fp16 operands instead: the
    // LayerNorm output and W^T carry three more mantissa bits into the
    // pre-activations at the bf16 MFMA rate (nk holds fp16; kn stays bf16 for
    // the input gradient, and the bf16 LayerNorm output for the weight gradient)
    bool f16 = false;
    bool present = false;
};
struct Norm {
    size_t g = 0, b = 0;
    int n = 0;
    int id = 0;                 // index among the partition's LayerNorms
    bool present = false;
};
struct LayerPlan {
    Norm ln1, ln2, ln3;
    Linear qkv, o, ffn1, ffn2, xq, xkv, xo;
};
struct HeadPlan {
    Norm lnf;
    Linear out;
};
struct ParamPlan {
    std::vector<LayerPlan> layers;
    HeadPlan head;
    size_t n32 = 0;  // floats in master (and in grads)
    size_t nelt = 0; // elements in the working copies
    size_t count = 0;
    std::vector<const Linear*> linears() const {
        std::vector<const Linear*> v;
        for (auto& l : layers)
            for (const Linear* x : {&l.qkv, &l.o, &l.ffn1, &l.ffn2, &l.xq, &l.xkv, &l.xo})
                if (x->present) v.push_back(x);
        if (head.out.present) v.push_back(&head.out);
        return v;
    }
    std::vector<const Norm*> norms() const {
        std::vector<const Norm*> v;
        for (auto& l : layers)
            for (const Norm* x : {&l.ln1, &l.ln2, &l.ln3})
                if (x->present) v.push_back(x);
        if (head.lnf.present) v.push_back(&head.lnf);
        return v;
    }
};

inline size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

inline ParamPlan plan_params(const Dims& d, const Geometry& g) {
    ParamPlan p;
    size_t f = 0, e = 0;
    auto lin = [&](Linear& x, int in, int out, int role, bool split = false) {
        x.present = true;
        x.role = role;
        x.in = in;
        x.out = out;
        x.split = split;
        x.w = f;
        x.b = f + (size_t)in * out;
        f = align_up(x.b + out, 64); // keep every block 256-byte aligned
        x.kn = e;
        x.nk = e + (size_t)in * out;
        e = align_up(x.nk + (size_t)in * out, 128);
        if (split) {  // bf16 elements: in / 2 bytes = in / 4 elements per row, one byte of scale per row
            x.q4 = e;
            e = align_up(x.q4 + (size_t)out * in / 4, 128);
            x.q4s = e;
            e = align_up(x.q4s + ((size_t)out + 1) / 2, 128);
        }
        p.count += (size_t)in * out + out;
    };
    int nnorm = 0;
    auto norm = [&](Norm& x, int n) {
        x.present = true;
        x.n = n;
        x.id = nnorm++;
        x.g = f;
        x.b = f + n;
        f = align_up(x.b + n, 64);
        p.count += 2 * (size_t)n;
    };
    const bool dec = g.kind == GP_DECODER_CROSS;
    p.layers.resize(d.L);
    for (auto& l : p.layers) {
        norm(l.ln1, d.D);
        lin(l.qkv, d.D, 3 * d.D, GP_K_QKV_FWD);
        lin(l.o, d.D, d.D, GP_K_O_FWD);
        norm(l.ln2, d.D);
        const bool f16 = g.dtype == GP_BF16 && g.ffn_f16 && d.D % 256 == 0 && d.D <= 2048 && d.F % 64 == 0;
        lin(l.ffn1, d.D, d.F, GP_K_FFN1_FWD, g.dtype == GP_BF16 && g.ffn_fp4 && !f16);
        l.ffn1.f16 = f16;
        lin(l.ffn2, d.F, d.D, GP_K_FFN2_FWD);
        if (dec) {
            lin(l.xq, d.D, d.D, GP_K_XQ_FWD);
            lin(l.xkv, d.D, 2 * d.D, GP_K_XKV_FWD);
            lin(l.xo, d.D, d.D, GP_K_XO_FWD);
            norm(l.ln3, d.D);
        }
    }
    if (g.loss == GP_LOSS_XENT_LS) {
        norm(p.head.lnf, d.D);
        lin(p.head.out, d.D, g.V, GP_K_HEAD_FWD);
    }
    p.n32 = f;
    p.nelt = e;
    return p;
}

// The bf16 update pass.  Each linear's W is updated in 64 x 64 tiles in the
// same pass that rewrites its working copies; every other parameter (the
// biases, LayerNorm gains and shifts) is updated from a list of (offset,
// count) float ranges, written to `ranges` as flat pairs.  Returns false (and
// leaves `ranges` empty) unless every linear is a whole number of tiles and
// the weights and ranges together cover the n32 master floats exactly once.
inline bool plan_update_ranges(const ParamPlan& p, std::vector<long>& ranges) {
    ranges.clear();
    std::vector<std::pair<size_t, size_t>> cover;  // (offset, count) of every block
    for (const Linear* l : p.linears()) {
        if (l->in % 64 || l->out % 64) {
            ranges.clear();
            return false;
        }
        cover.push_back({l->w, (size_t)l->in * l->out});
        cover.push_back({l->b, (size_t)l->out});
        ranges.push_back((long)l->b);
        ranges.push_back(l->out);
    }
    for (const Norm* n : p.norms()) {
        if (n->b != n->g + (size_t)n->n) {  // gains then shifts, contiguous
            ranges.clear();
            return false;
        }
        cover.push_back({n->g, 2 * (size_t)n->n});
        ranges.push_back((long)n->g);
        ranges.push_back(2L * n->n);
    }
    std::sort(cover.begin(), cover.end());
    size_t end = 0;
    for (const auto& c : cover) {
        if (c.first != end) {  // a gap (padding) or an overlap
            ranges.clear();
            return false;
        }
        end = c.first + c.second;
    }
    if (end != p.n32) ranges.clear();
    return end == p.n32;
}

// Where one logical parameter tensor lives in the fp32 master: `rows` rows of
// `cols` floats, row i at off + i * ld.  `lin` (if any) is the linear block
// whose working copies must be refreshed after a write.
struct ParamRef {
    size_t off = 0;
    int rows = 0, cols = 0, ld = 0;
    const Linear* lin = nullptr;
};

inline gp_status resolve_param(const ParamPlan& p, const Dims& d, int layer, int id, ParamRef& r,
                               std::string& msg) {
    const int D = d.D;
    auto mat = [&](const Linear& x, int c0, int c1) {
        if (!x.present) return false;
        r.off = x.w + c0;
        r.rows = x.in;
        r.cols = c1 - c0;
        r.ld = x.out;
        r.lin = &x;
        return true;
    };
    auto bias = [&](const Linear& x, int c0, int c1) {
        if (!x.present) return false;
        r.off = x.b + c0;
        r.rows = 1;
        r.cols = c1 - c0;
        r.ld = c1 - c0;
        r.lin = nullptr;
        return true;
    };
    auto vec = [&](const Norm& x, bool beta) {
        if (!x.present) return false;
        r.off = beta ? x.b : x.g;
        r.rows = 1;
        r.cols = x.n;
        r.ld = x.n;
        r.lin = nullptr;
        return true;
    };
    bool ok = false;
    if (layer == -1) {
        const HeadPlan& h = p.head;
        switch (id) {
        case GP_P_LNF_G: ok = vec(h.lnf, false); break;
        case GP_P_LNF_B: ok = vec(h.lnf, true); break;
        case GP_P_WOUT: ok = mat(h.out, 0, h.out.out); break;
        case GP_P_BOUT: ok = bias(h.out, 0, h.out.out); break;
        default: ok = false;
        }
    } else if (layer >= 0 && layer < (int)p.layers.size()) {
        const LayerPlan& l = p.layers[layer];
        switch (id) {
        case GP_P_LN1_G: ok = vec(l.ln1, false); break;
        case GP_P_LN1_B: ok = vec(l.ln1, true); break;
        case GP_P_WQ: ok = mat(l.qkv, 0, D); break;
        case GP_P_BQ: ok = bias(l.qkv, 0, D); break;
        case GP_P_WK: ok = mat(l.qkv, D, 2 * D); break;
        case GP_P_BK: ok = bias(l.qkv, D, 2 * D); break;
        case GP_P_WV: ok = mat(l.qkv, 2 * D, 3 * D); break;
        case GP_P_BV: ok = bias(l.qkv, 2 * D, 3 * D); break;
        case GP_P_WO: ok = mat(l.o, 0, D); break;
        case GP_P_BO: ok = bias(l.o, 0, D); break;
        case GP_P_LN2_G: ok = vec(l.ln2, false); break;
        case GP_P_LN2_B: ok = vec(l.ln2, true); break;
        case GP_P_W1: ok = mat(l.ffn1, 0, l.ffn1.out); break;
        case GP_P_B1: ok = bias(l.ffn1, 0, l.ffn1.out); break;
        case GP_P_W2: ok = mat(l.ffn2, 0, l.ffn2.out); break;
        case GP_P_B2: ok = bias(l.ffn2, 0, l.ffn2.out); break;
        case GP_P_XWQ: ok = mat(l.xq, 0, D); break;
        case GP_P_XBQ: ok = bias(l.xq, 0, D); break;
        case GP_P_XWK: ok = mat(l.xkv, 0, D); break;
        case GP_P_XBK: ok = bias(l.xkv, 0, D); break;
        case GP_P_XWV: ok = mat(l.xkv, D, 2 * D); break;
        case GP_P_XBV: ok = bias(l.xkv, D, 2 * D); break;
        case GP_P_XWO: ok = mat(l.xo, 0, D); break;
        case GP_P_XBO: ok = bias(l.xo, 0, D); break;
        case GP_P_LN3_G: ok = vec(l.ln3, false); break;
        case GP_P_LN3_B: ok = vec(l.ln3, true); break;
        default: ok = false;
        }
    } else {
        msg = "layer index out of range";
        return GP_ERR_INVALID_ARG;
    }
    if (!ok) {
        msg = "parameter id not present in this partition";
        return GP_ERR_INVALID_ARG;
    }
    return GP_OK;
}

// ------------------------------------------------------------ state machine
enum class Phase { Created, Idle, Forward, Backward, Ready };

class Sched {
  public:
    Phase phase = Phase::Created;
    int M = 0;
    int next_fwd = 0;
    int next_bwd = -1;

    gp_status configure(int m, std::string& msg) {
        if (phase != Phase::Created) { msg = "partition already configured"; return GP_ERR_STATE; }
        M = m;
        phase = Phase::Idle;
        next_fwd = 0;
        return GP_OK;
    }
    bool configured() const { return phase != Phase::Created; }
    // Parameters may change only between mini-batches.
    gp_status can_set_param(std::string& msg) const {
        if (phase == Phase::Created) { msg = "partition not configured"; return GP_ERR_STATE; }
        if (phase != Phase::Idle) { msg = "parameters may only change between mini-batches"; return GP_ERR_STATE; }
        return GP_OK;
    }
    gp_status can_forward(int mb, std::string& msg) const {
        if (phase == Phase::Created) { msg = "partition not configured"; return GP_ERR_STATE; }
        if (mb < 0 || mb >= M) { msg = "micro-batch index out of range"; return GP_ERR_INVALID_ARG; }
        if (phase != Phase::Idle && phase != Phase::Forward) { msg = "forward after the backward pass began"; return GP_ERR_STATE; }
        if (mb != next_fwd) { msg = "forward micro-batches must run in order 0..M-1"; return GP_ERR_STATE; }
        return GP_OK;
    }
    void did_forward() {
        ++next_fwd;
        phase = Phase::Forward;
        if (next_fwd == M) {
            phase = Phase::Backward;
            next_bwd = M - 1;
        }
    }
    gp_status can_backward(int mb, std::string& msg) const {
        if (phase == Phase::Created) { msg = "partition not configured"; return GP_ERR_STATE; }
        if (mb < 0 || mb >= M) { msg = "micro-batch index out of range"; return GP_ERR_INVALID_ARG; }
        if (phase != Phase::Backward) { msg = "backward needs all M forwards and precedes the step"; return GP_ERR_STATE; }
        if (mb != next_bwd) { msg = "backward micro-batches must run in order M-1..0"; return GP_ERR_STATE; }
        return GP_OK;
    }
    bool first_backward() const { return next_bwd == M - 1; }
    // micro-batch of the most recent backward of this mini-batch, or -1
    int last_backward() const {
        if (phase == Phase::Backward && next_bwd < M - 1) return next_bwd + 1;
        if (phase == Phase::Ready) return 0;
        return -1;
    }
    void did_backward() {
        --next_bwd;
        if (next_bwd < 0) phase = Phase::Ready;
    }
    gp_status can_step(std::string& msg) const {
        if (phase == Phase::Created) { msg = "partition not configured"; return GP_ERR_STATE; }
        if (phase != Phase::Ready) { msg = "step needs all M backward micro-batches"; return GP_ERR_STATE; }
        return GP_OK;
    }
    void did_step() {
        phase = Phase::Idle;
        next_fwd = 0;
        next_bwd = -1;
    }
};

} // namespace gp
