// kernels.hpp -- host-side launchers of the partition's HIP kernels.  All
// launchers enqueue on the given stream and return gp_status (launch errors
// only; device faults surface at the next synchronising call).
#pragma once

#include <hip/hip_runtime.h>
#include "../../include/gp.h"

namespace gp {

// ------------------------------------------------------------------ GEMM
enum {
    EPI_STORE = 0,     // C (elt) = act(acc + bias), act = ReLU when relu != 0
    EPI_RES_F32 = 1,   // C (f32) = aux (f32 residual) + acc + bias; C2 (elt, optional) = same, rounded
    EPI_F32 = 2,       // C (f32) = acc
    EPI_RELU_MASK = 3, // C (elt) = acc * [aux (elt) > 0]
    EPI_ACC_F32 = 4    // C (f32) = (accumulate ? C : 0) + acc
};

struct GemmArgs {
    int M = 0, N = 0, K = 0;
    const void* A = nullptr; long lda = 0; // element (m,k): k-major A[m lda + k], else A[k lda + m]
    const void* B = nullptr; long ldb = 0; // element (n,k): k-major B[n ldb + k], else B[k ldb + n]
    void* C = nullptr; long ldc = 0;
    void* C2 = nullptr; long ldc2 = 0;
    const float* bias = nullptr;
    const void* aux = nullptr; long ldaux = 0;
    int relu = 0;
    int accumulate = 0;
    float* ws = nullptr;   // split-K partials (fp32), ws_elems floats; nullptr disables split-K
    long ws_elems = 0;
    int force_cfg = -1;    // tile shape override (tests and tuning); -1 = heuristic
    int force_splits = 0;
    float* colsum = nullptr; // EPI_ACC_F32 with n-contiguous B: also colsum[n] (+)= sum_k B(n, k)
    // Optional fp4 correction term (bf16, k-contiguous, EPI_STORE): the GEMM
    // also adds sum_k a4(m, k) sa4[m] * b4(n, k) sb4[n].  a4 [M, K/2] and b4
    // [N, K/2] hold OCP e2m1 values (element k of a row in byte k/2, low
    // nibble first); sa4 [M] and sb4 [N] are E8M0 scales (2^(s - 127)).
    const void* a4 = nullptr;
    const void* b4 = nullptr;
    const unsigned char* sa4 = nullptr;
    const unsigned char* sb4 = nullptr;
    // EPI_RES_F32 and EPI_F32 only: when set, a split-K launch leaves its
    // partials in ws [splits][M][N] and stores the split count here instead of
    // running the reduce (the caller then reduces, e.g. fused with the next
    // LayerNorm); 1 when the GEMM completed its own epilogue.
    int* deferred = nullptr;
    // > 0: choose the tile shape and split count as for a problem of this many
    // rows (M) -- the problem one micro-batch poses -- and run them on the M
    // rows given.  Split-K changes each element's summation order, so a pass
    // over two micro-batches' rows then rounds exactly as two single passes
    // (the tile shape does not change any element's order).  ws must hold the
    // partials of the M rows.
    int split_rows = 0;
    // A and B hold fp16 values instead of bf16 (EPI_STORE, k-contiguous, no
    // fp4 term); the tile and split choice is the bf16 one
    int f16 = 0;
};

gp_status gemm(const GemmArgs& a, int epi, bool a_kmajor, bool b_kmajor, int dtype, hipStream_t st);
// Floats of a.ws that gemm() with these arguments writes (its split-K partial
// tiles and column-sum rows); 0 when it runs unsplit.  Host arithmetic only.
long gemm_workspace_need(const GemmArgs& a, int epi, bool a_kmajor, int dtype);
// The split-K reduce and epilogue of a bf16 GEMM whose partials are in a.ws.
gp_status gemm_reduce(const GemmArgs& a, int epi, int splits, hipStream_t st);

// ------------------------------------------------------------- LayerNorm
// out (elt) = gamma * (x - mu) * rstd + beta per row of D; stats[row] = {mu, rstd}.
// lo4 / lo_sc (optional; bf16, D % 64 == 0): the rounding residuals y - bf16(y)
// of the row as fp4 [rows, D/2] bytes with one E8M0 scale per row, the
// correction operand (GemmArgs::a4) of the GEMM that consumes out.
// out16 (optional; bf16, D % 256 == 0, D <= 2048): out also in fp16, the A
// operand of a GEMM with fp16 operands (GemmArgs::f16).
gp_status layernorm_fwd(int dtype, const float* x, long rows, int D, const float* gamma, const float* beta,
                        float eps, void* out, float* stats, void* lo4, unsigned char* lo_sc, hipStream_t st,
                        void* out16 = nullptr);
// The split-K reduce of a residual GEMM fused with the LayerNorm of its result:
// x = sum over s < splits of ws[s plane + row D + col], plus (res + bias), in
// the order of the GEMM's own reduce, is stored in xo (fp32) and xc (bf16, when
// not null), then normalised as layernorm_fwd does.  Rows of D contiguous;
// bf16 out, D % 256 == 0, D <= 2048, 16-byte aligned pointers
// (layernorm_fwd_res_ok); GP_ERR_UNSUPPORTED otherwise.
bool layernorm_fwd_res_ok(int dtype, int D, const void* ws, const float* bias, const float* res, const float* xo,
                          const void* xc);
gp_status layernorm_fwd_res(int dtype, const float* ws, int splits, long plane, const float* bias, const float* res,
                            float* xo, void* xc, long rows, int D, const float* gamma, const float* beta, float eps,
                            void* out, float* stats, void* lo4, unsigned char* lo_sc, hipStream_t st,
                            void* out16 = nullptr);
// dx = dres + rstd (g - mean g - xh mean(g xh)), g = dn * gamma; writes dx_f32 and/or dx_elt.
// Per-block partial sums of dn * xh and dn go to partial[blk][2][D] (added to
// what is there when accumulate != 0); *nblk receives the block count (for
// colsum_finalize over width 2 D).  The block count depends on rows only.
// dn_splits > 1 (D % 256 == 0, D <= 2048): dn holds that many split-K
// partial planes dn_plane floats apart, summed in plane order (the fused
// reduce of the GEMM that produced dn).
gp_status layernorm_bwd(int dtype, const float* dn, const float* x, const float* stats, const float* gamma,
                        long rows, int D, const float* dres, float* dx_f32, void* dx_elt, float* partial,
                        int accumulate, int* nblk, hipStream_t st, int dn_splits = 1, long dn_plane = 0);
// Blocks (rows of the partial buffer) layernorm_bwd uses for `rows` rows.
int layernorm_bwd_blocks(long rows);

// out[c] = (accumulate ? out[c] : 0) + sum_b partial[b * width + c]
gp_status colsum_finalize(const float* partial, int nblk, int width, float* out, int accumulate, hipStream_t st);

// ------------------------------------------------------------- attention
struct AttnArgs {
    int n = 0, H = 0, Sq = 0, Sk = 0, dh = 0;
    const void* q = nullptr; long ldq = 0; // row (b, i) of head h at q + (b Sq + i) ldq + h dh
    const void* k = nullptr; long ldk = 0; // row (b, j) at k + (b Sk + j) ldk + h dh
    const void* v = nullptr; long ldv = 0;
    void* o = nullptr; long ldo = 0;
    float* lse = nullptr;                  // [n, H, Sq] log-sum-exp of the scaled scores
    int causal = 0;
    float scale = 1.f;
    const void* dout = nullptr; long lddo = 0;
    void* dq = nullptr; long lddq = 0;
    void* dk = nullptr; long lddk = 0;
    void* dv = nullptr; long lddv = 0;
    float* delta = nullptr;                // [n, H, Sq] rowsum(dO * O) = rowsum(P * dP) scratch
    int split = 1;                         // allow the two-wave (half-loop) kernels where they apply
    int waves = 0;                         // waves (32-row blocks) per workgroup: 1, 2 or 4; 0 = by grid size
    int hint_n = 0;                        // > 0: choose the kernel variant as for this many sequences
                                           // (one micro-batch), so that a pass over two rounds alike
};
gp_status attention_fwd(int dtype, const AttnArgs& a, hipStream_t st);
gp_status attention_bwd(int dtype, const AttnArgs& a, hipStream_t st);

// ----------------------------------------------------------- elementwise
// x32 = float(src); stash (optional) = src.  count elements.
gp_status intake(int dtype, const void* src, void* stash, float* x32, long count, hipStream_t st);
// dst (elt) = src (f32) rounded.
gp_status cast_out(int dtype, const float* src, void* dst, long count, hipStream_t st);
// d = y - t; d32 = 2 d / norm; delt = rounded d32; partial[blk] = sum d^2 / norm (fp64)
gp_status mse_grad(int dtype, const float* y, const void* target, long count, double norm, float* d32,
                   void* delt, double* partial, int* nblk, hipStream_t st);
int loss_blocks();
// acc[0] = (accumulate ? acc[0] : 0) + sum_b partial[b]
gp_status loss_finalize(const double* partial, int nblk, double* acc, int accumulate, hipStream_t st);

// Label-smoothed softmax cross-entropy over rows of V logits (f32 or elt in
// z, overwritten by dZ in the elt type): dZ = (softmax(z) - q) / norm,
// partial[row] = -sum q log p / norm in fp64.  A label outside [0, V) is read
// as 0 and sets bad_label[0] = 1.  clip > 0: the logits are clipped to
// [-clip, clip] first, and dZ is zero where |z| > clip.
gp_status xent_ls(int dtype, void* z, long rows, int V, const int* labels, float ls, float clip, double norm,
                  double* partial, int* bad_label, hipStream_t st);
int xent_partials(long rows);

// --------------------------------------------------------------- update
// w[i] -= lr * g[i] for i < count (fp32 masters).
// Sustained bf16 MFMA rate of a register-only 32x32x16 loop on every CU
// (best of three timed runs after one warm-up), in TFLOP/s; synchronises st.
gp_status mfma_peak(hipStream_t st, double* tflops);
gp_status sgd_update(float* w, const float* g, float lr, long count, hipStream_t st);
// ms = rho ms + (1 - rho) g^2;  w -= lr g / sqrt(ms + eps)  (count % 4 == 0, 16-byte aligned).
gp_status rmsprop_update(float* w, const float* g, float* ms, float lr, float rho, float eps, long count,
                         hipStream_t st);
// Working copies of one linear layer from its fp32 master W [in, out], in the
// partition dtype: kn = W [in, out], nk = W^T [out, in].  q4 / q4s (optional,
// bf16): the rows of nk in fp4 [out, in/2] bytes with one E8M0 scale per row
// (GemmArgs::b4, sb4).  nk16 (bf16, in and out multiples of 64): nk in fp16
// instead (the B operand of a GEMM with fp16 operands, GemmArgs::f16).
gp_status refresh_linear(int dtype, const float* w, int in, int out, void* kn, void* nk, void* q4, void* q4s,
                         hipStream_t st, bool nk16 = false);
// The SGD (ms == nullptr) or RMSProp step of a linear's fp32 weights fused
// with the refresh of its bf16 working copies as refresh_linear makes them;
// in, out multiples of 64.
gp_status update_refresh_linear(float* w, const float* g, float* ms, float lr, float rho, float eps, int in,
                                int out, void* kn, void* nk, void* q4, void* q4s, hipStream_t st, bool nk16 = false);
// The same update over nranges float ranges (offset, count pairs in device
// memory), one workgroup each.
gp_status update_ranges(float* w, const float* g, float* ms, float lr, float rho, float eps, const long* ranges,
                        int nranges, hipStream_t st);
// An empty launch labelled by its grid (role x (edge + 1) workgroups of one
// wave): edge 0 before, 1 after a timed launch, so that per-dispatch profiler
// records can be attributed to launch roles.
gp_status role_marker(int role, int edge, hipStream_t st);
// Fill bytes [p, p + bytes) with 0xFF (NaN in every floating type); test mode only.
gp_status poison_fill(void* p, size_t bytes, hipStream_t st);
// flag[0] = 1 if any of x[0..count) is not finite (flag must be zeroed first).
gp_status finite_check(const float* x, long count, int* flag, hipStream_t st);

} // namespace gp
