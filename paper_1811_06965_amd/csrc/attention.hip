// attention.hip -- multi-head scaled dot-product attention, forward and
// backward, for fp32 partitions (and any head width <= 64 / length <= 1024).
//
// A = softmax(Q K^T s + mask), O = A V per (sequence, head), s = 1/sqrt(d_h);
// the causal mask removes keys j > i.  One wave owns one query row (forward,
// dQ) or one key row (dK, dV); the row's scores live in LDS and the wave
// reduces max and sum across its 64 lanes.  The backward is split into a
// query-row pass (dQ, and delta_i = rowsum(dO_i O_i)) and a key-row pass (dK,
// dV) so that no two waves ever add into the same output: results are
// deterministic and the re-materialised forward reproduces the first pass.
//
// bf16 partitions use the MFMA kernels in attention_mfma.hip.
#include "common.hpp"
#include "kernels.hpp"

namespace gp {

namespace {

constexpr int AW = 4;       // waves (rows) per block
constexpr int MAXS = 1024;  // longest key / query row held in LDS

// Each wave uses only its own LDS rows, so a wave-local ordering point is all
// the synchronisation needed: wait for the wave's LDS traffic and keep the
// compiler from moving memory operations across it.
__device__ __forceinline__ void wave_lds_sync() {
    __builtin_amdgcn_s_waitcnt(0);
    __builtin_amdgcn_wave_barrier();
}

template <typename T>
__device__ __forceinline__ float dot_row(const float* __restrict__ a_lds, const T* __restrict__ b, int dh) {
    float s = 0.f;
    for (int d = 0; d < dh; ++d) s += a_lds[d] * to_f32(b[d]);
    return s;
}

template <typename T>
__global__ void __launch_bounds__(256) attn_fwd_simt(AttnArgs a) {
    __shared__ float qs[AW][64];
    __shared__ float ps[AW][MAXS];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const long r = (long)blockIdx.x * AW + w;
    if (r >= (long)a.n * a.H * a.Sq) return;
    const int i = (int)(r % a.Sq), h = (int)((r / a.Sq) % a.H), b = (int)(r / ((long)a.Sq * a.H));
    const T* Q = reinterpret_cast<const T*>(a.q) + ((long)b * a.Sq + i) * a.ldq + h * a.dh;
    const T* K = reinterpret_cast<const T*>(a.k) + (long)b * a.Sk * a.ldk + h * a.dh;
    const T* V = reinterpret_cast<const T*>(a.v) + (long)b * a.Sk * a.ldv + h * a.dh;
    if (lane < a.dh) qs[w][lane] = to_f32(Q[lane]);
    wave_lds_sync();
    const int jmax = a.causal ? i + 1 : a.Sk;
    float m = -INFINITY;
    for (int j = lane; j < jmax; j += 64) {
        const float s = a.scale * dot_row(qs[w], K + (long)j * a.ldk, a.dh);
        ps[w][j] = s;
        m = fmaxf(m, s);
    }
    m = wave_max(m);
    float sum = 0.f;
    for (int j = lane; j < jmax; j += 64) {
        const float e = expf(ps[w][j] - m);
        ps[w][j] = e;
        sum += e;
    }
    sum = wave_sum(sum);
    wave_lds_sync();
    if (lane < a.dh) {
        float o = 0.f;
        for (int j = 0; j < jmax; ++j) o += ps[w][j] * to_f32(V[(long)j * a.ldv + lane]);
        T* O = reinterpret_cast<T*>(a.o) + ((long)b * a.Sq + i) * a.ldo + h * a.dh;
        O[lane] = to_elt<T>(o / sum);
    }
    if (a.lse && lane == 0) a.lse[r] = m + logf(sum);
}

// dQ pass: one wave per query row i.
template <typename T>
__global__ void __launch_bounds__(256) attn_bwd_dq_simt(AttnArgs a) {
    __shared__ float qs[AW][64], dos[AW][64];
    __shared__ float ds_[AW][MAXS];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const long r = (long)blockIdx.x * AW + w;
    const bool live = r < (long)a.n * a.H * a.Sq;
    const long rr = live ? r : 0;
    const int i = (int)(rr % a.Sq), h = (int)((rr / a.Sq) % a.H), b = (int)(rr / ((long)a.Sq * a.H));
    const long qrow = (long)b * a.Sq + i;
    const T* Q = reinterpret_cast<const T*>(a.q) + qrow * a.ldq + h * a.dh;
    const T* O = reinterpret_cast<const T*>(a.o) + qrow * a.ldo + h * a.dh;
    const T* dO = reinterpret_cast<const T*>(a.dout) + qrow * a.lddo + h * a.dh;
    const T* K = reinterpret_cast<const T*>(a.k) + (long)b * a.Sk * a.ldk + h * a.dh;
    const T* V = reinterpret_cast<const T*>(a.v) + (long)b * a.Sk * a.ldv + h * a.dh;
    float od = 0.f;
    if (lane < a.dh) {
        qs[w][lane] = to_f32(Q[lane]);
        const float g = to_f32(dO[lane]);
        dos[w][lane] = g;
        od = g * to_f32(O[lane]);
    }
    const float Di = wave_sum(od);
    wave_lds_sync();
    if (!live) return;
    const float lse = a.lse[rr];
    const int jmax = a.causal ? i + 1 : a.Sk;
    for (int j = lane; j < jmax; j += 64) {
        const float p = expf(a.scale * dot_row(qs[w], K + (long)j * a.ldk, a.dh) - lse);
        const float dp = dot_row(dos[w], V + (long)j * a.ldv, a.dh);
        ds_[w][j] = p * (dp - Di);
    }
    wave_lds_sync();
    if (lane < a.dh) {
        float g = 0.f;
        for (int j = 0; j < jmax; ++j) g += ds_[w][j] * to_f32(K[(long)j * a.ldk + lane]);
        T* dQ = reinterpret_cast<T*>(a.dq) + qrow * a.lddq + h * a.dh;
        dQ[lane] = to_elt<T>(a.scale * g);
    }
    if (lane == 0) a.delta[rr] = Di;
}

// dK, dV pass: one wave per key row j.
template <typename T>
__global__ void __launch_bounds__(256) attn_bwd_dkv_simt(AttnArgs a) {
    __shared__ float ks[AW][64], vs[AW][64];
    __shared__ float ps[AW][MAXS], ds_[AW][MAXS];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const long r = (long)blockIdx.x * AW + w;
    const bool live = r < (long)a.n * a.H * a.Sk;
    const long rr = live ? r : 0;
    const int j = (int)(rr % a.Sk), h = (int)((rr / a.Sk) % a.H), b = (int)(rr / ((long)a.Sk * a.H));
    const long krow = (long)b * a.Sk + j;
    const T* K = reinterpret_cast<const T*>(a.k) + krow * a.ldk + h * a.dh;
    const T* V = reinterpret_cast<const T*>(a.v) + krow * a.ldv + h * a.dh;
    const T* Q = reinterpret_cast<const T*>(a.q) + (long)b * a.Sq * a.ldq + h * a.dh;
    const T* dO = reinterpret_cast<const T*>(a.dout) + (long)b * a.Sq * a.lddo + h * a.dh;
    if (lane < a.dh) {
        ks[w][lane] = to_f32(K[lane]);
        vs[w][lane] = to_f32(V[lane]);
    }
    wave_lds_sync();
    if (!live) return;
    const float* lse = a.lse + ((long)b * a.H + h) * a.Sq;
    const float* delta = a.delta + ((long)b * a.H + h) * a.Sq;
    const int i0 = a.causal ? j : 0;
    for (int i = i0 + lane; i < a.Sq; i += 64) {
        const float p = expf(a.scale * dot_row(ks[w], Q + (long)i * a.ldq, a.dh) - lse[i]);
        const float dp = dot_row(vs[w], dO + (long)i * a.lddo, a.dh);
        ps[w][i] = p;
        ds_[w][i] = p * (dp - delta[i]);
    }
    wave_lds_sync();
    if (lane < a.dh) {
        float gv = 0.f, gk = 0.f;
        for (int i = i0; i < a.Sq; ++i) {
            gv += ps[w][i] * to_f32(dO[(long)i * a.lddo + lane]);
            gk += ds_[w][i] * to_f32(Q[(long)i * a.ldq + lane]);
        }
        T* dV = reinterpret_cast<T*>(a.dv) + krow * a.lddv + h * a.dh;
        T* dK = reinterpret_cast<T*>(a.dk) + krow * a.lddk + h * a.dh;
        dV[lane] = to_elt<T>(gv);
        dK[lane] = to_elt<T>(a.scale * gk);
    }
}

template <typename T>
gp_status fwd_t(const AttnArgs& a, hipStream_t st) {
    const long rows = (long)a.n * a.H * a.Sq;
    klaunch(attn_fwd_simt<T>, (unsigned)((rows + AW - 1) / AW), 256, 0, st, a);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

template <typename T>
gp_status bwd_t(const AttnArgs& a, hipStream_t st) {
    const long qrows = (long)a.n * a.H * a.Sq, krows = (long)a.n * a.H * a.Sk;
    klaunch(attn_bwd_dq_simt<T>, (unsigned)((qrows + AW - 1) / AW), 256, 0, st, a);
    GP_LAUNCH_CHECK();
    klaunch(attn_bwd_dkv_simt<T>, (unsigned)((krows + AW - 1) / AW), 256, 0, st, a);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

} // namespace

gp_status attention_fwd_simt(int dtype, const AttnArgs& a, hipStream_t st) {
    if (a.dh > 64 || a.Sk > MAXS || a.Sq > MAXS) return set_error(GP_ERR_UNSUPPORTED, "attention: d_h <= 64 and S <= 1024");
    if (dtype == GP_BF16) return fwd_t<bf16>(a, st);
    return fwd_t<float>(a, st);
}

gp_status attention_bwd_simt(int dtype, const AttnArgs& a, hipStream_t st) {
    if (a.dh > 64 || a.Sk > MAXS || a.Sq > MAXS) return set_error(GP_ERR_UNSUPPORTED, "attention: d_h <= 64 and S <= 1024");
    if (dtype == GP_BF16) return bwd_t<bf16>(a, st);
    return bwd_t<float>(a, st);
}

} // namespace gp
