// attention_mfma.hip -- scaled dot-product attention on the matrix cores
// (bf16 operands, fp32 accumulation), head width 64, up to 256 keys.
//
// Forward: one wave owns 32 queries of one (sequence, head) and all keys.  It
// computes the transposed score block S^T = K Q^T with v_mfma_f32_32x32x16_bf16
// so that in the accumulator layout each lane holds one query's scores (lanes
// l and l + 32 split the keys between them).  The row softmax is therefore an
// in-register max/sum plus one cross-half exchange, and the probabilities,
// rounded to bf16, are already laid out as the B operand of the second
// product O^T = V^T P^T; no LDS round trip for P.  K and V^T of the
// (sequence, head) are staged once per workgroup in LDS.  The workgroup also
// writes the row log-sum-exp for the backward pass.
//
// Backward (two kernels, no atomics, deterministic):
//   dQ pass (per 32 queries, loop over key blocks):  S^T, dP^T = V dO^T,
//     dS^T = P^T (dP^T - delta), dQ^T += K^T dS^T;  also writes
//     delta_i = sum_d dO_id O_id.
//   dK/dV pass (per 32 keys, loop over query blocks):  S = Q K^T, dP = dO V^T,
//     dS = P (dP - delta), dV^T += dO^T P, dK^T += Q^T dS.
// In every product the register-held operand's accumulator layout (lane =
// column; register r = rows 8 (r/4) + 4 (lane/32) + r%4) is consumed as the
// B operand of the next product, whose A operand is read from LDS with the
// matching k order (two runs of four consecutive rows per lane).
#include "common.hpp"
#include "kernels.hpp"

namespace gp {

gp_status attention_fwd_simt(int dtype, const AttnArgs& a, hipStream_t st);
gp_status attention_bwd_simt(int dtype, const AttnArgs& a, hipStream_t st);

namespace {

constexpr int DH = 64;         // head width
constexpr int LDR = DH + 8;    // row stride (elements) of [row][d] LDS tiles
constexpr int MAXK = 256;      // keys / queries per (sequence, head)
constexpr int LDT = MAXK + 8;  // row stride of transposed [d][row] LDS tiles
constexpr float LOG2E = 1.4426950408889634f;

__device__ __forceinline__ f32x16 mfma(const bf16x8& a, const bf16x8& b, const f32x16& c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 zero16() {
    f32x16 z;
#pragma unroll
    for (int i = 0; i < 16; ++i) z[i] = 0.f;
    return z;
}

// Stage rows [0, nrows) x 64 of a head into LDS as [row][d] (row stride LDR).
__device__ __forceinline__ void stage_rows(bf16* __restrict__ s, const bf16* __restrict__ g, long ld, int nrows,
                                           int tid, int nthr) {
    for (int i = tid; i < nrows * (DH / 8); i += nthr) {
        const int r = i >> 3, c = (i & 7) * 8;
        *reinterpret_cast<bf16x8*>(s + r * LDR + c) = *reinterpret_cast<const bf16x8*>(g + (long)r * ld + c);
    }
}

// Stage rows [0, nrows) x 64 of a head into LDS transposed, as [d][row]
// (row stride LDT): each thread moves 4 rows x 8 features.
__device__ __forceinline__ void stage_rows_t(bf16* __restrict__ s, const bf16* __restrict__ g, long ld, int nrows,
                                             int tid, int nthr) {
    for (int i = tid; i < (nrows / 4) * (DH / 8); i += nthr) {
        const int r0 = (i >> 3) * 4, c0 = (i & 7) * 8;
        bf16x8 v[4];
#pragma unroll
        for (int q = 0; q < 4; ++q) v[q] = *reinterpret_cast<const bf16x8*>(g + (long)(r0 + q) * ld + c0);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            bf16x4 t = {v[0][e], v[1][e], v[2][e], v[3][e]};
            *reinterpret_cast<bf16x4*>(s + (c0 + e) * LDT + r0) = t;
        }
    }
}

// A operand from an [row][d] tile: rows row0 + lane%32, d = s*16 + 8*(lane/32) .. +8.
__device__ __forceinline__ bf16x8 frag_rows(const bf16* s, int row0, int kstep, int lane) {
    return *reinterpret_cast<const bf16x8*>(s + (row0 + (lane & 31)) * LDR + kstep * 16 + (lane >> 5) * 8);
}

// A operand from a transposed [d][row] tile, matching the k order of a
// register-held accumulator chunk: feature d = d0 + lane%32; rows
// base + 4*(lane/32) + {0..3} and base + 8 + 4*(lane/32) + {0..3}.
__device__ __forceinline__ bf16x8 frag_t(const bf16* s, int d0, int base, int lane) {
    const bf16* p = s + (d0 + (lane & 31)) * LDT + base + (lane >> 5) * 4;
    const bf16x4 lo = *reinterpret_cast<const bf16x4*>(p);
    const bf16x4 hi = *reinterpret_cast<const bf16x4*>(p + 8);
    bf16x8 r;
#pragma unroll
    for (int e = 0; e < 4; ++e) {
        r[e] = lo[e];
        r[4 + e] = hi[e];
    }
    return r;
}

// B operand from a global row of the head: row (lane%32 of the caller's
// block), features s*16 + 8*(lane/32) .. +8.
__device__ __forceinline__ bf16x8 frag_global(const bf16* row, int kstep, int lane) {
    return *reinterpret_cast<const bf16x8*>(row + kstep * 16 + (lane >> 5) * 8);
}

// Accumulator registers [8c, 8c + 8) of a 32x32 block, rounded to bf16 as a B operand.
__device__ __forceinline__ bf16x8 pack_chunk(const f32x16& v, int c) {
    bf16x8 r;
#pragma unroll
    for (int e = 0; e < 8; ++e) r[e] = (bf16)v[8 * c + e];
    return r;
}

// Row (within a 32-row block) held by accumulator register r of this lane.
__device__ __forceinline__ int acc_row(int r, int lane) { return (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3); }

// Write a transposed 64 x 32 accumulator pair (d x rows) as rows [row0 + lane%32][d]
// of a row-major [.., ld] bf16 tensor, scaled.
__device__ __forceinline__ void store_t(bf16* __restrict__ g, long ld, const f32x16* acc, float scale, int lane) {
    bf16* row = g + (long)(lane & 31) * ld;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int rg = 0; rg < 4; ++rg) {
            const int d = db * 32 + rg * 8 + (lane >> 5) * 4;
            bf16x4 t = {(bf16)(acc[db][rg * 4 + 0] * scale), (bf16)(acc[db][rg * 4 + 1] * scale),
                        (bf16)(acc[db][rg * 4 + 2] * scale), (bf16)(acc[db][rg * 4 + 3] * scale)};
            *reinterpret_cast<bf16x4*>(row + d) = t;
        }
}

constexpr int FWD_WAVES = 4;

template <int NKB>
__global__ void __launch_bounds__(256) attn_fwd_mfma(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) bf16 Ks[MAXK * LDR];
    __shared__ __attribute__((aligned(16))) bf16 Vt[DH * LDT];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bh = blockIdx.y, b = bh / a.H, hh = bh % a.H;
    const int Sk = NKB * 32;
    const bf16* K = reinterpret_cast<const bf16*>(a.k) + (long)b * a.Sk * a.ldk + hh * DH;
    const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)b * a.Sk * a.ldv + hh * DH;
    stage_rows(Ks, K, a.ldk, Sk, tid, 256);
    stage_rows_t(Vt, V, a.ldv, Sk, tid, 256);
    __syncthreads();
    const int q0 = (blockIdx.x * FWD_WAVES + wave) * 32;
    if (q0 >= a.Sq) return;
    const int q = q0 + (lane & 31);
    const bf16* Qrow = reinterpret_cast<const bf16*>(a.q) + ((long)b * a.Sq + q) * a.ldq + hh * DH;
    bf16x8 qf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) qf[s] = frag_global(Qrow, s, lane);
    const float c = a.scale * LOG2E;
    f32x16 sc[NKB];
    float m = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        sc[kb] = zero16();
        if (a.causal && kb * 32 > q0 + 31) {
#pragma unroll
            for (int r = 0; r < 16; ++r) sc[kb][r] = -INFINITY;
            continue;
        }
#pragma unroll
        for (int s = 0; s < 4; ++s) sc[kb] = mfma(frag_rows(Ks, kb * 32, s, lane), qf[s], sc[kb]);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float v = sc[kb][r] * c;
            if (a.causal && kb * 32 + acc_row(r, lane) > q) v = -INFINITY;
            sc[kb][r] = v;
            m = fmaxf(m, v);
        }
    }
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    float sum = 0.f;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float p = exp2f(sc[kb][r] - m);
            sc[kb][r] = p;
            sum += p;
        }
    sum += __shfl_xor(sum, 32, 64);
    f32x16 o[2] = {zero16(), zero16()};
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        if (a.causal && kb * 32 > q0 + 31) continue;
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            const bf16x8 pf = pack_chunk(sc[kb], cc);
#pragma unroll
            for (int db = 0; db < 2; ++db) o[db] = mfma(frag_t(Vt, db * 32, kb * 32 + cc * 16, lane), pf, o[db]);
        }
    }
    bf16* O = reinterpret_cast<bf16*>(a.o) + ((long)b * a.Sq + q0) * a.ldo + hh * DH;
    store_t(O, a.ldo, o, 1.f / sum, lane);
    if (a.lse && lane < 32) a.lse[(long)bh * a.Sq + q] = (m + log2f(sum)) / LOG2E;
}

constexpr int BWD_WAVES = 4;

template <int NKB>
__global__ void __launch_bounds__(256) attn_bwd_dq_mfma(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) bf16 Ks[MAXK * LDR];
    __shared__ __attribute__((aligned(16))) bf16 Vs[MAXK * LDR];
    __shared__ __attribute__((aligned(16))) bf16 Kt[DH * LDT];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bh = blockIdx.y, b = bh / a.H, hh = bh % a.H;
    const int Sk = NKB * 32;
    const bf16* K = reinterpret_cast<const bf16*>(a.k) + (long)b * a.Sk * a.ldk + hh * DH;
    const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)b * a.Sk * a.ldv + hh * DH;
    stage_rows(Ks, K, a.ldk, Sk, tid, 256);
    stage_rows(Vs, V, a.ldv, Sk, tid, 256);
    stage_rows_t(Kt, K, a.ldk, Sk, tid, 256);
    __syncthreads();
    const int q0 = (blockIdx.x * BWD_WAVES + wave) * 32;
    if (q0 >= a.Sq) return;
    const int q = q0 + (lane & 31);
    const long qrow = (long)b * a.Sq + q;
    const bf16* Qrow = reinterpret_cast<const bf16*>(a.q) + qrow * a.ldq + hh * DH;
    const bf16* dOrow = reinterpret_cast<const bf16*>(a.dout) + qrow * a.lddo + hh * DH;
    const bf16* Orow = reinterpret_cast<const bf16*>(a.o) + qrow * a.ldo + hh * DH;
    bf16x8 qf[4], gf[4];
    float dpart = 0.f;
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        qf[s] = frag_global(Qrow, s, lane);
        gf[s] = frag_global(dOrow, s, lane);
        const bf16x8 of = frag_global(Orow, s, lane);
#pragma unroll
        for (int e = 0; e < 8; ++e) dpart += (float)gf[s][e] * (float)of[e];
    }
    const float delta = dpart + __shfl_xor(dpart, 32, 64);
    const float c = a.scale * LOG2E;
    const float lse2 = a.lse[(long)bh * a.Sq + q] * LOG2E;
    f32x16 dq[2] = {zero16(), zero16()};
#pragma unroll 2
    for (int kb = 0; kb < NKB; ++kb) {
        if (a.causal && kb * 32 > q0 + 31) break;
        f32x16 st = zero16(), dp = zero16();
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            st = mfma(frag_rows(Ks, kb * 32, s, lane), qf[s], st);
            dp = mfma(frag_rows(Vs, kb * 32, s, lane), gf[s], dp);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float p = exp2f(st[r] * c - lse2);
            if (a.causal && kb * 32 + acc_row(r, lane) > q) p = 0.f;
            st[r] = p * (dp[r] - delta);
        }
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            const bf16x8 df = pack_chunk(st, cc);
#pragma unroll
            for (int db = 0; db < 2; ++db) dq[db] = mfma(frag_t(Kt, db * 32, kb * 32 + cc * 16, lane), df, dq[db]);
        }
    }
    bf16* dQ = reinterpret_cast<bf16*>(a.dq) + ((long)b * a.Sq + q0) * a.lddq + hh * DH;
    store_t(dQ, a.lddq, dq, a.scale, lane);
    if (lane < 32) a.delta[(long)bh * a.Sq + q] = delta;
}

template <int NQB>
__global__ void __launch_bounds__(256) attn_bwd_dkv_mfma(AttnArgs a) {
    __shared__ __attribute__((aligned(16))) bf16 Qs[MAXK * LDR];
    __shared__ __attribute__((aligned(16))) bf16 Gs[MAXK * LDR];
    __shared__ __attribute__((aligned(16))) bf16 Qt[DH * LDT];
    __shared__ __attribute__((aligned(16))) bf16 Gt[DH * LDT];
    __shared__ float lse2s[MAXK], dls[MAXK];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int bh = blockIdx.y, b = bh / a.H, hh = bh % a.H;
    const int Sq = NQB * 32;
    const bf16* Q = reinterpret_cast<const bf16*>(a.q) + (long)b * a.Sq * a.ldq + hh * DH;
    const bf16* G = reinterpret_cast<const bf16*>(a.dout) + (long)b * a.Sq * a.lddo + hh * DH;
    stage_rows(Qs, Q, a.ldq, Sq, tid, 256);
    stage_rows(Gs, G, a.lddo, Sq, tid, 256);
    stage_rows_t(Qt, Q, a.ldq, Sq, tid, 256);
    stage_rows_t(Gt, G, a.lddo, Sq, tid, 256);
    for (int i = tid; i < Sq; i += 256) {
        lse2s[i] = a.lse[(long)bh * a.Sq + i] * LOG2E;
        dls[i] = a.delta[(long)bh * a.Sq + i];
    }
    __syncthreads();
    const int k0 = (blockIdx.x * BWD_WAVES + wave) * 32;
    if (k0 >= a.Sk) return;
    const int key = k0 + (lane & 31);
    const long krow = (long)b * a.Sk + key;
    const bf16* Krow = reinterpret_cast<const bf16*>(a.k) + krow * a.ldk + hh * DH;
    const bf16* Vrow = reinterpret_cast<const bf16*>(a.v) + krow * a.ldv + hh * DH;
    bf16x8 kf[4], vf[4];
#pragma unroll
    for (int s = 0; s < 4; ++s) {
        kf[s] = frag_global(Krow, s, lane);
        vf[s] = frag_global(Vrow, s, lane);
    }
    const float c = a.scale * LOG2E;
    f32x16 dk[2] = {zero16(), zero16()}, dv[2] = {zero16(), zero16()};
    const int qb0 = a.causal ? k0 / 32 : 0;
    for (int qb = qb0; qb < NQB; ++qb) {
        f32x16 st = zero16(), dp = zero16();
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            st = mfma(frag_rows(Qs, qb * 32, s, lane), kf[s], st);
            dp = mfma(frag_rows(Gs, qb * 32, s, lane), vf[s], dp);
        }
        f32x16 pm;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int qi = qb * 32 + acc_row(r, lane);
            float p = exp2f(st[r] * c - lse2s[qi]);
            if (a.causal && key > qi) p = 0.f;
            pm[r] = p;
            st[r] = p * (dp[r] - dls[qi]);
        }
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            const bf16x8 pf = pack_chunk(pm, cc);
            const bf16x8 df = pack_chunk(st, cc);
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                dv[db] = mfma(frag_t(Gt, db * 32, qb * 32 + cc * 16, lane), pf, dv[db]);
                dk[db] = mfma(frag_t(Qt, db * 32, qb * 32 + cc * 16, lane), df, dk[db]);
            }
        }
    }
    bf16* dK = reinterpret_cast<bf16*>(a.dk) + ((long)b * a.Sk + k0) * a.lddk + hh * DH;
    bf16* dV = reinterpret_cast<bf16*>(a.dv) + ((long)b * a.Sk + k0) * a.lddv + hh * DH;
    store_t(dK, a.lddk, dk, a.scale, lane);
    store_t(dV, a.lddv, dv, 1.f, lane);
}

#define GP_NB_SWITCH(NB, KERNEL, GRID)                                              \
    switch (NB) {                                                                   \
    case 1: klaunch(KERNEL<1>, GRID, 256, 0, st, a); break;                              \
    case 2: klaunch(KERNEL<2>, GRID, 256, 0, st, a); break;                              \
    case 3: klaunch(KERNEL<3>, GRID, 256, 0, st, a); break;                              \
    case 4: klaunch(KERNEL<4>, GRID, 256, 0, st, a); break;                              \
    case 5: klaunch(KERNEL<5>, GRID, 256, 0, st, a); break;                              \
    case 6: klaunch(KERNEL<6>, GRID, 256, 0, st, a); break;                              \
    case 7: klaunch(KERNEL<7>, GRID, 256, 0, st, a); break;                              \
    case 8: klaunch(KERNEL<8>, GRID, 256, 0, st, a); break;                              \
    default: return set_error(GP_ERR_UNSUPPORTED, "attention: sequence length > 256"); \
    }

bool mfma_ok(const AttnArgs& a) {
    return a.dh == DH && a.Sq % 32 == 0 && a.Sk % 32 == 0 && a.Sq <= MAXK && a.Sk <= MAXK &&
           a.ldq % 8 == 0 && a.ldk % 8 == 0 && a.ldv % 8 == 0 && a.ldo % 8 == 0;
}

} // namespace

gp_status attention_fwd(int dtype, const AttnArgs& a, hipStream_t st) {
    if (dtype != GP_BF16) return attention_fwd_simt(dtype, a, st);
    if (!mfma_ok(a)) return set_error(GP_ERR_UNSUPPORTED, "bf16 attention needs d_h = 64 and lengths multiple of 32, <= 256");
    dim3 grid((a.Sq + 32 * FWD_WAVES - 1) / (32 * FWD_WAVES), a.n * a.H);
    GP_NB_SWITCH(a.Sk / 32, attn_fwd_mfma, grid);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status attention_bwd(int dtype, const AttnArgs& a, hipStream_t st) {
    if (dtype != GP_BF16) return attention_bwd_simt(dtype, a, st);
    if (!mfma_ok(a)) return set_error(GP_ERR_UNSUPPORTED, "bf16 attention needs d_h = 64 and lengths multiple of 32, <= 256");
    dim3 gq((a.Sq + 32 * BWD_WAVES - 1) / (32 * BWD_WAVES), a.n * a.H);
    GP_NB_SWITCH(a.Sk / 32, attn_bwd_dq_mfma, gq);
    GP_LAUNCH_CHECK();
    dim3 gk((a.Sk + 32 * BWD_WAVES - 1) / (32 * BWD_WAVES), a.n * a.H);
    GP_NB_SWITCH(a.Sq / 32, attn_bwd_dkv_mfma, gk);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

} // namespace gp
