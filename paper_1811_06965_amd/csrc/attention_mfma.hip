// attention_mfma.hip -- scaled dot-product attention on the matrix cores
// (bf16 operands, fp32 accumulation), head width 64, up to 256 keys.
//
// Forward: one wave owns 32 queries of one (sequence, head) and all keys.  It
// computes the transposed score block S^T = K Q^T with v_mfma_f32_32x32x16_bf16
// so that in the accumulator layout each lane holds one query's scores (lanes
// l and l + 32 split the keys between them).  The row softmax is therefore an
// in-register max/sum plus one cross-half exchange, and the probabilities,
// rounded to bf16, are already laid out as the B operand of the second
// product O^T = V^T P^T; no LDS round trip for P.  K and V of the (sequence,
// head) are staged row-major once per workgroup in LDS; V^T fragments come
// from transposing LDS reads (ds_read_b64_tr_b16).  The workgroup also writes
// the row log-sum-exp for the backward pass.
//
// Backward (two kernels, no atomics, deterministic):
//   dQ pass (per 32 queries, two loops over key blocks): first
//     delta_i = sum_j P_ij dP_ij from the recomputed S^T and dP^T = V dO^T,
//     then S^T, dP^T again, dS^T = P^T (dP^T - delta), dQ^T += K^T dS^T;
//     writes delta for the second kernel.
// delta is formed from the very probabilities and dP the backward uses, not
// as dO . O: the forward's O comes from bf16-rounded probabilities (and is
// stored in bf16), and any mismatch leaves the rows of dS summing to a
// nonzero value.  A component that all keys (and queries) of a head share --
// it grows with depth in a residual stack -- multiplies that sum coherently
// over the keys in dQ = dS K and in the bias and weight gradients built from
// dQ and dK (several percent of dQ in a 16-layer stack with delta = dO . O).
//   dK/dV pass (per 32 keys, loop over query blocks):  S = Q K^T, dP = dO V^T,
//     dS = P (dP - delta), dV^T += dO^T P, dK^T += Q^T dS.
// In every product the register-held operand's accumulator layout (lane =
// column; register r = rows 8 (r/4) + 4 (lane/32) + r%4) is consumed as the
// B operand of the next product, whose A operand (K^T, Q^T, dO^T) is read
// transposed from the row-major LDS tile with the matching k order (two runs
// of four consecutive rows per lane).  A workgroup holds 1, 2 or 4 waves,
// chosen so that small micro-batches still launch enough workgroups.
#include "common.hpp"
#include "kernels.hpp"

namespace gp {

gp_status attention_fwd_simt(int dtype, const AttnArgs& a, hipStream_t st);
gp_status attention_bwd_simt(int dtype, const AttnArgs& a, hipStream_t st);

namespace {

constexpr int DH = 64;         // head width
constexpr int MAXK = 256;      // keys / queries per (sequence, head)
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

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16* LdsV4;

// LDS tiles hold rows of 64 features (128 bytes) without padding; the
// 16-byte chunk c of row r is stored at chunk position c ^ swz(r).  With this
// swizzle both access patterns are free of bank conflicts: 16 lanes reading
// the same chunk of 16 consecutive rows (row fragments), and a half-wave
// reading four consecutive chunks of 4 consecutive rows (transposing reads).
__device__ __forceinline__ int swz(int r) { return (((r >> 1) & 1) << 2) | ((r >> 2) & 3); }
__device__ __forceinline__ int lds_off(int r, int col) { return r * 128 + (((col >> 3) ^ swz(r)) << 4) + (col & 7) * 2; }

typedef __amdgpu_buffer_rsrc_t Rsrc;
typedef __attribute__((address_space(3))) void* LdsPtr;

// Stage NROWS rows x 64 features of a head (rows ld elements apart, base g)
// into the LDS tile s with direct-to-LDS buffer loads: each wave instruction
// fills 8 rows (1 KB) and each lane fetches the global chunk that belongs at
// its swizzled LDS position.  All loads are issued back to back; the caller
// waits (vmcnt 0) and synchronises before reading.
template <int NROWS, int NW>
__device__ __forceinline__ void stage_dl(char* s, const bf16* g, long ld, int wave, int lane) {
    static_assert(NROWS % (8 * NW) == 0, "staging split");
    constexpr int P = NROWS / (8 * NW);
    const Rsrc rs = __builtin_amdgcn_make_buffer_rsrc((void*)g, (short)0, (int)(((long)(NROWS - 1) * ld + DH) * 2), 0x00020000);
#pragma unroll
    for (int i = 0; i < P; ++i) {
        const int blk = wave * P + i, r = blk * 8 + (lane >> 3), c = (lane & 7) ^ swz(r);
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rs, (LdsPtr)(s + blk * 1024), 16, (int)(((long)r * ld + c * 8) * 2),
                                                 0, 0, 0);
    }
}

// s_waitcnt vmcnt(0), leaving the other counters unconstrained
__device__ __forceinline__ void wait_loads() { __builtin_amdgcn_s_waitcnt((0x7 << 4) | (0xF << 8)); }

// A operand from an [row][d] tile: rows row0 + lane%32, d = s*16 + 8*(lane/32) .. +8.
__device__ __forceinline__ bf16x8 frag_rows(const char* s, int row0, int kstep, int lane) {
    return *reinterpret_cast<const bf16x8*>(s + lds_off(row0 + (lane & 31), kstep * 16 + (lane >> 5) * 8));
}

// A operand of the transposed tile (m = feature d0 + lane%32) from an [row][d]
// tile, with the k order of a register-held accumulator chunk: rows
// base + 4 (lane/32) + {0..3} and base + 8 + 4 (lane/32) + {0..3}.  Two
// transposing LDS reads (ds_read_b64_tr_b16): in each 16-lane group, lane q
// addresses row k0 + q/4, features m0 + 4 (q%4) .. +3, and receives the four
// rows k0 .. k0+3 of feature m0 + q.
__device__ __forceinline__ bf16x8 frag_tr(const char* s, int d0, int base, int lane) {
    const int g = lane >> 4, q = lane & 15;
    const int row = base + 4 * (g >> 1) + (q >> 2), col = d0 + 16 * (g & 1) + 4 * (q & 3);
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LdsV4)(s + lds_off(row, col)));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LdsV4)(s + lds_off(row + 8, col)));
    const bf16x4 x = __builtin_bit_cast(bf16x4, lo), y = __builtin_bit_cast(bf16x4, hi);
    return bf16x8{x[0], x[1], x[2], x[3], y[0], y[1], y[2], y[3]};
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

// 2^x with the hardware transcendental (v_exp_f32); every argument here is
// <= 0 or a finite difference of scaled scores, and a result that flushes
// to zero below 2^-126 is irrelevant next to the row's largest term (1).
__device__ __forceinline__ float exp2_hw(float x) { return __builtin_amdgcn_exp2f(x); }

// Work item of this workgroup, remapped so that the workgroups of one
// (sequence, head) -- consecutive work items -- run on the same XCD (the
// hardware deals consecutive workgroup ids round-robin to the 8 XCDs, each
// with its own L2) and share its cached copy of the head's keys and values.
// Returns the row block in *blk and the (sequence, head) index.
__device__ __forceinline__ int xcd_work(int* blk) {
    const int G = gridDim.x * gridDim.y, G8 = G & ~7;
    int L = blockIdx.x + blockIdx.y * gridDim.x;
    if (L < G8) L = (L & 7) * (G8 >> 3) + (L >> 3);
    *blk = L % gridDim.x;
    return L / gridDim.x;
}

// Forward: QW waves per workgroup, 32 queries each, all keys of the head.
template <int NKB, int QW, bool CAUSAL>
__global__ void __launch_bounds__(64 * QW) attn_fwd_mfma(AttnArgs a) {
    __shared__ __attribute__((aligned(1024))) char Ks[NKB * 32 * 128];
    __shared__ __attribute__((aligned(1024))) char Vs[NKB * 32 * 128];
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int blk;
    const int bh = xcd_work(&blk), b = bh / a.H, hh = bh % a.H;
    const bf16* K = reinterpret_cast<const bf16*>(a.k) + (long)b * a.Sk * a.ldk + hh * DH;
    const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)b * a.Sk * a.ldv + hh * DH;
    // this wave's queries are fetched while the keys and values stream into LDS
    const int q0 = (blk * QW + wave) * 32;
    const int q = q0 + (lane & 31);
    bf16x8 qf[4];
    if (q0 < a.Sq) {
        const bf16* Qrow = reinterpret_cast<const bf16*>(a.q) + ((long)b * a.Sq + q) * a.ldq + hh * DH;
#pragma unroll
        for (int s = 0; s < 4; ++s) qf[s] = frag_global(Qrow, s, lane);
    }
    stage_dl<NKB * 32, QW>(Ks, K, a.ldk, wave, lane);
    stage_dl<NKB * 32, QW>(Vs, V, a.ldv, wave, lane);
    wait_loads();
    __syncthreads();
    if (q0 >= a.Sq) return;
    // key blocks at or below the diagonal (causal), else all
    const int nkb = CAUSAL ? min(NKB, q0 / 32 + 1) : NKB;
    f32x16 sc[NKB];
    float m = -INFINITY;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        sc[kb] = zero16();
        if (kb >= nkb) continue;
#pragma unroll
        for (int s = 0; s < 4; ++s) sc[kb] = mfma(frag_rows(Ks, kb * 32, s, lane), qf[s], sc[kb]);
        if (CAUSAL && kb == nkb - 1) {
            // the diagonal block: keys after the query are masked
#pragma unroll
            for (int r = 0; r < 16; ++r)
                if (kb * 32 + acc_row(r, lane) > q) sc[kb][r] = -INFINITY;
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) m = fmaxf(m, sc[kb][r]);
    }
    m = fmaxf(m, __shfl_xor(m, 32, 64));
    // p = 2^(c (s - m)) with c = scale log2(e): one FMA and one exp per score
    const float c = a.scale * LOG2E, mc = m * c;
    float sum = 0.f;
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        if (kb >= nkb) continue;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const float p = exp2_hw(fmaf(sc[kb][r], c, -mc));
            sc[kb][r] = p;
            sum += p;
        }
    }
    sum += __shfl_xor(sum, 32, 64);
    f32x16 o[2] = {zero16(), zero16()};
#pragma unroll
    for (int kb = 0; kb < NKB; ++kb) {
        if (kb >= nkb) continue;
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            const bf16x8 pf = pack_chunk(sc[kb], cc);
#pragma unroll
            for (int db = 0; db < 2; ++db) o[db] = mfma(frag_tr(Vs, db * 32, kb * 32 + cc * 16, lane), pf, o[db]);
        }
    }
    bf16* O = reinterpret_cast<bf16*>(a.o) + ((long)b * a.Sq + q0) * a.ldo + hh * DH;
    store_t(O, a.ldo, o, 1.f / sum, lane);
    if (a.lse && lane < 32) a.lse[(long)bh * a.Sq + q] = m * a.scale + logf(sum);
}

// Forward with the keys split in two halves (non-causal, even key-block
// count): 2 QW waves per workgroup, wave w takes query block w % QW and key
// half w / QW.  Each wave runs the softmax over its half with its own running
// maximum and sum and an unnormalised output; the second half's wave hands
// (O, m, sum) to the first through LDS (the K/V tiles' space once every wave
// is done with them), which rescales both to the common maximum, normalises
// and stores.  Twice the waves of attn_fwd_mfma on the same LDS, each with
// half the serial work.
template <int NKB, int QW>
__global__ void __launch_bounds__(128 * QW) attn_fwd_ks(AttnArgs a) {
    static_assert(NKB % 2 == 0, "key halves");
    constexpr int HB = NKB / 2;
    constexpr int KVB = NKB * 32 * 128, XB = QW * 64 * 34 * 4;
    __shared__ __attribute__((aligned(1024))) char KV[2 * KVB > XB ? 2 * KVB : XB];
    char* const Ks = KV;
    char* const Vs = KV + KVB;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = wave / QW, qw = wave % QW;
    int blk;
    const int bh = xcd_work(&blk), b = bh / a.H, hh = bh % a.H;
    const bf16* K = reinterpret_cast<const bf16*>(a.k) + (long)b * a.Sk * a.ldk + hh * DH;
    const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)b * a.Sk * a.ldv + hh * DH;
    const int q0 = (blk * QW + qw) * 32;
    const bool live = q0 < a.Sq;  // every wave takes part in all three barriers
    const int q = q0 + (lane & 31);
    bf16x8 qf[4];
    if (live) {
        const bf16* Qrow = reinterpret_cast<const bf16*>(a.q) + ((long)b * a.Sq + q) * a.ldq + hh * DH;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) qf[s2] = frag_global(Qrow, s2, lane);
    }
    stage_dl<NKB * 32, 2 * QW>(Ks, K, a.ldk, wave, lane);
    stage_dl<NKB * 32, 2 * QW>(Vs, V, a.ldv, wave, lane);
    wait_loads();
    __syncthreads();
    const float c = a.scale * LOG2E;
    f32x16 o[2] = {zero16(), zero16()};
    float m = -INFINITY, sum = 0.f;
    if (live) {
        f32x16 sc[HB];
#pragma unroll
        for (int j = 0; j < HB; ++j) {
            const int kb = half * HB + j;
            sc[j] = zero16();
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) sc[j] = mfma(frag_rows(Ks, kb * 32, s2, lane), qf[s2], sc[j]);
#pragma unroll
            for (int r = 0; r < 16; ++r) m = fmaxf(m, sc[j][r]);
        }
        m = fmaxf(m, __shfl_xor(m, 32, 64));
        const float mc = m * c;
#pragma unroll
        for (int j = 0; j < HB; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float pv = exp2_hw(fmaf(sc[j][r], c, -mc));
                sc[j][r] = pv;
                sum += pv;
            }
        sum += __shfl_xor(sum, 32, 64);
#pragma unroll
        for (int j = 0; j < HB; ++j) {
            const int kb = half * HB + j;
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
                const bf16x8 pf = pack_chunk(sc[j], cc);
#pragma unroll
                for (int db = 0; db < 2; ++db) o[db] = mfma(frag_tr(Vs, db * 32, kb * 32 + cc * 16, lane), pf, o[db]);
            }
        }
    }
    __syncthreads();  // K and V are no longer read: their space carries the hand-over
    float* xo = reinterpret_cast<float*>(KV) + (qw * 64 + lane) * 34;
    if (half == 1 && live) {
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) xo[db * 16 + r] = o[db][r];
        xo[32] = m;
        xo[33] = sum;
    }
    __syncthreads();
    if (half == 1 || !live) return;
    const float m1 = xo[32], s1 = xo[33];
    const float mn = fmaxf(m, m1);
    const float a0 = exp2_hw((m - mn) * c), a1 = exp2_hw((m1 - mn) * c);
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) o[db][r] = o[db][r] * a0 + xo[db * 16 + r] * a1;
    const float tot = sum * a0 + s1 * a1;
    bf16* O = reinterpret_cast<bf16*>(a.o) + ((long)b * a.Sq + q0) * a.ldo + hh * DH;
    store_t(O, a.ldo, o, 1.f / tot, lane);
    if (a.lse && lane < 32) a.lse[(long)bh * a.Sq + q] = mn * a.scale + logf(tot);
}

// dQ pass: QW waves per workgroup, 32 queries each; also writes delta.
template <int NKB, int QW, bool CAUSAL>
__global__ void __launch_bounds__(64 * QW) attn_bwd_dq_mfma(AttnArgs a) {
    __shared__ __attribute__((aligned(1024))) char Ks[NKB * 32 * 128];
    __shared__ __attribute__((aligned(1024))) char Vs[NKB * 32 * 128];
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int blk;
    const int bh = xcd_work(&blk), b = bh / a.H, hh = bh % a.H;
    const bf16* K = reinterpret_cast<const bf16*>(a.k) + (long)b * a.Sk * a.ldk + hh * DH;
    const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)b * a.Sk * a.ldv + hh * DH;
    // this wave's queries, output gradients and LSE are fetched while the
    // keys and values stream into LDS
    const int q0 = (blk * QW + wave) * 32;
    const int q = q0 + (lane & 31);
    bf16x8 qf[4], gf[4];
    float lse = 0.f;
    if (q0 < a.Sq) {
        const long qrow = (long)b * a.Sq + q;
        const bf16* Qrow = reinterpret_cast<const bf16*>(a.q) + qrow * a.ldq + hh * DH;
        const bf16* dOrow = reinterpret_cast<const bf16*>(a.dout) + qrow * a.lddo + hh * DH;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            qf[s] = frag_global(Qrow, s, lane);
            gf[s] = frag_global(dOrow, s, lane);
        }
        lse = a.lse[(long)bh * a.Sq + q];
    }
    stage_dl<NKB * 32, QW>(Ks, K, a.ldk, wave, lane);
    stage_dl<NKB * 32, QW>(Vs, V, a.ldv, wave, lane);
    wait_loads();
    __syncthreads();
    if (q0 >= a.Sq) return;
    const float c = a.scale * LOG2E;
    const float lse2 = lse * LOG2E;
    const int nkb = CAUSAL ? min(NKB, q0 / 32 + 1) : NKB;
    // delta = sum_j P_ij dP_ij; lanes l and l + 32 hold the two key halves of a block
    float dpart = 0.f;
#pragma unroll 2
    for (int kb = 0; kb < nkb; ++kb) {
        f32x16 st = zero16(), dp = zero16();
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            st = mfma(frag_rows(Ks, kb * 32, s, lane), qf[s], st);
            dp = mfma(frag_rows(Vs, kb * 32, s, lane), gf[s], dp);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float p = exp2_hw(fmaf(st[r], c, -lse2));
            if (CAUSAL && kb * 32 + acc_row(r, lane) > q) p = 0.f;
            dpart = fmaf(p, dp[r], dpart);
        }
    }
    const float delta = dpart + __shfl_xor(dpart, 32, 64);
    f32x16 dq[2] = {zero16(), zero16()};
#pragma unroll 2
    for (int kb = 0; kb < nkb; ++kb) {
        f32x16 st = zero16(), dp = zero16();
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            st = mfma(frag_rows(Ks, kb * 32, s, lane), qf[s], st);
            dp = mfma(frag_rows(Vs, kb * 32, s, lane), gf[s], dp);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float p = exp2_hw(fmaf(st[r], c, -lse2));
            if (CAUSAL && kb * 32 + acc_row(r, lane) > q) p = 0.f;
            st[r] = fmaf(p, dp[r], -p * delta);
        }
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            const bf16x8 df = pack_chunk(st, cc);
#pragma unroll
            for (int db = 0; db < 2; ++db) dq[db] = mfma(frag_tr(Ks, db * 32, kb * 32 + cc * 16, lane), df, dq[db]);
        }
    }
    bf16* dQ = reinterpret_cast<bf16*>(a.dq) + ((long)b * a.Sq + q0) * a.lddq + hh * DH;
    store_t(dQ, a.lddq, dq, a.scale, lane);
    if (lane < 32) a.delta[(long)bh * a.Sq + q] = delta;
}

// dK/dV pass: KW waves per workgroup, 32 keys each, looping over query blocks.
template <int NQB, int KW, bool CAUSAL>
__global__ void __launch_bounds__(64 * KW) attn_bwd_dkv_mfma(AttnArgs a) {
    __shared__ __attribute__((aligned(1024))) char Qs[NQB * 32 * 128];
    __shared__ __attribute__((aligned(1024))) char Gs[NQB * 32 * 128];
    __shared__ __attribute__((aligned(16))) float lse2s[NQB * 32], dls[NQB * 32];
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int blk;
    const int bh = xcd_work(&blk), b = bh / a.H, hh = bh % a.H;
    const int Sq = NQB * 32;
    const bf16* Q = reinterpret_cast<const bf16*>(a.q) + (long)b * a.Sq * a.ldq + hh * DH;
    const bf16* G = reinterpret_cast<const bf16*>(a.dout) + (long)b * a.Sq * a.lddo + hh * DH;
    // this wave's keys and values are fetched while the queries and output
    // gradients stream into LDS
    const int k0 = (blk * KW + wave) * 32;
    const int key = k0 + (lane & 31);
    bf16x8 kf[4], vf[4];
    if (k0 < a.Sk) {
        const long krow = (long)b * a.Sk + key;
        const bf16* Krow = reinterpret_cast<const bf16*>(a.k) + krow * a.ldk + hh * DH;
        const bf16* Vrow = reinterpret_cast<const bf16*>(a.v) + krow * a.ldv + hh * DH;
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            kf[s] = frag_global(Krow, s, lane);
            vf[s] = frag_global(Vrow, s, lane);
        }
    }
    stage_dl<NQB * 32, KW>(Qs, Q, a.ldq, wave, lane);
    stage_dl<NQB * 32, KW>(Gs, G, a.lddo, wave, lane);
    for (int i = tid; i < Sq; i += 64 * KW) {
        lse2s[i] = a.lse[(long)bh * a.Sq + i] * LOG2E;
        dls[i] = a.delta[(long)bh * a.Sq + i];
    }
    wait_loads();
    __syncthreads();
    if (k0 >= a.Sk) return;
    const float c = a.scale * LOG2E;
    f32x16 dk[2] = {zero16(), zero16()}, dv[2] = {zero16(), zero16()};
    const int qb0 = CAUSAL ? k0 / 32 : 0;
    for (int qb = qb0; qb < NQB; ++qb) {
        f32x16 st = zero16(), dp = zero16();
#pragma unroll
        for (int s = 0; s < 4; ++s) {
            st = mfma(frag_rows(Qs, qb * 32, s, lane), kf[s], st);
            dp = mfma(frag_rows(Gs, qb * 32, s, lane), vf[s], dp);
        }
        // this lane's rows of the block: 8 j + 4 (lane/32) + {0..3}, j = 0..3
        f32x4 l4[4], d4[4];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int r0 = qb * 32 + 8 * j + 4 * (lane >> 5);
            l4[j] = *reinterpret_cast<const f32x4*>(lse2s + r0);
            d4[j] = *reinterpret_cast<const f32x4*>(dls + r0);
        }
        f32x16 pm;
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float p = exp2_hw(fmaf(st[r], c, -l4[r >> 2][r & 3]));
            if (CAUSAL && key > qb * 32 + acc_row(r, lane)) p = 0.f;
            pm[r] = p;
            st[r] = fmaf(p, dp[r], -p * d4[r >> 2][r & 3]);
        }
#pragma unroll
        for (int cc = 0; cc < 2; ++cc) {
            const bf16x8 pf = pack_chunk(pm, cc);
            const bf16x8 df = pack_chunk(st, cc);
#pragma unroll
            for (int db = 0; db < 2; ++db) {
                dv[db] = mfma(frag_tr(Gs, db * 32, qb * 32 + cc * 16, lane), pf, dv[db]);
                dk[db] = mfma(frag_tr(Qs, db * 32, qb * 32 + cc * 16, lane), df, dk[db]);
            }
        }
    }
    bf16* dK = reinterpret_cast<bf16*>(a.dk) + ((long)b * a.Sk + k0) * a.lddk + hh * DH;
    bf16* dV = reinterpret_cast<bf16*>(a.dv) + ((long)b * a.Sk + k0) * a.lddv + hh * DH;
    store_t(dK, a.lddk, dk, a.scale, lane);
    store_t(dV, a.lddv, dv, 1.f, lane);
}

// dQ pass with the keys split in two halves (non-causal, even key-block
// count): 2 QW waves per workgroup, wave w takes query block w % QW and key
// half w / QW.  The two waves of a query block exchange their partial delta
// through LDS (both add the halves in the same order, so both hold the same
// delta), then each runs dS and dQ over its half; the second half's wave hands
// its dQ partial to the first, which adds it and stores.  Halves the serial
// chain of each wave.
template <int NKB, int QW>
__global__ void __launch_bounds__(128 * QW) attn_bwd_dq_ks(AttnArgs a) {
    static_assert(NKB % 2 == 0, "key halves");
    constexpr int HB = NKB / 2;
    constexpr int KVB = NKB * 32 * 128, XB = QW * 64 * 32 * 4;
    __shared__ __attribute__((aligned(1024))) char KV[2 * KVB > XB ? 2 * KVB : XB];
    __shared__ float xd[2 * QW * 64];
    char* const Ks = KV;
    char* const Vs = KV + KVB;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = wave / QW, qw = wave % QW;
    int blk;
    const int bh = xcd_work(&blk), b = bh / a.H, hh = bh % a.H;
    const bf16* K = reinterpret_cast<const bf16*>(a.k) + (long)b * a.Sk * a.ldk + hh * DH;
    const bf16* V = reinterpret_cast<const bf16*>(a.v) + (long)b * a.Sk * a.ldv + hh * DH;
    const int q0 = (blk * QW + qw) * 32;
    const bool live = q0 < a.Sq;  // every wave takes part in all four barriers
    const int q = q0 + (lane & 31);
    bf16x8 qf[4], gf[4];
    float lse = 0.f;
    if (live) {
        const long qrow = (long)b * a.Sq + q;
        const bf16* Qrow = reinterpret_cast<const bf16*>(a.q) + qrow * a.ldq + hh * DH;
        const bf16* dOrow = reinterpret_cast<const bf16*>(a.dout) + qrow * a.lddo + hh * DH;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
            qf[s2] = frag_global(Qrow, s2, lane);
            gf[s2] = frag_global(dOrow, s2, lane);
        }
        lse = a.lse[(long)bh * a.Sq + q];
    }
    stage_dl<NKB * 32, 2 * QW>(Ks, K, a.ldk, wave, lane);
    stage_dl<NKB * 32, 2 * QW>(Vs, V, a.ldv, wave, lane);
    wait_loads();
    __syncthreads();
    const float c = a.scale * LOG2E;
    const float lse2 = lse * LOG2E;
    const int kb0 = half * HB;
    // partial delta = sum over this half's keys of P dP
    float dpart = 0.f;
    if (live) {
#pragma unroll 2
        for (int j = 0; j < HB; ++j) {
            const int kb = kb0 + j;
            f32x16 st = zero16(), dp = zero16();
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                st = mfma(frag_rows(Ks, kb * 32, s2, lane), qf[s2], st);
                dp = mfma(frag_rows(Vs, kb * 32, s2, lane), gf[s2], dp);
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) dpart = fmaf(exp2_hw(fmaf(st[r], c, -lse2)), dp[r], dpart);
        }
        dpart += __shfl_xor(dpart, 32, 64);
    }
    xd[wave * 64 + lane] = dpart;
    __syncthreads();
    const float delta = xd[qw * 64 + lane] + xd[(QW + qw) * 64 + lane];
    f32x16 dq[2] = {zero16(), zero16()};
    if (live) {
#pragma unroll 2
        for (int j = 0; j < HB; ++j) {
            const int kb = kb0 + j;
            f32x16 st = zero16(), dp = zero16();
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                st = mfma(frag_rows(Ks, kb * 32, s2, lane), qf[s2], st);
                dp = mfma(frag_rows(Vs, kb * 32, s2, lane), gf[s2], dp);
            }
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = exp2_hw(fmaf(st[r], c, -lse2));
                st[r] = fmaf(p, dp[r], -p * delta);
            }
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
                const bf16x8 df = pack_chunk(st, cc);
#pragma unroll
                for (int db = 0; db < 2; ++db) dq[db] = mfma(frag_tr(Ks, db * 32, kb * 32 + cc * 16, lane), df, dq[db]);
            }
        }
    }
    __syncthreads();  // K and V are no longer read: their space carries the hand-over
    float* xo = reinterpret_cast<float*>(KV) + (qw * 32) * 64 + lane;  // register-major, lane fastest
    if (half == 1 && live) {
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) xo[(db * 16 + r) * 64] = dq[db][r];
    }
    __syncthreads();
    if (half == 1 || !live) return;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) dq[db][r] += xo[(db * 16 + r) * 64];
    bf16* dQ = reinterpret_cast<bf16*>(a.dq) + ((long)b * a.Sq + q0) * a.lddq + hh * DH;
    store_t(dQ, a.lddq, dq, a.scale, lane);
    if (lane < 32) a.delta[(long)bh * a.Sq + q] = delta;
}

// dK/dV pass with the queries split in two halves (non-causal, even
// query-block count): 2 KW waves per workgroup, wave w takes key block w % KW
// and query half w / KW; the second half's wave hands its dK and dV partials
// to the first through LDS, which adds them and stores.
template <int NQB, int KW>
__global__ void __launch_bounds__(128 * KW) attn_bwd_dkv_ks(AttnArgs a) {
    static_assert(NQB % 2 == 0, "query halves");
    constexpr int HQ = NQB / 2;
    constexpr int QGB = NQB * 32 * 128, XB = KW * 64 * 64 * 4;
    __shared__ __attribute__((aligned(1024))) char QG[2 * QGB > XB ? 2 * QGB : XB];
    __shared__ __attribute__((aligned(16))) float lse2s[NQB * 32], dls[NQB * 32];
    char* const Qs = QG;
    char* const Gs = QG + QGB;
    const int tid = threadIdx.x, lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int half = wave / KW, kw = wave % KW;
    int blk;
    const int bh = xcd_work(&blk), b = bh / a.H, hh = bh % a.H;
    const int Sq = NQB * 32;
    const bf16* Q = reinterpret_cast<const bf16*>(a.q) + (long)b * a.Sq * a.ldq + hh * DH;
    const bf16* G = reinterpret_cast<const bf16*>(a.dout) + (long)b * a.Sq * a.lddo + hh * DH;
    const int k0 = (blk * KW + kw) * 32;
    const bool live = k0 < a.Sk;  // every wave takes part in all three barriers
    const int key = k0 + (lane & 31);
    bf16x8 kf[4], vf[4];
    if (live) {
        const long krow = (long)b * a.Sk + key;
        const bf16* Krow = reinterpret_cast<const bf16*>(a.k) + krow * a.ldk + hh * DH;
        const bf16* Vrow = reinterpret_cast<const bf16*>(a.v) + krow * a.ldv + hh * DH;
#pragma unroll
        for (int s2 = 0; s2 < 4; ++s2) {
            kf[s2] = frag_global(Krow, s2, lane);
            vf[s2] = frag_global(Vrow, s2, lane);
        }
    }
    stage_dl<NQB * 32, 2 * KW>(Qs, Q, a.ldq, wave, lane);
    stage_dl<NQB * 32, 2 * KW>(Gs, G, a.lddo, wave, lane);
    for (int i = tid; i < Sq; i += 128 * KW) {
        lse2s[i] = a.lse[(long)bh * a.Sq + i] * LOG2E;
        dls[i] = a.delta[(long)bh * a.Sq + i];
    }
    wait_loads();
    __syncthreads();
    const float c = a.scale * LOG2E;
    f32x16 dk[2] = {zero16(), zero16()}, dv[2] = {zero16(), zero16()};
    if (live) {
        for (int j = 0; j < HQ; ++j) {
            const int qb = half * HQ + j;
            f32x16 st = zero16(), dp = zero16();
#pragma unroll
            for (int s2 = 0; s2 < 4; ++s2) {
                st = mfma(frag_rows(Qs, qb * 32, s2, lane), kf[s2], st);
                dp = mfma(frag_rows(Gs, qb * 32, s2, lane), vf[s2], dp);
            }
            // this lane's rows of the block: 8 i + 4 (lane/32) + {0..3}, i = 0..3
            f32x4 l4[4], d4[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const int r0 = qb * 32 + 8 * i + 4 * (lane >> 5);
                l4[i] = *reinterpret_cast<const f32x4*>(lse2s + r0);
                d4[i] = *reinterpret_cast<const f32x4*>(dls + r0);
            }
            f32x16 pm;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const float p = exp2_hw(fmaf(st[r], c, -l4[r >> 2][r & 3]));
                pm[r] = p;
                st[r] = fmaf(p, dp[r], -p * d4[r >> 2][r & 3]);
            }
#pragma unroll
            for (int cc = 0; cc < 2; ++cc) {
                const bf16x8 pf = pack_chunk(pm, cc);
                const bf16x8 df = pack_chunk(st, cc);
#pragma unroll
                for (int db = 0; db < 2; ++db) {
                    dv[db] = mfma(frag_tr(Gs, db * 32, qb * 32 + cc * 16, lane), pf, dv[db]);
                    dk[db] = mfma(frag_tr(Qs, db * 32, qb * 32 + cc * 16, lane), df, dk[db]);
                }
            }
        }
    }
    __syncthreads();  // Q and dO are no longer read: their space carries the hand-over
    float* xo = reinterpret_cast<float*>(QG) + (kw * 64) * 64 + lane;  // register-major, lane fastest
    if (half == 1 && live) {
#pragma unroll
        for (int db = 0; db < 2; ++db)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                xo[(db * 16 + r) * 64] = dk[db][r];
                xo[(32 + db * 16 + r) * 64] = dv[db][r];
            }
    }
    __syncthreads();
    if (half == 1 || !live) return;
#pragma unroll
    for (int db = 0; db < 2; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            dk[db][r] += xo[(db * 16 + r) * 64];
            dv[db][r] += xo[(32 + db * 16 + r) * 64];
        }
    bf16* dK = reinterpret_cast<bf16*>(a.dk) + ((long)b * a.Sk + k0) * a.lddk + hh * DH;
    bf16* dV = reinterpret_cast<bf16*>(a.dv) + ((long)b * a.Sk + k0) * a.lddv + hh * DH;
    store_t(dK, a.lddk, dk, a.scale, lane);
    store_t(dV, a.lddv, dv, 1.f, lane);
}

// Launch KERNEL<NB, W, C> for the runtime block count NB (1..8), W waves and causal flag C.
#define GP_NB_SWITCH(NB, W, C, KERNEL, GRID)                                               \
    switch (NB) {                                                                          \
    case 1: klaunch(KERNEL<1, W, C>, GRID, 64 * W, 0, st, a); break;                       \
    case 2: klaunch(KERNEL<2, W, C>, GRID, 64 * W, 0, st, a); break;                       \
    case 3: klaunch(KERNEL<3, W, C>, GRID, 64 * W, 0, st, a); break;                       \
    case 4: klaunch(KERNEL<4, W, C>, GRID, 64 * W, 0, st, a); break;                       \
    case 5: klaunch(KERNEL<5, W, C>, GRID, 64 * W, 0, st, a); break;                       \
    case 6: klaunch(KERNEL<6, W, C>, GRID, 64 * W, 0, st, a); break;                       \
    case 7: klaunch(KERNEL<7, W, C>, GRID, 64 * W, 0, st, a); break;                       \
    case 8: klaunch(KERNEL<8, W, C>, GRID, 64 * W, 0, st, a); break;                       \
    default: return set_error(GP_ERR_UNSUPPORTED, "attention: sequence length > 256");     \
    }
#define GP_WC_SWITCH(NB, W, CAUS, KERNEL, GRID)                                            \
    if (CAUS) {                                                                            \
        if (W == 4) { GP_NB_SWITCH(NB, 4, true, KERNEL, GRID) }                            \
        else if (W == 2) { GP_NB_SWITCH(NB, 2, true, KERNEL, GRID) }                       \
        else { GP_NB_SWITCH(NB, 1, true, KERNEL, GRID) }                                   \
    } else {                                                                               \
        if (W == 4) { GP_NB_SWITCH(NB, 4, false, KERNEL, GRID) }                           \
        else if (W == 2) { GP_NB_SWITCH(NB, 2, false, KERNEL, GRID) }                      \
        else { GP_NB_SWITCH(NB, 1, false, KERNEL, GRID) }                                  \
    }

// Waves per workgroup (32 rows each): as many as keep at least 2 x NUM_CU
// workgroups for a small batch, at most 4 (fewer waves per workgroup re-stage
// the head's keys and values more often).  AttnArgs::waves (1, 2 or 4)
// overrides the choice.
int waves_for(const AttnArgs& a, long row_blocks) {
    if (a.waves == 1 || a.waves == 2 || a.waves == 4) return a.waves;
    constexpr long CU2 = 2 * 256;
    return row_blocks >= 4 * CU2 ? 4 : row_blocks >= 2 * CU2 ? 2 : 1;
}

// Split variants (two waves per 32-row block, each over half of the loop's
// blocks): non-causal heads whose loop runs over an even block count, when
// the row blocks alone would leave a SIMD with at most one wave (there the
// one-wave kernels' serial chain sets the time; with more row blocks the two
// forms tie or the split loses to the doubled wave count).
// AttnArgs::split = 0 keeps the one-wave kernels.
bool split_ok(const AttnArgs& a, long row_blocks, int loop_blocks) {
    constexpr long SIMDS = 4 * 256;
    return a.split && !a.causal && loop_blocks % 2 == 0 && row_blocks <= SIMDS;
}

// Launch KERNEL<NB, W> (split variants: 128 W threads) for an even block count NB <= 8.
#define GP_KS_SWITCH(NB, W, KERNEL, GRID)                                                      \
    switch ((NB) * 8 + (W)) {                                                                  \
    case 2 * 8 + 1: klaunch(KERNEL<2, 1>, GRID, 128, 0, st, a); break;                         \
    case 2 * 8 + 2: klaunch(KERNEL<2, 2>, GRID, 256, 0, st, a); break;                         \
    case 2 * 8 + 4: klaunch(KERNEL<2, 4>, GRID, 512, 0, st, a); break;                         \
    case 4 * 8 + 1: klaunch(KERNEL<4, 1>, GRID, 128, 0, st, a); break;                         \
    case 4 * 8 + 2: klaunch(KERNEL<4, 2>, GRID, 256, 0, st, a); break;                         \
    case 4 * 8 + 4: klaunch(KERNEL<4, 4>, GRID, 512, 0, st, a); break;                         \
    case 6 * 8 + 1: klaunch(KERNEL<6, 1>, GRID, 128, 0, st, a); break;                         \
    case 6 * 8 + 2: klaunch(KERNEL<6, 2>, GRID, 256, 0, st, a); break;                         \
    case 6 * 8 + 4: klaunch(KERNEL<6, 4>, GRID, 512, 0, st, a); break;                         \
    case 8 * 8 + 1: klaunch(KERNEL<8, 1>, GRID, 128, 0, st, a); break;                         \
    case 8 * 8 + 2: klaunch(KERNEL<8, 2>, GRID, 256, 0, st, a); break;                         \
    case 8 * 8 + 4: klaunch(KERNEL<8, 4>, GRID, 512, 0, st, a); break;                         \
    default: return set_error(GP_ERR_UNSUPPORTED, "attention: sequence length > 256");         \
    }

bool mfma_ok(const AttnArgs& a) {
    return a.dh == DH && a.Sq % 32 == 0 && a.Sk % 32 == 0 && a.Sq <= MAXK && a.Sk <= MAXK &&
           a.ldq % 8 == 0 && a.ldk % 8 == 0 && a.ldv % 8 == 0 && a.ldo % 8 == 0;
}

} // namespace

gp_status attention_fwd(int dtype, const AttnArgs& a, hipStream_t st) {
    if (dtype != GP_BF16) return attention_fwd_simt(dtype, a, st);
    if (!mfma_ok(a)) return set_error(GP_ERR_UNSUPPORTED, "bf16 attention needs d_h = 64 and lengths multiple of 32, <= 256");
    const int w = waves_for(a, (long)(a.Sq / 32) * (a.hint_n ? a.hint_n : a.n) * a.H);
    dim3 grid((a.Sq + 32 * w - 1) / (32 * w), a.n * a.H);
    if (split_ok(a, (long)(a.Sq / 32) * (a.hint_n ? a.hint_n : a.n) * a.H, a.Sk / 32)) {
        GP_KS_SWITCH(a.Sk / 32, w, attn_fwd_ks, grid);
    } else {
        GP_WC_SWITCH(a.Sk / 32, w, a.causal, attn_fwd_mfma, grid);
    }
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status attention_bwd(int dtype, const AttnArgs& a, hipStream_t st) {
    if (dtype != GP_BF16) return attention_bwd_simt(dtype, a, st);
    if (!mfma_ok(a)) return set_error(GP_ERR_UNSUPPORTED, "bf16 attention needs d_h = 64 and lengths multiple of 32, <= 256");
    const int wq = waves_for(a, (long)(a.Sq / 32) * (a.hint_n ? a.hint_n : a.n) * a.H);
    dim3 gq((a.Sq + 32 * wq - 1) / (32 * wq), a.n * a.H);
    if (split_ok(a, (long)(a.Sq / 32) * (a.hint_n ? a.hint_n : a.n) * a.H, a.Sk / 32)) {
        GP_KS_SWITCH(a.Sk / 32, wq, attn_bwd_dq_ks, gq);
    } else {
        GP_WC_SWITCH(a.Sk / 32, wq, a.causal, attn_bwd_dq_mfma, gq);
    }
    GP_LAUNCH_CHECK();
    const int wk = waves_for(a, (long)(a.Sk / 32) * (a.hint_n ? a.hint_n : a.n) * a.H);
    dim3 gk((a.Sk + 32 * wk - 1) / (32 * wk), a.n * a.H);
    if (split_ok(a, (long)(a.Sk / 32) * (a.hint_n ? a.hint_n : a.n) * a.H, a.Sq / 32)) {
        GP_KS_SWITCH(a.Sq / 32, wk, attn_bwd_dkv_ks, gk);
    } else {
        GP_WC_SWITCH(a.Sq / 32, wk, a.causal, attn_bwd_dkv_mfma, gk);
    }
    GP_LAUNCH_CHECK();
    return GP_OK;
}

} // namespace gp
