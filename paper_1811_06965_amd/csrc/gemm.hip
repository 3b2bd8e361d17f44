// gemm.hip -- LDS-staged MFMA GEMM family of the partition (gfx950, wave64).
//
//   C[m, n] = sum_k A(m, k) B(n, k)     then a fused epilogue
//
// Every linear layer of the partition maps onto one of three operand forms:
//   forward    Y  = X W      A = X  [T, in]  k-contiguous,  B = W^T [out, in]  k-contiguous
//   input grad dX = dY W^T   A = dY [T, out] k-contiguous,  B = W   [in, out]  k-contiguous
//   weight grad dW = X^T dY  A = X  [T, in]  m-contiguous,  B = dY  [T, out]   n-contiguous
// The partition keeps both W and W^T working copies so the two activation
// GEMMs stream both operands along k.  The weight-gradient GEMM loads
// m-contiguous 16-byte vectors over 4 consecutive k and transposes them in
// registers, so LDS always holds k-contiguous rows and every MFMA fragment is
// one 16-byte LDS read per lane.
//
// Workgroup = 4 waves (2 x 2).  Tile shapes (bf16, BK = 64):
//   256 x 256: each wave 128 x 128 = 4 x 4 blocks of v_mfma_f32_32x32x16_bf16
//              (256 accumulator registers per lane, held in AGPRs); 144 KB LDS
//   256 x 128, 128 x 256, 128 x 128: smaller waves for short or thin problems.
// Per 16-deep k-step a wave reads (TM + TN) fragments for TM x TN MFMAs, so
// the 128 x 128 wave tile needs 64 B/clk/CU of LDS reads at full MFMA rate.
// Pipelining: global loads of k-tile t+1 are in flight while tile t is
// consumed; MFMA fragments are double-buffered across k-steps; the one
// barrier per k-tile sits before the last k-step's MFMAs, which then cover
// the latency of the first fragment reads from the new buffer.
//
// Split-K (for problems with too few output tiles to fill 256 CUs): k-tiles
// are divided among gridDim.y workgroups per output tile, each writes an fp32
// partial tile, and a reduce kernel sums the partials in a fixed order and
// applies the epilogue -- deterministic, no atomics.
//
// Workgroup ids are remapped so each XCD (which receives every 8th workgroup)
// works on a contiguous run of output tiles that share operand panels in its
// own L2.
#include <algorithm>

#include <cstdlib>
#include "common.hpp"
#include "kernels.hpp"

namespace gp {

namespace {

template <typename T> struct Frag;
template <> struct Frag<bf16> {
    bf16x8 v;
    __device__ __forceinline__ void load(const bf16* p) { v = *reinterpret_cast<const bf16x8*>(p); }
};
template <> struct Frag<float> {
    f32x4 lo, hi;
    __device__ __forceinline__ void load(const float* p) {
        lo = *reinterpret_cast<const f32x4*>(p);
        hi = *reinterpret_cast<const f32x4*>(p + 4);
    }
};

// One 32x32 output block advanced by 16 reduction steps.  Lane l supplies row
// (l % 32) of A and column (l % 32) of B over the 8 k-values
// [8 (l / 32), 8 (l / 32) + 8) of the 16-step chunk; A and B use the same
// k-assignment, so the sum is over all 16 k.
__device__ __forceinline__ void mma(f32x16& c, const Frag<bf16>& a, const Frag<bf16>& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a.v, b.v, c, 0, 0, 0);
}
// The same block with both operands' 16-bit elements read as fp16.
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
__device__ __forceinline__ void mma16(f32x16& c, const Frag<bf16>& a, const Frag<bf16>& b) {
    c = __builtin_amdgcn_mfma_f32_32x32x16_f16(__builtin_bit_cast(f16x8, a.v), __builtin_bit_cast(f16x8, b.v), c, 0,
                                               0, 0);
}
__device__ __forceinline__ void mma(f32x16& c, const Frag<float>& a, const Frag<float>& b) {
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[e], b.lo[e], c, 0, 0, 0);
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[e], b.hi[e], c, 0, 0, 0);
}

template <typename T> using V16 = typename Vec16<T>::type;
typedef int i32x4 __attribute__((ext_vector_type(4)));
typedef __amdgpu_buffer_rsrc_t Rsrc;

// Buffer resource over `bytes` bytes at p; raw buffer accesses beyond it read
// 0 and drop writes, which implements the tile-edge masking without branches.
constexpr uint32_t OOB = 0x80000000u;
__device__ __forceinline__ Rsrc make_rsrc(const void* p, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(p), (short)0, (int)bytes, 0x00020000);
}
template <typename T>
__device__ __forceinline__ V16<T> bload16(Rsrc r, uint32_t off) {
    return __builtin_bit_cast(V16<T>, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
}

// LDS tiles hold ROWS rows of BK elements (128 bytes) with no padding; the
// 16-byte chunk c of row r is stored at chunk c ^ swz(r).  swz varies over
// any 8 consecutive rows (conflict-free fragment reads, where 8 lanes read 8
// consecutive rows) and over rows 8 apart (conflict-free transposing stores,
// where 8 lanes write rows 8 apart).
__device__ __forceinline__ int swz(int r) { return (r ^ (r >> 3)) & 7; }
// fp4 rows of a stage are 32 bytes (two 16-byte chunks); swapping the chunks
// of rows 8 .. 15 (mod 16) spreads 16 lanes reading 16 consecutive rows over
// all banks
__device__ __forceinline__ int sw4(int r) { return (r >> 3) & 1; }

typedef int i32x8 __attribute__((ext_vector_type(8)));
// An empty use of registers loaded from memory: the compiler places its wait
// for the loads here (the host pass of the build sees no body: the VGPR
// constraint exists on the device only).
template <int A, int B>
__device__ __forceinline__ void pin_vgprs(int (&a)[A], int (&b)[B]) {
#if defined(__HIP_DEVICE_COMPILE__)
#pragma unroll
    for (int i = 0; i < A; ++i) asm volatile("" : "+v"(a[i]));
#pragma unroll
    for (int j = 0; j < B; ++j) asm volatile("" : "+v"(b[j]));
#endif
}
// OCP e2m1 x e2m1 (format code 4), both operands scaled per lane by E8M0 byte 0
__device__ __forceinline__ void mma_fp4(f32x16& c, const i32x4& a, const i32x4& b, int sa, int sb) {
    const i32x8 a8 = {a[0], a[1], a[2], a[3], 0, 0, 0, 0}, b8 = {b[0], b[1], b[2], b[3], 0, 0, 0, 0};
    c = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(a8, b8, c, 4, 4, 0, sa, 0, sb);
}
__device__ __forceinline__ int lds_byte(int row, int kbyte) {
    return row * 128 + ((((kbyte >> 4) ^ swz(row)) << 4) | (kbyte & 15));
}

// Tile loader for one operand: ROWS x BK elements of the operand (row index =
// m for A, n for B), k contiguous in LDS.
template <typename T, int ROWS, int BK, bool KMAJOR>
struct TileLoader {
    static constexpr int VEC = Vec16<T>::N;
    static constexpr int ESZ = sizeof(T);
    static_assert(BK * ESZ == 128, "one LDS row is 128 bytes");
    // k-major: each thread moves 16-byte vectors along k.
    static constexpr int TPR = BK / VEC;
    static constexpr int RPP = 256 / TPR;
    static constexpr int KPASS = ROWS / RPP;
    // m-major: each thread moves a VEC (rows) x KB (k) block, transposing it.
    static constexpr int KB = 4;
    static constexpr int MBLK = ROWS / VEC;
    static constexpr int NBLK = MBLK * (BK / KB);
    static constexpr int MPASS = NBLK / 256;
    static constexpr int NREG = KMAJOR ? KPASS : MPASS * KB;
    static_assert(KMAJOR ? (ROWS % RPP == 0) : (NBLK % 256 == 0), "tile shape");

    V16<T> r[NREG];

    __device__ __forceinline__ void load(Rsrc g, long ld, int row0, int nrows, int k0, int K, int tid) {
        if constexpr (KMAJOR) {
            const int rr = tid / TPR, kk = (tid % TPR) * VEC;
#pragma unroll
            for (int p = 0; p < KPASS; ++p) {
                const int row = row0 + p * RPP + rr, k = k0 + kk;
                const bool ok = row < nrows && k < K;
                r[p] = bload16<T>(g, ok ? (uint32_t)(((long)row * ld + k) * ESZ) : OOB);
            }
        } else {
#pragma unroll
            for (int p = 0; p < MPASS; ++p) {
                const int blk = p * 256 + tid;
                const int mb = blk % MBLK, kb = blk / MBLK;
                const int row = row0 + mb * VEC;
#pragma unroll
                for (int q = 0; q < KB; ++q) {
                    const int k = k0 + kb * KB + q;
                    const bool ok = row < nrows && k < K;
                    r[p * KB + q] = bload16<T>(g, ok ? (uint32_t)(((long)k * ld + row) * ESZ) : OOB);
                }
            }
        }
    }

    // m-major only: add this thread's loaded values over its KB k-rows into
    // cs[i] for its VEC rows (operand rows = output columns of a dW GEMM).
    __device__ __forceinline__ void colsum(float (&cs)[VEC]) const {
        if constexpr (!KMAJOR) {
#pragma unroll
            for (int p = 0; p < MPASS; ++p)
#pragma unroll
                for (int q = 0; q < KB; ++q)
#pragma unroll
                    for (int i = 0; i < VEC; ++i) cs[i] += (float)r[p * KB + q][i];
        }
    }

    __device__ __forceinline__ void store(char* __restrict__ s, int tid) const {
        if constexpr (KMAJOR) {
            const int rr = tid / TPR, kk = (tid % TPR) * VEC;
#pragma unroll
            for (int p = 0; p < KPASS; ++p)
                *reinterpret_cast<V16<T>*>(s + lds_byte(p * RPP + rr, kk * ESZ)) = r[p];
        } else {
#pragma unroll
            for (int p = 0; p < MPASS; ++p) {
                const int blk = p * 256 + tid;
                const int mb = blk % MBLK, kb = blk / MBLK;
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    char* dst = s + lds_byte(mb * VEC + i, kb * KB * ESZ);
                    if constexpr (sizeof(T) == 2) {
                        bf16x4 v = {r[p * KB + 0][i], r[p * KB + 1][i], r[p * KB + 2][i], r[p * KB + 3][i]};
                        *reinterpret_cast<bf16x4*>(dst) = v;
                    } else {
                        f32x4 v = {r[p * KB + 0][i], r[p * KB + 1][i], r[p * KB + 2][i], r[p * KB + 3][i]};
                        *reinterpret_cast<f32x4*>(dst) = v;
                    }
                }
            }
        }
    }
};

template <typename T> struct GemmCfg;
template <> struct GemmCfg<bf16> { static constexpr int BK = 64; };
template <> struct GemmCfg<float> { static constexpr int BK = 32; };

// Fragment read: 8 elements (16 bytes for bf16, 32 for fp32) of one LDS row.
template <typename T> struct FragRead;
template <> struct FragRead<bf16> {
    static __device__ __forceinline__ void load(Frag<bf16>& f, const char* s, int row, int kbyte) {
        f.v = *reinterpret_cast<const bf16x8*>(s + lds_byte(row, kbyte));
    }
};
template <> struct FragRead<float> {
    static __device__ __forceinline__ void load(Frag<float>& f, const char* s, int row, int kbyte) {
        f.lo = *reinterpret_cast<const f32x4*>(s + lds_byte(row, kbyte));
        f.hi = *reinterpret_cast<const f32x4*>(s + lds_byte(row, kbyte + 16));
    }
};

// Fused epilogue of one workgroup tile through buffer resources (out-of-range
// elements are dropped by the hardware).  Inputs are loaded in batches of one
// 32-row block strip (TN x 16 values per lane) before any store of that strip,
// so the loads are not serialised behind possibly-aliasing stores.
template <typename T, int EPI>
struct Epilogue {
    Rsrc c, c2, aux, bias;
    __device__ __forceinline__ void init(const GemmArgs& a) {
        const uint32_t esz = sizeof(T);
        const uint32_t cbytes = (uint32_t)(((long)(a.M - 1) * a.ldc + a.N) *
                                           (EPI == EPI_STORE || EPI == EPI_RELU_MASK ? esz : 4));
        c = make_rsrc(a.C, cbytes);
        if constexpr (EPI == EPI_RES_F32) {
            c2 = make_rsrc(a.C2, a.C2 ? (uint32_t)(((long)(a.M - 1) * a.ldc2 + a.N) * esz) : 0u);
            aux = make_rsrc(a.aux, (uint32_t)(((long)(a.M - 1) * a.ldaux + a.N) * 4));
        }
        if constexpr (EPI == EPI_RELU_MASK)
            aux = make_rsrc(a.aux, (uint32_t)(((long)(a.M - 1) * a.ldaux + a.N) * esz));
        bias = make_rsrc(a.bias, a.bias ? (uint32_t)a.N * 4 : 0u);
    }
    static __device__ __forceinline__ void store_elt(Rsrc r, uint32_t off, float v) {
        if constexpr (sizeof(T) == 2)
            __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, (bf16)v), r, off, 0, 0);
        else
            __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), r, off, 0, 0);
    }
    static __device__ __forceinline__ float load_f32(Rsrc r, uint32_t off) {
        return __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(r, off, 0, 0));
    }
    static __device__ __forceinline__ float load_elt(Rsrc r, uint32_t off) {
        if constexpr (sizeof(T) == 2)
            return (float)__builtin_bit_cast(bf16, __builtin_amdgcn_raw_buffer_load_b16(r, off, 0, 0));
        else
            return load_f32(r, off);
    }

    // acc[i][j][r] holds row row0 + 32 i + rowoff(r), column col0 + 32 j.
    template <int TM, int TN>
    __device__ __forceinline__ void run(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int row0, int col0,
                                        int lane) {
        float bv[TN];
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = col0 + j * 32;
            bv[j] = (EPI == EPI_STORE || EPI == EPI_RES_F32) ? load_f32(bias, col < a.N ? col * 4 : OOB) : 0.f;
        }
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            float in[TN][16];
            if constexpr (EPI == EPI_RES_F32 || EPI == EPI_RELU_MASK || EPI == EPI_ACC_F32) {
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const int row = row0 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                        const int col = col0 + j * 32;
                        const bool ok = row < a.M && col < a.N;
                        if constexpr (EPI == EPI_RES_F32)
                            in[j][r] = load_f32(aux, ok ? (uint32_t)(((long)row * a.ldaux + col) * 4) : OOB);
                        else if constexpr (EPI == EPI_RELU_MASK)
                            in[j][r] = load_elt(aux, ok ? (uint32_t)(((long)row * a.ldaux + col) * sizeof(T)) : OOB);
                        else
                            in[j][r] = a.accumulate ? load_f32(c, ok ? (uint32_t)(((long)row * a.ldc + col) * 4) : OOB) : 0.f;
                    }
            }
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = row0 + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                    const int col = col0 + j * 32;
                    const bool ok = row < a.M && col < a.N;
                    const long e = (long)row * a.ldc + col;
                    float v = acc[i][j][r];
                    if constexpr (EPI == EPI_STORE) {
                        v += bv[j];
                        if (a.relu) v = fmaxf(v, 0.f);
                        store_elt(c, ok ? (uint32_t)(e * sizeof(T)) : OOB, v);
                    } else if constexpr (EPI == EPI_RES_F32) {
                        v += in[j][r] + bv[j];
                        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), c, ok ? (uint32_t)(e * 4) : OOB, 0, 0);
                        if (a.C2) store_elt(c2, ok ? (uint32_t)(((long)row * a.ldc2 + col) * sizeof(T)) : OOB, v);
                    } else if constexpr (EPI == EPI_F32) {
                        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), c, ok ? (uint32_t)(e * 4) : OOB, 0, 0);
                    } else if constexpr (EPI == EPI_RELU_MASK) {
                        store_elt(c, ok ? (uint32_t)(e * sizeof(T)) : OOB, in[j][r] > 0.f ? v : 0.f);
                    } else if constexpr (EPI == EPI_ACC_F32) {
                        v += in[j][r];
                        __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), c, ok ? (uint32_t)(e * 4) : OOB, 0, 0);
                    }
                }
        }
    }
};

// Epilogue of the split-K reduction (global pointers, element granularity).
template <typename T, int EPI>
__device__ __forceinline__ void epilogue(const GemmArgs& a, int row, int col, float v) {
    const long i = (long)row * a.ldc + col;
    if constexpr (EPI == EPI_STORE) {
        if (a.bias) v += a.bias[col];
        if (a.relu) v = fmaxf(v, 0.f);
        reinterpret_cast<T*>(a.C)[i] = to_elt<T>(v);
    } else if constexpr (EPI == EPI_RES_F32) {
        v += reinterpret_cast<const float*>(a.aux)[(long)row * a.ldaux + col];
        if (a.bias) v += a.bias[col];
        reinterpret_cast<float*>(a.C)[i] = v;
        if (a.C2) reinterpret_cast<T*>(a.C2)[(long)row * a.ldc2 + col] = to_elt<T>(v);
    } else if constexpr (EPI == EPI_F32) {
        reinterpret_cast<float*>(a.C)[i] = v;
    } else if constexpr (EPI == EPI_RELU_MASK) {
        const float z = to_f32(reinterpret_cast<const T*>(a.aux)[(long)row * a.ldaux + col]);
        reinterpret_cast<T*>(a.C)[i] = to_elt<T>(z > 0.f ? v : 0.f);
    } else if constexpr (EPI == EPI_ACC_F32) {
        float* c = reinterpret_cast<float*>(a.C) + i;
        *c = a.accumulate ? *c + v : v;
    }
}

template <typename T, int BM, int BN, bool AK, bool BKM, int EPI, bool SPLIT>
__global__ void __launch_bounds__(256) gemm_kernel(GemmArgs args) {
    constexpr int BK = GemmCfg<T>::BK, KS = BK / 16;
    constexpr int WM = 2, WN = 2;
    constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
    using LA = TileLoader<T, BM, BK, AK>;
    using LB = TileLoader<T, BN, BK, BKM>;
    __shared__ __attribute__((aligned(16))) char As[2][BM * 128];
    __shared__ __attribute__((aligned(16))) char Bs[2][BN * 128];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // XCD-aware tile order: workgroup b runs on XCD b % 8; give XCD x the
    // contiguous logical range [x G/8, (x+1) G/8) (tiles walk down M inside a
    // column of N tiles, so neighbours share the B panel).
    const int tiles_m = (args.M + BM - 1) / BM;
    const int G = gridDim.x;
    int bid = blockIdx.x;
    const int G8 = G & ~7;
    if (bid < G8) bid = (bid & 7) * (G8 >> 3) + (bid >> 3);
    const int tm = bid % tiles_m, tn = bid / tiles_m;
    const int m0 = tm * BM, n0 = tn * BN;

    const int nk_all = (args.K + BK - 1) / BK;
    int kt0 = 0, kt1 = nk_all;
    if constexpr (SPLIT) {
        const int per = (nk_all + gridDim.y - 1) / gridDim.y;
        kt0 = blockIdx.y * per;
        kt1 = min(nk_all, kt0 + per);
    }

    constexpr int ESZ = sizeof(T);
    const Rsrc A = make_rsrc(args.A, (uint32_t)((AK ? (long)(args.M - 1) * args.lda + args.K
                                                    : (long)(args.K - 1) * args.lda + args.M) * ESZ));
    const Rsrc B = make_rsrc(args.B, (uint32_t)((BKM ? (long)(args.N - 1) * args.ldb + args.K
                                                     : (long)(args.K - 1) * args.ldb + args.N) * ESZ));
    LA la;
    LB lb;
    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // Fused bias gradient of a weight-gradient GEMM: the workgroups of the
    // first M tile see every k-row of B (= dY) for their columns (of their k
    // range, under split-K: then the sums go to the partial area after the
    // split partial tiles, one row of N per split).
    constexpr bool COLSUM = !BKM && (EPI == EPI_ACC_F32 || SPLIT);
    const bool do_colsum = COLSUM && args.colsum != nullptr && tm == 0;
    float cs[LB::VEC];
#pragma unroll
    for (int i = 0; i < LB::VEC; ++i) cs[i] = 0.f;

    const int fr = lane & 31, fk = (lane >> 5) * 8 * ESZ;
    const int arow = wm * (BM / WM) + fr, brow = wn * (BN / WN) + fr;
    Frag<T> fa[2][TM], fb[2][TN];
    auto load_frags = [&](int slot, const char* as, const char* bs, int s) {
#pragma unroll
        for (int i = 0; i < TM; ++i) FragRead<T>::load(fa[slot][i], as, arow + i * 32, s * 16 * ESZ + fk);
#pragma unroll
        for (int j = 0; j < TN; ++j) FragRead<T>::load(fb[slot][j], bs, brow + j * 32, s * 16 * ESZ + fk);
    };

    if (kt0 < kt1) {
        la.load(A, args.lda, m0, args.M, kt0 * BK, args.K, tid);
        lb.load(B, args.ldb, n0, args.N, kt0 * BK, args.K, tid);
        la.store(As[0], tid);
        lb.store(Bs[0], tid);
        if (do_colsum) lb.colsum(cs);
        __syncthreads();
        load_frags(0, As[0], Bs[0], 0);
        for (int kt = kt0; kt < kt1; ++kt) {
            const int buf = (kt - kt0) & 1;
            const bool next = kt + 1 < kt1;
            if (next) {
                la.load(A, args.lda, m0, args.M, (kt + 1) * BK, args.K, tid);
                lb.load(B, args.ldb, n0, args.N, (kt + 1) * BK, args.K, tid);
            }
#pragma unroll
            for (int s = 0; s < KS; ++s) {
                const int cur = s & 1;
                if (s + 1 < KS) {
                    load_frags(cur ^ 1, As[buf], Bs[buf], s + 1);
                } else if (next) {
                    la.store(As[buf ^ 1], tid);
                    lb.store(Bs[buf ^ 1], tid);
                    if (do_colsum) lb.colsum(cs);
                    __syncthreads();
                    load_frags(cur ^ 1, As[buf ^ 1], Bs[buf ^ 1], 0);
                }
#pragma unroll
                for (int i = 0; i < TM; ++i)
#pragma unroll
                    for (int j = 0; j < TN; ++j) mma(acc[i][j], fa[cur][i], fb[cur][j]);
            }
        }
    }

    // 32x32 accumulator layout: lane l holds column (l % 32); register r holds
    // row 8 (r / 4) + 4 (l / 32) + (r % 4).
    if constexpr (COLSUM) {
        if (do_colsum) {
            // threads tid = mb + MBLK j (j = 0, 1, ...) hold partial sums of the
            // same VEC columns; add them in increasing tid order.
            constexpr int MBLK = LB::MBLK, VEC = LB::VEC;
            float* red = reinterpret_cast<float*>(&As[0][0]);
            __syncthreads();
#pragma unroll
            for (int i = 0; i < VEC; ++i) red[tid * VEC + i] = cs[i];
            __syncthreads();
            if (tid < BN) {
                const int mb = tid / VEC, i = tid % VEC;
                float sum = 0.f;
                for (int t = mb; t < 256; t += MBLK) sum += red[t * VEC + i];
                const int col = n0 + tid;
                if constexpr (SPLIT) {
                    if (col < args.N) args.ws[((long)gridDim.y * args.M + blockIdx.y) * args.N + col] = sum;
                } else {
                    if (col < args.N) args.colsum[col] = args.accumulate ? args.colsum[col] + sum : sum;
                }
            }
        }
    }
    if constexpr (SPLIT) {
        const Rsrc ws = make_rsrc(args.ws, (uint32_t)((long)gridDim.y * args.M * args.N * 4));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = n0 + wn * (BN / WN) + j * 32 + (lane & 31);
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = m0 + wm * (BM / WM) + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                    const bool ok = row < args.M && col < args.N;
                    const uint32_t o = ok ? (uint32_t)((((long)blockIdx.y * args.M + row) * args.N + col) * 4) : OOB;
                    // Read the accumulator element into a plain float first: a bit-cast
                    // taken directly on the AGPR-held vector element was compiled into
                    // stores that all read the block's first register.
                    const float v = acc[i][j][r];
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), ws, o, 0, 0);
                }
            }
    } else {
        Epilogue<T, EPI> ep;
        ep.init(args);
        ep.template run<TM, TN>(args, acc, m0 + wm * (BM / WM), n0 + wn * (BN / WN) + (lane & 31), lane);
    }
}

// ---------------------------------------------------------------------------
// Direct-to-LDS pipeline for bf16 GEMMs with both operands k-contiguous (the
// forward and input-gradient GEMMs).  Tiles are copied global -> LDS with
// buffer_load_dwordx4 ... lds: each wave instruction fills 8 rows (1 KB) of a
// stage and each lane fetches the global 16-byte chunk that belongs at its
// (swizzled) LDS position, so no VGPRs hold staged data and no ds_write is
// issued.  NSTAGE stages form a ring; k-tile t + NSTAGE - 1 is in flight while
// tile t is consumed.  Waits use explicit vmcnt values (loads complete in
// order), and the single barrier per k-tile precedes the last k-step's MFMAs.
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
    static_assert(N >= 0 && N < 64, "vmcnt");
    __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}
__device__ __forceinline__ void wait_vmcnt_dyn(int n) {
    switch (n) {
    case 0: wait_vmcnt<0>(); break;
    case 4: wait_vmcnt<4>(); break;
    case 5: wait_vmcnt<5>(); break;
    case 6: wait_vmcnt<6>(); break;
    case 10: wait_vmcnt<10>(); break;
    case 20: wait_vmcnt<20>(); break;
    case 8: wait_vmcnt<8>(); break;
    case 12: wait_vmcnt<12>(); break;
    case 16: wait_vmcnt<16>(); break;
    case 24: wait_vmcnt<24>(); break;
    case 32: wait_vmcnt<32>(); break;
    case 48: wait_vmcnt<48>(); break;
    default: wait_vmcnt<0>(); break;
    }
}

// All waves of the workgroup meet once every LDS read of this wave has
// returned.  No memory fence: a fence would also wait for every outstanding
// direct-to-LDS load of the wave (vmcnt(0)) and so drain the prefetch ring;
// the loads a k-tile needs are waited for explicitly (wait_vmcnt) before.
// The memory clobber keeps the compiler from moving LDS accesses across it.
__device__ __forceinline__ void lds_barrier() {
    asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory");
}

typedef __attribute__((address_space(3))) void* LdsPtr;

// P direct loads of 8 rows (1 KB) each into consecutive LDS blocks at dst;
// lane offsets vo[i] are fixed, the k advance is the scalar offset so.
template <int P>
__device__ __forceinline__ void dl_load_blocks(Rsrc g, const uint32_t* vo, int so, char* dst) {
#pragma unroll
    for (int i = 0; i < P; ++i) __builtin_amdgcn_raw_ptr_buffer_load_lds(g, (LdsPtr)(dst + i * 1024), 16, vo[i], so, 0, 0);
}
// 1 KB direct-to-LDS blocks, each from its own buffer resource
template <int P>
__device__ __forceinline__ void dl_load_rsrcs(const Rsrc* g, const uint32_t* vo, int so, char* dst) {
#pragma unroll
    for (int i = 0; i < P; ++i) __builtin_amdgcn_raw_ptr_buffer_load_lds(g[i], (LdsPtr)(dst + i * 1024), 16, vo[i], so, 0, 0);
}

// The direct loads of one k-tile that go out in k-step `part` of KS: load
// slot q (PA A blocks, then PB B blocks, then F fp4 blocks, 1 KB each at the
// wave's place in the stage) belongs to k-step q KS / LPW.
template <int PA, int PB, int F, int LPW, int KS, int BM, int STAGE_BF>
__device__ __forceinline__ void dl_issue_part(int part, Rsrc A, Rsrc B, const uint32_t* voa, const uint32_t* vob,
                                              const Rsrc* R4, const uint32_t* vo4, int soa, int sob, int so4,
                                              char* st, int wave) {
#pragma unroll
    for (int q = 0; q < LPW; ++q) {
        if (q * KS / LPW != part) continue;
        if (q < PA) {
            __builtin_amdgcn_raw_ptr_buffer_load_lds(A, (LdsPtr)(st + (wave * PA + q) * 1024), 16, voa[q < PA ? q : 0], soa, 0, 0);
        } else if (q < PA + PB) {
            const int b = q - PA;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(B, (LdsPtr)(st + BM * 128 + (wave * PB + b) * 1024), 16,
                                                     vob[b < PB ? b : 0], sob, 0, 0);
        } else if constexpr (F > 0) {
            const int f = q - PA - PB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(R4[f < F ? f : 0], (LdsPtr)(st + STAGE_BF + (wave * F + f) * 1024), 16,
                                                     vo4[f < F ? f : 0], so4, 0, 0);
        }
    }
}

// Wave index as a wave-uniform (scalar) value, so LDS base addresses derived
// from it stay in SGPRs (M0 of the direct loads).
__device__ __forceinline__ int uniform_wave_id(int tid) { return __builtin_amdgcn_readfirstlane(tid >> 6); }

// Epilogue of a tile lying entirely inside C: per-lane column offsets are
// computed once; the row part of every offset is wave-uniform and passed as
// the buffer instruction's scalar offset.
template <int TM, int TN, int EPI>
__device__ __forceinline__ void dl_epilogue_full(const GemmArgs& a, const f32x16 (&acc)[TM][TN], int row0, int col0,
                                                 int lane) {
    constexpr bool OUT_F32 = EPI == EPI_RES_F32 || EPI == EPI_F32;
    const int h = lane >> 5;
    const uint32_t osz = OUT_F32 ? 4 : 2;
    const long big = (long)(a.M - 1) * a.ldc + a.N;
    const Rsrc c = make_rsrc(a.C, (uint32_t)(big * osz));
    const uint32_t vc = (uint32_t)(((long)(row0 + 4 * h) * a.ldc + col0) * osz);
    float bv[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) bv[j] = (EPI == EPI_STORE || EPI == EPI_RES_F32) && a.bias ? a.bias[col0 + j * 32] : 0.f;
    Rsrc aux, c2;
    uint32_t va = 0, vc2 = 0;
    if constexpr (EPI == EPI_RES_F32) {
        aux = make_rsrc(a.aux, (uint32_t)(((long)(a.M - 1) * a.ldaux + a.N) * 4));
        va = (uint32_t)(((long)(row0 + 4 * h) * a.ldaux + col0) * 4);
        c2 = make_rsrc(a.C2, a.C2 ? (uint32_t)(((long)(a.M - 1) * a.ldc2 + a.N) * 2) : 0u);
        vc2 = (uint32_t)(((long)(row0 + 4 * h) * a.ldc2 + col0) * 2);
    } else if constexpr (EPI == EPI_RELU_MASK) {
        aux = make_rsrc(a.aux, (uint32_t)(((long)(a.M - 1) * a.ldaux + a.N) * 2));
        va = (uint32_t)(((long)(row0 + 4 * h) * a.ldaux + col0) * 2);
    }
#pragma unroll
    for (int i = 0; i < TM; ++i) {
        float in[TN][16];
        if constexpr (EPI == EPI_RES_F32 || EPI == EPI_RELU_MASK) {
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int dr = i * 32 + (r >> 2) * 8 + (r & 3);
                    if constexpr (EPI == EPI_RES_F32)
                        in[j][r] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                                                                 aux, va, (dr * a.ldaux + j * 32) * 4, 0));
                    else
                        in[j][r] = (float)__builtin_bit_cast(
                            bf16, __builtin_amdgcn_raw_buffer_load_b16(aux, va, (dr * a.ldaux + j * 32) * 2, 0));
                }
        }
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int dr = i * 32 + (r >> 2) * 8 + (r & 3);
                const int so = (dr * a.ldc + j * 32) * osz;
                float v = acc[i][j][r];
                if constexpr (EPI == EPI_STORE) {
                    v += bv[j];
                    if (a.relu) v = fmaxf(v, 0.f);
                    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, (bf16)v), c, vc, so, 0);
                } else if constexpr (EPI == EPI_RES_F32) {
                    v += in[j][r] + bv[j];
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), c, vc, so, 0);
                    if (a.C2)
                        __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, (bf16)v), c2, vc2,
                                                              (dr * a.ldc2 + j * 32) * 2, 0);
                } else if constexpr (EPI == EPI_F32) {
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), c, vc, so, 0);
                } else if constexpr (EPI == EPI_RELU_MASK) {
                    v = in[j][r] > 0.f ? v : 0.f;
                    __builtin_amdgcn_raw_buffer_store_b16(__builtin_bit_cast(unsigned short, (bf16)v), c, vc, so, 0);
                }
            }
    }
}

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16* LdsV4;

// Two transposing LDS reads (ds_read_b64_tr_b16) make one bf16 MFMA fragment
// from a k-row-major tile: each gives the lane 4 consecutive k of its m.
__device__ __forceinline__ bf16x8 tr_frag(const char* p, int second) {
    const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LdsV4)(p));
    const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((LdsV4)(p + second));
    const bf16x4 a = __builtin_bit_cast(bf16x4, lo), b = __builtin_bit_cast(bf16x4, hi);
    return bf16x8{a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
}

// Direct-to-LDS GEMM (requires K % 64 == 0).  KM: both operands k-contiguous
// (A[m lda + k], B[n ldb + k]: forward and input-gradient GEMMs); else both
// m/n-contiguous (A[k lda + m], B[k ldb + n]: weight-gradient GEMMs, read as
// the activations are stored).
//   KM:  a stage holds rows of 64 k (128 bytes) per m, 16-byte chunks
//        XOR-swizzled by swz(row); fragments are plain 16-byte LDS reads.
//   !KM: a stage holds rows of W m-values per k (2W bytes), 16-byte chunk c of
//        row k stored at c ^ 4 (k % 4); fragments come from transposing reads
//        (tr_frag), whose four k-rows then fall in distinct bank groups.
// Address arithmetic is hoisted: each lane's global offsets are computed once
// and the k advance rides in the scalar offset of the buffer load; M0 (the LDS
// destination) is wave-uniform; fragment offsets are precomputed and the stage
// base folds into the ds_read immediate because the k-tile loop is unrolled
// over the stages.
//   MX: the fp4 correction term of GemmArgs (a4, b4, sa4, sb4).  Each stage
//   also holds the k-tile's 32 bytes (64 e2m1 values) of every A and B row,
//   loaded directly like the bf16 tiles (16-byte chunk h of row r at slot
//   2 r + (h ^ sw4(r))); once per k-tile each output block takes one
//   v_mfma_scale_f32_32x32x64_f8f6f4 into the same fp32 accumulator, the
//   per-lane scale being the E8M0 byte of the lane's row (A) or column (B),
//   which are loaded once, before the k loop.
//   KG: k-groups.  With KG = 2 the workgroup holds two groups of WM x WN
//   waves (two per SIMD for 4-wave groups); group g takes k-tiles g, g + 2,
//   ... of the same output tile through its own stage ring, both groups in
//   lockstep (one workgroup barrier per k-tile each), and at the end group 1
//   hands its accumulators to group 0 through LDS, which adds them and runs
//   the epilogue.  The k-tile count must be a multiple of KG.
// F16: A and B hold fp16 values (k-contiguous, no fp4 stage, one k-group).
template <int BM, int BN, int WM, int WN, int NSTAGE, int EPI, int SM, bool KM, bool MX = false, int KG = 1,
          bool F16 = false>
__global__ void __launch_bounds__(64 * WM * WN * KG) gemm_dl(GemmArgs args) {
    static_assert(!F16 || (KM && !MX && KG == 1), "fp16 operands: k-contiguous, no fp4 stage, one k-group");
    // SM: 0 no split-K; 1 split-K, partial tiles only (summed by splitk_reduce)
    constexpr bool SPLIT = SM != 0;
    constexpr int BK = 64, KS = 4, NW = WM * WN;  // NW: waves per k-group
    static_assert(KG == 1 || (KG == 2 && KM && !MX && !SPLIT), "k-groups: k-contiguous, unsplit, bf16 only");
    constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
    constexpr int STAGE_BF = (BM + BN) * 128;
    constexpr int STAGE = STAGE_BF + (MX ? (BM + BN) * 32 : 0);
    constexpr int PA = BM / (8 * NW), PB = BN / (8 * NW);  // 1 KB load blocks per wave for A and B
    static_assert(PA * 8 * NW == BM && PB * 8 * NW == BN, "load blocks");
    // m-contiguous tiles swizzle 16-byte chunks by 4 (k % 4): rows need >= 16 chunks
    static_assert(KM || (BM >= 128 && BN >= 128), "m-contiguous tiles must be at least 128 wide");
    constexpr int NL4 = MX ? (BM + BN) * 2 / (64 * NW) : 0;  // 1 KB fp4 load blocks per wave
    static_assert(!MX || (KM && NL4 * 64 * NW == (BM + BN) * 2 && (2 * BM) % 64 == 0), "fp4 load blocks");
    static_assert(KG * NSTAGE * STAGE <= 160 * 1024, "LDS");
    static_assert(KG == 1 || BM * BN * 4 <= NSTAGE * STAGE * KG, "LDS for the k-group hand-over");
    constexpr int LPW = PA + PB + NL4;         // load instructions per wave per k-tile
    __shared__ __attribute__((aligned(1024))) char smem_all[KG * NSTAGE * STAGE];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave_all = uniform_wave_id(tid);
    const int kg = wave_all / NW, wave = wave_all % NW;  // k-group, wave within the group
    char* const smem = smem_all + kg * NSTAGE * STAGE;   // the group's stage ring
    const int wm = wave / WN, wn = wave % WN;
    const int tiles_m = (args.M + BM - 1) / BM;
    const int G = gridDim.x;
    int bid = blockIdx.x;
    const int G8 = G & ~7;
    if (bid < G8) bid = (bid & 7) * (G8 >> 3) + (bid >> 3);
    // XCD x now holds a contiguous run of ids; number the tiles in bands of
    // H tile rows, column by column within a band, so that the tiles one XCD
    // runs at a time form a compact block (4 x 8 for 32 workgroups) and its
    // L2 serves each A row panel and B column panel to several of them
    // (a run down whole tile columns would stream all of A through every XCD)
    // The band height H suits the tiles an XCD runs at once (P: its 32 CUs
    // times the workgroups that fit a CU): about sqrt(P BN / BM) rows.
    constexpr int RES = (160 * 1024) / (KG * NSTAGE * STAGE) < 1 ? 1 : (160 * 1024) / (KG * NSTAGE * STAGE);
    const int P = min(max(G >> 3, 1), 32 * min(RES, 3));
    const int H = P * BN >= 64 * BM ? 8 : 4;
    const int tiles_n = (args.N + BN - 1) / BN;
    const int band = bid / (H * tiles_n), in_band = bid - band * H * tiles_n;
    const int bh = min(H, tiles_m - band * H);
    const int tm = band * H + in_band % bh, tn = in_band / bh;
    const int m0 = tm * BM, n0 = tn * BN;

    const int nk_all = args.K / BK;
    int kt0 = 0, kt1 = nk_all;
    if constexpr (SPLIT) {
        const int per = (nk_all + gridDim.y - 1) / gridDim.y;
        kt0 = blockIdx.y * per;
        kt1 = min(nk_all, kt0 + per);
    }
    // group-local k-tile i is global k-tile kt0 + i KG + kg
    const int nkt = (kt1 - kt0) / KG;
    kt0 += kg;

    Rsrc A, B;
    uint32_t voa[PA], vob[PB];
    int ka, kb;  // bytes per k-tile advance of A and B
    if constexpr (KM) {
        A = make_rsrc(args.A, (uint32_t)(((long)(args.M - 1) * args.lda + args.K) * 2));
        B = make_rsrc(args.B, (uint32_t)(((long)(args.N - 1) * args.ldb + args.K) * 2));
#pragma unroll
        for (int i = 0; i < PA; ++i) {
            const int r = (wave * PA + i) * 8 + (lane >> 3);
            const int row = m0 + r;
            voa[i] = row < args.M ? (uint32_t)(((long)row * args.lda + ((lane & 7) ^ swz(r)) * 8) * 2) : OOB;
        }
#pragma unroll
        for (int i = 0; i < PB; ++i) {
            const int r = (wave * PB + i) * 8 + (lane >> 3);
            const int row = n0 + r;
            vob[i] = row < args.N ? (uint32_t)(((long)row * args.ldb + ((lane & 7) ^ swz(r)) * 8) * 2) : OOB;
        }
        ka = kb = BK * 2;
    } else {
        A = make_rsrc(args.A, (uint32_t)(((long)(args.K - 1) * args.lda + args.M) * 2));
        B = make_rsrc(args.B, (uint32_t)(((long)(args.K - 1) * args.ldb + args.N) * 2));
#pragma unroll
        for (int i = 0; i < PA; ++i) {
            const int pos = (wave * PA + i) * 1024 + 16 * lane;
            const int k = pos / (2 * BM), c = ((pos % (2 * BM)) >> 4) ^ ((k & 3) << 2);
            const int m = m0 + 8 * c;
            voa[i] = m < args.M ? (uint32_t)(((long)k * args.lda + m) * 2) : OOB;
        }
#pragma unroll
        for (int i = 0; i < PB; ++i) {
            const int pos = (wave * PB + i) * 1024 + 16 * lane;
            const int k = pos / (2 * BN), c = ((pos % (2 * BN)) >> 4) ^ ((k & 3) << 2);
            const int n = n0 + 8 * c;
            vob[i] = n < args.N ? (uint32_t)(((long)k * args.ldb + n) * 2) : OOB;
        }
        ka = (int)(BK * args.lda * 2);
        kb = (int)(BK * args.ldb * 2);
    }
    // fp4 correction operands: per-lane chunk offsets, and the scales of the
    // lane's rows (A) and columns (B), issued before the bf16 prologue so
    // that the prologue's wait covers them
    // (a conditional expression over buffer resources drops the kernel's host
    // stub: the operand is chosen by pointer and size, one resource per block)
    constexpr int NL4A = NL4 > 0 ? NL4 : 1;
    Rsrc R4[NL4A];
    uint32_t vo4[NL4A];
    int sca[TM], scb[TN];
    if constexpr (MX) {
        const int kb4 = args.K / 2;  // bytes per fp4 row
#pragma unroll
        for (int p = 0; p < NL4; ++p) {
            const int blk = wave * NL4 + p;     // 64 chunks per block, never straddling A and B
            const int c = blk * 64 + lane;
            const bool isa = blk * 64 < 2 * BM;
            const int cc = isa ? c : c - 2 * BM, r = cc >> 1;
            const int row = (isa ? m0 : n0) + r, lim = isa ? args.M : args.N;
            R4[p] = make_rsrc(isa ? args.a4 : args.b4, (uint32_t)((long)lim * kb4));
            vo4[p] = row < lim ? (uint32_t)((long)row * kb4 + (((cc & 1) ^ sw4(r)) << 4)) : OOB;
        }
        const Rsrc SA = make_rsrc(args.sa4, (uint32_t)args.M);
        const Rsrc SB = make_rsrc(args.sb4, (uint32_t)args.N);
#pragma unroll
        for (int i = 0; i < TM; ++i)
            sca[i] = __builtin_amdgcn_raw_buffer_load_b8(SA, (uint32_t)(m0 + wm * (BM / WM) + i * 32 + (lane & 31)), 0, 0);
#pragma unroll
        for (int j = 0; j < TN; ++j)
            scb[j] = __builtin_amdgcn_raw_buffer_load_b8(SB, (uint32_t)(n0 + wn * (BN / WN) + j * 32 + (lane & 31)), 0, 0);
    }
#define GP_DL_ISSUE(t, st)                                                                   \
    do {                                                                                     \
        dl_load_blocks<PA>(A, voa, (kt0 + ((t) - kt0) * KG) * ka, (st) + wave * PA * 1024);  \
        dl_load_blocks<PB>(B, vob, (kt0 + ((t) - kt0) * KG) * kb, (st) + BM * 128 + wave * PB * 1024); \
        if constexpr (MX) dl_load_rsrcs<NL4>(R4, vo4, (t) * 32, (st) + STAGE_BF + wave * NL4 * 1024); \
    } while (0)

    // Rings of 3+ stages spread a tile's direct loads over the KS k-steps of
    // the tile after the one whose stage they refill: load slot q (A blocks,
    // then B blocks, then fp4 blocks) goes out in k-step q KS / LPW.  Issued
    // in one burst right after the barrier, the loads of all waves queued at
    // the CU's texture unit together and held up the MFMAs behind them.
    constexpr bool SPREAD = NSTAGE >= 3;
#define GP_DL_ISSUE_PART(t, st, part)                                                                        \
    dl_issue_part<PA, PB, (MX ? NL4 : 0), LPW, KS, BM, STAGE_BF>((part), A, B, voa, vob, R4, vo4,               \
                                                                 (kt0 + ((t) - kt0) * KG) * ka,                  \
                                                                 (kt0 + ((t) - kt0) * KG) * kb, (t) * 32, (st), wave)

    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    // Fragment byte offsets within a stage.  KM: the lane's fragment of block
    // i, k-step s is chunk (2 s + h) ^ swz(row) of row r = wm (BM / WM) + 32 i + fr.
    // swz reads bits 0..5 of r: bits 0..4 are fr's, and bit 5 is the parity
    // p of (wm (BM / WM)) / 32 + i.  So swz(r) = w ^ 4 p with w = swz(fr), and
    // the offset is base + 4096 i + ((s ^ (w >> 1) ^ 2 p) << 5), the chunk's
    // low bit h ^ (w & 1) folded into the base: per operand a base and a
    // per-lane term with the wave's parity in it, the block's parity an XOR
    // with 64 -- instead of one register per (k-step, block).
    // !KM: k-step s moves the fragment down 16 k-rows, a constant stride, and
    // leaves the k-row's swizzle (k % 4) unchanged: one offset per block.
    const int fr = lane & 31, h = lane >> 5;
    int fa_base = 0, fb_base = 0, swa = 0, swb = 0;
    int fa_off[KM ? 1 : TM], fb_off[KM ? 1 : TN];
    if constexpr (KM) {
        const int w = swz(fr);
        fa_base = (wm * (BM / WM) + fr) * 128 + ((h ^ (w & 1)) << 4);
        fb_base = BM * 128 + (wn * (BN / WN) + fr) * 128 + ((h ^ (w & 1)) << 4);
        swa = (w >> 1) ^ ((((wm * (BM / WM)) >> 5) & 1) << 1);
        swb = (w >> 1) ^ ((((wn * (BN / WN)) >> 5) & 1) << 1);
    } else {
        // lane l of a 16-lane group g = l / 16 addresses k-row 8 (g / 2) + (l % 16) / 4
        // and m 16 (g % 2) + 4 (l % 4) of its fragment (plus 4 k-rows for the second read)
        const int g = lane >> 4, q = lane & 15;
        const int kr = 8 * (g >> 1) + (q >> 2), mo = 16 * (g & 1) + 4 * (q & 3);
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int m = wm * (BM / WM) + i * 32 + mo;
            fa_off[i] = kr * (2 * BM) + ((((m >> 3) ^ ((kr & 3) << 2))) << 4) + (m & 7) * 2;
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int n = wn * (BN / WN) + j * 32 + mo;
            fb_off[j] = BM * 128 + kr * (2 * BN) + ((((n >> 3) ^ ((kr & 3) << 2))) << 4) + (n & 7) * 2;
        }
    }
    int f4a_off[TM], f4b_off[TN];
    if constexpr (MX) {
#pragma unroll
        for (int i = 0; i < TM; ++i) {
            const int r = wm * (BM / WM) + i * 32 + fr;
            f4a_off[i] = STAGE_BF + (2 * r + (h ^ sw4(r))) * 16;
        }
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int r = wn * (BN / WN) + j * 32 + fr;
            f4b_off[j] = STAGE_BF + (2 * BM + 2 * r + (h ^ sw4(r))) * 16;
        }
    }
    Frag<bf16> fa[2][TM], fb[2][TN];
    auto load_frags = [&](int slot, const char* stg, int s) {
        if constexpr (KM) {
            const int ta = (s ^ swa) << 5, tb = (s ^ swb) << 5;
            const char* pa[2] = {stg + fa_base + ta, stg + fa_base + (ta ^ 64)};
            const char* pb[2] = {stg + fb_base + tb, stg + fb_base + (tb ^ 64)};
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[slot][i].v = *reinterpret_cast<const bf16x8*>(pa[i & 1] + i * 4096);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[slot][j].v = *reinterpret_cast<const bf16x8*>(pb[j & 1] + j * 4096);
        } else {
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[slot][i].v = tr_frag(stg + fa_off[i] + s * 32 * BM, 4 * 2 * BM);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[slot][j].v = tr_frag(stg + fb_off[j] + s * 32 * BN, 4 * 2 * BN);
        }
    };

    // Fused bias gradient (weight-gradient GEMMs): the waves of the first M-tile
    // with wm == 0 hold every k of their B columns in their fragments.
    constexpr bool COLSUM = !KM && (EPI == EPI_ACC_F32 || SPLIT);
    const bool do_colsum = COLSUM && args.colsum != nullptr && tm == 0 && wm == 0;
    float cs[TN];
#pragma unroll
    for (int j = 0; j < TN; ++j) cs[j] = 0.f;

    if (nkt > 0) {
        // prologue: fill every stage; wait for tile 0 (tiles 1 .. NSTAGE-1 may be in flight)
#pragma unroll
        for (int p = 0; p < NSTAGE; ++p)
            if (p < nkt) GP_DL_ISSUE(kt0 + p, smem + p * STAGE);
        if (nkt >= NSTAGE)
            wait_vmcnt<(NSTAGE - 1) * LPW>();
        else
            wait_vmcnt<0>();
        if constexpr (MX) pin_vgprs<TM, TN>(sca, scb);
        lds_barrier();
        load_frags(0, smem, 0);
        for (int i0 = 0; i0 < nkt; i0 += NSTAGE) {
#pragma unroll
            for (int st = 0; st < NSTAGE; ++st) {
                const int i = i0 + st;
                if (i >= nkt) break;
                const char* stg = smem + st * STAGE;
                const char* nxt = smem + ((st + 1) % NSTAGE) * STAGE;
#pragma unroll
                for (int s = 0; s < KS; ++s) {
                    const int cur = s & 1;
                    if constexpr (SPREAD) {
                        // part s of tile i - 1 + NSTAGE, into the stage tile i - 1 left
                        if (i >= 1 && i - 1 + NSTAGE < nkt)
                            GP_DL_ISSUE_PART(kt0 + i - 1 + NSTAGE, smem + ((st + NSTAGE - 1) % NSTAGE) * STAGE, s);
                    }
                    if constexpr (COLSUM) {
                        if (do_colsum) {
#pragma unroll
                            for (int j = 0; j < TN; ++j)
#pragma unroll
                                for (int e = 0; e < 8; ++e) cs[j] += (float)fb[cur][j].v[e];
                        }
                    }
                    if (s + 1 < KS) {
                        load_frags(cur ^ 1, stg, s + 1);
                    } else {
                        // Tiles issued: 0 .. min(i + NSTAGE - 1, nkt - 1).  Tile i+1 must have
                        // landed (tiles i+2 .. i+NSTAGE-1 may be in flight; near the end of
                        // the ring everything is waited for); then every wave is past tile i,
                        // whose stage is refilled with tile i + NSTAGE.  Branch-free around
                        // the LDS reads; on the last tile the fragment read is unused.
                        if (i + NSTAGE - 1 < nkt)
                            wait_vmcnt<(NSTAGE - 2) * LPW>();
                        else
                            wait_vmcnt<0>();
                        lds_barrier();
                        if constexpr (!SPREAD) {
                            if (i + NSTAGE < nkt) GP_DL_ISSUE(kt0 + i + NSTAGE, smem + st * STAGE);
                        }
                        load_frags(cur ^ 1, nxt, 0);
                    }
                    i32x4 a4[MX ? TM : 1], b4[MX ? TN : 1];
                    if constexpr (MX) {
                        if (s == 1) {
#pragma unroll
                            for (int ii = 0; ii < TM; ++ii) a4[ii] = *reinterpret_cast<const i32x4*>(stg + f4a_off[ii]);
#pragma unroll
                            for (int j = 0; j < TN; ++j) b4[j] = *reinterpret_cast<const i32x4*>(stg + f4b_off[j]);
                        }
                    }
                    // The next k-step's fragment reads stay ahead of this
                    // k-step's MFMAs (left to itself the scheduler sinks them
                    // below the MFMAs into the same registers, which exposes
                    // the LDS latency once per k-step).
                    __builtin_amdgcn_sched_barrier(0);
#pragma unroll
                    for (int ii = 0; ii < TM; ++ii)
#pragma unroll
                        for (int j = 0; j < TN; ++j) {
                            if constexpr (F16)
                                mma16(acc[ii][j], fa[cur][ii], fb[cur][j]);
                            else
                                mma(acc[ii][j], fa[cur][ii], fb[cur][j]);
                        }
                    if constexpr (MX) {
                        if (s == 1) {
#pragma unroll
                            for (int ii = 0; ii < TM; ++ii)
#pragma unroll
                                for (int j = 0; j < TN; ++j) mma_fp4(acc[ii][j], a4[ii], b4[j], sca[ii], scb[j]);
                        }
                    }
                }
            }
        }
    }

#undef GP_DL_ISSUE
#undef GP_DL_ISSUE_PART
    if constexpr (KG == 2) {
        // group 1 hands its partial sums to group 0 through the (now idle) stage rings;
        // lane-fastest layout, so both the writes and the reads are conflict-free
        float* red = reinterpret_cast<float*>(smem_all) + (long)(wm * WN + wn) * TM * TN * 16 * 64 + lane;
        lds_barrier();
        if (kg == 1) {
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j)
#pragma unroll
                    for (int r = 0; r < 16; ++r) {
                        const float v = acc[i][j][r];
                        red[((i * TN + j) * 16 + r) * 64] = v;
                    }
        }
        lds_barrier();
        if (kg == 1) return;
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc[i][j][r] += red[((i * TN + j) * 16 + r) * 64];
    }
    const int row0 = m0 + wm * (BM / WM), col0 = n0 + wn * (BN / WN) + (lane & 31);
    if constexpr (COLSUM) {
        // lanes l and l + 32 hold the two k-halves of column l % 32
#pragma unroll
        for (int j = 0; j < TN; ++j) cs[j] += __shfl_xor(cs[j], 32);
        if (do_colsum && lane < 32) {
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = col0 + j * 32;
                if (col < args.N) {
                    if constexpr (SPLIT)
                        args.ws[((long)gridDim.y * args.M + blockIdx.y) * args.N + col] = cs[j];
                    else
                        args.colsum[col] = args.accumulate ? args.colsum[col] + cs[j] : cs[j];
                }
            }
        }
    }
    if constexpr (SPLIT) {
        const Rsrc ws = make_rsrc(args.ws, (uint32_t)((long)gridDim.y * args.M * args.N * 4));
#pragma unroll
        for (int i = 0; i < TM; ++i)
#pragma unroll
            for (int j = 0; j < TN; ++j) {
                const int col = col0 + j * 32;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int row = row0 + i * 32 + (r >> 2) * 8 + h * 4 + (r & 3);
                    const bool ok = row < args.M && col < args.N;
                    const uint32_t o = ok ? (uint32_t)((((long)blockIdx.y * args.M + row) * args.N + col) * 4) : OOB;
                    const float v = acc[i][j][r];  // see the note in gemm_kernel
                    __builtin_amdgcn_raw_buffer_store_b32(__builtin_bit_cast(int, v), ws, o, 0, 0);
                }
            }
    } else {
        if (EPI != EPI_ACC_F32 && m0 + BM <= args.M && n0 + BN <= args.N) {
            dl_epilogue_full<TM, TN, EPI>(args, acc, row0, col0, lane);
        } else {
            Epilogue<bf16, EPI> ep;
            ep.init(args);
            ep.template run<TM, TN>(args, acc, row0, col0, lane);
        }
    }
}

// Sum the split-K partials in split order and apply the epilogue; 4 columns
// per thread.  An accumulating (weight-gradient) GEMM with fused bias
// gradient also sums the splits' column-sum rows, stored after the partial
// tiles, into colsum.
template <typename T, int EPI>
__global__ void __launch_bounds__(256) splitk_reduce(GemmArgs args, int splits) {
    const long nq = (long)args.M * (args.N / 4);
    const long plane = (long)args.M * args.N;
    if constexpr (EPI == EPI_ACC_F32) {
        if (args.colsum) {
            for (long c = ((long)blockIdx.x * 256 + threadIdx.x) * 4; c < args.N; c += (long)gridDim.x * 256 * 4) {
                const float* p = args.ws + (long)splits * plane + c;
                f32x4 v = *reinterpret_cast<const f32x4*>(p);
                for (int k = 1; k < splits; ++k) {
                    const f32x4 t = *reinterpret_cast<const f32x4*>(p + (long)k * args.N);
                    v += t;
                }
                f32x4* o = reinterpret_cast<f32x4*>(args.colsum + c);
                if (args.accumulate) v += *o;
                *o = v;
            }
        }
    }
    for (long i = (long)blockIdx.x * 256 + threadIdx.x; i < nq; i += (long)gridDim.x * 256) {
        const int row = (int)(i / (args.N / 4)), col = (int)(i % (args.N / 4)) * 4;
        const float* p = args.ws + (long)row * args.N + col;
        f32x4 s = *reinterpret_cast<const f32x4*>(p);
        for (int k = 1; k < splits; ++k) {
            const f32x4 t = *reinterpret_cast<const f32x4*>(p + k * plane);
            s += t;
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) epilogue<T, EPI>(args, row, col + j, s[j]);
    }
}

// The same reduction with 16-byte accesses throughout (every leading
// dimension a multiple of 4 and every base 16-byte aligned, which the host
// checks): thread t of a block owns columns 4 t .. 4 t + 3 of a 1024-column
// chunk (blockIdx.x) over `rows` consecutive rows (blockIdx.y), so no index
// division is needed and each row of partials is read as whole 4 KB runs.
template <int EPI>
__global__ void __launch_bounds__(256) splitk_reduce_v4(GemmArgs args, int splits, int rows) {
    const int col = blockIdx.x * 1024 + threadIdx.x * 4;
    if (col >= args.N) return;
    const long plane = (long)args.M * args.N;
    if constexpr (EPI == EPI_ACC_F32) {
        if (args.colsum && blockIdx.y == 0) {
            const float* p = args.ws + (long)splits * plane + col;
            f32x4 v = *reinterpret_cast<const f32x4*>(p);
            for (int k = 1; k < splits; ++k) v += *reinterpret_cast<const f32x4*>(p + (long)k * args.N);
            f32x4* o = reinterpret_cast<f32x4*>(args.colsum + col);
            if (args.accumulate) v += *o;
            *o = v;
        }
    }
    f32x4 bv = {0.f, 0.f, 0.f, 0.f};
    if constexpr (EPI == EPI_STORE || EPI == EPI_RES_F32)
        if (args.bias) bv = *reinterpret_cast<const f32x4*>(args.bias + col);
    const int r0 = blockIdx.y * rows, r1 = min(args.M, r0 + rows);
    for (int row = r0; row < r1; ++row) {
        const float* p = args.ws + (long)row * args.N + col;
        f32x4 s = *reinterpret_cast<const f32x4*>(p);
        for (int k = 1; k < splits; ++k) s += *reinterpret_cast<const f32x4*>(p + (long)k * plane);
        const long i = (long)row * args.ldc + col;
        if constexpr (EPI == EPI_STORE) {
            s += bv;
            if (args.relu)
#pragma unroll
                for (int j = 0; j < 4; ++j) s[j] = fmaxf(s[j], 0.f);
            *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(args.C) + i) = {(bf16)s[0], (bf16)s[1], (bf16)s[2], (bf16)s[3]};
        } else if constexpr (EPI == EPI_RES_F32) {
            s += *reinterpret_cast<const f32x4*>(reinterpret_cast<const float*>(args.aux) + (long)row * args.ldaux + col) + bv;
            *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(args.C) + i) = s;
            if (args.C2)
                *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(args.C2) + (long)row * args.ldc2 + col) =
                    {(bf16)s[0], (bf16)s[1], (bf16)s[2], (bf16)s[3]};
        } else if constexpr (EPI == EPI_F32) {
            *reinterpret_cast<f32x4*>(reinterpret_cast<float*>(args.C) + i) = s;
        } else if constexpr (EPI == EPI_RELU_MASK) {
            const bf16x4 z = *reinterpret_cast<const bf16x4*>(reinterpret_cast<const bf16*>(args.aux) + (long)row * args.ldaux + col);
            *reinterpret_cast<bf16x4*>(reinterpret_cast<bf16*>(args.C) + i) = {
                (bf16)((float)z[0] > 0.f ? s[0] : 0.f), (bf16)((float)z[1] > 0.f ? s[1] : 0.f),
                (bf16)((float)z[2] > 0.f ? s[2] : 0.f), (bf16)((float)z[3] > 0.f ? s[3] : 0.f)};
        } else if constexpr (EPI == EPI_ACC_F32) {
            f32x4* c = reinterpret_cast<f32x4*>(reinterpret_cast<float*>(args.C) + i);
            if (args.accumulate) s += *c;
            *c = s;
        }
    }
}

enum TileCfg {
    T256x256 = 0, T256x128 = 1, T128x256 = 2, T128x128 = 3,  // register-staged (any operand form)
    T_DL128x128_S2 = 4, T_DL128x128_S3 = 5, T_DL256x128_S2 = 6, T_DL256x256_S2 = 7,  // direct-to-LDS, k-contiguous
    T_DL256x256_W8 = 8, T_DL256x128_W8 = 9, T_DL128x256_W8 = 10,                          // ... with 8 waves
    T_DL128x128_W8A = 11, T_DL128x128_W8B = 12, T_DL256x128_W8S3 = 13, T_DL128x256_W8S3 = 14,
    T_DL128x64 = 15, T_DL64x128 = 16, T_DL128x64_S3 = 17,
    T_DL128x128_W8S4 = 18, T_DL128x64_S4 = 19, T_DL128x128_W8S3 = 20,  // deeper prefetch rings
    T_DL128x64_KG2 = 21, T_DL128x128_KG2 = 22, T_DL64x128_KG2 = 23,     // two k-groups (8 waves)
    T_LAST = T_DL64x128_KG2
};

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

// The split-K reduce of a bf16 GEMM: 16-byte accesses when every operand of
// the epilogue allows them, element accesses otherwise.
gp_status launch_reduce(const GemmArgs& a, int epi, int splits, hipStream_t st) {
    const bool res = epi == EPI_RES_F32, mask = epi == EPI_RELU_MASK;
    const bool v4 = a.N % 4 == 0 && a.ldc % 4 == 0 && aligned16(a.C) && aligned16(a.ws) &&
                    (!(epi == EPI_STORE || res) || !a.bias || aligned16(a.bias)) &&
                    (!(res || mask) || (a.ldaux % 4 == 0 && aligned16(a.aux))) &&
                    (!res || !a.C2 || (a.ldc2 % 4 == 0 && aligned16(a.C2))) &&
                    (epi != EPI_ACC_F32 || !a.colsum || aligned16(a.colsum));
    if (v4) {
        const int cx = (a.N + 1023) / 1024;
        // about 2048 workgroups, each over a run of whole rows
        const int rows = std::max(1, (int)((long)a.M * cx / 2048));
        const dim3 grid(cx, (a.M + rows - 1) / rows);
        switch (epi) {
        case EPI_STORE: klaunch(splitk_reduce_v4<EPI_STORE>, grid, 256, 0, st, a, splits, rows); break;
        case EPI_RES_F32: klaunch(splitk_reduce_v4<EPI_RES_F32>, grid, 256, 0, st, a, splits, rows); break;
        case EPI_F32: klaunch(splitk_reduce_v4<EPI_F32>, grid, 256, 0, st, a, splits, rows); break;
        case EPI_RELU_MASK: klaunch(splitk_reduce_v4<EPI_RELU_MASK>, grid, 256, 0, st, a, splits, rows); break;
        case EPI_ACC_F32: klaunch(splitk_reduce_v4<EPI_ACC_F32>, grid, 256, 0, st, a, splits, rows); break;
        default: return set_error(GP_ERR_INVALID_ARG, "gemm: split-K epilogue");
        }
        GP_LAUNCH_CHECK();
        return GP_OK;
    }
    const long nq = (long)a.M * (a.N / 4);
    const int rg = (int)std::min<long>((nq + 255) / 256, 2048);
    switch (epi) {
    case EPI_STORE: klaunch(splitk_reduce<bf16, EPI_STORE>, rg, 256, 0, st, a, splits); break;
    case EPI_RES_F32: klaunch(splitk_reduce<bf16, EPI_RES_F32>, rg, 256, 0, st, a, splits); break;
    case EPI_F32: klaunch(splitk_reduce<bf16, EPI_F32>, rg, 256, 0, st, a, splits); break;
    case EPI_RELU_MASK: klaunch(splitk_reduce<bf16, EPI_RELU_MASK>, rg, 256, 0, st, a, splits); break;
    case EPI_ACC_F32: klaunch(splitk_reduce<bf16, EPI_ACC_F32>, rg, 256, 0, st, a, splits); break;
    default: return set_error(GP_ERR_INVALID_ARG, "gemm: split-K epilogue");
    }
    GP_LAUNCH_CHECK();
    return GP_OK;
}

template <typename T, int BM, int BN, bool AK, bool BKM>
gp_status launch_tile(const GemmArgs& a, int epi, int splits, hipStream_t st) {
    const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    if (splits > 1) {
        dim3 grid(tiles, splits);
        klaunch(gemm_kernel<T, BM, BN, AK, BKM, EPI_F32, true>, grid, 256, 0, st, a);
        GP_LAUNCH_CHECK();
        const long nq = (long)a.M * (a.N / 4);
        const int rg = (int)std::min<long>((nq + 255) / 256, 2048);
        switch (epi) {
        case EPI_STORE: klaunch(splitk_reduce<T, EPI_STORE>, rg, 256, 0, st, a, splits); break;
        case EPI_RES_F32: klaunch(splitk_reduce<T, EPI_RES_F32>, rg, 256, 0, st, a, splits); break;
        case EPI_F32: klaunch(splitk_reduce<T, EPI_F32>, rg, 256, 0, st, a, splits); break;
        case EPI_RELU_MASK: klaunch(splitk_reduce<T, EPI_RELU_MASK>, rg, 256, 0, st, a, splits); break;
        case EPI_ACC_F32: klaunch(splitk_reduce<T, EPI_ACC_F32>, rg, 256, 0, st, a, splits); break;
        default: return set_error(GP_ERR_INVALID_ARG, "gemm: split-K epilogue");
        }
        GP_LAUNCH_CHECK();

        return GP_OK;
    }
    switch (epi) {
    case EPI_STORE: klaunch(gemm_kernel<T, BM, BN, AK, BKM, EPI_STORE, false>, tiles, 256, 0, st, a); break;
    case EPI_RES_F32: klaunch(gemm_kernel<T, BM, BN, AK, BKM, EPI_RES_F32, false>, tiles, 256, 0, st, a); break;
    case EPI_F32: klaunch(gemm_kernel<T, BM, BN, AK, BKM, EPI_F32, false>, tiles, 256, 0, st, a); break;
    case EPI_RELU_MASK: klaunch(gemm_kernel<T, BM, BN, AK, BKM, EPI_RELU_MASK, false>, tiles, 256, 0, st, a); break;
    case EPI_ACC_F32: klaunch(gemm_kernel<T, BM, BN, AK, BKM, EPI_ACC_F32, false>, tiles, 256, 0, st, a); break;
    default: return set_error(GP_ERR_INVALID_ARG, "gemm: unknown epilogue");
    }
    GP_LAUNCH_CHECK();
    return GP_OK;
}

template <int BM, int BN, int WM, int WN, int NSTAGE, bool KM>
gp_status launch_dl(const GemmArgs& a, int epi, int splits, hipStream_t st) {
    constexpr int NT = 64 * WM * WN;
    const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    if (splits > 1) {
        dim3 grid(tiles, splits);
        klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_F32, 1, KM>, grid, NT, 0, st, a);
        GP_LAUNCH_CHECK();
        if (a.deferred && (epi == EPI_RES_F32 || epi == EPI_F32)) {
            *a.deferred = splits;  // the caller reduces
            return GP_OK;
        }
        return launch_reduce(a, epi, splits, st);
    }
    if constexpr (KM) {
        switch (epi) {
        case EPI_STORE: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_STORE, 0, KM>, tiles, NT, 0, st, a); break;
        case EPI_RES_F32: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_RES_F32, 0, KM>, tiles, NT, 0, st, a); break;
        case EPI_F32: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_F32, 0, KM>, tiles, NT, 0, st, a); break;
        case EPI_RELU_MASK: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_RELU_MASK, 0, KM>, tiles, NT, 0, st, a); break;
        case EPI_ACC_F32: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_ACC_F32, 0, KM>, tiles, NT, 0, st, a); break;
        default: return set_error(GP_ERR_INVALID_ARG, "gemm: epilogue not instantiated for k-contiguous operands");
        }
    } else {
        switch (epi) {
        case EPI_ACC_F32: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_ACC_F32, 0, KM>, tiles, NT, 0, st, a); break;
        default: return set_error(GP_ERR_INVALID_ARG, "gemm: epilogue not instantiated for m-contiguous operands");
        }
    }
    GP_LAUNCH_CHECK();
    return GP_OK;
}

// Two k-groups per workgroup (k-contiguous operands, no split-K; the host
// guarantees an even k-tile count).
template <int BM, int BN, int WM, int WN, int NSTAGE>
gp_status launch_dl_kg2(const GemmArgs& a, int epi, hipStream_t st) {
    constexpr int NT = 64 * WM * WN * 2;
    const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    switch (epi) {
    case EPI_STORE: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_STORE, 0, true, false, 2>, tiles, NT, 0, st, a); break;
    case EPI_RES_F32: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_RES_F32, 0, true, false, 2>, tiles, NT, 0, st, a); break;
    case EPI_F32: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_F32, 0, true, false, 2>, tiles, NT, 0, st, a); break;
    case EPI_RELU_MASK: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_RELU_MASK, 0, true, false, 2>, tiles, NT, 0, st, a); break;
    case EPI_ACC_F32: klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_ACC_F32, 0, true, false, 2>, tiles, NT, 0, st, a); break;
    default: return set_error(GP_ERR_INVALID_ARG, "gemm: epilogue not instantiated for k-groups");
    }
    GP_LAUNCH_CHECK();
    return GP_OK;
}

// The fp4-corrected forward GEMM (EPI_STORE, k-contiguous operands).
template <int BM, int BN, int WM, int WN, int NSTAGE>
gp_status launch_dl_mx(const GemmArgs& a, int splits, hipStream_t st) {
    constexpr int NT = 64 * WM * WN;
    const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    if (splits > 1) {
        klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_F32, 1, true, true>, dim3(tiles, splits), NT, 0, st, a);
        GP_LAUNCH_CHECK();
        return launch_reduce(a, EPI_STORE, splits, st);
    } else {
        klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_STORE, 0, true, true>, tiles, NT, 0, st, a);
    }
    GP_LAUNCH_CHECK();
    return GP_OK;
}

// The fp16 forward GEMM (EPI_STORE, k-contiguous fp16 operands).
template <int BM, int BN, int WM, int WN, int NSTAGE>
gp_status launch_dl16(const GemmArgs& a, int splits, hipStream_t st) {
    constexpr int NT = 64 * WM * WN;
    const int tiles = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    if (splits > 1) {
        klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_F32, 1, true, false, 1, true>, dim3(tiles, splits), NT, 0, st, a);
        GP_LAUNCH_CHECK();
        return launch_reduce(a, EPI_STORE, splits, st);
    }
    klaunch(gemm_dl<BM, BN, WM, WN, NSTAGE, EPI_STORE, 0, true, false, 1, true>, tiles, NT, 0, st, a);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

// The chooser's k-contiguous shapes, with fp16 operands.
gp_status launch_f16(const GemmArgs& a, int cfg, int splits, hipStream_t st) {
    switch (cfg) {
    case T_DL256x256_W8: return launch_dl16<256, 256, 2, 4, 2>(a, splits, st);
    case T_DL256x128_W8: return launch_dl16<256, 128, 4, 2, 2>(a, splits, st);
    case T_DL128x256_W8: return launch_dl16<128, 256, 2, 4, 2>(a, splits, st);
    case T_DL256x128_W8S3: return launch_dl16<256, 128, 4, 2, 3>(a, splits, st);
    case T_DL128x256_W8S3: return launch_dl16<128, 256, 2, 4, 3>(a, splits, st);
    case T_DL128x128_W8S4: return launch_dl16<128, 128, 2, 4, 4>(a, splits, st);
    case T_DL128x128_W8S3: return launch_dl16<128, 128, 2, 4, 3>(a, splits, st);
    case T_DL128x64_S4: return launch_dl16<128, 64, 2, 2, 4>(a, splits, st);
    case T_DL128x64: return launch_dl16<128, 64, 2, 2, 2>(a, splits, st);
    case T_DL64x128: return launch_dl16<64, 128, 2, 2, 2>(a, splits, st);
    default: return launch_dl16<128, 128, 2, 4, 2>(a, splits, st);  // T_DL128x128_W8A and any other
    }
}

// Tile shapes whose fp4 stage splits into whole 1 KB blocks per wave.
bool mx_capable(int cfg) {
    return cfg == T_DL128x128_S2 || cfg == T_DL128x128_S3 || cfg == T_DL256x128_S2 || cfg == T_DL256x256_S2 ||
           cfg == T_DL256x256_W8 || cfg == T_DL128x128_W8A || cfg == T_DL128x128_W8B || cfg == T_DL128x128_W8S3 ||
           cfg == T_DL128x128_W8S4;
}

gp_status launch_mx(const GemmArgs& a, int cfg, int splits, hipStream_t st) {
    switch (cfg) {
    case T_DL128x128_S3: return launch_dl_mx<128, 128, 2, 2, 3>(a, splits, st);
    case T_DL256x128_S2: return launch_dl_mx<256, 128, 2, 2, 2>(a, splits, st);
    case T_DL256x256_S2: return launch_dl_mx<256, 256, 2, 2, 2>(a, splits, st);
    case T_DL256x256_W8: return launch_dl_mx<256, 256, 2, 4, 2>(a, splits, st);
    case T_DL128x128_W8A: return launch_dl_mx<128, 128, 2, 4, 2>(a, splits, st);
    case T_DL128x128_W8B: return launch_dl_mx<128, 128, 4, 2, 2>(a, splits, st);
    case T_DL128x128_W8S3: return launch_dl_mx<128, 128, 2, 4, 3>(a, splits, st);
    case T_DL128x128_W8S4: return launch_dl_mx<128, 128, 2, 4, 4>(a, splits, st);
    default: return launch_dl_mx<128, 128, 2, 2, 2>(a, splits, st);
    }
}

template <bool AK, bool BKM>
gp_status launch_bf16(const GemmArgs& a, int epi, int cfg, int splits, hipStream_t st) {
    if constexpr (AK == BKM) {
        constexpr bool KM = AK;
        switch (cfg) {
        case T_DL128x128_S2: return launch_dl<128, 128, 2, 2, 2, KM>(a, epi, splits, st);
        case T_DL128x128_S3: return launch_dl<128, 128, 2, 2, 3, KM>(a, epi, splits, st);
        case T_DL256x128_S2: return launch_dl<256, 128, 2, 2, 2, KM>(a, epi, splits, st);
        case T_DL256x256_S2: return launch_dl<256, 256, 2, 2, 2, KM>(a, epi, splits, st);
        case T_DL256x256_W8: return launch_dl<256, 256, 2, 4, 2, KM>(a, epi, splits, st);
        case T_DL256x128_W8: return launch_dl<256, 128, 4, 2, 2, KM>(a, epi, splits, st);
        case T_DL128x256_W8: return launch_dl<128, 256, 2, 4, 2, KM>(a, epi, splits, st);
        case T_DL128x128_W8A: return launch_dl<128, 128, 2, 4, 2, KM>(a, epi, splits, st);
        case T_DL128x128_W8B: return launch_dl<128, 128, 4, 2, 2, KM>(a, epi, splits, st);
        case T_DL256x128_W8S3: return launch_dl<256, 128, 4, 2, 3, KM>(a, epi, splits, st);
        case T_DL128x256_W8S3: return launch_dl<128, 256, 2, 4, 3, KM>(a, epi, splits, st);
        case T_DL128x128_W8S4: return launch_dl<128, 128, 2, 4, 4, KM>(a, epi, splits, st);
        case T_DL128x128_W8S3: return launch_dl<128, 128, 2, 4, 3, KM>(a, epi, splits, st);
        case T_DL128x64_S4:
            if constexpr (KM) return launch_dl<128, 64, 2, 2, 4, KM>(a, epi, splits, st);
            break;
        case T_DL128x64_KG2:
            if constexpr (KM) return launch_dl_kg2<128, 64, 2, 2, 3>(a, epi, st);
            break;
        case T_DL128x128_KG2:
            if constexpr (KM) return launch_dl_kg2<128, 128, 2, 2, 2>(a, epi, st);
            break;
        case T_DL64x128_KG2:
            if constexpr (KM) return launch_dl_kg2<64, 128, 2, 2, 3>(a, epi, st);
            break;
        case T_DL128x64:
            if constexpr (KM) return launch_dl<128, 64, 2, 2, 2, KM>(a, epi, splits, st);
            break;
        case T_DL64x128:
            if constexpr (KM) return launch_dl<64, 128, 2, 2, 2, KM>(a, epi, splits, st);
            break;
        case T_DL128x64_S3:
            if constexpr (KM) return launch_dl<128, 64, 2, 2, 3, KM>(a, epi, splits, st);
            break;
        default: break;
        }
    }
    switch (cfg) {
    case T256x256: return launch_tile<bf16, 256, 256, AK, BKM>(a, epi, splits, st);
    case T256x128: return launch_tile<bf16, 256, 128, AK, BKM>(a, epi, splits, st);
    case T128x256: return launch_tile<bf16, 128, 256, AK, BKM>(a, epi, splits, st);
    default: return launch_tile<bf16, 128, 128, AK, BKM>(a, epi, splits, st);
    }
}

constexpr int NUM_CU = 256;

// Pick the tile shape and split count.  Cost = full-machine rounds x per-tile
// time, where a round holds NUM_CU x (workgroups resident per CU) tiles and
// co-resident tiles share their CU; per-tile time is the tile's k-steps over
// a measured relative efficiency; split-K adds its partial-tile traffic.
// Split-K needs the partial tiles (and, for a fused bias gradient, one row of
// column sums per split) to fit the workspace, N % 4 == 0 for the reduce, and
// at least four k-steps per split.
bool split_fits(const GemmArgs& a, int s, int nk) {
    const long need = (long)s * a.M * a.N + (a.colsum ? (long)s * a.N : 0);
    return a.ws != nullptr && nk / s >= 4 && need <= a.ws_elems && a.N % 4 == 0;
}

// Direct-to-LDS tiles (K % 64 == 0): time = fixed launch cost + rounds x
// k-steps x per-step time of the tile shape (with the tile running alone on
// its CU or sharing it with a second one) + the fp32 read-modify-write of an
// accumulating epilogue + the split-K partial traffic and reduce.  The
// constants were fitted to measurements of the d_model 1024 partition's GEMMs
// on MI355X at 512, 1024, 2048 and 4096 token rows (random bf16 operands,
// splits up to 4), separately for k-contiguous operands (forward and
// input-gradient GEMMs) and m/n-contiguous ones (weight gradients, whose
// transposing LDS reads cost more per step).  Units: us.
// Weight of the split-K cost terms (GP_SPLIT_WEIGHT, default 1): the fit was
// made on GEMMs running alone; next to concurrent work the partial traffic
// can cost more.
double split_weight() {
    static const double w = [] {
        const char* e = std::getenv("GP_SPLIT_WEIGHT");
        return e ? std::atof(e) : 1.0;
    }();
    return w;
}

void choose_dl_model(const GemmArgs& a, int epi, bool kmaj, int& cfg, int& splits);

// The choice depends only on the problem's shape and operand form; a small
// per-thread memo (direct-mapped, full key checked) keeps the cost model off
// the launch path for the handful of shapes a partition launches repeatedly.
void choose_dl(const GemmArgs& a, int epi, bool kmaj, int& cfg, int& splits) {
    struct Entry { long long key[4]; int cfg, splits; bool used; };
    static thread_local Entry memo[64] = {};
    const long long key[4] = {((long long)a.M << 32) | (unsigned)a.N,
                              ((long long)a.K << 32) | (unsigned)(epi | (kmaj ? 256 : 0) | (a.a4 ? 512 : 0) |
                                                                   (a.colsum ? 1024 : 0) | (a.ws ? 2048 : 0)),
                              (long long)a.ws_elems, 0};
    unsigned long long h = 1469598103934665603ull;
    for (long long k : key) h = (h ^ (unsigned long long)k) * 1099511628211ull;
    Entry& e = memo[(h >> 20) & 63];
    if (e.used && e.key[0] == key[0] && e.key[1] == key[1] && e.key[2] == key[2]) {
        cfg = e.cfg;
        splits = e.splits;
        return;
    }
    choose_dl_model(a, epi, kmaj, cfg, splits);
    e = Entry{{key[0], key[1], key[2], 0}, cfg, splits, true};
}

void choose_dl_model(const GemmArgs& a, int epi, bool kmaj, int& cfg, int& splits) {
    // the fp4 correction adds one MFMA of a quarter of the bf16 time per k-tile
    // and a quarter more tile traffic; only some shapes carry it
    const bool mx = a.a4 != nullptr;
    const double mx_step = mx ? 1.25 : 1.0;
    // per-k-tile time with 1, 2 or 3 tiles sharing a CU (0 = cannot share)
    struct Cand { int cfg, bm, bn, resident; double step[3]; };
    static const Cand kc[] = {  // k-contiguous operands
        {T_DL256x256_W8, 256, 256, 1, {1.263, 0, 0}},    {T_DL256x128_W8, 256, 128, 1, {0.801, 0, 0}},
        {T_DL128x256_W8, 128, 256, 1, {0.790, 0, 0}},    {T_DL128x128_W8A, 128, 128, 2, {0.511, 0.879, 0}},
        {T_DL256x128_W8S3, 256, 128, 1, {0.688, 0, 0}},  {T_DL128x256_W8S3, 128, 256, 1, {0.682, 0, 0}},
        {T_DL128x64, 128, 64, 3, {0.402, 0.561, 0.714}}, {T_DL64x128, 64, 128, 3, {0.398, 0.552, 0.712}},
        {T_DL128x128_W8S4, 128, 128, 1, {0.410, 0, 0}},  {T_DL128x64_S4, 128, 64, 1, {0.320, 0, 0}},
        {T_DL128x128_W8S3, 128, 128, 1, {0.402, 0, 0}}};
    static const Cand mc[] = {  // m/n-contiguous operands (weight gradients)
        {T_DL256x256_W8, 256, 256, 1, {1.865, 0, 0}},    {T_DL256x128_W8, 256, 128, 1, {1.256, 0, 0}},
        {T_DL128x256_W8, 128, 256, 1, {1.236, 0, 0}},    {T_DL128x128_W8A, 128, 128, 2, {0.831, 0.940, 0}},
        {T_DL128x128_W8B, 128, 128, 2, {0.898, 1.012, 0}}, {T_DL256x128_W8S3, 256, 128, 1, {1.350, 0, 0}},
        {T_DL128x256_W8S3, 128, 256, 1, {1.335, 0, 0}},  {T_DL128x128_W8S4, 128, 128, 1, {1.040, 0, 0}},
        {T_DL128x128_W8S3, 128, 128, 1, {1.049, 0, 0}}};
    const Cand* cands = kmaj ? kc : mc;
    const int ncand = kmaj ? (int)(sizeof(kc) / sizeof(kc[0])) : (int)(sizeof(mc) / sizeof(mc[0]));
    const double c0 = kmaj ? 4.147 : 0.0, BW = kmaj ? 1.969e6 : 5.084e6, red0 = kmaj ? 3.285 : 7.821;
    // The m/n-contiguous shapes are the weight gradients, which run beside the
    // backward's dX chain and the recompute: a split spends more CU time
    // (partial planes and a reduce) to finish sooner alone, so it is costed
    // three times over for them.
    const double split_w = (kmaj ? 1.0 : 3.0) * split_weight();
    const int nk = a.K / 64;
    double best = 1e300;
    cfg = T_DL128x128_W8A;
    splits = 1;
    for (int ci = 0; ci < ncand; ++ci) {
        const Cand& c = cands[ci];
        if (mx && !mx_capable(c.cfg)) continue;
        const long tiles = (long)((a.M + c.bm - 1) / c.bm) * ((a.N + c.bn - 1) / c.bn);
        for (int s = 1; s <= 4; s *= 2) {
            if (s > 1 && !split_fits(a, s, nk)) continue;
            const long per_cu = (tiles * s + NUM_CU - 1) / NUM_CU;
            const long rounds = (per_cu + c.resident - 1) / c.resident;
            const int occ = (int)std::min<long>(per_cu, c.resident);
            double t = c0 + rounds * (double)((nk + s - 1) / s) * c.step[occ - 1] * mx_step;
            if (epi == EPI_ACC_F32) t += (kmaj ? 3.0 : 0.0) + (double)a.M * a.N * 8.0 / BW;
            if (s > 1) t += split_w * ((double)a.M * a.N * 4.0 * (s + 1.0) / 2.0 / BW + red0);
            if (t < best * 0.999) {
                best = t;
                cfg = c.cfg;
                splits = s;
            }
        }
    }
}

void choose(const GemmArgs& a, int epi, int& cfg, int& splits) {
    static const int BMs[4] = {256, 256, 128, 128}, BNs[4] = {256, 128, 256, 128};
    static const int resident[4] = {1, 1, 1, 2};
    static const double eff[4] = {0.95, 0.8, 0.8, 1.0};
    double best = 1e300;
    cfg = T128x128;
    splits = 1;
    const int nk = (a.K + 63) / 64;
    for (int c = 0; c < 4; ++c) {
        const long tiles = (long)((a.M + BMs[c] - 1) / BMs[c]) * ((a.N + BNs[c] - 1) / BNs[c]);
        for (int s = 1; s <= 8; s *= 2) {
            if (s > 1 && !split_fits(a, s, nk)) continue;
            const long wgs = tiles * s;
            const long slots = (long)NUM_CU * resident[c];
            const long rounds = (wgs + slots - 1) / slots;
            const long per_cu = std::min<long>(resident[c], (wgs + NUM_CU - 1) / NUM_CU);
            const double kt = (double)((nk + s - 1) / s);
            // time in units of one 128x128x64 tile step of a CU running alone
            // two co-resident tiles hide each other's latencies: 1.5x, not 2x, the time of one
            double t = rounds * (per_cu == 2 ? 1.5 : 1.0) * (BMs[c] / 128.0) * (BNs[c] / 128.0) * kt / eff[c];
            // split-K: partial-tile traffic at ~1.75 TB/s and the reduce launch (one
            // unit = one 128x128x64 step of a lone tile, ~0.58 us on MI355X)
            if (s > 1) t += (double)a.M * a.N * 4.0 * (s + 1.0) / 2.0 / 1.0e6 + 4.0;
            if (t < best * 0.999) {
                best = t;
                cfg = c;
                splits = s;
            }
        }
    }
}

template <typename T>
gp_status check_args(const GemmArgs& a, bool a_kmajor, bool b_kmajor) {
    constexpr int VEC = Vec16<T>::N;
    if (a.M <= 0 || a.N <= 0 || a.K <= 0) return set_error(GP_ERR_INVALID_ARG, "gemm: empty problem");
    if (a.K % VEC || a.lda % VEC || a.ldb % VEC)
        return set_error(GP_ERR_INVALID_ARG, "gemm: K and leading dimensions must be multiples of 16 bytes");
    if ((!a_kmajor && a.M % VEC) || (!b_kmajor && a.N % VEC))
        return set_error(GP_ERR_INVALID_ARG, "gemm: m/n-contiguous operands need M, N multiples of 16 bytes");
    if (((uintptr_t)a.A | (uintptr_t)a.B) & 15) return set_error(GP_ERR_INVALID_ARG, "gemm: operands must be 16-byte aligned");
    if (a_kmajor != b_kmajor) return set_error(GP_ERR_UNSUPPORTED, "gemm: mixed operand majorness not instantiated");
    return GP_OK;
}

} // namespace

gp_status gemm_reduce(const GemmArgs& a, int epi, int splits, hipStream_t st) {
    if (!a.ws || splits < 2) return set_error(GP_ERR_INVALID_ARG, "gemm_reduce: no split-K partials");
    return launch_reduce(a, epi, splits, st);
}

namespace {
// The tile shape and split count gemm() launches a bf16 problem with.
void decide_bf16(const GemmArgs& args, int epi, bool a_kmajor, int& cfg, int& splits) {
    GemmArgs a = args;
    if (args.split_rows > 0) a.M = args.split_rows;
    if (a.a4) {
        choose_dl(a, epi, true, cfg, splits);
        if (a.force_cfg >= 0 && a.force_cfg <= T_LAST) {
            // a forced shape without an fp4 stage falls back to the 128 x 128 tile
            cfg = mx_capable(a.force_cfg) ? a.force_cfg : T_DL128x128_S2;
            splits = a.force_splits > 0 ? a.force_splits : 1;
            if (splits > 1 && !split_fits(a, splits, a.K / 64)) splits = 1;
        }
        return;
    }
    if (a.K % 64 == 0)
        choose_dl(a, epi, a_kmajor, cfg, splits);
    else
        choose(a, epi, cfg, splits);
    if (a.force_cfg >= 0 && a.force_cfg <= T_LAST) {
        cfg = a.force_cfg;
        splits = a.force_splits > 0 ? a.force_splits : 1;
        if (splits > 1 && !split_fits(a, splits, (a.K + 63) / 64)) splits = 1;
    }
    if (cfg > T128x128 && a.K % 64) cfg = T128x128;
    const bool narrow = cfg == T_DL128x64 || cfg == T_DL64x128 || cfg == T_DL128x64_S3 || cfg == T_DL128x64_S4;
    const bool kg2 = cfg == T_DL128x64_KG2 || cfg == T_DL128x128_KG2 || cfg == T_DL64x128_KG2;
    if (!a_kmajor && (narrow || kg2)) cfg = T_DL128x128_W8A;  // no 64-wide or k-group m-contiguous tiles
    if (kg2 && (splits > 1 || (a.K / 64) % 2)) {               // k-groups: unsplit, even k-tile count
        cfg = T_DL128x64_S4;
        splits = 1;
    }
}
} // namespace

long gemm_workspace_need(const GemmArgs& a, int epi, bool a_kmajor, int dtype) {
    if (dtype != GP_BF16 || !a.ws) return 0;
    int cfg = 0, splits = 1;
    decide_bf16(a, epi, a_kmajor, cfg, splits);
    return splits > 1 ? (long)splits * a.M * a.N + (a.colsum ? (long)splits * a.N : 0) : 0;
}

gp_status gemm(const GemmArgs& a, int epi, bool a_kmajor, bool b_kmajor, int dtype, hipStream_t st) {
    if (a.deferred) *a.deferred = 1;
    if (a.f16) {
        if (dtype != GP_BF16 || !a_kmajor || !b_kmajor || epi != EPI_STORE || a.K % 64 || a.a4)
            return set_error(GP_ERR_UNSUPPORTED, "gemm: fp16 operands need k-contiguous operands, a stored epilogue, "
                                                 "K % 64 == 0 and no fp4 term");
        gp_status s = check_args<bf16>(a, true, true);
        if (s != GP_OK) return s;
        int cfg, splits;
        decide_bf16(a, epi, true, cfg, splits);
        return launch_f16(a, cfg, splits, st);
    }
    if (a.a4) {
        if (dtype != GP_BF16 || !a_kmajor || !b_kmajor || epi != EPI_STORE || a.K % 64 || !a.b4 || !a.sa4 || !a.sb4)
            return set_error(GP_ERR_UNSUPPORTED, "gemm: the fp4 correction needs bf16, k-contiguous operands, "
                                                 "a stored epilogue and K % 64 == 0");
        gp_status s = check_args<bf16>(a, true, true);
        if (s != GP_OK) return s;
        int cfg, splits;
        decide_bf16(a, epi, true, cfg, splits);
        return launch_mx(a, cfg, splits, st);
    }
    if (dtype == GP_BF16) {
        gp_status s = check_args<bf16>(a, a_kmajor, b_kmajor);
        if (s != GP_OK) return s;
        int cfg, splits;
        decide_bf16(a, epi, a_kmajor, cfg, splits);
        return a_kmajor ? launch_bf16<true, true>(a, epi, cfg, splits, st)
                        : launch_bf16<false, false>(a, epi, cfg, splits, st);
    }
    gp_status s = check_args<float>(a, a_kmajor, b_kmajor);
    if (s != GP_OK) return s;
    return a_kmajor ? launch_tile<float, 128, 128, true, true>(a, epi, 1, st)
                    : launch_tile<float, 128, 128, false, false>(a, epi, 1, st);
}

} // namespace gp
