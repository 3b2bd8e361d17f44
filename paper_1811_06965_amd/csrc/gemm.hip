// gemm.hip -- LDS-staged MFMA GEMM family of the partition (gfx950, wave64).
//
//   C[m, n] = sum_k A(m, k) B(n, k)     then a fused epilogue
//
// Every linear layer of the partition maps onto one of three operand forms:
//   forward   Y  = X W      A = X  [T, in]  k-contiguous,  B = W^T [out, in]  k-contiguous
//   input grad dX = dY W^T  A = dY [T, out] k-contiguous,  B = W   [in, out]  k-contiguous
//   weight grad dW = X^T dY A = X  [T, in]  m-contiguous,  B = dY  [T, out]   n-contiguous
// The partition keeps both W and W^T working copies so the two activation
// GEMMs stream both operands along k.  The weight-gradient GEMM loads
// m-contiguous 16-byte vectors over 4 consecutive k and transposes them in
// registers, so LDS always holds k-contiguous rows and the MFMA fragment read
// is one 16-byte LDS load per lane.
//
// Tiles: 128 x 128 x BK per workgroup of 4 waves (2 x 2), each wave 64 x 64 =
// 2 x 2 MFMA blocks of 32 x 32.  bf16 uses v_mfma_f32_32x32x16_bf16 (fp32
// accumulate), fp32 uses v_mfma_f32_32x32x2_f32.  Global tiles are prefetched
// into registers while the current LDS buffer is consumed (two LDS buffers,
// one barrier per k-tile).  Workgroup ids are remapped so each XCD (which
// receives every 8th workgroup) works on a contiguous run of output tiles
// that share weight panels in its own L2.
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
__device__ __forceinline__ void mma(f32x16& c, const Frag<float>& a, const Frag<float>& b) {
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.lo[e], b.lo[e], c, 0, 0, 0);
#pragma unroll
    for (int e = 0; e < 4; ++e) c = __builtin_amdgcn_mfma_f32_32x32x2f32(a.hi[e], b.hi[e], c, 0, 0, 0);
}

template <typename T> using V16 = typename Vec16<T>::type;

template <typename T>
__device__ __forceinline__ V16<T> load16(const T* p, bool ok) {
    if (ok) return *reinterpret_cast<const V16<T>*>(p);
    V16<T> z;
#pragma unroll
    for (int i = 0; i < Vec16<T>::N; ++i) z[i] = (T)0.f;
    return z;
}

// Tile loader for one operand: ROWS x BK elements of the operand (row index =
// m for A, n for B) into LDS laid out [ROWS][BK + PAD], k contiguous.
template <typename T, int ROWS, int BK, bool KMAJOR>
struct TileLoader {
    static constexpr int VEC = Vec16<T>::N;
    static constexpr int PAD = VEC;
    static constexpr int LDK = BK + PAD;
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

    __device__ __forceinline__ void load(const T* __restrict__ g, long ld, int row0, int nrows, int k0, int K,
                                         int tid) {
        if (KMAJOR) {
            const int rr = tid / TPR, kk = (tid % TPR) * VEC;
#pragma unroll
            for (int p = 0; p < KPASS; ++p) {
                const int row = row0 + p * RPP + rr, k = k0 + kk;
                const bool ok = row < nrows && k < K;
                r[p] = load16<T>(g + (long)(ok ? row : 0) * ld + (ok ? k : 0), ok);
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
                    r[p * KB + q] = load16<T>(g + (long)(ok ? k : 0) * ld + (ok ? row : 0), ok);
                }
            }
        }
    }

    __device__ __forceinline__ void store(T* __restrict__ s, int tid) const {
        if (KMAJOR) {
            const int rr = tid / TPR, kk = (tid % TPR) * VEC;
#pragma unroll
            for (int p = 0; p < KPASS; ++p)
                *reinterpret_cast<V16<T>*>(s + (p * RPP + rr) * LDK + kk) = r[p];
        } else {
#pragma unroll
            for (int p = 0; p < MPASS; ++p) {
                const int blk = p * 256 + tid;
                const int mb = blk % MBLK, kb = blk / MBLK;
#pragma unroll
                for (int i = 0; i < VEC; ++i) {
                    T* dst = s + (mb * VEC + i) * LDK + kb * KB;
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

// Epilogue on one output element (row, col) of value v = sum_k A B.
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
        float* c = reinterpret_cast<float*>(a.C);
        c[i] = a.accumulate ? c[i] + v : v;
    }
}

template <typename T, bool AK, bool BKM, int EPI>
__global__ void __launch_bounds__(256) gemm_kernel(GemmArgs args) {
    constexpr int BM = 128, BN = 128, BK = GemmCfg<T>::BK;
    constexpr int WM = 2, WN = 2;
    constexpr int TM = BM / WM / 32, TN = BN / WN / 32;
    using LA = TileLoader<T, BM, BK, AK>;
    using LB = TileLoader<T, BN, BK, BKM>;
    constexpr int LDK = LA::LDK;
    __shared__ __attribute__((aligned(16))) T As[2][BM * LDK];
    __shared__ __attribute__((aligned(16))) T Bs[2][BN * LDK];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int wm = wave / WN, wn = wave % WN;

    // XCD-aware tile order: workgroup b runs on XCD b % 8; give XCD x the
    // contiguous logical range [x G/8, (x+1) G/8) (tiles walk down M inside a
    // column of N tiles, so neighbours share the B panel).
    const int tiles_m = (args.M + BM - 1) / BM, tiles_n = (args.N + BN - 1) / BN;
    const int G = tiles_m * tiles_n;
    int bid = blockIdx.x;
    const int G8 = G & ~7;
    if (bid < G8) bid = (bid & 7) * (G8 >> 3) + (bid >> 3);
    const int tm = bid % tiles_m, tn = bid / tiles_m;
    const int m0 = tm * BM, n0 = tn * BN;

    const T* A = reinterpret_cast<const T*>(args.A);
    const T* B = reinterpret_cast<const T*>(args.B);
    LA la;
    LB lb;
    f32x16 acc[TM][TN];
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.f;

    const int nk = (args.K + BK - 1) / BK;
    la.load(A, args.lda, m0, args.M, 0, args.K, tid);
    lb.load(B, args.ldb, n0, args.N, 0, args.K, tid);
    la.store(As[0], tid);
    lb.store(Bs[0], tid);
    __syncthreads();

    const int fr = lane & 31, fk = (lane >> 5) * 8;
    for (int kt = 0; kt < nk; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < nk) {
            la.load(A, args.lda, m0, args.M, (kt + 1) * BK, args.K, tid);
            lb.load(B, args.ldb, n0, args.N, (kt + 1) * BK, args.K, tid);
        }
        const T* as = As[buf];
        const T* bs = Bs[buf];
#pragma unroll
        for (int s = 0; s < BK / 16; ++s) {
            Frag<T> fa[TM], fb[TN];
#pragma unroll
            for (int i = 0; i < TM; ++i) fa[i].load(as + (wm * (BM / WM) + i * 32 + fr) * LDK + s * 16 + fk);
#pragma unroll
            for (int j = 0; j < TN; ++j) fb[j].load(bs + (wn * (BN / WN) + j * 32 + fr) * LDK + s * 16 + fk);
#pragma unroll
            for (int i = 0; i < TM; ++i)
#pragma unroll
                for (int j = 0; j < TN; ++j) mma(acc[i][j], fa[i], fb[j]);
        }
        if (kt + 1 < nk) {
            la.store(As[buf ^ 1], tid);
            lb.store(Bs[buf ^ 1], tid);
        }
        __syncthreads();
    }

    // 32x32 accumulator layout: lane l holds column (l % 32); register r holds
    // row 8 (r / 4) + 4 (l / 32) + (r % 4).
#pragma unroll
    for (int i = 0; i < TM; ++i)
#pragma unroll
        for (int j = 0; j < TN; ++j) {
            const int col = n0 + wn * (BN / WN) + j * 32 + (lane & 31);
            if (col >= args.N) continue;
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int row = m0 + wm * (BM / WM) + i * 32 + (r >> 2) * 8 + (lane >> 5) * 4 + (r & 3);
                if (row < args.M) epilogue<T, EPI>(args, row, col, acc[i][j][r]);
            }
        }
}

template <typename T, bool AK, bool BKM>
gp_status launch_epi(const GemmArgs& a, int epi, hipStream_t st) {
    constexpr int BM = 128, BN = 128;
    const int grid = ((a.M + BM - 1) / BM) * ((a.N + BN - 1) / BN);
    switch (epi) {
    case EPI_STORE: gemm_kernel<T, AK, BKM, EPI_STORE><<<grid, 256, 0, st>>>(a); break;
    case EPI_RES_F32: gemm_kernel<T, AK, BKM, EPI_RES_F32><<<grid, 256, 0, st>>>(a); break;
    case EPI_F32: gemm_kernel<T, AK, BKM, EPI_F32><<<grid, 256, 0, st>>>(a); break;
    case EPI_RELU_MASK: gemm_kernel<T, AK, BKM, EPI_RELU_MASK><<<grid, 256, 0, st>>>(a); break;
    case EPI_ACC_F32: gemm_kernel<T, AK, BKM, EPI_ACC_F32><<<grid, 256, 0, st>>>(a); break;
    default: return set_error(GP_ERR_INVALID_ARG, "gemm: unknown epilogue");
    }
    GP_LAUNCH_CHECK();
    return GP_OK;
}

template <typename T>
gp_status gemm_t(const GemmArgs& a, int epi, bool a_kmajor, bool b_kmajor, hipStream_t st) {
    constexpr int VEC = Vec16<T>::N;
    if (a.M <= 0 || a.N <= 0 || a.K <= 0) return set_error(GP_ERR_INVALID_ARG, "gemm: empty problem");
    if (a.K % VEC || a.lda % VEC || a.ldb % VEC) return set_error(GP_ERR_INVALID_ARG, "gemm: K and leading dimensions must be multiples of 16 bytes");
    if ((!a_kmajor && a.M % VEC) || (!b_kmajor && a.N % VEC)) return set_error(GP_ERR_INVALID_ARG, "gemm: m/n-contiguous operands need M, N multiples of 16 bytes");
    if (((uintptr_t)a.A | (uintptr_t)a.B) & 15) return set_error(GP_ERR_INVALID_ARG, "gemm: operands must be 16-byte aligned");
    if (a_kmajor && b_kmajor) return launch_epi<T, true, true>(a, epi, st);
    if (!a_kmajor && !b_kmajor) return launch_epi<T, false, false>(a, epi, st);
    return set_error(GP_ERR_UNSUPPORTED, "gemm: mixed operand majorness not instantiated");
}

} // namespace

gp_status gemm(const GemmArgs& a, int epi, bool a_kmajor, bool b_kmajor, int dtype, hipStream_t st) {
    if (dtype == GP_BF16) return gemm_t<bf16>(a, epi, a_kmajor, b_kmajor, st);
    return gemm_t<float>(a, epi, a_kmajor, b_kmajor, st);
}

} // namespace gp
