// norm.hip -- LayerNorm forward/backward and deterministic column reductions.
//
// LayerNorm over the feature dimension D of each token row (biased variance,
// eps inside the square root).  Optionally the forward also writes the bf16
// rounding residuals of its output in fp4 with one scale per row (see
// layernorm_fwd).  One wave owns one row; lane l holds features
// l, l + 64, ... so every global access is a coalesced 256-byte row segment.
// Parameter gradients are reduced in two deterministic stages: per-block
// partial sums, then a fixed-order column sum (no atomics), so re-running a
// micro-batch reproduces its gradients bit for bit.
#include "common.hpp"
#include "kernels.hpp"

namespace gp {

namespace {

constexpr int LN_WAVES = 4;

template <typename T, int C>
__global__ void __launch_bounds__(256) ln_fwd_kernel(const float* __restrict__ x, long rows, int D,
                                                     const float* __restrict__ gamma,
                                                     const float* __restrict__ beta, float eps,
                                                     T* __restrict__ out, float* __restrict__ stats,
                                                     unsigned char* __restrict__ lo4, unsigned char* __restrict__ lo_sc) {
    const int lane = threadIdx.x & 63;
    const long row = (long)blockIdx.x * LN_WAVES + (threadIdx.x >> 6);
    if (row >= rows) return;
    const float* xr = x + row * D;
    float v[C];
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int d = lane + c * 64;
        v[c] = d < D ? xr[d] : 0.f;
        s += v[c];
    }
    const float mu = wave_sum(s) / D;
    float q = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int d = lane + c * 64;
        const float t = d < D ? v[c] - mu : 0.f;
        q += t * t;
    }
    const float rstd = 1.f / sqrtf(wave_sum(q) / D + eps);
    T* orow = out + row * D;
    float lo[C];
    float amax = 0.f;
#pragma unroll
    for (int c = 0; c < C; ++c) {
        const int d = lane + c * 64;
        lo[c] = 0.f;
        if (d < D) {
            const float y = gamma[d] * ((v[c] - mu) * rstd) + beta[d];
            const T hi = to_elt<T>(y);
            orow[d] = hi;
            lo[c] = y - (float)hi;
            amax = fmaxf(amax, fabsf(lo[c]));
        }
    }
    if (lo4) {
        // fp4 rounding residuals (D % 64 == 0): features d, d + 1 of lanes 2k, 2k + 1 share a byte
        const unsigned sc = e8m0_for_amax(wave_max(amax));
        const float inv = e8m0_inv(sc);
        unsigned char* lrow = lo4 + row * (D / 2);
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const unsigned q = e2m1_code(lo[c] * inv);
            const unsigned nb = (unsigned)__shfl_xor((int)q, 1, 64);
            const int d = lane + c * 64;
            if (!(lane & 1) && d < D) lrow[d / 2] = (unsigned char)(q | (nb << 4));
        }
        if (lane == 0) lo_sc[row] = (unsigned char)sc;
    }
    if (stats && lane == 0) {
        stats[2 * row] = mu;
        stats[2 * row + 1] = rstd;
    }
}

int ln_bwd_rows_per_wave(long rows) {
    long r = rows / (LN_WAVES * 256);
    return r < 1 ? 1 : (int)r;
}

template <typename T, int C>
__global__ void __launch_bounds__(256) ln_bwd_kernel(const float* __restrict__ dn, const float* __restrict__ x,
                                                     const float* __restrict__ stats,
                                                     const float* __restrict__ gamma, long rows, int D, int rpw,
                                                     const float* __restrict__ dres, float* __restrict__ dx32,
                                                     T* __restrict__ dxe, float* __restrict__ partial,
                                                     int accumulate) {
    __shared__ float red[LN_WAVES][2][C * 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    float pg[C], pb[C];
#pragma unroll
    for (int c = 0; c < C; ++c) pg[c] = pb[c] = 0.f;
    const long row0 = ((long)blockIdx.x * LN_WAVES + wave) * rpw;
    for (int rr = 0; rr < rpw; ++rr) {
        const long row = row0 + rr;
        if (row >= rows) break;
        const float mu = stats[2 * row], rstd = stats[2 * row + 1];
        float g[C], xh[C];
        float sg = 0.f, sgx = 0.f;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int d = lane + c * 64;
            if (d < D) {
                const float dv = dn[row * D + d];
                xh[c] = (x[row * D + d] - mu) * rstd;
                g[c] = dv * gamma[d];
                pg[c] += dv * xh[c];
                pb[c] += dv;
            } else {
                xh[c] = g[c] = 0.f;
            }
            sg += g[c];
            sgx += g[c] * xh[c];
        }
        sg = wave_sum(sg) / D;
        sgx = wave_sum(sgx) / D;
#pragma unroll
        for (int c = 0; c < C; ++c) {
            const int d = lane + c * 64;
            if (d < D) {
                float r = rstd * (g[c] - sg - xh[c] * sgx);
                if (dres) r += dres[row * D + d];
                if (dx32) dx32[row * D + d] = r;
                if (dxe) dxe[row * D + d] = to_elt<T>(r);
            }
        }
    }
#pragma unroll
    for (int c = 0; c < C; ++c) {
        red[wave][0][lane + c * 64] = pg[c];
        red[wave][1][lane + c * 64] = pb[c];
    }
    __syncthreads();
    for (int i = threadIdx.x; i < 2 * D; i += 256) {
        const int which = i / D, d = i % D;
        float s = 0.f;
#pragma unroll
        for (int w = 0; w < LN_WAVES; ++w) s += red[w][which][d];
        float* pp = partial + (long)blockIdx.x * 2 * D + i;
        *pp = accumulate ? *pp + s : s;
    }
}

// 16 waves per block, 64 columns per block: wave w adds rows w, w + 16, ...
// (lanes = columns, coalesced), then the 16 wave sums are added in order.
__global__ void __launch_bounds__(1024) colsum_kernel(const float* __restrict__ partial, int nblk, int width,
                                                      float* __restrict__ out, int accumulate) {
    __shared__ float red[16][64];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int c = blockIdx.x * 64 + lane;
    float s = 0.f;
    if (c < width)
        for (int b = w; b < nblk; b += 16) s += partial[(long)b * width + c];
    red[w][lane] = s;
    __syncthreads();
    if (w == 0 && c < width) {
        float t = 0.f;
#pragma unroll
        for (int i = 0; i < 16; ++i) t += red[i][lane];
        out[c] = accumulate ? out[c] + t : t;
    }
}

// ---- 16-byte vectorised LayerNorm for D a multiple of 256 (lane l owns
// features 4 (l + 64 c) .. +3, c < C4 = D / 256).
template <typename T> struct Out4;
template <> struct Out4<float> {
    static __device__ __forceinline__ void store(float* p, f32x4 v) { *reinterpret_cast<f32x4*>(p) = v; }
    static __device__ __forceinline__ f32x4 residual(f32x4) { return f32x4{0.f, 0.f, 0.f, 0.f}; }
};
template <> struct Out4<bf16> {
    static __device__ __forceinline__ void store(bf16* p, f32x4 v) {
        bf16x4 b = {(bf16)v[0], (bf16)v[1], (bf16)v[2], (bf16)v[3]};
        *reinterpret_cast<bf16x4*>(p) = b;
    }
    // the rounding residual v - bf16(v)
    static __device__ __forceinline__ f32x4 residual(f32x4 v) {
        f32x4 r;
#pragma unroll
        for (int i = 0; i < 4; ++i) r[i] = v[i] - (float)(bf16)v[i];
        return r;
    }
};

__device__ __forceinline__ float hsum(f32x4 v) { return (v[0] + v[1]) + (v[2] + v[3]); }

typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));

// o16 (optional): the output also in fp16 (the operand of a GEMM that takes
// fp16 inputs).
template <typename T, int C4>
__device__ __forceinline__ void ln_row_v4(const f32x4 (&v)[C4], int lane, long row, int D,
                                          const float* __restrict__ gamma, const float* __restrict__ beta, float eps,
                                          T* __restrict__ out, float* __restrict__ stats,
                                          unsigned char* __restrict__ lo4, unsigned char* __restrict__ lo_sc,
                                          _Float16* __restrict__ o16) {
    float s = 0.f;
#pragma unroll
    for (int c = 0; c < C4; ++c) s += hsum(v[c]);
    const float mu = wave_sum(s) / D;
    float q = 0.f;
#pragma unroll
    for (int c = 0; c < C4; ++c) {
        const f32x4 t = v[c] - mu;
        q += hsum(t * t);
    }
    const float rstd = 1.f / sqrtf(wave_sum(q) / D + eps);
    const f32x4* g4 = reinterpret_cast<const f32x4*>(gamma);
    const f32x4* b4 = reinterpret_cast<const f32x4*>(beta);
    T* orow = out + row * D;
    f32x4 lo[C4];
    float amax = 0.f;
#pragma unroll
    for (int c = 0; c < C4; ++c) {
        const int i = lane + 64 * c;
        const f32x4 y = g4[i] * ((v[c] - mu) * rstd) + b4[i];
        Out4<T>::store(orow + 4 * i, y);
        if (o16)
            *reinterpret_cast<f16x4*>(o16 + row * D + 4 * i) = {(_Float16)y[0], (_Float16)y[1], (_Float16)y[2],
                                                                (_Float16)y[3]};
        lo[c] = Out4<T>::residual(y);
        amax = fmaxf(amax, fmaxf(fmaxf(fabsf(lo[c][0]), fabsf(lo[c][1])), fmaxf(fabsf(lo[c][2]), fabsf(lo[c][3]))));
    }
    if (lo4) {
        // fp4 rounding residuals: the lane's 4 consecutive features fill 2 bytes
        const unsigned sc = e8m0_for_amax(wave_max(amax));
        const float inv = e8m0_inv(sc);
        unsigned short* lrow = reinterpret_cast<unsigned short*>(lo4 + row * (D / 2));
#pragma unroll
        for (int c = 0; c < C4; ++c) {
            const unsigned q = e2m1_code(lo[c][0] * inv) | (e2m1_code(lo[c][1] * inv) << 4) |
                               (e2m1_code(lo[c][2] * inv) << 8) | (e2m1_code(lo[c][3] * inv) << 12);
            lrow[lane + 64 * c] = (unsigned short)q;
        }
        if (lane == 0) lo_sc[row] = (unsigned char)sc;
    }
    if (stats && lane == 0) {
        stats[2 * row] = mu;
        stats[2 * row + 1] = rstd;
    }
}

// One wave per row: the row's float4 chunks lane + 64 c (c < C4), then ln_row_v4.
template <typename T, int C4>
__global__ void __launch_bounds__(256) ln_fwd_v4(const float* __restrict__ x, long rows, int D,
                                                 const float* __restrict__ gamma, const float* __restrict__ beta,
                                                 float eps, T* __restrict__ out, float* __restrict__ stats,
                                                 unsigned char* __restrict__ lo4, unsigned char* __restrict__ lo_sc,
                                                 _Float16* __restrict__ o16) {
    const int lane = threadIdx.x & 63;
    const long row = (long)blockIdx.x * LN_WAVES + (threadIdx.x >> 6);
    if (row >= rows) return;
    const f32x4* xr = reinterpret_cast<const f32x4*>(x + row * D);
    f32x4 v[C4];
#pragma unroll
    for (int c = 0; c < C4; ++c) v[c] = xr[lane + 64 * c];
    ln_row_v4<T, C4>(v, lane, row, D, gamma, beta, eps, out, stats, lo4, lo_sc, o16);
}

// The split-K reduce of a residual GEMM fused with the LayerNorm of its
// result (same wave-per-row layout as ln_fwd_v4): each chunk of x is the sum
// of the split partials, in split order, plus (residual + bias) -- the
// operations of the GEMM's own reduce -- stored in fp32 (and as a bf16 copy
// when xc is given) and normalised from registers.
template <typename T, int C4>
__global__ void __launch_bounds__(256) ln_fwd_res_v4(const float* __restrict__ ws, int splits, long plane,
                                                     const float* __restrict__ bias, const float* res, float* xo,
                                                     bf16* __restrict__ xc, long rows, int D,
                                                     const float* __restrict__ gamma, const float* __restrict__ beta,
                                                     float eps, T* __restrict__ out, float* __restrict__ stats,
                                                     unsigned char* __restrict__ lo4, unsigned char* __restrict__ lo_sc,
                                                     _Float16* __restrict__ o16) {
    const int lane = threadIdx.x & 63;
    const long row = (long)blockIdx.x * LN_WAVES + (threadIdx.x >> 6);
    if (row >= rows) return;
    const f32x4* p4 = reinterpret_cast<const f32x4*>(ws + row * D);
    const f32x4* r4 = reinterpret_cast<const f32x4*>(res + row * D);
    const f32x4* b4 = reinterpret_cast<const f32x4*>(bias);
    f32x4* x4 = reinterpret_cast<f32x4*>(xo + row * D);
    const long plane4 = plane / 4;
    f32x4 v[C4];
#pragma unroll
    for (int c = 0; c < C4; ++c) {
        const int i = lane + 64 * c;
        f32x4 s = p4[i];
        for (int k = 1; k < splits; ++k) s += p4[i + k * plane4];
        const f32x4 bv = bias ? b4[i] : f32x4{0.f, 0.f, 0.f, 0.f};
        s += r4[i] + bv;
        v[c] = s;
        x4[i] = s;
        if (xc) *reinterpret_cast<bf16x4*>(xc + row * D + 4 * i) = {(bf16)s[0], (bf16)s[1], (bf16)s[2], (bf16)s[3]};
    }
    ln_row_v4<T, C4>(v, lane, row, D, gamma, beta, eps, out, stats, lo4, lo_sc, o16);
}

template <typename T, int C4>
__global__ void __launch_bounds__(256) ln_bwd_v4(const float* __restrict__ dn, const float* __restrict__ x,
                                                 const float* __restrict__ stats, const float* __restrict__ gamma,
                                                 long rows, int D, int rpw, const float* __restrict__ dres,
                                                 float* __restrict__ dx32, T* __restrict__ dxe,
                                                 float* __restrict__ partial, int accumulate, int dn_splits,
                                                 long dn_plane) {
    __shared__ f32x4 red[LN_WAVES][2][C4 * 64];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const f32x4* g4 = reinterpret_cast<const f32x4*>(gamma);
    f32x4 pg[C4], pb[C4];
#pragma unroll
    for (int c = 0; c < C4; ++c) pg[c] = pb[c] = f32x4{0.f, 0.f, 0.f, 0.f};
    const long row0 = ((long)blockIdx.x * LN_WAVES + wave) * rpw;
    const int nr = (int)max(0L, min((long)rpw, rows - row0));
    // the next row's operands are loaded while the current row is computed
    f32x4 dv[C4], xv[C4], rv[C4];
    float mu = 0.f, rstd = 0.f;
    auto load = [&](long row, f32x4* d, f32x4* xx, f32x4* r, float& m, float& s) {
        m = stats[2 * row];
        s = stats[2 * row + 1];
        const f32x4* dn4 = reinterpret_cast<const f32x4*>(dn + row * D);
        const f32x4* x4 = reinterpret_cast<const f32x4*>(x + row * D);
        const f32x4* r4 = reinterpret_cast<const f32x4*>(dres + row * D);
#pragma unroll
        for (int c = 0; c < C4; ++c) {
            // dn_splits > 1: dn is the split-K partials of the GEMM that produced
            // it, summed here in split order (the order of that GEMM's reduce)
            d[c] = dn4[lane + 64 * c];
            for (int k = 1; k < dn_splits; ++k) d[c] += dn4[lane + 64 * c + k * (dn_plane / 4)];
            xx[c] = x4[lane + 64 * c];
            r[c] = dres ? r4[lane + 64 * c] : f32x4{0.f, 0.f, 0.f, 0.f};
        }
    };
    if (nr > 0) load(row0, dv, xv, rv, mu, rstd);
    for (int rr = 0; rr < nr; ++rr) {
        const long row = row0 + rr;
        f32x4 dv2[C4], xv2[C4], rv2[C4];
        float mu2 = 0.f, rstd2 = 0.f;
        if (rr + 1 < nr) load(row + 1, dv2, xv2, rv2, mu2, rstd2);
        f32x4 g[C4], xh[C4];
        float sg = 0.f, sgx = 0.f;
#pragma unroll
        for (int c = 0; c < C4; ++c) {
            const int i = lane + 64 * c;
            xh[c] = (xv[c] - mu) * rstd;
            g[c] = dv[c] * g4[i];
            pg[c] += dv[c] * xh[c];
            pb[c] += dv[c];
            sg += hsum(g[c]);
            sgx += hsum(g[c] * xh[c]);
        }
        sg = wave_sum(sg) / D;
        sgx = wave_sum(sgx) / D;
#pragma unroll
        for (int c = 0; c < C4; ++c) {
            const int i = lane + 64 * c;
            const f32x4 r = rstd * (g[c] - sg - xh[c] * sgx) + rv[c];
            if (dx32) reinterpret_cast<f32x4*>(dx32 + row * D)[i] = r;
            if (dxe) Out4<T>::store(dxe + row * D + 4 * i, r);
        }
        if (rr + 1 < nr) {
#pragma unroll
            for (int c = 0; c < C4; ++c) {
                dv[c] = dv2[c];
                xv[c] = xv2[c];
                rv[c] = rv2[c];
            }
            mu = mu2;
            rstd = rstd2;
        }
    }
#pragma unroll
    for (int c = 0; c < C4; ++c) {
        red[wave][0][lane + c * 64] = pg[c];
        red[wave][1][lane + c * 64] = pb[c];
    }
    __syncthreads();
    const int n4 = D / 4;
    for (int i = threadIdx.x; i < 2 * n4; i += 256) {
        const int which = i / n4, d = i % n4;
        f32x4 t = red[0][which][d];
#pragma unroll
        for (int w = 1; w < LN_WAVES; ++w) t += red[w][which][d];
        f32x4* pp = reinterpret_cast<f32x4*>(partial + (long)blockIdx.x * 2 * D + which * D) + d;
        if (accumulate) t += *pp;
        *pp = t;
    }
}

template <typename T>
gp_status ln_fwd_t(const float* x, long rows, int D, const float* g, const float* b, float eps, void* out,
                   float* stats, unsigned char* lo4, unsigned char* lo_sc, _Float16* o16, hipStream_t st) {
    const int grid = (int)((rows + LN_WAVES - 1) / LN_WAVES);
    T* o = reinterpret_cast<T*>(out);
    if (D % 256 == 0 && D <= 2048) {
        switch (D / 256) {
        case 1: klaunch(ln_fwd_v4<T, 1>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc, o16); break;
        case 2: klaunch(ln_fwd_v4<T, 2>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc, o16); break;
        case 3: klaunch(ln_fwd_v4<T, 3>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc, o16); break;
        case 4: klaunch(ln_fwd_v4<T, 4>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc, o16); break;
        case 5: klaunch(ln_fwd_v4<T, 5>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc, o16); break;
        case 6: klaunch(ln_fwd_v4<T, 6>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc, o16); break;
        case 7: klaunch(ln_fwd_v4<T, 7>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc, o16); break;
        default: klaunch(ln_fwd_v4<T, 8>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc, o16); break;
        }
        GP_LAUNCH_CHECK();
        return GP_OK;
    }
    const int C = (D + 63) / 64;
    if (C <= 1) klaunch(ln_fwd_kernel<T, 1>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc);
    else if (C <= 2) klaunch(ln_fwd_kernel<T, 2>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc);
    else if (C <= 4) klaunch(ln_fwd_kernel<T, 4>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc);
    else if (C <= 8) klaunch(ln_fwd_kernel<T, 8>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc);
    else if (C <= 16) klaunch(ln_fwd_kernel<T, 16>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc);
    else if (C <= 32) klaunch(ln_fwd_kernel<T, 32>, grid, 256, 0, st, x, rows, D, g, b, eps, o, stats, lo4, lo_sc);
    else return set_error(GP_ERR_UNSUPPORTED, "layernorm: d_model > 2048");
    GP_LAUNCH_CHECK();
    return GP_OK;
}

template <typename T>
gp_status ln_bwd_t(const float* dn, const float* x, const float* stats, const float* gamma, long rows, int D,
                   const float* dres, float* dx32, void* dxe, float* partial, int accumulate, int* nblk,
                   int dn_splits, long dn_plane, hipStream_t st) {
    const int rpw = ln_bwd_rows_per_wave(rows);
    const int grid = (int)((rows + (long)LN_WAVES * rpw - 1) / ((long)LN_WAVES * rpw));
    *nblk = grid;
    T* e = reinterpret_cast<T*>(dxe);
    if (D % 256 == 0 && D <= 2048) {
#define GP_LNV(CC) klaunch(ln_bwd_v4<T, CC>, grid, 256, 0, st, dn, x, stats, gamma, rows, D, rpw, dres, dx32, e, partial, \
                           accumulate, dn_splits, dn_plane)
        switch (D / 256) {
        case 1: GP_LNV(1); break;
        case 2: GP_LNV(2); break;
        case 3: GP_LNV(3); break;
        case 4: GP_LNV(4); break;
        case 5: GP_LNV(5); break;
        case 6: GP_LNV(6); break;
        case 7: GP_LNV(7); break;
        default: GP_LNV(8); break;
        }
#undef GP_LNV
        GP_LAUNCH_CHECK();
        return GP_OK;
    }
    if (dn_splits > 1) return set_error(GP_ERR_UNSUPPORTED, "layernorm backward over split-K partials: d_model % 256");
    const int C = (D + 63) / 64;
#define GP_LNB(CC) klaunch(ln_bwd_kernel<T, CC>, grid, 256, 0, st, dn, x, stats, gamma, rows, D, rpw, dres, dx32, e, partial, accumulate)
    if (C <= 1) GP_LNB(1);
    else if (C <= 2) GP_LNB(2);
    else if (C <= 4) GP_LNB(4);
    else if (C <= 8) GP_LNB(8);
    else if (C <= 16) GP_LNB(16);
    else if (C <= 32) GP_LNB(32);
    else return set_error(GP_ERR_UNSUPPORTED, "layernorm: d_model > 2048");
#undef GP_LNB
    GP_LAUNCH_CHECK();
    return GP_OK;
}

} // namespace

int layernorm_bwd_blocks(long rows) {
    const int rpw = ln_bwd_rows_per_wave(rows);
    return (int)((rows + (long)LN_WAVES * rpw - 1) / ((long)LN_WAVES * rpw));
}

gp_status layernorm_fwd(int dtype, const float* x, long rows, int D, const float* gamma, const float* beta,
                        float eps, void* out, float* stats, void* lo4, unsigned char* lo_sc, hipStream_t st,
                        void* out16) {
    unsigned char* l4 = static_cast<unsigned char*>(lo4);
    if (l4 && (dtype != GP_BF16 || D % 64 || !lo_sc))
        return set_error(GP_ERR_UNSUPPORTED, "layernorm: fp4 residuals need bf16 output and d_model % 64 == 0");
    if (out16 && (dtype != GP_BF16 || D % 256 || D > 2048))
        return set_error(GP_ERR_UNSUPPORTED, "layernorm: an fp16 copy needs bf16 output and d_model % 256 == 0");
    _Float16* o16 = static_cast<_Float16*>(out16);
    if (dtype == GP_BF16) return ln_fwd_t<bf16>(x, rows, D, gamma, beta, eps, out, stats, l4, lo_sc, o16, st);
    return ln_fwd_t<float>(x, rows, D, gamma, beta, eps, out, stats, nullptr, nullptr, nullptr, st);
}

bool layernorm_fwd_res_ok(int dtype, int D, const void* ws, const float* bias, const float* res, const float* xo,
                          const void* xc) {
    auto a16 = [](const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; };
    return dtype == GP_BF16 && D % 256 == 0 && D >= 256 && D <= 2048 && ws && res && xo && a16(ws) && a16(bias) &&
           a16(res) && a16(xo) && (!xc || (reinterpret_cast<uintptr_t>(xc) & 7) == 0);
}

gp_status layernorm_fwd_res(int dtype, const float* ws, int splits, long plane, const float* bias, const float* res,
                            float* xo, void* xc, long rows, int D, const float* gamma, const float* beta, float eps,
                            void* out, float* stats, void* lo4, unsigned char* lo_sc, hipStream_t st, void* out16) {
    if (!layernorm_fwd_res_ok(dtype, D, ws, bias, res, xo, xc) || splits < 1 || plane % 4 || plane < rows * D)
        return set_error(GP_ERR_UNSUPPORTED, "layernorm with split-K reduce: bf16, d_model % 256 == 0 (<= 2048), "
                                             "aligned rows");
    unsigned char* l4 = static_cast<unsigned char*>(lo4);
    if (l4 && (D % 64 || !lo_sc)) return set_error(GP_ERR_UNSUPPORTED, "layernorm: fp4 residuals need an E8M0 scale row");
    const int grid = (int)((rows + LN_WAVES - 1) / LN_WAVES);
    bf16* o = reinterpret_cast<bf16*>(out);
    bf16* c = reinterpret_cast<bf16*>(xc);
    _Float16* o16 = static_cast<_Float16*>(out16);
#define GP_LNR(C4) klaunch(ln_fwd_res_v4<bf16, C4>, grid, 256, 0, st, ws, splits, plane, bias, res, xo, c, rows, D, \
                           gamma, beta, eps, o, stats, l4, lo_sc, o16)
    switch (D / 256) {
    case 1: GP_LNR(1); break;
    case 2: GP_LNR(2); break;
    case 3: GP_LNR(3); break;
    case 4: GP_LNR(4); break;
    case 5: GP_LNR(5); break;
    case 6: GP_LNR(6); break;
    case 7: GP_LNR(7); break;
    default: GP_LNR(8); break;
    }
#undef GP_LNR
    GP_LAUNCH_CHECK();
    return GP_OK;
}

gp_status layernorm_bwd(int dtype, const float* dn, const float* x, const float* stats, const float* gamma,
                        long rows, int D, const float* dres, float* dx_f32, void* dx_elt, float* partial,
                        int accumulate, int* nblk, hipStream_t st, int dn_splits, long dn_plane) {
    if (dn_splits < 1 || (dn_splits > 1 && (dn_plane < rows * D || dn_plane % 4)))
        return set_error(GP_ERR_INVALID_ARG, "layernorm backward: split-K partial layout");
    if (dtype == GP_BF16)
        return ln_bwd_t<bf16>(dn, x, stats, gamma, rows, D, dres, dx_f32, dx_elt, partial, accumulate, nblk,
                              dn_splits, dn_plane, st);
    return ln_bwd_t<float>(dn, x, stats, gamma, rows, D, dres, dx_f32, dx_elt, partial, accumulate, nblk, dn_splits,
                           dn_plane, st);
}

gp_status colsum_finalize(const float* partial, int nblk, int width, float* out, int accumulate, hipStream_t st) {
    klaunch(colsum_kernel, (width + 63) / 64, 1024, 0, st, partial, nblk, width, out, accumulate);
    GP_LAUNCH_CHECK();
    return GP_OK;
}

} // namespace gp
