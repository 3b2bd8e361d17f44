"""Host check of the GEMM's LDS fragment addressing (csrc/gemm.hip, gemm_dl).

The direct-to-LDS tiles store 16-byte chunk c of row r at c ^ swz(r), with
swz(r) = (r ^ (r >> 3)) & 7 (k-contiguous operands), or chunk c of k-row k at
c ^ 4 (k % 4) (m-contiguous operands).  The kernel does not keep one offset per
(k-step, block): it rebuilds them from a base register, a per-lane swizzle
term and compile-time strides.  This test checks, for every tile shape the
library instantiates, every wave and lane, k-step and block, that the
rebuilt offsets equal the direct formula (the GPU tile-shape parity tests then
check the kernels that use them)."""

TILES = [  # (BM, BN, WM, WN)
    (128, 128, 2, 2), (256, 128, 2, 2), (256, 256, 2, 2), (256, 256, 2, 4), (256, 128, 4, 2), (128, 256, 2, 4),
    (128, 128, 2, 4), (128, 128, 4, 2), (128, 64, 2, 2), (64, 128, 2, 2)]
KS = 4  # 16-deep k-steps per 64-deep k-tile


def swz(r):
    return (r ^ (r >> 3)) & 7


def test_k_contiguous_offsets_rebuild_the_swizzled_chunk_address():
    for BM, BN, WM, WN in TILES:
        TM, TN = BM // WM // 32, BN // WN // 32
        for wave in range(WM * WN):
            wm, wn = wave // WN, wave % WN
            for lane in range(64):
                fr, h = lane & 31, lane >> 5
                w = swz(fr)
                fa_base = (wm * (BM // WM) + fr) * 128 + ((h ^ (w & 1)) << 4)
                fb_base = BM * 128 + (wn * (BN // WN) + fr) * 128 + ((h ^ (w & 1)) << 4)
                swa = (w >> 1) ^ ((((wm * (BM // WM)) >> 5) & 1) << 1)
                swb = (w >> 1) ^ ((((wn * (BN // WN)) >> 5) & 1) << 1)
                for s in range(KS):
                    ta, tb = (s ^ swa) << 5, (s ^ swb) << 5
                    for i in range(TM):
                        row = wm * (BM // WM) + i * 32 + fr
                        want = row * 128 + (((2 * s + h) ^ swz(row)) << 4)
                        assert fa_base + i * 4096 + ((ta ^ 64) if i & 1 else ta) == want, (BM, BN, wave, lane, s, i)
                    for j in range(TN):
                        row = wn * (BN // WN) + j * 32 + fr
                        want = BM * 128 + row * 128 + (((2 * s + h) ^ swz(row)) << 4)
                        assert fb_base + j * 4096 + ((tb ^ 64) if j & 1 else tb) == want, (BM, BN, wave, lane, s, j)


def test_m_contiguous_offsets_step_by_sixteen_k_rows():
    for BM, BN, WM, WN in TILES:
        if BM < 128 or BN < 128:
            continue  # m-contiguous tiles are at least 128 wide
        TM, TN = BM // WM // 32, BN // WN // 32
        for wave in range(WM * WN):
            wm, wn = wave // WN, wave % WN
            for lane in range(64):
                g, q = lane >> 4, lane & 15
                kr, mo = 8 * (g >> 1) + (q >> 2), 16 * (g & 1) + 4 * (q & 3)
                for s in range(KS):
                    k = 16 * s + kr
                    for i in range(TM):
                        m = wm * (BM // WM) + i * 32 + mo
                        want = k * (2 * BM) + (((m >> 3) ^ ((k & 3) << 2)) << 4) + (m & 7) * 2
                        got = kr * (2 * BM) + (((m >> 3) ^ ((kr & 3) << 2)) << 4) + (m & 7) * 2 + s * 32 * BM
                        assert got == want
                    for j in range(TN):
                        n = wn * (BN // WN) + j * 32 + mo
                        want = BM * 128 + k * (2 * BN) + (((n >> 3) ^ ((k & 3) << 2)) << 4) + (n & 7) * 2
                        got = BM * 128 + kr * (2 * BN) + (((n >> 3) ^ ((kr & 3) << 2)) << 4) + (n & 7) * 2 + s * 32 * BN
                        assert got == want
