"""Index arithmetic of the direct-to-LDS loaders, restated from the kernels
(`kdev.hpp` KM / swz, `wgrad.hip` wgrad_rowg_kernel, `kconv.hpp` lane-order
copies) and checked exhaustively on the CPU:

* a copy instruction writes 1 KiB of LDS in lane order; for every tile
  shape the kernels use, the (k row, 16-byte vector) each lane fetches lands
  exactly once at the byte the swizzled layout assigns to it;
* 16-lane phases of the row-major fragment reads hit 16 distinct 4-bank
  groups for 4- and 8-vector rows;
* the weight gradient's scalar walk of 8-pixel groups over padded rows
  reproduces direct indexing of (image, row, column) and of both operands'
  byte offsets, for random shapes, strides, paddings and split chunks.
"""
import random


def km_sw(W, k):
    c = W // 32
    return (k & 3) if c >= 4 else ((k >> 1) & 1) if c == 2 else 0


def km_off(W, k, col):
    """Element offset of (k, col) in a W-wide k-major bf16 tile."""
    return k * W + (col ^ (km_sw(W, k) << 5))


def swz(kr, row, vec):
    return vec ^ ((row >> 1) & 7) if kr == 8 else vec ^ ((row >> 2) & 3)


def test_weight_gradient_copies_fill_km_tiles():
    # A tiles (W = 64 or 128 output channels) and B tiles (W = 128 columns),
    # 32 k rows: wave w's copy j covers rows (w * NI + j) * R .. + R - 1
    for W in (64, 128):
        V, R = W // 8, 64 // (W // 8)
        NI = 32 // R // 4
        seen = {}
        for wave in range(4):
            for lane in range(64):
                vec = (lane % V) ^ (km_sw(W, lane // V) << 2)
                for j in range(NI):
                    k = (wave * NI + j) * R + lane // V
                    addr = (wave * NI + j) * 1024 + lane * 16
                    assert addr == km_off(W, k, vec * 8) * 2
                    assert (k, vec) not in seen
                    seen[(k, vec)] = addr
        assert len(seen) == 32 * V


def test_input_gradient_weight_copies_fill_km_tiles():
    # k-major weight tile of the stride-1 bf16 input gradient: thread tid,
    # copy j, row bk0 + BKS j, column vector permuted within its row
    for BN in (64, 128):
        for kr in (4, 8):
            BV = BN // 8
            BKS = 256 // BV
            NBL = BN * kr // 256
            seen = set()
            for tid in range(256):
                wave, lane = tid // 64, tid % 64
                bk0 = tid // BV
                col = 8 * ((tid % BV) ^ (km_sw(BN, bk0) << 2))
                for j in range(NBL):
                    k = bk0 + BKS * j
                    addr = ((wave * 64) // BV + BKS * j) * BN * 2 + lane * 16
                    assert addr == km_off(BN, k, col) * 2
                    assert (k, col) not in seen
                    seen.add((k, col))
            assert len(seen) == 8 * kr * BV


def test_row_major_lane_order_copies_and_reads():
    for kr in (4, 8):
        rs = 256 // kr
        for tid in range(256):
            kv = ((tid & 7) ^ ((tid >> 4) & 7)) if kr == 8 else ((tid & 3) ^ ((tid >> 4) & 3))
            wave, lane = tid // 64, tid % 64
            for i in range(kr // 2):
                row = tid // kr + rs * i
                assert swz(kr, row, kv) == tid % kr
                assert row * kr * 16 + swz(kr, row, kv) * 16 == \
                    (wave * (64 // kr) + rs * i) * kr * 16 + lane * 16
        for r0 in range(0, 128, 16):
            for v in range(kr):
                groups = {((row * kr * 16 + swz(kr, row, v) * 16) // 16) % 16
                          for row in range(r0, r0 + 16)}
                assert len(groups) == 16


def _walk(B, R, Wv, sh, sw, ph, pw, y0, row0, srow, srcC, bs, Co, kchunk_steps):
    BK = 32
    Wp = (Wv + 7) // 8 * 8
    K = B * R * Wp
    wdx, wdy, wdb = BK % Wp, (BK // Wp) % R, BK // (Wp * R)
    dA0 = ((wdb * R + wdy) * Wv + wdx) * Co * 2
    dA1 = (Wv - Wp) * Co * 2
    dyb, ryb = wdy * sh, R * sh
    dB0 = (wdb * bs + dyb * srow + wdx * sw * srcC) * 2
    dB1 = (sh * srow - Wp * sw * srcC) * 2
    dB2 = (bs - ryb * srow) * 2
    kchunk = kchunk_steps * BK
    for z in range((K + kchunk - 1) // kchunk):
        kbeg, kend = z * kchunk, min(K, z * kchunk + kchunk)
        for wave in range(4):
            q = kbeg + 8 * wave
            xs, ys, b = q % Wp, (q // Wp) % R, q // (Wp * R)
            offA = ((b * R + ys) * Wv + xs) * Co * 2
            sy, sx = (y0 + ys) * sh - ph, xs * sw - pw
            offB = (b * bs + (sy - row0) * srow + sx * srcC) * 2
            kl = kend - q
            for step in range((kend - kbeg + BK - 1) // BK):
                qq = kbeg + BK * step + 8 * wave
                X, Y, Bb = qq % Wp, (qq // Wp) % R, qq // (Wp * R)
                assert (xs, ys) == (X, Y) and X % 8 == 0 and X + 8 <= Wp
                assert offA == ((Bb * R + Y) * Wv + X) * Co * 2
                SY, SX = (y0 + Y) * sh - ph, X * sw - pw
                assert (sy, sx) == (SY, SX)
                assert offB == (Bb * bs + (SY - row0) * srow + SX * srcC) * 2
                assert kl == kend - qq
                xs += wdx; ys += wdy; offA += dA0; offB += dB0; sy += dyb
                sx += wdx * sw; kl -= BK
                if xs >= Wp:
                    xs -= Wp; ys += 1; offA += dA1; offB += dB1; sy += sh; sx -= Wp * sw
                if ys >= R:
                    ys -= R; offB += dB2; sy -= ryb


def test_weight_gradient_scalar_walk_matches_direct_indexing():
    rnd = random.Random(7)
    for _ in range(600):
        R, srcW, srcC = rnd.randint(1, 9), rnd.randint(8, 300), rnd.choice([8, 16, 64])
        _walk(B=rnd.randint(1, 4), R=R,
              Wv=rnd.choice([1, 3, 7, 8, 9, 15, 16, 17, 31, 32, 33, 37, 56, 113, 225]),
              sh=rnd.choice([1, 2]), sw=rnd.choice([1, 2]), ph=rnd.randint(0, 3),
              pw=rnd.randint(0, 3), y0=rnd.randint(0, 20), row0=rnd.randint(-2, 5),
              srow=srcW * srcC, srcC=srcC, bs=(2 * R + 8) * srcW * srcC,
              Co=rnd.choice([8, 64, 256]), kchunk_steps=rnd.randint(1, 9))
