"""Host emulation of gemm_bf16_kernel's (csrc/gemm.hip) index arithmetic: for
its one allowed geometry (128 x 128 tiles, 2 x 2 waves, 4 stages, 2 blocks
per CU) and for the larger geometries an earlier sweep built (256 x 256 with
4 stages, 256 x 128 with 6, 128 x 256 with 4), every LDS write of the
operand loads, every LDS fragment read, every epilogue staging access and the
memory-counter arithmetic stay within their ranges.  What separates the
swept geometries is the register budget: their accumulators and operand
fragments alone leave a wave too few registers for addresses, loop state and
the epilogue, so those builds spill (the kernel's inline-asm LDS reads must
not be spilled between issue and wait), which is why the kernel now rejects
them at compile time."""
import itertools

import pytest

BK = 32


def hsw(k):
    return 2 * ((k & 3) | (((k >> 3) & 1) << 2))


def check_geometry(BM, BN, WGM, WGN, STAGES):
    NW = WGM * WGN
    WTM, WTN = BM // WGM, BN // WGN
    FM, FN = WTM // 16, WTN // 16
    STAGE = (BM + BN) * BK                                    # elements per stage
    lds_elems = STAGES * STAGE
    # loads: K-contiguous tile (one 1 KiB fragment per wave instruction) and MN-contiguous tile
    for ROWS in (BM, BN):
        NI = ROWS // 16 // NW
        assert NI >= 1 and ROWS % (16 * NW) == 0
        for i, wid in itertools.product(range(NI), range(NW)):
            q = i * NW + wid
            assert 0 <= q * 512 and q * 512 + 512 <= ROWS * BK   # K-contiguous: fragment q
        CPR = ROWS // 8
        NIm = BK * CPR // 64 // NW
        assert NIm >= 1 and CPR >= 16
        for i, wid in itertools.product(range(NIm), range(NW)):
            q = i * NW + wid
            assert q * 512 + 512 <= BK * ROWS                      # MN-contiguous: 64 chunks per instruction
    # fragment reads (K-contiguous: fragment (r0 / 16 + c) of the stage, 16 bytes per lane)
    for wm, wn, lane in itertools.product(range(WGM), range(WGN), range(64)):
        for u in range(FM):
            a = ((wm * WTM) // 16 + u) * 512 + lane * 8
            assert 0 <= a and a + 8 <= BM * BK
        for u in range(FN):
            b = ((wn * WTN) // 16 + u) * 512 + lane * 8
            assert 0 <= b and b + 8 <= BN * BK
        # MN-contiguous (transposed) reads: rows k and k + 4, 4 columns each
        j = lane & 15
        k = 8 * (lane >> 4) + (j >> 2)
        for COLS, c0, NF in ((BM, wm * WTM, FM), (BN, wn * WTN, FN)):
            for c in range(NF):
                col = c0 + 16 * c + 4 * (j & 3)
                for kk in (k, k + 4):
                    off = kk * COLS + (((col >> 3) ^ hsw(kk)) << 3) + (col & 7)
                    assert 0 <= off and off + 4 <= BK * COLS
    # epilogue staging through LDS (float), one slice per wave
    EPI_LD = WTN + 4
    EPI_ROWS = 32 if NW * 32 * EPI_LD * 4 <= STAGES * STAGE * 2 else 16
    assert WTM % EPI_ROWS == 0 and NW * EPI_ROWS * EPI_LD * 4 <= STAGES * STAGE * 2
    for wid in range(NW):
        base = wid * EPI_ROWS * EPI_LD
        for ii, g4, v, jj, l in itertools.product(range(EPI_ROWS // 16), range(4), range(4), range(FN), range(16)):
            idx = base + (ii * 16 + 4 * g4 + v) * EPI_LD + jj * 16 + l
            assert idx < base + EPI_ROWS * EPI_LD and idx * 4 < lds_elems * 2
        for q in range(EPI_ROWS * (WTN // 8)):
            rr, cc = q // (WTN // 8), q % (WTN // 8)
            assert base + rr * EPI_LD + cc * 8 + 8 <= base + EPI_ROWS * EPI_LD
    # memory counter: loads per wave per stage times the stages in flight fit vmcnt's 6 bits
    LPS = BM // 16 // NW + BN // 16 // NW
    assert LPS * (STAGES - 1) < 64
    return dict(acc=FM * FN * 4, frags=2 * (FM + FN) * 4, lds_bytes=lds_elems * 2 + (64 + 1) * 4)


def test_allowed_geometry_fits():
    r = check_geometry(128, 128, 2, 2, 4)
    assert r["lds_bytes"] * 2 <= 160 * 1024          # two blocks per CU
    assert r["acc"] + r["frags"] <= 256 - 32          # registers at two waves per SIMD, with room for addresses


@pytest.mark.parametrize("geom", [(256, 256, 2, 2, 4), (256, 128, 2, 2, 6), (128, 256, 2, 2, 4)])
def test_swept_geometries_index_in_range_but_crowd_the_registers(geom):
    r = check_geometry(*geom)
    assert r["lds_bytes"] <= 160 * 1024
    # the allowed geometry keeps half of a wave's 256 registers free of accumulators and
    # fragments; these keep 32 or fewer
    assert r["acc"] + r["frags"] >= 256 - 32
    ok = check_geometry(128, 128, 2, 2, 4)
    assert ok["acc"] + ok["frags"] == 128
