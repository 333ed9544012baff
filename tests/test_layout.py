"""CPU checks of the packed-layout transform used by the parity tests
(tests/packed_layout.py) against the layout as include/micromix.h states it,
written out byte by byte, and of its round trip."""

import numpy as np
import pytest

from tests import packed_layout as L


def _rand_rowmajor(rng, rows, split):
    p4, p6, p8 = split
    return (rng.integers(0, 256, (rows, p4 // 2), dtype=np.uint8), rng.integers(0, 256, (rows, 3 * p6 // 4), dtype=np.uint8),
            rng.integers(0, 256, (rows, p8), dtype=np.uint8), rng.integers(0, 256, (rows, sum(split) // 32), dtype=np.uint8))


@pytest.mark.parametrize("rows,split", [(5, (96, 160, 96)), (33, (128, 128, 128)), (64, (32, 0, 288)), (1, (0, 64, 0))])
def test_tile_matches_header_formula(rows, split):
    """Every code byte lands where the header's formula puts it; padding is zero."""
    rng = np.random.default_rng(rows)
    q4, q6, q8, sc = _rand_rowmajor(rng, rows, split)
    t = L.tile(q4, q6, q8, sc, rows, split)
    geo = L.geometry(rows, split)
    rp = geo["rp"]
    seen = {k: np.zeros(len(v), bool) for k, v in t.items()}
    for g, (name, arr) in enumerate((("q4", q4), ("q6", q6), ("q8", q8))):
        RB, bb = L.STEP_ROW_BYTES[g], L.BLOCK_BYTES[g]
        for n in range(rows):
            for b in range(geo["nb"][g]):
                s, j, q, r = b // 4, b % 4, n // 32, n % 32
                rec = s * rp * RB + q * 32 * RB
                blk = arr[n, b * bb:(b + 1) * bb]
                if g == 0:
                    pos = [rec + j * 512 + r * 16 + i for i in range(16)]
                elif g == 1:
                    pos = [rec + j * 768 + r * 24 + i for i in range(24)]
                else:
                    pos = [rec + (2 * j + i // 16) * 512 + r * 16 + i % 16 for i in range(32)]
                assert np.array_equal(t[name][pos], blk)
                seen[name][pos] = True
    t0 = [0, geo["steps"][0], geo["steps"][0] + geo["steps"][1]]
    b0 = [0, geo["nb"][0], geo["nb"][0] + geo["nb"][1]]
    for g in range(3):
        for n in range(rows):
            for b in range(geo["nb"][g]):
                pos = ((t0[g] + b // 4) * rp + n) * 4 + b % 4
                assert t["sc"][pos] == sc[n, b0[g] + b]
                seen["sc"][pos] = True
    for k in t:
        assert len(t[k]) == geo["bytes"]["q4 q6 q8 sc".split().index(k)]
        assert not t[k][~seen[k]].any(), f"{k}: padding not zero"


@pytest.mark.parametrize("rows,split", [(7, (64, 96, 32)), (70, (256, 0, 64))])
def test_untile_inverts_tile(rows, split):
    rng = np.random.default_rng(7 + rows)
    q4, q6, q8, sc = _rand_rowmajor(rng, rows, split)
    back = L.untile(L.tile(q4, q6, q8, sc, rows, split), rows, split)
    for name, ref in (("q4", q4), ("q6", q6), ("q8", q8), ("sc", sc)):
        assert np.array_equal(back[name], ref), name
