"""Index algebra of the frame-wise kernels' register tile layouts, checked on
the CPU (the GPU parity tests check the kernels themselves).

* P32 accumulator tiles of a Gram matrix: lane (li, lg), value q of tile
  (r, c) holds G[32 (r // 2) + 8 lg + 4 (r % 2) + q][32 (c // 2) + 8 (li // 4)
  + 4 (c % 2) + li % 4].  The split partials keep the tiles with c >= r; the
  reduction rebuilds a tile below the diagonal from its mirror: lane (li, lg)
  value q of tile (r, c) is lane (4 lg + q) + 16 (li // 4) value li % 4 of
  tile (c, r).
* The fused output deals channel 32 kb + 8 m + 4 e + q to row 4 m + q of tile
  2 kb + e (fused_out_chan), so that accumulator lane (li, lg) of tiles 2 kb
  and 2 kb + 1 holds the 8 consecutive channels 32 kb + 8 lg .. + 7.
"""
import numpy as np
import pytest


def p32_tile(G, r, c):
    T = np.zeros((64, 4))
    for lane in range(64):
        li, lg = lane % 16, lane // 16
        for q in range(4):
            T[lane, q] = G[32 * (r // 2) + 8 * lg + 4 * (r % 2) + q,
                           32 * (c // 2) + 8 * (li // 4) + 4 * (c % 2) + li % 4]
    return T


def mirrored(T):
    U = np.zeros((64, 4))
    for lane in range(64):
        li, lg = lane % 16, lane // 16
        for q in range(4):
            U[lane, q] = T[(4 * lg + q) + 16 * (li // 4), li % 4]
    return U


def fused_out_chan(jo, i):
    return 32 * (jo >> 1) + 8 * (i >> 2) + 4 * (jo & 1) + (i & 3)


@pytest.mark.parametrize("dk", [64, 128])
def test_gram_mirror_rebuilds_lower_tiles(dk):
    rng = np.random.default_rng(dk)
    a = rng.standard_normal((dk, dk))
    G = a @ a.T                                      # symmetric, as K^T B K is
    R = dk // 16
    for r in range(R):
        for c in range(R):
            assert np.array_equal(p32_tile(G, r, c), mirrored(p32_tile(G, c, r))), (r, c)
    # a non-symmetric matrix is not rebuilt: the mapping relies on symmetry
    b = rng.standard_normal((dk, dk))
    assert not np.array_equal(p32_tile(b, 1, 0), mirrored(p32_tile(b, 0, 1)))


@pytest.mark.parametrize("dv", [64, 128])
def test_fused_output_channel_order(dv):
    tiles = dv // 16
    chans = sorted(fused_out_chan(jo, i) for jo in range(tiles) for i in range(16))
    assert chans == list(range(dv))                  # every channel exactly once
    for kb in range(dv // 32):
        for lg in range(4):
            # accumulator rows 4 lg + q of tiles 2 kb (q = 0..3) and 2 kb + 1
            got = [fused_out_chan(2 * kb + e, 4 * lg + q) for e in range(2) for q in range(4)]
            assert got == list(range(32 * kb + 8 * lg, 32 * kb + 8 * lg + 8))
