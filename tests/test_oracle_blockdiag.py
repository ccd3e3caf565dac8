"""Pins for the oracle's per-block diagnostic (oracle_attn_diag): the gap of
each block below the running maximum and the zero codes per block.

The paper replaces the single sink gap Delta by the gap of each block when
sinks are spread over the sequence (Limitations and Future Work, "Multi-sink
patterns").  The oracle measures, per row and visited block, g = -(the
block's largest exponent argument), so the block's largest P is 2^-g, and
bins floor(g).  The checks tie it to an independent numpy computation of the
same gap in FP64 from the definition (running maximum over the visited blocks,
block maximum, scaled by log2(e)/sqrt(d)), to closed-form row and key counts,
to the per-row counts, to Theorem 2 (reverse order with S = 256 zeroes
nothing outside the sink's block), and to Prop. 1 (a block whose gap reaches
10 + log2 S is zeroed whole).
"""
import numpy as np
import pytest

import oracle
from paper_2606_06521_amd.inputs import make_inputs

NB = 32


def _numpy_gaps(q, k, Bc, order, causal, scale):
    """g[r, j] (NaN where row r does not visit block j) in FP64 from the
    definition: m = running max of the raw dots over the blocks visited so
    far (this one included), M = block j's max, g = (m - M) log2(e) scale."""
    N = q.shape[0]
    D = q.astype(np.float64) @ k.astype(np.float64).T
    nblk = (N + Bc - 1) // Bc
    g = np.full((N, nblk), np.nan)
    for r in range(N):
        L = r + 1 if causal else N
        nb = (L + Bc - 1) // Bc
        seq = range(nb) if order == "forward" else range(nb - 1, -1, -1)
        m = -np.inf
        for j in seq:
            M = D[r, j * Bc:min((j + 1) * Bc, L)].max()
            m = max(m, M)
            g[r, j] = (m - M) * np.log2(np.e) * scale
    return g


@pytest.mark.parametrize("order", ["forward", "reverse"])
@pytest.mark.parametrize("causal", [False, True])
def test_gap_histogram_matches_numpy_definition(order, causal):
    inp = make_inputs(1, 2, 1, 300, 64, fmt="f32", delta=9.0, seed=71)
    Bc = 64
    _, _, cnt, hist, bz = oracle.block_diag(inp.q32, inp.k32, inp.v32, S=256.0, order=order,
                                            block_kv=Bc, causal=causal, nbins=NB)
    amb = 0
    for h in range(2):
        g = _numpy_gaps(inp.q32[0, h], inp.k32[0, 0], Bc, order, causal, 1.0 / np.sqrt(64))
        want = np.zeros((g.shape[1], NB), np.int64)
        for j in range(g.shape[1]):
            col = g[:, j][~np.isnan(g[:, j])]
            # a gap within 1e-4 of an integer may fall on either side in FP32
            amb += int(np.sum((np.abs(col - np.rint(col)) < 1e-4) & (col > 0.5)))
            b = np.clip(np.floor(col), 0, NB - 1).astype(int)
            np.add.at(want[j], b, 1)
        diff = np.abs(hist[0, h].astype(np.int64) - want).sum()
        assert diff <= 2 * amb, (h, diff, amb)


@pytest.mark.parametrize("order", ["forward", "reverse"])
@pytest.mark.parametrize("causal", [False, True])
def test_counts_add_up(order, causal):
    N, Bc = 333, 64
    inp = make_inputs(2, 4, 2, N, 64, fmt="bf16_e4m3", delta=10.0, seed=72)
    _, _, cnt, hist, bz = oracle.block_diag(inp.q32, inp.k32, inp.v32, S=256.0, order=order,
                                            block_kv=Bc, causal=causal, nbins=NB)
    nblk = (N + Bc - 1) // Bc
    # every row visits every block (non-causal) or the blocks with a key <= r
    visits = np.array([N if not causal else N - j * Bc for j in range(nblk)])
    assert np.array_equal(hist.sum(axis=3), np.broadcast_to(visits, hist.shape[:3]))
    # the per-block zero codes are the per-row counts regrouped
    per_bh = cnt.reshape(2, 4, N, 3).sum(axis=(2, 3))
    assert np.array_equal(bz.sum(axis=2), per_bh)
    if order == "reverse":
        # the first block a row visits holds the running maximum: gap 0
        first = visits.copy()
        first[:-1] -= visits[1:]          # rows whose last block is j
        assert np.all(hist[..., 0] >= first)
        # Theorem 2: reverse order with S = 256 zeroes nothing outside block 0
        assert bz[..., 1:].sum() == 0


def test_blocks_far_below_the_maximum_are_zeroed_whole():
    # a sink gap far past the collapse point: in forward order every later
    # block sits >= 18 = 10 + log2(256) below the sink, so by Prop. 1 all its
    # keys are cast to zero, and its gap lands in the top bin
    N, Bc = 512, 64
    inp = make_inputs(1, 2, 1, N, 64, fmt="f32", delta=60.0, seed=73)
    _, _, cnt, hist, bz = oracle.block_diag(inp.q32, inp.k32, inp.v32, S=256.0, order="forward",
                                            block_kv=Bc, causal=False, nbins=NB)
    assert np.all(hist[0, :, 1:, NB - 1] == N)
    assert np.all(bz[0, :, 1:] == N * Bc)
    # and with the cast off nothing is counted
    _, _, _, _, bz0 = oracle.block_diag(inp.q32, inp.k32, inp.v32, S=256.0, order="forward",
                                        block_kv=Bc, cast=False, nbins=NB)
    assert bz0.sum() == 0


def test_rejects_bad_bins():
    inp = make_inputs(1, 1, 1, 64, 64, fmt="f32", delta=5.0, seed=74)
    for nb in (0, 65):
        with pytest.raises(ValueError):
            oracle.block_diag(inp.q32, inp.k32, inp.v32, S=256.0, order="forward", block_kv=64,
                              nbins=nb)
