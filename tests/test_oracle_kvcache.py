"""The oracle on the KV-cache prefill shape: Nq query rows against Nk cached
keys (the short-query shape of Exp. 1, q_len = 32 against N = 4096).  Query
row r sits at key position Nk - Nq + r; under causal masking it sees keys up
to that position.

Pins: every row equals the same row of the full N x N problem bit for bit
(the alignment), with the cast off it equals a numpy FP64 attention written
here with bottom-right causal masking, and the FP64 reference agrees with the
same numpy attention.
"""
import numpy as np
import pytest

import oracle
from paper_2606_06521_amd.inputs import last_queries, make_inputs


def _numpy_attention(q, k, v, causal):
    nq, nk = q.shape[0], k.shape[0]
    z = (q.astype(np.float64) @ k.astype(np.float64).T) / np.sqrt(q.shape[1])
    if causal:
        pos = nk - nq + np.arange(nq)
        z = np.where(np.arange(nk)[None, :] <= pos[:, None], z, -np.inf)
    z = z - z.max(axis=1, keepdims=True)
    p = np.exp(z)
    return (p @ v.astype(np.float64)) / p.sum(axis=1, keepdims=True)


@pytest.mark.parametrize("order", ["forward", "reverse"])
@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("nq", [1, 32, 77])
def test_rows_equal_the_square_problem(order, causal, nq):
    full = make_inputs(2, 4, 2, 300, 64, fmt="bf16_e4m3", delta=8.0, seed=61)
    kv = last_queries(full, nq)
    rows = np.concatenate([bh * 300 + np.arange(300 - nq, 300) for bh in range(8)])
    want = oracle.attn(full.q32, full.k32, full.v32, S=256.0, order=order, block_kv=64,
                       causal=causal, rows=rows)
    got = oracle.attn(kv.q32, kv.k32, kv.v32, S=256.0, order=order, block_kv=64, causal=causal)
    for a, b in zip(want, got):
        assert np.array_equal(a, b)
    # and the per-block diagnostic aggregates the same rows
    _, _, c1, h1, z1 = oracle.block_diag(full.q32, full.k32, full.v32, S=256.0, order=order,
                                         block_kv=64, causal=causal, rows=rows, nbins=16)
    _, _, c2, h2, z2 = oracle.block_diag(kv.q32, kv.k32, kv.v32, S=256.0, order=order,
                                         block_kv=64, causal=causal, nbins=16)
    assert np.array_equal(h1, h2) and np.array_equal(z1, z2) and np.array_equal(c1, c2)


@pytest.mark.parametrize("causal", [False, True])
def test_cast_off_matches_numpy_attention(causal):
    full = make_inputs(1, 2, 1, 250, 64, fmt="f32", delta=6.0, seed=62)
    kv = last_queries(full, 40)
    out, _, _ = oracle.attn(kv.q32, kv.k32, kv.v32, S=16.0, order="reverse", block_kv=64,
                            causal=causal, cast=False)
    ref, _ = oracle.ref_fp64(kv.q32, kv.k32, kv.v32, causal=causal)
    for h in range(2):
        want = _numpy_attention(kv.q32[0, h], kv.k32[0, 0], kv.v32[0, 0], causal)
        assert np.abs(out.reshape(2, 40, 64)[h] - want).max() < 1e-5
        assert np.abs(ref.reshape(2, 40, 64)[h] - want).max() < 1e-12


def test_rejects_more_queries_than_keys():
    full = make_inputs(1, 1, 1, 64, 64, fmt="f32", delta=6.0, seed=63)
    q = np.concatenate([full.q32, full.q32], axis=2)
    with pytest.raises(ValueError):
        oracle.attn(q, full.k32, full.v32, S=256.0, order="forward", block_kv=64)


@pytest.mark.parametrize("nq,nk,causal", [(5, 5, True), (3, 17, True), (7, 7, False), (4, 9, False), (1, 1, True)])
def test_workload_pair_count_is_the_visible_pairs(nq, nk, causal):
    """Workload.pairs() (the exp2 count the benchmark reports) equals a brute
    count of the (row, key) pairs the mask leaves visible, with row r of nq at
    key position nk - nq + r."""
    from paper_2606_06521_amd.workloads import Workload
    w = Workload("t", 2, 3, 3, nk, 64, causal, "fast", 64, (0.0,), (256.0,), ("reverse",),
                 nq=nq if nq < nk else 0)
    brute = sum(1 for r in range(nq) for t in range(nk) if not causal or t <= nk - nq + r)
    assert w.pairs() == 2 * 3 * brute
