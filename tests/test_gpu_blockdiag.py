"""Per-block diagnostic on the device (attn_fp8_block_gap_diag) against the
oracle: the gap histogram and the per-block zero codes are integers decided
by the same FP32 operations on both sides, so they must agree exactly, as the
per-row counts do (faithful mode at any S, the fast modes at S = 2^k)."""
import itertools

import numpy as np
import pytest
import torch

import oracle
from paper_2606_06521_amd.inputs import make_inputs, with_sink_cluster
from paper_2606_06521_amd.workloads import WORKLOADS
from tests.gpu_helpers import log, to_device

pytestmark = pytest.mark.gpu

FMT = {"faithful": "f32", "fast": "bf16_e4m3", "fp8qk": "e4m3"}


def _run(dev, mode, S, order, causal, bkv, scale="static", nbins=32, tile=None):
    from paper_2606_06521_amd import attn_fp8 as A
    q, k, v = dev
    hist, bz, cnt = A.block_gap_diag(q, k, v, S=S, order=order, causal=causal, block_kv=bkv,
                                     mode=mode, nbins=nbins, scale=scale, tile=tile)
    torch.cuda.synchronize()
    return (hist.cpu().numpy().view(np.uint32), bz.cpu().numpy().view(np.uint32),
            cnt.cpu().numpy().view(np.uint32))


@pytest.mark.parametrize("mode,tile", [("faithful", None), ("fast", 256), ("fast", 128),
                                       ("fp8qk", 256), ("fp8qk", 128)])
@pytest.mark.parametrize("d,bkv", [(64, 64), (128, 128), (128, 64)])
def test_small_exact(mode, tile, d, bkv):
    inp = make_inputs(2, 4, 2, 333, d, fmt=FMT[mode], delta=9.0, seed=800 + d + bkv)
    dev = to_device(inp)
    for (causal, order), (S, scale) in itertools.product(
            itertools.product([False, True], ["forward", "reverse"]),
            [(256.0, "static"), (16.0, "dynamic"), (1.0, "static")]):
        label = f"diag {mode} d={d} bkv={bkv} causal={causal} {order} S={S} {scale} tile={tile}"
        log(label)
        hist, bz, cnt = _run(dev, mode, S, order, causal, bkv, scale, tile=tile)
        _, _, o_cnt, o_hist, o_bz = oracle.block_diag(inp.q32, inp.k32, inp.v32, S=S,
                                                      order=order, block_kv=bkv, causal=causal,
                                                      scale=scale, nbins=32)
        assert np.array_equal(hist, o_hist), label
        assert np.array_equal(bz, o_bz), label
        assert np.array_equal(cnt.reshape(-1, 3), o_cnt), label


@pytest.mark.parametrize("mode,tile", [("faithful", None), ("fast", 256), ("fast", 128)])
def test_multi_sink_exact(mode, tile):
    # sinks spread over the sequence: gap 8 at keys 0-3, gap 30 at keys
    # 160-163, gap 12 at keys 700-703 (blocks 0, 2 and 10 of 64; 5 and 2 of 128)
    for d, bkv in ((64, 64), (128, 128)):
        inp = make_inputs(1, 4, 2, 777, d, fmt=FMT[mode], delta=8.0, seed=802 + d)
        inp = with_sink_cluster(with_sink_cluster(inp, 160, 4, 30.0), 700, 4, 12.0)
        dev = to_device(inp)
        for causal, order in itertools.product([False, True], ["forward", "reverse"]):
            label = f"diag multi-sink {mode} d={d} bkv={bkv} causal={causal} {order} tile={tile}"
            log(label)
            hist, bz, cnt = _run(dev, mode, 256.0, order, causal, bkv, tile=tile)
            _, _, o_cnt, o_hist, o_bz = oracle.block_diag(inp.q32, inp.k32, inp.v32, S=256.0,
                                                          order=order, block_kv=bkv,
                                                          causal=causal, nbins=32)
            assert np.array_equal(hist, o_hist), label
            assert np.array_equal(bz, o_bz), label
            assert np.array_equal(cnt.reshape(-1, 3), o_cnt), label


def test_sweep_head_exact():
    # one head group of the Delta sweep shape (N = 4096, d = 128, block 128)
    # at the collapse point, forward order, both device modes
    for mode in ("faithful", "fast"):
        inp = make_inputs(1, 2, 1, 4096, 128, fmt=FMT[mode], delta=9.0, seed=801)
        dev = to_device(inp)
        for order in ("forward", "reverse"):
            label = f"diag sweep {mode} {order}"
            log(label)
            hist, bz, _ = _run(dev, mode, 256.0, order, False, 128)
            _, _, _, o_hist, o_bz = oracle.block_diag(inp.q32, inp.k32, inp.v32, S=256.0,
                                                      order=order, block_kv=128, nbins=32)
            assert np.array_equal(hist, o_hist), label
            assert np.array_equal(bz, o_bz), label


def test_headline_workload_invariants():
    # full size: rows per block, per-block zeros = per-row counts regrouped,
    # reverse order with S = 256 zeroes nothing outside the sink's block
    w = WORKLOADS["causal_mha_b4_h32_n8192_d128_fast"]
    inp = make_inputs(w.B, w.Hq, w.Hkv, w.N, w.d, fmt=w.fmt, delta=w.deltas[0], seed=w.seed_base)
    dev = to_device(inp)
    log(f"diag {w.name}")
    hist, bz, cnt = _run(dev, w.mode, 256.0, "reverse", w.causal, w.block_kv)
    nblk = w.N // w.block_kv
    visits = np.array([w.N - j * w.block_kv for j in range(nblk)])
    assert np.array_equal(hist.astype(np.int64).sum(axis=3),
                          np.broadcast_to(visits, hist.shape[:3]))
    per_bh = cnt.reshape(w.B, w.Hq, w.N, 3).astype(np.int64).sum(axis=(2, 3))
    assert np.array_equal(bz.astype(np.int64).sum(axis=2), per_bh)
    assert bz[..., 1:].sum() == 0
    # the last block is every row's first: all of its rows sit in bin 0
    assert np.array_equal(hist[:, :, nblk - 1, 0], np.full((w.B, w.Hq), w.block_kv))
