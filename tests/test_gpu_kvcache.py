"""Queries against a KV cache (Nq < Nk) on the device against the oracle:
the prefill kernel (fast modes) and the faithful kernel with a query offset.
Same bar as the square problems: counts exact where claimed, outputs within
the mode's tolerance (plus the code-ambiguity bound in the fast modes), lse
within 1e-4."""
import itertools

import numpy as np
import pytest

from paper_2606_06521_amd.inputs import last_queries, make_inputs
from paper_2606_06521_amd.workloads import WORKLOADS
from tests.gpu_helpers import compare, log, run_gpu, to_device

pytestmark = pytest.mark.gpu

FMT = {"faithful": "f32", "nocast": "f32", "fast": "bf16_e4m3", "fp8qk": "e4m3"}


@pytest.mark.parametrize("mode", ["fast", "fp8qk", "faithful"])
@pytest.mark.parametrize("d,bkv", [(64, 64), (128, 128), (64, 128), (128, 64)])
def test_small(mode, d, bkv):
    full = make_inputs(2, 4, 2, 333, d, fmt=FMT[mode], delta=9.0, seed=900 + d + bkv)
    for nq in (1, 32, 77):
        inp = last_queries(full, nq)
        dev = to_device(inp)
        for (causal, order), (S, scale) in itertools.product(
                itertools.product([False, True], ["forward", "reverse"]),
                [(256.0, "static"), (448.0, "static"), (16.0, "dynamic")]):
            label = f"kv {mode} nq={nq} nk=333 d={d} bkv={bkv} causal={causal} {order} S={S} {scale}"
            log(label)
            gpu = run_gpu(dev, mode, S, order, causal, bkv, scale=scale)
            compare(inp, gpu, mode, S, order, causal, bkv, label=label, scale=scale)


@pytest.mark.parametrize("tile", [256, 128])
@pytest.mark.parametrize("mode", ["fast", "fp8qk"])
@pytest.mark.parametrize("bkv", [64, 128])
def test_long_chunks(mode, bkv, tile):
    # 256 queries with a block-aligned offset (Nk = 640) take the persistent
    # kernel (on either schedule); 200 queries at offset 133 (Nk = 333) the
    # prefill kernel (where the schedule flag has no effect)
    for nk, nq in ((640, 256), (333, 200)):
        full = make_inputs(1, 4, 2, nk, 128, fmt=FMT[mode], delta=9.0, seed=960 + nk + bkv)
        inp = last_queries(full, nq)
        dev = to_device(inp)
        for (causal, order), (S, scale) in itertools.product(
                itertools.product([False, True], ["forward", "reverse"]),
                [(256.0, "static"), (448.0, "static"), (16.0, "dynamic")]):
            label = f"kv {mode} nq={nq} nk={nk} bkv={bkv} causal={causal} {order} S={S} {scale} tile={tile}"
            log(label)
            gpu = run_gpu(dev, mode, S, order, causal, bkv, scale=scale, tile=tile)
            compare(inp, gpu, mode, S, order, causal, bkv, label=label, scale=scale)


@pytest.mark.parametrize("mode", ["fast", "fp8qk"])
@pytest.mark.parametrize("d,bkv,nk", [(128, 128, 2000), (64, 64, 4500), (128, 64, 1100), (64, 128, 3000)])
def test_split_over_workgroups(mode, d, bkv, nk):
    # Few 32-row tiles against many KV blocks: the prefill kernel splits each
    # tile's visit order over C = min(CUs / tiles, blocks / 8, 8) workgroups
    # (on 256 CUs: C = 2, 8, 2 and 3 for these caches), two launches and a
    # cross-workgroup merge.  Ragged caches, one row and a ragged 45-row chunk.
    full = make_inputs(1, 2, 1, nk, d, fmt=FMT[mode], delta=9.0, seed=970 + d + bkv + nk)
    for nq in (1, 45):
        inp = last_queries(full, nq)
        dev = to_device(inp)
        for (causal, order), (S, scale) in itertools.product(
                itertools.product([False, True], ["forward", "reverse"]),
                [(256.0, "static"), (448.0, "static"), (16.0, "dynamic")]):
            label = f"kv split {mode} nq={nq} nk={nk} d={d} bkv={bkv} causal={causal} {order} S={S} {scale}"
            log(label)
            gpu = run_gpu(dev, mode, S, order, causal, bkv, scale=scale)
            compare(inp, gpu, mode, S, order, causal, bkv, label=label, scale=scale)


@pytest.mark.parametrize("mode", ["fast", "fp8qk"])
def test_split_over_workgroups_gqa(mode):
    # GQA 8:1 with two batches: 2 * 8 * 2 = 32 tiles of 32 rows against 2500
    # keys (20 blocks of 128): C = min(256 / 32, 20 / 8, 8) = 2 workgroups per tile
    full = make_inputs(2, 8, 1, 2500, 128, fmt=FMT[mode], delta=9.0, seed=990)
    inp = last_queries(full, 50)
    dev = to_device(inp)
    for causal, order in itertools.product([False, True], ["forward", "reverse"]):
        label = f"kv split gqa {mode} causal={causal} {order}"
        log(label)
        gpu = run_gpu(dev, mode, 256.0, order, causal, 128)
        compare(inp, gpu, mode, 256.0, order, causal, 128, label=label)


def test_split_over_workgroups_descaled():
    # a split tile (C = 4) with per-tensor descales on E4M3 Q, K and V
    full = make_inputs(1, 2, 1, 4096, 128, fmt="e4m3", delta=8.0, seed=985)
    inp = last_queries(full, 32)
    dev = to_device(inp)
    ds = (0.75, 1.5, 2.0)
    for order in ("forward", "reverse"):
        label = f"kv split fp8qk descales {order}"
        log(label)
        gpu = run_gpu(dev, "fp8qk", 256.0, order, True, 128, descales=ds)
        compare(inp, gpu, "fp8qk", 256.0, order, True, 128, label=label, descales=ds)


def test_nocast_and_descales():
    full = make_inputs(1, 2, 1, 300, 128, fmt="f32", delta=7.0, seed=950)
    inp = last_queries(full, 40)
    dev = to_device(inp)
    for causal in (False, True):
        label = f"kv nocast causal={causal}"
        log(label)
        gpu = run_gpu(dev, "nocast", 256.0, "forward", causal, 64)
        compare(inp, gpu, "nocast", 256.0, "forward", causal, 64, label=label)
    full8 = make_inputs(1, 4, 2, 300, 128, fmt="e4m3", delta=7.0, seed=951)
    inp8 = last_queries(full8, 50)
    dev8 = to_device(inp8)
    ds = (0.75, 1.5, 2.0)
    label = "kv fp8qk descales"
    log(label)
    gpu = run_gpu(dev8, "fp8qk", 256.0, "reverse", True, 128, descales=ds)
    compare(inp8, gpu, "fp8qk", 256.0, "reverse", True, 128, label=label, descales=ds)


@pytest.mark.parametrize("order", ["forward", "reverse"])
def test_exp1_prefill_shape_all_rows(order):
    # Exp. 1's shape (q_len = 32 against N = 4096, 64 problems) in full
    w = WORKLOADS["prefill_q32_b64_n4096_d128_fast"]
    full = make_inputs(w.B, w.Hq, w.Hkv, w.N, w.d, fmt=w.fmt, delta=w.deltas[0], seed=w.seed_base)
    inp = last_queries(full, w.nq)
    dev = to_device(inp)
    for S in (256.0, 1.0):
        label = f"{w.name} S={S} {order}"
        log(label)
        gpu = run_gpu(dev, w.mode, S, order, w.causal, w.block_kv)
        res = compare(inp, gpu, w.mode, S, order, w.causal, w.block_kv, label=label)
        log(str(res))
        if order == "reverse" and S == 256.0:
            assert gpu[2][..., 2].sum() == 0, label


def test_square_call_through_kv_entry_is_unchanged():
    # Nq = Nk through the KV entry point runs the square kernels: bit-identical
    from paper_2606_06521_amd import attn_fp8 as A
    import torch
    inp = make_inputs(1, 4, 2, 300, 128, fmt="bf16_e4m3", delta=8.0, seed=952)
    q, k, v = to_device(inp)
    o1, l1 = A.fwd(q, k, v, S=256.0, order="reverse", causal=True, block_kv=128, mode="fast")
    o2 = torch.empty_like(o1)
    l2 = torch.empty_like(l1)
    st = A.attn_fp8_fwd_kv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o2.data_ptr(), l2.data_ptr(),
                           1, 4, 2, 300, 300, 128, 1, 128, 1, 256.0, 1, 1.0, 1.0, 1.0, None, 0,
                           torch.cuda.current_stream().cuda_stream)
    torch.cuda.synchronize()
    assert st == 0
    assert torch.equal(o1, o2) and torch.equal(l1, l2)


def test_split_workspace_is_the_callers():
    # A split shape through the C ABI: with the caller's workspace (split
    # launches), without one (NULL: the tiles run unsplit) and with one that
    # is too small (rejected before any launch).  The workspace starts filled
    # with NaN bytes: nothing is read before the call writes it.  Both runs
    # equal the oracle, codes and counts included.
    import torch
    from paper_2606_06521_amd import attn_fp8 as A
    inp = last_queries(make_inputs(2, 4, 2, 3000, 128, fmt="bf16_e4m3", delta=8.0, seed=995), 20)
    q, k, v = to_device(inp)
    B, Hq, Hkv, Nq, Nk, d = 2, 4, 2, 20, 3000, 128
    st, nbytes = A.attn_fp8_kv_workspace_bytes(B, Hq, Hkv, Nq, Nk, d, 1, 128, A.ATTN_MODE_FAST)
    assert st == 0 and nbytes > 0
    # square problems and the faithful mode never split
    assert A.attn_fp8_kv_workspace_bytes(B, Hq, Hkv, Nk, Nk, d, 1, 128, A.ATTN_MODE_FAST) == (0, 0)
    assert A.attn_fp8_kv_workspace_bytes(B, Hq, Hkv, Nq, Nk, d, 1, 128, A.ATTN_MODE_FAITHFUL) == (0, 0)
    ws = torch.full((nbytes,), 0xFF, dtype=torch.uint8, device="cuda")
    sptr = torch.cuda.current_stream().cuda_stream
    for label, wptr, wbytes in (("with workspace", ws.data_ptr(), nbytes), ("no workspace", None, 0)):
        o = torch.empty((B, Hq, Nq, d), dtype=torch.float32, device="cuda")
        l = torch.empty((B, Hq, Nq), dtype=torch.float32, device="cuda")
        c = torch.empty((B, Hq, Nq, 3), dtype=torch.int32, device="cuda")
        st = A.attn_fp8_fwd_kv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), l.data_ptr(),
                               B, Hq, Hkv, Nq, Nk, d, 1, 128, 1, 256.0, 1, 1.0, 1.0, 1.0, wptr,
                               wbytes, sptr)
        assert st == 0, label
        st = A.attn_fp8_p_underflow_count_kv(q.data_ptr(), k.data_ptr(), v.data_ptr(), B, Hq, Hkv,
                                             Nq, Nk, d, 1, 128, 1, 256.0, 1, 4, 1.0, 1.0, 1.0,
                                             c.data_ptr(), None, None, wptr, wbytes, sptr)
        assert st == 0, label
        torch.cuda.synchronize()
        log(f"kv split: {label}")
        compare(inp, (o.cpu().numpy(), l.cpu().numpy(), c.cpu().numpy().view(np.uint32)), "fast",
                256.0, "reverse", True, 128, label=label)
    st = A.attn_fp8_fwd_kv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), None, B, Hq,
                           Hkv, Nq, Nk, d, 1, 128, 1, 256.0, 1, 1.0, 1.0, 1.0, ws.data_ptr(),
                           nbytes - 1, sptr)
    assert st == A.ATTN_ERR_INVALID_ARG
    st = A.attn_fp8_fwd_kv(q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), None, B, Hq,
                           Hkv, Nq, Nk, d, 1, 128, 1, 256.0, 1, 1.0, 1.0, 1.0,
                           ws.data_ptr() + 16, nbytes - 16, sptr)
    assert st == A.ATTN_ERR_INVALID_ARG    # a workspace must be 256-byte aligned


def test_split_call_in_a_captured_graph():
    # A split KV-cache call captured in a HIP graph (its workspace comes from
    # the graph's own pool) and replayed several times, with eager work and a
    # synchronisation between replays; every replay equals the eager result
    # bit for bit, and that result equals the oracle.
    import torch
    from paper_2606_06521_amd import attn_fp8 as A
    inp = last_queries(make_inputs(1, 8, 2, 2600, 128, fmt="bf16_e4m3", delta=8.0, seed=981), 24)
    q, k, v = to_device(inp)
    o_eager, l_eager = A.fwd(q, k, v, S=256.0, order="reverse", causal=True, block_kv=128,
                             mode="fast")
    torch.cuda.synchronize()
    compare(inp, (o_eager.cpu().numpy(), l_eager.cpu().numpy(), None), "fast", 256.0, "reverse",
            True, 128, label="kv split eager")
    s = torch.cuda.Stream()
    s.wait_stream(torch.cuda.current_stream())
    with torch.cuda.stream(s):           # warm-up on the capture stream
        A.fwd(q, k, v, S=256.0, order="reverse", causal=True, block_kv=128, mode="fast")
    torch.cuda.current_stream().wait_stream(s)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        o_g, l_g = A.fwd(q, k, v, S=256.0, order="reverse", causal=True, block_kv=128, mode="fast")
    for i in range(4):
        o_g.fill_(float("nan"))
        l_g.fill_(float("nan"))
        g.replay()
        other, _ = A.fwd(q, k, v, S=1.0, order="forward", causal=True, block_kv=128, mode="fast")
        torch.cuda.synchronize()
        log(f"kv split graph replay {i}")
        assert torch.equal(o_g, o_eager) and torch.equal(l_g, l_eager), i
        del other


def test_split_workspace_two_host_threads():
    # Two host threads, each on its own stream, enqueue different split
    # problems over and over (ctypes releases the GIL during the calls, so
    # the library is entered concurrently; each call has its own workspace);
    # every thread's last result equals the oracle.
    import threading
    import torch
    from paper_2606_06521_amd import attn_fp8 as A
    probs = [last_queries(make_inputs(1, 2, 1, 2500, 128, fmt="bf16_e4m3", delta=8.0, seed=997), 24),
             last_queries(make_inputs(2, 4, 2, 3000, 128, fmt="bf16_e4m3", delta=9.0, seed=998), 33)]
    devs = [to_device(p) for p in probs]
    results = [None, None]
    errors = []

    def worker(i):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                q, k, v = devs[i]
                for _ in range(20):
                    o, l = A.fwd(q, k, v, S=256.0, order="reverse", causal=True, block_kv=128, mode="fast")
                s.synchronize()
                results[i] = (o.cpu().numpy(), l.cpu().numpy(), None)
        except Exception as e:   # surfaced below
            errors.append(e)

    torch.cuda.synchronize()
    threads = [threading.Thread(target=worker, args=(i,)) for i in range(2)]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for i in range(2):
        label = f"kv split two threads, problem {i}"
        log(label)
        compare(probs[i], results[i], "fast", 256.0, "reverse", True, 128, label=label)


def test_workload_prefill_q256_full_size_both_schedules():
    """The KV-cache prefill workload at full size (4 x 32 query heads, 8 KV
    heads, the last 256 of 32768 positions, d = 128): 128 tiles of 256 rows
    would leave half of the CUs idle, so the library picks the 128-row
    schedule.  Both schedules are run.  Their E4M3 codes are the same by
    construction, so the counts must agree on every row; the outputs only in
    FP32 rounding.  Sampled rows are checked against the oracle."""
    w = WORKLOADS["prefill_q256_b4_h32kv8_n32768_d128_fast"]
    full = make_inputs(w.B, w.Hq, w.Hkv, w.N, w.d, fmt=w.fmt, delta=w.deltas[0], seed=w.seed_base)
    inp = last_queries(full, w.nq)
    del full
    dev = to_device(inp)
    nq = w.nq
    rng = np.random.default_rng(5)
    heads = np.array([0, 45, 127])                      # flat (batch, head) ids
    rows = np.concatenate([bh * nq + np.concatenate([np.arange(0, 8), rng.integers(0, nq, 16),
                                                     np.arange(nq - 8, nq)]) for bh in heads])
    rows = np.unique(rows)
    res = {}
    for tile in (None, 128, 256):
        label = f"{w.name} S=256 reverse tile={tile} (rows {rows.size})"
        log(label)
        gpu = run_gpu(dev, w.mode, 256.0, "reverse", w.causal, w.block_kv, tile=tile)
        log(str(compare(inp, gpu, w.mode, 256.0, "reverse", w.causal, w.block_kv, rows=rows,
                        label=label)))
        res[tile] = gpu
    for tile in (None, 256):
        assert np.array_equal(res[tile][2], res[128][2]), tile             # counts, every row
        assert np.allclose(res[tile][0], res[128][0], rtol=1e-5, atol=1e-6), tile
        assert np.allclose(res[tile][1], res[128][1], rtol=0, atol=1e-5), tile
    assert np.array_equal(res[None][0], res[128][0])                       # the automatic choice
