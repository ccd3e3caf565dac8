"""The allocation-free KV-cache entry point (attn_fp8_fwd_kv_noalloc) against
attn_fp8_fwd_kv with the caller's workspace, through the C ABI.

Two calls in a row on split shapes, the second smaller than the first, so it
runs over scratch the first call left behind: each equals the workspace entry
point's result bit for bit (same kernels, same split, same summation order),
and the first also equals the oracle.  A shape that does not split and a
square problem take the same path with no scratch at all.
"""
import numpy as np
import pytest
import torch

from paper_2606_06521_amd.inputs import last_queries, make_inputs
from tests.gpu_helpers import compare, log, to_device

pytestmark = pytest.mark.gpu


def _pair(A, inp, B, Hq, Hkv, Nq, Nk, d=128, order=1, S=256.0, mode=1):
    q, k, v = to_device(inp)
    st, nbytes = A.attn_fp8_kv_workspace_bytes(B, Hq, Hkv, Nq, Nk, d, 1, 128, mode)
    assert st == 0
    ws = torch.empty(max(nbytes, 1), dtype=torch.uint8, device="cuda")
    sptr = torch.cuda.current_stream().cuda_stream
    outs = []
    for noalloc in (False, True):
        o = torch.full((B, Hq, Nq, d), float("nan"), dtype=torch.float32, device="cuda")
        l = torch.full((B, Hq, Nq), float("nan"), dtype=torch.float32, device="cuda")
        args = (q.data_ptr(), k.data_ptr(), v.data_ptr(), o.data_ptr(), l.data_ptr(), B, Hq, Hkv,
                Nq, Nk, d, 1, 128, order, S, mode, 1.0, 1.0, 1.0)
        if noalloc:
            st = A.attn_fp8_fwd_kv_noalloc(*args, sptr)
        else:
            st = A.attn_fp8_fwd_kv(*args, ws.data_ptr() if nbytes else None, nbytes, sptr)
        assert st == 0, (noalloc, A.attn_fp8_strerror(st))
        outs.append((o, l))
    torch.cuda.synchronize()
    return nbytes, outs


def test_noalloc_matches_workspace_entry_point_twice():
    from paper_2606_06521_amd import attn_fp8 as A
    shapes = [(2, 8, 2, 40, 3000, 901), (1, 4, 1, 20, 2000, 902)]   # the second is smaller
    for i, (B, Hq, Hkv, Nq, Nk, seed) in enumerate(shapes):
        inp = last_queries(make_inputs(B, Hq, Hkv, Nk, 128, fmt="bf16_e4m3", delta=8.0, seed=seed), Nq)
        log(f"noalloc call {i}: B={B} Hq={Hq} Hkv={Hkv} Nq={Nq} Nk={Nk}")
        nbytes, ((o_ws, l_ws), (o_na, l_na)) = _pair(A, inp, B, Hq, Hkv, Nq, Nk)
        assert nbytes > 0, "the shape must split to use the scratch"
        assert torch.equal(o_ws, o_na) and torch.equal(l_ws, l_na), i
        if i == 0:
            compare(inp, (o_na.cpu().numpy(), l_na.cpu().numpy(), None), "fast", 256.0, "reverse",
                    True, 128, label="noalloc vs oracle")


def test_noalloc_without_split_and_square():
    from paper_2606_06521_amd import attn_fp8 as A
    # enough tiles to fill the GPU (no split), and a square problem
    for B, Hq, Hkv, Nq, Nk, seed in [(4, 64, 8, 32, 700, 903), (1, 4, 2, 300, 300, 904)]:
        inp = last_queries(make_inputs(B, Hq, Hkv, Nk, 128, fmt="bf16_e4m3", delta=8.0, seed=seed), Nq)
        log(f"noalloc no split: B={B} Hq={Hq} Hkv={Hkv} Nq={Nq} Nk={Nk}")
        nbytes, ((o_ws, l_ws), (o_na, l_na)) = _pair(A, inp, B, Hq, Hkv, Nq, Nk)
        assert nbytes == 0
        assert torch.equal(o_ws, o_na) and torch.equal(l_ws, l_na)
