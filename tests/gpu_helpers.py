"""Helpers shared by the GPU tests: move seeded inputs to the device, run the
library through its binding, run the oracle on the same values, compare."""
from __future__ import annotations

import sys

import numpy as np
import torch

import oracle

TOL_OUT = {"faithful": 2e-3, "nocast": 2e-3, "fast": 2e-2, "fp8qk": 2e-2}
TOL_LSE = 1e-4
# The fast kernels take exp2 from v_exp_f32 (within 2 ulp of exact, see
# test_gpu_probes), the oracle from a correctly rounded double.  With the
# roundings of P and of P*S on both sides a P*S value can differ by up to
# 3.5 ulp, so where it lies within 6 ulp of an E4M3 rounding midpoint both
# codes are valid; the oracle's amb bounds what those choices move.
AMB_WINDOW = 6.0 * 2.0 ** -23


def log(msg: str) -> None:
    print(msg, flush=True)
    sys.stdout.flush()


def to_device(inp):
    if inp.fmt == "f32":
        q = torch.from_numpy(inp.q_dev).cuda()
        k = torch.from_numpy(inp.k_dev).cuda()
        v = torch.from_numpy(inp.v_dev).cuda()
    elif inp.fmt == "e4m3":
        q = torch.from_numpy(inp.q_dev).cuda().view(torch.float8_e4m3fn)
        k = torch.from_numpy(inp.k_dev).cuda().view(torch.float8_e4m3fn)
        v = torch.from_numpy(inp.v_dev).cuda().view(torch.float8_e4m3fn)
    else:
        q = torch.from_numpy(inp.q_dev.view(np.int16)).cuda().view(torch.bfloat16)
        k = torch.from_numpy(inp.k_dev.view(np.int16)).cuda().view(torch.bfloat16)
        v = torch.from_numpy(inp.v_dev).cuda().view(torch.float8_e4m3fn)
    return q, k, v


def run_gpu(dev, mode, S, order, causal, block_kv, n_sink=4, counts=True, scale="static",
            descales=(1.0, 1.0, 1.0), tile=None):
    from paper_2606_06521_amd import attn_fp8 as A
    q, k, v = dev
    out, lse = A.fwd(q, k, v, S=S, order=order, causal=causal, block_kv=block_kv, mode=mode,
                     scale=scale, descales=descales, tile=tile)
    cnt = None
    if counts:
        cnt = A.p_underflow_count(q, k, v, S=S, order=order, causal=causal, block_kv=block_kv,
                                  mode=mode, n_sink=n_sink, scale=scale, descales=descales,
                                  tile=tile)
    torch.cuda.synchronize()
    res = (out.cpu().numpy(), lse.cpu().numpy(), None if cnt is None else cnt.cpu().numpy().view(np.uint32))
    return res


def counts_are_exact(mode, S) -> bool:
    """Count parity is claimed wherever both sides take the zero-code decision
    on identical P values: faithful mode (exp2 in FP64 on both sides, any S),
    and fast mode for S = 2^k, where the decision is the integer threshold
    x <= -(10 + k) and the hardware exp2 is exact at integers and monotone
    around them (see test_gpu_probes).  The dynamic scale keeps that property:
    block j's threshold is the integer x <= -(10 + kj)."""
    if mode == "faithful":
        return True
    if mode in ("fast", "fp8qk"):
        return float(np.log2(S)).is_integer()
    return False


def compare(inp, gpu, mode, S, order, causal, block_kv, rows=None, n_sink=4, label="",
            scale="static", descales=(1.0, 1.0, 1.0)):
    """Oracle on `rows` (flat ids, None = all); asserts counts bit-exact (where
    claimed) and out / lse within tolerance.  Returns the measured differences."""
    out_g, lse_g, cnt_g = gpu
    d = inp.d
    hw_exp2 = mode in ("fast", "fp8qk")
    o_out, o_lse, o_cnt, amb = oracle.attn(inp.q32, inp.k32, inp.v32, S=S, order=order,
                                           block_kv=block_kv, causal=causal,
                                           cast=(mode != "nocast"), n_sink=n_sink, rows=rows,
                                           scale=scale, descales=descales,
                                           bound_rel=AMB_WINDOW if hw_exp2 else 0.0)
    g_out = out_g.reshape(-1, d)
    g_lse = lse_g.reshape(-1)
    if rows is not None:
        g_out, g_lse = g_out[rows], g_lse[rows]
    diff = np.abs(g_out.astype(np.float64) - o_out)
    err = float(diff.max()) if g_out.size else 0.0
    lerr = float(np.abs(g_lse - o_lse).max()) if g_lse.size else 0.0
    # elements past the plain tolerance that the code-ambiguity bound covers
    over = diff > TOL_OUT[mode]
    res = {"max_abs_out": err, "max_abs_lse": lerr, "n_ambiguous_over_tol": int(over.sum())}
    assert np.all(np.isfinite(g_out)), label
    bad = diff > TOL_OUT[mode] + amb
    assert not bad.any(), (label, err, float((diff - amb)[bad].max()) if bad.any() else 0.0)
    if over.any():
        log(f"  {label}: {int(over.sum())} outputs past {TOL_OUT[mode]} (max {err:.4g}), "
            f"all within the code-ambiguity bound")
    assert lerr <= TOL_LSE, (label, lerr)
    if cnt_g is not None and counts_are_exact(mode, S):
        g_cnt = cnt_g.reshape(-1, 3)
        if rows is not None:
            g_cnt = g_cnt[rows]
        bad = np.nonzero(np.any(g_cnt != o_cnt, axis=1))[0]
        assert bad.size == 0, (label, [(int(i), g_cnt[i].tolist(), o_cnt[i].tolist()) for i in bad[:5]])
        res["counts"] = o_cnt.sum(0).tolist()
    return res
