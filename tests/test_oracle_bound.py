"""The oracle's code-ambiguity bound (oracle_attn_bound).

An implementation whose exp2 is a few ulps off the correctly rounded one (the
GPU's v_exp_f32, two ulps at most by the probe test) can put a P*S value that
sits next to an E4M3 rounding midpoint on the neighbouring code.  The bound
amb says how far that can move each output.  It is pinned here by planting
such an error in the oracle itself (a fixed +-jitter on every exp2 of a P
value) and checking that the outputs move by no more than amb, that they do
move (codes really flip), and that the check fails without the bound.
"""
import numpy as np
import pytest

import oracle
from paper_2606_06521_amd.inputs import make_inputs

ULP = 2.0 ** -23
# A planted exp2 error of J moves P*S by at most J + 2 ulp once the roundings
# of P and of P*S on both sides are counted, so a window of J + 2.5 ulp must
# hold every move.  1.5 ulp is the size of the GPU's exp2 error; 64 ulp makes
# flips common enough to show in every case.
JITTERS = (1.5 * ULP, 64 * ULP)
WINDOW = 4.0 * ULP


def _inputs(fmt, seed, N=333, d=64):
    return make_inputs(2, 4, 2, N, d, fmt=fmt, delta=8.0, seed=seed)


CASES = [("e4m3", 448.0, "static", "forward", False), ("e4m3", 3.0, "static", "reverse", True),
         ("bf16_e4m3", 256.0, "static", "reverse", False), ("bf16_e4m3", 448.0, "static", "forward", True),
         ("e4m3", 16.0, "dynamic", "forward", False), ("bf16_e4m3", 256.0, "dynamic", "reverse", True)]


@pytest.mark.parametrize("jitter", JITTERS)
@pytest.mark.parametrize("fmt,S,scale,order,causal", CASES)
def test_planted_exp2_error_stays_within_bound(fmt, S, scale, order, causal, jitter):
    inp = _inputs(fmt, 900 + int(S))
    args = dict(S=S, order=order, block_kv=64, causal=causal, scale=scale)
    out, lse, cnt, amb = oracle.attn(inp.q32, inp.k32, inp.v32, bound_rel=jitter + 2.5 * ULP,
                                     **args)
    for sign in (1.0, -1.0):
        o2, l2, c2 = oracle.attn(inp.q32, inp.k32, inp.v32, jitter_rel=sign * jitter, **args)
        diff = np.abs(o2.astype(np.float64) - out)
        # l moves by the jitter itself (1e-7 relative); everything above that
        # comes from flipped codes and must sit under amb
        assert np.all(diff <= amb + 1e-5), float((diff - amb).max())
        assert np.abs(l2 - lse).max() < 1e-5
    # flips that matter are rare (test_check_fails_without_the_bound shows
    # one); some of these cases have no P*S near a midpoint at all
    assert np.all(amb >= 0)


def test_bound_is_zero_without_window_or_cast():
    inp = _inputs("bf16_e4m3", 7)
    out, _, _, amb = oracle.attn(inp.q32, inp.k32, inp.v32, S=448.0, order="forward",
                                 block_kv=64, bound_rel=0.0)
    assert np.all(amb == 0)
    ref = oracle.attn(inp.q32, inp.k32, inp.v32, S=448.0, order="forward", block_kv=64)
    assert np.array_equal(out, ref[0])
    _, _, _, amb = oracle.attn(inp.q32, inp.k32, inp.v32, S=448.0, order="forward",
                               block_kv=64, cast=False, bound_rel=WINDOW)
    assert np.all(amb == 0)


def test_check_fails_without_the_bound():
    # the plant flips codes that move outputs far above the FP32 noise floor:
    # judged with a window that misses it, the same check fails
    inp = _inputs("e4m3", 1300)
    args = dict(S=448.0, order="forward", block_kv=64)
    J = JITTERS[1]
    out, _, _, amb = oracle.attn(inp.q32, inp.k32, inp.v32, bound_rel=J + 2.5 * ULP, **args)
    _, _, _, amb_small = oracle.attn(inp.q32, inp.k32, inp.v32, bound_rel=WINDOW, **args)
    o2, _, _ = oracle.attn(inp.q32, inp.k32, inp.v32, jitter_rel=J, **args)
    diff = np.abs(o2.astype(np.float64) - out)
    assert diff.max() > 1e-3
    assert np.all(diff <= amb + 1e-5)
    assert not np.all(diff <= amb_small + 1e-5)


def test_bound_closed_form_single_key():
    # one key per row (N = 1): P = 1 exactly, y = S; the window spans a
    # midpoint only when S itself is one, and then amb = step * |v| / S
    q = np.zeros((1, 1, 1, 4), np.float32)
    k = np.zeros((1, 1, 1, 4), np.float32)
    v = np.array([[[[1.0, -2.0, 0.5, 0.0]]]], np.float32)
    for S, step in ((3.0, 0.0), (17.0, 2.0), (272.0, 32.0)):
        # 17 lies halfway between 16 and 18, 272 halfway between 256 and 288
        out, _, _, amb = oracle.attn(q, k, v, S=S, order="forward", block_kv=1, bound_rel=WINDOW)
        assert np.allclose(amb[0], step * np.abs(v[0, 0, 0]) / S, rtol=1e-6, atol=0)
