"""Per-tensor descales in the oracle (Sec. 6.1: the QKV quantization carries
its own qscale/kscale/vscale, separate from the P-scale S) and the E4M3 Q/K
input recipe, pinned against exact identities and an independent FP64
attention written here in numpy."""
import numpy as np
import pytest

import oracle
from paper_2606_06521_amd.inputs import make_inputs


def _inp(fmt="f32", N=200, d=64, seed=31, delta=8.0):
    return make_inputs(1, 2, 1, N, d, fmt=fmt, delta=delta, seed=seed)


def test_unit_descales_change_nothing():
    inp = _inp()
    a = oracle.attn(inp.q32, inp.k32, inp.v32, S=256.0, order="forward", block_kv=64)
    b = oracle.attn(inp.q32, inp.k32, inp.v32, S=256.0, order="forward", block_kv=64,
                    descales=(1.0, 1.0, 1.0))
    for x, y in zip(a, b):
        assert np.array_equal(x, y)


@pytest.mark.parametrize("which", [0, 1, 2])
@pytest.mark.parametrize("order", ["forward", "reverse"])
def test_power_of_two_descale_equals_prescaled_tensor(which, order):
    # storing x * 2 with descale 1/2 is the same problem: scores, every P, every
    # zero code and every output agree bit for bit (powers of two commute with
    # every rounding on the path)
    inp = _inp()
    t = [inp.q32, inp.k32, inp.v32]
    ref = oracle.attn(*t, S=256.0, order=order, block_kv=64, causal=True)
    t2 = list(t)
    t2[which] = (t[which] * np.float32(2.0)).astype(np.float32)
    ds = [1.0, 1.0, 1.0]
    ds[which] = 0.5
    got = oracle.attn(*t2, S=256.0, order=order, block_kv=64, causal=True, descales=tuple(ds))
    for x, y in zip(ref, got):
        assert np.array_equal(x, y)


def _numpy_attention(q, k, v, causal):
    """Plain softmax attention in FP64 over [N, d] arrays (no blocks, no cast)."""
    z = (q @ k.T) / np.sqrt(q.shape[1])
    if causal:
        z = np.where(np.tril(np.ones(z.shape, bool)), z, -np.inf)
    z = z - z.max(axis=1, keepdims=True)
    p = np.exp(z)
    return (p @ v) / p.sum(axis=1, keepdims=True)


@pytest.mark.parametrize("causal", [False, True])
def test_descaled_without_cast_matches_fp64_attention(causal):
    inp = _inp(N=150, seed=32)
    qd, kd, vd = 0.75, 1.5, 3.0
    out, _, _ = oracle.attn(inp.q32, inp.k32, inp.v32, S=16.0, order="reverse", block_kv=64,
                            causal=causal, cast=False, descales=(qd, kd, vd))
    ref, _ = oracle.ref_fp64(inp.q32, inp.k32, inp.v32, causal=causal, descales=(qd, kd, vd))
    for h in range(2):
        want = _numpy_attention(inp.q32[0, h].astype(np.float64) * qd,
                                inp.k32[0, 0].astype(np.float64) * kd,
                                inp.v32[0, 0].astype(np.float64) * vd, causal)
        rows = slice(h * inp.N, (h + 1) * inp.N)
        assert np.abs(ref[rows] - want).max() < 1e-12
        assert np.abs(out[rows] - want).max() < 1e-5 * vd


def test_e4m3_inputs_are_e4m3_values_with_exact_dots():
    inp = _inp(fmt="e4m3", N=257, d=128, seed=33, delta=9.0)
    q = inp.q32[0, 0].astype(np.float64)
    k = inp.k32[0, 0].astype(np.float64)
    # stored bytes decode to exactly the values the oracle sees
    assert np.array_equal(oracle.e4m3_decode(inp.q_dev[0, 0]), inp.q32[0, 0])
    assert np.array_equal(oracle.e4m3_decode(inp.k_dev[0, 0]), inp.k32[0, 0])
    assert np.array_equal(oracle.e4m3_decode(inp.v_dev[0, 0]), inp.v32[0, 0])
    # every dot is a multiple of 2^-8 below 2^11: FP32 sums in any order are exact
    D = q @ k.T
    assert np.abs(D).max() < 2 ** 11 and np.all(np.mod(D * 256, 1) == 0)
    # and so are the FP8 matrix cores' group sums: in each group of eight
    # consecutive channels every product is a multiple of 2^(e - 13), e the
    # exponent of the group's largest product (the alignment they keep)
    prod = q[:, None, :] * k[None, :, :]
    g = np.abs(prod).reshape(prod.shape[0], prod.shape[1], -1, 8).max(axis=3)
    e = np.floor(np.log2(np.where(g > 0, g, 1.0)))
    unit = np.repeat(np.exp2(e - 13), 8, axis=2)
    assert np.all(np.mod(prod / unit, 1) == 0)
    rng = np.random.default_rng(0)
    acc = np.zeros(D.shape, np.float32)
    for i in rng.permutation(128):
        acc += (q[:, i:i + 1] * k[:, i:i + 1].T).astype(np.float32)
    assert np.array_equal(acc.astype(np.float64), D)
    # the sink offset: the first n_sink keys sit Delta_eff above the rest on average
    z = D / np.sqrt(128)
    assert abs(inp.delta_eff - 9.0) < 0.2
    assert abs((z[:, :4].mean() - z[:, 4:].mean()) - inp.delta_eff) < 0.3
