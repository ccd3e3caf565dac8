"""Pins for the oracle's Algorithm 1 (FP8 online-softmax attention).

Each check compares the oracle with something it does not share code with:
a textbook FP64 softmax attention written here in numpy, a per-key closed
form of the underflow decision, torch's E4M3 conversion in the single-block
case, IEEE facts (Prop. 2), and the paper's fixed points (Theorem 2 and the
P-collapse corollary).
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import analysis
from paper_2606_06521_amd.inputs import make_inputs, sample_rows, with_delta

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def numpy_attention_fp64(q, k, v, causal):
    """Textbook softmax(q k^T / sqrt(d)) v in float64 with GQA head sharing."""
    B, Hq, N, d = q.shape
    Hkv = k.shape[1]
    g = Hq // Hkv
    kk = np.repeat(k.astype(np.float64), g, axis=1)
    vv = np.repeat(v.astype(np.float64), g, axis=1)
    z = np.einsum("bhnd,bhtd->bhnt", q.astype(np.float64), kk) / math.sqrt(d)
    if causal:
        z = np.where(np.tril(np.ones((N, N), dtype=bool)), z, -np.inf)
    m = z.max(-1, keepdims=True)
    p = np.exp(z - m)
    ell = p.sum(-1, keepdims=True)
    out = np.einsum("bhnt,bhtd->bhnd", p, vv) / ell
    lse = (m + np.log(ell))[..., 0]
    return out, lse


def c_const(d):
    return np.float32(1.4426950408889634 / math.sqrt(d))


def direct_underflow_counts(inp, causal, Bc, order, k_pow, n_sink):
    """Per-key closed form of the cast-to-zero decision, independent of the
    oracle's loop: key t (block j) is cast to zero iff
    fl32(D_t c - fl32(m_j c)) <= -(10 + k) for S = 2^k, where m_j is the maximum
    raw score over the valid keys of every block visited up to and including j
    (forward: blocks 0..j; reverse: blocks j..last).  Uses the monotonicity of
    exp2 and its exactness at integers."""
    q, kmat = inp.q32, inp.k32
    B, Hq, N, d = q.shape
    g = Hq // kmat.shape[1]
    c = c_const(d)
    out = np.zeros((B, Hq, N, 3), dtype=np.uint32)
    for b in range(B):
        for h in range(Hq):
            D = (q[b, h].astype(np.float64) @ kmat[b, h // g].astype(np.float64).T).astype(np.float32)
            for r in range(N):
                L = r + 1 if causal else N
                nblk = (L + Bc - 1) // Bc
                row = D[r, :L]
                bmax = np.array([row[j * Bc:(j + 1) * Bc].max() for j in range(nblk)], dtype=np.float32)
                if order == "forward":
                    run = np.maximum.accumulate(bmax)
                else:
                    run = np.maximum.accumulate(bmax[::-1])[::-1]
                m_key = np.repeat(run, Bc)[:L]
                mc = (m_key * c).astype(np.float32)
                x = (row.astype(np.float64) * np.float64(c) - mc.astype(np.float64)).astype(np.float32)
                zero = x <= -(10 + k_pow)
                t = np.arange(L)
                out[b, h, r, 0] = np.count_nonzero(zero & (t < n_sink))
                out[b, h, r, 1] = np.count_nonzero(zero & (t >= n_sink) & (t < Bc))
                out[b, h, r, 2] = np.count_nonzero(zero & (t >= Bc))
    return out


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("order", ["forward", "reverse"])
def test_cast_off_matches_fp64(causal, order):
    """Fixed point (e): with the cast disabled Algorithm 1 is exact softmax
    attention up to FP32 rounding, for any S, any order, GQA and ragged N."""
    inp = make_inputs(1, 4, 2, 200, 16, fmt="f32", delta=6.0, seed=11)
    want, want_lse = numpy_attention_fp64(inp.q32, inp.k32, inp.v32, causal)
    for S in (1.0, 3.0, 256.0, 448.0):
        out, lse, _ = oracle.attn(inp.q32, inp.k32, inp.v32, S=S, order=order, block_kv=64,
                                  causal=causal, cast=False)
        err = np.abs(out.reshape(want.shape) - want).max()
        assert err <= 1e-5, (S, err)
        assert np.abs(lse.reshape(want_lse.shape) - want_lse).max() <= 1e-5
    # the C FP64 reference agrees with the numpy one
    ref, ref_lse = oracle.ref_fp64(inp.q32, inp.k32, inp.v32, causal=causal)
    assert np.abs(ref.reshape(want.shape) - want).max() <= 1e-12
    assert np.abs(ref_lse.reshape(want_lse.shape) - want_lse).max() <= 1e-12


def test_cast_off_d64_n1024_both_orders():
    inp = make_inputs(1, 1, 1, 1024, 64, fmt="f32", delta=8.0, seed=12)
    ref, _ = oracle.ref_fp64(inp.q32, inp.k32, inp.v32)
    outs = {}
    for order in ("forward", "reverse"):
        out, _, _ = oracle.attn(inp.q32, inp.k32, inp.v32, S=256.0, order=order, block_kv=64, cast=False)
        assert np.abs(out - ref).max() <= 1e-5
        outs[order] = out
    assert np.abs(outs["forward"] - outs["reverse"]).max() <= 2e-6


def test_power_of_two_scale_is_bit_exact_end_to_end():
    """Fixed point (a), Prop. 2: with the cast off, S = 2^k gives results
    bit-identical to S = 1 (scaling by 2^k commutes with every rounding); a
    non-power-of-two S does not."""
    inp = make_inputs(1, 2, 2, 300, 32, fmt="f32", delta=7.0, seed=13)
    base, base_lse, _ = oracle.attn(inp.q32, inp.k32, inp.v32, S=1.0, order="forward", block_kv=64, cast=False)
    for k in range(1, 9):
        out, lse, _ = oracle.attn(inp.q32, inp.k32, inp.v32, S=2.0 ** k, order="forward", block_kv=64, cast=False)
        assert np.array_equal(out.view(np.uint32), base.view(np.uint32)), k
        assert np.array_equal(lse.view(np.uint32), base_lse.view(np.uint32))
    out448, _, _ = oracle.attn(inp.q32, inp.k32, inp.v32, S=448.0, order="forward", block_kv=64, cast=False)
    assert not np.array_equal(out448.view(np.uint32), base.view(np.uint32))
    assert np.abs(out448 - base).max() < 1e-5


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("order", ["forward", "reverse"])
@pytest.mark.parametrize("k_pow", [0, 4, 8])
def test_counts_match_per_key_closed_form(causal, order, k_pow):
    """Prop. 1 per key: the oracle's zero-code counts equal the direct count of
    x_t <= -(10 + k) under the running maximum each block sees."""
    inp = make_inputs(1, 2, 1, 300, 32, fmt="f32", delta=9.0, seed=14 + k_pow)
    Bc = 64
    _, _, counts = oracle.attn(inp.q32, inp.k32, inp.v32, S=2.0 ** k_pow, order=order, block_kv=Bc,
                               causal=causal, cast=True, n_sink=4)
    want = direct_underflow_counts(inp, causal, Bc, order, k_pow, 4)
    assert np.array_equal(counts.reshape(want.shape), want)
    if k_pow == 0 and not causal:
        assert want.sum() > 0


def test_single_block_reduces_to_direct_formula():
    """With one KV block there is no rescaling: out = sum(E4M3(P*S) v)/(S l)
    with P = exp2(fma(D, c, -m c)); the cast here is torch's float8_e4m3fn."""
    inp = make_inputs(1, 1, 1, 64, 64, fmt="f32", delta=7.0, seed=15)
    q, k, v = inp.q32[0, 0], inp.k32[0, 0], inp.v32[0, 0]
    c = c_const(64)
    for S in (1.0, 256.0, 448.0):
        out, _, _ = oracle.attn(inp.q32, inp.k32, inp.v32, S=S, order="forward", block_kv=64)
        D = (q.astype(np.float64) @ k.astype(np.float64).T).astype(np.float32)
        mc = (D.max(1, keepdims=True) * c).astype(np.float32)
        x = (D.astype(np.float64) * np.float64(c) - mc.astype(np.float64)).astype(np.float32)
        P = np.exp2(x.astype(np.float64)).astype(np.float32)
        ell = P.astype(np.float64).sum(1, keepdims=True)
        y = (P * np.float32(S)).astype(np.float32)
        Pt = torch.from_numpy(y).to(torch.float8_e4m3fn).float().numpy().astype(np.float64)
        want = (Pt @ v.astype(np.float64)) / (S * ell)
        assert np.abs(out - want).max() <= 2e-6


def test_reverse_s256_no_noncausal_block_underflow_small():
    """Fixed point (c), Theorem 2: reverse order with S = 256 leaves no key
    outside the sink's block cast to zero (N = 1024, d = 64, Delta = 8)."""
    inp = make_inputs(1, 1, 1, 1024, 64, fmt="f32", delta=8.0, seed=20260100)
    _, _, cnt = oracle.attn(inp.q32, inp.k32, inp.v32, S=256.0, order="reverse", block_kv=64, n_sink=4)
    assert cnt[:, 2].sum() == 0
    # the same keys do collapse under forward order with S = 1
    _, _, cnt1 = oracle.attn(inp.q32, inp.k32, inp.v32, S=1.0, order="forward", block_kv=64, n_sink=4)
    frac = cnt1[:, 2].sum() / (1024 * (1024 - 64))
    assert frac > 0.9


@pytest.fixture(scope="module")
def sweep_base():
    inp = make_inputs(1, 8, 8, 4096, 128, fmt="f32", delta=0.0, seed=20260200)
    rows = np.concatenate([np.arange(h * 4096, h * 4096 + 4096, 64) + (h * 7) % 64 for h in range(8)])
    return inp, rows


def test_sweep_reverse_s256_zero_outside_sink_block(sweep_base):
    inp0, rows = sweep_base
    for D in range(0, 13):
        inp = with_delta(inp0, float(D))
        _, _, cnt = oracle.attn(inp.q32, inp.k32, inp.v32, S=256.0, order="reverse", block_kv=128,
                                rows=rows, n_sink=4)
        assert cnt[:, 2].sum() == 0, D


def test_sweep_forward_fraction_tracks_closed_form(sweep_base):
    """Fixed point (d): the measured forward-order fraction of non-sink P cast
    to zero tracks F(Delta_eff, S) = Phi(Delta_eff + delta_4 - 10 ln 2 - ln S)."""
    inp0, rows = sweep_base
    n_nonsink = rows.size * (4096 - 4)
    worst = 0.0
    for S in (1.0, 16.0, 256.0):
        for D in range(0, 13):
            inp = with_delta(inp0, float(D))
            _, _, cnt = oracle.attn(inp.q32, inp.k32, inp.v32, S=S, order="forward", block_kv=128,
                                    rows=rows, n_sink=4)
            frac = (cnt[:, 1].sum() + cnt[:, 2].sum()) / n_nonsink
            F = analysis.collapse_fraction(inp.delta_eff, S)
            worst = max(worst, abs(frac - F))
            assert abs(frac - F) <= 0.06, (S, D, frac, F)
    assert worst > 0.0


def test_sink_block_counts_agree_between_orders(sweep_base):
    """When block 0 holds the row maximum, its keys see that maximum in both
    orders, so category-0/1 counts agree row by row."""
    inp0, rows = sweep_base
    inp = with_delta(inp0, 10.0)
    _, _, cf = oracle.attn(inp.q32, inp.k32, inp.v32, S=256.0, order="forward", block_kv=128, rows=rows)
    _, _, cr = oracle.attn(inp.q32, inp.k32, inp.v32, S=256.0, order="reverse", block_kv=128, rows=rows)
    B, Hq, N, d = inp.q32.shape
    flat_q = inp.q32.reshape(-1, d)[rows].astype(np.float64)
    heads = rows // N
    holds = np.zeros(rows.size, dtype=bool)
    for h in np.unique(heads):
        sel = heads == h
        D = flat_q[sel] @ inp.k32[0, h].astype(np.float64).T
        holds[sel] = D[:, :128].max(1) >= D[:, 128:].max(1)
    assert holds.sum() > rows.size // 2
    assert np.array_equal(cf[holds, :2], cr[holds, :2])
    assert cr[:, 1].sum() > 0   # keys 4..127 do underflow at Delta = 10 in both orders


def test_table1_statistical_context():
    """Table 1 (N = 4096, block 64, forward): loose agreement of the measured
    S = 1 and S = 256 fractions with the paper's own simulation."""
    with open(os.path.join(GOLD, "table1_collapse.json")) as f:
        t = json.load(f)
    inp0 = make_inputs(1, 2, 2, 4096, 128, fmt="f32", delta=0.0, seed=20260201)
    rows = np.concatenate([np.arange(h * 4096, (h + 1) * 4096, 97) for h in range(2)])
    n_nonsink = rows.size * (4096 - 4)
    for D, s1, s256 in zip(t["delta"], t["frac_zeroed_S1"], t["frac_zeroed_S256"]):
        inp = with_delta(inp0, float(D))
        got = []
        for S in (1.0, 256.0):
            _, _, cnt = oracle.attn(inp.q32, inp.k32, inp.v32, S=S, order="forward", block_kv=64,
                                    rows=rows, n_sink=4)
            got.append((cnt[:, 1].sum() + cnt[:, 2].sum()) / n_nonsink)
        assert abs(got[0] - s1) <= 0.08, (D, got[0], s1)
        assert abs(got[1] - s256) <= 0.08, (D, got[1], s256)


def test_row_sampling_and_argument_checks():
    rows = sample_rows(2, 3, 1000, 128, 4, seed=0)
    assert rows.min() >= 0 and rows.max() < 2 * 3 * 1000
    assert np.all(np.diff(rows) > 0)
    inp = make_inputs(1, 2, 2, 64, 16, fmt="f32", delta=1.0, seed=1)
    with pytest.raises(ValueError):
        oracle.attn(inp.q32, inp.k32, inp.v32, S=0.0, order="forward", block_kv=64)
    with pytest.raises(ValueError):
        oracle.attn(inp.q32, inp.k32, inp.v32, S=1.0, order="forward", block_kv=64, rows=[128])


@pytest.mark.parametrize("causal", [False, True])
@pytest.mark.parametrize("order", ["forward", "reverse"])
@pytest.mark.parametrize("S", [1.0, 256.0])
def test_two_level_scores_closed_form(causal, order, S):
    """Several blocks with the cast on, against a closed form.  q = e_0 and
    k_t = (X if t < 4 else Y) e_0 give raw scores X on the four sink keys and
    Y on every other key.  Forward, block 0 fixes the maximum X at once: every
    non-sink key has P_y = exp2(x_y) and code E(P_y S) (zero at S = 1: the
    collapse).  Reverse, the later blocks come first with maximum Y (P = 1,
    code E(S)); block 0 then raises the maximum and rescales O and l by
    alpha = exp2(fl(Y c) - fl(X c)).  Codes from torch's float8_e4m3fn, sums
    in FP64.  The oracle accumulates l and O in FP32 over up to 256 equal
    addends, so the bar is 3e-5 relative (about n u); Y puts P_y S about 4 %
    away from its E4M3 code, so a plausible slip (l summed over the cast P, a
    missing alpha, a wrong code) moves the result by 1e-3 or more."""
    N, d, Bc, X, Y = 256, 64, 64, 64.0, 0.34375
    rng = np.random.default_rng(31)
    q = np.zeros((1, 1, N, d), np.float32)
    q[..., 0] = 1.0
    k = np.zeros((1, 1, N, d), np.float32)
    k[0, 0, :, 0] = Y
    k[0, 0, :4, 0] = X
    v = rng.standard_normal((1, 1, N, d)).astype(np.float32)
    out, lse, _ = oracle.attn(q, k, v, S=S, order=order, causal=causal, block_kv=Bc)

    c = c_const(d)
    f32 = np.float32
    mcX, mcY = f32(X * c), f32(Y * c)

    def p_of(D, mc):       # P = exp2(fl32(fma(D, c, -mc))), FP64 exp2 rounded once
        x = f32(np.float64(D) * np.float64(c) - np.float64(mc))
        return f32(np.exp2(np.float64(x)))

    def code(p):           # decoded E4M3 code of fl32(P S)
        y = torch.tensor([float(f32(p * f32(S)))], dtype=torch.float32)
        return float(y.to(torch.float8_e4m3fn).float()[0])

    Ps, Py = p_of(X, mcX), p_of(Y, mcX)           # relative to the sink maximum
    P1 = p_of(Y, mcY)                              # relative to Y (= 1)
    alpha = f32(np.exp2(np.float64(mcY) - np.float64(mcX)))
    vv = v[0, 0].astype(np.float64)
    for r in range(N):
        L = r + 1 if causal else N
        sink = vv[:min(4, L)].sum(0)
        ns = min(4, L)
        y0 = vv[ns:min(L, Bc)].sum(0)
        n0 = min(L, Bc) - ns
        y1 = vv[Bc:L].sum(0) if L > Bc else np.zeros(d)
        n1 = max(0, L - Bc)
        if order == "forward" or n1 == 0:
            o = code(Ps) * sink + code(Py) * (y0 + y1)
            ell = ns * np.float64(Ps) + (n0 + n1) * np.float64(Py)
        else:
            o = np.float64(alpha) * code(P1) * y1 + code(Ps) * sink + code(Py) * y0
            ell = np.float64(alpha) * n1 * np.float64(P1) + ns * np.float64(Ps) + n0 * np.float64(Py)
        want = o / (S * ell)
        assert np.all(np.abs(out[r] - want) <= 2e-6 + 3e-5 * np.abs(want)), (r, order, causal, S)
        want_lse = (np.float64(mcX) + math.log2(ell)) * math.log(2.0)
        assert abs(lse[r] - want_lse) <= 3e-5, (r, order, causal, S)
    if S == 1.0:
        assert code(Py) == 0.0          # the non-sink keys collapse under the sink maximum
    else:
        assert abs(code(Py) / (np.float64(Py) * S) - 1.0) > 0.03
