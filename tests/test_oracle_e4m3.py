"""Pins for the oracle's bit-level E4M3 codec (Sec. 2.1).

The encoder is checked against things it does not share code with: the format
constants printed in the paper, a brute-force nearest-value search written
here, and torch's float8_e4m3fn conversion (a library routine).
"""
import json
import os

import numpy as np
import pytest
import torch

import oracle
from oracle import analysis

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def _gold(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def test_decode_table_matches_printed_format():
    g = _gold("e4m3_format.json")
    codes = np.arange(256, dtype=np.uint8)
    vals = oracle.e4m3_decode(codes)
    pos = vals[1:128]                                   # codes 0x01..0x7F
    finite = pos[np.isfinite(pos)]
    assert finite.size == g["positive_finite_values"]
    assert np.isnan(vals[0x7F]) and np.isnan(vals[0xFF])
    assert vals[0] == 0.0 and np.signbit(vals[0x80])
    assert finite.max() == g["max_representable"]
    sub = finite[finite < g["min_normal"]]
    assert sub.size == g["subnormal_count"]
    assert (finite >= g["min_normal"]).sum() == g["normal_count"]
    assert sub.min() == g["min_subnormal"]
    assert [sub.min(), sub.max()] == g["subnormal_span"]
    # 8 equispaced values in every full normal binade [2^n, 2^(n+1))
    for n in range(-6, 8):
        inb = finite[(finite >= 2.0 ** n) & (finite < 2.0 ** (n + 1))]
        assert inb.size == g["values_per_normal_binade"]
        assert np.allclose(np.diff(inb), 2.0 ** (n - 3))
    # negative codes mirror positive ones
    assert np.array_equal(vals[128:][np.isfinite(vals[128:])], -vals[:128][np.isfinite(vals[:128])])
    # the closed-form list of the analysis module agrees with the decoder
    assert np.array_equal(np.sort(finite), analysis.e4m3_positive_values().astype(np.float32))


def test_round_trip_all_codes():
    codes = np.arange(256, dtype=np.uint8)
    vals = oracle.e4m3_decode(codes)
    back = oracle.e4m3_encode(vals)
    fin = np.isfinite(vals)
    assert np.array_equal(back[fin], codes[fin])
    assert np.all(back[~fin] & 0x7F == 0x7F)


def test_round_to_zero_threshold():
    g = _gold("e4m3_format.json")
    t = np.float32(g["round_to_zero_below"])            # 2^-10
    above = np.nextafter(t, np.float32(1))
    below = np.nextafter(t, np.float32(0))
    enc = oracle.e4m3_encode(np.array([below, t, above], dtype=np.float32))
    # below 2^-10 -> 0; exactly 2^-10 is a tie between 0 and 2^-9 and goes to
    # the even code 0x00; just above -> 2^-9 (code 0x01)
    assert enc.tolist() == [0, 0, 1]


def _brute_force(y: np.ndarray) -> np.ndarray:
    """Nearest finite E4M3 value, ties to the even code, saturate |y| >= 448 to
    448, NaN -> 0x7F | sign.  Independent of the oracle's bit manipulation."""
    grid = np.concatenate([[0.0], analysis.e4m3_positive_values()])   # index == code
    with np.errstate(invalid="ignore"):
        a = np.abs(y.astype(np.float64))
    sign = np.signbit(y).astype(np.uint8) << 7
    idx = np.searchsorted(grid, a)                                     # grid[idx-1] < a <= grid[idx]
    idx = np.clip(idx, 1, grid.size - 1)
    lo, hi = grid[idx - 1], grid[idx]
    dlo, dhi = a - lo, hi - a
    pick_hi = (dhi < dlo) | ((dhi == dlo) & ((idx % 2) == 0))
    code = np.where(pick_hi, idx, idx - 1).astype(np.int64)
    code = np.where(a >= 448.0, 126, code)
    code = np.where(a == 0, 0, code)
    out = (code.astype(np.uint8) | sign)
    out = np.where(np.isnan(y), 0x7F | sign, out)
    return out.astype(np.uint8)


def _structured_patterns():
    hi = np.arange(1 << 16, dtype=np.uint32) << 16
    lows = np.array([0, 1, 0x7FFF, 0x8000, 0x8001, 0xFFFF, 0x1234, 0xC000], dtype=np.uint32)
    return (hi[:, None] | lows[None, :]).ravel()


def test_encoder_vs_brute_force_all_exponents():
    bits = _structured_patterns()
    rng = np.random.default_rng(1)
    bits = np.concatenate([bits, rng.integers(0, 1 << 32, size=2_000_000, dtype=np.uint64).astype(np.uint32)])
    y = bits.view(np.float32)
    got = oracle.e4m3_encode(y)
    want = _brute_force(y)
    bad = np.nonzero(got != want)[0]
    assert bad.size == 0, [(hex(int(bits[i])), float(y[i]), int(got[i]), int(want[i])) for i in bad[:10]]


def test_encoder_dense_below_464():
    # every FP32 value in [2^-12, 464) on a stride, plus the exact ties
    lo = np.float32(2.0 ** -12).view(np.uint32)
    hi = np.float32(464.0).view(np.uint32)
    bits = np.arange(lo, hi, 97, dtype=np.uint32)
    y = bits.view(np.float32)
    assert np.array_equal(oracle.e4m3_encode(y), _brute_force(y))


def test_encoder_vs_torch_float8():
    # torch's float8_e4m3fn conversion (round to nearest even) for |y| <= 448
    rng = np.random.default_rng(2)
    y = np.concatenate([
        (rng.standard_normal(1_000_000) * 40).astype(np.float32),
        np.exp2(rng.uniform(-14, 8.8, 1_000_000)).astype(np.float32),
        analysis.e4m3_positive_values().astype(np.float32),
        ((analysis.e4m3_positive_values()[1:] + analysis.e4m3_positive_values()[:-1]) / 2).astype(np.float32),
    ])
    y = y[np.abs(y) <= 448]
    y = np.concatenate([y, -y])
    t = torch.from_numpy(y).to(torch.float8_e4m3fn).view(torch.uint8).numpy()
    assert np.array_equal(oracle.e4m3_encode(y), t)


def test_saturation_and_specials():
    y = np.array([448, 449, 463.9, 464, 1e6, np.inf, -np.inf, -500, np.nan], dtype=np.float32)
    got = oracle.e4m3_encode(y).tolist()
    assert got[:6] == [0x7E] * 6
    assert got[6] == 0xFE and got[7] == 0xFE
    assert got[8] & 0x7F == 0x7F


@pytest.mark.parametrize("S", [1.0, 256.0, 448.0])
def test_pipeline_max_error_is_half_step(S):
    """Sec. 5.2: through P~ = Round(P*S)/S the pointwise error is at most dp(S)/2,
    and the bound is attained (at the ties of the widest step)."""
    rng = np.random.default_rng(3)
    lo, hi = 0, np.float32(1.0).view(np.uint32)
    bits = np.concatenate([np.arange(lo, hi, 1021, dtype=np.uint32),
                           rng.integers(lo, hi, size=1_000_000).astype(np.uint32)])
    P = bits.view(np.float32)
    # midpoints of the widest step below S, mapped back to the P domain
    grid = np.concatenate([[0.0], analysis.e4m3_positive_values()])
    mids = ((grid[1:] + grid[:-1]) / 2)
    mids = mids[mids < min(S, 448)] / S
    P = np.concatenate([P, mids.astype(np.float32)])
    Pt = oracle.e4m3_decode(oracle.e4m3_encode(P * np.float32(S))).astype(np.float64) / S
    err = np.abs(Pt - P.astype(np.float64)).max()
    bound = analysis.dp(S) / 2
    pow2 = float(np.log2(S)).is_integer()
    # S = 2^k: P*S is exact (Prop. 2), so the bound holds exactly; otherwise the
    # FP32 product adds one rounding, at most 2^-24 in the P domain
    slack = 0.0 if pow2 else 2.0 ** -24
    assert err <= bound + slack
    assert err >= bound * (1 - 1e-6)
