"""Randomised parity sweep: shapes, modes and settings drawn from a fixed seed,
every one checked against the oracle to the same bar as the other parity
tests (counts exact where claimed, outputs within the mode's tolerance plus
the code-ambiguity bound, lse within 1e-4).  Covers combinations the
structured tests do not enumerate: odd lengths, GQA ratios, KV-cache offsets
that are and are not block-aligned, S below 1 and above 448, descales."""
import numpy as np
import pytest

from paper_2606_06521_amd.inputs import last_queries, make_inputs
from tests.gpu_helpers import compare, log, run_gpu, to_device

pytestmark = pytest.mark.gpu

FMT = {"faithful": "f32", "nocast": "f32", "fast": "bf16_e4m3", "fp8qk": "e4m3"}


def _draw(rng):
    mode = rng.choice(["faithful", "fast", "fast", "fp8qk", "fp8qk", "nocast"])
    d = int(rng.choice([64, 128]))
    bkv = int(rng.choice([64, 128]))
    hkv = int(rng.choice([1, 2]))
    hq = hkv * int(rng.choice([1, 2, 4]))
    b = int(rng.integers(1, 3))
    nk = int(rng.integers(1, 700))
    nq = nk if rng.random() < 0.6 else int(rng.integers(1, nk + 1))
    causal = bool(rng.integers(0, 2))
    order = str(rng.choice(["forward", "reverse"]))
    scale = "static"
    if mode != "nocast" and rng.random() < 0.3:
        scale = "dynamic"
        S = float(2.0 ** int(rng.integers(0, 9)))
    else:
        S = float(rng.choice([1.0, 256.0, 448.0, 3.0, 0.25, 1024.0, 16.0]))
    ds = (1.0, 1.0, 1.0)
    if mode == "fp8qk" and rng.random() < 0.5:
        ds = tuple(float(x) for x in rng.choice([0.5, 0.75, 1.25, 2.0], 3))
    delta = float(rng.uniform(0.0, 12.0))
    return dict(mode=mode, d=d, bkv=bkv, hkv=hkv, hq=hq, b=b, nk=nk, nq=nq, causal=causal,
                order=order, scale=scale, S=S, ds=ds, delta=delta)


@pytest.mark.parametrize("seed", range(48))
def test_random_config(seed):
    c = _draw(np.random.default_rng(7000 + seed))
    label = f"random seed={seed} {c}"
    log(label)
    full = make_inputs(c["b"], c["hq"], c["hkv"], c["nk"], c["d"], fmt=FMT[c["mode"]],
                       delta=c["delta"], seed=7100 + seed)
    inp = last_queries(full, c["nq"]) if c["nq"] < c["nk"] else full
    dev = to_device(inp)
    gpu = run_gpu(dev, c["mode"], c["S"], c["order"], c["causal"], c["bkv"], scale=c["scale"],
                  descales=c["ds"])
    compare(inp, gpu, c["mode"], c["S"], c["order"], c["causal"], c["bkv"], label=label,
            scale=c["scale"], descales=c["ds"])


def _draw_split(rng):
    # few heads and a short query chunk against a long cache: the prefill
    # kernel splits each 32-row tile over C = min(256 / tiles, blocks / 8, 8)
    # workgroups (C = 2 .. 8 on 256 CUs)
    mode = str(rng.choice(["fast", "fp8qk"]))
    d = int(rng.choice([64, 128]))
    bkv = int(rng.choice([64, 128]))
    hkv = int(rng.choice([1, 2]))
    hq = hkv * int(rng.choice([1, 2, 4]))
    b = int(rng.integers(1, 3))
    nk = int(rng.integers(1100, 6000))
    nq = int(rng.integers(1, 65))
    causal = bool(rng.integers(0, 2))
    order = str(rng.choice(["forward", "reverse"]))
    scale = "dynamic" if rng.random() < 0.3 else "static"
    S = float(2.0 ** int(rng.integers(0, 9))) if scale == "dynamic" else float(rng.choice([1.0, 256.0, 448.0, 3.0]))
    ds = (1.0, 1.0, 1.0)
    if mode == "fp8qk" and rng.random() < 0.5:
        ds = tuple(float(x) for x in rng.choice([0.5, 0.75, 1.25, 2.0], 3))
    delta = float(rng.uniform(0.0, 12.0))
    return dict(mode=mode, d=d, bkv=bkv, hkv=hkv, hq=hq, b=b, nk=nk, nq=nq, causal=causal,
                order=order, scale=scale, S=S, ds=ds, delta=delta)


@pytest.mark.parametrize("seed", range(24))
def test_random_split_prefill(seed):
    c = _draw_split(np.random.default_rng(8000 + seed))
    label = f"random split seed={seed} {c}"
    log(label)
    full = make_inputs(c["b"], c["hq"], c["hkv"], c["nk"], c["d"], fmt=FMT[c["mode"]],
                       delta=c["delta"], seed=8100 + seed)
    inp = last_queries(full, c["nq"])
    dev = to_device(inp)
    gpu = run_gpu(dev, c["mode"], c["S"], c["order"], c["causal"], c["bkv"], scale=c["scale"],
                  descales=c["ds"])
    compare(inp, gpu, c["mode"], c["S"], c["order"], c["causal"], c["bkv"], label=label,
            scale=c["scale"], descales=c["ds"])
