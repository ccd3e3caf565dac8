"""Seeded synthetic inputs shaped like the paper's sink workload.

This module only draws and lays out numbers; it contains none of the
attention arithmetic.  Both the device path and the CPU oracle consume what it
produces, so they see bit-identical values.

Workload structure (Sec. 3.1): one head per (batch, head) pair, non-sink
logits s ~ N(0, 1) after the 1/sqrt(d) scaling, the first ``n_sink`` keys lifted
by Delta (Sec. 3.2: the sink scores carry the same N(0,1) fluctuation as the
others).  Recipe:

* Q and K entries: N(0, 1) snapped to the 2^-5 grid and clipped to
  +-(8 - 2^-5).  Every product q_i k_i is then a multiple of 2^-10 below 64 in
  magnitude, so any dot product over d <= 128 terms is exact in FP32 whatever
  the summation order, and every entry is exact in bfloat16.
* The sink offset travels in the last channel: Q[..., d-1] = 1 and
  K[..., t, d-1] = snap(sqrt(d) * (Delta * [t < n_sink] + b_t)), so the logit of
  key t gains Delta (+ b_t); b_t ~ N(0, bias_var) when ``bias_var > 0``.  For
  bfloat16 inputs that channel is additionally rounded to bfloat16 (it is the
  only channel that can leave the exact range).  The realised sink offset is
  reported as ``delta_eff``.  Non-sink logits then have variance (d-1)/d.
* V: float32 N(0, 1) for the FP32 modes; for the fast mode N(0, 1) divided by
  its per-tensor max |V| and rounded to OCP E4M3 (torch's float8_e4m3fn
  conversion, round to nearest even), so |V| <= 1.
* E4M3 Q/K (fmt "e4m3", the FP8 x FP8 scores of Algorithm 1): N(0, 1)
  clipped to +-4 and rounded to E4M3, values below 2^-1 in magnitude snapped
  to the 2^-4 grid instead (every value is then an E4M3 value and a multiple
  of 2^-4).  Products are multiples of 2^-8 of magnitude <= 16, so dots over
  d <= 128 terms stay below 2^11 and are exact in FP32 in any order.  They are
  also exact on the FP8 matrix cores of gfx950, which add products in groups
  of eight aligned to the group's largest product and drop the bits more than
  13 places below it (measured; a product <= 16 keeps bits down to 2^-9).  The sink
  offset travels in the last SINK_CH8 channels: Q = 4 there, K = the E4M3 grid
  value u with 4 * SINK_CH8 * u ~ sqrt(d) (Delta [t < n_sink] + b_t) (the same
  u in every one of them); those channels are 0 for the other keys' offset
  part.  Non-sink logits then have variance (d - SINK_CH8)/d.  V as in the
  fast mode.

Seeds: numpy PCG64; head (b, h) of each tensor draws from its own stream
seeded by SeedSequence([seed, tensor, b, h]) (q = 1, k = 2, v = 3; the per-key
bias uses [seed, 4]).
"""
from __future__ import annotations

import concurrent.futures as cf
import os
from dataclasses import dataclass, field

import numpy as np
import torch

GRID = 2.0 ** -5
CLIP = 8.0 - GRID
GRID8 = 2.0 ** -4      # E4M3 Q/K: grid of the small values
CLIP8 = 4.0
SINK_CH8 = 10          # E4M3 Q/K: channels carrying the sink offset


@dataclass
class AttnInputs:
    """Host arrays for one problem.

    ``q32``/``k32``/``v32`` are float32 arrays holding exactly the values the
    device consumes (decoded where the device format is narrower); ``q_dev`` /
    ``k_dev`` / ``v_dev`` are the arrays in device format (float32, or raw
    bfloat16 / E4M3 bit patterns as uint16 / uint8).
    """
    B: int
    Hq: int
    Hkv: int
    N: int
    d: int
    fmt: str                    # "f32", "bf16_e4m3" or "e4m3"
    delta: float
    n_sink: int
    q32: np.ndarray
    k32: np.ndarray
    v32: np.ndarray
    q_dev: np.ndarray
    k_dev: np.ndarray
    v_dev: np.ndarray
    delta_eff: float
    meta: dict = field(default_factory=dict)


def _snap_inplace(x: np.ndarray) -> None:
    """Snap float32 data to the 2^-5 grid (round half to even) and clip, in place."""
    x *= np.float32(1.0 / GRID)
    np.rint(x, out=x)
    np.clip(x, -CLIP / GRID, CLIP / GRID, out=x)
    x *= np.float32(GRID)


def _bf16_round(x: np.ndarray) -> np.ndarray:
    """Round float32 to the nearest bfloat16 value (ties to even), as float32."""
    return torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.bfloat16).float().numpy()


def _bf16_bits(x: np.ndarray) -> np.ndarray:
    """Raw bfloat16 bit patterns of float32 values that are exact in bfloat16."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    if np.any(u[..., ::7] & 0xFFFF):
        raise AssertionError("value not exact in bfloat16")
    # little-endian: the high 16 bits of each float32 are the odd uint16 halves
    return np.ascontiguousarray(u.view(np.uint16)[..., 1::2])


def _e4m3_grid_inplace(x: np.ndarray) -> None:
    """E4M3 values that are multiples of 2^-4, |x| <= 4, in place (E4M3 steps
    are 2^-4 or coarser from 2^-1 up, so only smaller values need the grid)."""
    np.clip(x, -CLIP8, CLIP8, out=x)
    small = np.abs(x) < np.float32(0.5)
    t = torch.from_numpy(x).to(torch.float8_e4m3fn).float().numpy()
    x[...] = np.where(small, np.rint(x * np.float32(1 / GRID8)) * np.float32(GRID8), t)


def _e4m3_codes(x: np.ndarray) -> tuple[np.ndarray, np.ndarray]:
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32)).to(torch.float8_e4m3fn)
    return t.view(torch.uint8).numpy().copy(), t.float().numpy()


def _workers() -> int:
    try:
        return max(1, min(16, len(os.sched_getaffinity(0))))
    except AttributeError:  # pragma: no cover
        return 4


def _normal_heads(seed: int, tag: int, B: int, H: int, N: int, d: int) -> np.ndarray:
    """[B][H][N][d] float32 N(0,1); head (b, h) draws from its own PCG64 stream
    seeded by (seed, tag, b, h), so heads can be generated in parallel."""
    out = np.empty((B, H, N, d), dtype=np.float32)

    def fill(bh):
        b, h = divmod(bh, H)
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, tag, b, h])))
        rng.standard_normal((N, d), dtype=np.float32, out=out[b, h])

    with cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(fill, range(B * H)))
    return out


def _parallel_heads(fn, B: int, H: int) -> None:
    with cf.ThreadPoolExecutor(_workers()) as ex:
        list(ex.map(lambda bh: fn(*divmod(bh, H)), range(B * H)))


def sink_channel(N: int, d: int, delta: float, n_sink: int, bias: np.ndarray | None,
                 bf16: bool) -> np.ndarray:
    """Values of K[..., :, d-1] for one KV head (length N)."""
    off = np.zeros(N, dtype=np.float64)
    off[:n_sink] = delta
    if bias is not None:
        off = off + bias
    ch = np.round(np.sqrt(d) * off / GRID) * GRID
    ch = ch.astype(np.float32)
    if bf16:
        ch = _bf16_round(ch)
    return ch


def make_inputs(B: int, Hq: int, Hkv: int, N: int, d: int, *, fmt: str, delta: float,
                seed: int, n_sink: int = 4, bias_var: float = 0.0,
                sink_channel_on: bool = True) -> AttnInputs:
    """Draw one problem.  fmt: "f32" (faithful / nocast), "bf16_e4m3" (fast) or
    "e4m3" (E4M3 Q/K/V)."""
    if fmt not in ("f32", "bf16_e4m3", "e4m3"):
        raise ValueError(fmt)
    if fmt == "e4m3":
        return _make_inputs_e4m3(B, Hq, Hkv, N, d, delta=delta, seed=seed, n_sink=n_sink,
                                 bias_var=bias_var, sink_channel_on=sink_channel_on)
    q = _normal_heads(seed, 1, B, Hq, N, d)
    k = _normal_heads(seed, 2, B, Hkv, N, d)
    v = _normal_heads(seed, 3, B, Hkv, N, d)
    bias = None
    if bias_var > 0:
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 4])))
        bias = rng.standard_normal((B, Hkv, N)) * np.sqrt(bias_var)
    bf16 = fmt == "bf16_e4m3"
    _parallel_heads(lambda b, h: _snap_inplace(q[b, h]), B, Hq)
    _parallel_heads(lambda b, h: _snap_inplace(k[b, h]), B, Hkv)
    delta_eff = float("nan")
    if sink_channel_on and N > 0:
        q[..., d - 1] = 1.0
        for b in range(B):
            for h in range(Hkv):
                k[b, h, :, d - 1] = sink_channel(N, d, delta, n_sink,
                                                 None if bias is None else bias[b, h], bf16)
        delta_eff = float(sink_channel(max(n_sink, 1), d, delta, n_sink, None, bf16)[0] / np.sqrt(d))
    meta = {"seed": seed, "bias_var": bias_var}
    if bf16:
        amax = float(max(v.max(), -v.min())) if v.size else 1.0
        v_codes = np.empty(v.shape, dtype=np.uint8)

        def enc(b, h):
            v[b, h] /= np.float32(amax)
            v_codes[b, h], v[b, h] = _e4m3_codes(v[b, h])

        _parallel_heads(enc, B, Hkv)
        meta["v_amax"] = amax
        return AttnInputs(B, Hq, Hkv, N, d, fmt, delta, n_sink, q, k, v,
                          _bf16_bits(q), _bf16_bits(k), v_codes, delta_eff, meta)
    return AttnInputs(B, Hq, Hkv, N, d, fmt, delta, n_sink, q, k, v, q, k, v, delta_eff, meta)


def sink_channel8(N: int, d: int, delta: float, n_sink: int, bias: np.ndarray | None) -> np.ndarray:
    """E4M3 Q/K: the value u of K in each of the SINK_CH8 sink channels (Q = 4 there)."""
    off = np.zeros(N, dtype=np.float64)
    off[:n_sink] = delta
    if bias is not None:
        off = off + bias
    u = (np.sqrt(d) * off / (4.0 * SINK_CH8)).astype(np.float32)
    _e4m3_grid_inplace(u)
    return u


def _make_inputs_e4m3(B, Hq, Hkv, N, d, *, delta, seed, n_sink, bias_var, sink_channel_on):
    q = _normal_heads(seed, 1, B, Hq, N, d)
    k = _normal_heads(seed, 2, B, Hkv, N, d)
    v = _normal_heads(seed, 3, B, Hkv, N, d)
    bias = None
    if bias_var > 0:
        rng = np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, 4])))
        bias = rng.standard_normal((B, Hkv, N)) * np.sqrt(bias_var)
    _parallel_heads(lambda b, h: _e4m3_grid_inplace(q[b, h]), B, Hq)
    _parallel_heads(lambda b, h: _e4m3_grid_inplace(k[b, h]), B, Hkv)
    delta_eff = float("nan")
    nc = min(SINK_CH8, d)
    if sink_channel_on and N > 0:
        q[..., d - nc:] = 4.0
        for b in range(B):
            for h in range(Hkv):
                k[b, h, :, d - nc:] = sink_channel8(N, d, delta, n_sink,
                                                    None if bias is None else bias[b, h])[:, None]
        u0 = sink_channel8(max(n_sink, 1), d, delta, n_sink, None)[0]
        delta_eff = float(4.0 * nc * u0 / np.sqrt(d))
    amax = float(max(v.max(), -v.min())) if v.size else 1.0
    v_codes = np.empty(v.shape, dtype=np.uint8)
    q_codes = np.empty(q.shape, dtype=np.uint8)
    k_codes = np.empty(k.shape, dtype=np.uint8)

    def enc_v(b, h):
        v[b, h] /= np.float32(amax)
        v_codes[b, h], v[b, h] = _e4m3_codes(v[b, h])

    def enc_q(b, h):
        q_codes[b, h], dec = _e4m3_codes(q[b, h])
        assert np.array_equal(dec, q[b, h])

    def enc_k(b, h):
        k_codes[b, h], dec = _e4m3_codes(k[b, h])
        assert np.array_equal(dec, k[b, h])

    _parallel_heads(enc_v, B, Hkv)
    _parallel_heads(enc_q, B, Hq)
    _parallel_heads(enc_k, B, Hkv)
    meta = {"seed": seed, "bias_var": bias_var, "v_amax": amax}
    return AttnInputs(B, Hq, Hkv, N, d, "e4m3", delta, n_sink, q, k, v, q_codes, k_codes,
                      v_codes, delta_eff, meta)


def with_delta(inp: AttnInputs, delta: float) -> AttnInputs:
    """Same base Q/K/V with only the sink keys' channel rewritten for a new Delta
    (paired runs, as in the paper's paired comparisons).  Requires bias_var == 0."""
    if inp.meta.get("bias_var", 0.0) > 0:
        raise ValueError("with_delta needs inputs without a per-key bias")
    if inp.fmt == "e4m3":
        raise ValueError("with_delta covers the f32 and bf16 formats")
    bf16 = inp.fmt == "bf16_e4m3"
    k32 = inp.k32.copy()
    ns = min(inp.n_sink, inp.N)
    ch = sink_channel(max(inp.n_sink, 1), inp.d, delta, inp.n_sink, None, bf16)[:ns]
    k32[:, :, :ns, inp.d - 1] = ch
    k_dev = _bf16_bits(k32) if bf16 else k32
    delta_eff = float(ch[0] / np.sqrt(inp.d)) if ns else float("nan")
    return AttnInputs(inp.B, inp.Hq, inp.Hkv, inp.N, inp.d, inp.fmt, delta, inp.n_sink,
                      inp.q32, k32, inp.v32, inp.q_dev, k_dev, inp.v_dev, delta_eff,
                      dict(inp.meta))


def with_sink_cluster(inp: AttnInputs, start: int, count: int, delta: float) -> AttnInputs:
    """A second sink cluster: keys start .. start+count-1 of every KV head get
    the sink channel of a sink with gap ``delta`` (the same rounding as the
    first cluster), so sinks are spread over the sequence rather than all at
    position 0.  Q, V and every other key are unchanged.  f32 and bf16 inputs."""
    if inp.fmt not in ("f32", "bf16_e4m3"):
        raise ValueError("sink clusters are built for the f32 and bf16 formats")
    if not (0 <= start and count > 0 and start + count <= inp.N):
        raise ValueError("cluster outside the keys")
    bf16 = inp.fmt == "bf16_e4m3"
    val = sink_channel(1, inp.d, delta, 1, None, bf16)[0]
    k32 = inp.k32.copy()
    k32[:, :, start:start + count, inp.d - 1] = val
    k_dev = _bf16_bits(k32) if bf16 else k32
    clusters = list(inp.meta.get("sink_clusters", [])) + [(start, count, delta)]
    return AttnInputs(inp.B, inp.Hq, inp.Hkv, inp.N, inp.d, inp.fmt, inp.delta, inp.n_sink,
                      inp.q32, k32, inp.v32, inp.q_dev, k_dev, inp.v_dev, inp.delta_eff,
                      dict(inp.meta, sink_clusters=clusters))


def last_queries(inp: AttnInputs, nq: int) -> AttnInputs:
    """The KV-cache prefill shape: the same keys and values, and only the last
    ``nq`` query rows (positions N - nq .. N - 1 of the sequence)."""
    if not 0 < nq <= inp.N:
        raise ValueError("need 0 < nq <= N")
    cut = slice(inp.N - nq, inp.N)
    return AttnInputs(inp.B, inp.Hq, inp.Hkv, inp.N, inp.d, inp.fmt, inp.delta, inp.n_sink,
                      np.ascontiguousarray(inp.q32[:, :, cut]), inp.k32, inp.v32,
                      np.ascontiguousarray(inp.q_dev[:, :, cut]), inp.k_dev, inp.v_dev,
                      inp.delta_eff, dict(inp.meta, nq=nq))


def sample_rows(B: int, Hq: int, N: int, tile: int, every: int, seed: int,
                per_tile: int = 2) -> np.ndarray:
    """Flat row ids ((b*Hq + h)*N + r) for row-sampled checks: in every head, the
    first and last query tile in full plus ``per_tile`` random rows from every
    ``every``-th tile (and always the very last row)."""
    rng = np.random.Generator(np.random.PCG64(seed))
    ntile = (N + tile - 1) // tile
    rows = []
    for bh in range(B * Hq):
        base = bh * N
        for t in range(ntile):
            r0, r1 = t * tile, min(N, (t + 1) * tile)
            if t == 0 or t == ntile - 1:
                rows.extend(range(base + r0, base + r1))
            elif t % every == 0:
                rows.extend(base + rng.integers(r0, r1, size=per_tile))
        rows.append(base + N - 1)
    return np.unique(np.asarray(rows, dtype=np.int64))
