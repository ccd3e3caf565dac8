"""CPU oracle for FP8 online-softmax attention (test infrastructure).

Only ``tests/``, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` may import this package.  The product path (the HIP library and
its binding) never touches it, and the two share no code.

``liboracle.so`` is built from ``oracle.c`` with gcc (``build()``); the
Python side only marshals numpy arrays.  ``analysis`` holds the closed forms of
the paper (dp(S), F(Delta, S), delta_k).
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "oracle.c")
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
# test build with the planted exp2 error compiled in (-DORACLE_TEST_PLANTS);
# used only by the code-ambiguity bound's own tests
_PLANT_PATH = os.path.join(_HERE, "liboracle_plant.so")
_lib = None
_plant_lib = None

ORDER = {"forward": 0, "reverse": 1}
SCALE = {"static": 0, "dynamic": 1}


CFLAGS = ["-O2", "-std=c11", "-fno-fast-math", "-ffp-contract=off", "-fPIC", "-shared",
          "-pthread"]


def _compile(path: str, extra=()) -> None:
    tmp = path + ".tmp%d" % os.getpid()
    cmd = ["gcc", *CFLAGS, *extra, "-o", tmp, _SRC, "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(tmp, path)


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (no fast-math, no FMA contraction), and
    the test build liboracle_plant.so."""
    if force or not os.path.exists(_LIB_PATH):
        _compile(_LIB_PATH)
    if force or not os.path.exists(_PLANT_PATH):
        _compile(_PLANT_PATH, ["-DORACLE_TEST_PLANTS"])
    return _LIB_PATH


def _declare(L: ctypes.CDLL) -> ctypes.CDLL:
    P = ctypes.c_void_p
    i32, i64, f32, f64 = ctypes.c_int, ctypes.c_int64, ctypes.c_float, ctypes.c_double
    L.oracle_e4m3_encode.argtypes = [f32]
    L.oracle_e4m3_encode.restype = ctypes.c_uint8
    L.oracle_e4m3_decode.argtypes = [ctypes.c_uint8]
    L.oracle_e4m3_decode.restype = f32
    L.oracle_e4m3_encode_array.argtypes = [P, P, i64]
    L.oracle_e4m3_encode_array.restype = None
    L.oracle_e4m3_decode_array.argtypes = [P, P, i64]
    L.oracle_e4m3_decode_array.restype = None
    L.oracle_attn_full.argtypes = ([P] * 9 + [i32] + [i32] * 9 + [f32, i32, i32, i32]
                                   + [f32, f32, f32, f64, f64, P, i64, i32])
    L.oracle_attn_full.restype = i32
    L.oracle_ref_fp64_kv.argtypes = [P, P, P, P, P] + [i32] * 7 + [f64, f64, f64, P, i64, i32]
    L.oracle_ref_fp64_kv.restype = i32
    L.oracle_version.restype = i32
    return L


def plant_lib() -> ctypes.CDLL:
    """The test build (planted exp2 error available through jitter_rel)."""
    global _plant_lib
    if _plant_lib is None:
        if not os.path.exists(_PLANT_PATH):
            _compile(_PLANT_PATH, ["-DORACLE_TEST_PLANTS"])
        _plant_lib = _declare(ctypes.CDLL(_PLANT_PATH))
    return _plant_lib


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH):
            _compile(_LIB_PATH)
        _lib = _declare(ctypes.CDLL(_LIB_PATH))
    return _lib


def default_threads() -> int:
    """Usable host cores, capped at 16 (the CPU share of one GPU on the GPU hosts)."""
    try:
        n = len(os.sched_getaffinity(0))
    except AttributeError:  # pragma: no cover
        n = os.cpu_count() or 1
    return max(1, min(16, n))


def _ptr(a: np.ndarray | None):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def e4m3_encode(x) -> np.ndarray:
    """Bit-level OCP E4M3 encoding (RNE, subnormals, satfinite) of float32 data."""
    x = np.ascontiguousarray(np.asarray(x, dtype=np.float32))
    out = np.empty(x.shape, dtype=np.uint8)
    lib().oracle_e4m3_encode_array(_ptr(x), _ptr(out), x.size)
    return out


def e4m3_decode(codes) -> np.ndarray:
    codes = np.ascontiguousarray(np.asarray(codes, dtype=np.uint8))
    out = np.empty(codes.shape, dtype=np.float32)
    lib().oracle_e4m3_decode_array(_ptr(codes), _ptr(out), codes.size)
    return out


def attn(q, k, v, *, S: float, order: str, block_kv: int, causal: bool = False,
         cast: bool = True, n_sink: int = 4, rows=None, nthreads: int | None = None,
         scale: str = "static", descales=(1.0, 1.0, 1.0), bound_rel: float | None = None,
         jitter_rel: float = 0.0):
    """Algorithm 1 on the given rows.

    q: [B,Hq,Nq,d]; k, v: [B,Hkv,Nk,d] (Nq <= Nk; query row r sits at key
    position Nk - Nq + r, so Nq = Nk is plain self-attention); float32 arrays
    holding the exact values the device consumed.  rows: flat row ids
    ((b*Hq+hq)*Nq + r) or None for all.
    scale: "static" (one S for every block) or "dynamic" (per-block 2^kj from
    the block's P range, S = 2^k0 its floor; see oracle.c).
    descales: per-tensor (q, k, v) descales of the stored values (Sec. 6.1).
    bound_rel: if given, also return amb [n_rows,d], the bound on how far out
    can move when every P*S within bound_rel (relative) of an E4M3 rounding
    midpoint takes the other code (see oracle_attn_full in oracle.c).
    jitter_rel: planted exp2 error for the bound's own tests (runs the test
    build liboracle_plant.so); 0 for the method itself.
    Returns (out [n_rows,d] float32, lse [n_rows] float32, counts [n_rows,3]
    uint32[, amb [n_rows,d] float32]).
    """
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k, dtype=np.float32)
    v = np.ascontiguousarray(v, dtype=np.float32)
    B, Hq, Nq, d = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    if rows is None:
        n_rows = B * Hq * Nq
        rows_a = None
    else:
        rows_a = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        n_rows = rows_a.size
    out = np.empty((n_rows, d), dtype=np.float32)
    lse = np.empty(n_rows, dtype=np.float32)
    counts = np.zeros((n_rows, 3), dtype=np.uint32)
    amb = None if bound_rel is None else np.empty((n_rows, d), dtype=np.float32)
    qd, kd, vd = (float(x) for x in descales)
    L = plant_lib() if jitter_rel else lib()
    rc = L.oracle_attn_full(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _ptr(counts),
                            _ptr(amb), None, None, 0, B, Hq, Hkv, Nq, Nk, d,
                            int(bool(causal)), int(block_kv), ORDER[order], float(S),
                            int(bool(cast)), SCALE[scale], int(n_sink), qd, kd, vd,
                            float(bound_rel or 0.0), float(jitter_rel), _ptr(rows_a), n_rows,
                            nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle_attn rejected its arguments")
    if amb is not None:
        return out, lse, counts, amb
    return out, lse, counts


def block_diag(q, k, v, *, S: float, order: str, block_kv: int, causal: bool = False,
               cast: bool = True, n_sink: int = 4, rows=None, nthreads: int | None = None,
               scale: str = "static", descales=(1.0, 1.0, 1.0), nbins: int = 32):
    """Algorithm 1 with the per-block diagnostic (see oracle_attn_full in
    oracle.c), accumulated over the given rows.
    Returns (out, lse, counts, gap_hist [B,Hq,nblk,nbins] uint32,
    blk_zero [B,Hq,nblk] uint32)."""
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k, dtype=np.float32)
    v = np.ascontiguousarray(v, dtype=np.float32)
    B, Hq, Nq, d = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    if rows is None:
        n_rows = B * Hq * Nq
        rows_a = None
    else:
        rows_a = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        n_rows = rows_a.size
    nblk = (Nk + block_kv - 1) // block_kv
    out = np.empty((n_rows, d), dtype=np.float32)
    lse = np.empty(n_rows, dtype=np.float32)
    counts = np.zeros((n_rows, 3), dtype=np.uint32)
    hist = np.empty((B, Hq, nblk, nbins), dtype=np.uint32)
    bz = np.empty((B, Hq, nblk), dtype=np.uint32)
    qd, kd, vd = (float(x) for x in descales)
    rc = lib().oracle_attn_full(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), _ptr(counts),
                                None, _ptr(hist), _ptr(bz), int(nbins), B, Hq, Hkv, Nq, Nk, d,
                                int(bool(causal)), int(block_kv), ORDER[order], float(S),
                                int(bool(cast)), SCALE[scale], int(n_sink), qd, kd, vd, 0.0, 0.0,
                                _ptr(rows_a), n_rows, nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle_attn_full rejected its arguments")
    return out, lse, counts, hist, bz


def ref_fp64(q, k, v, *, causal: bool = False, rows=None, nthreads: int | None = None,
             descales=(1.0, 1.0, 1.0)):
    """Textbook softmax attention in FP64 (no blocks, no cast) on the given rows.

    Returns (out [n_rows,d] float64, lse [n_rows] float64).
    """
    q = np.ascontiguousarray(q, dtype=np.float32)
    k = np.ascontiguousarray(k, dtype=np.float32)
    v = np.ascontiguousarray(v, dtype=np.float32)
    B, Hq, Nq, d = q.shape
    Hkv, Nk = k.shape[1], k.shape[2]
    if rows is None:
        n_rows = B * Hq * Nq
        rows_a = None
    else:
        rows_a = np.ascontiguousarray(np.asarray(rows, dtype=np.int64))
        n_rows = rows_a.size
    out = np.empty((n_rows, d), dtype=np.float64)
    lse = np.empty(n_rows, dtype=np.float64)
    qd, kd, vd = (float(x) for x in descales)
    rc = lib().oracle_ref_fp64_kv(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse),
                                  B, Hq, Hkv, Nq, Nk, d, int(bool(causal)), qd, kd, vd,
                                  _ptr(rows_a), n_rows, nthreads or default_threads())
    if rc != 0:
        raise ValueError("oracle_ref_fp64 rejected its arguments")
    return out, lse
