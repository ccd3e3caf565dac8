"""Python binding of libattn_fp8.so (argument marshalling only).

The C entry points are exposed under their C names; ``fwd`` and
``p_underflow_count`` are thin conveniences that take torch tensors on the GPU,
check their dtypes and shapes, allocate outputs with torch and pass the
current torch stream.  Every step of the computation runs in the HIP kernels;
there is no fallback.  If the shared library is missing the import fails.
"""
from __future__ import annotations

import ctypes
import os

import torch

_HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_HERE, "libattn_fp8.so")

ATTN_MODE_FAITHFUL, ATTN_MODE_FAST, ATTN_MODE_NOCAST, ATTN_MODE_FP8QK = 0, 1, 2, 3
ATTN_ORDER_FORWARD, ATTN_ORDER_REVERSE = 0, 1
ATTN_OK, ATTN_ERR_INVALID_ARG, ATTN_ERR_UNSUPPORTED, ATTN_ERR_HIP = 0, -1, -2, -3
ATTN_ERR_SCRATCH = -4
ATTN_SCALE_DYNAMIC = 0x100
ATTN_TILE_256, ATTN_TILE_128 = 0x200, 0x400

MODES = {"faithful": ATTN_MODE_FAITHFUL, "fast": ATTN_MODE_FAST, "nocast": ATTN_MODE_NOCAST,
         "fp8qk": ATTN_MODE_FP8QK}
ORDERS = {"forward": ATTN_ORDER_FORWARD, "reverse": ATTN_ORDER_REVERSE}
SCALES = {"static": 0, "dynamic": ATTN_SCALE_DYNAMIC}
TILES = {None: 0, 256: ATTN_TILE_256, 128: ATTN_TILE_128}   # fast kernel schedule (None: automatic)

if not os.path.exists(LIB_PATH):
    raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                      "(hipcc --offload-arch=gfx950)")
_lib = ctypes.CDLL(LIB_PATH)

_P, _I, _F, _Z = ctypes.c_void_p, ctypes.c_int, ctypes.c_float, ctypes.c_size_t
_lib.attn_fp8_fwd.argtypes = [_P, _P, _P, _P, _P] + [_I] * 8 + [_F, _I, _P]
_lib.attn_fp8_fwd.restype = _I
_lib.attn_fp8_p_underflow_count.argtypes = [_P, _P, _P] + [_I] * 8 + [_F, _I, _I, _P, _P, _P, _P]
_lib.attn_fp8_p_underflow_count.restype = _I
_lib.attn_fp8_fwd_descaled.argtypes = [_P, _P, _P, _P, _P] + [_I] * 8 + [_F, _I, _F, _F, _F, _P]
_lib.attn_fp8_fwd_descaled.restype = _I
_lib.attn_fp8_p_underflow_count_descaled.argtypes = ([_P, _P, _P] + [_I] * 8 + [_F, _I, _I]
                                                     + [_F, _F, _F, _P, _P, _P, _P])
_lib.attn_fp8_p_underflow_count_descaled.restype = _I
_lib.attn_fp8_fwd_kv.argtypes = [_P] * 5 + [_I] * 9 + [_F, _I, _F, _F, _F, _P, _Z, _P]
_lib.attn_fp8_fwd_kv.restype = _I
_lib.attn_fp8_p_underflow_count_kv.argtypes = ([_P] * 3 + [_I] * 9 + [_F, _I, _I, _F, _F, _F]
                                               + [_P] * 4 + [_Z, _P])
_lib.attn_fp8_p_underflow_count_kv.restype = _I
_lib.attn_fp8_fwd_kv_noalloc.argtypes = [_P] * 5 + [_I] * 9 + [_F, _I, _F, _F, _F, _P]
_lib.attn_fp8_fwd_kv_noalloc.restype = _I
_lib.attn_fp8_kv_workspace_bytes.argtypes = [_I] * 9 + [ctypes.POINTER(_Z)]
_lib.attn_fp8_kv_workspace_bytes.restype = _I
_lib.attn_fp8_block_gap_diag.argtypes = ([_P, _P, _P] + [_I] * 8 + [_F, _I, _I, _F, _F, _F, _I]
                                         + [_P] * 5 + [_P])
_lib.attn_fp8_block_gap_diag.restype = _I
_lib.attn_fp8_strerror.argtypes = [_I]
_lib.attn_fp8_strerror.restype = ctypes.c_char_p
_lib.attn_fp8_version.argtypes = []
_lib.attn_fp8_version.restype = _I


class AttnError(RuntimeError):
    def __init__(self, status: int):
        super().__init__(f"attn_fp8 status {status}: {attn_fp8_strerror(status)}")
        self.status = status


# ---- the C entry points, same names, raw pointers (ints) and sizes ----

def attn_fp8_fwd(q, k, v, out, lse, B, Hq, Hkv, N, d, causal, block_kv, order, S, mode, stream):
    return _lib.attn_fp8_fwd(q, k, v, out, lse, B, Hq, Hkv, N, d, causal, block_kv, order,
                             float(S), mode, stream)


def attn_fp8_p_underflow_count(q, k, v, B, Hq, Hkv, N, d, causal, block_kv, order, S, mode,
                               n_sink, counts, out, lse, stream):
    return _lib.attn_fp8_p_underflow_count(q, k, v, B, Hq, Hkv, N, d, causal, block_kv, order,
                                           float(S), mode, n_sink, counts, out, lse, stream)


def attn_fp8_fwd_descaled(q, k, v, out, lse, B, Hq, Hkv, N, d, causal, block_kv, order, S, mode,
                          q_descale, k_descale, v_descale, stream):
    return _lib.attn_fp8_fwd_descaled(q, k, v, out, lse, B, Hq, Hkv, N, d, causal, block_kv,
                                      order, float(S), mode, float(q_descale), float(k_descale),
                                      float(v_descale), stream)


def attn_fp8_p_underflow_count_descaled(q, k, v, B, Hq, Hkv, N, d, causal, block_kv, order, S,
                                        mode, n_sink, q_descale, k_descale, v_descale, counts,
                                        out, lse, stream):
    return _lib.attn_fp8_p_underflow_count_descaled(q, k, v, B, Hq, Hkv, N, d, causal, block_kv,
                                                    order, float(S), mode, n_sink,
                                                    float(q_descale), float(k_descale),
                                                    float(v_descale), counts, out, lse, stream)


def attn_fp8_fwd_kv(q, k, v, out, lse, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order, S, mode,
                    q_descale, k_descale, v_descale, workspace, workspace_bytes, stream):
    return _lib.attn_fp8_fwd_kv(q, k, v, out, lse, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order,
                                float(S), mode, float(q_descale), float(k_descale),
                                float(v_descale), workspace, workspace_bytes, stream)


def attn_fp8_fwd_kv_noalloc(q, k, v, out, lse, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order, S,
                            mode, q_descale, k_descale, v_descale, stream):
    return _lib.attn_fp8_fwd_kv_noalloc(q, k, v, out, lse, B, Hq, Hkv, Nq, Nk, d, causal,
                                        block_kv, order, float(S), mode, float(q_descale),
                                        float(k_descale), float(v_descale), stream)


def attn_fp8_p_underflow_count_kv(q, k, v, B, Hq, Hkv, Nq, Nk, d, causal, block_kv, order, S,
                                  mode, n_sink, q_descale, k_descale, v_descale, counts, out,
                                  lse, workspace, workspace_bytes, stream):
    return _lib.attn_fp8_p_underflow_count_kv(q, k, v, B, Hq, Hkv, Nq, Nk, d, causal, block_kv,
                                              order, float(S), mode, n_sink, float(q_descale),
                                              float(k_descale), float(v_descale), counts, out,
                                              lse, workspace, workspace_bytes, stream)


def attn_fp8_kv_workspace_bytes(B, Hq, Hkv, Nq, Nk, d, causal, block_kv, mode):
    """Returns (status, bytes)."""
    n = _Z(0)
    st = _lib.attn_fp8_kv_workspace_bytes(B, Hq, Hkv, Nq, Nk, d, causal, block_kv, mode,
                                          ctypes.byref(n))
    return st, n.value


def attn_fp8_block_gap_diag(q, k, v, B, Hq, Hkv, N, d, causal, block_kv, order, S, mode, n_sink,
                            q_descale, k_descale, v_descale, nbins, gap_hist, blk_zero, counts,
                            out, lse, stream):
    return _lib.attn_fp8_block_gap_diag(q, k, v, B, Hq, Hkv, N, d, causal, block_kv, order,
                                        float(S), mode, n_sink, float(q_descale),
                                        float(k_descale), float(v_descale), nbins, gap_hist,
                                        blk_zero, counts, out, lse, stream)


def attn_fp8_strerror(status: int) -> str:
    return _lib.attn_fp8_strerror(status).decode()


def attn_fp8_version() -> int:
    return _lib.attn_fp8_version()


# ---- torch conveniences ----

_FAST_QK = (torch.bfloat16, torch.int16, torch.uint16)
_FAST_V = (torch.float8_e4m3fn, torch.uint8)


def _check(q, k, v, mode):
    if q.dim() != 4 or k.dim() != 4 or v.dim() != 4:
        raise ValueError("q, k, v must be [B, H, N, d]")
    B, Hq, N, d = q.shape
    if k.shape != v.shape or k.shape[0] != B or k.shape[2] < N or k.shape[3] != d:
        raise ValueError(f"shape mismatch: q {tuple(q.shape)} k {tuple(k.shape)} v {tuple(v.shape)}")
    for t in (q, k, v):
        if not t.is_cuda or not t.is_contiguous():
            raise ValueError("q, k, v must be contiguous device tensors")
    if mode == ATTN_MODE_FAST:
        if q.dtype not in _FAST_QK or k.dtype not in _FAST_QK or v.dtype not in _FAST_V:
            raise TypeError("fast mode takes bfloat16 q/k and float8_e4m3fn (or uint8) v")
    elif mode == ATTN_MODE_FP8QK:
        if q.dtype not in _FAST_V or k.dtype not in _FAST_V or v.dtype not in _FAST_V:
            raise TypeError("fp8qk mode takes float8_e4m3fn (or uint8) q, k and v")
    elif q.dtype != torch.float32 or k.dtype != torch.float32 or v.dtype != torch.float32:
        raise TypeError("faithful / nocast modes take float32 q, k, v")
    return B, Hq, k.shape[1], N, d, k.shape[2]


def _ptr(t):
    return None if t is None else t.data_ptr()


def _stream(stream):
    s = stream if stream is not None else torch.cuda.current_stream()
    return s.cuda_stream


def kv_workspace(B, Hq, Hkv, N, Nk, d, causal, block_kv, mode, device):
    """A device workspace (torch-allocated) for a KV-cache call of this shape,
    or None when the call does not split."""
    st, n = attn_fp8_kv_workspace_bytes(B, Hq, Hkv, N, Nk, d, int(bool(causal)), int(block_kv),
                                        mode)
    if st != ATTN_OK:
        raise AttnError(st)
    return torch.empty(n, dtype=torch.uint8, device=device) if n else None


def fwd(q, k, v, *, S: float = 256.0, order: str = "reverse", causal: bool = False,
        block_kv: int = 128, mode: str = "fast", out=None, lse=None, want_lse: bool = True,
        stream=None, scale: str = "static", descales=(1.0, 1.0, 1.0), tile=None):
    """Attention forward; returns (out [B,Hq,N,d] float32, lse [B,Hq,N] float32 or None).
    k, v may hold more keys than q has rows (a KV cache): query row r then
    sits at key position Nk - N + r; the call's workspace, if it splits, is
    taken from torch's allocator on q's device.
    scale="dynamic" ORs ATTN_SCALE_DYNAMIC into the mode (S = 2^k0, k0 <= 8);
    descales = per-tensor (q, k, v) descales of the stored values; tile = 256 or
    128 forces the fast kernel's schedule (ATTN_TILE_*), None lets the library pick."""
    m = MODES[mode]
    B, Hq, Hkv, N, d, Nk = _check(q, k, v, m)
    if out is None:
        out = torch.empty((B, Hq, N, d), dtype=torch.float32, device=q.device)
    if lse is None and want_lse:
        lse = torch.empty((B, Hq, N), dtype=torch.float32, device=q.device)
    ws = kv_workspace(B, Hq, Hkv, N, Nk, d, causal, block_kv, m, q.device) if Nk != N else None
    st = attn_fp8_fwd_kv(_ptr(q), _ptr(k), _ptr(v), _ptr(out), _ptr(lse), B, Hq, Hkv, N, Nk, d,
                         int(bool(causal)), int(block_kv), ORDERS[order], S,
                         m | SCALES[scale] | TILES[tile], *descales, _ptr(ws),
                         0 if ws is None else ws.numel(), _stream(stream))
    if st != ATTN_OK:
        raise AttnError(st)
    return out, lse


def p_underflow_count(q, k, v, *, S: float = 256.0, order: str = "reverse", causal: bool = False,
                      block_kv: int = 128, mode: str = "fast", n_sink: int = 4, out=None, lse=None,
                      stream=None, scale: str = "static", descales=(1.0, 1.0, 1.0), tile=None):
    """P-underflow diagnostic; returns counts [B,Hq,N,3] uint32 (as int32 storage)."""
    m = MODES[mode]
    B, Hq, Hkv, N, d, Nk = _check(q, k, v, m)
    counts = torch.empty((B, Hq, N, 3), dtype=torch.int32, device=q.device)
    ws = kv_workspace(B, Hq, Hkv, N, Nk, d, causal, block_kv, m, q.device) if Nk != N else None
    st = attn_fp8_p_underflow_count_kv(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, Nk, d,
                                       int(bool(causal)), int(block_kv), ORDERS[order], S,
                                       m | SCALES[scale] | TILES[tile], int(n_sink), *descales,
                                       _ptr(counts),
                                       _ptr(out), _ptr(lse), _ptr(ws),
                                       0 if ws is None else ws.numel(), _stream(stream))
    if st != ATTN_OK:
        raise AttnError(st)
    return counts


def block_gap_diag(q, k, v, *, S: float = 256.0, order: str = "reverse", causal: bool = False,
                   block_kv: int = 128, mode: str = "fast", n_sink: int = 4, nbins: int = 32,
                   stream=None, scale: str = "static", descales=(1.0, 1.0, 1.0), tile=None):
    """Per-block diagnostic; returns (gap_hist [B,Hq,nblk,nbins], blk_zero [B,Hq,nblk],
    counts [B,Hq,N,3]), all uint32 held in int32 storage."""
    m = MODES[mode]
    B, Hq, Hkv, N, d, Nk = _check(q, k, v, m)
    if Nk != N:
        raise ValueError("block_gap_diag takes square problems (as many keys as query rows)")
    nblk = (N + block_kv - 1) // block_kv
    hist = torch.empty((B, Hq, nblk, nbins), dtype=torch.int32, device=q.device)
    bz = torch.empty((B, Hq, nblk), dtype=torch.int32, device=q.device)
    counts = torch.empty((B, Hq, N, 3), dtype=torch.int32, device=q.device)
    st = attn_fp8_block_gap_diag(_ptr(q), _ptr(k), _ptr(v), B, Hq, Hkv, N, d, int(bool(causal)),
                                 int(block_kv), ORDERS[order], S, m | SCALES[scale] | TILES[tile],
                                 int(n_sink),
                                 *descales, int(nbins), _ptr(hist), _ptr(bz), _ptr(counts), None,
                                 None, _stream(stream))
    if st != ATTN_OK:
        raise AttnError(st)
    return hist, bz, counts
