"""Builds and loads libgpu_probes.so (hardware probes used by the GPU tests)."""
from __future__ import annotations

import ctypes
import os
import subprocess

HERE = os.path.dirname(os.path.abspath(__file__))
SRC = os.path.join(HERE, "gpu_probes.hip")
LIB = os.path.join(HERE, "libgpu_probes.so")
FLAGS = ["--offload-arch=gfx950", "-O3", "-std=c++17", "-fPIC", "-shared",
         "-Xclang", "-target-feature", "-Xclang", "-packed-fp32-ops"]
_lib = None


def build() -> str:
    tmp = LIB + ".tmp%d" % os.getpid()
    subprocess.run([os.environ.get("HIPCC", "/opt/rocm/bin/hipcc"), *FLAGS, SRC, "-o", tmp],
                   check=True, capture_output=True, text=True)
    os.replace(tmp, LIB)
    return LIB


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(LIB):
            raise ImportError(f"{LIB} is not built; run __graft_entry__.build()")
        L = ctypes.CDLL(LIB)
        P, I64, F, I, U32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_float, ctypes.c_int, ctypes.c_uint32
        L.probe_cvt_range.argtypes = [U32, I64, P, P]
        L.probe_cvt_list.argtypes = [P, I64, P, F, I, I, P]
        L.probe_exp2.argtypes = [P, I64, P, P]
        L.probe_mfma.argtypes = [I, P, P, P, P]
        L.probe_mfma_fp8_scaled.argtypes = [P, P, P, P, P, P]
        L.probe_cvt_scaled_vec.argtypes = [P, P, I64, P, P]
        L.probe_exp2_rate.argtypes = [I, I, P, P]
        L.probe_lds_rate.argtypes = [I, I, I, I, I, P, P, P, P]
        L.probe_coexec.argtypes = [I, I, I, I, P, P, P]
        for f in (L.probe_cvt_range, L.probe_cvt_list, L.probe_exp2, L.probe_mfma,
                  L.probe_mfma_fp8_scaled, L.probe_cvt_scaled_vec, L.probe_exp2_rate,
                  L.probe_lds_rate, L.probe_coexec):
            f.restype = I
        _lib = L
    return _lib
