"""The C ABI on the host (no GPU needed): the library loads, exports every
symbol include/attn_fp8.h declares, and rejects bad arguments before any HIP
call is made."""
import ctypes
import os
import re

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "attn_fp8.h")


@pytest.fixture(scope="module")
def A():
    from paper_2606_06521_amd import attn_fp8
    return attn_fp8


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(attn_fp8_\w+)\s*\(", text)))


def test_exports_every_declared_symbol(A):
    names = declared_functions()
    assert names == ["attn_fp8_block_gap_diag", "attn_fp8_fwd", "attn_fp8_fwd_descaled",
                     "attn_fp8_fwd_kv", "attn_fp8_fwd_kv_noalloc", "attn_fp8_kv_workspace_bytes",
                     "attn_fp8_p_underflow_count",
                     "attn_fp8_p_underflow_count_descaled", "attn_fp8_p_underflow_count_kv",
                     "attn_fp8_strerror", "attn_fp8_version"]
    lib = ctypes.CDLL(A.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), n


def test_version_and_strerror(A):
    assert A.attn_fp8_version() >= 100
    for st in (A.ATTN_OK, A.ATTN_ERR_INVALID_ARG, A.ATTN_ERR_UNSUPPORTED, A.ATTN_ERR_HIP,
               A.ATTN_ERR_SCRATCH, 12345):
        assert isinstance(A.attn_fp8_strerror(st), str) and A.attn_fp8_strerror(st)


def test_enum_values_match_header(A):
    text = open(HEADER).read()
    for name in ["ATTN_MODE_FAITHFUL", "ATTN_MODE_FAST", "ATTN_MODE_NOCAST", "ATTN_MODE_FP8QK",
                 "ATTN_ORDER_FORWARD",
                 "ATTN_ORDER_REVERSE", "ATTN_OK", "ATTN_ERR_INVALID_ARG", "ATTN_ERR_UNSUPPORTED",
                 "ATTN_ERR_HIP", "ATTN_ERR_SCRATCH"]:
        m = re.search(name + r"\s*=\s*(-?\d+)", text)
        assert m and int(m.group(1)) == getattr(A, name), name
    for name in ["ATTN_SCALE_DYNAMIC", "ATTN_TILE_256", "ATTN_TILE_128"]:
        m = re.search(name + r"\s*=\s*(0x[0-9a-fA-F]+)", text)
        assert m and int(m.group(1), 16) == getattr(A, name), name


FAKE = 0x1000   # never dereferenced: every case below fails validation first


def fwd(A, **kw):
    a = dict(q=FAKE, k=FAKE, v=FAKE, out=FAKE, lse=None, B=1, Hq=4, Hkv=2, N=128, d=128, causal=1,
             block_kv=128, order=1, S=256.0, mode=1, stream=None)
    a.update(kw)
    return A.attn_fp8_fwd(a["q"], a["k"], a["v"], a["out"], a["lse"], a["B"], a["Hq"], a["Hkv"],
                          a["N"], a["d"], a["causal"], a["block_kv"], a["order"], a["S"], a["mode"],
                          a["stream"])


@pytest.mark.parametrize("kw,status", [
    (dict(q=None), -1), (dict(k=None), -1), (dict(v=None), -1), (dict(out=None), -1),
    (dict(Hkv=3), -1), (dict(Hq=0), -1), (dict(B=-1), -1), (dict(N=-5), -1),
    (dict(causal=2), -1), (dict(order=2), -1), (dict(mode=4), -1), (dict(mode=-1), -1),
    (dict(S=0.0), -1), (dict(S=-1.0), -1), (dict(S=float("inf")), -1), (dict(S=float("nan")), -1),
    (dict(d=96), -2), (dict(d=256), -2), (dict(block_kv=32), -2), (dict(block_kv=256), -2),
    (dict(d=0), -1), (dict(N=(1 << 30) + 1), -2),
    # the dynamic scale needs S = 2^k0 with 0 <= k0 <= 8; at most one ATTN_TILE_* flag;
    # no other flag bit exists
    (dict(mode=1 | 0x100, S=3.0), -1), (dict(mode=1 | 0x100, S=512.0), -1),
    (dict(mode=0 | 0x100, S=0.5), -1), (dict(mode=1 | 0x600), -1), (dict(mode=1 | 0x800), -1),
    (dict(mode=1 | 0x80), -1),
])
def test_fwd_rejects_bad_arguments(A, kw, status):
    assert fwd(A, **kw) == status


def test_empty_problems_return_ok_without_touching_pointers(A):
    assert fwd(A, N=0, q=None, k=None, v=None, out=None) == 0
    assert fwd(A, B=0, q=None, k=None, v=None, out=None) == 0


def test_count_rejects_bad_arguments(A):
    def cnt(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, B=1, Hq=2, Hkv=1, N=64, d=64, causal=0, block_kv=64,
                 order=0, S=1.0, mode=0, n_sink=4, counts=FAKE, out=None, lse=None, stream=None)
        a.update(kw)
        return A.attn_fp8_p_underflow_count(a["q"], a["k"], a["v"], a["B"], a["Hq"], a["Hkv"],
                                            a["N"], a["d"], a["causal"], a["block_kv"], a["order"],
                                            a["S"], a["mode"], a["n_sink"], a["counts"], a["out"],
                                            a["lse"], a["stream"])
    assert cnt(counts=None) == -1
    assert cnt(n_sink=-1) == -1
    # sink keys beyond block 0 would fall in two count categories at once
    assert cnt(n_sink=64 + 8) == -1
    assert cnt(n_sink=64 + 8, block_kv=128, N=0, counts=None) == 0
    assert cnt(d=32) == -2
    assert cnt(N=0, counts=None) == 0


def test_binding_checks_dtypes_before_calling(A):
    import torch
    q = torch.zeros((1, 1, 4, 64), dtype=torch.float32)
    with pytest.raises(ValueError):
        A.fwd(q, q, q, mode="faithful")          # host tensors are refused


def test_descaled_entry_points_validate_descales(A):
    base = dict(q=FAKE, k=FAKE, v=FAKE, out=FAKE, lse=None, B=1, Hq=2, Hkv=1, N=64, d=64,
                causal=0, block_kv=64, order=0, S=1.0, mode=3)

    def f(qd, kd, vd, **kw):
        a = dict(base, **kw)
        return A.attn_fp8_fwd_descaled(a["q"], a["k"], a["v"], a["out"], a["lse"], a["B"],
                                       a["Hq"], a["Hkv"], a["N"], a["d"], a["causal"],
                                       a["block_kv"], a["order"], a["S"], a["mode"], qd, kd, vd,
                                       None)
    for bad in (0.0, -1.0, float("inf"), float("nan")):
        assert f(bad, 1.0, 1.0) == -1
        assert f(1.0, bad, 1.0) == -1
        assert f(1.0, 1.0, bad) == -1
    assert f(1.0, 1.0, 1.0, N=0, q=None, k=None, v=None, out=None) == 0
    cnt = A.attn_fp8_p_underflow_count_descaled(FAKE, FAKE, FAKE, 1, 2, 1, 64, 64, 0, 64, 0, 1.0, 3,
                                                4, 1.0, -2.0, 1.0, FAKE, None, None, None)
    assert cnt == -1


def test_block_gap_diag_validates_before_any_launch(A):
    def g(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, B=1, Hq=2, Hkv=1, N=64, d=64, causal=0, block_kv=64,
                 order=0, S=256.0, mode=1, n_sink=4, qd=1.0, kd=1.0, vd=1.0, nbins=16,
                 hist=FAKE, bz=FAKE, counts=FAKE)
        a.update(kw)
        return A.attn_fp8_block_gap_diag(a["q"], a["k"], a["v"], a["B"], a["Hq"], a["Hkv"],
                                         a["N"], a["d"], a["causal"], a["block_kv"], a["order"],
                                         a["S"], a["mode"], a["n_sink"], a["qd"], a["kd"],
                                         a["vd"], a["nbins"], a["hist"], a["bz"], a["counts"],
                                         None, None, None)
    for bad in (0, 65, -3):
        assert g(nbins=bad) == -1
    assert g(hist=None) == -1
    assert g(bz=None) == -1
    assert g(counts=None) == -1
    assert g(qd=0.0) == -1
    assert g(d=32) == -2
    assert g(N=0, q=None, k=None, v=None, hist=None, bz=None, counts=None) == 0


def test_kv_entry_points_validate(A):
    def f(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, out=FAKE, B=1, Hq=2, Hkv=1, Nq=32, Nk=4096, d=128,
                 causal=1, block_kv=128, order=1, S=256.0, mode=1)
        a.update(kw)
        return A.attn_fp8_fwd_kv(a["q"], a["k"], a["v"], a["out"], None, a["B"], a["Hq"],
                                 a["Hkv"], a["Nq"], a["Nk"], a["d"], a["causal"], a["block_kv"],
                                 a["order"], a["S"], a["mode"], 1.0, 1.0, 1.0, a.get("ws"),
                                 a.get("ws_bytes", 0), None)
    assert f(Nq=4097) == -1            # more queries than keys
    assert f(Nk=-1) == -1
    assert f(Nk=(1 << 30) + 1) == -2   # key positions must stay well inside int
    assert f(out=None) == -1
    assert f(d=96) == -2
    assert f(Nq=0, q=None, k=None, v=None, out=None) == 0
    assert f(ws=FAKE + 16, ws_bytes=1 << 20) == -1     # workspace not 256-byte aligned
    cnt = A.attn_fp8_p_underflow_count_kv(FAKE, FAKE, FAKE, 1, 2, 1, 32, 4096, 128, 1, 128, 1,
                                          256.0, 1, 4, 1.0, 1.0, 1.0, None, None, None, None, 0,
                                          None)
    assert cnt == -1
    cnt = A.attn_fp8_p_underflow_count_kv(FAKE, FAKE, FAKE, 1, 2, 1, 32, 4096, 128, 1, 128, 1,
                                          256.0, 1, 129, 1.0, 1.0, 1.0, FAKE, None, None, None, 0,
                                          None)
    assert cnt == -1                   # n_sink > block_kv


def test_noalloc_entry_point_validates(A):
    def f(**kw):
        a = dict(q=FAKE, k=FAKE, v=FAKE, out=FAKE, B=1, Hq=2, Hkv=1, Nq=32, Nk=4096, d=128,
                 causal=1, block_kv=128, order=1, S=256.0, mode=1)
        a.update(kw)
        return A.attn_fp8_fwd_kv_noalloc(a["q"], a["k"], a["v"], a["out"], None, a["B"], a["Hq"],
                                         a["Hkv"], a["Nq"], a["Nk"], a["d"], a["causal"],
                                         a["block_kv"], a["order"], a["S"], a["mode"], 1.0, 1.0,
                                         1.0, None)
    assert f(Nq=4097) == -1
    assert f(out=None) == -1
    assert f(q=FAKE + 8) == -1
    assert f(d=96) == -2
    assert f(Nq=0, q=None, k=None, v=None, out=None) == 0


def test_kv_workspace_query_validates(A):
    import ctypes
    assert A._lib.attn_fp8_kv_workspace_bytes(1, 2, 1, 32, 4096, 128, 1, 128, 1, None) == -1
    assert A.attn_fp8_kv_workspace_bytes(1, 2, 1, 33, 32, 128, 1, 128, 1)[0] == -1   # Nq > Nk
    assert A.attn_fp8_kv_workspace_bytes(1, 2, 1, 32, 4096, 96, 1, 128, 1)[0] == -2
    # no split without a kernel that splits: square problems, faithful mode, empty problems
    assert A.attn_fp8_kv_workspace_bytes(1, 2, 1, 64, 64, 128, 1, 128, 1) == (0, 0)
    assert A.attn_fp8_kv_workspace_bytes(1, 2, 1, 32, 4096, 128, 1, 128, 0) == (0, 0)
    assert A.attn_fp8_kv_workspace_bytes(0, 2, 1, 32, 4096, 128, 1, 128, 1) == (0, 0)


def test_misaligned_pointers_are_rejected(A):
    base = 1 << 20
    def f(**kw):
        a = dict(q=base, k=base, v=base, out=base, lse=None, mode=1)
        a.update(kw)
        return A.attn_fp8_fwd(a["q"], a["k"], a["v"], a["out"], a["lse"], 1, 2, 1, 64, 64, 0, 64, 0,
                              256.0, a["mode"], None)
    assert f(q=base + 8) == -1
    assert f(k=base + 2) == -1
    assert f(v=base + 1) == -1
    assert f(out=base + 4) == -1
    assert f(lse=base + 2) == -1
    cnt = A.attn_fp8_p_underflow_count(base, base, base, 1, 2, 1, 64, 64, 0, 64, 0, 256.0, 1, 4,
                                       base + 1, None, None, None)
    assert cnt == -1


def test_header_is_plain_c_and_links(A, tmp_path):
    # a C99 program that includes the header, links the library and calls the
    # entry points that need no GPU (version, strerror, a validation error)
    import shutil
    import subprocess
    gcc = shutil.which("gcc")
    if gcc is None:
        pytest.skip("no C compiler")
    src = tmp_path / "use_abi.c"
    src.write_text(r'''
#include <stdio.h>
#include "attn_fp8.h"
int main(void) {
    int st = attn_fp8_fwd(0, 0, 0, 0, 0, -1, 1, 1, 8, 64, 0, 64, 0, 256.0f, 1, 0);
    printf("%d %d %s\n", attn_fp8_version(), st == ATTN_ERR_INVALID_ARG, attn_fp8_strerror(st));
    return st == ATTN_ERR_INVALID_ARG ? 0 : 1;
}
''')
    exe = tmp_path / "use_abi"
    libdir = os.path.dirname(A.LIB_PATH)
    subprocess.run([gcc, "-std=c99", "-Wall", "-Werror", "-pedantic-errors", "-I", os.path.join(ROOT, "include"),
                    str(src), "-o", str(exe), "-L", libdir, "-lattn_fp8", "-Wl,-rpath," + libdir],
                   check=True, capture_output=True, text=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stdout + r.stderr
    version, rejected, _ = r.stdout.split(" ", 2)
    assert int(version) == A.attn_fp8_version() and rejected == "1"
