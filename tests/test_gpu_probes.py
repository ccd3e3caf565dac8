"""Hardware facts the parity argument rests on (gfx950), checked against the
CPU oracle or exact host arithmetic:

- the E4M3 convert is OCP E4M3 (bias 7, max 448) with round-to-nearest-even,
  bit-identical to the oracle's encoder on every non-negative FP32 input below
  464 (the whole range P*S can take for S <= 448);
- the scaled convert with scale 2^-k equals the plain convert of x * 2^k;
- v_exp_f32 is exact at integers and monotone around them, so for S = 2^k the
  zero-code decision is x <= -(10 + k) on both sides;
- the MFMA operand / accumulator lane layouts the kernels assume;
- how the matrix cores add products: the FP8 MFMA sums groups of eight
  consecutive products aligned to the group's largest one and drops what lies
  more than 13 bits below it (toward zero); the bf16 MFMA keeps 23 bits below
  its largest product.  On the seeded inputs both are exact, which is what
  makes the scores identical to the oracle's exact dot products.
"""
import numpy as np
import pytest
import torch

import oracle

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def probes():
    from tests import probes as pr
    return pr.lib()


def _stream():
    return torch.cuda.current_stream().cuda_stream


def test_cvt_exhaustive_nonnegative_below_464(probes):
    hi = int(np.float32(464.0).view(np.uint32))
    chunk = 1 << 26
    out = torch.empty(chunk, dtype=torch.uint8, device="cuda")
    for lo in range(0, hi, chunk):
        n = min(chunk, hi - lo)
        assert probes.probe_cvt_range(lo, n, out.data_ptr(), _stream()) == 0
        got = out[:n].cpu().numpy()
        want = oracle.e4m3_encode(np.arange(lo, lo + n, dtype=np.uint32).view(np.float32))
        bad = np.nonzero(got != want)[0]
        assert bad.size == 0, [(hex(lo + int(i)), int(got[i]), int(want[i])) for i in bad[:8]]


def test_cvt_negative_and_specials(probes):
    rng = np.random.default_rng(5)
    neg = -np.abs(rng.standard_normal(1 << 20).astype(np.float32) * 50)
    neg = neg[neg > -448]
    x = np.concatenate([neg, np.float32([2.0 ** -10, 2.0 ** -9, 7.5 * 2.0 ** -9, 448, 0.0, -0.0])])
    if x.size % 2:
        x = np.append(x, np.float32(1.0))
    xt = torch.from_numpy(x).cuda()
    out = torch.empty(x.size, dtype=torch.uint8, device="cuda")
    assert probes.probe_cvt_list(xt.data_ptr(), x.size, out.data_ptr(), 1.0, 0, 0, _stream()) == 0
    assert np.array_equal(out.cpu().numpy(), oracle.e4m3_encode(x))
    # the high-word form writes the same codes into bytes 2..3
    assert probes.probe_cvt_list(xt.data_ptr(), x.size, out.data_ptr(), 1.0, 0, 1, _stream()) == 0
    assert np.array_equal(out.cpu().numpy(), oracle.e4m3_encode(x))


@pytest.mark.parametrize("k", [0, 4, 8])
def test_scaled_cvt_equals_cvt_of_scaled(probes, k):
    rng = np.random.default_rng(6 + k)
    P = np.concatenate([rng.uniform(0, 1, 1 << 20), np.exp2(rng.uniform(-40, 0, 1 << 20)),
                        2.0 ** -np.arange(0, 40), [1.0, 0.0]]).astype(np.float32)
    if P.size % 2:
        P = np.append(P, np.float32(0.5))
    S = np.float32(2.0 ** k)
    Pt = torch.from_numpy(P).cuda()
    out = torch.empty(P.size, dtype=torch.uint8, device="cuda")
    for hi in (0, 1):
        assert probes.probe_cvt_list(Pt.data_ptr(), P.size, out.data_ptr(), float(1 / S), 1, hi, _stream()) == 0
        assert np.array_equal(out.cpu().numpy(), oracle.e4m3_encode(P * S)), hi


def test_exp2_exact_at_integers_and_monotone(probes):
    """For S = 2^k the zero-code threshold is x = -(10 + k); with |x| >= 8 one
    FP32 step of x moves 2^x by more than 5 ulps, so the hardware result must
    sit strictly on the correct side of 2^n for every neighbour of n."""
    ints = np.arange(-126, 1, dtype=np.float32)
    nb = []
    for n in range(-40, -7):
        c = np.float32(n).view(np.uint32)
        # negative floats: a larger bit pattern is more negative
        nb.append(np.arange(c - 256, c + 257, dtype=np.uint32).view(np.float32))
    x = np.concatenate([ints] + nb).astype(np.float32)
    xt = torch.from_numpy(x).cuda()
    out = torch.empty_like(xt)
    assert probes.probe_exp2(xt.data_ptr(), x.size, out.data_ptr(), _stream()) == 0
    y = out.cpu().numpy().astype(np.float64)
    xi = x.astype(np.float64)
    assert np.array_equal(y[:ints.size], np.exp2(ints.astype(np.float64)))
    rest_x, rest_y = xi[ints.size:], y[ints.size:]
    n = np.round(rest_x)
    below, above = rest_x < n, rest_x > n
    assert np.all(rest_y[below] < np.exp2(n[below]))
    assert np.all(rest_y[above] > np.exp2(n[above]))


def test_exp2_accuracy(probes):
    rng = np.random.default_rng(7)
    x = rng.uniform(-60, 0.001, 1 << 22).astype(np.float32)
    xt = torch.from_numpy(x).cuda()
    out = torch.empty_like(xt)
    assert probes.probe_exp2(xt.data_ptr(), x.size, out.data_ptr(), _stream()) == 0
    y = out.cpu().numpy()
    ref = np.exp2(x.astype(np.float64))
    ulp = np.spacing(ref.astype(np.float32)).astype(np.float64)
    err = np.abs(y.astype(np.float64) - ref) / ulp
    assert err.max() <= 2.0, err.max()


def test_exp2_issue_rate(probes):
    """Chip-wide v_exp_f32 rate, the exp2 peak the benchmark reports the
    attention kernels against: 2048 workgroups x 256 lanes x 16 independent
    chains x 4096 rounds, timed with events on the launch stream (median of
    five launches).  The results must be finite and each lane's sum of its 16
    chains in [8, 16]."""
    blocks, iters, chains = 2048, 4096, 16
    out = torch.empty(blocks * 256, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()
    assert probes.probe_exp2_rate(blocks, 64, out.data_ptr(), s.cuda_stream) == 0   # warm-up
    times = []
    for _ in range(5):
        e0, e1 = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
        e0.record(s)
        assert probes.probe_exp2_rate(blocks, iters, out.data_ptr(), s.cuda_stream) == 0
        e1.record(s)
        torch.cuda.synchronize()
        times.append(e0.elapsed_time(e1) / 1e3)
    sec = float(np.median(times))
    rate = blocks * 256 * iters * chains / sec
    y = out.cpu().numpy()
    assert np.all(np.isfinite(y)) and y.min() >= 8.0 and y.max() <= 16.0
    print(f"v_exp_f32 issue rate: {rate:.4e} exp2/s ({sec * 1e3:.3f} ms per launch)", flush=True)
    # between 1/64 and 1 evaluation per lane per cycle at 2.4 GHz on 256 CUs
    assert 256 * 256 * 2.4e9 / 64 < rate < 256 * 256 * 2.4e9


def test_lds_read_rate(probes):
    """LDS read rate of one CU, in bytes per shader cycle (s_memtime), for the
    two reads of the fast kernel's MFMA phase: ds_read_b128 (the K operand)
    and ds_read_b64_tr_b8 (the transposed V operand).  8 reader waves, then 4
    reader waves alone and beside 4 waves that copy global memory into LDS
    with global_load_lds_dwordx4 (the stage copies).  One workgroup per CU,
    256 workgroups; the median over workgroups of (bytes read / the slowest
    reader's cycles).  The ds_read_b128 checksums are compared with the host."""
    blocks, iters = 256, 2049
    cyc = torch.zeros(blocks * 8, dtype=torch.int64, device="cuda")
    sink = torch.zeros(blocks * 512, dtype=torch.int32, device="cuda")
    src = torch.zeros(65536, dtype=torch.uint8, device="cuda")
    s = torch.cuda.current_stream()
    words = (np.arange(16384, dtype=np.uint64) * 2654435761) % (1 << 32)
    res = {}
    for mode, readers, copiers in [(0, 8, 0), (1, 8, 0), (0, 4, 0), (0, 4, 4), (1, 4, 0), (1, 4, 4)]:
        assert probes.probe_lds_rate(blocks, 64, mode, readers, copiers, src.data_ptr(), cyc.data_ptr(),
                                     sink.data_ptr(), s.cuda_stream) == 0   # warm-up
        assert probes.probe_lds_rate(blocks, iters, mode, readers, copiers, src.data_ptr(), cyc.data_ptr(),
                                     sink.data_ptr(), s.cuda_stream) == 0
        torch.cuda.synchronize()
        c = cyc.cpu().numpy().reshape(blocks, 8)[:, :readers].max(axis=1).astype(np.float64)
        per_instr = 1024 if mode == 0 else 512
        rate = float(np.median(readers * iters * 8 * per_instr / c))
        res[(mode, readers, copiers)] = rate
        print(f"LDS {'ds_read_b128' if mode == 0 else 'ds_read_b64_tr_b8'}: {readers} reader waves, "
              f"{copiers} copier waves: {rate:.1f} B/cycle per CU", flush=True)
        assert 16.0 < rate < 1024.0
        if mode == 0:
            # an odd number of rounds leaves one round's XOR in every lane
            got = sink.cpu().numpy().view(np.uint32).reshape(blocks, 8, 64)
            for w in range(readers):
                lanes = np.arange(64)
                idx = [(w * 8192 + 16 * lanes + 1024 * k) // 4 + (k % 4) for k in range(8)]
                want = np.bitwise_xor.reduce(np.stack([words[i] for i in idx]), axis=0).astype(np.uint32)
                assert np.all(got[:, w, :] == want[None, :]), w



def test_mfma_valu_coexec(probes):
    """How one SIMD's matrix core and vector ALU overlap, in shader cycles per
    iteration (s_memtime, median over 256 workgroups of the slowest wave of a
    kind).  The vector stream is the softmax's instruction mix of one wave and
    128-key block.  Matrix streams of 1536 cycles at the documented rates:
    pattern 0 is the fast kernel's matrix work per wave-block (32 bf16
    32x32x16 + 8 FP8 32x32x64), 1 is 24 FP8 32x32x64, 2 is 48 bf16 32x32x16,
    3 is 96 bf16 16x16x32.  Layouts: each stream alone (one wave per SIMD);
    the fast kernel's ping-pong (an MFMA wave and a vector wave on every SIMD);
    one wave per SIMD running pattern 0 and the vector stream.  Every matrix
    stream alone pins the 1536-cycle cost (the three shapes' rates); the vector
    wave's slowdown beside each pattern is reported per MFMA instruction."""
    blocks, iters = 256, 1001
    cyc = torch.zeros(blocks * 8, dtype=torch.int64, device="cuda")
    sink = torch.zeros(blocks * 512, dtype=torch.float32, device="cuda")
    s = torch.cuda.current_stream()

    def run(layout, pattern):
        cyc.zero_()
        assert probes.probe_coexec(blocks, 8, layout, pattern, cyc.data_ptr(), sink.data_ptr(),
                                   s.cuda_stream) == 0
        assert probes.probe_coexec(blocks, iters, layout, pattern, cyc.data_ptr(), sink.data_ptr(),
                                   s.cuda_stream) == 0
        torch.cuda.synchronize()
        c = cyc.cpu().numpy().reshape(blocks, 8).astype(np.float64) / iters
        nw = 8 if layout == 2 else 4
        assert np.all(c[:, :nw] > 0)
        assert np.all(np.isfinite(sink.cpu().numpy().reshape(blocks, 512)[:, :64 * nw]))
        return (float(np.median(c[:, :4].max(axis=1))),
                float(np.median(c[:, 4:8].max(axis=1))) if layout == 2 else None)

    valu = run(1, 0)[0]
    one = run(3, 0)[0]
    n_instr = {0: 40, 1: 24, 2: 48, 3: 96}
    for pattern in range(4):
        mfma = run(0, pattern)[0]
        split_m, split_v = run(2, pattern)
        per = (split_v - valu) / n_instr[pattern]
        print(f"pattern {pattern}: matrix stream alone {mfma:.0f} cycles/iteration, vector stream alone "
              f"{valu:.0f}; ping-pong: MFMA wave {split_m:.0f}, vector wave {split_v:.0f} "
              f"({100 * (split_v / valu - 1):+.1f} %, {per:.1f} cycles per MFMA instruction)", flush=True)
        assert 1536 * 0.98 < mfma < 1536 * 1.1
        assert split_m >= 0.95 * mfma and split_v >= 0.95 * valu
    print(f"one wave per SIMD running pattern 0 and the vector stream: {one:.0f}", flush=True)
    assert one >= 0.95 * max(1536, valu)

def test_mfma_bf16_layout(probes):
    rng = np.random.default_rng(8)
    A = rng.integers(-8, 9, (32, 16)).astype(np.float32)
    B = rng.integers(-8, 9, (16, 32)).astype(np.float32)
    At = torch.from_numpy(A).to(torch.bfloat16).cuda()
    Bt = torch.from_numpy(B).to(torch.bfloat16).cuda()
    D = torch.zeros((32, 32), dtype=torch.float32, device="cuda")
    assert probes.probe_mfma(0, At.data_ptr(), Bt.data_ptr(), D.data_ptr(), _stream()) == 0
    assert np.array_equal(D.cpu().numpy(), A @ B)


def test_mfma_fp8_layout(probes):
    rng = np.random.default_rng(9)
    A = rng.integers(-8, 9, (32, 64)).astype(np.float32) / 4
    B = rng.integers(-8, 9, (64, 32)).astype(np.float32) / 8
    Ac = torch.from_numpy(A).to(torch.float8_e4m3fn).view(torch.uint8).cuda()
    Bc = torch.from_numpy(B).to(torch.float8_e4m3fn).view(torch.uint8).cuda()
    D = torch.zeros((32, 32), dtype=torch.float32, device="cuda")
    assert probes.probe_mfma(1, Ac.data_ptr(), Bc.data_ptr(), D.data_ptr(), _stream()) == 0
    assert np.array_equal(D.cpu().numpy(), A @ B)


def test_mfma_f32_layout(probes):
    rng = np.random.default_rng(10)
    A = rng.integers(-8, 9, (32, 2)).astype(np.float32)
    B = rng.integers(-8, 9, (2, 32)).astype(np.float32)
    At, Bt = torch.from_numpy(A).cuda(), torch.from_numpy(B).cuda()
    D = torch.zeros((32, 32), dtype=torch.float32, device="cuda")
    assert probes.probe_mfma(2, At.data_ptr(), Bt.data_ptr(), D.data_ptr(), _stream()) == 0
    assert np.array_equal(D.cpu().numpy(), A @ B)


def test_mfma_fp8_block_scales_per_lane(probes):
    """Block scales of the FP8 MFMA (byte 0 of each lane's scale operand):
    lane m + 32 g (g = 0, 1) scales row m of A (column m of B) at the K
    positions k with (k mod 32) div 16 == g, i.e. the first 16 operand
    elements of both lanes of the row take lane m's scale and the last 16
    take lane m + 32's.  The dynamic P-scale gives both lanes of a query row
    the same byte, so the whole column of P of that row is scaled by it."""
    rng = np.random.default_rng(11)
    A = rng.integers(-8, 9, (32, 64)).astype(np.float32) / 4
    B = rng.integers(-8, 9, (64, 32)).astype(np.float32) / 8
    sa = rng.integers(120, 135, 64).astype(np.uint8)
    sb = rng.integers(100, 128, 64).astype(np.uint8)
    k = np.arange(64)
    g = (k % 32) // 16
    As = A * np.exp2(sa[np.arange(32)[:, None] + 32 * g[None, :]].astype(np.float64) - 127)
    Bs = B * np.exp2(sb[np.arange(32)[None, :] + 32 * g[:, None]].astype(np.float64) - 127)

    def run(sa_, sb_):
        Ac = torch.from_numpy(A).to(torch.float8_e4m3fn).view(torch.uint8).cuda()
        Bc = torch.from_numpy(B).to(torch.float8_e4m3fn).view(torch.uint8).cuda()
        sat, sbt = torch.from_numpy(sa_).cuda(), torch.from_numpy(sb_).cuda()
        D = torch.zeros((32, 32), dtype=torch.float32, device="cuda")
        assert probes.probe_mfma_fp8_scaled(Ac.data_ptr(), Bc.data_ptr(), sat.data_ptr(),
                                            sbt.data_ptr(), D.data_ptr(), _stream()) == 0
        return D.cpu().numpy().astype(np.float64)

    got = run(sa, sb)
    want = As @ Bs
    # FP32 accumulation of 64 terms: within 64 ulps of the sum of magnitudes
    bound = (np.abs(As) @ np.abs(Bs)) * 64 * 2.0 ** -24
    assert np.all(np.abs(got - want) <= bound), np.abs(got - want).max()
    # the kernel's use: one byte per column of B, in both of its lanes
    col = rng.integers(9, 128, 32).astype(np.uint8)
    got = run(np.full(64, 127, np.uint8), np.concatenate([col, col]))
    want = A.astype(np.float64) @ (B * np.exp2(col.astype(np.float64) - 127)[None, :])
    bound = (np.abs(A) @ np.abs(B * np.exp2(col.astype(np.float64) - 127)[None, :])) * 64 * 2.0 ** -24
    assert np.all(np.abs(got - want) <= bound)


@pytest.mark.parametrize("kmax", [8, 40, 126])
def test_scaled_cvt_per_element_power_of_two(probes, kmax):
    """The dynamic P-scale casts P * 2^kj with kj up to 126 through the scaled
    convert (scale 2^-kj, one per lane): bit-equal to the cast of the exact
    product, for products in the range the rule produces (at most S = 2^8)."""
    rng = np.random.default_rng(12 + kmax)
    n = 1 << 20
    k = rng.integers(0, kmax + 1, n // 2).repeat(2)
    # P * 2^k in (0, 256]: P = 2^(u - k) with u in [-20, 8]
    u = rng.uniform(-20, 8, n)
    P = np.exp2(u - k).astype(np.float32)
    P[::97] = np.float32(0.0)
    scale = np.exp2(-k.astype(np.float64)).astype(np.float32)
    xt, st = torch.from_numpy(P).cuda(), torch.from_numpy(scale).cuda()
    out = torch.empty(n, dtype=torch.uint8, device="cuda")
    assert probes.probe_cvt_scaled_vec(xt.data_ptr(), st.data_ptr(), n, out.data_ptr(), _stream()) == 0
    exact = (P.astype(np.float64) * np.exp2(k)).astype(np.float32)
    assert np.all(exact.astype(np.float64) == P.astype(np.float64) * np.exp2(k))
    assert np.array_equal(out.cpu().numpy(), oracle.e4m3_encode(exact))


def _fp8_dot(probes, A, B):
    Ac = torch.from_numpy(np.ascontiguousarray(A, np.float32)).to(torch.float8_e4m3fn)
    Bc = torch.from_numpy(np.ascontiguousarray(B, np.float32)).to(torch.float8_e4m3fn)
    assert np.array_equal(Ac.float().numpy(), A) and np.array_equal(Bc.float().numpy(), B)
    D = torch.zeros((32, 32), dtype=torch.float32, device="cuda")
    assert probes.probe_mfma(1, Ac.view(torch.uint8).cuda().data_ptr(),
                             Bc.view(torch.uint8).cuda().data_ptr(), D.data_ptr(), _stream()) == 0
    return D.cpu().numpy().astype(np.float64)


def _bf16_dot(probes, A, B):
    At = torch.from_numpy(np.ascontiguousarray(A, np.float32)).to(torch.bfloat16)
    Bt = torch.from_numpy(np.ascontiguousarray(B, np.float32)).to(torch.bfloat16)
    assert np.array_equal(At.float().numpy(), A) and np.array_equal(Bt.float().numpy(), B)
    D = torch.zeros((32, 32), dtype=torch.float32, device="cuda")
    assert probes.probe_mfma(0, At.cuda().data_ptr(), Bt.cuda().data_ptr(), D.data_ptr(),
                             _stream()) == 0
    return D.cpu().numpy().astype(np.float64)


def _two_products(K, big, i, small):
    """A, B (power-of-two entries, E4M3 and bf16 exact) whose dot in every
    output is big (channel 0) + small (channel i)."""
    A = np.zeros((32, K), np.float32)
    B = np.zeros((K, 32), np.float32)
    for ch, v in ((0, big), (i, small)):
        e = int(np.log2(abs(v)))
        ea = max(e // 2, -9)
        A[:, ch] = np.sign(v) * 2.0 ** ea
        B[ch, :] = 2.0 ** (e - ea)
    return A, B


@pytest.mark.parametrize("big_exp", [0, 4])
def test_mfma_fp8_groups_of_eight_truncate_13_bits_below(probes, big_exp):
    big = 2.0 ** big_exp
    for i in range(1, 64):
        for f, sign in ((13, 1.0), (14, 1.0), (14, -1.0)):
            small = sign * 2.0 ** (big_exp - f)
            got = _fp8_dot(probes, *_two_products(64, big, i, small))
            kept = f <= 13 or i >= 8
            want = big + small if kept else big
            assert np.all(got == want), (big_exp, i, f, sign, got[0, 0])


def test_mfma_bf16_keeps_23_bits_below(probes):
    for i in (1, 8, 15):
        assert np.all(_bf16_dot(probes, *_two_products(16, 1.0, i, 2.0 ** -23)) == 1.0 + 2.0 ** -23)
        assert np.all(_bf16_dot(probes, *_two_products(16, 1.0, i, 2.0 ** -24)) == 1.0)


@pytest.mark.parametrize("d", [64, 128])
def test_matrix_core_dots_exact_on_seeded_inputs(probes, d):
    from paper_2606_06521_amd.inputs import make_inputs
    for fmt, K, dot in (("e4m3", 64, _fp8_dot), ("bf16_e4m3", 16, _bf16_dot)):
        inp = make_inputs(1, 1, 1, 96, d, fmt=fmt, delta=9.0, seed=40 + d)
        q, k = inp.q32[0, 0], inp.k32[0, 0]
        # keys 0..31 hold the sink offset (n_sink = 4) and the rest; every
        # K-wide slice of the channels, including the sink channels at the end
        for c0 in range(0, d, K):
            for r0 in (0, 32, 64):
                A = q[r0:r0 + 32, c0:c0 + K]
                B = k[0:32, c0:c0 + K].T
                got = dot(probes, A, B)
                assert np.array_equal(got, A.astype(np.float64) @ B.astype(np.float64)), (fmt, c0, r0)
