"""Throughput benchmark of the FP8 attention forward on one MI355X.

One step = one attn_fp8_fwd call over the whole workload (every query row of
every batch and head: QK^T, online softmax over the KV blocks in the chosen
order, E4M3 P-cast, P.V, epilogue).  Inputs are seeded synthetic sink-shaped
tensors already resident in HBM when the timed region starts.

Prints ONE JSON line:
  value      whole-job TFLOP/s (FlashAttention convention 4*B*H*N^2*d, halved
             under causal masking) over K timed steps bracketed by device syncs;
  roofline   the attention kernel's algorithmic FLOPs per launch divided by the
             median of its launch times from HIP events on its stream, against the
             dense FP8 MFMA peak (and, for reference, the mixed bf16+FP8 peak
             this kernel's instruction mix can reach);
  cpu_baseline  the CPU oracle timed on a bounded row sample of the same
             workload (rank 0 only), plus the P-cast MSE of the GPU and of the
             oracle against FP64 attention on those rows.
"""
from __future__ import annotations

import argparse
import hashlib
import json
import os
import sys
import time

ROOT = os.path.dirname(os.path.abspath(__file__))
if ROOT not in sys.path:
    sys.path.insert(0, ROOT)

PEAK_TFLOPS = {"fp8": 5000.0, "bf16": 2500.0}
# half of the FLOPs (QK^T) run on the bf16 MFMA, half (P.V) on the FP8 MFMA
MIXED_PEAK = 2.0 / (1.0 / PEAK_TFLOPS["bf16"] + 1.0 / PEAK_TFLOPS["fp8"])
# the arithmetic type of each mode's two contractions
DTYPES = {"fast": "bf16 QK^T + e4m3 P.V, fp32 accumulate",
          "fp8qk": "e4m3 QK^T + e4m3 P.V, fp32 accumulate",
          "faithful": "fp32", "nocast": "fp32"}
KERNEL_SOURCES = ["paper_2606_06521_amd/csrc/attn_fast_kernel.hpp",
                  "paper_2606_06521_amd/csrc/attn_fast_dispatch.hpp",
                  "paper_2606_06521_amd/csrc/attn_fast.hip",
                  "paper_2606_06521_amd/csrc/attn_fast_pair.hip",
                  "paper_2606_06521_amd/csrc/attn_fast_qk8.hip",
                  "paper_2606_06521_amd/csrc/attn_fast_qk8_pair.hip",
                  "paper_2606_06521_amd/csrc/attn_prefill.hip",
                  "paper_2606_06521_amd/csrc/attn_common.hpp"]
HBM_PEAK_GBS = 8000.0
# chip-wide v_exp_f32 rate measured by tests/test_gpu_probes.py::test_exp2_issue_rate
# (16 independent chains per lane, all CUs): 1.83e13 exp2/s, i.e. one wave64
# instruction per ~8.6 cycles per SIMD at 2.4 GHz
EXP2_PEAK_PER_S = 1.83e13


def traffic_file(workload: str) -> str:
    return os.path.join(ROOT, "profiles", f"traffic_fast_kernel_{workload}.json")


def kernel_source_hash() -> str:
    h = hashlib.sha256()
    for p in KERNEL_SOURCES:
        with open(os.path.join(ROOT, p), "rb") as f:
            h.update(f.read())
    return h.hexdigest()


def measured_traffic(workload: str):
    """HBM bytes per launch from the committed rocprofv3 counter summary, only
    if it was taken on the current kernel source and this workload."""
    try:
        with open(traffic_file(workload)) as f:
            t = json.load(f)
    except (OSError, ValueError):
        return None
    if t.get("kernel_source_sha256") != kernel_source_hash() or t.get("workload") != workload:
        return None
    return t.get("hbm_bytes_per_launch")


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--settle-ms", type=float, default=100.0,
                    help="after the warm-up steps, keep running untimed steps until this much wall time "
                         "has passed since the first warm-up step (the GPU clock's ramp under load; "
                         "reported as settle_ms / settle_steps; 0 turns it off)")
    ap.add_argument("--workload", default=None)
    ap.add_argument("--order", default=None, choices=[None, "forward", "reverse"])
    ap.add_argument("--S", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one device copy of this size (for counter calibration)")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter CSVs (FETCH_SIZE, WRITE_SIZE) of a "
                         "run with --copy-calibration-mib into the traffic summary and exit")
    ap.add_argument("--report", metavar="JSONL", default=None,
                    help="per-run report of the five measured configurations (one JSON line per "
                         "run: GPU time and roofline fraction, MSE of the GPU and of the oracle "
                         "against FP64 attention, counts, the collapse fraction F, oracle time); "
                         "writes JSONL and a markdown summary next to it, then exits")
    ap.add_argument("--report-configs", default="C1,C2,C3,C4,C5",
                    help="which configurations the report covers")
    return ap.parse_args()


def write_traffic(fetch_csv: str, write_csv: str, workload: str, copy_mib: int = 1024) -> dict:
    """HBM bytes per call of the attention path from the two counter passes.
    Each counter is scaled by bytes_copied / counter_reading of the largest
    device copy in the same run (a plain copy of ``copy_mib`` MiB).  A call is
    one kernel, or for a split prefill its three launches (range maxima,
    pass 2, merge): the average of each kind of launch is summed."""
    import csv

    def read(path):
        rows = list(csv.DictReader(open(path)))
        name = lambda r: r["Kernel_Name"]
        kinds = [
            # the timed launches: causal, no counts, static power-of-two scale
            lambda r: "_kernel<" in name(r) and ", true, false, 1," in name(r),
            # a split prefill's range-maxima launch and its merge
            lambda r: "prefill_kernel<" in name(r) and name(r).split("(")[0].endswith(", 1>"),
            lambda r: "prefill_merge<" in name(r),
        ]
        per_call = 0.0
        for k in kinds:
            vals = [float(r["Counter_Value"]) for r in rows if k(r)]
            if vals:
                per_call += sum(vals) / len(vals)
        copy = max(float(r["Counter_Value"]) for r in rows if "copyBuffer" in r["Kernel_Name"])
        return per_call, copy

    f_kib, f_copy = read(fetch_csv)
    w_kib, w_copy = read(write_csv)
    true_kib = copy_mib * 1024.0
    f_scale, w_scale = true_kib / f_copy, true_kib / w_copy
    t = {
        "workload": workload,
        "kernel_source_sha256": kernel_source_hash(),
        "fetch_kib_per_launch_raw": f_kib,
        "write_kib_per_launch_raw": w_kib,
        "copy_calibration_mib": copy_mib,
        "fetch_scale": f_scale,
        "write_scale": w_scale,
        "hbm_read_bytes_per_launch": f_kib * 1024 * f_scale,
        "hbm_write_bytes_per_launch": w_kib * 1024 * w_scale,
        "hbm_bytes_per_launch": f_kib * 1024 * f_scale + w_kib * 1024 * w_scale,
    }
    with open(traffic_file(workload), "w") as f:
        json.dump(t, f, indent=1)
    return t


def main() -> int:
    args = parse()
    if args.write_traffic:
        from paper_2606_06521_amd.workloads import HEADLINE
        print(json.dumps(write_traffic(*args.write_traffic, args.workload or HEADLINE)))
        return 0
    world = int(os.environ.get("WORLD_SIZE", "1"))
    if args.report:
        if args.gpus != 1 or world != 1:
            print("bench.py --report: one GPU only", file=sys.stderr)
            return 2
        return report(args.report, args.report_configs.split(","))
    if args.gpus != 1 or world != 1:
        print("bench.py: measures one GPU only; the attention path shards over (batch, KV-head) "
              "groups with no communication, so a multi-GPU figure is not measured.",
              file=sys.stderr)
        return 2

    import numpy as np
    import torch

    from paper_2606_06521_amd import attn_fp8 as A
    from paper_2606_06521_amd.inputs import last_queries, make_inputs, sample_rows
    from paper_2606_06521_amd.workloads import HEADLINE, WORKLOADS

    w = WORKLOADS[args.workload or HEADLINE]
    order = args.order or w.orders[-1]
    S = args.S or w.scales[-1]
    delta = w.deltas[0]
    torch.cuda.set_device(0)
    t_gen = time.time()
    inp = make_inputs(w.B, w.Hq, w.Hkv, w.N, w.d, fmt=w.fmt, delta=delta, seed=w.seed_base,
                      bias_var=w.bias_var)
    if w.nq:
        inp = last_queries(inp, w.nq)     # w.nq queries against the w.N-key cache
    if w.fmt == "f32":
        q = torch.from_numpy(inp.q_dev).cuda()
        k = torch.from_numpy(inp.k_dev).cuda()
        v = torch.from_numpy(inp.v_dev).cuda()
    elif w.fmt == "e4m3":
        q = torch.from_numpy(inp.q_dev).cuda().view(torch.float8_e4m3fn)
        k = torch.from_numpy(inp.k_dev).cuda().view(torch.float8_e4m3fn)
        v = torch.from_numpy(inp.v_dev).cuda().view(torch.float8_e4m3fn)
    else:
        q = torch.from_numpy(inp.q_dev.view(np.int16)).cuda().view(torch.bfloat16)
        k = torch.from_numpy(inp.k_dev.view(np.int16)).cuda().view(torch.bfloat16)
        v = torch.from_numpy(inp.v_dev).cuda().view(torch.float8_e4m3fn)
    out = torch.empty((w.B, w.Hq, w.rows, w.d), dtype=torch.float32, device="cuda")
    lse = torch.empty((w.B, w.Hq, w.rows), dtype=torch.float32, device="cuda")
    gen_s = time.time() - t_gen

    if args.copy_calibration_mib > 0:
        src = torch.empty(args.copy_calibration_mib << 18, dtype=torch.float32, device="cuda").fill_(1.0)
        dst = torch.empty_like(src)
        torch.cuda.synchronize()
        dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst

    stream = torch.cuda.current_stream()
    sptr = stream.cuda_stream
    mode = A.MODES[w.mode]
    ordc = A.ORDERS[order]
    ptrs = (q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr())
    # the KV-cache split's workspace (the caller's memory), taken once
    ws = A.kv_workspace(w.B, w.Hq, w.Hkv, w.rows, w.N, w.d, w.causal, w.block_kv, mode,
                        q.device) if w.nq else None
    ws_ptr, ws_bytes = (None, 0) if ws is None else (ws.data_ptr(), ws.numel())

    def step():
        if w.nq:
            st = A.attn_fp8_fwd_kv(*ptrs, w.B, w.Hq, w.Hkv, w.rows, w.N, w.d, int(w.causal),
                                   w.block_kv, ordc, S, mode, 1.0, 1.0, 1.0, ws_ptr, ws_bytes, sptr)
        else:
            st = A.attn_fp8_fwd(*ptrs, w.B, w.Hq, w.Hkv, w.N, w.d, int(w.causal), w.block_kv,
                                ordc, S, mode, sptr)
        if st != A.ATTN_OK:
            raise A.AttnError(st)

    t_w0 = time.perf_counter()
    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
    # The GPU's clock ramps up over the first tens of milliseconds of sustained
    # load: in kernel traces of this step the first launches take up to 1.35x
    # the settled time and the time keeps falling for about 25 launches.
    # Untimed steps continue until settle_ms have passed since the first
    # warm-up step, so the K timed steps see the settled clock.
    settle_steps = 0
    while (time.perf_counter() - t_w0) * 1e3 < args.settle_ms:
        for _ in range(4):
            step()
        torch.cuda.synchronize()
        settle_steps += 4
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(args.steps)]
    t0 = time.perf_counter()
    for s_ev, e_ev in ev:
        s_ev.record(stream)
        step()
        e_ev.record(stream)
    torch.cuda.synchronize()
    t1 = time.perf_counter()
    ms_per_step = (t1 - t0) * 1e3 / args.steps
    kernel_ms = [s_ev.elapsed_time(e_ev) for s_ev, e_ev in ev]
    # the statistic of the roofline: the median of the timed launches (mean
    # and minimum reported beside it)
    kernel_ms_med = float(np.median(kernel_ms))
    flops = w.flops()
    # dense peak of the contraction dtype: FP8 MFMA for the fast modes (the
    # spec denominator), FP32 matrix for the faithful ones
    peak = PEAK_TFLOPS["fp8"] if w.mode in ("fast", "fp8qk") else 157.3
    value = flops / (ms_per_step * 1e-3) / 1e12
    achieved = flops / (kernel_ms_med * 1e-3) / 1e12
    # algorithmic HBM bytes: q, k, v once, out and lse written once
    qk_bytes = 1 if w.fmt == "e4m3" else (2 if w.fmt == "bf16_e4m3" else 4)
    v_bytes = 4 if w.fmt == "f32" else 1
    hbm_bytes = float(w.B * (w.Hq * w.rows * w.d * qk_bytes + w.Hkv * w.N * w.d * (qk_bytes + v_bytes)
                             + w.Hq * w.rows * (4 * w.d + 4)))
    hbm_bound = flops / hbm_bytes < peak / HBM_PEAK_GBS * 1e3
    timing = {"kernel_ms_median": round(kernel_ms_med, 4),
              "kernel_ms_mean": round(float(np.mean(kernel_ms)), 4),
              "kernel_ms_min": round(float(np.min(kernel_ms)), 4),
              "timed_launches": len(kernel_ms)}

    # P-underflow diagnostic on the same inputs (timed separately, not reported as throughput)
    cnt = A.p_underflow_count(q, k, v, S=S, order=order, causal=w.causal, block_kv=w.block_kv,
                              mode=w.mode, n_sink=inp.n_sink)
    torch.cuda.synchronize()
    cnt_np = cnt.cpu().numpy().view(np.uint32).reshape(-1, 3)
    counts_total = [int(x) for x in cnt_np.sum(0, dtype=np.uint64)]

    res = {
        "metric": "FP8-attn fwd TFLOP/s (% MFMA peak) at N=8192 d=128; P-cast MSE vs FP64",
        "value": round(value, 2),
        "unit": "TFLOP/s",
        "n_gpus": 1,
        "steps": args.steps,
        "warmup": args.warmup,
        "settle_ms": args.settle_ms,
        "settle_steps": settle_steps,
        "ms_per_step": round(ms_per_step, 4),
        "higher_is_better": True,
        "scaling": "weak",
        "vs_baseline": None,
        "dtype": DTYPES[w.mode],
        "data": "synthetic (seeded sink workload, Delta=%g, 4 sink keys)" % delta,
        "config": {"workload": w.name, "B": w.B, "Hq": w.Hq, "Hkv": w.Hkv, "N": w.N,
                   "query_rows": w.rows, "d": w.d,
                   "causal": w.causal, "mode": w.mode, "block_kv": w.block_kv, "order": order,
                   "S": S, "delta_eff": round(inp.delta_eff, 4), "parallelism": "single GPU"},
        "roofline": {
            "bound": "hbm",
            "achieved": round(hbm_bytes / (kernel_ms_med * 1e-3) / 1e9, 1),
            "peak": HBM_PEAK_GBS,
            "unit": "GB/s",
            "frac": round(hbm_bytes / (kernel_ms_med * 1e-3) / 1e9 / HBM_PEAK_GBS, 4),
            "algorithmic_bytes_per_launch": hbm_bytes,
            "traffic": measured_traffic(w.name),
            **timing,
            "flops_per_launch": flops,
            "tflops": round(achieved, 2),
        } if hbm_bound else {
            "bound": "mfma",
            "achieved": round(achieved, 2),
            "peak": peak,
            "unit": "TFLOP/s",
            "frac": round(achieved / peak, 4),
            "traffic": measured_traffic(w.name),
            **timing,
            "flops_per_launch": flops,
            "mixed_bf16_fp8_peak": round(MIXED_PEAK, 1) if w.mode == "fast" else None,
            "frac_of_mixed_peak": round(achieved / MIXED_PEAK, 4) if w.mode == "fast" else None,
        },
        # one exp2 per visible (row, key) pair, against the measured v_exp_f32 rate
        "exp2": {"per_launch": w.pairs(),
                 "achieved_per_s": float("%.4g" % (w.pairs() / (kernel_ms_med * 1e-3))),
                 "peak_per_s": EXP2_PEAK_PER_S,
                 "frac": round(w.pairs() / (kernel_ms_med * 1e-3) / EXP2_PEAK_PER_S, 4)},
        "p_underflow_counts": {"sink": counts_total[0], "sink_block_nonsink": counts_total[1],
                               "other_blocks": counts_total[2]},
        "input_gen_s": round(gen_s, 2),
    }

    if not args.no_cpu_baseline:
        # the same workload with the dynamic per-block scale (S = 2^k0), for its MSE
        out_dyn = None
        if float(np.log2(S)).is_integer() and 0 <= np.log2(S) <= 8:
            out_dyn, _ = A.fwd(q, k, v, S=S, order=order, causal=w.causal, block_kv=w.block_kv,
                               mode=w.mode, want_lse=False, scale="dynamic")
            torch.cuda.synchronize()
        res["cpu_baseline"] = cpu_baseline(inp, w, order, S, out, lse, cnt_np, sample_rows, out_dyn)
    print(json.dumps(res), flush=True)
    return 0


def cpu_baseline(inp, w, order, S, out_dev, lse_dev, cnt_gpu, sample_rows, out_dyn_dev=None):
    """The oracle (as it stands) on a bounded row sample of the same workload,
    plus P-cast MSE of the GPU output and of the oracle against FP64 attention,
    the largest GPU-oracle differences, and the sample's underflow fractions
    per key category next to the paper's collapse fraction F(Delta, S)."""
    import numpy as np

    import oracle
    from oracle import analysis

    nthreads = min(16, oracle.default_threads())
    # about 10-15 s of oracle work on 16 host threads at the headline size
    every = max(1, (w.B * w.Hq * w.rows) // 524288)
    rows = np.arange(0, w.B * w.Hq * w.rows, every, dtype=np.int64)
    rows = np.unique(np.concatenate([rows, sample_rows(w.B, w.Hq, w.rows, 128, 10 ** 9,
                                                       seed=0)[:64]]))
    keys = (rows % w.rows + (w.N - w.rows) + 1) if w.causal else np.full(rows.size, w.N)
    flops = float(4.0 * w.d * keys.sum())
    fast = w.mode in ("fast", "fp8qk")
    t0 = time.perf_counter()
    res = oracle.attn(inp.q32, inp.k32, inp.v32, S=S, order=order, block_kv=w.block_kv,
                      causal=w.causal, n_sink=inp.n_sink, rows=rows, nthreads=nthreads,
                      bound_rel=6.0 * 2.0 ** -23 if fast else None)
    dt = time.perf_counter() - t0
    o_out, o_lse, o_cnt = res[:3]
    ref, _ = oracle.ref_fp64(inp.q32, inp.k32, inp.v32, causal=w.causal, rows=rows, nthreads=nthreads)
    g = out_dev.cpu().numpy().reshape(-1, w.d)[rows]
    mse_gpu = float(np.mean((g.astype(np.float64) - ref) ** 2))
    mse_oracle = float(np.mean((o_out.astype(np.float64) - ref) ** 2))
    gl = lse_dev.cpu().numpy().reshape(-1)[rows]
    # visible keys of each sampled row per category: sink keys, the rest of
    # block 0, the other blocks
    n_s = np.minimum(inp.n_sink, keys)
    n_b0 = np.minimum(w.block_kv, keys) - n_s
    n_o = keys - np.minimum(w.block_kv, keys)
    frac = {name: (float(o_cnt[:, i].sum() / n.sum()) if n.sum() else None)
            for i, (name, n) in enumerate((("sink", n_s), ("sink_block_nonsink", n_b0),
                                           ("other_blocks", n_o)))}
    extra = {}
    if fast:
        # elements past the spec bar (2e-2), and past it plus the
        # per-element code-ambiguity bound the parity tests allow
        diff = np.abs(g.astype(np.float64) - o_out)
        extra["n_out_past_2e-2"] = int((diff > 2e-2).sum())
        extra["n_out_past_2e-2_plus_amb"] = int((diff > 2e-2 + res[3]).sum())
    if out_dyn_dev is not None:
        gd = out_dyn_dev.cpu().numpy().reshape(-1, w.d)[rows]
        extra["mse_gpu_dynamic_scale_vs_fp64"] = float(np.mean((gd.astype(np.float64) - ref) ** 2))
    return {
        "value": round(flops / dt / 1e12, 6),
        "unit": "TFLOP/s",
        "cores": nthreads,
        "kind": "oracle",
        "sample": f"{rows.size} query rows (every {every}th flat row of all batches/heads, "
                  f"{int(keys.sum())} (row, key) pairs, {flops:.3e} FLOP) in {dt:.2f} s",
        "oracle_s": round(dt, 3),
        "mse_gpu_vs_fp64": mse_gpu,
        "mse_oracle_vs_fp64": mse_oracle,
        "max_abs_gpu_minus_oracle": float(np.abs(g - o_out).max()),
        "max_abs_lse_gpu_minus_oracle": float(np.abs(gl.astype(np.float64) - o_lse).max()),
        # fraction of the sample's visible (row, key) pairs per category whose
        # E4M3 code is zero; F(Delta, S) is the paper's collapse fraction of
        # non-sink keys under the sink maximum (forward order: every block;
        # reverse order: block 0 only, none elsewhere by Theorem 2)
        "underflow_fraction": frac,
        "collapse_fraction_F": analysis.collapse_fraction(inp.delta_eff, S, inp.n_sink),
        "counts_equal_on_sample": bool(np.array_equal(cnt_gpu[rows], o_cnt)),
        **extra,
    }


# ---------------------------------------------------------------------------
# Per-run report
# ---------------------------------------------------------------------------

# The paper's own figures, quoted as context only: they come from its
# kernel-faithful simulation (FP32 Q/K/V, block 64, q_len 32 for the MSE
# table, an FP32 reference), not from a kernel or this hardware.
PAPER_TABLE1 = {   # Table 1 (Sec. 3.3): fraction of non-sink P zeroed, forward order, N = 4096
    "delta": [5, 6, 7, 8, 9, 10, 12],
    "S1": [0.223, 0.516, 0.820, 0.948, 0.995, 1.0, 1.0],
    "S256": [0.0, 0.0, 0.0, 0.003, 0.023, 0.117, 0.679],
}
PAPER_TABLE2_N4096 = {   # Table 2 (Sec. 6.5): MSE at Delta = 7, N = 4096 (x 1e-5)
    ("forward", 1.0): 5.65e-5, ("reverse", 1.0): 1.70e-5, ("forward", 448.0): 1.81e-5,
    ("forward", 256.0): 1.64e-5, ("reverse", 256.0): 1.64e-5,
}

# configuration label -> (workload, runs [(S, order, Delta)], oracle row stride)
REPORT_CONFIGS = {
    "C1": "sink_n1024_d64_faithful",
    "C2": "sink_sweep_h8_n4096_d128_faithful",
    "C3": "causal_mha_b4_h32_n8192_d128_fast",
    "C4": "causal_gqa_h64kv8_n32768_d128_fast",
    "C5": "causal_gqa_h32kv8_n131072_d128_fast_bias",
}
REPORT_STRIDE = {"C1": 1, "C2": 4, "C3": 64, "C4": 512, "C5": 2048}


def _paper_context(label, order, S, delta):
    ctx = {}
    if label == "C2" and order == "forward" and delta in PAPER_TABLE1["delta"] and S in (1.0, 256.0):
        i = PAPER_TABLE1["delta"].index(delta)
        ctx["table1_frac_zeroed"] = PAPER_TABLE1["S1" if S == 1.0 else "S256"][i]
    if label == "C2" and delta == 7.0 and (order, S) in PAPER_TABLE2_N4096:
        ctx["table2_mse"] = PAPER_TABLE2_N4096[(order, S)]
    if ctx:
        ctx["note"] = ("the paper's simulation (block 64, FP32 reference; Table 2 with "
                       "32 queries per problem): context, not a target")
    return ctx


def report(path: str, labels) -> int:
    """Runs every (S, order, Delta) of the selected configurations once on the
    GPU (timed, and again with the underflow count), the oracle on a fixed row
    sample, FP64 attention on the same rows; one JSON line per run."""
    import numpy as np
    import torch

    import oracle
    from oracle import analysis
    from paper_2606_06521_amd import attn_fp8 as A
    from paper_2606_06521_amd.inputs import make_inputs, with_delta
    from paper_2606_06521_amd.workloads import WORKLOADS

    torch.cuda.set_device(0)
    nthreads = oracle.default_threads()
    stream = torch.cuda.current_stream()
    out_f = open(path, "w")
    for label in labels:
        w = WORKLOADS[REPORT_CONFIGS[label]]
        every = REPORT_STRIDE[label]
        print(f"report {label}: inputs for {w.name}", flush=True)
        t_gen = time.perf_counter()
        base = make_inputs(w.B, w.Hq, w.Hkv, w.N, w.d, fmt=w.fmt, delta=w.deltas[0],
                           seed=w.seed_base, bias_var=w.bias_var)
        gen_s = time.perf_counter() - t_gen
        rows_total = w.B * w.Hq * w.N
        rows = np.arange(0, rows_total, every, dtype=np.int64)
        # visible keys per row and per count category, over all rows
        r_all = np.arange(w.N, dtype=np.int64)
        keys = (r_all + 1) if w.causal else np.full(w.N, w.N, dtype=np.int64)
        n_s = np.minimum(4, keys)
        denom = [int(n_s.sum()) * w.B * w.Hq,
                 int((np.minimum(w.block_kv, keys) - n_s).sum()) * w.B * w.Hq,
                 int((keys - np.minimum(w.block_kv, keys)).sum()) * w.B * w.Hq]
        keys_s = (rows % w.N + 1) if w.causal else np.full(rows.size, w.N)
        peak = PEAK_TFLOPS["fp8"] if w.mode in ("fast", "fp8qk") else 157.3
        # the headline-sized runs get the bench's own 5 warm-up and 20 timed
        # launches (fewer warm-ups read the clock still ramping up)
        reps, warm = (20, 5) if w.flops() < 1e13 else (10, 5)
        for delta in w.deltas:
            inp = base if delta == w.deltas[0] else with_delta(base, delta)
            dev = _to_device(inp, torch, np)
            ref, _ = oracle.ref_fp64(inp.q32, inp.k32, inp.v32, causal=w.causal, rows=rows,
                                     nthreads=nthreads)
            for S in w.scales:
                for order in w.orders:
                    rec = _report_run(label, w, inp, dev, S, order, rows, keys_s, ref, denom,
                                      peak, reps, warm, nthreads, stream, A, oracle, analysis,
                                      torch, np)
                    rec["input_gen_s"] = round(gen_s, 2)
                    out_f.write(json.dumps(rec) + "\n")
                    out_f.flush()
                    print(f"report {label} Delta={delta:g} S={S:g} {order}: "
                          f"{rec['gpu_ms_median']} ms, {rec['tflops']} TFLOP/s, "
                          f"MSE gpu {rec['mse_gpu_vs_fp64']:.3e} oracle {rec['mse_oracle_vs_fp64']:.3e}",
                          flush=True)
            del dev
            torch.cuda.empty_cache()
    out_f.close()
    write_report_md(path)
    return 0


def _to_device(inp, torch, np):
    if inp.fmt == "f32":
        return tuple(torch.from_numpy(a).cuda() for a in (inp.q_dev, inp.k_dev, inp.v_dev))
    if inp.fmt == "e4m3":
        return tuple(torch.from_numpy(a).cuda().view(torch.float8_e4m3fn)
                     for a in (inp.q_dev, inp.k_dev, inp.v_dev))
    return (torch.from_numpy(inp.q_dev.view(np.int16)).cuda().view(torch.bfloat16),
            torch.from_numpy(inp.k_dev.view(np.int16)).cuda().view(torch.bfloat16),
            torch.from_numpy(inp.v_dev).cuda().view(torch.float8_e4m3fn))


def _report_run(label, w, inp, dev, S, order, rows, keys_s, ref, denom, peak, reps, warm,
                nthreads, stream, A, oracle, analysis, torch, np):
    q, k, v = dev
    out = torch.empty((w.B, w.Hq, w.N, w.d), dtype=torch.float32, device="cuda")
    lse = torch.empty((w.B, w.Hq, w.N), dtype=torch.float32, device="cuda")
    ptrs = (q.data_ptr(), k.data_ptr(), v.data_ptr(), out.data_ptr(), lse.data_ptr())
    mode = A.MODES[w.mode]
    ordc = A.ORDERS[order]

    def step():
        st = A.attn_fp8_fwd(*ptrs, w.B, w.Hq, w.Hkv, w.N, w.d, int(w.causal), w.block_kv, ordc,
                            S, mode, stream.cuda_stream)
        if st != A.ATTN_OK:
            raise A.AttnError(st)

    # warm-up launches, then untimed ones until the clock has settled (as in
    # the bench line: 100 ms after the first warm-up launch)
    t_w0 = time.perf_counter()
    for _ in range(warm):
        step()
    torch.cuda.synchronize()
    while (time.perf_counter() - t_w0) * 1e3 < 100.0:
        step()
        torch.cuda.synchronize()
    ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True))
          for _ in range(reps)]
    for s_ev, e_ev in ev:
        s_ev.record(stream)
        step()
        e_ev.record(stream)
    torch.cuda.synchronize()
    ms = float(np.median([a.elapsed_time(b) for a, b in ev]))
    cnt = A.p_underflow_count(q, k, v, S=S, order=order, causal=w.causal, block_kv=w.block_kv,
                              mode=w.mode, n_sink=inp.n_sink)
    torch.cuda.synchronize()
    cnt_all = cnt.cpu().numpy().view(np.uint32).reshape(-1, 3)
    g_out = out.cpu().numpy().reshape(-1, w.d)[rows]
    g_lse = lse.cpu().numpy().reshape(-1)[rows]
    fast = w.mode in ("fast", "fp8qk")
    t0 = time.perf_counter()
    res = oracle.attn(inp.q32, inp.k32, inp.v32, S=S, order=order, block_kv=w.block_kv,
                      causal=w.causal, n_sink=inp.n_sink, rows=rows, nthreads=nthreads,
                      bound_rel=6.0 * 2.0 ** -23 if fast else None)
    oracle_s = time.perf_counter() - t0
    o_out, o_lse, o_cnt = res[:3]
    diff = np.abs(g_out.astype(np.float64) - o_out)
    tol = 2e-2 if fast else 2e-3
    counts = [int(x) for x in cnt_all.sum(0, dtype=np.uint64)]
    flops = w.flops()
    rec = {
        "config": label, "workload": w.name, "mode": w.mode, "S": S, "order": order,
        "delta": inp.delta, "delta_eff": round(inp.delta_eff, 4),
        "gpu_ms_median": round(ms, 4), "timed_launches": reps,
        "tflops": round(flops / (ms * 1e-3) / 1e12, 2), "peak_tflops": peak,
        "frac_of_peak": round(flops / (ms * 1e-3) / 1e12 / peak, 4),
        "mse_gpu_vs_fp64": float(np.mean((g_out.astype(np.float64) - ref) ** 2)),
        "mse_oracle_vs_fp64": float(np.mean((o_out.astype(np.float64) - ref) ** 2)),
        "max_abs_gpu_minus_oracle": float(diff.max()),
        "max_abs_lse_gpu_minus_oracle": float(np.abs(g_lse.astype(np.float64) - o_lse).max()),
        "counts_gpu_all_rows": {"sink": counts[0], "sink_block_nonsink": counts[1],
                                "other_blocks": counts[2]},
        "pairs_all_rows": {"sink": denom[0], "sink_block_nonsink": denom[1],
                           "other_blocks": denom[2]},
        "zero_fraction_nonsink": (counts[1] + counts[2]) / max(1, denom[1] + denom[2]),
        "collapse_fraction_F": analysis.collapse_fraction(inp.delta_eff, S, inp.n_sink),
        "counts_equal_on_oracle_rows": bool(np.array_equal(cnt_all[rows], o_cnt)),
        "oracle": {"rows": int(rows.size), "rows_total": int(w.B * w.Hq * w.N),
                   "sample": f"every {REPORT_STRIDE[label]}th flat row",
                   "pairs": int(keys_s.sum()), "seconds": round(oracle_s, 3), "cores": nthreads,
                   "tflops": round(4.0 * w.d * float(keys_s.sum()) / oracle_s / 1e12, 6)},
    }
    if fast:
        amb = res[3]
        rec["n_out_past_tol"] = int((diff > tol).sum())
        rec["n_out_past_tol_and_amb"] = int((diff > tol + amb).sum())
    ctx = _paper_context(label, order, S, inp.delta)
    if ctx:
        rec["paper_context"] = ctx
    return rec


def write_report_md(path: str) -> str:
    """Markdown summary of a report JSONL (written next to it, .md)."""
    recs = [json.loads(l) for l in open(path) if l.strip()]
    md = os.path.splitext(path)[0] + ".md"
    lines = ["# Per-run report: the five measured configurations", "",
             "Generated by `python bench.py --report " + os.path.relpath(path, ROOT) + "` "
             "(one MI355X; seeded synthetic inputs).  One row per run.  MSE is the mean "
             "over output elements against FP64 softmax attention on the oracle's row "
             "sample; counts and zero fractions cover every row; F is the collapse "
             "fraction of the Corollary at Delta_eff, a prediction for the forward order "
             "(reverse order zeroes only the sink block's non-sink keys).  Paper figures "
             "are context only.", "",
             "| cfg | Delta_eff | S | order | GPU ms | TFLOP/s | of peak | MSE GPU | MSE oracle "
             "| max |GPU-oracle| | zeroed non-sink | F | counts equal | oracle s (cores, rows) "
             "| paper |",
             "|---|---|---|---|---|---|---|---|---|---|---|---|---|---|---|"]
    for r in recs:
        ctx = r.get("paper_context", {})
        paper = ", ".join(f"{k}={v}" for k, v in ctx.items() if k != "note")
        o = r["oracle"]
        lines.append(
            f"| {r['config']} | {r['delta_eff']} | {r['S']:g} | {r['order']} | "
            f"{r['gpu_ms_median']} | {r['tflops']} | {r['frac_of_peak']:.3f} | "
            f"{r['mse_gpu_vs_fp64']:.3e} | {r['mse_oracle_vs_fp64']:.3e} | "
            f"{r['max_abs_gpu_minus_oracle']:.2e} | {r['zero_fraction_nonsink']:.4g} | "
            f"{r['collapse_fraction_F']:.4g} | {r['counts_equal_on_oracle_rows']} | "
            f"{o['seconds']} ({o['cores']}, {o['rows']}) | {paper} |")
    # the paper's MSE-improvement figures beside the measured ratio (context)
    c2 = [r for r in recs if r["config"] == "C2" and r["delta"] == 7.0]
    f1 = [r["mse_gpu_vs_fp64"] for r in c2 if r["order"] == "forward" and r["S"] == 1.0]
    best = [r["mse_gpu_vs_fp64"] for r in c2 if r["S"] == 256.0]
    if f1 and best:
        lines += ["", f"MSE improvement at Delta = 7, N = 4096 (C2): MSE(forward, S = 1) / MSE(best "
                  f"S = 256 run) = {f1[0] / min(best):.2f}x measured.  Context only: the paper's "
                  "Table 2 (Sec. 6.5) gives 3.4x at N = 4096 (5.5x at 8192, 10.5x at 16384), and its "
                  "Exp. 2 (Sec. 6.4) a ratio growing from 1.3x at N = 512 to 10x at N = 16384, from "
                  "its kernel-faithful simulation (FP32 Q/K/V, block 64)."]
    open(md, "w").write("\n".join(lines) + "\n")
    return md


if __name__ == "__main__":
    sys.exit(main())
