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
                  "paper_2606_06521_amd/csrc/attn_fast.hip",
                  "paper_2606_06521_amd/csrc/attn_fast_qk8.hip",
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
    ap.add_argument("--workload", default=None)
    ap.add_argument("--order", default=None, choices=[None, "forward", "reverse"])
    ap.add_argument("--S", type=float, default=None)
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--copy-calibration-mib", type=int, default=0,
                    help="also run one device copy of this size (for counter calibration)")
    ap.add_argument("--write-traffic", nargs=2, metavar=("FETCH_CSV", "WRITE_CSV"),
                    help="turn two rocprofv3 --pmc counter CSVs (FETCH_SIZE, WRITE_SIZE) of a "
                         "run with --copy-calibration-mib into the traffic summary and exit")
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

    for _ in range(args.warmup):
        step()
    torch.cuda.synchronize()
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
    t0 = time.perf_counter()
    o_out, o_lse, o_cnt = oracle.attn(inp.q32, inp.k32, inp.v32, S=S, order=order,
                                      block_kv=w.block_kv, causal=w.causal, n_sink=inp.n_sink,
                                      rows=rows, nthreads=nthreads)
    dt = time.perf_counter() - t0
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


if __name__ == "__main__":
    sys.exit(main())
