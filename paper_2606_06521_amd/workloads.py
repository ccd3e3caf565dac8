"""Named synthetic workloads (shapes and settings of the measured problems).

Every workload is the paper's sink setting (Sec. 3.1) at a given size; the
names say what each one is.  ``seed_base`` feeds ``inputs.make_inputs``.
"""
from __future__ import annotations

from dataclasses import dataclass


@dataclass(frozen=True)
class Workload:
    name: str
    B: int
    Hq: int
    Hkv: int
    N: int
    d: int
    causal: bool
    mode: str                 # "faithful" or "fast"
    block_kv: int
    deltas: tuple
    scales: tuple
    orders: tuple
    bias_var: float = 0.0
    seed_base: int = 0
    nq: int = 0               # query rows against N cached keys (0: all N rows)

    @property
    def rows(self) -> int:
        return self.nq or self.N

    @property
    def fmt(self) -> str:
        if self.mode == "fp8qk":
            return "e4m3"
        return "f32" if self.mode in ("faithful", "nocast") else "bf16_e4m3"

    def pairs(self) -> int:
        """Visible (query row, key) pairs per launch: one exp2, one P and one
        E4M3 code each.  Row r of nq sits at key position N - nq + r."""
        nq = self.rows
        if not self.causal:
            per_head = nq * self.N
        else:
            per_head = nq * (self.N - nq) + nq * (nq + 1) // 2
        return self.B * self.Hq * per_head

    def flops(self) -> float:
        """FlashAttention convention: 4*B*Hq*N^2*d, halved under causal masking.
        With nq query rows against N cached keys: 4 d per (row, visible key)."""
        if not self.nq:
            f = 4.0 * self.B * self.Hq * self.N * self.N * self.d
            return f / 2 if self.causal else f
        keys = (self.nq * (self.N - self.nq) + self.nq * (self.nq + 1) / 2 if self.causal
                else self.nq * self.N)
        return 4.0 * self.B * self.Hq * keys * self.d


WORKLOADS = {
    w.name: w for w in [
        # single head, four sink keys at Delta = 8, both orders, S in {1, 256}
        Workload("sink_n1024_d64_faithful", 1, 1, 1, 1024, 64, False, "faithful", 64,
                 (8.0,), (1.0, 256.0), ("forward", "reverse"), seed_base=20260100),
        # Delta sweep 0..12 over S in {1, 16, 256, 448}, both orders, 8 heads
        Workload("sink_sweep_h8_n4096_d128_faithful", 1, 8, 8, 4096, 128, False, "faithful", 128,
                 tuple(float(x) for x in range(13)), (1.0, 16.0, 256.0, 448.0),
                 ("forward", "reverse"), seed_base=20260200),
        # causal MHA prefill, bf16 Q/K, e4m3 V, Delta = 7, reverse, S = 256
        Workload("causal_mha_b4_h32_n8192_d128_fast", 4, 32, 32, 8192, 128, True, "fast", 128,
                 (7.0,), (256.0,), ("reverse",), seed_base=20260300),
        # the same with E4M3 Q and K (S^T on the FP8 MFMA as well)
        Workload("causal_mha_b4_h32_n8192_d128_fp8qk", 4, 32, 32, 8192, 128, True, "fp8qk", 128,
                 (7.0,), (256.0,), ("reverse",), seed_base=20260310),
        # causal GQA 64/8 heads at 32k, Delta = 9, S in {1, 256}, both orders
        Workload("causal_gqa_h64kv8_n32768_d128_fast", 1, 64, 8, 32768, 128, True, "fast", 128,
                 (9.0,), (1.0, 256.0), ("forward", "reverse"), seed_base=20260400),
        # causal GQA 32/8 heads at 128k, Delta = 10 plus a N(0, 0.5) per-key bias
        Workload("causal_gqa_h32kv8_n131072_d128_fast_bias", 1, 32, 8, 131072, 128, True, "fast",
                 128, (10.0,), (256.0,), ("reverse",), bias_var=0.5, seed_base=20260500),
        # Exp. 1's shape: 32 new queries against a 4096-key cache, 64 problems
        Workload("prefill_q32_b64_n4096_d128_fast", 64, 1, 1, 4096, 128, True, "fast", 128,
                 (7.0,), (256.0,), ("reverse",), seed_base=20260600, nq=32),
        # a serving-sized prefill chunk: 256 queries against a 32k cache, GQA 32/8
        Workload("prefill_q256_b4_h32kv8_n32768_d128_fast", 4, 32, 8, 32768, 128, True, "fast",
                 128, (9.0,), (256.0,), ("reverse",), seed_base=20260700, nq=256),
    ]
}

HEADLINE = "causal_mha_b4_h32_n8192_d128_fast"
