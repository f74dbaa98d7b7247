"""Benchmark of deferred normalization on one MI355X.

    python bench.py [--steps K] [--warmup W] [--workload NAME] [--no-cpu-baseline]

A step is one pass of the whole hot path over one batch of synthetic input:
the deferred LayerNorm -> Linear (Sec. II-A, Eq. (5)) and the deferred
Softmax -> P.V (Sec. II-B, Eq. (8)).  The default workload is a 7B-class
Transformer layer's two fusion sites: LN -> QKV projection, x[4096, 4096] .
W[4096, 12288], and causal Softmax -> P.V over 32 heads, 8192 keys, d = 128.

Warmup: the W untimed steps, continued until at least --warm-seconds (0.3 s)
of them have run, so that the timed steps see the chip's steady clocks rather
than its ramp out of idle (which costs 10-25 % on the first few milliseconds).

Prints ONE JSON line.  `value` is whole-step throughput (TFLOP/s, algorithmic
FLOP of both products) with inputs already resident in HBM; per-kernel times
come from HIP events recorded on the stream the kernels are launched on.  The
unfused comparators (LayerNorm + GEMM; Softmax + GEMM) run in the same process
on the same inputs; speedups compare each path timed on its own, back to back.
`cpu_baseline` times the fp64 oracle on a bounded row sample of the same
workload on this host's cores and extrapolates by work.

Other workloads (--workload): ln_qkv, causal_softmax_pv, ffn_prefill,
ffn_decode_t{1,4,16} (LayerNorm -> FFN up-projection, 8192 x 28672),
qkv_t{32,128,1024} (the LN -> QKV projection over 32 / 128 tokens of batched
decode and a 1024-token prefill chunk), rms_qkv,
rms_ffn_decode_t1 (RMSNorm, Eq. (6)), swiglu_prefill, swiglu_decode_t1
(RMSNorm -> gated MLP input), causal_attention (scores formed in the kernel),
decode_attention, decode_attention_gqa (keys split to fill the chip), small.  Per kernel
the line also carries the ablations the workload supports: statistics from a
pre-pass (serial_stats_ms), normalize-on-load without deferral
(norm_on_load_ms), the post-LN placement (post_ln_ms), the eager dense softmax
pair (unfused_dense_ms), decode without the key split (single_pass_ms).
"""
from __future__ import annotations

import argparse
import json
import os
import sys
import time

import numpy as np
import torch

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

METRIC = "TFLOP/s fused LN→GEMM & softmax→PV, % MFMA peak, speedup vs unfused"
PEAK_BF16_TFLOPS = 2516.6   # 256 CU x 2.4 GHz x 4096 flop/clk (dense bf16 MFMA)
PEAK_F32_TFLOPS = 157.3     # fp32 MFMA / vector
PEAK_HBM_GBS = 8000.0       # HBM3E
ROUNDS = 7                  # rounds of the alternating isolated timings

# HBM traffic per launch, from two rocprofv3 --pmc runs of this script (FETCH_SIZE, then WRITE_SIZE,
# KiB per dispatch, averaged over the timed launches), each scaled by what the same counter reads for
# a plain device copy of 1 GiB in the same run (--calib-copy-mib 1024): FETCH_SIZE reads 524306 KiB
# for its 1048576 KiB (x 1.99993), WRITE_SIZE reads 1048576 KiB (x 1.0).  A figure is only valid for
# the kernel source it was taken on: each entry carries the sha256 of its kernel's source files, and
# the bench reports null once they differ.
KERNEL_SOURCES = {"softmax_pv_deferred": ("softmax_pv.hip", "dn_device.hpp"),
                  "attention_deferred": ("attention.hip", "dn_device.hpp"),
                  "attention_decode_deferred": ("attention.hip", "dn_device.hpp"),
                  "ln_linear_deferred": ("ln_gemm.hip", "dn_device.hpp"),
                  "rms_linear_deferred": ("ln_gemm.hip", "dn_device.hpp"),
                  "rms_swiglu_deferred": ("ln_gemm.hip", "dn_device.hpp")}
TRAFFIC = {
    ("softmax_pv_deferred", "causal_softmax_pv_bf16_32x8192x8192_d128"): {
        "sha256": ("8348feaf7e161752c3966e3a1e5f5235f20f8403ef203d36c1487a1565ffb446",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 1131128, "fetch_scale": 1.99988, "write_kib": 65962, "write_scale": 1.0},
    ("softmax_pv_deferred", "softmax_pv_bf16_12x512x512_d64"): {
        "sha256": ("8348feaf7e161752c3966e3a1e5f5235f20f8403ef203d36c1487a1565ffb446",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 3676, "fetch_scale": 1.99990, "write_kib": 768, "write_scale": 1.0},
    ("ln_linear_deferred", "ln_qkv_bf16_4096x4096x12288"): {
        "sha256": ("70ff13ee8dfa009c3eb542e1df3eb31c525d39718e9311900f3f1a3c58b46307",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 298905, "fetch_scale": 1.99992, "write_kib": 109686, "write_scale": 1.0},
    ("ln_linear_deferred", "ln_ffn_up_bf16_8192x8192x28672"): {
        "sha256": ("70ff13ee8dfa009c3eb542e1df3eb31c525d39718e9311900f3f1a3c58b46307",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 2768553, "fetch_scale": 1.99993, "write_kib": 481424, "write_scale": 1.0},
    ("ln_linear_deferred", "ln_ffn_up_bf16_decode_t1_8192x28672"): {
        "sha256": ("70ff13ee8dfa009c3eb542e1df3eb31c525d39718e9311900f3f1a3c58b46307",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 233660, "fetch_scale": 1.99986, "write_kib": 56, "write_scale": 1.0},
    ("ln_linear_deferred", "ln_linear_f32_128x768x3072"): {
        "sha256": ("70ff13ee8dfa009c3eb542e1df3eb31c525d39718e9311900f3f1a3c58b46307",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 6296, "fetch_scale": 1.99992, "write_kib": 1536, "write_scale": 1.0},
    ("rms_linear_deferred", "rms_qkv_bf16_4096x4096x6144"): {
        "sha256": ("70ff13ee8dfa009c3eb542e1df3eb31c525d39718e9311900f3f1a3c58b46307",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 164194, "fetch_scale": 1.99993, "write_kib": 52852, "write_scale": 1.0},
    ("rms_swiglu_deferred", "rms_swiglu_bf16_decode_t1_8192x28672"): {
        "sha256": ("70ff13ee8dfa009c3eb542e1df3eb31c525d39718e9311900f3f1a3c58b46307",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 459121, "fetch_scale": 1.99994, "write_kib": 56, "write_scale": 1.0},
    ("attention_deferred", "causal_attention_bf16_32x8192x8192_d128"): {
        "sha256": ("7a22d31fdb1a62b1da07e531c37abb39162f3075d1df416b61aae2ba1f2a525e",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 144248, "fetch_scale": 1.99991, "write_kib": 65536, "write_scale": 1.0},
    # 256 heads fill the chip with one workgroup per head: no key split, no merge kernel
    ("attention_decode_deferred", "decode_attention_bf16_256x1x8192_d128"): {
        "sha256": ("7a22d31fdb1a62b1da07e531c37abb39162f3075d1df416b61aae2ba1f2a525e",
                   "ac9c5fe92ec45f657c9519fcd8d54a4977d6a85897f645cae15b69abf72ca89a"),
        "fetch_kib": 524463, "fetch_scale": 1.99990, "write_kib": 64, "write_scale": 1.0},
}


def measured_traffic(kernel: str, workload: str):
    """HBM bytes per launch from the counter table, or None when absent or taken on other sources."""
    import hashlib
    t = TRAFFIC.get((kernel, workload))
    if t is None:
        return None
    csrc = os.path.join(ROOT, "paper_2502_17728_amd", "csrc")
    now = tuple(hashlib.sha256(open(os.path.join(csrc, f), "rb").read()).hexdigest()
                for f in KERNEL_SOURCES[kernel])
    if now != t["sha256"]:
        return None
    return 1024.0 * (t["fetch_kib"] * t["fetch_scale"] + t["write_kib"] * t["write_scale"])


def parse():
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=20)
    ap.add_argument("--warmup", type=int, default=5)
    ap.add_argument("--warm-seconds", type=float, default=0.3,
                    help="keep running warmup steps until this much wall time has passed")
    ap.add_argument("--workload", default="layer",
                    choices=["layer", "small", "ln_qkv", "causal_softmax_pv", "ffn_prefill",
                             "ffn_decode_t1", "ffn_decode_t4", "ffn_decode_t16", "qkv_t32", "qkv_t128",
                             "qkv_t1024", "rms_qkv",
                             "rms_ffn_decode_t1", "swiglu_prefill", "swiglu_decode_t1", "causal_attention",
                             "decode_attention", "decode_attention_gqa"])
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-unfused", action="store_true")
    ap.add_argument("--path", default="fused", choices=["fused", "unfused", "library"],
                    help="what the timed steps run: the deferred kernels (default), the unfused "
                         "comparators, or (LN workloads) the plain product from the vendor library "
                         "-- for profiling each on its own")
    ap.add_argument("--no-workloads", action="store_true",
                    help="skip the other named workloads (timed on their own after the layer step)")
    ap.add_argument("--cpu-threads", type=int, default=None)
    ap.add_argument("--cpu-seconds", type=float, default=12.0,
                    help="approximate CPU time of the oracle sample behind cpu_baseline")
    ap.add_argument("--calib-copy-mib", type=int, default=0,
                    help="after the timed steps, copy a buffer of this many MiB twice (a plain copy "
                         "kernel of known size, to scale hardware traffic counters)")
    return ap.parse_args()


# ------------------------------------------------------------------------------ workloads
def ln_bytes(w) -> float:
    """Algorithmic bytes of deferred LN->Linear: read x and W' (+c, b), write out."""
    es = 4 if w.dtype == "f32" else 2
    return es * (w.M * w.K + w.K * w.N + w.M * w.N) + 8.0 * w.N


def sm_bytes(w) -> float:
    """Algorithmic bytes of deferred Softmax->P.V: the kept scores, V, and the output."""
    return 2.0 * (w.pairs() + 2.0 * w.BH * w.L * w.d)


class LNSite:
    """LayerNorm -> Linear (Eq. (5)), or RMSNorm -> Linear (Eq. (6)) when the workload says so."""

    def __init__(self, ops, I, w, case=None, copies=1):
        """case: the workload's tensors when already generated; copies: how many separately
        prepared copies of the static weights the calls rotate through (HBM-bound shapes take
        enough of them that the weights cannot stay in the 256 MB last-level cache)."""
        self.w = w
        self.rms = w.norm == "rms"
        self.kernel = "rms_linear_deferred" if self.rms else "ln_linear_deferred"
        self.case = I.make_ln(w) if case is None else case
        c = self.case
        cuda = lambda t: None if t is None else t.cuda()
        self.x = c["x"].cuda()
        W = c["W"].cuda()
        self.g, self.b = c["gamma"].cuda(), cuda(c["beta"])
        self.bias = cuda(c["bias"])
        self.preps = [ops.ln_linear_prepare(W, self.g, self.b, self.bias) for _ in range(copies)]
        self.prep = self.preps[0]
        self.out = torch.empty((w.M, w.N), dtype=self.x.dtype, device="cuda")
        # unfused comparator: the same static weights packed the same way (gamma = 1 folds
        # nothing), so both paths run the same weight layout and MFMA main loop
        one = torch.ones(w.K, dtype=W.dtype, device="cuda")
        self.Wpks = [ops.ln_linear_prepare(W, one) for _ in range(copies)]
        # vendor-library reference for the plain product (hipBLASLt through torch), on
        # MFMA-bound bf16 shapes: W^T stored [N][K], the layout the library runs fastest
        self.Wt = W.t().contiguous() if self.library_supported() else None
        del W
        self.copies, self.it = copies, 0
        self.y = torch.empty_like(self.x)
        self.stats = torch.empty(2 * w.M, dtype=torch.float32, device="cuda")
        self.ops = ops
        torch.cuda.synchronize()

    def _next(self):
        """Index of the weight copy for this call (round robin)."""
        self.it = (self.it + 1) % self.copies
        return self.it

    def serial(self):
        # ablation: the row statistics in a pre-pass kernel, then the same deferred epilogue
        self.ops.ln_linear_serial(self.x, self.preps[self._next()], self.w.eps, stats=self.stats, out=self.out)

    def on_load_supported(self):
        return (not self.rms and self.w.dtype == "bf16" and self.w.K % 64 == 0
                and ((self.w.M + 255) // 256) * ((self.w.N + 255) // 256) >= 256)

    def post(self):
        # post-LN placement: the deferred product plus the normalized rows (the residual branch)
        self.ops.linear_deferred_post(self.x, self.preps[self._next()], self.g, None if self.rms else self.b,
                                      self.w.eps,
                                      rms=self.rms, stats=self.stats, y=self.y, out=self.out)

    def norm_on_load(self):
        # ablation without deferral: pre-pass statistics, x normalized on load into the product
        self.ops.ln_linear_norm_on_load(self.x, self.preps[self._next()], self.w.eps, stats=self.stats,
                                        out=self.out)

    def fused(self):
        f = self.ops.rms_linear_deferred if self.rms else self.ops.ln_linear_deferred
        f(self.x, self.preps[self._next()], self.w.eps, out=self.out)

    def gemm_only(self):
        # the product alone on the same packed weights: no statistics, no normalization
        self.ops.gemm(self.x, self.Wpks[self._next()], self.bias, out=self.out.view(1, self.w.M, self.w.N))

    def library_supported(self):
        return self.w.dtype == "bf16" and self.w.M > 128

    def library(self):
        # the same plain product (x . W + bias, bf16 out) from the vendor library: a reference for
        # what the chip's own GEMM reaches on this shape, not part of the deferred path
        if self.bias is None:
            torch.matmul(self.x, self.Wt.t(), out=self.out)
        else:
            torch.addmm(self.bias, self.x, self.Wt.t(), out=self.out)

    def unfused(self):
        if self.rms:
            self.ops.rmsnorm(self.x, self.g, self.w.eps, out=self.y)
        else:
            self.ops.layernorm(self.x, self.g, self.b, self.w.eps, out=self.y)
        self.ops.gemm(self.y, self.Wpks[self._next()], self.bias, out=self.out.view(1, self.w.M, self.w.N))

    def flops(self):
        return self.w.flops()

    def bytes(self):
        return ln_bytes(self.w)

    def peak_tflops(self):
        return PEAK_F32_TFLOPS if self.w.dtype == "f32" else PEAK_BF16_TFLOPS

    def oracle_sample(self, oracle, I, threads, rows):
        idx = I.sample_rows(self.w.M, rows, seed=7)
        c = self.case
        xs = c["x"][torch.as_tensor(idx)]
        t0 = time.perf_counter()
        if self.rms:
            oracle.rms_linear(xs, c["gamma"], c["W"], c["bias"], c["eps"], nthreads=threads)
        else:
            oracle.ln_linear(xs, c["gamma"], c["beta"], c["W"], c["bias"], c["eps"], nthreads=threads)
        dt = time.perf_counter() - t0
        norm = "RMSNorm" if self.rms else "LayerNorm"
        return dt, len(idx) / self.w.M, f"{len(idx)} of {self.w.M} {norm}->Linear rows"


class SwiGLUSite:
    """RMSNorm -> gate and up projections -> SiLU(gate) * up, the Llama MLP input stage."""
    kernel = "rms_swiglu_deferred"

    def __init__(self, ops, I, w):
        self.w = w
        self.case = I.make_swiglu(w)
        c = self.case
        self.x = c["x"].cuda()
        Wg, Wu, self.g = c["Wg"].cuda(), c["Wu"].cuda(), c["gamma"].cuda()
        self.prep = ops.swiglu_prepare(Wg, Wu, self.g)
        one = torch.ones(w.K, dtype=Wg.dtype, device="cuda")
        self.Wg_pk, self.Wu_pk = ops.ln_linear_prepare(Wg, one), ops.ln_linear_prepare(Wu, one)
        del Wg, Wu
        self.out = torch.empty((w.M, w.N), dtype=self.x.dtype, device="cuda")
        self.y = torch.empty_like(self.x)
        self.gate = torch.empty((1, w.M, w.N), dtype=self.x.dtype, device="cuda")
        self.up = torch.empty_like(self.gate)
        self.ops = ops
        torch.cuda.synchronize()

    def fused(self):
        self.ops.rms_swiglu_deferred(self.x, self.prep, self.w.eps, out=self.out)

    def unfused(self):
        self.ops.rmsnorm(self.x, self.g, self.w.eps, out=self.y)
        self.ops.gemm(self.y, self.Wg_pk, out=self.gate)
        self.ops.gemm(self.y, self.Wu_pk, out=self.up)
        self.ops.silu_mul(self.gate, self.up, out=self.out.view(1, self.w.M, self.w.N))

    def flops(self):
        return 2.0 * self.w.flops()

    def bytes(self):
        w = self.w
        return 2.0 * (w.M * w.K + 2 * w.K * w.N + w.M * w.N) + 16.0 * w.N

    def peak_tflops(self):
        return PEAK_BF16_TFLOPS

    def oracle_sample(self, oracle, I, threads, rows):
        idx = I.sample_rows(self.w.M, rows, seed=9)
        c = self.case
        t0 = time.perf_counter()
        oracle.rms_swiglu(c["x"][torch.as_tensor(idx)], c["gamma"], c["Wg"], c["Wu"], c["eps"], nthreads=threads)
        dt = time.perf_counter() - t0
        return dt, len(idx) / self.w.M, f"{len(idx)} of {self.w.M} RMSNorm->SwiGLU rows"


class SMSite:
    def __init__(self, ops, I, w):
        self.w = w
        self.case = I.make_sm(w)
        self.S = self.case["S"].cuda()
        self.V = self.case["V"].cuda()
        self.out = torch.empty((w.BH, w.L, w.d), dtype=torch.bfloat16, device="cuda")
        self.P = torch.empty_like(self.S)
        self.ops = ops
        torch.cuda.synchronize()

    def fused(self):
        self.ops.softmax_pv_deferred(self.S, self.V, causal=self.w.causal, out=self.out)

    def unfused(self):
        # strongest conventional pair: softmax writes the kept triangle, the GEMM skips masked tiles
        self.ops.softmax(self.S, causal=2 if self.w.causal else 0, out=self.P)
        self.ops.gemm(self.P, self.V, a_causal=self.w.causal, out=self.out)

    def unfused_dense(self):
        # the eager conventional pair: dense probabilities (zeros above the diagonal), dense GEMM
        self.ops.softmax(self.S, causal=1 if self.w.causal else 0, out=self.P)
        self.ops.gemm(self.P, self.V, out=self.out)

    def flops(self):
        return self.w.flops()

    def bytes(self):
        return sm_bytes(self.w)

    def peak_tflops(self):
        return PEAK_BF16_TFLOPS

    def oracle_sample(self, oracle, I, threads, rows):
        w = self.w
        idx = I.sample_rows(w.BH * w.L, rows, seed=8)
        head, q = idx // w.L, idx % w.L
        S_rows = self.case["S"].reshape(w.BH * w.L, w.L)[torch.as_tensor(idx)]
        t0 = time.perf_counter()
        oracle.softmax_pv(S_rows, self.case["V"], head=head, qpos=q if w.causal else None, nthreads=threads)
        dt = time.perf_counter() - t0
        kept = float(np.sum(q + 1)) if w.causal else float(len(idx) * w.L)
        return dt, kept / w.pairs(), f"{len(idx)} of {w.BH * w.L} Softmax->P.V rows"


class AttnSite:
    """Attention with the scores formed in the kernel (Q, K, V in; S never stored)."""
    kernel = "attention_deferred"

    def __init__(self, ops, I, w):
        self.w = w
        self.case = I.make_qkv(w)
        c = self.case
        self.Q, self.K, self.V = c["Q"].cuda(), c["K"].cuda(), c["V"].cuda()
        self.out = torch.empty_like(self.Q)
        # conventional comparators: S = (scale Q) K^T stored (the scale folded into Q once, untimed),
        # then the deferred Softmax -> P.V on S, or softmax + P.V
        self.Qs = (self.Q.float() * c["scale"]).to(torch.bfloat16)
        self.S = torch.empty((w.BH, w.L, w.L), dtype=torch.bfloat16, device="cuda")
        self.P = torch.empty_like(self.S)
        self.ops = ops
        torch.cuda.synchronize()

    def fused(self):
        self.ops.attention_deferred(self.Q, self.K, self.V, causal=self.w.causal, scale=self.case["scale"],
                                    out=self.out)

    def unfused(self):
        # the materialized-score path: QK^T GEMM writes S, then deferred Softmax -> P.V reads it
        self.ops.gemm(self.Qs, self.K, b_layout=1, out=self.S)
        self.ops.softmax_pv_deferred(self.S, self.V, causal=self.w.causal, out=self.out)

    def unfused_dense(self):
        # the eager conventional chain: QK^T, softmax (dense P), P.V
        self.ops.gemm(self.Qs, self.K, b_layout=1, out=self.S)
        self.ops.softmax(self.S, causal=1 if self.w.causal else 0, out=self.P)
        self.ops.gemm(self.P, self.V, out=self.out)

    def flops(self):
        return 2.0 * self.w.flops()

    def bytes(self):
        w = self.w
        return 2.0 * 4 * w.BH * w.L * w.d

    def peak_tflops(self):
        return PEAK_BF16_TFLOPS

    def oracle_sample(self, oracle, I, threads, rows):
        w = self.w
        idx = I.sample_rows(w.BH * w.L, rows, seed=10)
        head, q = idx // w.L, idx % w.L
        Qr = self.case["Q"].reshape(w.BH * w.L, w.d)[torch.as_tensor(idx)]
        t0 = time.perf_counter()
        oracle.attention(Qr, self.case["K"], self.case["V"], self.case["scale"], head=head,
                         qpos=q if w.causal else None, nthreads=threads)
        dt = time.perf_counter() - t0
        kept = float(np.sum(q + 1)) if w.causal else float(len(idx) * w.L)
        return dt, kept / w.pairs(), f"{len(idx)} of {w.BH * w.L} attention rows"


class DecodeAttnSite:
    """Decode attention: the keys of each head split over enough workgroups to fill the chip, partials
    merged (Eq. (8) over key ranges); 256 heads at d = 128 fill it with one workgroup per head."""
    kernel = "attention_decode_deferred"

    def __init__(self, ops, I, w):
        self.w = w
        self.case = I.make_decode(w)
        c = self.case
        self.Q, self.K, self.V = c["Q"].cuda(), c["K"].cuda(), c["V"].cuda()
        self.out = torch.empty_like(self.Q)
        self.ws = torch.empty(ops.attention_decode_workspace_bytes(w.BH, w.group * w.Lq, w.Lk, w.d),
                              dtype=torch.uint8, device="cuda")
        # conventional comparator: S = (scale Q) K^T stored, then deferred Softmax -> P.V on S (the
        # query heads of one key/value head batched together as its rows)
        gq = w.group * w.Lq
        self.Qs = (self.Q.float() * c["scale"]).to(torch.bfloat16).reshape(w.BH, gq, w.d)
        self.S = torch.empty((w.BH, gq, w.Lk), dtype=torch.bfloat16, device="cuda")
        self.Qg, self.out_g = self.Q.reshape(w.BH, gq, w.d), self.out.view(w.BH, gq, w.d)
        self.ops = ops
        torch.cuda.synchronize()

    def fused(self):
        self.ops.attention_decode_deferred(self.Q, self.K, self.V, scale=self.case["scale"], workspace=self.ws,
                                           out=self.out)

    def unfused(self):
        self.ops.gemm(self.Qs, self.K, b_layout=1, out=self.S)
        self.ops.softmax_pv_deferred(self.S, self.V, out=self.out_g)

    def single_pass(self):
        # ablation: the same computation without the key split (one workgroup per key/value head)
        self.ops.attention_deferred(self.Qg, self.K, self.V, causal=False, scale=self.case["scale"], out=self.out_g)

    def flops(self):
        return self.w.flops()

    def bytes(self):
        return self.w.bytes()

    def peak_tflops(self):
        return PEAK_BF16_TFLOPS

    def oracle_sample(self, oracle, I, threads, rows):
        w = self.w
        gq = w.group * w.Lq
        heads = I.sample_rows(w.BH, max(1, rows // gq), seed=12)
        hsel = torch.as_tensor(heads)
        Qg = self.case["Q"].reshape(w.BH, gq, w.d)[hsel].reshape(-1, w.d)
        t0 = time.perf_counter()
        oracle.attention(Qg, self.case["K"][hsel], self.case["V"][hsel], self.case["scale"],
                         head=np.repeat(np.arange(len(heads)), gq), nthreads=threads)
        dt = time.perf_counter() - t0
        return dt, len(heads) / w.BH, f"{len(heads)} of {w.BH} decode key/value heads"


def build_sites(ops, I, name):
    if name == "layer":
        return [LNSite(ops, I, I.LN_QKV), SMSite(ops, I, I.SM_CAUSAL)], \
            "llama7b-class layer: LN->QKV x[4096,4096].W[4096,12288] + causal softmax->PV 32h x 8192 x 8192, d128"
    if name == "small":
        return [LNSite(ops, I, I.LN_F32_SMALL), SMSite(ops, I, I.SM_BF16_SMALL)], \
            "small: LN->Linear fp32 x[128,768].W[768,3072] + softmax->PV 12h x 512 x 512, d64"
    if name == "ln_qkv":
        return [LNSite(ops, I, I.LN_QKV)], I.LN_QKV.name
    if name == "causal_softmax_pv":
        return [SMSite(ops, I, I.SM_CAUSAL)], I.SM_CAUSAL.name
    if name == "ffn_prefill":
        return [LNSite(ops, I, I.LN_FFN_PREFILL)], I.LN_FFN_PREFILL.name
    if name == "rms_qkv":
        return [LNSite(ops, I, I.RMS_QKV)], I.RMS_QKV.name
    if name == "causal_attention":
        return [AttnSite(ops, I, I.ATTN_CAUSAL)], I.ATTN_CAUSAL.name
    if name == "decode_attention":
        return [DecodeAttnSite(ops, I, I.ATTN_DECODE)], I.ATTN_DECODE.name
    if name == "decode_attention_gqa":
        return [DecodeAttnSite(ops, I, I.ATTN_DECODE_GQA)], I.ATTN_DECODE_GQA.name
    if name == "swiglu_prefill":
        return [SwiGLUSite(ops, I, I.SWIGLU_PREFILL)], I.SWIGLU_PREFILL.name
    if name == "swiglu_decode_t1":
        w = I.swiglu_decode(1)
        return [SwiGLUSite(ops, I, w)], w.name
    t = int(name.rsplit("t", 1)[1])
    if name.startswith("qkv_"):
        w = I.ln_qkv_tokens(t)
    else:
        w = I.rms_ffn_decode(t) if name.startswith("rms_") else I.ln_ffn_decode(t)
    return [LNSite(ops, I, w, copies=weight_copies(w))], w.name


# ------------------------------------------------------------------------------ timing
def warm(fns, steps, seconds):
    """Untimed: `steps` steps, then more until `seconds` of wall time have passed."""
    t0 = time.perf_counter()
    done = 0
    while done < steps or time.perf_counter() - t0 < seconds:
        for f in fns:
            f()
        done += 1
        if done % 16 == 0:
            torch.cuda.synchronize()
    torch.cuda.synchronize()


def time_steps(fns, steps, warmup, warm_seconds=0.0):
    """Run `fns` in order per step; per-fn HIP-event durations and the total, in ms.

    The total comes from a pass with events only around the K steps; a second
    pass of K steps with an event after every kernel gives the per-kernel times.
    """
    warm(fns, warmup, warm_seconds)
    stream = torch.cuda.current_stream()
    t_begin = torch.cuda.Event(enable_timing=True)
    t_end = torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    t_begin.record(stream)
    for _ in range(steps):
        for f in fns:
            f()
    t_end.record(stream)
    torch.cuda.synchronize()
    total = t_begin.elapsed_time(t_end) / steps
    ev = [[torch.cuda.Event(enable_timing=True) for _ in range(len(fns) + 1)] for _ in range(steps)]
    for s in range(steps):
        ev[s][0].record(stream)
        for i, f in enumerate(fns):
            f()
            ev[s][i + 1].record(stream)
    torch.cuda.synchronize()
    per = [sum(ev[s][i].elapsed_time(ev[s][i + 1]) for s in range(steps)) / steps for i in range(len(fns))]
    return per, total


def weight_copies(w) -> int:
    """Prepared weight copies for an HBM-bound LN shape: enough that the calls rotate through
    about 1 GB of weights, four times the 256 MB last-level cache (1 for MFMA-bound shapes)."""
    es = 4 if w.dtype == "f32" else 2
    peak = PEAK_F32_TFLOPS if w.dtype == "f32" else PEAK_BF16_TFLOPS
    if 2.0 * w.M * w.K * w.N / (es * (w.M * w.K + w.K * w.N + w.M * w.N)) >= peak / PEAK_HBM_GBS * 1e3:
        return 1
    return int(min(16, max(1, -(-1.0e9 // (es * w.K * w.N)))))


def roof_of(s, ms):
    """Bound ("hbm" below the ridge point of the site's arithmetic intensity, else "mfma"), the
    achieved rate at `ms` per launch and its fraction of that roof's peak."""
    hbm = isinstance(s, (SMSite, DecodeAttnSite)) or \
        s.flops() / s.bytes() < s.peak_tflops() * 1e12 / (PEAK_HBM_GBS * 1e9)
    if hbm:
        a = s.bytes() / (ms * 1e-3) / 1e9
        return {"bound": "hbm", "achieved": round(a, 1), "unit": "GB/s", "peak": PEAK_HBM_GBS,
                "frac": round(a / PEAK_HBM_GBS, 4)}
    a = s.flops() / (ms * 1e-3) / 1e12
    return {"bound": "mfma", "achieved": round(a, 2), "unit": "TFLOP/s", "peak": s.peak_tflops(),
            "frac": round(a / s.peak_tflops(), 4)}


def workload_entries(ops, I, steps):
    """The other named workloads, each timed on its own (isolated median over ROUNDS rounds) with its
    unfused comparator: LayerNorm -> Linear fp32 128 x 768 x 3072, Softmax -> P.V 12 x 512 x 512
    (d 64), the LayerNorm -> FFN up-projection 8192 -> 28672 over 8192 tokens (prefill) and over
    1, 4 and 16 tokens (decode, rotating through weight copies so every call streams W' from HBM).
    The decode tokens are the first t rows of the prefill batch (the same stream)."""
    out = {}

    def one(site, extra=None):
        k = isolated(site, steps)
        e = {"isolated_ms": k["isolated_ms"], "isolated_spread_ms": k["isolated_spread_ms"],
             "tflops": round(site.flops() / (k["isolated_ms"] * 1e-3) / 1e12, 2),
             "gbs": round(site.bytes() / (k["isolated_ms"] * 1e-3) / 1e9, 1),
             "alg_gflop": round(site.flops() / 1e9, 3), "alg_mbytes": round(site.bytes() / 1e6, 2)}
        e["roofline"] = roof_of(site, k["isolated_ms"])
        tr = measured_traffic(site.kernel if isinstance(site, LNSite) else "softmax_pv_deferred", site.w.name)
        e["hbm_traffic_mbytes"] = None if tr is None else round(tr / 1e6, 2)
        e.update({a: b for a, b in k.items() if a not in e})
        if extra:
            e.update(extra)
        out[site.w.name] = e
        torch.cuda.synchronize()

    one(LNSite(ops, I, I.LN_F32_SMALL))
    one(SMSite(ops, I, I.SM_BF16_SMALL))
    case = I.make_ln(I.LN_FFN_PREFILL)
    site = LNSite(ops, I, I.LN_FFN_PREFILL, case=case)
    one(site)
    del site
    torch.cuda.empty_cache()
    for t in (1, 4, 16):
        w = I.ln_ffn_decode(t)
        c = dict(case, x=case["x"][:t].clone())
        r = weight_copies(w)
        site = LNSite(ops, I, w, case=c, copies=r)
        one(site, {"weight_copies": r})
        del site
        torch.cuda.empty_cache()
    return out


def copy_bandwidth(mib=1024, reps=10):
    """A plain device-to-device copy of `mib` MiB, event-timed: bytes read + written per second."""
    src = torch.ones(mib << 20, dtype=torch.uint8, device="cuda")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    stream = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    torch.cuda.synchronize()
    a.record(stream)
    for _ in range(reps):
        dst.copy_(src)
    b.record(stream)
    torch.cuda.synchronize()
    ms = a.elapsed_time(b) / reps
    del src, dst
    torch.cuda.empty_cache()
    gbs = 2.0 * (mib << 20) / (ms * 1e-3) / 1e9
    return {"bytes": 2 * (mib << 20), "ms": round(ms, 4), "gbs": round(gbs, 1), "frac_of_spec": round(gbs / PEAK_HBM_GBS, 4)}


def cpu_model() -> str:
    try:
        for ln in open("/proc/cpuinfo"):
            if ln.startswith("model name"):
                return ln.split(":", 1)[1].strip()
    except OSError:
        pass
    return "unknown"


def time_graph(fn, n, replays=3):
    """Mean device time of one call of `fn`, in ms, from `replays` replays of a HIP graph that
    holds n calls: for kernels of a few microseconds, back-to-back calls from Python measure the
    host's launch rate instead (the library allocates nothing and sets no memory, so its launches
    can be recorded)."""
    fn()
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        for _ in range(n):
            fn()
    g.replay()
    torch.cuda.synchronize()
    stream = torch.cuda.current_stream()
    a, b = torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)
    a.record(stream)
    for _ in range(replays):
        g.replay()
    b.record(stream)
    torch.cuda.synchronize()
    return a.elapsed_time(b) / (replays * n)


def floor_us(s) -> float:
    """The site's roofline floor: algorithmic FLOP at the MFMA peak or bytes at the HBM peak."""
    return 1e6 * max(s.flops() / (s.peak_tflops() * 1e12), s.bytes() / (PEAK_HBM_GBS * 1e9))


def isolated(s, steps):
    """Each path of a site timed on its own: the deferred kernel, the unfused comparator and the
    ablations the site supports, alternating over ROUNDS rounds of at least 20 launches; medians
    and min-max spreads over the rounds."""
    k = {}
    # speedups compare like with like: each path timed alone, back to back on its own inputs
    # (inside the step the kernel follows the other site, whose traffic evicts the caches);
    # the paths alternate over ROUNDS rounds and each reports its median
    n = max(20, steps)  # iterations per round (each round: every path, in turn)
    fis, us, uds, sers, sps, nols, posts, gos, libs = [], [], [], [], [], [], [], [], []
    serial = isinstance(s, LNSite) and not s.rms and s.w.K <= 16384
    on_load = serial and s.on_load_supported()
    # kernels whose roofline floor is a few microseconds are timed from graph replays
    graph = floor_us(s) < 20.0
    k["timing"] = "graph replay" if graph else "stream"

    def tm(fn, iters=n):
        return time_graph(fn, iters) if graph else time_steps([fn], iters, 2)[0][0]

    paths = [(fis, s.fused, n), (us, s.unfused, n)]
    if isinstance(s, LNSite):
        paths.append((gos, s.gemm_only, n))
        if s.library_supported():
            paths.append((libs, s.library, n))
    if isinstance(s, (SMSite, AttnSite)) and s.w.causal:
        paths.append((uds, s.unfused_dense, max(3, n // 2)))
    if serial:
        paths.append((sers, s.serial, n))
    if isinstance(s, DecodeAttnSite):
        paths.append((sps, s.single_pass, n))
    if on_load:
        paths.append((nols, s.norm_on_load, n))
    if isinstance(s, LNSite):
        paths.append((posts, s.post, n))
    for r in range(ROUNDS):
        # alternate the order round by round, so no path always follows the same one
        for dst, fn, iters in (paths if r % 2 == 0 else paths[::-1]):
            dst.append(tm(fn, iters))
    fi, u = float(np.median(fis)), float(np.median(us))
    k["isolated_ms"] = round(fi, 4)
    k["unfused_ms"] = round(u, 4)
    k["isolated_spread_ms"] = [round(min(fis), 4), round(max(fis), 4)]  # over the rounds
    k["unfused_spread_ms"] = [round(min(us), 4), round(max(us), 4)]
    k["speedup_vs_unfused"] = round(u / fi, 3)
    if gos:  # the product alone: what deferral adds on top of it
        go = float(np.median(gos))
        k["gemm_only_ms"] = round(go, 4)
        k["deferred_overhead_us"] = round(1e3 * (fi - go), 1)
    if libs:  # reference: the plain product from the vendor library (no normalization)
        lb = float(np.median(libs))
        k["library_gemm_ms"] = round(lb, 4)
        k["library_gemm_tflops"] = round(s.flops() / (lb * 1e-3) / 1e12, 2)
    if uds:
        ud = float(np.median(uds))
        k["unfused_dense_ms"] = round(ud, 4)
        k["speedup_vs_unfused_dense"] = round(ud / fi, 3)
    if sers:  # ablation: statistics from a pre-pass instead of concurrently
        se = float(np.median(sers))
        k["serial_stats_ms"] = round(se, 4)
        k["speedup_vs_serial_stats"] = round(se / fi, 3)
    if posts:  # post-LN placement: deferred product + normalized rows, against the unfused pair
        po = float(np.median(posts))
        k["post_ln_ms"] = round(po, 4)
        k["post_ln_speedup_vs_unfused"] = round(u / po, 3)
    if nols:  # ablation: fused without deferral (normalize on load)
        nl = float(np.median(nols))
        k["norm_on_load_ms"] = round(nl, 4)
        k["speedup_vs_norm_on_load"] = round(nl / fi, 3)
    if sps:  # ablation: no key split (one workgroup per head)
        sp = float(np.median(sps))
        k["single_pass_ms"] = round(sp, 4)
        k["speedup_vs_single_pass"] = round(sp / fi, 3)
    return k


def main():
    args = parse()
    if args.gpus != 1:
        print(f"bench.py measures one GPU: the kernels run on a single MI355X and there is no multi-GPU path "
              f"(asked for --gpus {args.gpus}).", file=sys.stderr)
        sys.exit(2)
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        sys.exit(2)
    from paper_2502_17728_amd import inputs as I
    from paper_2502_17728_amd import ops

    t_setup = time.perf_counter()
    sites, wl_name = build_sites(ops, I, args.workload)
    setup_s = time.perf_counter() - t_setup

    if args.path == "library" and not all(isinstance(s, LNSite) and s.library_supported() for s in sites):
        print("--path library runs the plain bf16 product of an LN workload with more than 128 rows",
              file=sys.stderr)
        sys.exit(2)
    fns = [{"fused": s.fused, "unfused": s.unfused, "library": getattr(s, "library", None)}[args.path]
           for s in sites]
    per, total = time_steps(fns, args.steps, args.warmup, args.warm_seconds)
    if args.calib_copy_mib > 0:
        src = torch.ones(args.calib_copy_mib << 20, dtype=torch.uint8, device="cuda")
        dst = torch.empty_like(src)
        for _ in range(2):
            dst.copy_(src)
        torch.cuda.synchronize()
        del src, dst
    flops = sum(s.flops() for s in sites)
    value = flops / (total * 1e-3) / 1e12

    kernels = {}
    dom = max(range(len(sites)), key=lambda i: per[i])
    for i, s in enumerate(sites):
        name = s.kernel if isinstance(s, (LNSite, SwiGLUSite, AttnSite, DecodeAttnSite)) else "softmax_pv_deferred"
        tf = s.flops() / (per[i] * 1e-3) / 1e12
        gbs = s.bytes() / (per[i] * 1e-3) / 1e9
        k = {"workload": s.w.name, "ms": round(per[i], 4), "tflops": round(tf, 2),
             "frac_mfma_peak": round(tf / s.peak_tflops(), 4), "gbs": round(gbs, 1),
             "frac_hbm_peak": round(gbs / PEAK_HBM_GBS, 4), "alg_gflop": round(s.flops() / 1e9, 3),
             "alg_mbytes": round(s.bytes() / 1e6, 2)}
        tr = measured_traffic(name, s.w.name)
        k["hbm_traffic_mbytes"] = None if tr is None else round(tr / 1e6, 2)
        if not args.no_unfused:
            k.update(isolated(s, args.steps))
        kernels[name] = k

    d = sites[dom]
    dname = list(kernels)[dom]
    # the roof the dominant kernel's arithmetic intensity (algorithmic FLOP per algorithmic
    # byte) meets first: HBM below the ridge point (peak FLOP/s over peak bytes/s), else MFMA
    hbm_bound = isinstance(d, (SMSite, DecodeAttnSite)) or \
        d.flops() / d.bytes() < d.peak_tflops() * 1e12 / (PEAK_HBM_GBS * 1e9)
    if hbm_bound:
        ach = d.bytes() / (per[dom] * 1e-3) / 1e9
        roof = {"kernel": dname, "bound": "hbm", "achieved": round(ach, 1), "peak": PEAK_HBM_GBS,
                "unit": "GB/s", "frac": round(ach / PEAK_HBM_GBS, 4),
                "traffic": kernels[dname]["hbm_traffic_mbytes"] and round(kernels[dname]["hbm_traffic_mbytes"] * 1e6)}
    else:
        ach = d.flops() / (per[dom] * 1e-3) / 1e12
        pk = d.peak_tflops()
        roof = {"kernel": dname, "bound": "mfma", "achieved": round(ach, 2), "peak": pk,
                "unit": "TFLOP/s", "frac": round(ach / pk, 4),
                "traffic": kernels[dname]["hbm_traffic_mbytes"] and round(kernels[dname]["hbm_traffic_mbytes"] * 1e6)}

    workloads = None
    if args.workload == "layer" and not args.no_workloads:
        workloads = workload_entries(ops, I, args.steps)
    hbm_copy = copy_bandwidth() if args.workload == "layer" else None

    cpu = None
    if not args.no_cpu_baseline:
        import oracle
        # the host's share of CPU threads for one GPU is 16, whatever the affinity mask shows
        affinity = len(os.sched_getaffinity(0))
        threads = args.cpu_threads or min(16, affinity)
        t_cpu, frac_cpu, descs = 0.0, 0.0, []
        extrap = 0.0
        for s in sites:
            rows = 16 if isinstance(s, (LNSite, SwiGLUSite)) and s.w.K * s.w.N > 1e8 else 64
            if isinstance(s, (LNSite, SwiGLUSite)) and s.w.M <= 16:
                rows = s.w.M
            if isinstance(s, (SMSite, AttnSite)):
                rows = 1024 if s.w.L >= 4096 else 2048
            if isinstance(s, DecodeAttnSite):
                rows = 128
            # a short calibration sample, then one sized to about cpu_seconds / sites of work
            dt, frac, desc = s.oracle_sample(oracle, I, threads, rows)
            budget = args.cpu_seconds / len(sites)
            for _ in range(3):  # fixed costs make small samples look slow per row: refine
                if dt >= 0.5 * budget or frac >= 1.0:
                    break
                rows = max(rows + 1, int(rows * min(budget / max(dt, 1e-3), 1.0 / frac)))
                dt, frac, desc = s.oracle_sample(oracle, I, threads, rows)
            extrap += dt / frac
            descs.append(f"{desc} ({dt:.1f} s)")
        cpu = {"value": round(flops / extrap / 1e12, 6), "unit": "TFLOP/s", "cores": threads, "kind": "oracle",
               "sample": "; ".join(descs) + f"; time extrapolated by work to the whole step "
                         f"({extrap:.1f} s per step on {threads} threads)",
               "cpu_model": cpu_model(), "affinity_cores": affinity}
        # one thread, the whole LayerNorm -> Linear fp32 128 x 768 x 3072 workload
        small = I.make_ln(I.LN_F32_SMALL)
        t0 = time.perf_counter()
        oracle.ln_linear(small["x"], small["gamma"], small["beta"], small["W"], small["bias"], small["eps"],
                         nthreads=1)
        dt1 = time.perf_counter() - t0
        cpu["single_thread"] = {"workload": I.LN_F32_SMALL.name, "s": round(dt1, 3),
                                "tflops": round(I.LN_F32_SMALL.flops() / dt1 / 1e12, 6)}

    line = {
        "metric": METRIC, "value": round(value, 2), "unit": "TFLOP/s", "n_gpus": 1, "steps": args.steps,
        "warmup": args.warmup, "ms_per_step": round(total, 4), "higher_is_better": True, "scaling": "weak",
        "vs_baseline": None, "dtype": "f32" if all(getattr(s.w, "dtype", "bf16") == "f32" for s in sites) else "bf16",
        "data": "synthetic",
        "config": {"workload": wl_name} if args.path == "fused" else {"workload": wl_name, "path": args.path},
        "roofline": roof, "cpu_baseline": cpu, "kernels": kernels, "workloads": workloads, "hbm_copy": hbm_copy,
        "frac_mfma_peak_step": round(value / PEAK_BF16_TFLOPS, 4), "setup_s": round(setup_s, 1),
    }
    print(json.dumps(line), flush=True)


if __name__ == "__main__":
    main()
