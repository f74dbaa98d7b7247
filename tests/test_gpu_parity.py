"""GPU parity: the HIP path, called through the C ABI, against the fp64 oracle.

Small cases span several tiles and ragged tails; the named workloads run at
full size in the bench's launch configuration and every output row is
compared with the oracle.
"""
import os

import numpy as np
import pytest
import torch

import oracle
from paper_2502_17728_amd import inputs as I
from tests.parity import TOL, cuda, rowwise_rel_err

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def ops():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    from paper_2502_17728_amd import ops as _ops
    return _ops


def _ln_check(ops, case, rows=None, tol=None):
    """LayerNorm -> Linear, or RMSNorm -> Linear when case["norm"] == "rms"."""
    rms = case.get("norm") == "rms"
    x, W = cuda(case["x"]), cuda(case["W"])
    w = ops.ln_linear_prepare(W, cuda(case["gamma"]), cuda(case["beta"]), cuda(case["bias"]))
    out = (ops.rms_linear_deferred if rms else ops.ln_linear_deferred)(x, w, case["eps"])
    torch.cuda.synchronize()
    xs = case["x"] if rows is None else case["x"][torch.as_tensor(rows)]
    if rms:
        ref = oracle.rms_linear(xs, case["gamma"], case["W"], case["bias"], case["eps"], beta=case["beta"])
    else:
        ref = oracle.ln_linear(xs, case["gamma"], case["beta"], case["W"], case["bias"], case["eps"])
    got = out.cpu() if rows is None else out.cpu()[torch.as_tensor(rows)]
    err = rowwise_rel_err(got, ref)
    name = "rms_linear_deferred" if rms else "ln_linear_deferred"
    print(f"{name} {tuple(case['x'].shape)}x{tuple(case['W'].shape)} {case['x'].dtype}: err={err:.3e}")
    assert err <= (tol or TOL[case["x"].dtype]), err
    return out, w


# Full-row checks of the large workloads: the oracle's normalization in C, the product as one
# fp64 library matmul (oracle.norm_linear_matmul), compared chunk by chunk over every row.
ORACLE_THREADS = min(16, len(os.sched_getaffinity(0)))


def _all_rows_err(got, ref_rows, M, chunk):
    err = 0.0
    for r0 in range(0, M, chunk):
        r1 = min(M, r0 + chunk)
        err = max(err, rowwise_rel_err(got[r0:r1], ref_rows(r0, r1)))
    return err


def _ln_check_all_rows(ops, case, name, chunk=1024):
    rms = case.get("norm") == "rms"
    x, W = cuda(case["x"]), cuda(case["W"])
    w = ops.ln_linear_prepare(W, cuda(case["gamma"]), cuda(case["beta"]), cuda(case["bias"]))
    del W
    out = (ops.rms_linear_deferred if rms else ops.ln_linear_deferred)(x, w, case["eps"])
    got = out.cpu()
    del out, w, x
    W64 = oracle.to_f64(case["W"])
    M = case["x"].shape[0]
    err = _all_rows_err(got, lambda r0, r1: oracle.norm_linear_matmul(
        case["x"][r0:r1], case["gamma"], case["beta"], W64, case["bias"], case["eps"], rms=rms,
        nthreads=ORACLE_THREADS), M, chunk)
    print(f"{name}: all {M} rows, err={err:.3e}", flush=True)
    assert err <= TOL[case["x"].dtype], err


# ---------------------------------------------------------------------------- LN -> Linear
def test_ln_linear_f32_workload(ops):
    _ln_check(ops, I.make_ln(I.LN_F32_SMALL))


@pytest.mark.parametrize("M,K,N", [(37, 104, 72), (1, 8, 8), (300, 512, 200)])
def test_ln_linear_f32_ragged(ops, M, K, N):
    _ln_check(ops, I.make_ln_case(M, K, N, "f32", seed=M))


@pytest.mark.parametrize("M,K,N", [(17, 64, 136), (200, 520, 392), (200, 512, 392), (129, 256, 8),
                                   (257, 1024, 264), (300, 72, 8),
                                   (128, 768, 3072), (1, 8, 8)])
def test_ln_linear_bf16_ragged(ops, M, K, N):
    _ln_check(ops, I.make_ln_case(M, K, N, "bf16", seed=M + K))


# token counts on both sides of each decode-layout switch (16 | 17..32 | 33..48 |
# 49..64 | 65..96 | 97..128 | 129 = the tiled kernels), partial row fragments; K = 8
# leaves most K-slices empty, N = 24 / 520 leave a partial group of column blocks
@pytest.mark.parametrize("M", [1, 3, 4, 5, 8, 9, 16, 17, 32, 33, 48, 49, 63, 64, 65, 81, 96, 97, 127, 128, 129])
@pytest.mark.parametrize("K,N", [(1024, 520), (8200, 64), (8, 24)])
def test_ln_linear_bf16_decode_shapes(ops, M, K, N):
    _ln_check(ops, I.make_ln_case(M, K, N, "bf16", seed=M * 7 + 1, outliers=4))


@pytest.mark.parametrize("M,N", [(100, 20352), (100, 20608), (128, 20352)])
def test_ln_linear_bf16_batched_decode_switch(ops, M, N):
    # 65-128 tokens take the streaming kernel below 160 tiles of 128 x 128 (159 here) and
    # the tiled kernel from 160 tiles (161)
    _ln_check(ops, I.make_ln_case(M, 256, N, "bf16", seed=N % 97, outliers=2))


def test_ln_linear_bf16_outliers(ops):
    _ln_check(ops, I.make_ln_case(96, 2048, 384, "bf16", seed=5, outliers=8))


def test_ln_linear_mean_offset_stress(ops):
    # rows with mean 4 and unit spread: the deferred form subtracts mean*c after
    # the product, losing about (|mean|/std) * 2^-24 * sqrt(K) relative; well
    # inside the bf16 bound, and documented as the method's cancellation limit
    _ln_check(ops, I.make_ln_case(64, 1024, 256, "bf16", seed=9, mean_offset=4.0))


def test_ln_linear_constant_rows_give_b(ops):
    case = I.make_ln_case(20, 256, 136, "bf16", seed=11)
    case["x"] = torch.full_like(case["x"], 0.75)
    _ln_check(ops, case)


@pytest.mark.parametrize("M,K,N", [(4000, 544, 4104), (4000, 520, 4104), (4096, 4096, 4096)])
def test_ln_linear_bf16_large_tiles(ops, M, K, N):
    # >= 256 output tiles of 256x256: the pipelined main loop with ragged M and N (K % 32 == 0);
    # K = 520 takes the 128x128 loop with its K tail
    case = I.make_ln_case(M, K, N, "bf16", seed=M % 97, outliers=3)
    _ln_check(ops, case)


# K >= 8192 on the 256x256 loop, one tile per workgroup and the row moments shared between the
# column groups of each row block: (2100, 8256, 4200) ragged M and N over 9 x 17 tiles,
# (2048, 8192, 4096) 8 x 16; every 7th row (all 16-row fragments of every row block) against the
# oracle
@pytest.mark.parametrize("M,K,N,norm", [(2100, 8256, 4200, "layernorm"), (2048, 8192, 4096, "layernorm"),
                                        (2100, 8256, 4200, "rms")])
def test_norm_linear_bf16_long_k(ops, M, K, N, norm):
    case = I.make_ln_case(M, K, N, "bf16", seed=M % 91, outliers=3, norm=norm)
    _ln_check(ops, case, rows=np.arange(0, M, 7))


@pytest.mark.parametrize("M,K,N,layout", [(4104, 320, 4096, 2), (4104, 264, 4096, 2), (4104, 264, 4096, 1),
                                           (300, 136, 264, 2), (257, 512, 1032, 2), (2100, 8256, 4200, 2)])
def test_gemm_large(ops, M, K, N, layout):
    # layout 2 (packed weights, gamma = 1) with K % 64 == 0 runs the pipelined loop, on
    # 256 x 256 tiles at 4104 rows and at 2100 x 4200 with K = 8256 (every 7th row checked) and
    # on 128 x 128 tiles at 257 x 1032 (27 tiles); K = 264 and K = 136 run the two-stage
    # 128 x 128 loop
    g = torch.Generator().manual_seed(5)
    A = torch.randn(M, K, generator=g).to(torch.bfloat16)
    B = torch.randn(K, N, generator=g).to(torch.bfloat16)
    bias = torch.randn(N, generator=g).to(torch.bfloat16)
    if layout == 2:
        Bd = ops.ln_linear_prepare(cuda(B), torch.ones(K, dtype=torch.bfloat16, device="cuda"))
    else:
        Bd = cuda(B.t().contiguous())
    C = ops.gemm(cuda(A), Bd, cuda(bias), b_layout=layout)
    rows = torch.arange(0, M, 7) if K > 4096 else torch.arange(M)
    ref = oracle.to_f64(A[rows]) @ oracle.to_f64(B) + oracle.to_f64(bias)
    assert rowwise_rel_err(C.cpu()[rows], ref) <= TOL[torch.bfloat16]


@pytest.mark.parametrize("M,K,N", [(1, 1024, 520), (5, 8200, 264), (16, 512, 72), (3, 8, 8), (17, 1024, 520),
                                   (40, 2048, 264), (64, 512, 4104), (90, 1024, 520), (128, 512, 4104)])
def test_gemm_packed_decode(ops, M, K, N):
    # decode shapes with packed weights: the streaming kernel without moments (the unfused
    # comparators' GEMM at M <= 128), bias added once; ragged N and K
    g = torch.Generator().manual_seed(M + K)
    A = torch.randn(M, K, generator=g).to(torch.bfloat16)
    B = (torch.randn(K, N, generator=g) / K ** 0.5).to(torch.bfloat16)
    bias = torch.randn(N, generator=g).to(torch.bfloat16)
    Bd = ops.ln_linear_prepare(cuda(B), torch.ones(K, dtype=torch.bfloat16, device="cuda"))
    C = ops.gemm(cuda(A), Bd, cuda(bias), b_layout=2)
    assert rowwise_rel_err(C.cpu(), oracle.linear(A, B, bias)) <= TOL[torch.bfloat16]


def test_gemm_packed_f32(ops):
    g = torch.Generator().manual_seed(6)
    A, B = torch.randn(45, 72, generator=g), torch.randn(72, 40, generator=g)
    Bd = ops.ln_linear_prepare(cuda(B), torch.ones(72, device="cuda"))
    C = ops.gemm(cuda(A), Bd)
    assert rowwise_rel_err(C.cpu(), oracle.linear(A, B)) <= TOL[torch.float32]


def test_ln_linear_ffn_prefill_workload_all_rows(ops):
    # the 8192 x 8192 x 28672 up-projection at full size in the bench's launch configuration
    # (the 256x256 kernel, 14 column tiles per workgroup), every row against the oracle
    _ln_check_all_rows(ops, I.make_ln(I.LN_FFN_PREFILL), "ln_linear_deferred ffn prefill 8192x8192x28672")


def test_ln_linear_qkv_workload_all_rows(ops):
    _ln_check_all_rows(ops, I.make_ln(I.LN_QKV), "ln_linear_deferred qkv 4096x4096x12288")


@pytest.mark.parametrize("t", [1, 4, 8, 16])
def test_ln_linear_ffn_decode_workload(ops, t):
    _ln_check(ops, I.make_ln(I.ln_ffn_decode(t)))


@pytest.mark.parametrize("t", [32, 128, 1024])
def test_ln_linear_qkv_tokens_workload_all_rows(ops, t):
    # the QKV projection at the bench's batched-decode and prefill-chunk sizes, in the
    # launch configurations it times: 2 and 8 row fragments of the streaming kernel, and
    # 4 x 48 tiles of 256 x 256 (one tile per workgroup, each reducing its rows' moments)
    _ln_check_all_rows(ops, I.make_ln(I.ln_qkv_tokens(t)), f"ln_linear_deferred qkv {t} tokens")


def test_ln_linear_deterministic(ops):
    case = I.make_ln_case(130, 512, 256, "bf16", seed=2)
    x = cuda(case["x"])
    w = ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"]))
    a = ops.ln_linear_deferred(x, w)
    b = ops.ln_linear_deferred(x, w)
    assert torch.equal(a, b)


def test_ln_linear_guard_band(ops):
    case = I.make_ln_case(33, 256, 72, "bf16", seed=4)
    w = ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"]))
    buf = torch.full((33 * 72 + 2 * 512,), 7.0, dtype=torch.bfloat16, device="cuda")
    out = buf[512:512 + 33 * 72].view(33, 72)
    ops.ln_linear_deferred(cuda(case["x"]), w, out=out)
    torch.cuda.synchronize()
    assert (buf[:512] == 7.0).all() and (buf[-512:] == 7.0).all()


# Shared row moments: on the pipelined kernels the workgroups of a row block each reduce a share
# of its rows' moments and exchange them through a device mailbox, every word stamped with its
# call's number.  A bound of 0 on the wait for the peers' shares makes every workgroup reduce all
# its rows itself -- the path taken when a peer is not resident.
@pytest.mark.parametrize("M,K,N", [(4096, 1024, 4096), (300, 256, 4104), (4000, 544, 4104), (520, 256, 8200)])
@pytest.mark.parametrize("norm", ["layernorm", "rms"])
def test_ln_linear_moments_reduced_locally(ops, M, K, N, norm, monkeypatch):
    monkeypatch.setenv("DN_MOMENT_WAIT_TICKS", "0")
    _ln_check(ops, I.make_ln_case(M, K, N, "bf16", seed=M + 5, outliers=3, norm=norm))


def test_swiglu_moments_reduced_locally(ops, monkeypatch):
    monkeypatch.setenv("DN_MOMENT_WAIT_TICKS", "0")
    _swiglu_check(ops, I.make_swiglu_case(1100, 512, 2056, "bf16", seed=6, outliers=2))


def test_ln_linear_shared_moments_follow_each_call(ops):
    # calls of one shape on different rows, back to back: each call's workgroups take only
    # their own call's moments (a stale share would shift whole rows), and a repeated call
    # gives the same bits
    a = I.make_ln_case(4096, 512, 4104, "bf16", seed=40, outliers=2)
    b = I.make_ln_case(4096, 512, 4104, "bf16", seed=41, outliers=2, mean_offset=1.0)
    w = ops.ln_linear_prepare(cuda(a["W"]), cuda(a["gamma"]), cuda(a["beta"]))
    xa, xb = cuda(a["x"]), cuda(b["x"])
    oa = ops.ln_linear_deferred(xa, w, a["eps"])
    ob = ops.ln_linear_deferred(xb, w, a["eps"])
    oa2 = ops.ln_linear_deferred(xa, w, a["eps"])
    torch.cuda.synchronize()
    for x, out in ((a["x"], oa), (b["x"], ob)):
        ref = oracle.ln_linear(x, a["gamma"], a["beta"], a["W"], None, a["eps"])
        assert rowwise_rel_err(out.cpu(), ref) <= TOL[torch.bfloat16]
    assert torch.equal(oa, oa2)


def test_ln_linear_graph_replays_follow_new_inputs(ops):
    # a deferred LayerNorm product recorded in a HIP graph (a shape that takes the row-moment
    # exchange when launched directly) and replayed on new contents of the same x buffer: every
    # replay normalizes with the new rows' statistics; eager work and a synchronization run
    # between the replays
    cases = [I.make_ln_case(1024, 512, 4096, "bf16", seed=60 + i, outliers=2, mean_offset=0.5 * i)
             for i in range(3)]
    a = cases[0]
    w = ops.ln_linear_prepare(cuda(a["W"]), cuda(a["gamma"]), cuda(a["beta"]))
    x = cuda(a["x"])
    out = torch.empty((1024, 4096), dtype=torch.bfloat16, device="cuda")
    ops.ln_linear_deferred(x, w, a["eps"], out=out)  # first call outside the capture
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ops.ln_linear_deferred(x, w, a["eps"], out=out)
    for rep in range(2):
        for c in cases:
            x.copy_(cuda(c["x"]))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            eager = ops.ln_linear_deferred(x, w, a["eps"])
            torch.cuda.synchronize()
            ref = oracle.ln_linear(c["x"], a["gamma"], a["beta"], a["W"], None, a["eps"])
            err, err_e = rowwise_rel_err(out.cpu(), ref), rowwise_rel_err(eager.cpu(), ref)
            print(f"graph replay {rep}: err={err:.3e}, eager err={err_e:.3e}")
            assert err <= TOL[torch.bfloat16] and err_e <= TOL[torch.bfloat16], (err, err_e)


# Non-finite inputs propagate as in the plain definition (Eq. (1)-(2), Eq. (6)): a row holding
# NaN, +inf or -inf gives an all-NaN output row and leaves every other row untouched; with
# eps = 0 a constant row (LayerNorm: zero variance) or an all-zero row (RMSNorm) gives 0/0 = NaN.
# The shapes take every kernel: fp32 tiles, the 128 x 128 two-stage loop (K % 64 != 0), the
# pipelined 128 x 128 and 256 x 256 kernels, and the decode kernel with 1 and 3 row fragments.
NONFINITE_SHAPES = [(37, 104, 72, "f32"), (200, 520, 392, "bf16"), (300, 256, 4104, "bf16"),
                    (520, 256, 8200, "bf16"), (5, 1024, 520, "bf16"), (40, 1024, 520, "bf16")]


@pytest.mark.parametrize("M,K,N,dtype", NONFINITE_SHAPES)
@pytest.mark.parametrize("norm", ["layernorm", "rms"])
def test_ln_linear_nonfinite_rows(ops, M, K, N, dtype, norm):
    case = I.make_ln_case(M, K, N, dtype, seed=M + N, outliers=2, norm=norm)
    x = case["x"].clone()
    x[1, K // 3] = float("nan")
    x[2, K - 1] = float("inf")
    x[M - 1, 0] = float("-inf")
    case["x"] = x
    out, _ = _ln_check(ops, case)
    o = out.cpu().float()
    assert torch.isnan(o[[1, 2, M - 1]]).all() and torch.isfinite(o[3:M - 1]).all()


@pytest.mark.parametrize("M,K,N,dtype", NONFINITE_SHAPES)
@pytest.mark.parametrize("norm", ["layernorm", "rms"])
def test_ln_linear_eps0_degenerate_rows(ops, M, K, N, dtype, norm):
    case = I.make_ln_case(M, K, N, dtype, seed=M + K, norm=norm)
    case["eps"] = 0.0
    x = case["x"].clone()
    # values whose sums and squares are exact in fp32, so the one-pass variance is exactly 0
    if norm == "rms":
        x[0] = 0
        x[M - 1] = 0
    else:
        x[0] = 0.75
        x[M - 1] = -1.5
    case["x"] = x
    out, _ = _ln_check(ops, case)
    o = out.cpu().float()
    assert torch.isnan(o[[0, M - 1]]).all() and torch.isfinite(o[1:M - 1]).all()


# ---------------------------------------------------------------------------- ablations
@pytest.mark.parametrize("M,K,N,dtype", [(37, 104, 72, "f32"), (257, 1024, 264, "bf16"), (5, 1024, 520, "bf16"),
                                         (4000, 544, 4104, "bf16")])
def test_ln_linear_centered_weight(ops, M, K, N, dtype):
    # Eq. (5) literally: (I - E/n) Gamma W folded into the static weight, no mean term in the epilogue
    case = I.make_ln_case(M, K, N, dtype, seed=M + 3, outliers=2)
    w = ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"]), centered=True)
    out = ops.ln_linear_deferred(cuda(case["x"]), w, case["eps"])
    ref = oracle.ln_linear(case["x"], case["gamma"], case["beta"], case["W"], None, case["eps"])
    assert rowwise_rel_err(out.cpu(), ref) <= TOL[case["x"].dtype]


def test_centered_weight_loses_accuracy_on_offset_rows(ops):
    # rows with mean 4 and unit spread: the rounded W'' columns no longer sum to 0, an error of
    # about |mean|/std * 2^-9 that the mean * c epilogue (c summed from the rounded W') cancels
    case = I.make_ln_case(64, 1024, 256, "bf16", seed=9, mean_offset=4.0)
    x, W, g, b = cuda(case["x"]), cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"])
    ref = oracle.ln_linear(case["x"], case["gamma"], case["beta"], case["W"], None, case["eps"])
    e_epi = rowwise_rel_err(ops.ln_linear_deferred(x, ops.ln_linear_prepare(W, g, b)).cpu(), ref)
    e_lit = rowwise_rel_err(ops.ln_linear_deferred(x, ops.ln_linear_prepare(W, g, b, centered=True)).cpu(), ref)
    print(f"mean-offset rows: epilogue form {e_epi:.3e}, literal Eq. (5) weight {e_lit:.3e}")
    assert e_epi <= TOL[torch.bfloat16] and e_lit <= TOL[torch.bfloat16]
    assert e_epi < e_lit


@pytest.mark.parametrize("M,K,N,dtype", [(37, 104, 72, "f32"), (257, 1024, 264, "bf16"), (3, 1024, 520, "bf16"),
                                         (12, 8200, 64, "bf16"), (45, 1024, 264, "bf16"), (100, 1024, 264, "bf16"),
                                         (4000, 544, 4104, "bf16")])
def test_ln_linear_serial_stats(ops, M, K, N, dtype):
    # statistics from a pre-pass kernel, then the same product and deferred epilogue
    case = I.make_ln_case(M, K, N, dtype, seed=M + 4, outliers=2)
    w = ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"]))
    stats = torch.empty(2 * M, dtype=torch.float32, device="cuda")
    out = ops.ln_linear_serial(cuda(case["x"]), w, case["eps"], stats=stats)
    ref = oracle.ln_linear(case["x"], case["gamma"], case["beta"], case["W"], None, case["eps"])
    assert rowwise_rel_err(out.cpu(), ref) <= TOL[case["x"].dtype]
    st = stats.cpu().double().numpy().reshape(M, 2)
    xd = oracle.to_f64(case["x"])
    np.testing.assert_allclose(st[:, 0], xd.mean(1), rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(st[:, 1], 1 / np.sqrt(xd.var(1) + case["eps"]), rtol=1e-4)


@pytest.mark.parametrize("M,K,N,offset", [(4000, 576, 4104, 0.0), (4104, 320, 4096, 0.0), (4096, 256, 4096, 4.0)])
def test_ln_linear_norm_on_load(ops, M, K, N, offset):
    # ablation without deferral: pre-pass statistics, x normalized on load into the product;
    # ragged M and N over the large tiles, and rows with a large mean (normalized before the
    # product, so no cancellation)
    case = I.make_ln_case(M, K, N, "bf16", seed=M + K, outliers=2, mean_offset=offset)
    w = ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"]))
    stats = torch.empty(2 * M, dtype=torch.float32, device="cuda")
    out = ops.ln_linear_norm_on_load(cuda(case["x"]), w, case["eps"], stats=stats)
    ref = oracle.norm_linear_matmul(case["x"], case["gamma"], case["beta"], case["W"], None, case["eps"])
    err = rowwise_rel_err(out.cpu(), ref)
    print(f"ln_linear_norm_on_load {M}x{K}x{N} offset {offset}: err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err


def test_ln_linear_norm_on_load_qkv_workload_all_rows(ops):
    w = I.LN_QKV
    case = I.make_ln(w)
    prep = ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"]))
    got = ops.ln_linear_norm_on_load(cuda(case["x"]), prep, case["eps"]).cpu()
    W64 = oracle.to_f64(case["W"])
    err = _all_rows_err(got, lambda r0, r1: oracle.norm_linear_matmul(
        case["x"][r0:r1], case["gamma"], case["beta"], W64, None, case["eps"], nthreads=ORACLE_THREADS), w.M, 1024)
    print(f"ln_linear_norm_on_load qkv: all {w.M} rows, err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err


def test_ln_linear_norm_on_load_rejects_small_shapes(ops):
    case = I.make_ln_case(64, 256, 256, "bf16", seed=3)
    w = ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"]))
    with pytest.raises(ops.DNError) as e:
        ops.ln_linear_norm_on_load(cuda(case["x"]), w, case["eps"])
    assert e.value.status == 2  # DN_ERR_UNSUPPORTED: the ablation runs on the large tiles only


# (1024, 512, 4096): 128 x 128 pipelined tiles whose workgroups exchange row moments;
# (4104, 320, 4096): 256 x 256 tiles exchanging them; (100, 1024, 520): 8 decode fragments
@pytest.mark.parametrize("M,K,N,dtype,norm", [(37, 104, 72, "f32", "layernorm"), (257, 1024, 264, "bf16", "layernorm"),
                                              (5, 1024, 520, "bf16", "layernorm"), (50, 1024, 520, "bf16", "layernorm"),
                                              (100, 1024, 520, "bf16", "layernorm"),
                                              (4104, 320, 4096, "bf16", "layernorm"), (1024, 512, 4096, "bf16", "layernorm"),
                                              (1024, 512, 4096, "bf16", "rms"),
                                              (300, 512, 200, "bf16", "rms"), (3, 8200, 64, "bf16", "rms")])
def test_linear_deferred_post(ops, M, K, N, dtype, norm):
    # post-LN placement: the deferred product and the normalized rows (the residual branch) from
    # the statistics the product's kernel reduced; covers the fp32, 128x128, decode and 256x256
    # kernels, each exporting the statistics once per row
    rms = norm == "rms"
    case = I.make_ln_case(M, K, N, dtype, seed=M + K + 7, outliers=2, norm=norm)
    g, b = cuda(case["gamma"]), cuda(case["beta"])
    w = ops.ln_linear_prepare(cuda(case["W"]), g, b, cuda(case["bias"]))
    out, y, st = ops.linear_deferred_post(cuda(case["x"]), w, g, None if rms else b, case["eps"], rms=rms)
    torch.cuda.synchronize()
    xs = case["x"]
    if rms:
        ref = oracle.rms_linear(xs, case["gamma"], case["W"], case["bias"], case["eps"])
        yref = oracle.rmsnorm(xs, case["gamma"], case["eps"])
    else:
        ref = oracle.ln_linear(xs, case["gamma"], case["beta"], case["W"], case["bias"], case["eps"])
        yref = oracle.layernorm(xs, case["gamma"], case["beta"], case["eps"])
    tol = TOL[case["x"].dtype]
    e_out, e_y = rowwise_rel_err(out.cpu(), ref), rowwise_rel_err(y.cpu(), yref)
    print(f"linear_deferred_post {M}x{K}x{N} {dtype} {norm}: out err={e_out:.3e}, y err={e_y:.3e}")
    assert e_out <= tol and e_y <= (tol if dtype == "f32" else tol / 4)
    sd = st.cpu().double().reshape(M, 2).numpy()
    xd = oracle.to_f64(xs)
    mean = np.zeros(len(xd)) if rms else xd.mean(1)
    var = (xd * xd).mean(1) if rms else xd.var(1)
    np.testing.assert_allclose(sd[:, 0], mean, rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(sd[:, 1], 1 / np.sqrt(var + case["eps"]), rtol=1e-4)


def test_linear_deferred_post_qkv_workload_statistics(ops):
    # the row statistics the LN -> QKV workload's kernel reduces (4096 x 4096 x 12288, the
    # bench's launch configuration: 256 x 256 tiles, moments shared between the 16 column
    # groups of each row block), exported and checked on every row: a share of the moments
    # lost or counted twice shifts a row's mean far beyond this bound, where it can hide
    # inside the bf16 tolerance of the outputs
    w = I.LN_QKV
    case = I.make_ln(w)
    g, b = cuda(case["gamma"]), cuda(case["beta"])
    wp = ops.ln_linear_prepare(cuda(case["W"]), g, b, cuda(case["bias"]))
    out, y, st = ops.linear_deferred_post(cuda(case["x"]), wp, g, b, case["eps"])
    torch.cuda.synchronize()
    sd = st.cpu().double().reshape(w.M, 2).numpy()
    del out, wp
    xd = oracle.to_f64(case["x"])
    np.testing.assert_allclose(sd[:, 0], xd.mean(1), rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(sd[:, 1], 1 / np.sqrt(xd.var(1) + case["eps"]), rtol=1e-4)
    yref = oracle.layernorm(case["x"], case["gamma"], case["beta"], case["eps"], nthreads=ORACLE_THREADS)
    assert rowwise_rel_err(y.cpu(), yref) <= TOL[torch.bfloat16] / 4


def test_linear_deferred_post_long_k_statistics(ops):
    # the statistics exported by the 256 x 256 kernel at K = 8192 with the row moments shared
    # between 16 column groups: every row's (mean, rstd) against the definition, the product on
    # every 7th row
    M, K, N = 2048, 8192, 4096
    case = I.make_ln_case(M, K, N, "bf16", seed=17, outliers=2)
    g, b = cuda(case["gamma"]), cuda(case["beta"])
    wp = ops.ln_linear_prepare(cuda(case["W"]), g, b, cuda(case["bias"]))
    out, y, st = ops.linear_deferred_post(cuda(case["x"]), wp, g, b, case["eps"])
    torch.cuda.synchronize()
    sd = st.cpu().double().reshape(M, 2).numpy()
    xd = oracle.to_f64(case["x"])
    np.testing.assert_allclose(sd[:, 0], xd.mean(1), rtol=1e-4, atol=1e-5)
    np.testing.assert_allclose(sd[:, 1], 1 / np.sqrt(xd.var(1) + case["eps"]), rtol=1e-4)
    rows = np.arange(0, M, 7)
    ref = oracle.norm_linear_matmul(case["x"][torch.as_tensor(rows)], case["gamma"], case["beta"],
                                    oracle.to_f64(case["W"]), case["bias"], case["eps"], nthreads=ORACLE_THREADS)
    assert rowwise_rel_err(out.cpu()[torch.as_tensor(rows)], ref) <= TOL[torch.bfloat16]


def test_linear_deferred_post_deterministic(ops):
    case = I.make_ln_case(4104, 320, 4096, "bf16", seed=23)
    g, b = cuda(case["gamma"]), cuda(case["beta"])
    w = ops.ln_linear_prepare(cuda(case["W"]), g, b)
    x = cuda(case["x"])
    r1 = ops.linear_deferred_post(x, w, g, b, case["eps"])
    r2 = ops.linear_deferred_post(x, w, g, b, case["eps"])
    assert all(torch.equal(p, q) for p, q in zip(r1, r2))


# ---------------------------------------------------------------------------- RMSNorm -> Linear
@pytest.mark.parametrize("M,K,N", [(37, 104, 72), (1, 8, 8), (300, 512, 200)])
def test_rms_linear_f32_ragged(ops, M, K, N):
    _ln_check(ops, I.make_ln_case(M, K, N, "f32", seed=M + 1, norm="rms"))


@pytest.mark.parametrize("M,K,N", [(17, 64, 136), (257, 1024, 264), (128, 768, 3072), (1, 8, 8)])
def test_rms_linear_bf16_ragged(ops, M, K, N):
    _ln_check(ops, I.make_ln_case(M, K, N, "bf16", seed=M + K + 1, norm="rms"))


@pytest.mark.parametrize("M", [1, 5, 16, 20, 40, 64, 100, 128])
@pytest.mark.parametrize("K,N", [(1024, 520), (8, 24)])
def test_rms_linear_bf16_decode_shapes(ops, M, K, N):
    _ln_check(ops, I.make_ln_case(M, K, N, "bf16", seed=M * 5 + 2, outliers=4, norm="rms"))


@pytest.mark.parametrize("M,K,N", [(4000, 544, 4104), (4000, 520, 4104)])
def test_rms_linear_bf16_large_tiles(ops, M, K, N):
    case = I.make_ln_case(M, K, N, "bf16", seed=M % 89, outliers=3, norm="rms")
    _ln_check(ops, case)


def test_rms_linear_qkv_workload_all_rows(ops):
    _ln_check_all_rows(ops, I.make_ln(I.RMS_QKV), "rms_linear_deferred qkv 4096x4096x6144")


def test_rms_linear_ffn_decode_workload(ops):
    _ln_check(ops, I.make_ln(I.rms_ffn_decode(1)))


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rms_linear_with_beta_and_bias(ops, dtype):
    # a shift folded at prepare adds beta W for every row, as the oracle's optional beta does
    case = I.make_ln_case(70, 256, 136, dtype, seed=8, norm="rms")
    case["beta"] = I.make_ln_case(1, 256, 8, dtype, seed=9)["beta"]
    case["bias"] = I.make_ln_case(1, 136, 8, dtype, seed=10)["beta"]
    _ln_check(ops, case)


def test_rms_linear_zero_rows_give_b(ops):
    # an all-zero row: sum x^2 = 0, rstd = 1/sqrt(eps) times acc = 0 -> out = b (= bias here)
    case = I.make_ln_case(40, 512, 264, "bf16", seed=14, norm="rms")
    case["x"][3:9] = 0
    case["bias"] = I.make_ln_case(1, 264, 8, "bf16", seed=15)["beta"]
    out, _ = _ln_check(ops, case)
    assert torch.equal(out.cpu()[3:9], case["bias"].expand(6, -1))


# ---------------------------------------------------------------------------- RMSNorm -> SwiGLU
def _swiglu_check(ops, case, rows=None):
    w = ops.swiglu_prepare(cuda(case["Wg"]), cuda(case["Wu"]), cuda(case["gamma"]))
    h = ops.rms_swiglu_deferred(cuda(case["x"]), w, case["eps"])
    torch.cuda.synchronize()
    xs = case["x"] if rows is None else case["x"][torch.as_tensor(rows)]
    ref = oracle.rms_swiglu(xs, case["gamma"], case["Wg"], case["Wu"], case["eps"])
    got = h.cpu() if rows is None else h.cpu()[torch.as_tensor(rows)]
    err = rowwise_rel_err(got, ref)
    print(f"rms_swiglu_deferred {tuple(case['x'].shape)}x{tuple(case['Wg'].shape)} {case['x'].dtype}: err={err:.3e}")
    assert err <= TOL[case["x"].dtype], err
    return h


def test_rms_swiglu_graph_replays_follow_new_inputs(ops):
    # the gated product recorded in a HIP graph (a shape whose direct launches exchange row
    # moments between workgroups) and replayed on new contents of the same x buffer
    cases = [I.make_swiglu_case(1024, 512, 2048, "bf16", seed=70 + i, outliers=2) for i in range(3)]
    a = cases[0]
    w = ops.swiglu_prepare(cuda(a["Wg"]), cuda(a["Wu"]), cuda(a["gamma"]))
    x = cuda(a["x"])
    out = torch.empty((1024, 2048), dtype=torch.bfloat16, device="cuda")
    ops.rms_swiglu_deferred(x, w, a["eps"], out=out)
    torch.cuda.synchronize()
    g = torch.cuda.CUDAGraph()
    with torch.cuda.graph(g):
        ops.rms_swiglu_deferred(x, w, a["eps"], out=out)
    for rep in range(2):
        for c in cases:
            x.copy_(cuda(c["x"]))
            torch.cuda.synchronize()
            g.replay()
            torch.cuda.synchronize()
            ref = oracle.rms_swiglu(c["x"], a["gamma"], a["Wg"], a["Wu"], a["eps"])
            err = rowwise_rel_err(out.cpu(), ref)
            print(f"swiglu graph replay {rep}: err={err:.3e}")
            assert err <= TOL[torch.bfloat16], err


@pytest.mark.parametrize("M,K,N", [(37, 104, 72), (1, 8, 8), (130, 256, 200)])
def test_rms_swiglu_f32_ragged(ops, M, K, N):
    _swiglu_check(ops, I.make_swiglu_case(M, K, N, "f32", seed=M))


# (1, 64, 12304), (16, 128, 28688), (3, 64, 4112): 4, 7 and 2 gate/up pairs per decode
# workgroup, each with a last workgroup holding a single pair
@pytest.mark.parametrize("M,K,N", [(17, 64, 136), (257, 1024, 264), (128, 768, 1032), (1, 8, 8),
                                   (1, 64, 12304), (16, 128, 28688), (3, 64, 4112)])
def test_rms_swiglu_bf16_ragged(ops, M, K, N):
    _swiglu_check(ops, I.make_swiglu_case(M, K, N, "bf16", seed=M + K, outliers=2))


@pytest.mark.parametrize("M", [1, 8, 9, 16, 17, 33, 48, 49, 63, 64, 65, 96, 97, 128])
@pytest.mark.parametrize("K,N", [(1024, 520), (8, 24)])
def test_rms_swiglu_bf16_decode_shapes(ops, M, K, N):
    # 1-7 gate/up pairs per workgroup, 1-8 row fragments (33, 49 and 63 rows leave the last
    # fragment partial under the two-pair layout); N = 520 / 24 leave a partial pair group
    _swiglu_check(ops, I.make_swiglu_case(M, K, N, "bf16", seed=M * 3 + 1, outliers=4))


@pytest.mark.parametrize("M,K,N", [(4000, 544, 2056), (4000, 520, 2056), (2100, 8256, 2104)])
def test_rms_swiglu_bf16_large_tiles(ops, M, K, N):
    # 2 x 2056 packed columns: 16 x 17 tiles of 256 x 256 (pipelined loop, ragged M and N); K = 520
    # takes the 128 x 128 loop; K = 8256 runs 129 stages (every 7th row checked)
    _swiglu_check(ops, I.make_swiglu_case(M, K, N, "bf16", seed=M % 83, outliers=3),
                  rows=np.arange(0, M, 7) if K > 4096 else None)


def test_rms_swiglu_prefill_workload_all_rows(ops):
    w = I.SWIGLU_PREFILL
    case = I.make_swiglu(w)
    pw = ops.swiglu_prepare(cuda(case["Wg"]), cuda(case["Wu"]), cuda(case["gamma"]))
    got = ops.rms_swiglu_deferred(cuda(case["x"]), pw, case["eps"]).cpu()
    del pw
    Wg, Wu = oracle.to_f64(case["Wg"]), oracle.to_f64(case["Wu"])
    err = _all_rows_err(got, lambda r0, r1: oracle.rms_swiglu_matmul(
        case["x"][r0:r1], case["gamma"], Wg, Wu, case["eps"], nthreads=ORACLE_THREADS), w.M, 1024)
    print(f"rms_swiglu_deferred prefill 4096x4096x2x14336: all {w.M} rows, err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err


def test_rms_swiglu_decode_workload(ops):
    _swiglu_check(ops, I.make_swiglu(I.swiglu_decode(1)))


def test_rms_swiglu_matches_unfused_chain(ops):
    case = I.make_swiglu_case(150, 512, 264, "bf16", seed=16)
    x, one = cuda(case["x"]), torch.ones(512, dtype=torch.bfloat16, device="cuda")
    fused = _swiglu_check(ops, case)
    y = ops.rmsnorm(x, cuda(case["gamma"]), case["eps"])
    g = ops.gemm(y, ops.ln_linear_prepare(cuda(case["Wg"]), one))
    u = ops.gemm(y, ops.ln_linear_prepare(cuda(case["Wu"]), one))
    h = ops.silu_mul(g, u)
    ref = oracle.rms_swiglu(case["x"], case["gamma"], case["Wg"], case["Wu"], case["eps"])
    assert rowwise_rel_err(h.cpu(), ref) <= TOL[torch.bfloat16]
    assert rowwise_rel_err(fused.cpu(), oracle.to_f64(h.cpu())) <= TOL[torch.bfloat16]


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_silu_mul_unfused(ops, dtype):
    g = torch.Generator().manual_seed(17)
    a = (torch.randn(33, 40, generator=g) * 6).to(I.DTYPES[dtype])
    b = torch.randn(33, 40, generator=g).to(I.DTYPES[dtype])
    h = ops.silu_mul(cuda(a), cuda(b))
    ref = torch.nn.functional.silu(a.double()) * b.double()
    assert rowwise_rel_err(h.cpu(), ref.numpy()) <= TOL[a.dtype] / 4


# ---------------------------------------------------------------------------- Softmax -> P.V
def _sm_check(ops, case, rows=None):
    S, V = case["S"], case["V"]
    BH, L, _ = S.shape
    causal = case["causal"]
    out = ops.softmax_pv_deferred(cuda(S), cuda(V), causal=causal)
    torch.cuda.synchronize()
    if rows is None:
        rows = np.arange(BH * L)
    rows = np.asarray(rows)
    head, q = rows // L, rows % L
    S_rows = S.reshape(BH * L, L)[torch.as_tensor(rows)]
    ref = oracle.softmax_pv(S_rows, V, head=head, qpos=q if causal else None)
    got = out.cpu().reshape(BH * L, -1)[torch.as_tensor(rows)]
    err = rowwise_rel_err(got, ref)
    print(f"softmax_pv_deferred {tuple(S.shape)} d={V.shape[-1]} causal={causal}: err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err
    return out


def test_softmax_pv_small_workload(ops):
    _sm_check(ops, I.make_sm(I.SM_BF16_SMALL))


@pytest.mark.parametrize("BH,L,d,causal", [(3, 200, 64, True), (2, 136, 128, False), (2, 8, 64, True),
                                           (1, 392, 128, True), (5, 64, 64, False), (2, 520, 128, False),
                                           # enough 256-query blocks to fill the chip: the 8-wave kernel
                                           (256, 136, 64, True), (128, 264, 128, False), (86, 776, 64, True)])
def test_softmax_pv_ragged(ops, BH, L, d, causal):
    _sm_check(ops, I.make_sm_case(BH, L, d, causal, seed=L, from_qk=causal))


def test_softmax_pv_causal_workload_all_rows(ops):
    # the causal 32 x 8192 x 8192, d = 128 workload in the bench's launch configuration; every
    # row of every head against the oracle, one head at a time
    w = I.SM_CAUSAL
    case = I.make_sm(w)
    out = ops.softmax_pv_deferred(cuda(case["S"]), cuda(case["V"]), causal=True)
    got = out.cpu()
    del out
    err, qpos = 0.0, np.arange(w.L)
    for h in range(w.BH):
        ref = oracle.softmax_pv(case["S"][h], case["V"][h], qpos=qpos, nthreads=ORACLE_THREADS)
        err = max(err, rowwise_rel_err(got[h], ref))
    print(f"softmax_pv_deferred causal 32x8192x8192 d128: all {w.BH * w.L} rows, err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err


@pytest.mark.parametrize("BH,Lq,Lk,d", [(2, 100, 304, 64), (3, 300, 72, 128), (1, 7, 1000, 128),
                                        (2, 257, 520, 64)])
def test_softmax_pv_cross_lengths(ops, BH, Lq, Lk, d):
    # non-causal with Lq != Lk: every query row takes all Lk keys (Eq. (7) per row)
    case = I.make_sm_case(BH, max(Lq, Lk), d, False, seed=Lq + Lk)
    S = case["S"][:, :Lq, :Lk].contiguous()
    V = case["V"][:, :Lk].contiguous()
    out = ops.softmax_pv_deferred(cuda(S), cuda(V))
    torch.cuda.synchronize()
    ref = oracle.softmax_pv(S.reshape(BH * Lq, Lk), V, head=np.repeat(np.arange(BH), Lq))
    err = rowwise_rel_err(out.cpu().reshape(BH * Lq, d), ref)
    print(f"softmax_pv_deferred S{tuple(S.shape)} V{tuple(V.shape)}: err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err


def test_softmax_pv_causal_row0_exact(ops):
    case = I.make_sm_case(2, 256, 128, True, seed=3)
    out = ops.softmax_pv_deferred(cuda(case["S"]), cuda(case["V"]), causal=True)
    assert torch.equal(out[:, 0].cpu(), case["V"][:, 0])


@pytest.mark.parametrize("BH,L", [(256, 264), (2, 264)])
def test_softmax_pv_causal_flag_matches_premasked(ops, BH, L):
    # S carries -inf above the diagonal; with the causal flag the kernel skips those keys, without
    # it they give zero numerators.  On a grid that fills the chip both take the same kernel and
    # agree bitwise; on a small one the non-causal call splits the keys between two groups of
    # waves (another summation order), so both are held to the oracle instead.
    case = I.make_sm_case(BH, L, 64, True, seed=8, from_qk=True)
    S, V = cuda(case["S"]), cuda(case["V"])
    a = ops.softmax_pv_deferred(S, V, causal=True)
    b = ops.softmax_pv_deferred(S, V, causal=False)
    if BH * ((L + 255) // 256) >= 256:
        assert torch.equal(a, b)
    else:
        rows = np.arange(BH * L)
        ref = oracle.softmax_pv(case["S"].reshape(BH * L, L), case["V"], head=rows // L, qpos=rows % L)
        for o in (a, b):
            assert rowwise_rel_err(o.cpu().reshape(BH * L, -1), ref) <= TOL[torch.bfloat16]


def test_softmax_pv_fully_masked_row_is_nan(ops):
    case = I.make_sm_case(1, 64, 64, False, seed=1)
    case["S"][0, 5, :] = float("-inf")
    out = _sm_check(ops, case)
    assert torch.isnan(out[0, 5].float()).all()


def test_softmax_pv_key_groups_merge(ops):
    # small non-causal grids split the keys between two groups of waves and merge their partial
    # sums: rows whose unmasked keys all lie in one group's half (the other group's reference
    # maximum stays -inf), a row masked entirely (NaN) and a row masked but for one key
    case = I.make_sm_case(2, 200, 64, False, seed=21)
    S = case["S"]
    S[0, 3, :128] = float("-inf")     # keys only in the second group's steps
    S[0, 4, 128:] = float("-inf")     # keys only in the first group's steps
    S[1, 5, :] = float("-inf")        # nothing: 0/0
    S[1, 6, :] = float("-inf")
    S[1, 6, 150] = 3.0                # one key: exactly V[150]
    out = _sm_check(ops, case, rows=[r for r in range(400) if r != 205])
    assert torch.isnan(out[1, 5].float()).all()
    assert torch.equal(out[1, 6].cpu(), case["V"][1, 150])


@pytest.mark.parametrize("BH,L,d,causal", [(256, 264, 128, True), (2, 520, 64, False), (3, 392, 128, True)])
def test_softmax_pv_reference_rises_mid_row(ops, BH, L, d, causal):
    # scores that climb along the keys (the reference maximum rises step after step, the partial
    # sums rescaled each time), fall, stay flat, or jump once late in the row (a single lane's
    # keys ask for the rise while the others do not), on the 8-wave, split and small kernels
    case = I.make_sm_case(BH, L, d, causal, seed=BH + L)
    g = torch.Generator().manual_seed(BH * L)
    S = case["S"].float()
    slopes = torch.tensor([0.0, 0.05, 0.2, -0.05])[torch.randint(0, 4, (BH, L, 1), generator=g)]
    S = S + slopes * torch.arange(L, dtype=torch.float32)
    spike_q = torch.randint(0, L, (BH, 8), generator=g)
    for h in range(BH):
        for q in spike_q[h].tolist():
            k = q if causal else int(torch.randint(0, L, (1,), generator=g))
            S[h, q, k] += 30.0
    case["S"] = S.to(torch.bfloat16)
    _sm_check(ops, case)


@pytest.mark.parametrize("BH,L,d,causal", [(256, 264, 128, True), (2, 520, 64, False), (3, 392, 128, True)])
def test_softmax_pv_nonfinite_scores(ops, BH, L, d, causal):
    # a NaN score and a +inf score (kept keys) each make their row all NaN, as the plain
    # definition does (exp(s - m) with m = +inf gives inf - inf); the other rows are unaffected
    # (8-wave, split and small kernels)
    case = I.make_sm_case(BH, L, d, causal, seed=L + d)
    S = case["S"]
    S[0, 5, 3] = float("nan")
    S[0, 150, 100] = float("inf")
    S[BH - 1, L - 1, L // 2] = float("nan")
    out = _sm_check(ops, case)
    for h, q in ((0, 5), (0, 150), (BH - 1, L - 1)):
        assert torch.isnan(out[h, q].float()).all()
    assert not torch.isnan(out[0, 4].float()).any()


def test_softmax_pv_deterministic(ops):
    case = I.make_sm_case(2, 296, 128, True, seed=6)
    S, V = cuda(case["S"]), cuda(case["V"])
    assert torch.equal(ops.softmax_pv_deferred(S, V, causal=True), ops.softmax_pv_deferred(S, V, causal=True))


def test_softmax_pv_rejects_ragged_key_length(ops):
    case = I.make_sm_case(1, 300, 64, False, seed=6)
    with pytest.raises(ops.DNError) as e:
        ops.softmax_pv_deferred(cuda(case["S"]), cuda(case["V"]))
    assert e.value.status == 2  # DN_ERR_UNSUPPORTED: Lk must be a multiple of 8


# ---------------------------------------------------------------------------- attention from Q, K
def _attn_check(ops, case, rows=None, Lk=None):
    Q, K, V = case["Q"], case["K"], case["V"]
    BH, Lq, d = Q.shape
    causal = case["causal"]
    out = ops.attention_deferred(cuda(Q), cuda(K), cuda(V), causal=causal, scale=case["scale"])
    torch.cuda.synchronize()
    rows = np.arange(BH * Lq) if rows is None else np.asarray(rows)
    head, q = rows // Lq, rows % Lq
    ref = oracle.attention(Q.reshape(BH * Lq, d)[torch.as_tensor(rows)], K, V, case["scale"], head=head,
                           qpos=q if causal else None)
    got = out.cpu().reshape(BH * Lq, d)[torch.as_tensor(rows)]
    err = rowwise_rel_err(got, ref)
    print(f"attention_deferred Q{tuple(Q.shape)} K{tuple(K.shape)} causal={causal}: err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err
    return out


@pytest.mark.parametrize("BH,L,d,causal", [(3, 200, 64, True), (2, 136, 128, False), (2, 8, 64, True),
                                           (1, 1000, 128, True), (2, 64, 128, True), (1, 1, 64, True),
                                           (2, 520, 64, False)])
def test_attention_shapes(ops, BH, L, d, causal):
    # ragged lengths (not multiples of the 64-key step or the 256-query block), one-key rows
    _attn_check(ops, I.make_qkv_case(BH, L, d, causal, seed=L + d))


@pytest.mark.parametrize("Lq,Lk,d", [(100, 300, 64), (300, 72, 128), (7, 1000, 128)])
def test_attention_cross_lengths(ops, Lq, Lk, d):
    # non-causal with different query and key lengths
    a = I.make_qkv_case(2, Lq, d, False, seed=Lq)
    b = I.make_qkv_case(2, Lk, d, False, seed=Lk + 1)
    _attn_check(ops, dict(Q=a["Q"], K=b["K"], V=b["V"], causal=False, scale=a["scale"]))


@pytest.mark.parametrize("BH,g,Lq,Lk,d,causal", [(2, 4, 300, 300, 128, True), (3, 2, 100, 520, 64, False),
                                                 (1, 8, 260, 260, 64, True)])
def test_attention_grouped_query(ops, BH, g, Lq, Lk, d, causal):
    # grouped-query attention: g consecutive query heads read one key/value head
    q = I.make_qkv_case(BH * g, Lq, d, causal, seed=Lq + g)["Q"]
    kv = I.make_qkv_case(BH, Lk, d, causal, seed=Lk + 3)
    scale = 1.0 / d ** 0.5
    out = ops.attention_deferred(cuda(q), cuda(kv["K"]), cuda(kv["V"]), causal=causal, scale=scale)
    torch.cuda.synchronize()
    rows = np.arange(BH * g * Lq)
    qh, pos = rows // Lq, rows % Lq
    ref = oracle.attention(q.reshape(-1, d), kv["K"], kv["V"], scale, head=qh // g, qpos=pos if causal else None)
    err = rowwise_rel_err(out.cpu().reshape(-1, d), ref)
    print(f"attention GQA Q{tuple(q.shape)} K{tuple(kv['K'].shape)} causal={causal}: err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err


def test_attention_matches_softmax_pv_on_materialized_scores(ops):
    # the same workload through S = Q K^T / sqrt(d) stored in bf16 and softmax_pv_deferred:
    # the two differ only by the rounding of S to bf16
    w = I.SMWorkload("attn_vs_sm", 202, 2, 384, 128, True, from_qk=True)
    qkv, sm = I.make_qkv(w), I.make_sm(w)
    a = ops.attention_deferred(cuda(qkv["Q"]), cuda(qkv["K"]), cuda(qkv["V"]), causal=True)
    b = ops.softmax_pv_deferred(cuda(sm["S"]), cuda(sm["V"]), causal=True)
    assert rowwise_rel_err(a.cpu().reshape(-1, 128), oracle.to_f64(b.cpu()).reshape(-1, 128)) <= TOL[torch.bfloat16]


def test_attention_causal_workload_all_rows(ops):
    # causal 32 x 8192 x 8192, d = 128 with the scores formed in the kernel; every row of
    # every head against the oracle, one head at a time
    w = I.ATTN_CAUSAL
    case = I.make_qkv(w)
    out = ops.attention_deferred(cuda(case["Q"]), cuda(case["K"]), cuda(case["V"]), causal=True,
                                 scale=case["scale"])
    got = out.cpu()
    del out
    err, qpos = 0.0, np.arange(w.L)
    for h in range(w.BH):
        ref = oracle.attention(case["Q"][h], case["K"][h], case["V"][h], case["scale"], qpos=qpos,
                               nthreads=ORACLE_THREADS)
        err = max(err, rowwise_rel_err(got[h], ref))
    print(f"attention_deferred causal 32x8192x8192 d128: all {w.BH * w.L} rows, err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err


# ---------------------------------------------------------------------------- decode attention (split keys + merge)
def _decode_check(ops, case, heads=None):
    Q, K, V = case["Q"], case["K"], case["V"]
    BH, Lq, d = Q.shape
    out = ops.attention_decode_deferred(cuda(Q), cuda(K), cuda(V), scale=case["scale"])
    torch.cuda.synchronize()
    heads = np.arange(BH) if heads is None else np.asarray(heads)
    rows = (heads[:, None] * Lq + np.arange(Lq)[None, :]).reshape(-1)
    hsel = torch.as_tensor(heads)
    # the oracle sees only the sampled heads' caches (row r belongs to sampled head r // Lq)
    ref = oracle.attention(Q[hsel].reshape(-1, d), K[hsel], V[hsel], case["scale"],
                           head=np.repeat(np.arange(len(heads)), Lq))
    got = out.cpu().reshape(BH * Lq, d)[torch.as_tensor(rows)]
    err = rowwise_rel_err(got, ref)
    print(f"attention_decode_deferred Q{tuple(Q.shape)} K{tuple(K.shape)}: err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err
    return out


@pytest.mark.parametrize("BH,Lq,Lk,d", [(1, 1, 1, 64), (3, 1, 100, 128), (2, 4, 8200, 128), (5, 16, 8192, 64),
                                        (1, 7, 70001, 128), (2048, 1, 130, 64), (8, 3, 64, 128),
                                        (600, 2, 3000, 128), (255, 1, 4100, 128), (511, 2, 1000, 64)])
def test_attention_decode_shapes(ops, BH, Lq, Lk, d):
    # single key; ragged caches (not whole steps); splits of one step and of many steps (one head,
    # long cache); enough heads for a single pass without the merge; partial query tiles; one head
    # short of a full resident round (255 at d = 128, 511 at d = 64: two ranges per head)
    _decode_check(ops, I.make_decode_case(BH, Lq, Lk, d, seed=Lk + Lq))


@pytest.mark.parametrize("causal", [True, False])
def test_attention_nonfinite_inputs(ops, causal):
    # a NaN in a query row makes that row NaN; a NaN in a key row makes NaN every row that
    # keeps that key (causal: the rows at or after it), as the plain definition does
    case = I.make_qkv_case(2, 300, 128, causal, seed=31)
    case["Q"][0, 10, 7] = float("nan")
    case["K"][1, 200, 3] = float("nan")
    out = _attn_check(ops, case)
    assert torch.isnan(out[0, 10].float()).all()
    assert torch.isnan(out[1, 299].float()).all()
    if causal:  # the rows before key 200 do not keep it
        assert not torch.isnan(out[1, 199].float()).any()


def test_attention_decode_nonfinite_inputs(ops):
    # split keys and the merge: a NaN key row poisons its head's rows only
    case = I.make_decode_case(4, 2, 3000, 128, seed=13)
    case["K"][2, 1234, 5] = float("nan")
    out = _decode_check(ops, case)
    assert torch.isnan(out[2].float()).all()
    assert not torch.isnan(out[1].float()).any()


def test_attention_decode_matches_single_pass(ops):
    # the split + merge against the single-pass kernel on the same inputs: both bf16 outputs
    # of the same exact quantity, so they agree to twice the bf16 output rounding
    case = I.make_decode_case(4, 16, 3000, 128, seed=12)
    q, k, v = cuda(case["Q"]), cuda(case["K"]), cuda(case["V"])
    a = ops.attention_decode_deferred(q, k, v)
    b = ops.attention_deferred(q, k, v, causal=False)
    assert rowwise_rel_err(a.cpu().reshape(-1, 128), oracle.to_f64(b.cpu()).reshape(-1, 128)) <= 2 ** -7


def test_attention_decode_workspace_reuse(ops):
    # one workspace serves a large call and then a smaller one; a caller-provided output is used
    big = I.make_decode_case(16, 2, 5000, 128, seed=13)
    ws = torch.empty(ops.attention_decode_workspace_bytes(16, 2, 5000, 128), dtype=torch.uint8, device="cuda")
    out = torch.empty((16, 2, 128), dtype=torch.bfloat16, device="cuda")
    ops.attention_decode_deferred(cuda(big["Q"]), cuda(big["K"]), cuda(big["V"]), workspace=ws, out=out)
    small = I.make_decode_case(3, 1, 700, 128, seed=14)
    assert ops.attention_decode_workspace_bytes(3, 1, 700, 128) <= ws.numel()
    got = ops.attention_decode_deferred(cuda(small["Q"]), cuda(small["K"]), cuda(small["V"]), workspace=ws)
    torch.cuda.synchronize()
    ref = oracle.attention(small["Q"].reshape(-1, 128), small["K"], small["V"], small["scale"],
                           head=np.arange(3))
    assert rowwise_rel_err(got.cpu().reshape(-1, 128), ref) <= TOL[torch.bfloat16]
    refb = oracle.attention(big["Q"].reshape(-1, 128), big["K"], big["V"], big["scale"],
                            head=np.repeat(np.arange(16), 2))
    assert rowwise_rel_err(out.cpu().reshape(-1, 128), refb) <= TOL[torch.bfloat16]


def _decode_gqa_check(ops, case, heads=None):
    Q, K, V = case["Q"], case["K"], case["V"]
    BH, d = K.shape[0], K.shape[2]
    gq = Q.shape[0] // BH * Q.shape[1]  # query rows per key/value head
    out = ops.attention_decode_deferred(cuda(Q), cuda(K), cuda(V), scale=case["scale"])
    torch.cuda.synchronize()
    hs = torch.as_tensor(np.arange(BH) if heads is None else np.asarray(heads))
    ref = oracle.attention(Q.reshape(BH, gq, d)[hs].reshape(-1, d), K[hs], V[hs], case["scale"],
                           head=np.repeat(np.arange(len(hs)), gq))
    got = out.cpu().reshape(BH, gq, d)[hs].reshape(-1, d)
    err = rowwise_rel_err(got, ref)
    print(f"attention_decode_deferred GQA Q{tuple(Q.shape)} K{tuple(K.shape)}: err={err:.3e}")
    assert err <= TOL[torch.bfloat16], err


@pytest.mark.parametrize("BH,g,Lq,Lk,d", [(8, 4, 1, 3000, 128), (3, 8, 2, 777, 64), (2, 16, 1, 64, 128),
                                          (600, 4, 1, 1000, 128)])
def test_attention_decode_grouped_query(ops, BH, g, Lq, Lk, d):
    # g query heads per key/value head go through the kernel as g * Lq rows of that head
    _decode_gqa_check(ops, I.make_decode_case(BH, Lq, Lk, d, seed=BH + g, group=g))


def test_attention_decode_gqa_workload_all_heads(ops):
    _decode_gqa_check(ops, I.make_decode(I.ATTN_DECODE_GQA))


def test_attention_deterministic(ops):
    # no atomics anywhere: the same inputs give the same bits, causal and decode
    case = I.make_qkv_case(2, 700, 128, True, seed=21)
    q, k, v = cuda(case["Q"]), cuda(case["K"]), cuda(case["V"])
    assert torch.equal(ops.attention_deferred(q, k, v, causal=True), ops.attention_deferred(q, k, v, causal=True))
    dec = I.make_decode_case(4, 3, 5000, 128, seed=22)
    q, k, v = cuda(dec["Q"]), cuda(dec["K"]), cuda(dec["V"])
    assert torch.equal(ops.attention_decode_deferred(q, k, v), ops.attention_decode_deferred(q, k, v))


def test_attention_decode_workload_all_heads(ops):
    # the benchmarked decode workload at full size, in its own launch configuration, every head
    _decode_check(ops, I.make_decode(I.ATTN_DECODE))


# ---------------------------------------------------------------------------- unfused comparators
@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_layernorm_unfused(ops, dtype):
    case = I.make_ln_case(77, 1032, 8, dtype, seed=3, outliers=2)
    y = ops.layernorm(cuda(case["x"]), cuda(case["gamma"]), cuda(case["beta"]), case["eps"])
    ref = oracle.layernorm(case["x"], case["gamma"], case["beta"], case["eps"])
    err = rowwise_rel_err(y.cpu(), ref)
    assert err <= TOL[case["x"].dtype] / (4 if dtype == "bf16" else 1), err


@pytest.mark.parametrize("dtype", ["f32", "bf16"])
def test_rmsnorm_unfused(ops, dtype):
    case = I.make_ln_case(77, 1032, 8, dtype, seed=5, outliers=2, norm="rms")
    y = ops.rmsnorm(cuda(case["x"]), cuda(case["gamma"]), case["eps"])
    ref = oracle.rmsnorm(case["x"], case["gamma"], case["eps"])
    err = rowwise_rel_err(y.cpu(), ref)
    assert err <= TOL[case["x"].dtype] / (4 if dtype == "bf16" else 1), err


@pytest.mark.parametrize("causal", [0, 1])
def test_softmax_unfused(ops, causal):
    case = I.make_sm_case(2, 136, 64, bool(causal), seed=4)
    P = ops.softmax(cuda(case["S"]), causal=causal)
    L = 136
    ref = oracle.softmax(case["S"].reshape(-1, L), np.tile(np.arange(L), 2) if causal else None)
    assert rowwise_rel_err(P.cpu().reshape(-1, L), ref) <= 1e-2


@pytest.mark.parametrize("b_layout,M", [(0, 136), (1, 136), (1, 1)])
def test_gemm_unfused(ops, b_layout, M):
    # M = 1: one row per batch entry (the score product of a decode step)
    g = torch.Generator().manual_seed(1)
    A = torch.randn(3, M, 200, generator=g).to(torch.bfloat16)
    B = torch.randn(3, 200, 72, generator=g).to(torch.bfloat16)
    bias = torch.randn(72, generator=g).to(torch.bfloat16)
    Bd = B if b_layout == 0 else B.transpose(1, 2).contiguous()
    C = ops.gemm(cuda(A), cuda(Bd), cuda(bias), b_layout=b_layout)
    ref = oracle.linear(A, B, bias)
    assert rowwise_rel_err(C.cpu().reshape(-1, 72), ref.reshape(-1, 72)) <= TOL[torch.bfloat16]


def test_gemm_unfused_f32(ops):
    g = torch.Generator().manual_seed(2)
    A, B = torch.randn(70, 96, generator=g), torch.randn(96, 40, generator=g)
    C = ops.gemm(cuda(A), cuda(B.t().contiguous()), b_layout=1)
    assert rowwise_rel_err(C.cpu(), oracle.linear(A, B)) <= TOL[torch.float32]


def test_gemm_causal_matches_dense_lower_triangular(ops):
    g = torch.Generator().manual_seed(3)
    L, d = 264, 64
    A = torch.tril(torch.rand(2, L, L, generator=g)).to(torch.bfloat16)
    V = torch.randn(2, L, d, generator=g).to(torch.bfloat16)
    junk = A.clone()
    junk[:, torch.triu(torch.ones(L, L, dtype=torch.bool), 1)] = float("nan")   # never used
    C = ops.gemm(cuda(junk), cuda(V), a_causal=True)
    ref = oracle.linear(A, V)
    assert rowwise_rel_err(C.cpu().reshape(-1, d), ref.reshape(-1, d)) <= TOL[torch.bfloat16]


def test_unfused_chains_match_deferred(ops):
    case = I.make_ln_case(150, 512, 264, "bf16", seed=12)
    x = cuda(case["x"])
    w = ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"]), cuda(case["beta"]))
    fused = ops.ln_linear_deferred(x, w)
    y = ops.layernorm(x, cuda(case["gamma"]), cuda(case["beta"]))
    unfused = ops.gemm(y, ops.ln_linear_prepare(cuda(case["W"]), torch.ones(512, dtype=torch.bfloat16,
                                                                          device="cuda")))
    ref = oracle.ln_linear(case["x"], case["gamma"], case["beta"], case["W"], None, case["eps"])
    assert rowwise_rel_err(unfused.cpu(), ref) <= TOL[torch.bfloat16]
    assert rowwise_rel_err(fused.cpu(), oracle.to_f64(unfused.cpu())) <= TOL[torch.bfloat16]
    rfused = ops.rms_linear_deferred(x, ops.ln_linear_prepare(cuda(case["W"]), cuda(case["gamma"])))
    y = ops.rmsnorm(x, cuda(case["gamma"]))
    runfused = ops.gemm(y, ops.ln_linear_prepare(cuda(case["W"]), torch.ones(512, dtype=torch.bfloat16,
                                                                            device="cuda")))
    rref = oracle.rms_linear(case["x"], case["gamma"], case["W"], None, case["eps"])
    assert rowwise_rel_err(runfused.cpu(), rref) <= TOL[torch.bfloat16]
    assert rowwise_rel_err(rfused.cpu(), rref) <= TOL[torch.bfloat16]
    sm = I.make_sm_case(2, 256, 128, True, seed=13)
    S, V = cuda(sm["S"]), cuda(sm["V"])
    P = ops.softmax(S, causal=2)
    o2 = ops.gemm(P, V, a_causal=True)
    o1 = ops.softmax(S, causal=1)
    o1 = ops.gemm(o1, V)
    fused = ops.softmax_pv_deferred(S, V, causal=True)
    ref = oracle.softmax_pv(sm["S"].reshape(-1, 256), sm["V"], head=np.repeat([0, 1], 256),
                            qpos=np.tile(np.arange(256), 2))
    for o in (o1, o2, fused):
        assert rowwise_rel_err(o.cpu().reshape(-1, 128), ref) <= TOL[torch.bfloat16]
