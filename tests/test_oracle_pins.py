"""Pins of the fp64 oracle against what the paper and mathematics fix.

The oracle (``oracle/``) is the plain definition of Eq. (1), (2), (4), (6) and (7),
and of attention formed from Q and K ahead of Eq. (7).
Before it may judge the GPU path it is tied here to things other than itself:

- hand-worked examples stored in ``tests/golden`` (exact values);
- closed forms and special cases (K = 2, constant rows, one-hot scores, V = I);
- library routines: ``torch.nn.functional.layer_norm``, ``rms_norm``, ``silu``,
  ``scaled_dot_product_attention`` and ``torch.softmax``
  in fp64, which the oracle does not call;
- the paper's fused forms, Eq. (5) and Eq. (8), evaluated independently here
  with numpy, which reach the same result by different arithmetic;
- invariants: probabilities sum to 1, the pre-affine LayerNorm output has
  mean 0 and variance var/(var+eps), shift and scale invariance;
- a 50-digit mpmath brute force on tiny inputs.

A dropped term, a wrong sign or index, a transposed operand, an unbiased
variance, eps outside the root or a causal off-by-one each fails at least one.
"""
import json
import math
import os

import numpy as np
import pytest
import torch

import oracle


def _num(v):
    """Golden entries are numbers or strings "lnK" / "A+lnK" (natural log of an integer)."""
    if isinstance(v, str):
        base, _, ln = v.rpartition("ln")
        return (float(base.rstrip("+")) if base else 0.0) + math.log(int(ln))
    return float(v)


def _arr(rows):
    return np.array([[_num(v) for v in r] for r in rows], dtype=np.float64)


# --------------------------------------------------------------------------- goldens
def test_golden_ln_linear(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "ln_linear_worked.json")))
    x, W = _arr(g["x"]), _arr(g["W"])
    gamma, beta, bias = (np.array(g[k], np.float64) for k in ("gamma", "beta", "bias"))
    y = oracle.layernorm(x, gamma, beta, g["eps"])
    np.testing.assert_array_equal(y, _arr(g["y"]))
    out = oracle.ln_linear(x, gamma, beta, W, bias, g["eps"])
    np.testing.assert_array_equal(out, _arr(g["out"]))
    np.testing.assert_array_equal(oracle.linear(y, W, bias), _arr(g["out"]))


def test_golden_rms_linear(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "rms_linear_worked.json")))
    x, W = _arr(g["x"]), _arr(g["W"])
    gamma, bias = (np.array(g[k], np.float64) for k in ("gamma", "bias"))
    y = oracle.rmsnorm(x, gamma, g["eps"])
    np.testing.assert_array_equal(y, _arr(g["y"]))
    np.testing.assert_array_equal(oracle.rms_linear(x, gamma, W, bias, g["eps"]), _arr(g["out"]))
    np.testing.assert_array_equal(oracle.linear(y, W, bias), _arr(g["out"]))


@pytest.mark.parametrize("case", ["plain", "large"])
def test_golden_softmax_pv(golden_dir, case):
    g = json.load(open(os.path.join(golden_dir, "softmax_pv_worked.json")))[case]
    S, V = _arr(g["S"]), _arr(g["V"])
    # the stored score 1000 + ln 3 is itself rounded by ulp(1000) ~ 1.1e-13, which moves the
    # probabilities by about that much; the small-score case is exact to a few fp64 ulps
    tol = 4 * np.spacing(np.abs(S).max())
    np.testing.assert_allclose(oracle.softmax(S), _arr(g["P"]), rtol=max(tol, 1e-15), atol=0)
    np.testing.assert_allclose(oracle.softmax_pv(S, V), _arr(g["out"]), rtol=max(tol, 1e-15), atol=1e-15)


def test_golden_softmax_pv_causal(golden_dir):
    g = json.load(open(os.path.join(golden_dir, "softmax_pv_worked.json")))["causal"]
    S, V = _arr(g["S"]), _arr(g["V"])
    out = oracle.softmax_pv(S, V, qpos=[0, 1, 2])
    np.testing.assert_allclose(out, _arr(g["out"]), rtol=1e-15, atol=1e-15)
    assert out[0].tolist() == [6.0, 0.0]  # row 0 keeps key 0 only: exact


# --------------------------------------------------------------------------- closed forms
def test_layernorm_k2_closed_form():
    # x = [a, b]: mean (a+b)/2, variance ((a-b)/2)^2 -> normalized +-h/sqrt(h^2+eps), h=(a-b)/2
    rng = np.random.default_rng(1)
    for _ in range(20):
        a, b, eps = rng.normal(size=2).tolist() + [float(rng.uniform(0, 1))]
        h = (a - b) / 2
        want = h / math.sqrt(h * h + eps)
        y = oracle.layernorm(np.array([[a, b]]), np.ones(2), np.zeros(2), eps)
        np.testing.assert_allclose(y[0], [want, -want], rtol=1e-14, atol=1e-15)


def test_layernorm_constant_row_gives_beta_projection():
    rng = np.random.default_rng(2)
    K, N = 16, 5
    x = np.full((3, K), 0.375)
    gamma, beta, W, bias = rng.normal(size=K), rng.normal(size=K), rng.normal(size=(K, N)), rng.normal(size=N)
    out = oracle.ln_linear(x, gamma, beta, W, bias, 1e-5)
    np.testing.assert_allclose(out, np.broadcast_to(beta @ W + bias, out.shape), rtol=1e-14, atol=1e-14)


def test_linear_identity_and_one_hot_columns():
    rng = np.random.default_rng(3)
    y = rng.normal(size=(4, 6))
    np.testing.assert_array_equal(oracle.linear(y, np.eye(6)), y)
    W = np.zeros((6, 3)); W[4, 0] = 1; W[1, 2] = 1
    out = oracle.linear(y, W)
    np.testing.assert_array_equal(out[:, 0], y[:, 4])
    np.testing.assert_array_equal(out[:, 1], 0 * y[:, 0])
    np.testing.assert_array_equal(out[:, 2], y[:, 1])


def test_softmax_constant_row_gives_mean_of_kept_values():
    rng = np.random.default_rng(4)
    L, d = 9, 4
    V = rng.normal(size=(L, d))
    S = np.full((L, L), 1.25)
    out = oracle.softmax_pv(S, V, qpos=np.arange(L))
    for i in range(L):
        np.testing.assert_allclose(out[i], V[: i + 1].mean(axis=0), rtol=1e-13, atol=1e-14)


def test_softmax_dominant_score_selects_value_row():
    rng = np.random.default_rng(5)
    L, d = 8, 3
    V = rng.normal(size=(L, d))
    S = rng.normal(size=(L, L))
    S[np.arange(L), (np.arange(L) * 3) % L] = 1000.0
    out = oracle.softmax_pv(S, V)
    np.testing.assert_allclose(out, V[(np.arange(L) * 3) % L], rtol=0, atol=1e-12)


def test_softmax_values_identity_and_ones():
    rng = np.random.default_rng(6)
    L = 7
    S = rng.normal(size=(L, L)) * 3
    np.testing.assert_allclose(oracle.softmax_pv(S, np.eye(L)), oracle.softmax(S), rtol=1e-15, atol=1e-17)
    np.testing.assert_allclose(oracle.softmax_pv(S, np.ones((L, 5))), np.ones((L, 5)), rtol=1e-14)


def test_softmax_causal_row0_is_first_value_row_exactly():
    rng = np.random.default_rng(7)
    L, d = 6, 4
    S, V = rng.normal(size=(L, L)), rng.normal(size=(L, d))
    out = oracle.softmax_pv(S, V, qpos=np.arange(L))
    np.testing.assert_array_equal(out[0], V[0])


def test_softmax_fully_masked_row_is_nan():
    S = np.array([[-np.inf, -np.inf, -np.inf]])
    assert np.isnan(oracle.softmax_pv(S, np.ones((3, 2)))).all()


def test_causal_ignores_stored_values_above_diagonal():
    rng = np.random.default_rng(8)
    L, d = 10, 3
    S, V = rng.normal(size=(L, L)), rng.normal(size=(L, d))
    masked = S.copy()
    masked[np.triu_indices(L, 1)] = -np.inf
    a = oracle.softmax_pv(S, V, qpos=np.arange(L))
    b = oracle.softmax_pv(masked, V)  # no causal flag: -inf scores carry the mask
    np.testing.assert_allclose(a, b, rtol=1e-15, atol=1e-16)
    garbage = S.copy()
    garbage[np.triu_indices(L, 1)] = 1e6
    np.testing.assert_array_equal(oracle.softmax_pv(garbage, V, qpos=np.arange(L)), a)


# --------------------------------------------------------------------------- library routines
@pytest.mark.parametrize("M,K,N,eps", [(5, 7, 3, 1e-5), (13, 64, 17, 0.1), (2, 1, 4, 1e-3)])
def test_ln_linear_matches_torch_layer_norm(M, K, N, eps):
    rng = np.random.default_rng(M * K * N)
    x = rng.normal(size=(M, K)) * 3 + 0.5
    gamma, beta = rng.uniform(0.5, 1.5, K), rng.normal(size=K) * 0.1
    W, bias = rng.normal(size=(K, N)), rng.normal(size=N)
    ref = torch.nn.functional.layer_norm(torch.from_numpy(x), (K,), torch.from_numpy(gamma),
                                         torch.from_numpy(beta), eps)
    np.testing.assert_allclose(oracle.layernorm(x, gamma, beta, eps), ref.numpy(), rtol=1e-12, atol=1e-13)
    want = (ref @ torch.from_numpy(W) + torch.from_numpy(bias)).numpy()
    np.testing.assert_allclose(oracle.ln_linear(x, gamma, beta, W, bias, eps), want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("M,K,N,eps", [(5, 7, 3, 1e-5), (13, 64, 17, 0.1), (2, 1, 4, 0.0)])
def test_rms_linear_matches_torch_rms_norm(M, K, N, eps):
    rng = np.random.default_rng(M * K * N + 1)
    x = rng.normal(size=(M, K)) * 3 + 0.5
    gamma, beta = rng.uniform(0.5, 1.5, K), rng.normal(size=K) * 0.1
    W, bias = rng.normal(size=(K, N)), rng.normal(size=N)
    ref = torch.nn.functional.rms_norm(torch.from_numpy(x), (K,), torch.from_numpy(gamma), eps)
    np.testing.assert_allclose(oracle.rmsnorm(x, gamma, eps), ref.numpy(), rtol=1e-12, atol=1e-13)
    np.testing.assert_allclose(oracle.rmsnorm(x, gamma, eps, beta=beta), ref.numpy() + beta, rtol=1e-12,
                               atol=1e-13)
    want = (ref @ torch.from_numpy(W) + torch.from_numpy(bias)).numpy()
    np.testing.assert_allclose(oracle.rms_linear(x, gamma, W, bias, eps), want, rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("M,K,N,eps", [(5, 7, 3, 1e-5), (9, 64, 17, 0.1)])
def test_rms_swiglu_matches_torch(M, K, N, eps):
    rng = np.random.default_rng(M * K + N)
    x = rng.normal(size=(M, K)) * 2 + 0.3
    gamma = rng.uniform(0.5, 1.5, K)
    Wg, Wu = rng.normal(size=(K, N)) * 2, rng.normal(size=(K, N))
    y = torch.nn.functional.rms_norm(torch.from_numpy(x), (K,), torch.from_numpy(gamma), eps)
    want = torch.nn.functional.silu(y @ torch.from_numpy(Wg)) * (y @ torch.from_numpy(Wu))
    np.testing.assert_allclose(oracle.rms_swiglu(x, gamma, Wg, Wu, eps), want.numpy(), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("M,K,N,eps", [(5, 7, 3, 1e-5), (13, 64, 17, 0.1), (2, 1, 4, 0.0)])
def test_matmul_step_entries_match_plain_rows(M, K, N, eps):
    # the library-matmul entries used for full-row checks of the large workloads equal the plain
    # row loops (ln_linear, rms_linear, rms_swiglu, themselves pinned above) to rounding; a
    # transposed W, a dropped bias or a swapped gate/up fails here
    rng = np.random.default_rng(M + 7 * K + 11 * N)
    x = rng.normal(size=(M, K)) * 3 + 0.5
    gamma, beta = rng.uniform(0.5, 1.5, K), rng.normal(size=K) * 0.1
    W, Wu, bias = rng.normal(size=(K, N)), rng.normal(size=(K, N)), rng.normal(size=N)
    np.testing.assert_allclose(oracle.norm_linear_matmul(x, gamma, beta, W, bias, eps),
                               oracle.ln_linear(x, gamma, beta, W, bias, eps), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.norm_linear_matmul(x, gamma, None, W, None, eps, rms=True),
                               oracle.rms_linear(x, gamma, W, None, eps), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.norm_linear_matmul(x, gamma, beta, W, bias, eps, rms=True),
                               oracle.rms_linear(x, gamma, W, bias, eps, beta=beta), rtol=1e-12, atol=1e-12)
    np.testing.assert_allclose(oracle.rms_swiglu_matmul(x, gamma, W, Wu, eps),
                               oracle.rms_swiglu(x, gamma, W, Wu, eps), rtol=1e-12, atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_softmax_pv_matches_torch_softmax(causal):
    rng = np.random.default_rng(11)
    H, L, d = 3, 19, 5
    S, V = rng.normal(size=(H, L, L)) * 2, rng.normal(size=(H, L, d))
    St = torch.from_numpy(S)
    if causal:
        St = St.masked_fill(torch.triu(torch.ones(L, L, dtype=torch.bool), 1), float("-inf"))
    P = torch.softmax(St, dim=-1)
    want = torch.bmm(P, torch.from_numpy(V)).numpy().reshape(H * L, d)
    head = np.repeat(np.arange(H), L)
    qpos = np.tile(np.arange(L), H) if causal else None
    np.testing.assert_allclose(oracle.softmax(S.reshape(H * L, L), qpos), P.numpy().reshape(H * L, L),
                               rtol=1e-13, atol=1e-16)
    got = oracle.softmax_pv(S.reshape(H * L, L), V, head=head, qpos=qpos)
    np.testing.assert_allclose(got, want, rtol=1e-12, atol=1e-14)


def test_batched_linear_matches_matmul():
    rng = np.random.default_rng(12)
    a, W, bias = rng.normal(size=(3, 4, 6)), rng.normal(size=(3, 6, 5)), rng.normal(size=5)
    np.testing.assert_allclose(oracle.linear(a, W, bias), a @ W + bias, rtol=1e-13, atol=1e-13)


# --------------------------------------------------------------------------- the paper's fused forms
@pytest.mark.parametrize("M,K,N", [(6, 32, 9), (3, 5, 2)])
def test_eq5_fused_layernorm_equals_oracle(M, K, N):
    """Eq. (5): yF = 1/sqrt(var+eps) * (x (I - E/n) Gamma F) + beta F (+ bias)."""
    rng = np.random.default_rng(21)
    eps = 1e-3
    x = rng.normal(size=(M, K)) + 0.7
    gamma, beta, W, bias = rng.uniform(0.5, 1.5, K), rng.normal(size=K), rng.normal(size=(K, N)), rng.normal(size=N)
    centering = np.eye(K) - np.ones((K, K)) / K          # I - E/n, Eq. (3)
    static = centering @ np.diag(gamma) @ W              # computed once, as for static weights
    r = 1.0 / np.sqrt(np.var(x, axis=1) + eps)           # the collective sub-operation
    fused = r[:, None] * (x @ static) + beta @ W + bias
    np.testing.assert_allclose(oracle.ln_linear(x, gamma, beta, W, bias, eps), fused, rtol=1e-11, atol=1e-12)
    # the deferred form with the centering moved to the epilogue: r (x Gamma F - mean * 1 Gamma F) + beta F
    Wg = np.diag(gamma) @ W
    epi = r[:, None] * (x @ Wg - x.mean(axis=1)[:, None] * Wg.sum(axis=0)[None, :]) + beta @ W + bias
    np.testing.assert_allclose(oracle.ln_linear(x, gamma, beta, W, bias, eps), epi, rtol=1e-11, atol=1e-12)


@pytest.mark.parametrize("M,K,N", [(6, 32, 9), (3, 5, 2)])
def test_eq6_deferred_rmsnorm_equals_oracle(M, K, N):
    """Eq. (6) deferred past the product: r (x Gamma F) + beta F (+ bias), r = 1/sqrt(mean(x^2) + eps)."""
    rng = np.random.default_rng(23)
    eps = 1e-3
    x = rng.normal(size=(M, K)) + 0.7
    gamma, beta, W, bias = rng.uniform(0.5, 1.5, K), rng.normal(size=K), rng.normal(size=(K, N)), rng.normal(size=N)
    r = 1.0 / np.sqrt((x * x).mean(axis=1) + eps)        # the collective sub-operation
    fused = r[:, None] * (x @ (np.diag(gamma) @ W)) + beta @ W + bias
    np.testing.assert_allclose(oracle.rms_linear(x, gamma, W, bias, eps, beta=beta), fused, rtol=1e-11,
                               atol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_attention_matches_torch_sdpa(causal):
    rng = np.random.default_rng(24 + causal)
    H, L, d = 3, 19, 8
    Q, K, V = rng.normal(size=(H, L, d)), rng.normal(size=(H, L, d)), rng.normal(size=(H, L, d))
    scale = 1 / math.sqrt(d)
    want = torch.nn.functional.scaled_dot_product_attention(
        torch.from_numpy(Q), torch.from_numpy(K), torch.from_numpy(V), is_causal=causal, scale=scale).numpy()
    head, qpos = np.repeat(np.arange(H), L), np.tile(np.arange(L), H)
    got = oracle.attention(Q.reshape(-1, d), K, V, scale, head=head, qpos=qpos if causal else None)
    np.testing.assert_allclose(got, want.reshape(-1, d), rtol=1e-12, atol=1e-13)
    # and against the pinned softmax . V on scores formed independently
    S = np.einsum("hqd,hkd->hqk", Q, K) * scale
    ref = oracle.softmax_pv(S.reshape(-1, L), V, head=head, qpos=qpos if causal else None)
    np.testing.assert_allclose(got, ref, rtol=1e-12, atol=1e-13)


def test_attention_closed_forms():
    # K = 0: every score is 0, so row i averages the kept values (causal: V[0..i])
    rng = np.random.default_rng(25)
    L, d = 7, 3
    Q, V = rng.normal(size=(L, d)), rng.normal(size=(L, d))
    got = oracle.attention(Q, np.zeros((L, d)), V, 0.5, qpos=np.arange(L))
    want = np.cumsum(V, axis=0) / np.arange(1, L + 1)[:, None]
    np.testing.assert_allclose(got, want, rtol=1e-13, atol=1e-14)
    # one key aligned with the query and a huge scale: that key's value row
    K = np.eye(L, d)
    got = oracle.attention(np.eye(L, d)[2:3] * 50.0, K, V, 40.0)
    np.testing.assert_allclose(got[0], V[2], rtol=1e-12)


@pytest.mark.parametrize("causal", [False, True])
def test_eq8_fused_softmax_equals_oracle(causal):
    """Eq. (8): yV = (1 / sum_i e^{x_i}) ([e^{x_1} ... e^{x_n}] V)."""
    rng = np.random.default_rng(22)
    L, d = 12, 4
    S, V = rng.normal(size=(L, L)) * 2, rng.normal(size=(L, d))
    if causal:
        S = S.copy()
        S[np.triu_indices(L, 1)] = -np.inf
    e = np.exp(S - S.max(axis=1, keepdims=True))
    fused = (e @ V) / e.sum(axis=1, keepdims=True)
    np.testing.assert_allclose(oracle.softmax_pv(S, V, qpos=np.arange(L) if causal else None), fused,
                               rtol=1e-12, atol=1e-14)


# --------------------------------------------------------------------------- invariants
def test_layernorm_pre_affine_moments():
    rng = np.random.default_rng(31)
    M, K, eps = 8, 257, 0.05
    x = rng.normal(size=(M, K)) * rng.uniform(0.1, 3, size=(M, 1)) + rng.normal(size=(M, 1))
    y = oracle.layernorm(x, np.ones(K), np.zeros(K), eps)
    var = ((x - x.mean(1, keepdims=True)) ** 2).mean(1)
    np.testing.assert_allclose(y.mean(1), 0, atol=1e-14)
    np.testing.assert_allclose((y ** 2).mean(1), var / (var + eps), rtol=1e-13)


def test_layernorm_shift_and_scale_invariance_without_eps():
    rng = np.random.default_rng(32)
    K = 40
    x = rng.normal(size=(4, K))
    gamma, beta = rng.normal(size=K), rng.normal(size=K)
    a = oracle.layernorm(x, gamma, beta, 0.0)
    b = oracle.layernorm(3.5 * x - 2.25, gamma, beta, 0.0)
    np.testing.assert_allclose(a, b, rtol=1e-12, atol=1e-13)


def test_rmsnorm_k1_and_constant_rows():
    # K = 1: y = x / sqrt(x^2 + eps) * gamma; eps = 0 gives sign(x) * gamma
    for xv, eps in ((3.0, 16.0), (-0.5, 0.0), (2.0, 0.0)):
        want = xv / math.sqrt(xv * xv + eps) * 1.5
        assert oracle.rmsnorm(np.array([[xv]]), np.array([1.5]), eps)[0, 0] == pytest.approx(want, rel=1e-15)
    # constant row c (eps = 0): the root mean square is |c|, so y = sign(c) * gamma exactly
    gamma = np.array([0.5, -2.0, 3.0, 1.25])
    for c in (7.0, -0.375):
        np.testing.assert_array_equal(oracle.rmsnorm(np.full((1, 4), c), gamma, 0.0)[0], np.sign(c) * gamma)
    # a zero row: eps > 0 gives zeros (the linear layer then yields beta W + bias); eps = 0 gives 0/0
    assert (oracle.rmsnorm(np.zeros((1, 3)), np.ones(3), 1e-5) == 0).all()
    assert np.isnan(oracle.rmsnorm(np.zeros((1, 3)), np.ones(3), 0.0)).all()


def test_rmsnorm_pre_affine_mean_square_and_scale_invariance():
    rng = np.random.default_rng(36)
    M, K, eps = 8, 257, 0.05
    x = rng.normal(size=(M, K)) * rng.uniform(0.1, 3, size=(M, 1)) + rng.normal(size=(M, 1))
    y = oracle.rmsnorm(x, np.ones(K), eps)
    ms = (x * x).mean(1)
    np.testing.assert_allclose((y ** 2).mean(1), ms / (ms + eps), rtol=1e-13)
    gamma = rng.normal(size=K)
    a = oracle.rmsnorm(x, gamma, 0.0)
    np.testing.assert_allclose(oracle.rmsnorm(-2.5 * x, gamma, 0.0), -a, rtol=1e-13, atol=1e-14)
    # unlike LayerNorm it is not shift invariant ...
    assert not np.allclose(oracle.rmsnorm(x + 1.0, gamma, 0.0), a)
    # ... and on zero-mean rows it is LayerNorm (the pinned oracle) exactly in R
    xc = x - x.mean(1, keepdims=True)
    np.testing.assert_allclose(oracle.rmsnorm(xc, gamma, eps), oracle.layernorm(xc, gamma, None, eps),
                               rtol=1e-12, atol=1e-13)


def test_silu_closed_forms():
    # K = 1, x = 1, eps = 0: y = gamma exactly, so g = gamma * Wg and u = gamma * Wu.
    # SiLU(ln a) = ln a * a / (1 + a): ln 3 -> 0.75 ln 3, -ln 3 -> -0.25 ln 3
    l3 = math.log(3.0)
    h = oracle.rms_swiglu(np.ones((1, 1)), np.array([l3]), np.array([[1.0, -1.0]]), np.array([[2.0, 2.0]]), 0.0)
    np.testing.assert_allclose(h[0], [0.75 * l3 * 2 * l3, -0.25 * l3 * 2 * l3], rtol=4e-16)
    # a zero gate gives exactly zero; a large gate passes through (SiLU(z) -> z)
    rng = np.random.default_rng(37)
    x, g = rng.normal(size=(4, 16)), rng.uniform(0.5, 1.5, 16)
    Wu = rng.normal(size=(16, 5))
    assert (oracle.rms_swiglu(x, g, np.zeros((16, 5)), Wu, 1e-5) == 0).all()
    big = oracle.rms_swiglu(np.ones((1, 1)), np.array([1.0]), np.array([[60.0]]), np.array([[1.0]]), 0.0)
    assert big[0, 0] == 60.0


def test_swiglu_odd_part_identity():
    # SiLU(z) - SiLU(-z) = z, so h(Wg) - h(-Wg) = (y Wg) * (y Wu), with y Wg and y Wu from the
    # pinned RMSNorm -> Linear; a sign slip inside exp(-z) or a swapped gate/up fails this
    rng = np.random.default_rng(38)
    M, K, N, eps = 6, 24, 7, 1e-3
    x, gamma = rng.normal(size=(M, K)) + 0.2, rng.uniform(0.5, 1.5, K)
    Wg, Wu = rng.normal(size=(K, N)), rng.normal(size=(K, N))
    d = oracle.rms_swiglu(x, gamma, Wg, Wu, eps) - oracle.rms_swiglu(x, gamma, -Wg, Wu, eps)
    want = oracle.rms_linear(x, gamma, Wg, None, eps) * oracle.rms_linear(x, gamma, Wu, None, eps)
    np.testing.assert_allclose(d, want, rtol=1e-12, atol=1e-13)
    # and the deferred form: SiLU(r (x Gamma Wg)) * (r (x Gamma Wu)), r applied before the SiLU
    r = 1.0 / np.sqrt((x * x).mean(1) + eps)
    gg, uu = r[:, None] * (x @ (np.diag(gamma) @ Wg)), r[:, None] * (x @ (np.diag(gamma) @ Wu))
    np.testing.assert_allclose(oracle.rms_swiglu(x, gamma, Wg, Wu, eps), gg / (1 + np.exp(-gg)) * uu,
                               rtol=1e-12, atol=1e-13)


def test_softmax_rows_sum_to_one_and_shift_invariance():
    rng = np.random.default_rng(33)
    L = 50
    S = rng.normal(size=(L, L)) * 4
    for qpos in (None, np.arange(L)):
        P = oracle.softmax(S, qpos)
        np.testing.assert_allclose(P.sum(1), 1.0, rtol=1e-14)
        np.testing.assert_allclose(oracle.softmax(S + 7.5, qpos), P, rtol=1e-12, atol=1e-16)
    Pc = oracle.softmax(S, np.arange(L))
    assert (Pc[np.triu_indices(L, 1)] == 0).all()


def test_softmax_pv_output_within_value_hull():
    rng = np.random.default_rng(34)
    L, d = 30, 6
    S, V = rng.normal(size=(L, L)) * 3, rng.normal(size=(L, d))
    out = oracle.softmax_pv(S, V, qpos=np.arange(L))
    for i in range(L):
        assert np.all(out[i] <= V[: i + 1].max(0) + 1e-12)
        assert np.all(out[i] >= V[: i + 1].min(0) - 1e-12)


def test_threads_do_not_change_results():
    rng = np.random.default_rng(35)
    x, W = rng.normal(size=(37, 24)), rng.normal(size=(24, 11))
    g, b = rng.normal(size=24), rng.normal(size=24)
    np.testing.assert_array_equal(oracle.ln_linear(x, g, b, W, None, 1e-5, nthreads=1),
                                  oracle.ln_linear(x, g, b, W, None, 1e-5, nthreads=5))
    np.testing.assert_array_equal(oracle.rms_linear(x, g, W, None, 1e-5, nthreads=1),
                                  oracle.rms_linear(x, g, W, None, 1e-5, nthreads=6))
    S, V = rng.normal(size=(37, 37)), rng.normal(size=(37, 3))
    np.testing.assert_array_equal(oracle.softmax_pv(S, V, qpos=np.arange(37), nthreads=1),
                                  oracle.softmax_pv(S, V, qpos=np.arange(37), nthreads=7))


# --------------------------------------------------------------------------- brute force
def test_bruteforce_mpmath_tiny():
    mp = pytest.importorskip("mpmath")
    mp.mp.dps = 50
    rng = np.random.default_rng(41)
    M, K, N, eps = 3, 6, 4, 1e-3
    x, W = rng.normal(size=(M, K)), rng.normal(size=(K, N))
    g, b, bias = rng.normal(size=K), rng.normal(size=K), rng.normal(size=N)
    got = oracle.ln_linear(x, g, b, W, bias, eps)
    for m in range(M):
        xs = [mp.mpf(float(v)) for v in x[m]]
        mean = mp.fsum(xs) / K
        var = mp.fsum((v - mean) ** 2 for v in xs) / K
        y = [(xs[k] - mean) / mp.sqrt(var + mp.mpf(eps)) * mp.mpf(float(g[k])) + mp.mpf(float(b[k]))
             for k in range(K)]
        for n in range(N):
            ref = mp.fsum(y[k] * mp.mpf(float(W[k, n])) for k in range(K)) + mp.mpf(float(bias[n]))
            assert abs(float(ref) - got[m, n]) <= 1e-13 * max(1.0, abs(float(ref)))
    got = oracle.rms_linear(x, g, W, bias, eps, beta=b)
    for m in range(M):
        xs = [mp.mpf(float(v)) for v in x[m]]
        rms = mp.sqrt(mp.fsum(v * v for v in xs) / K + mp.mpf(eps))
        y = [xs[k] / rms * mp.mpf(float(g[k])) + mp.mpf(float(b[k])) for k in range(K)]
        for n in range(N):
            ref = mp.fsum(y[k] * mp.mpf(float(W[k, n])) for k in range(K)) + mp.mpf(float(bias[n]))
            assert abs(float(ref) - got[m, n]) <= 1e-13 * max(1.0, abs(float(ref)))
    Wu = rng.normal(size=(K, N))
    got = oracle.rms_swiglu(x, g, W, Wu, eps)
    for m in range(M):
        xs = [mp.mpf(float(v)) for v in x[m]]
        rms = mp.sqrt(mp.fsum(v * v for v in xs) / K + mp.mpf(eps))
        y = [xs[k] / rms * mp.mpf(float(g[k])) for k in range(K)]
        for n in range(N):
            gate = mp.fsum(y[k] * mp.mpf(float(W[k, n])) for k in range(K))
            up = mp.fsum(y[k] * mp.mpf(float(Wu[k, n])) for k in range(K))
            ref = gate / (1 + mp.exp(-gate)) * up
            assert abs(float(ref) - got[m, n]) <= 1e-13 * max(1.0, abs(float(ref)))
    L, d = 5, 3
    S, V = rng.normal(size=(L, L)) * 2, rng.normal(size=(L, d))
    got = oracle.softmax_pv(S, V, qpos=np.arange(L))
    for i in range(L):
        e = [mp.exp(mp.mpf(float(S[i, j]))) for j in range(i + 1)]
        tot = mp.fsum(e)
        for t in range(d):
            ref = mp.fsum(e[j] / tot * mp.mpf(float(V[j, t])) for j in range(i + 1))
            assert abs(float(ref) - got[i, t]) <= 1e-14 * max(1.0, abs(float(ref)))


def test_oracle_rejects_bad_arguments():
    with pytest.raises(ValueError):
        oracle.linear(np.zeros((1, 0)), np.zeros((0, 3)))


def test_bf16_inputs_widen_exactly():
    t = torch.tensor([1.0, -2.5, 3.140625, 1e-40, float("inf")], dtype=torch.bfloat16)
    np.testing.assert_array_equal(oracle.to_f64(t), t.double().numpy())
