"""The seeded synthetic workloads: determinism, shapes, distributions, rounding."""
import math

import numpy as np
import pytest
import torch

from paper_2502_17728_amd import inputs as I


def _rne_bf16_bits(f32: np.ndarray) -> np.ndarray:
    """Round-to-nearest-even fp32 -> bf16 written from the IEEE definition (finite inputs)."""
    u = f32.view(np.uint32).astype(np.uint64)
    lower = u & 0xFFFF
    upper = u >> 16
    round_up = (lower > 0x8000) | ((lower == 0x8000) & ((upper & 1) == 1))
    return (upper + round_up).astype(np.uint16)


def test_storage_cast_is_round_to_nearest_even():
    rng = np.random.default_rng(0)
    vals = np.concatenate([
        rng.normal(size=20000).astype(np.float32) * np.float32(3.0),
        # exact ties between two bf16 neighbours, both parities of the kept bit
        (np.arange(0x3F800000, 0x3F800000 + 64 * 0x10000, 0x10000, dtype=np.uint32) + 0x8000).view(np.float32),
        (np.arange(0x3F810000, 0x3F810000 + 64 * 0x10000, 0x10000, dtype=np.uint32) + 0x8000).view(np.float32),
        np.array([1e-40, -1e-40, 3.0e38, 0.0, -0.0], dtype=np.float32),
    ])
    got = I.to_storage(vals, "bf16").view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(got, _rne_bf16_bits(vals))


def test_generation_is_deterministic_and_seeded():
    a = I.make_ln_case(33, 64, 40, "bf16", seed=3)
    b = I.make_ln_case(33, 64, 40, "bf16", seed=3)
    c = I.make_ln_case(33, 64, 40, "bf16", seed=4)
    for k in ("x", "gamma", "beta", "W"):
        assert torch.equal(a[k], b[k])
        assert not torch.equal(a[k], c[k])


def test_head_subsets_equal_full_slices():
    w = I.SMWorkload("t", 9, 4, 40, 16, causal=True, from_qk=True)
    full = I.make_sm(w)
    part = I.make_sm(w, heads=[2, 0])
    assert torch.equal(part["S"][0], full["S"][2]) and torch.equal(part["V"][1], full["V"][0])


def test_decode_head_subsets_and_query_groups():
    # key/value head h carries query heads h*g .. h*g+g-1, each from its own stream, so a head
    # subset reproduces the matching slices of the full draw and g = 1 is the plain layout
    w = I.DecodeAttnWorkload("t", 12, 5, 2, 40, 16, group=3)
    full = I.make_decode(w)
    assert full["Q"].shape == (15, 2, 16) and full["K"].shape == (5, 40, 16)
    part = I.make_decode(w, heads=[4, 1])
    assert torch.equal(part["Q"][0:3], full["Q"][12:15]) and torch.equal(part["Q"][3:6], full["Q"][3:6])
    assert torch.equal(part["K"][0], full["K"][4]) and torch.equal(part["V"][1], full["V"][1])
    w1 = I.DecodeAttnWorkload("t1", 12, 5, 2, 40, 16)
    assert torch.equal(I.make_decode(w1)["Q"][1], full["Q"][1])  # query head 1 draws stream 1 in both layouts
    assert not torch.equal(full["Q"][0], full["Q"][1])
    g = I.ATTN_DECODE_GQA
    assert (g.BH, g.group, g.Lq, g.Lk, g.d) == (256, 4, 1, 8192, 128)
    assert g.bytes() == 2.0 * (2 * 256 * 8192 * 128 + 2 * 1024 * 128)


def test_ln_distributions():
    w = I.LNWorkload("t", 7, 512, 1024, 256, "f32", outliers=8)
    c = I.make_ln(w)
    x = c["x"].double()
    norm_cols = torch.tensor([(x[:, j].std() < 5).item() for j in range(w.K)])
    assert int((~norm_cols).sum()) == 8                              # eight fixed outlier channels
    xo = x[:, ~norm_cols]
    assert 17 < xo.std().item() < 23                                 # scaled x20
    xn = x[:, norm_cols]
    assert abs(xn.mean().item()) < 0.01 and abs(xn.std().item() - 1) < 0.01
    g = c["gamma"]
    assert g.min() >= 0.5 and g.max() <= 1.5
    assert abs(c["beta"].double().std().item() - math.sqrt(0.02)) < 0.02
    assert abs(c["W"].double().std().item() - 1 / math.sqrt(w.K)) < 0.01 / math.sqrt(w.K) * 10
    assert c["bias"] is None


def test_named_workloads_have_stated_shapes():
    assert (I.LN_F32_SMALL.M, I.LN_F32_SMALL.K, I.LN_F32_SMALL.N, I.LN_F32_SMALL.dtype) == (128, 768, 3072, "f32")
    assert (I.SM_BF16_SMALL.BH, I.SM_BF16_SMALL.L, I.SM_BF16_SMALL.d) == (12, 512, 64)
    assert (I.LN_QKV.M, I.LN_QKV.K, I.LN_QKV.N, I.LN_QKV.outliers) == (4096, 4096, 12288, 8)
    assert (I.SM_CAUSAL.BH, I.SM_CAUSAL.L, I.SM_CAUSAL.d, I.SM_CAUSAL.causal) == (32, 8192, 128, True)
    assert (I.LN_FFN_PREFILL.M, I.LN_FFN_PREFILL.K, I.LN_FFN_PREFILL.N) == (8192, 8192, 28672)
    assert I.ln_ffn_decode(4).M == 4
    c = I.make_ln(I.LN_F32_SMALL)
    assert c["x"].shape == (128, 768) and c["W"].shape == (768, 3072) and c["x"].dtype == torch.float32
    assert torch.count_nonzero(c["bias"]) == 0


def test_causal_scores_masked_and_scaled():
    w = I.SMWorkload("t", 8, 2, 256, 128, causal=True, from_qk=True)
    s = I.make_sm(w)["S"].float()
    L = w.L
    upper = torch.triu(torch.ones(L, L, dtype=torch.bool), 1)
    assert torch.isneginf(s[:, upper]).all()
    low = s[:, ~upper]
    assert torch.isfinite(low).all()
    assert abs(low.std().item() - 1.0) < 0.05          # Q.K / sqrt(d) with unit normals
    d = I.make_sm_case(3, 64, 64, False, s_std=2.0)
    assert abs(d["S"].float().std().item() - 2.0) < 0.05 and not torch.isinf(d["S"].float()).any()


def test_sample_rows():
    r = I.sample_rows(1000, 16, seed=1)
    assert len(r) == 16 and r[0] == 0 and r[-1] == 999 and len(set(r.tolist())) == 16
    assert I.sample_rows(5, 16).tolist() == [0, 1, 2, 3, 4]
