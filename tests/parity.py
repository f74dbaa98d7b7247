"""Shared helpers of the GPU parity tests (no method arithmetic here).

Error metric: per-row normwise relative error
    e = max_rows  max_n |gpu - oracle| / max_n |oracle|
(rows whose oracle output is all zero are compared absolutely).  An
element-wise relative error is ill-posed where outputs cross zero, as
LayerNorm->Linear outputs do.  Bounds: 1e-5 for fp32 inputs, 2e-2 for bf16
inputs with fp32 accumulation.
"""
import numpy as np
import torch

import oracle

TOL = {torch.float32: 1e-5, torch.bfloat16: 2e-2}


def rowwise_rel_err(got, ref) -> float:
    g = oracle.to_f64(got).reshape(-1, np.shape(ref)[-1])
    r = np.asarray(ref, np.float64).reshape(g.shape)
    nan_r = np.isnan(r)
    assert np.array_equal(np.isnan(g), nan_r), "NaN pattern differs from the oracle"
    g = np.where(nan_r, 0.0, g)
    r = np.where(nan_r, 0.0, r)
    assert np.isfinite(g).all(), "non-finite output where the oracle is finite"
    num = np.abs(g - r).max(axis=1)
    den = np.abs(r).max(axis=1)
    e = np.where(den > 0, num / np.where(den > 0, den, 1.0), num)
    return float(e.max()) if e.size else 0.0


def cuda(t):
    return None if t is None else t.cuda()
