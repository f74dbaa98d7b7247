"""fp64 CPU oracle for deferred normalization (arXiv 2502.17728).

TEST INFRASTRUCTURE ONLY.  The tests, the package smoke check and the
benchmark's CPU-baseline leg are the only callers; the product path never
imports this package.  It shares no code with the HIP library.

The arithmetic lives in ``dn_oracle.c`` (plain fp64 loops, see the header
comment there for the equations and readings).  This module only loads the
shared library, converts stored inputs exactly to fp64 and passes them in.

Stored bf16 values are widened bit-exactly (a bf16 is the top half of an
fp32), so the oracle sees exactly the values the GPU sees.
"""
from __future__ import annotations

import ctypes
import os
import subprocess

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_SRC = os.path.join(_HERE, "dn_oracle.c")
_LIB = os.path.join(_HERE, "liboracle.so")
_lib = None


def build(force: bool = True) -> str:
    """Compile dn_oracle.c into liboracle.so beside it (gcc, -O2, fp64)."""
    if force or not os.path.exists(_LIB):
        tmp = _LIB + ".tmp%d" % os.getpid()
        subprocess.check_call(
            ["gcc", "-O2", "-std=c11", "-Wall", "-Wextra", "-fPIC", "-shared",
             "-fno-fast-math", "-ffp-contract=off", _SRC, "-o", tmp,
             "-lm", "-lpthread"])
        os.replace(tmp, _LIB)
    return _LIB


def _load():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            build(force=True)
        lib = ctypes.CDLL(_LIB)
        d, i64, i32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int
        lib.oracle_layernorm.argtypes = [d, d, d, i64, i64, ctypes.c_double, d, i32]
        lib.oracle_linear.argtypes = [d, d, d, i64, i64, i64, i64, d, i32]
        lib.oracle_ln_linear.argtypes = [d, d, d, d, d, i64, i64, i64, ctypes.c_double, d, i32]
        lib.oracle_rmsnorm.argtypes = [d, d, d, i64, i64, ctypes.c_double, d, i32]
        lib.oracle_rms_linear.argtypes = [d, d, d, d, d, i64, i64, i64, ctypes.c_double, d, i32]
        lib.oracle_rms_swiglu.argtypes = [d, d, d, d, i64, i64, i64, ctypes.c_double, d, i32]
        lib.oracle_softmax.argtypes = [d, d, i64, i64, d, i32]
        lib.oracle_attention.argtypes = [d, d, d, d, d, i64, i64, i64, ctypes.c_double, d, i32]
        lib.oracle_softmax_pv.argtypes = [d, d, d, d, i64, i64, i64, d, i32]
        for f in ("oracle_layernorm", "oracle_linear", "oracle_ln_linear", "oracle_rmsnorm",
                  "oracle_rms_linear", "oracle_rms_swiglu", "oracle_softmax", "oracle_softmax_pv",
                  "oracle_attention"):
            getattr(lib, f).restype = ctypes.c_int
        _lib = lib
    return _lib


def to_f64(a) -> np.ndarray:
    """Exact widening of a stored input (torch bf16/fp32 tensor or numpy) to fp64."""
    try:
        import torch
        if isinstance(a, torch.Tensor):
            a = a.detach().cpu()
            if a.dtype == torch.bfloat16:
                bits = a.contiguous().view(torch.int16).numpy().astype(np.uint16)
                return (bits.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
            return a.contiguous().numpy().astype(np.float64)
    except ImportError:  # pragma: no cover
        pass
    return np.ascontiguousarray(np.asarray(a), dtype=np.float64)


def _ptr(a):
    return None if a is None else a.ctypes.data_as(ctypes.c_void_p)


def _threads(nthreads):
    if nthreads is None:
        return len(os.sched_getaffinity(0))
    return int(nthreads)


def _check(rc, name):
    if rc != 0:
        raise ValueError(f"{name}: invalid arguments (rc={rc})")


def layernorm(x, gamma, beta, eps, nthreads=None):
    """Eq. (1)-(2) per row of x[M, K]; returns y[M, K] in fp64."""
    x = to_f64(x)
    M, K = x.shape
    g = to_f64(gamma).reshape(K)
    b = None if beta is None else to_f64(beta).reshape(K)
    y = np.empty((M, K), np.float64)
    _check(_load().oracle_layernorm(_ptr(x), _ptr(g), _ptr(b), M, K, float(eps),
                                    _ptr(y), _threads(nthreads)), "layernorm")
    return y


def linear(a, W, bias=None, nthreads=None):
    """Eq. (4) product a[..., M, K] . W[..., K, N] + bias[N] in fp64 (batched over the leading dim)."""
    a = to_f64(a)
    W = to_f64(W)
    squeeze = a.ndim == 2
    if squeeze:
        a, W = a[None], W[None]
    B, M, K = a.shape
    N = W.shape[-1]
    assert W.shape == (B, K, N), (a.shape, W.shape)
    bb = None if bias is None else to_f64(bias).reshape(N)
    out = np.empty((B, M, N), np.float64)
    _check(_load().oracle_linear(_ptr(a), _ptr(W), _ptr(bb), B, M, K, N, _ptr(out),
                                 _threads(nthreads)), "linear")
    return out[0] if squeeze else out


def ln_linear(x, gamma, beta, W, bias, eps, nthreads=None):
    """Eq. (4): LayerNorm(x[M, K]) . W[K, N] + bias, fp64."""
    x = to_f64(x)
    M, K = x.shape
    W = to_f64(W)
    N = W.shape[1]
    g = to_f64(gamma).reshape(K)
    b = None if beta is None else to_f64(beta).reshape(K)
    bb = None if bias is None else to_f64(bias).reshape(N)
    out = np.empty((M, N), np.float64)
    _check(_load().oracle_ln_linear(_ptr(x), _ptr(g), _ptr(b), _ptr(W), _ptr(bb), M, K, N,
                                    float(eps), _ptr(out), _threads(nthreads)), "ln_linear")
    return out


def rmsnorm(x, gamma, eps, beta=None, nthreads=None):
    """Eq. (6) per row of x[M, K] (eps inside the root; beta optional); returns y[M, K] in fp64."""
    x = to_f64(x)
    M, K = x.shape
    g = to_f64(gamma).reshape(K)
    b = None if beta is None else to_f64(beta).reshape(K)
    y = np.empty((M, K), np.float64)
    _check(_load().oracle_rmsnorm(_ptr(x), _ptr(g), _ptr(b), M, K, float(eps),
                                  _ptr(y), _threads(nthreads)), "rmsnorm")
    return y


def rms_linear(x, gamma, W, bias, eps, beta=None, nthreads=None):
    """RMSNorm(x[M, K]) (Eq. (6)) . W[K, N] + bias, fp64."""
    x = to_f64(x)
    M, K = x.shape
    W = to_f64(W)
    N = W.shape[1]
    g = to_f64(gamma).reshape(K)
    b = None if beta is None else to_f64(beta).reshape(K)
    bb = None if bias is None else to_f64(bias).reshape(N)
    out = np.empty((M, N), np.float64)
    _check(_load().oracle_rms_linear(_ptr(x), _ptr(g), _ptr(b), _ptr(W), _ptr(bb), M, K, N,
                                     float(eps), _ptr(out), _threads(nthreads)), "rms_linear")
    return out


def rms_swiglu(x, gamma, Wg, Wu, eps, nthreads=None):
    """SiLU(RMSNorm(x) . Wg) * (RMSNorm(x) . Wu) for x[M, K], Wg/Wu[K, N]; returns h[M, N] fp64."""
    x = to_f64(x)
    M, K = x.shape
    Wg, Wu = to_f64(Wg), to_f64(Wu)
    N = Wg.shape[1]
    assert Wg.shape == (K, N) and Wu.shape == (K, N), (x.shape, Wg.shape, Wu.shape)
    g = to_f64(gamma).reshape(K)
    h = np.empty((M, N), np.float64)
    _check(_load().oracle_rms_swiglu(_ptr(x), _ptr(g), _ptr(Wg), _ptr(Wu), M, K, N, float(eps), _ptr(h),
                                     _threads(nthreads)), "rms_swiglu")
    return h


def _rows_meta(R, head, qpos):
    h = None if head is None else np.ascontiguousarray(np.asarray(head, np.int64).reshape(R))
    q = None if qpos is None else np.ascontiguousarray(np.asarray(qpos, np.int64).reshape(R))
    return h, q


def softmax(S_rows, qpos=None, nthreads=None):
    """Eq. (7) softmax of rows S_rows[R, Lk]; qpos[r] >= 0 applies the causal mask j <= qpos[r]."""
    S = to_f64(S_rows)
    R, Lk = S.shape
    _, q = _rows_meta(R, None, qpos)
    P = np.empty((R, Lk), np.float64)
    _check(_load().oracle_softmax(_ptr(S), _ptr(q), R, Lk, _ptr(P), _threads(nthreads)),
           "softmax")
    return P


def softmax_pv(S_rows, V, head=None, qpos=None, nthreads=None):
    """Eq. (7): softmax(S_rows[R, Lk]) . V[head[r]] with V[H, Lk, d]; returns [R, d] fp64."""
    S = to_f64(S_rows)
    R, Lk = S.shape
    V = to_f64(V)
    if V.ndim == 2:
        V = V[None]
    assert V.shape[1] == Lk, (S.shape, V.shape)
    d = V.shape[2]
    h, q = _rows_meta(R, head, qpos)
    if h is not None:
        assert h.min() >= 0 and h.max() < V.shape[0]
    out = np.empty((R, d), np.float64)
    _check(_load().oracle_softmax_pv(_ptr(S), _ptr(V), _ptr(h), _ptr(q), R, Lk, d, _ptr(out),
                                     _threads(nthreads)), "softmax_pv")
    return out


def attention(Q_rows, K, V, scale, head=None, qpos=None, nthreads=None):
    """softmax(scale * Q_rows[R, d] . K[head[r]]^T) . V[head[r]], K/V[H, Lk, d]; returns [R, d] fp64."""
    Q = to_f64(Q_rows)
    R, d = Q.shape
    K, V = to_f64(K), to_f64(V)
    if K.ndim == 2:
        K, V = K[None], V[None]
    assert K.shape == V.shape and K.shape[2] == d, (Q.shape, K.shape, V.shape)
    Lk = K.shape[1]
    h, q = _rows_meta(R, head, qpos)
    if h is not None:
        assert h.min() >= 0 and h.max() < K.shape[0]
    out = np.empty((R, d), np.float64)
    _check(_load().oracle_attention(_ptr(Q), _ptr(K), _ptr(V), _ptr(h), _ptr(q), R, Lk, d, float(scale),
                                    _ptr(out), _threads(nthreads)), "attention")
    return out


def norm_linear_matmul(x, gamma, beta, W, bias, eps, rms=False, nthreads=None):
    """LayerNorm (Eq. (1)-(2)) or RMSNorm (Eq. (6)) of x[M, K] by the C oracle, then the Eq. (4)
    product y . W + bias as one fp64 library matmul (numpy's BLAS), in place of the C row loop that
    streams all of W once per row.  Same definition, same fp64 operands; used to check every row of
    the large workloads.  Pinned against ln_linear / rms_linear in the oracle's tests."""
    y = rmsnorm(x, gamma, eps, beta=beta, nthreads=nthreads) if rms else \
        layernorm(x, gamma, beta, eps, nthreads=nthreads)
    out = y @ to_f64(W)
    if bias is not None:
        out += to_f64(bias).reshape(1, -1)
    return out


def rms_swiglu_matmul(x, gamma, Wg, Wu, eps, nthreads=None):
    """SiLU(RMSNorm(x) . Wg) * (RMSNorm(x) . Wu) with both products as fp64 library matmuls;
    SiLU(z) = z / (1 + e^-z).  Pinned against rms_swiglu in the oracle's tests."""
    y = rmsnorm(x, gamma, eps, nthreads=nthreads)
    g = y @ to_f64(Wg)
    u = y @ to_f64(Wu)
    return g / (1.0 + np.exp(-g)) * u
