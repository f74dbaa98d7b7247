"""Python binding of libdn (include/dn.h): argument marshalling only.

Every function here has the name of the C entry point it calls, takes torch
tensors that live on the GPU, passes their device pointers and sizes through
ctypes, and launches on the current torch stream (or the one given).  All
arithmetic happens in the HIP kernels; nothing here computes on the host, and
there is no fallback: if ``libdn.so`` is missing the import fails.
"""
from __future__ import annotations

import ctypes
import dataclasses
import os
from typing import Optional

import torch

_LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libdn.so")

DN_F32, DN_BF16 = 0, 1
DN_LN_LAYOUT_VERSION = 2
DN_SWIGLU_LAYOUT_VERSION = 0x102
STATUS = {0: "DN_OK", 1: "DN_ERR_INVALID_ARG", 2: "DN_ERR_UNSUPPORTED", 3: "DN_ERR_MISALIGNED", 4: "DN_ERR_HIP"}
SYMBOLS = ("dn_status_string", "dn_version", "ln_linear_packed_bytes", "ln_linear_prepare",
           "ln_linear_deferred", "rms_linear_deferred", "ln_linear_prepare_centered", "ln_linear_serial",
           "ln_linear_norm_on_load", "ln_linear_deferred_post", "rms_linear_deferred_post",
           "swiglu_packed_bytes", "swiglu_prepare", "rms_swiglu_deferred", "softmax_pv_deferred",
           "attention_deferred", "attention_gqa_deferred", "attention_decode_workspace_bytes",
           "attention_decode_deferred", "attention_decode_deferred_noalloc", "layernorm",
           "rmsnorm", "silu_mul", "softmax", "gemm")


class DNError(RuntimeError):
    def __init__(self, fn: str, status: int):
        super().__init__(f"{fn} failed: {STATUS.get(status, status)}")
        self.status = status


class LnLinearWeights(ctypes.Structure):
    """Mirror of ``ln_linear_weights`` in dn.h."""
    _fields_ = [("K", ctypes.c_int64), ("N", ctypes.c_int64), ("dtype", ctypes.c_int32),
                ("layout_version", ctypes.c_int32), ("packed", ctypes.c_void_p)]


def load_library(path: str = _LIB_PATH) -> ctypes.CDLL:
    if not os.path.exists(path):
        raise ImportError(f"libdn.so not found at {path}; build it with "
                          f"`python -m paper_2502_17728_amd.build` (needs hipcc for gfx950)")
    lib = ctypes.CDLL(path)
    vp, i64, i32, f32 = ctypes.c_void_p, ctypes.c_int64, ctypes.c_int, ctypes.c_float
    lib.dn_status_string.argtypes, lib.dn_status_string.restype = [i32], ctypes.c_char_p
    lib.dn_version.argtypes, lib.dn_version.restype = [], i32
    lib.ln_linear_packed_bytes.argtypes, lib.ln_linear_packed_bytes.restype = [i64, i64, i32], ctypes.c_size_t
    lib.ln_linear_prepare.argtypes = [vp, vp, vp, vp, i64, i64, i32, vp, ctypes.c_size_t,
                                      ctypes.POINTER(LnLinearWeights), vp]
    lib.ln_linear_deferred.argtypes = [vp, ctypes.POINTER(LnLinearWeights), i64, f32, vp, vp]
    lib.ln_linear_prepare_centered.argtypes = lib.ln_linear_prepare.argtypes
    lib.ln_linear_serial.argtypes = [vp, ctypes.POINTER(LnLinearWeights), i64, f32, vp, vp, vp]
    lib.ln_linear_norm_on_load.argtypes = [vp, ctypes.POINTER(LnLinearWeights), i64, f32, vp, vp, vp]
    lib.ln_linear_deferred_post.argtypes = [vp, ctypes.POINTER(LnLinearWeights), i64, f32, vp, vp, vp, vp, vp, vp]
    lib.rms_linear_deferred_post.argtypes = [vp, ctypes.POINTER(LnLinearWeights), i64, f32, vp, vp, vp, vp, vp]
    lib.rms_linear_deferred.argtypes = [vp, ctypes.POINTER(LnLinearWeights), i64, f32, vp, vp]
    lib.swiglu_packed_bytes.argtypes, lib.swiglu_packed_bytes.restype = [i64, i64, i32], ctypes.c_size_t
    lib.swiglu_prepare.argtypes = [vp, vp, vp, i64, i64, i32, vp, ctypes.c_size_t, ctypes.POINTER(LnLinearWeights),
                                   vp]
    lib.rms_swiglu_deferred.argtypes = [vp, ctypes.POINTER(LnLinearWeights), i64, f32, vp, vp]
    lib.silu_mul.argtypes = [vp, vp, i64, i32, vp, vp]
    lib.softmax_pv_deferred.argtypes = [vp, vp, i64, i64, i64, i64, i32, i32, vp, vp]
    lib.attention_deferred.argtypes = [vp, vp, vp, i64, i64, i64, i64, i32, f32, i32, vp, vp]
    lib.attention_gqa_deferred.argtypes = [vp, vp, vp, i64, i64, i64, i64, i64, i32, f32, i32, vp, vp]
    lib.attention_decode_workspace_bytes.argtypes = [i64, i64, i64, i64]
    lib.attention_decode_workspace_bytes.restype = ctypes.c_size_t
    lib.attention_decode_deferred.argtypes = [vp, vp, vp, i64, i64, i64, i64, f32, i32, vp, ctypes.c_size_t, vp, vp]
    lib.attention_decode_deferred_noalloc.argtypes = [vp, vp, vp, i64, i64, i64, i64, f32, i32, vp, vp]
    lib.layernorm.argtypes = [vp, vp, vp, i64, i64, f32, i32, vp, vp]
    lib.rmsnorm.argtypes = [vp, vp, i64, i64, f32, i32, vp, vp]
    lib.softmax.argtypes = [vp, i64, i64, i64, i32, i32, vp, vp]
    lib.gemm.argtypes = [vp, vp, vp, i64, i64, i64, i64, i32, i32, i32, vp, vp]
    for f in ("ln_linear_prepare", "ln_linear_deferred", "rms_linear_deferred", "ln_linear_prepare_centered",
              "ln_linear_serial", "ln_linear_norm_on_load", "ln_linear_deferred_post",
              "rms_linear_deferred_post", "swiglu_prepare", "rms_swiglu_deferred", "softmax_pv_deferred",
              "attention_deferred", "attention_gqa_deferred", "attention_decode_deferred",
              "attention_decode_deferred_noalloc", "layernorm", "rmsnorm",
              "silu_mul", "softmax",
              "gemm"):
        getattr(lib, f).restype = i32
    return lib


_lib = load_library()


def library_path() -> str:
    return _LIB_PATH


def _dt(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return DN_F32
    if t.dtype == torch.bfloat16:
        return DN_BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _dev(t: Optional[torch.Tensor], name: str):
    if t is None:
        return None
    if not t.is_cuda:
        raise ValueError(f"{name} must be a GPU tensor")
    if not t.is_contiguous():
        raise ValueError(f"{name} must be contiguous")
    return ctypes.c_void_p(t.data_ptr())


def _expect(t: Optional[torch.Tensor], name: str, shape=None, dtype=None, device=None, numel=None):
    """Check a tensor before its pointer reaches the C ABI, which sees only raw pointers and
    sizes: a wrong shape there becomes an out-of-bounds access on the GPU.  Raises ValueError
    on any mismatch; shape entries of None match any size."""
    if t is None:
        return
    if not isinstance(t, torch.Tensor):
        raise TypeError(f"{name} must be a torch.Tensor")
    if shape is not None:
        ok = t.dim() == len(shape) and all(s is None or int(a) == int(s) for a, s in zip(t.shape, shape))
        if not ok:
            want = "[" + ", ".join("*" if s is None else str(int(s)) for s in shape) + "]"
            raise ValueError(f"{name} has shape {list(t.shape)}, expected {want}")
    if numel is not None and t.numel() != numel:
        raise ValueError(f"{name} has {t.numel()} elements, expected {numel}")
    if dtype is not None and t.dtype != dtype:
        raise ValueError(f"{name} has dtype {t.dtype}, expected {dtype}")
    if device is not None and t.device != device:
        raise ValueError(f"{name} is on {t.device}, expected {device} (all tensors of a call share one device)")


_TORCH_DT = {DN_F32: torch.float32, DN_BF16: torch.bfloat16}


def _stream(stream) -> ctypes.c_void_p:
    if stream is None:
        stream = torch.cuda.current_stream()
    return ctypes.c_void_p(stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream))


def _check(fn: str, status: int):
    if status != 0:
        raise DNError(fn, status)


def _check_rows(x: torch.Tensor, w, out: Optional[torch.Tensor], stats: Optional[torch.Tensor] = None) -> int:
    """x[M, w.K] in the weights' dtype; out (if given) [M, w.N] like x; stats (if given) 2 M fp32."""
    if not isinstance(w, PreparedLinear):
        raise TypeError("w must come from ln_linear_prepare / swiglu_prepare")
    if x.dim() != 2:
        raise ValueError(f"x has shape {list(x.shape)}, expected [M, {w.K}]")
    M = x.shape[0]
    _expect(x, "x", (M, w.K), _TORCH_DT.get(w.desc.dtype), w.packed.device)
    _expect(out, "out", (M, w.N), x.dtype, x.device)
    _expect(stats, "stats", None, torch.float32, x.device, numel=2 * M)
    return M


@dataclasses.dataclass
class PreparedLinear:
    """Prepared static weights: the packed device buffer and its descriptor."""
    packed: torch.Tensor
    desc: LnLinearWeights

    @property
    def K(self):
        return self.desc.K

    @property
    def N(self):
        return self.desc.N


def ln_linear_packed_bytes(K: int, N: int, dtype: int) -> int:
    return int(_lib.ln_linear_packed_bytes(K, N, dtype))


def ln_linear_prepare(W: torch.Tensor, gamma: torch.Tensor, beta: Optional[torch.Tensor] = None,
                      bias: Optional[torch.Tensor] = None, stream=None, centered: bool = False) -> PreparedLinear:
    """centered=True calls ln_linear_prepare_centered (the literal Eq. (5) weight)."""
    if W.dim() != 2:
        raise ValueError(f"W has shape {list(W.shape)}, expected [K, N]")
    K, N = W.shape
    dt = _dt(W)
    _expect(gamma, "gamma", (K,), W.dtype, W.device)
    _expect(beta, "beta", (K,), W.dtype, W.device)
    _expect(bias, "bias", (N,), W.dtype, W.device)
    nbytes = ln_linear_packed_bytes(K, N, dt)
    if nbytes == 0:
        raise DNError("ln_linear_packed_bytes", 1)
    packed = torch.empty(nbytes, dtype=torch.uint8, device=W.device)
    desc = LnLinearWeights()
    fn = "ln_linear_prepare_centered" if centered else "ln_linear_prepare"
    _check(fn, getattr(_lib, fn)(
        _dev(W, "W"), _dev(gamma, "gamma"), _dev(beta, "beta"), _dev(bias, "bias"), K, N, dt,
        _dev(packed, "packed"), nbytes, ctypes.byref(desc), _stream(stream)))
    return PreparedLinear(packed, desc)


def ln_linear_deferred(x: torch.Tensor, w: PreparedLinear, eps: float = 1e-5,
                       out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    M = _check_rows(x, w, out)
    if out is None:
        out = torch.empty((M, w.N), dtype=x.dtype, device=x.device)
    _check("ln_linear_deferred", _lib.ln_linear_deferred(
        _dev(x, "x"), ctypes.byref(w.desc), M, eps, _dev(out, "out"), _stream(stream)))
    return out


def ln_linear_serial(x: torch.Tensor, w: PreparedLinear, eps: float = 1e-5, stats: Optional[torch.Tensor] = None,
                     out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    M = _check_rows(x, w, out, stats)
    if out is None:
        out = torch.empty((M, w.N), dtype=x.dtype, device=x.device)
    if stats is None:
        stats = torch.empty(2 * M, dtype=torch.float32, device=x.device)
    _check("ln_linear_serial", _lib.ln_linear_serial(
        _dev(x, "x"), ctypes.byref(w.desc), M, eps, _dev(stats, "stats"), _dev(out, "out"), _stream(stream)))
    return out


def ln_linear_norm_on_load(x: torch.Tensor, w: PreparedLinear, eps: float = 1e-5,
                           stats: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                           stream=None) -> torch.Tensor:
    """Ablation: statistics pre-pass, then x normalized on load into the product (no deferral)."""
    M = _check_rows(x, w, out, stats)
    if out is None:
        out = torch.empty((M, w.N), dtype=x.dtype, device=x.device)
    if stats is None:
        stats = torch.empty(2 * M, dtype=torch.float32, device=x.device)
    _check("ln_linear_norm_on_load", _lib.ln_linear_norm_on_load(
        _dev(x, "x"), ctypes.byref(w.desc), M, eps, _dev(stats, "stats"), _dev(out, "out"), _stream(stream)))
    return out


def linear_deferred_post(x: torch.Tensor, w: PreparedLinear, gamma: torch.Tensor, beta: Optional[torch.Tensor] = None,
                         eps: float = 1e-5, rms: bool = False, stats: Optional[torch.Tensor] = None,
                         y: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                         stream=None):
    """Post-LN placement: (out, y, stats) -- the deferred product and the normalized rows."""
    M = _check_rows(x, w, out, stats)
    K = w.K
    _expect(gamma, "gamma", (K,), x.dtype, x.device)
    _expect(beta, "beta", (K,), x.dtype, x.device)
    _expect(y, "y", (M, K), x.dtype, x.device)
    if out is None:
        out = torch.empty((M, w.N), dtype=x.dtype, device=x.device)
    if y is None:
        y = torch.empty_like(x)
    if stats is None:
        stats = torch.empty(2 * M, dtype=torch.float32, device=x.device)
    if rms:
        if beta is not None:
            raise ValueError("RMSNorm has no shift")
        st = _lib.rms_linear_deferred_post(_dev(x, "x"), ctypes.byref(w.desc), M, eps, _dev(gamma, "gamma"),
                                           _dev(stats, "stats"), _dev(y, "y"), _dev(out, "out"), _stream(stream))
        _check("rms_linear_deferred_post", st)
    else:
        st = _lib.ln_linear_deferred_post(_dev(x, "x"), ctypes.byref(w.desc), M, eps, _dev(gamma, "gamma"),
                                          _dev(beta, "beta"), _dev(stats, "stats"), _dev(y, "y"), _dev(out, "out"),
                                          _stream(stream))
        _check("ln_linear_deferred_post", st)
    return out, y, stats


def rms_linear_deferred(x: torch.Tensor, w: PreparedLinear, eps: float = 1e-5,
                        out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    M = _check_rows(x, w, out)
    if out is None:
        out = torch.empty((M, w.N), dtype=x.dtype, device=x.device)
    _check("rms_linear_deferred", _lib.rms_linear_deferred(
        _dev(x, "x"), ctypes.byref(w.desc), M, eps, _dev(out, "out"), _stream(stream)))
    return out


def swiglu_packed_bytes(K: int, N: int, dtype: int) -> int:
    return int(_lib.swiglu_packed_bytes(K, N, dtype))


def swiglu_prepare(W_gate: torch.Tensor, W_up: torch.Tensor, gamma: torch.Tensor, stream=None) -> PreparedLinear:
    if W_gate.dim() != 2:
        raise ValueError(f"W_gate has shape {list(W_gate.shape)}, expected [K, N]")
    K, N = W_gate.shape
    _expect(W_up, "W_up", (K, N), W_gate.dtype, W_gate.device)
    _expect(gamma, "gamma", (K,), W_gate.dtype, W_gate.device)
    dt = _dt(W_gate)
    nbytes = swiglu_packed_bytes(K, N, dt)
    if nbytes == 0:
        raise DNError("swiglu_packed_bytes", 1)
    packed = torch.empty(nbytes, dtype=torch.uint8, device=W_gate.device)
    desc = LnLinearWeights()
    _check("swiglu_prepare", _lib.swiglu_prepare(
        _dev(W_gate, "W_gate"), _dev(W_up, "W_up"), _dev(gamma, "gamma"), K, N, dt, _dev(packed, "packed"),
        nbytes, ctypes.byref(desc), _stream(stream)))
    return PreparedLinear(packed, desc)


def rms_swiglu_deferred(x: torch.Tensor, w: PreparedLinear, eps: float = 1e-5,
                        out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    M = _check_rows(x, w, out)
    if out is None:
        out = torch.empty((M, w.N), dtype=x.dtype, device=x.device)
    _check("rms_swiglu_deferred", _lib.rms_swiglu_deferred(
        _dev(x, "x"), ctypes.byref(w.desc), M, eps, _dev(out, "out"), _stream(stream)))
    return out


def softmax_pv_deferred(S: torch.Tensor, V: torch.Tensor, causal: bool = False,
                        out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    if S.dim() != 3 or V.dim() != 3:
        raise ValueError(f"S must be [BH, Lq, Lk] and V [BH, Lk, d]; got {list(S.shape)} and {list(V.shape)}")
    BH, Lq, Lk = S.shape
    d = V.shape[-1]
    _expect(V, "V", (BH, Lk, d), S.dtype, S.device)
    _expect(out, "out", (BH, Lq, d), S.dtype, S.device)
    if out is None:
        out = torch.empty((BH, Lq, d), dtype=S.dtype, device=S.device)
    _check("softmax_pv_deferred", _lib.softmax_pv_deferred(
        _dev(S, "S"), _dev(V, "V"), BH, Lq, Lk, d, int(causal), _dt(S), _dev(out, "out"), _stream(stream)))
    return out


def _check_qkv(Q, K, V, out):
    """Q[BHq, Lq, d], K and V [BH, Lk, d] with BHq a multiple of BH, one dtype and device; out like Q."""
    if Q.dim() != 3 or K.dim() != 3:
        raise ValueError(f"Q must be [BHq, Lq, d] and K, V [BH, Lk, d]; got {list(Q.shape)} and {list(K.shape)}")
    BHq, Lq, d = Q.shape
    BH, Lk = K.shape[0], K.shape[1]
    _expect(K, "K", (BH, Lk, d), Q.dtype, Q.device)
    _expect(V, "V", (BH, Lk, d), Q.dtype, Q.device)
    if BH < 1 or BHq % BH:
        raise ValueError(f"the query heads ({BHq}) must be a multiple of the key/value heads ({BH})")
    _expect(out, "out", tuple(Q.shape), Q.dtype, Q.device)
    return BHq, Lq, d, BH, Lk


def attention_deferred(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, causal: bool = False,
                       scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                       stream=None) -> torch.Tensor:
    """softmax(scale * Q K^T) V per query head; scale defaults to 1/sqrt(d).

    Q[BH * g, Lq, d], K/V[BH, Lk, d]: g = 1 is one key/value head per query head; g > 1 is
    grouped-query attention, query head h reading key/value head h // g.
    """
    BHq, Lq, d, BH, Lk = _check_qkv(Q, K, V, out)
    g = BHq // BH
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    if out is None:
        out = torch.empty_like(Q)
    if g == 1:
        st = _lib.attention_deferred(_dev(Q, "Q"), _dev(K, "K"), _dev(V, "V"), BH, Lq, Lk, d, int(causal),
                                     float(scale), _dt(Q), _dev(out, "out"), _stream(stream))
        _check("attention_deferred", st)
    else:
        st = _lib.attention_gqa_deferred(_dev(Q, "Q"), _dev(K, "K"), _dev(V, "V"), BH, g, Lq, Lk, d, int(causal),
                                         float(scale), _dt(Q), _dev(out, "out"), _stream(stream))
        _check("attention_gqa_deferred", st)
    return out


def attention_decode_workspace_bytes(BH: int, Lq: int, Lk: int, d: int) -> int:
    return int(_lib.attention_decode_workspace_bytes(BH, Lq, Lk, d))


def attention_decode_deferred(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, scale: Optional[float] = None,
                              workspace: Optional[torch.Tensor] = None, out: Optional[torch.Tensor] = None,
                              stream=None) -> torch.Tensor:
    """Decode attention (every key visible) split over key ranges, then merged.

    Q[BH * g, Lq, d] against K, V[BH, Lk, d]: with g > 1 (grouped-query attention) query
    heads h * g .. h * g + g - 1 share key/value head h, and the g heads' rows go through
    the kernel together as g * Lq (<= 16) queries of that head.
    """
    BHq, Lq, d, BH, Lk = _check_qkv(Q, K, V, out)
    _expect(workspace, "workspace", None, torch.uint8, Q.device)
    g = BHq // BH
    if out is None:
        out = torch.empty_like(Q)
    Q, out_k = Q.reshape(BH, g * Lq, d), out.view(BH, g * Lq, d)
    Lq = g * Lq
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    nbytes = attention_decode_workspace_bytes(BH, Lq, Lk, d)
    if workspace is None:
        workspace = torch.empty(max(nbytes, 16), dtype=torch.uint8, device=Q.device)
    _check("attention_decode_deferred", _lib.attention_decode_deferred(
        _dev(Q, "Q"), _dev(K, "K"), _dev(V, "V"), BH, Lq, Lk, d, float(scale), _dt(Q), _dev(workspace, "workspace"),
        workspace.numel() * workspace.element_size(), _dev(out_k, "out"), _stream(stream)))
    return out


def attention_decode_deferred_noalloc(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor,
                                      scale: Optional[float] = None, out: Optional[torch.Tensor] = None,
                                      stream=None) -> torch.Tensor:
    """attention_decode_deferred without a workspace: the partials live in the library's own
    device array (the C call allocates nothing; pass `out` to keep this wrapper from allocating
    the output).  Calls overlapping on one GPU share that array."""
    BHq, Lq, d, BH, Lk = _check_qkv(Q, K, V, out)
    g = BHq // BH
    if out is None:
        out = torch.empty_like(Q)
    if not (Q.is_contiguous() and out.is_contiguous()):
        raise ValueError("Q and out must be contiguous")
    Qg, out_k = Q.view(BH, g * Lq, d), out.view(BH, g * Lq, d)
    if scale is None:
        scale = 1.0 / float(d) ** 0.5
    _check("attention_decode_deferred_noalloc", _lib.attention_decode_deferred_noalloc(
        _dev(Qg, "Q"), _dev(K, "K"), _dev(V, "V"), BH, g * Lq, Lk, d, float(scale), _dt(Q), _dev(out_k, "out"),
        _stream(stream)))
    return out


def _check_norm(x, gamma, beta, out):
    if x.dim() != 2:
        raise ValueError(f"x has shape {list(x.shape)}, expected [M, K]")
    M, K = x.shape
    _expect(gamma, "gamma", (K,), x.dtype, x.device)
    _expect(beta, "beta", (K,), x.dtype, x.device)
    _expect(out, "out", (M, K), x.dtype, x.device)
    return M, K


def layernorm(x: torch.Tensor, gamma: torch.Tensor, beta: Optional[torch.Tensor] = None, eps: float = 1e-5,
              out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    M, K = _check_norm(x, gamma, beta, out)
    if out is None:
        out = torch.empty_like(x)
    _check("layernorm", _lib.layernorm(_dev(x, "x"), _dev(gamma, "gamma"), _dev(beta, "beta"), M, K, eps,
                                       _dt(x), _dev(out, "out"), _stream(stream)))
    return out


def rmsnorm(x: torch.Tensor, gamma: torch.Tensor, eps: float = 1e-5, out: Optional[torch.Tensor] = None,
            stream=None) -> torch.Tensor:
    M, K = _check_norm(x, gamma, None, out)
    if out is None:
        out = torch.empty_like(x)
    _check("rmsnorm", _lib.rmsnorm(_dev(x, "x"), _dev(gamma, "gamma"), M, K, eps, _dt(x), _dev(out, "out"),
                                   _stream(stream)))
    return out


def silu_mul(g: torch.Tensor, u: torch.Tensor, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    _expect(u, "u", tuple(g.shape), g.dtype, g.device)
    _expect(out, "out", None, g.dtype, g.device, numel=g.numel())
    if out is None:
        out = torch.empty_like(g)
    _check("silu_mul", _lib.silu_mul(_dev(g, "g"), _dev(u, "u"), g.numel(), _dt(g), _dev(out, "out"),
                                     _stream(stream)))
    return out


def softmax(S: torch.Tensor, causal: int = 0, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    if S.dim() != 3:
        raise ValueError(f"S has shape {list(S.shape)}, expected [BH, Lq, Lk]")
    BH, Lq, Lk = S.shape
    _expect(out, "out", tuple(S.shape), S.dtype, S.device)
    if out is None:
        out = torch.empty_like(S)
    _check("softmax", _lib.softmax(_dev(S, "S"), BH, Lq, Lk, int(causal), _dt(S), _dev(out, "out"),
                                   _stream(stream)))
    return out


def gemm(A: torch.Tensor, B, bias: Optional[torch.Tensor] = None, b_layout: int = 0,
         a_causal: bool = False, out: Optional[torch.Tensor] = None, stream=None) -> torch.Tensor:
    """C = A . B (+ bias).  B is a tensor ([K, N] for b_layout 0, [N, K] for 1, optionally
    batched) or a PreparedLinear (b_layout 2: the packed weights of ln_linear_prepare)."""
    if A.dim() not in (2, 3):
        raise ValueError(f"A has shape {list(A.shape)}, expected [M, K] or [batch, M, K]")
    squeeze = A.dim() == 2
    A3 = A.unsqueeze(0) if squeeze else A
    batch, M, K = A3.shape
    if isinstance(B, PreparedLinear):
        if B.K != K or _TORCH_DT.get(B.desc.dtype) != A.dtype:
            raise ValueError(f"the prepared weights are [{B.K}, {B.N}] of dtype {_TORCH_DT.get(B.desc.dtype)}; "
                             f"A is [*, {K}] of dtype {A.dtype}")
        if batch != 1:
            raise ValueError("prepared (packed) weights take an unbatched A")
        _expect(B.packed, "B", None, None, A.device)
        b_layout, N = 2, B.N
        bptr = None
    else:
        if b_layout not in (0, 1) or B.dim() not in (2, 3):
            raise ValueError("B must be [K, N] (b_layout 0) or [N, K] (b_layout 1), optionally batched")
        B3 = B.unsqueeze(0) if B.dim() == 2 else B
        N = B3.shape[2] if b_layout == 0 else B3.shape[1]
        _expect(B3, "B", (batch, K, N) if b_layout == 0 else (batch, N, K), A.dtype, A.device)
        bptr = None
    _expect(bias, "bias", (N,), A.dtype, A.device)
    _expect(out, "out", (batch, M, N), A.dtype, A.device)
    bptr = _dev(B.packed, "B") if isinstance(B, PreparedLinear) else _dev(B3, "B")
    if out is None:
        out = torch.empty((batch, M, N), dtype=A.dtype, device=A.device)
    _check("gemm", _lib.gemm(_dev(A3, "A"), bptr, _dev(bias, "bias"), batch, M, K, N, int(b_layout),
                             int(a_causal), _dt(A), _dev(out, "out"), _stream(stream)))
    return out[0] if squeeze else out
