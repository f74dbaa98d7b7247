"""The C ABI on the host: the library loads, exports every entry point that
include/dn.h declares, and rejects invalid calls before any HIP call (so
these run without a GPU; every call below fails validation)."""
import ctypes
import os
import re

import pytest

from paper_2502_17728_amd import ops

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
INVALID, UNSUPPORTED, MISALIGNED = 1, 2, 3
P = 0x7F0000000000  # aligned fake device addresses: never dereferenced by validation
P2 = P + (1 << 36)
P3 = P + (2 << 36)


def declared_symbols():
    text = open(os.path.join(ROOT, "include", "dn.h")).read()
    return sorted(set(re.findall(r"DN_API\s+[\w\s\*]+?\b(\w+)\s*\(", text)))


def test_header_and_binding_agree():
    assert declared_symbols() == sorted(ops.SYMBOLS)


def test_library_exports_every_declared_symbol():
    lib = ctypes.CDLL(ops.library_path())
    for name in declared_symbols():
        assert hasattr(lib, name), name


def test_status_strings_and_version():
    lib = ops._lib
    assert [lib.dn_status_string(i).decode() for i in range(5)] == [ops.STATUS[i] for i in range(5)]
    assert lib.dn_status_string(99) == b"DN_ERR_UNKNOWN"
    assert lib.dn_version() >= 1


def test_packed_bytes():
    f = ops.ln_linear_packed_bytes
    assert f(0, 8, 1) == 0 and f(8, 0, 1) == 0 and f(8, 8, 7) == 0
    assert f(4096, 12288, 1) == 4096 * 12288 * 2 + 2 * 12288 * 4   # Wt' + c + b, 256-aligned pieces
    assert f(768, 3072, 0) == 768 * 3072 * 4 + 2 * 3072 * 4
    assert f(8, 8, 1) % 256 == 0
    assert f(8, 8, 1) >= 16 * 32 * 2      # K padded to a 32-element chunk, N to 16 rows
    assert f(520, 24, 1) == (32 * 544 * 2) + 2 * 256


def _w(K=64, N=64, dtype=1, version=2, packed=P3):
    return ops.LnLinearWeights(K, N, dtype, version, packed)


@pytest.mark.parametrize("entry", ["ln_linear_deferred", "rms_linear_deferred"])
def test_ln_linear_deferred_validation(entry):
    f = getattr(ops._lib, entry)
    w = _w()
    assert f(None, ctypes.byref(w), 4, 1e-5, P2, None) == INVALID
    assert f(P, None, 4, 1e-5, P2, None) == INVALID
    assert f(P, ctypes.byref(w), 0, 1e-5, P2, None) == INVALID
    assert f(P, ctypes.byref(w), 4, -1.0, P2, None) == INVALID
    assert f(P, ctypes.byref(w), 4, float("nan"), P2, None) == INVALID
    assert f(P, ctypes.byref(w), 4, float("inf"), P2, None) == INVALID
    assert f(P, ctypes.byref(_w(version=0)), 4, 1e-5, P2, None) == INVALID
    assert f(P, ctypes.byref(_w(packed=None)), 4, 1e-5, P2, None) == INVALID
    assert f(P, ctypes.byref(_w(dtype=5)), 4, 1e-5, P2, None) == INVALID
    assert f(P, ctypes.byref(_w(K=60)), 4, 1e-5, P2, None) == UNSUPPORTED
    assert f(P + 8, ctypes.byref(w), 4, 1e-5, P2, None) == MISALIGNED
    assert f(P, ctypes.byref(w), 4, 1e-5, P2 + 2, None) == MISALIGNED
    assert f(P, ctypes.byref(_w(packed=P3 + 16)), 4, 1e-5, P2, None) == MISALIGNED
    assert f(P, ctypes.byref(w), 4, 1e-5, P + 128, None) == INVALID          # out overlaps x
    assert f(P, ctypes.byref(w), 4, 1e-5, P3 + 256, None) == INVALID         # out overlaps packed


def test_swiglu_validation():
    prep, f = ops._lib.swiglu_prepare, ops._lib.rms_swiglu_deferred
    nb = ops.swiglu_packed_bytes(64, 64, 1)
    assert nb > ops.ln_linear_packed_bytes(64, 64, 1)
    assert ops.swiglu_packed_bytes(0, 64, 1) == 0
    w = ops.LnLinearWeights()
    assert prep(None, P, P2, 64, 64, 1, P3, nb, ctypes.byref(w), None) == INVALID
    assert prep(P, P, P2, 64, 64, 1, P3, nb - 1, ctypes.byref(w), None) == INVALID
    assert prep(P, P, P2, 64, 60, 1, P3, 1 << 20, ctypes.byref(w), None) == UNSUPPORTED
    assert prep(P, P, P2, 64, 64, 1, P3 + 16, nb, ctypes.byref(w), None) == MISALIGNED
    assert prep(P, P2, P2 + 4096, 64, 64, 1, P2, nb, ctypes.byref(w), None) == INVALID  # packed overlaps W_up
    assert w.layout_version == 0
    sw = _w()
    sw.layout_version = ops.DN_SWIGLU_LAYOUT_VERSION
    assert f(P, ctypes.byref(_w()), 4, 1e-5, P2, None) == INVALID          # LayerNorm weights
    assert ops._lib.ln_linear_deferred(P, ctypes.byref(sw), 4, 1e-5, P2, None) == INVALID  # and back
    assert f(P, ctypes.byref(sw), 4, -1.0, P2, None) == INVALID
    assert f(P + 8, ctypes.byref(sw), 4, 1e-5, P2, None) == MISALIGNED
    assert f(P, ctypes.byref(sw), 4, 1e-5, P + 64, None) == INVALID         # h overlaps x
    sm = ops._lib.silu_mul
    assert sm(None, P2, 64, 1, P3, None) == INVALID
    assert sm(P, P2, 60, 1, P3, None) == UNSUPPORTED
    assert sm(P, P2 + 8, 64, 1, P3, None) == MISALIGNED
    assert sm(P, P2, 64, 1, P2, None) == INVALID


def test_ln_linear_serial_validation():
    f = ops._lib.ln_linear_serial
    w = _w()
    assert f(P, ctypes.byref(w), 4, 1e-5, None, P2, None) == INVALID                 # stats required
    assert f(P, ctypes.byref(w), 4, 1e-5, P3 + (1 << 30) + 4, P2, None) == MISALIGNED
    assert f(P, ctypes.byref(w), 4, 1e-5, P + 16, P2, None) == INVALID               # stats overlap x
    assert f(P, ctypes.byref(_w(K=1 << 15)), 4, 1e-5, P3 + (1 << 30), P2, None) == UNSUPPORTED  # K > row kernel
    assert f(P, ctypes.byref(_w(version=0)), 4, 1e-5, P3 + (1 << 30), P2, None) == INVALID


@pytest.mark.parametrize("rms", [False, True])
def test_linear_deferred_post_validation(rms):
    S, Y = P3 + (1 << 34), P3 + (1 << 35)
    w = _w()

    def f(x, g, b, st, y, out, ww=w, eps=1e-5):
        if rms:
            return ops._lib.rms_linear_deferred_post(x, ctypes.byref(ww), 4, eps, g, st, y, out, None)
        return ops._lib.ln_linear_deferred_post(x, ctypes.byref(ww), 4, eps, g, b, st, y, out, None)
    G = P + (1 << 33)
    assert f(P, None, None, S, Y, P2) == INVALID          # gamma required
    assert f(P, G, None, None, Y, P2) == INVALID          # stats required
    assert f(P, G, None, S, None, P2) == INVALID          # y required
    assert f(P, G, None, S, Y + 8, P2) == MISALIGNED
    assert f(P, G, None, S + 4, Y, P2) == MISALIGNED
    assert f(P, G, None, S, P + 64, P2) == INVALID        # y overlaps x
    assert f(P, G, None, P2 + 16, Y, P2) == INVALID       # stats overlap out
    assert f(P, G, None, S, Y, P2, ww=_w(K=68)) == UNSUPPORTED
    assert f(P, G, None, S, Y, P2, ww=_w(version=0)) == INVALID
    assert f(P, G, None, S, Y, P2, eps=-1.0) == INVALID  # the product's own checks still apply


def test_ln_linear_norm_on_load_validation():
    f = ops._lib.ln_linear_norm_on_load
    S = P3 + (1 << 34)
    big = _w(K=4096, N=4096)
    assert f(P, ctypes.byref(big), 4096, 1e-5, None, P2, None) == INVALID            # stats required
    assert f(P, ctypes.byref(_w()), 4, 1e-5, S, P2, None) == UNSUPPORTED            # below the large tiles
    assert f(P, ctypes.byref(_w(K=4096, N=4096, dtype=0)), 4096, 1e-5, S, P2, None) == UNSUPPORTED  # fp32
    assert f(P, ctypes.byref(_w(K=4104, N=4096)), 4096, 1e-5, S, P2, None) == UNSUPPORTED  # K % 64
    assert f(P, ctypes.byref(big), 4096, 1e-5, S + 4, P2, None) == MISALIGNED
    assert f(P, ctypes.byref(big), 4096, -1.0, S, P2, None) == INVALID


@pytest.mark.parametrize("entry", ["ln_linear_prepare", "ln_linear_prepare_centered"])
def test_ln_linear_prepare_validation(entry):
    f = getattr(ops._lib, entry)
    w = ops.LnLinearWeights()
    nb = ops.ln_linear_packed_bytes(64, 64, 1)
    assert f(None, P2, None, None, 64, 64, 1, P3, nb, ctypes.byref(w), None) == INVALID
    assert f(P, P2, None, None, 64, 64, 1, P3, nb - 1, ctypes.byref(w), None) == INVALID
    assert f(P, P2, None, None, 64, 64, 1, P3, nb, None, None) == INVALID
    assert f(P, P2, None, None, 64, 68, 1, P3, 1 << 20, ctypes.byref(w), None) == UNSUPPORTED
    assert f(P, P2, None, None, 64, 64, 1, P3 + 16, nb, ctypes.byref(w), None) == MISALIGNED
    assert f(P, P2, None, None, 64, 64, 1, P, nb, ctypes.byref(w), None) == INVALID   # packed overlaps W
    assert w.layout_version == 0  # untouched on failure


def test_softmax_pv_deferred_validation():
    f = ops._lib.softmax_pv_deferred
    assert f(None, P2, 1, 64, 64, 64, 0, 1, P3, None) == INVALID
    assert f(P, P2, 1, 64, 64, 64, 2, 1, P3, None) == INVALID            # causal must be 0/1
    assert f(P, P2, 1, 32, 64, 64, 1, 1, P3, None) == INVALID            # causal needs Lq == Lk
    assert f(P, P2, 0, 64, 64, 64, 0, 1, P3, None) == INVALID
    assert f(P, P2, 1, 64, 64, 64, 0, 0, P3, None) == UNSUPPORTED        # fp32 not implemented
    assert f(P, P2, 1, 64, 64, 96, 0, 1, P3, None) == UNSUPPORTED        # d must be 64 or 128
    assert f(P, P2, 1, 64, 60, 64, 0, 1, P3, None) == UNSUPPORTED        # Lk % 8
    assert f(P, P2, 1, 65536, 65536, 64, 1, 1, P3, None) == UNSUPPORTED  # one head's scores > 4 GiB
    assert f(P, P2, 1, 8, 1 << 24, 128, 0, 1, P3, None) == UNSUPPORTED    # one head's values >= 4 GiB
    assert f(P, P2 + 4, 1, 64, 64, 64, 0, 1, P3, None) == MISALIGNED
    assert f(P, P2, 1, 64, 64, 64, 0, 1, P + 64, None) == INVALID        # out overlaps S


def test_attention_deferred_validation():
    f = ops._lib.attention_deferred
    assert f(None, P2, P3, 1, 64, 64, 64, 0, 0.125, 1, P3 + (1 << 30), None) == INVALID
    assert f(P, P2, P3, 1, 64, 64, 64, 2, 0.125, 1, P3 + (1 << 30), None) == INVALID      # causal 0/1
    assert f(P, P2, P3, 1, 32, 64, 64, 1, 0.125, 1, P3 + (1 << 30), None) == INVALID      # causal: Lq == Lk
    assert f(P, P2, P3, 1, 64, 64, 64, 0, 0.0, 1, P3 + (1 << 30), None) == INVALID        # scale > 0
    assert f(P, P2, P3, 1, 64, 64, 64, 0, float("nan"), 1, P3 + (1 << 30), None) == INVALID
    assert f(P, P2, P3, 1, 64, 64, 64, 0, 0.125, 0, P3 + (1 << 30), None) == UNSUPPORTED  # bf16 only
    assert f(P, P2, P3, 1, 64, 64, 96, 0, 0.125, 1, P3 + (1 << 30), None) == UNSUPPORTED  # d 64 / 128
    assert f(P, P2, P3, 1, 1 << 23, 64, 128, 0, 0.125, 1, P3 + (1 << 30), None) == UNSUPPORTED
    assert f(P + 8, P2, P3, 1, 64, 64, 64, 0, 0.125, 1, P3 + (1 << 30), None) == MISALIGNED
    assert f(P, P2, P3, 1, 64, 64, 64, 0, 0.125, 1, P + 64, None) == INVALID              # out overlaps Q


def test_attention_gqa_validation():
    f = ops._lib.attention_gqa_deferred
    O = P + (1 << 33)
    assert f(P, P2, P3, 2, 0, 64, 64, 128, 1, 0.1, 1, O, None) == INVALID        # group >= 1
    assert f(P, P2, P3, 2, 4, 64, 32, 128, 1, 0.1, 1, O, None) == INVALID        # causal needs Lq == Lk
    assert f(P, P2, P3, 1 << 40, 1 << 40, 64, 64, 128, 0, 0.1, 1, O, None) == INVALID  # head count overflow
    assert f(P, P2, P3, 2, 4, 64, 64, 96, 0, 0.1, 1, O, None) == UNSUPPORTED
    assert f(P, P2, P3, 2, 4, 64, 64, 128, 0, 0.1, 1, O + 8, None) == MISALIGNED
    assert f(P, P2, P3, 2, 4, 64, 64, 128, 0, 0.1, 1, P + 4096, None) == INVALID  # out overlaps Q (8 heads)


def test_attention_decode_validation():
    f, wb = ops._lib.attention_decode_deferred, ops._lib.attention_decode_workspace_bytes
    assert wb(32, 1, 8192, 128) > 0
    assert wb(32, 17, 8192, 128) == 0 and wb(32, 1, 8192, 96) == 0 and wb(0, 1, 8, 64) == 0
    n = wb(2, 4, 1000, 64)
    W = P3 + (1 << 30)
    assert f(P, P2, P3, 2, 4, 1000, 64, 0.125, 1, None, n, P + (1 << 32), None) == INVALID   # workspace required
    assert f(P, P2, P3, 2, 4, 1000, 64, 0.125, 1, W, n - 1, P + (1 << 32), None) == INVALID  # too small
    assert f(P, P2, P3, 2, 17, 1000, 64, 0.125, 1, W, 1 << 20, P + (1 << 32), None) == UNSUPPORTED
    assert f(P, P2, P3, 2, 4, 1000, 64, -1.0, 1, W, n, P + (1 << 32), None) == INVALID
    assert f(P, P2, P3, 2, 4, 1000, 64, 0.125, 1, W + 4, n, P + (1 << 32), None) == MISALIGNED
    assert f(P, P2, P3, 2, 4, 1000, 64, 0.125, 1, P2, n, P + (1 << 32), None) == INVALID     # workspace over K


def test_attention_decode_noalloc_validation():
    f = ops._lib.attention_decode_deferred_noalloc
    O = P + (1 << 32)
    assert f(None, P2, P3, 2, 4, 1000, 64, 0.125, 1, O, None) == INVALID
    assert f(P, P2, P3, 2, 4, 1000, 64, 0.125, 1, None, None) == INVALID
    assert f(P, P2, P3, 0, 4, 1000, 64, 0.125, 1, O, None) == INVALID
    assert f(P, P2, P3, 2, 4, 1000, 64, float("nan"), 1, O, None) == INVALID
    assert f(P, P2, P3, 2, 17, 1000, 64, 0.125, 1, O, None) == UNSUPPORTED   # Lq > 16
    assert f(P, P2, P3, 2, 4, 1000, 96, 0.125, 1, O, None) == UNSUPPORTED    # d
    assert f(P, P2, P3, 2, 4, 1000, 64, 0.125, 0, O, None) == UNSUPPORTED    # fp32
    assert f(P, P2, P3, 2, 4, 1000, 64, 0.125, 1, O + 8, None) == MISALIGNED
    assert f(P, P2, P3, 2, 4, 1000, 64, 0.125, 1, P2, None) == INVALID       # out over K


def test_unfused_validation():
    ln, sm, gm = ops._lib.layernorm, ops._lib.softmax, ops._lib.gemm
    assert ln(None, P2, None, 4, 64, 1e-5, 1, P3, None) == INVALID
    assert ln(P, P2, None, 4, 64, -1e-5, 1, P3, None) == INVALID
    assert ln(P, P2, None, 4, 20, 1e-5, 1, P3, None) == UNSUPPORTED
    assert ln(P, P2, None, 4, 1 << 20, 1e-5, 1, P3, None) == UNSUPPORTED  # row kept in registers
    assert ln(P, P2, P + 8, 4, 64, 1e-5, 1, P3, None) == MISALIGNED
    assert ln(P, P2, None, 4, 64, 1e-5, 1, P, None) == INVALID           # in place not allowed
    rms = ops._lib.rmsnorm
    assert rms(None, P2, 4, 64, 1e-5, 1, P3, None) == INVALID
    assert rms(P, P2, 4, 64, float("nan"), 1, P3, None) == INVALID
    assert rms(P, P2, 0, 64, 1e-5, 1, P3, None) == INVALID
    assert rms(P, P2, 4, 20, 1e-5, 1, P3, None) == UNSUPPORTED
    assert rms(P, P2 + 8, 4, 64, 1e-5, 1, P3, None) == MISALIGNED
    assert rms(P, P2, 4, 64, 1e-5, 1, P + 64, None) == INVALID         # y overlaps x
    assert sm(P, 1, 64, 64, 3, 1, P2, None) == INVALID
    assert sm(P, 1, 64, 32, 1, 1, P2, None) == INVALID
    assert sm(P, 1, 64, 64, 0, 0, P2, None) == UNSUPPORTED
    assert sm(P, 1, 64, 64, 0, 1, P, None) == INVALID
    assert gm(P, P2, None, 1, 64, 64, 64, 3, 0, 1, P3, None) == INVALID   # b_layout
    assert gm(P, P2, None, 2, 64, 64, 64, 2, 0, 1, P3, None) == INVALID   # packed B is not batched
    assert gm(P, P2, None, 1, 64, 64, 64, 2, 1, 1, P3, None) == UNSUPPORTED  # causal A with packed B
    assert gm(P, P2 + 16, None, 1, 64, 64, 64, 2, 0, 1, P3, None) == MISALIGNED  # packed B is 256-aligned
    assert gm(P, P2, None, 1, 64, 32, 64, 0, 1, 1, P3, None) == INVALID   # causal needs M == K
    assert gm(P, P2, None, 1, 64, 64, 60, 0, 0, 1, P3, None) == UNSUPPORTED
    assert gm(P, P2, None, 1, 64, 64, 64, 0, 0, 0, P3, None) == UNSUPPORTED  # fp32 needs [N][K] B
    assert gm(P, P2, None, 70000, 8, 8, 8, 1, 0, 1, P3, None) == UNSUPPORTED
    assert gm(P, P2, None, 1, 64, 64, 64, 1, 0, 1, P2 + 64, None) == INVALID  # C overlaps B
    assert gm(P, P2, P3 + 2, 1, 64, 64, 64, 1, 0, 1, P3 + 4096, None) == MISALIGNED


def test_binding_rejects_host_tensors():
    import torch
    with pytest.raises(ValueError):
        ops.layernorm(torch.zeros(4, 64, dtype=torch.bfloat16), torch.ones(64, dtype=torch.bfloat16),
                      out=torch.zeros(4, 64, dtype=torch.bfloat16))


# ------------------------------------------------------------------ the binding's shape checks
# The C ABI sees raw pointers and sizes, so a mis-shaped tensor would reach the GPU as an
# out-of-bounds access.  The binding checks every tensor against the sizes it passes before
# taking any pointer; these calls use host tensors and fail on the shape (or dtype), never
# reaching the device check or the library.
def _bf(*shape):
    import torch
    return torch.zeros(*shape, dtype=torch.bfloat16)


def _prepared(K, N, dtype=1):
    import torch
    return ops.PreparedLinear(torch.zeros(64, dtype=torch.uint8), ops.LnLinearWeights(K, N, dtype, 2, None))


@pytest.mark.parametrize("fn", ["ln_linear_deferred", "rms_linear_deferred", "rms_swiglu_deferred",
                                "ln_linear_serial", "ln_linear_norm_on_load"])
def test_binding_checks_ln_shapes(fn):
    import torch
    f = getattr(ops, fn)
    w = _prepared(64, 32)
    with pytest.raises(ValueError, match="x has shape"):
        f(_bf(4, 72), w)                                   # K differs from the weights'
    with pytest.raises(ValueError, match="x has shape"):
        f(_bf(4, 8, 8), w)                                 # not 2-D
    with pytest.raises(ValueError, match="x has dtype"):
        f(torch.zeros(4, 64), w)                           # fp32 x, bf16 weights
    with pytest.raises(ValueError, match="out has shape"):
        f(_bf(4, 64), w, out=_bf(4, 16))
    with pytest.raises(ValueError, match="out has shape"):
        f(_bf(4, 64), w, out=_bf(5, 32))
    with pytest.raises(ValueError, match="out has dtype"):
        f(_bf(4, 64), w, out=torch.zeros(4, 32))
    with pytest.raises(ValueError, match="must be a GPU tensor"):
        f(_bf(4, 64), w, out=_bf(4, 32))                   # shapes right: only the device is wrong
    if fn in ("ln_linear_serial", "ln_linear_norm_on_load"):
        with pytest.raises(ValueError, match="stats has"):
            f(_bf(4, 64), w, stats=torch.zeros(6))
        with pytest.raises(ValueError, match="stats has dtype"):
            f(_bf(4, 64), w, stats=torch.zeros(8, dtype=torch.float64))


def test_binding_checks_post_and_prepare_shapes():
    import torch
    w = _prepared(64, 32)
    g = _bf(64)
    with pytest.raises(ValueError, match="gamma has shape"):
        ops.linear_deferred_post(_bf(4, 64), w, _bf(63))
    with pytest.raises(ValueError, match="beta has shape"):
        ops.linear_deferred_post(_bf(4, 64), w, g, _bf(32))
    with pytest.raises(ValueError, match="y has shape"):
        ops.linear_deferred_post(_bf(4, 64), w, g, y=_bf(4, 32))
    with pytest.raises(ValueError, match="stats has"):
        ops.linear_deferred_post(_bf(4, 64), w, g, stats=torch.zeros(4))
    with pytest.raises(ValueError, match="gamma has shape"):
        ops.ln_linear_prepare(_bf(64, 32), _bf(32))
    with pytest.raises(ValueError, match="bias has shape"):
        ops.ln_linear_prepare(_bf(64, 32), _bf(64), None, _bf(64))
    with pytest.raises(ValueError, match="gamma has dtype"):
        ops.ln_linear_prepare(_bf(64, 32), torch.ones(64))
    with pytest.raises(ValueError, match="W_up has shape"):
        ops.swiglu_prepare(_bf(64, 32), _bf(64, 24), _bf(64))
    with pytest.raises(ValueError, match="gamma has shape"):
        ops.swiglu_prepare(_bf(64, 32), _bf(64, 32), _bf(32))


def test_binding_checks_softmax_and_attention_shapes():
    import torch
    with pytest.raises(ValueError, match="V has shape"):
        ops.softmax_pv_deferred(_bf(2, 64, 128), _bf(2, 64, 64))       # V rows != Lk
    with pytest.raises(ValueError, match="V has shape"):
        ops.softmax_pv_deferred(_bf(2, 64, 64), _bf(1, 64, 64))        # heads differ
    with pytest.raises(ValueError, match="V has dtype"):
        ops.softmax_pv_deferred(_bf(2, 64, 64), torch.zeros(2, 64, 64))
    with pytest.raises(ValueError, match="out has shape"):
        ops.softmax_pv_deferred(_bf(2, 64, 64), _bf(2, 64, 128), out=_bf(2, 64, 64))
    with pytest.raises(ValueError, match="out has shape"):
        ops.softmax(_bf(2, 64, 64), out=_bf(2, 64, 32))
    for call in (ops.attention_deferred, ops.attention_decode_deferred):
        with pytest.raises(ValueError, match="K has shape"):
            call(_bf(4, 1, 128), _bf(4, 100, 64), _bf(4, 100, 64))     # head dims differ
        with pytest.raises(ValueError, match="V has shape"):
            call(_bf(4, 1, 128), _bf(4, 100, 128), _bf(4, 90, 128))
        with pytest.raises(ValueError, match="multiple of the key/value heads"):
            call(_bf(6, 1, 128), _bf(4, 100, 128), _bf(4, 100, 128))
        with pytest.raises(ValueError, match="out has shape"):
            call(_bf(4, 1, 128), _bf(4, 100, 128), _bf(4, 100, 128), out=_bf(4, 2, 128))
    with pytest.raises(ValueError, match="workspace has dtype"):
        ops.attention_decode_deferred(_bf(4, 1, 128), _bf(4, 100, 128), _bf(4, 100, 128),
                                      workspace=torch.zeros(16))


def test_binding_checks_norm_and_gemm_shapes():
    import torch
    with pytest.raises(ValueError, match="gamma has shape"):
        ops.layernorm(_bf(4, 64), _bf(32))
    with pytest.raises(ValueError, match="beta has shape"):
        ops.layernorm(_bf(4, 64), _bf(64), _bf(32))
    with pytest.raises(ValueError, match="out has shape"):
        ops.rmsnorm(_bf(4, 64), _bf(64), out=_bf(4, 32))
    with pytest.raises(ValueError, match="u has shape"):
        ops.silu_mul(_bf(4, 64), _bf(4, 32))
    with pytest.raises(ValueError, match="B has shape"):
        ops.gemm(_bf(4, 64), _bf(32, 16))                  # [K, N] with K != A's K
    with pytest.raises(ValueError, match="B has shape"):
        ops.gemm(_bf(2, 4, 64), _bf(3, 64, 16))            # batch differs
    with pytest.raises(ValueError, match="B has shape"):
        ops.gemm(_bf(4, 64), _bf(16, 32), b_layout=1)      # [N, K] with K != 64
    with pytest.raises(ValueError, match="bias has shape"):
        ops.gemm(_bf(4, 64), _bf(64, 16), bias=_bf(32))
    with pytest.raises(ValueError, match="out has shape"):
        ops.gemm(_bf(4, 64), _bf(64, 16), out=_bf(1, 4, 8))
    with pytest.raises(ValueError, match="prepared"):
        ops.gemm(_bf(4, 72), _prepared(64, 16))
    with pytest.raises(ValueError, match="B has dtype"):
        ops.gemm(_bf(4, 64), torch.zeros(64, 16))
