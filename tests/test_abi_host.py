"""The C-ABI library on the host: it loads, exports every declared symbol, and
its descriptor validation (no device access) accepts and rejects the right
groups."""
import ctypes
import os
import re

import pytest

from paper_2607_02945_amd import binding as B

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
OK, INVALID, UNSUPPORTED, ALIASING = 0, -1, -2, -3

pytestmark = pytest.mark.skipif(not os.path.exists(B.LIBPATH), reason="liboptimus.so not built")


def test_exports_match_header():
    hdr = open(os.path.join(ROOT, "include", "optimus.h")).read()
    declared = set(re.findall(r"\b(optimus_[a-z0-9_]+)\s*\(", hdr))
    assert declared == set(B.EXPORTS)
    lib = B.lib()
    for name in declared:
        assert hasattr(lib, name), name
    assert "gfx950" in B.optimus_version()


def lin(x, w, y, M=64, N=32, K=48, ldx=None, ldw=None, ldy=None, bias=None):
    return B.LinearDesc(x, ldx or K, w, ldw or K, bias, y, ldy or N, M, N, K)


def lin_arr(*descs):
    a = (B.LinearDesc * len(descs))(*descs)
    return a, len(descs)


MB = 1 << 20


def test_linear_validation():
    a, G = lin_arr(lin(1 * MB, 2 * MB, 3 * MB), lin(4 * MB, 5 * MB, 6 * MB, M=7, N=5, K=3))
    assert B.optimus_validate_linear(a, G, B.BF16) == OK
    assert B.optimus_validate_linear(a, 0, B.BF16) == OK
    assert B.optimus_validate_linear(a, -1, B.BF16) == INVALID
    assert B.optimus_validate_linear(a, G, 7) == UNSUPPORTED
    assert B.optimus_validate_linear(a, G, B.F32, 9) == UNSUPPORTED
    for bad in [lin(0, 2 * MB, 3 * MB), lin(1 * MB, 0, 3 * MB), lin(1 * MB, 2 * MB, 0),
                lin(1 * MB, 2 * MB, 3 * MB, M=0), lin(1 * MB, 2 * MB, 3 * MB, K=0),
                lin(1 * MB, 2 * MB, 3 * MB, ldx=47), lin(1 * MB, 2 * MB, 3 * MB, ldy=31),
                lin(1 * MB, 2 * MB, 3 * MB, M=1 << 31)]:
        a, G = lin_arr(bad)
        assert B.optimus_validate_linear(a, G, B.BF16) == INVALID
        assert B.optimus_last_error()


def test_linear_aliasing():
    # output of member 1 lands inside member 0's input
    a, G = lin_arr(lin(1 * MB, 2 * MB, 3 * MB), lin(4 * MB, 5 * MB, 1 * MB + 1024))
    assert B.optimus_validate_linear(a, G, B.BF16) == ALIASING
    assert "independent" in B.optimus_last_error()
    # in place is never allowed for a GEMM
    a, G = lin_arr(lin(1 * MB, 2 * MB, 1 * MB, M=8, N=8, K=8))
    assert B.optimus_validate_linear(a, G, B.F32) == ALIASING
    # two outputs overlapping
    a, G = lin_arr(lin(1 * MB, 2 * MB, 3 * MB), lin(4 * MB, 5 * MB, 3 * MB + 64))
    assert B.optimus_validate_linear(a, G, B.BF16) == ALIASING
    # shared input and shared weights are fine (inputs may overlap inputs)
    a, G = lin_arr(lin(1 * MB, 2 * MB, 3 * MB), lin(1 * MB, 2 * MB, 4 * MB))
    assert B.optimus_validate_linear(a, G, B.BF16) == OK
    # bias overlapping an output
    a, G = lin_arr(lin(1 * MB, 2 * MB, 3 * MB, bias=3 * MB + 2))
    assert B.optimus_validate_linear(a, G, B.BF16) == ALIASING


def ptrs(*vals):
    return (ctypes.c_void_p * len(vals))(*vals)


def test_linear_layernorm_validation():
    """The fused Linear + LayerNorm: the Linear checks, a finite eps >= 0, rows
    that fit one output tile (bf16 256, fp32 128), gamma/beta never overlapping
    an output."""
    a, G = lin_arr(lin(1 * MB, 2 * MB, 3 * MB, N=256), lin(4 * MB, 5 * MB, 6 * MB, N=17))
    g, b = ptrs(7 * MB, 8 * MB), ptrs(9 * MB, None)
    V = B.optimus_validate_linear_layernorm
    assert V(a, g, b, G, B.BF16) == OK
    assert V(a, None, None, G, B.BF16) == OK
    assert V(a, g, b, 0, B.BF16) == OK
    assert V(a, g, b, G, B.BF16, eps=-1.0) == INVALID
    assert V(a, g, b, G, B.BF16, eps=float("inf")) == INVALID
    assert V(a, g, b, G, B.BF16, act=9) == UNSUPPORTED
    assert V(a, g, b, G, B.F32) == UNSUPPORTED  # N = 256 > 128 for fp32
    assert "at most 128" in B.optimus_last_error()
    a1, G1 = lin_arr(lin(1 * MB, 2 * MB, 3 * MB, N=257))
    assert V(a1, None, None, G1, B.BF16) == UNSUPPORTED
    a2, G2 = lin_arr(lin(1 * MB, 2 * MB, 3 * MB, N=128))
    assert V(a2, None, None, G2, B.F32) == OK
    # gamma inside member 1's output
    assert V(a, ptrs(7 * MB, 6 * MB + 8), b, G, B.BF16) == ALIASING
    # the plain Linear rule still holds (no in place)
    a3, G3 = lin_arr(lin(1 * MB, 2 * MB, 1 * MB, M=8, N=8, K=8))
    assert V(a3, None, None, G3, B.BF16) == ALIASING


def pw(x, y, rows, cols, ldx, ldy):
    return B.PointwiseDesc(x, ldx, y, ldy, rows, cols)


def test_column_slices_of_one_buffer_are_independent():
    # 4 outputs: column slices [0,16) [16,48) [48,64) [64,128) of one [100, 128] bf16 buffer
    out, inp = 8 * MB, 16 * MB
    cuts = [0, 16, 48, 64, 128]
    ds = [pw(inp + 2 * c0, out + 2 * c0, 100, c1 - c0, 128, 128) for c0, c1 in zip(cuts, cuts[1:])]
    arr = (B.PointwiseDesc * 4)(*ds)
    assert B.optimus_validate_pointwise(arr, 4, B.BF16) == OK
    # exact in-place members are allowed
    ds = [pw(out + 2 * c0, out + 2 * c0, 100, c1 - c0, 128, 128) for c0, c1 in zip(cuts, cuts[1:])]
    arr = (B.PointwiseDesc * 4)(*ds)
    assert B.optimus_validate_pointwise(arr, 4, B.BF16) == OK
    # one column of overlap between neighbouring slices
    ds = [pw(inp, out, 100, 17, 128, 128), pw(inp + 32, out + 32, 100, 16, 128, 128)]
    arr = (B.PointwiseDesc * 2)(*ds)
    assert B.optimus_validate_pointwise(arr, 2, B.BF16) == ALIASING
    # disjoint columns but the second slice's rows wrap into the first (stride mismatch -> conservative)
    ds = [pw(inp, out, 100, 16, 128, 128), pw(inp + 64, out + 64, 100, 16, 64, 64)]
    arr = (B.PointwiseDesc * 2)(*ds)
    assert B.optimus_validate_pointwise(arr, 2, B.BF16) == ALIASING
    # an in-place member whose input is shifted by one row is not in place
    ds = [pw(out, out + 256, 100, 128, 128, 128)]
    arr = (B.PointwiseDesc * 1)(*ds)
    assert B.optimus_validate_pointwise(arr, 1, B.BF16) == ALIASING


def test_layernorm_validation():
    d = B.LayerNormDesc(1 * MB, 64, 2 * MB, 64, 3 * MB, 3 * MB + 4096, 100, 64, 1e-5)
    arr = (B.LayerNormDesc * 1)(d)
    assert B.optimus_validate_layernorm(arr, 1, B.F32, "tanh") == OK
    for field, val, want in [("rows", 0, INVALID), ("cols", 0, INVALID), ("ldx", 63, INVALID),
                             ("eps", -1.0, INVALID), ("eps", float("nan"), INVALID), ("x", None, INVALID),
                             ("gamma", 2 * MB + 128, ALIASING)]:
        bad = B.LayerNormDesc(1 * MB, 64, 2 * MB, 64, 3 * MB, 3 * MB + 4096, 100, 64, 1e-5)
        setattr(bad, field, val)
        arr = (B.LayerNormDesc * 1)(bad)
        assert B.optimus_validate_layernorm(arr, 1, B.F32) == want, field
    # in place is allowed for LayerNorm
    d = B.LayerNormDesc(1 * MB, 64, 1 * MB, 64, None, None, 100, 64, 1e-5)
    assert B.optimus_validate_layernorm((B.LayerNormDesc * 1)(d), 1, B.BF16) == OK


def soc(inp, out, widths, rows=10, ld=None, gam=None, bet=None, ln=1):
    n = len(widths)
    D = sum(widths)
    w = (ctypes.c_int64 * n)(*widths)
    g = None if gam is None else (ctypes.c_void_p * n)(*gam)
    b = None if bet is None else (ctypes.c_void_p * n)(*bet)
    d = B.SplitOpCatDesc(inp, ld or D, out, ld or D, rows, D, n, w, g, b, ln, 1e-5, 4)
    return d, (w, g, b)


def test_split_op_cat_validation():
    d, keep = soc(1 * MB, 2 * MB, [2, 2, 2])
    assert B.optimus_validate_split_op_cat(d, B.BF16) == OK
    d, keep = soc(1 * MB, 1 * MB, [16, 48])   # in place
    assert B.optimus_validate_split_op_cat(d, B.BF16) == OK
    d, keep = soc(1 * MB, 1 * MB + 64, [16, 48])   # shifted: overlaps
    assert B.optimus_validate_split_op_cat(d, B.BF16) == ALIASING
    d, keep = soc(1 * MB, 2 * MB, [2, 0, 4])
    assert B.optimus_validate_split_op_cat(d, B.BF16) == INVALID
    d, keep = soc(1 * MB, 2 * MB, [2, 2, 2])
    d.D = 7
    d.ldin = d.ldout = 7
    assert B.optimus_validate_split_op_cat(d, B.BF16) == INVALID
    assert "sum" in B.optimus_last_error()
    d, keep = soc(1 * MB, 2 * MB, [8, 8], gam=[3 * MB, 2 * MB + 8], bet=[None, None])
    assert B.optimus_validate_split_op_cat(d, B.BF16) == ALIASING
    d, keep = soc(1 * MB, 2 * MB, [8, 8])
    d.act = 11
    assert B.optimus_validate_split_op_cat(d, B.BF16) == UNSUPPORTED


def q8(x, q, scale=None, rows=64, cols=48, ldx=None, ldq=None):
    return B.Fp8QuantDesc(x, ldx or cols, q, ldq or cols, scale, rows, cols)


def dq8(q, y, scale=None, rows=64, cols=48, ldq=None, ldy=None):
    return B.Fp8DequantDesc(q, ldq or cols, scale, y, ldy or cols, rows, cols)


def test_fp8_codec_validation():
    arr = lambda T, *ds: ((T * len(ds))(*ds), len(ds))
    a, G = arr(B.Fp8QuantDesc, q8(1 * MB, 2 * MB, 3 * MB), q8(4 * MB, 5 * MB, 3 * MB + 4, rows=7, cols=5))
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 1) == OK
    assert B.optimus_validate_quantize_fp8(a, G, B.F32, 0) == OK
    assert B.optimus_validate_quantize_fp8(a, 0, B.BF16, 1) == OK
    assert B.optimus_validate_quantize_fp8(a, -1, B.BF16, 1) == INVALID
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 2) == INVALID
    assert "use_scaling" in B.optimus_last_error()
    assert B.optimus_validate_quantize_fp8(a, G, 5, 1) == UNSUPPORTED
    # scaled needs a scale pointer; unscaled does not
    a, G = arr(B.Fp8QuantDesc, q8(1 * MB, 2 * MB))
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 1) == INVALID
    assert "scale" in B.optimus_last_error()
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 0) == OK
    for bad in [q8(0, 2 * MB), q8(1 * MB, 0), q8(1 * MB, 2 * MB, rows=0), q8(1 * MB, 2 * MB, cols=0),
                q8(1 * MB, 2 * MB, ldx=47), q8(1 * MB, 2 * MB, ldq=40), q8(1 * MB, 2 * MB, rows=1 << 31)]:
        a, G = arr(B.Fp8QuantDesc, bad)
        assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 0) == INVALID, bad
    # codes over the values (bf16 values take 2 bytes each: 64 x 48 x 2 = 6 KiB)
    a, G = arr(B.Fp8QuantDesc, q8(1 * MB, 1 * MB + 4096))
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 0) == ALIASING
    a, G = arr(B.Fp8QuantDesc, q8(1 * MB, 1 * MB + 6144))
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 0) == OK
    # no in-place, even at equal pointers and strides
    a, G = arr(B.Fp8QuantDesc, q8(1 * MB, 1 * MB))
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 0) == ALIASING
    # two members writing one scale, or a scale inside a member's codes
    a, G = arr(B.Fp8QuantDesc, q8(1 * MB, 2 * MB, 3 * MB), q8(4 * MB, 5 * MB, 3 * MB))
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 1) == ALIASING
    a, G = arr(B.Fp8QuantDesc, q8(1 * MB, 2 * MB, 2 * MB + 100))
    assert B.optimus_validate_quantize_fp8(a, G, B.BF16, 1) == ALIASING

    a, G = arr(B.Fp8DequantDesc, dq8(1 * MB, 2 * MB, 3 * MB), dq8(4 * MB, 5 * MB))
    assert B.optimus_validate_dequantize_fp8(a, G, B.BF16) == OK
    assert B.optimus_validate_dequantize_fp8(a, G, 9) == UNSUPPORTED
    # members may share one read-only scale
    a, G = arr(B.Fp8DequantDesc, dq8(1 * MB, 2 * MB, 3 * MB), dq8(4 * MB, 5 * MB, 3 * MB))
    assert B.optimus_validate_dequantize_fp8(a, G, B.F32) == OK
    for bad in [dq8(0, 2 * MB), dq8(1 * MB, 0), dq8(1 * MB, 2 * MB, cols=-3), dq8(1 * MB, 2 * MB, ldy=47)]:
        a, G = arr(B.Fp8DequantDesc, bad)
        assert B.optimus_validate_dequantize_fp8(a, G, B.BF16) == INVALID, bad
    # the output over another member's codes, or over the scale
    a, G = arr(B.Fp8DequantDesc, dq8(1 * MB, 2 * MB), dq8(2 * MB + 512, 5 * MB))
    assert B.optimus_validate_dequantize_fp8(a, G, B.BF16) == ALIASING
    a, G = arr(B.Fp8DequantDesc, dq8(1 * MB, 2 * MB, 2 * MB + 8))
    assert B.optimus_validate_dequantize_fp8(a, G, B.BF16) == ALIASING


def test_backward_validation():
    arr = lambda T, *ds: ((T * len(ds))(*ds), len(ds))
    # Linear: M=64, N=32, K=48
    lg = lambda **kw: B.LinearGradDesc(*[kw.get(k, v) for k, v in [
        ("x", 1 * MB), ("ldx", 48), ("w", 2 * MB), ("ldw", 48), ("dy", 3 * MB), ("lddy", 32), ("dx", 4 * MB),
        ("lddx", 48), ("dw", 5 * MB), ("lddw", 48), ("db", 6 * MB), ("M", 64), ("N", 32), ("K", 48)]])
    a, G = arr(B.LinearGradDesc, lg(), lg(x=7 * MB, w=8 * MB, dy=9 * MB, dx=10 * MB, dw=11 * MB, db=12 * MB))
    assert B.optimus_validate_linear_backward(a, G, B.BF16) == OK
    assert B.optimus_validate_linear_backward(a, -1, B.BF16) == INVALID
    assert B.optimus_validate_linear_backward(a, G, 3) == UNSUPPORTED
    for bad in [lg(dy=None), lg(w=None), lg(x=None), lg(M=0), lg(lddy=31), lg(lddx=40), lg(lddw=47), lg(ldx=47)]:
        a, G = arr(B.LinearGradDesc, bad)
        assert B.optimus_validate_linear_backward(a, G, B.BF16) == INVALID, bad
    a, G = arr(B.LinearGradDesc, lg(dw=None))     # db without dw
    assert B.optimus_validate_linear_backward(a, G, B.BF16) == UNSUPPORTED
    a, G = arr(B.LinearGradDesc, lg(dw=None, db=None, x=None))   # dX only: x not needed
    assert B.optimus_validate_linear_backward(a, G, B.F32) == OK
    a, G = arr(B.LinearGradDesc, lg(dx=None, w=None))            # dW and db only: w not needed
    assert B.optimus_validate_linear_backward(a, G, B.F32) == OK
    a, G = arr(B.LinearGradDesc, lg(dx=3 * MB + 64))              # dX over dY
    assert B.optimus_validate_linear_backward(a, G, B.BF16) == ALIASING
    a, G = arr(B.LinearGradDesc, lg(), lg(x=7 * MB, w=8 * MB, dy=9 * MB, dx=10 * MB, dw=11 * MB, db=6 * MB))
    assert B.optimus_validate_linear_backward(a, G, B.BF16) == ALIASING   # two members' db
    # Linear with a fused activation backward: act_x checks (all before any device call)
    f = B.lib().optimus_grouped_linear_act_backward
    a, G = arr(B.LinearGradDesc, lg())
    ptrs = lambda *p: (ctypes.c_void_p * 1)(*p)
    lds = lambda *v: (ctypes.c_int64 * 1)(*v)
    assert f(a, ptrs(5 * MB + 96), lds(48), G, B.BF16, 1, None) == ALIASING     # over dW
    assert f(a, ptrs(6 * MB), lds(48), G, B.BF16, 1, None) == ALIASING          # over db
    assert f(a, ptrs(None), lds(48), G, B.BF16, 1, None) == INVALID             # NULL act_x
    assert f(a, ptrs(13 * MB), lds(47), G, B.BF16, 1, None) == INVALID          # ld < K
    assert f(a, None, None, G, B.BF16, 3, None) == INVALID                       # no arrays
    assert f(a, ptrs(13 * MB), lds(48), G, B.BF16, 9, None) == UNSUPPORTED      # unknown activation
    # LayerNorm: rows 64, cols 48
    ln = lambda **kw: B.LayerNormGradDesc(*[kw.get(k, v) for k, v in [
        ("x", 1 * MB), ("ldx", 48), ("gamma", 2 * MB), ("dy", 3 * MB), ("lddy", 48), ("dx", 4 * MB), ("lddx", 48),
        ("dgamma", 5 * MB), ("dbeta", 6 * MB), ("rows", 64), ("cols", 48), ("eps", 1e-5)]])
    a, G = arr(B.LayerNormGradDesc, ln(), ln(x=7 * MB, gamma=None, dy=8 * MB, dx=8 * MB, dgamma=None, dbeta=None))
    assert B.optimus_validate_layernorm_backward(a, G, B.BF16) == OK        # in place dx == dy allowed
    for bad in [ln(x=None), ln(dy=None), ln(dx=None), ln(cols=0), ln(lddx=40), ln(eps=-1.0), ln(eps=float("inf"))]:
        a, G = arr(B.LayerNormGradDesc, bad)
        assert B.optimus_validate_layernorm_backward(a, G, B.BF16) == INVALID, bad
    a, G = arr(B.LayerNormGradDesc, ln(dgamma=6 * MB + 8))
    assert B.optimus_validate_layernorm_backward(a, G, B.BF16) == ALIASING
    # activation
    ag = lambda **kw: B.ActGradDesc(*[kw.get(k, v) for k, v in [
        ("x", 1 * MB), ("ldx", 48), ("dy", 2 * MB), ("lddy", 48), ("dx", 2 * MB), ("lddx", 48), ("rows", 64),
        ("cols", 48)]])
    a, G = arr(B.ActGradDesc, ag())
    assert B.optimus_validate_act_backward(a, G, B.BF16, "silu") == OK
    assert B.optimus_validate_act_backward(a, G, B.BF16, 9) == UNSUPPORTED
    a, G = arr(B.ActGradDesc, ag(dx=1 * MB + 2))
    assert B.optimus_validate_act_backward(a, G, B.BF16, "relu") == ALIASING
