"""ctypes binding of liboptimus (include/optimus.h): argument marshalling only.

Every entry point here has the name of the C function it calls. Tensors are
torch tensors on the GPU (device memory and streams come from PyTorch); every
step of the work runs in the library's HIP kernels. If liboptimus.so is not
built this module raises -- there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os
from typing import List, Optional, Sequence

import torch

_PKG = os.path.dirname(os.path.abspath(__file__))
LIBPATH = os.path.join(_PKG, "liboptimus.so")

F32, BF16 = 0, 1
ACTS = {"none": 0, "relu": 1, "sigmoid": 2, "tanh": 3, "silu": 4}
EXEC_MODES = {"grouped": 0, "chain": 1, "horizontal": 2}
STATUS = {0: "OK", -1: "INVALID_ARG", -2: "UNSUPPORTED", -3: "ALIASING", -4: "HIP", -5: "OOM"}

c_i64, c_i32, c_vp = ctypes.c_int64, ctypes.c_int32, ctypes.c_void_p


class LinearDesc(ctypes.Structure):
    _fields_ = [("x", c_vp), ("ldx", c_i64), ("w", c_vp), ("ldw", c_i64), ("bias", c_vp), ("y", c_vp),
                ("ldy", c_i64), ("M", c_i64), ("N", c_i64), ("K", c_i64)]


class LayerNormDesc(ctypes.Structure):
    _fields_ = [("x", c_vp), ("ldx", c_i64), ("y", c_vp), ("ldy", c_i64), ("gamma", c_vp), ("beta", c_vp),
                ("rows", c_i64), ("cols", c_i64), ("eps", ctypes.c_float)]


class PointwiseDesc(ctypes.Structure):
    _fields_ = [("x", c_vp), ("ldx", c_i64), ("y", c_vp), ("ldy", c_i64), ("rows", c_i64), ("cols", c_i64)]


class SplitOpCatDesc(ctypes.Structure):
    _fields_ = [("in_", c_vp), ("ldin", c_i64), ("out", c_vp), ("ldout", c_i64), ("rows", c_i64), ("D", c_i64),
                ("n_slices", c_i32), ("widths", ctypes.POINTER(c_i64)), ("gamma", ctypes.POINTER(c_vp)),
                ("beta", ctypes.POINTER(c_vp)), ("apply_layernorm", c_i32), ("eps", ctypes.c_float),
                ("act", ctypes.c_int)]


class LinearGradDesc(ctypes.Structure):
    _fields_ = [("x", c_vp), ("ldx", c_i64), ("w", c_vp), ("ldw", c_i64), ("dy", c_vp), ("lddy", c_i64),
                ("dx", c_vp), ("lddx", c_i64), ("dw", c_vp), ("lddw", c_i64), ("db", c_vp), ("M", c_i64),
                ("N", c_i64), ("K", c_i64)]


class LayerNormGradDesc(ctypes.Structure):
    _fields_ = [("x", c_vp), ("ldx", c_i64), ("gamma", c_vp), ("dy", c_vp), ("lddy", c_i64), ("dx", c_vp),
                ("lddx", c_i64), ("dgamma", c_vp), ("dbeta", c_vp), ("rows", c_i64), ("cols", c_i64),
                ("eps", ctypes.c_float)]


class ActGradDesc(ctypes.Structure):
    _fields_ = [("x", c_vp), ("ldx", c_i64), ("dy", c_vp), ("lddy", c_i64), ("dx", c_vp), ("lddx", c_i64),
                ("rows", c_i64), ("cols", c_i64)]


class Fp8QuantDesc(ctypes.Structure):
    _fields_ = [("x", c_vp), ("ldx", c_i64), ("q", c_vp), ("ldq", c_i64), ("scale", c_vp), ("rows", c_i64),
                ("cols", c_i64)]


class Fp8DequantDesc(ctypes.Structure):
    _fields_ = [("q", c_vp), ("ldq", c_i64), ("scale", c_vp), ("y", c_vp), ("ldy", c_i64), ("rows", c_i64),
                ("cols", c_i64)]


class PlanOptions(ctypes.Structure):
    """optimus_plan_options: gemm_tile (TILES key or OPTIMUS_TILE_* value; 0 = the
    planner's), wgrad_splits (0 = the planner's), soc_waves_per_row (0 = the planner's)."""
    _fields_ = [("gemm_tile", c_i32), ("wgrad_splits", c_i32), ("soc_waves_per_row", c_i32), ("reserved", c_i32)]


# optimus_gemm_tile values, keyed by the kernel-table index the plan's kernel name reports
TILES = {"auto": 0, "bf16_128x64": 1, "bf16_128x128": 2, "bf16_256x256": 3, "f32_64x64": 4, "bf16_dma_256x256": 5,
         "bf16_dma_128x128": 6, "f32_64x128": 7, "skinny": 8, "f32_32x128": 9, "bf16_stream": 10,
         "f32_16x128": 11}


def plan_options(gemm_tile=0, wgrad_splits=0, soc_waves_per_row=0) -> PlanOptions:
    t = TILES[gemm_tile] if isinstance(gemm_tile, str) else int(gemm_tile)
    return PlanOptions(t, int(wgrad_splits), int(soc_waves_per_row), 0)


def _opts(options):
    if options is None:
        return None
    if isinstance(options, dict):
        options = plan_options(**options)
    return ctypes.byref(options)


class PlanInfo(ctypes.Structure):
    _fields_ = [("kind", c_i32), ("group_size", c_i32), ("launches", c_i32), ("chain_launches", c_i32),
                ("work_items", c_i64), ("grid", c_i32), ("block", c_i32), ("flops", ctypes.c_double),
                ("bytes", ctypes.c_double), ("kernel", ctypes.c_char_p)]


# Every symbol include/optimus.h declares.
EXPORTS = [
    "optimus_grouped_linear", "optimus_grouped_linear_layernorm", "optimus_grouped_layernorm",
    "optimus_grouped_pointwise", "optimus_split_op_cat", "optimus_grouped_quantize_fp8",
    "optimus_grouped_dequantize_fp8", "optimus_grouped_linear_backward", "optimus_grouped_layernorm_backward",
    "optimus_grouped_act_backward", "optimus_plan_linear_backward", "optimus_plan_layernorm_backward",
    "optimus_plan_act_backward", "optimus_validate_linear_backward", "optimus_validate_layernorm_backward",
    "optimus_grouped_layernorm_act_backward", "optimus_plan_layernorm_act_backward",
    "optimus_grouped_linear_act_backward", "optimus_plan_linear_act_backward",
    "optimus_validate_act_backward",
    "optimus_plan_linear", "optimus_plan_linear_layernorm", "optimus_plan_layernorm", "optimus_plan_pointwise",
    "optimus_plan_split_op_cat", "optimus_plan_quantize_fp8", "optimus_plan_dequantize_fp8",
    "optimus_plan_linear_ex", "optimus_plan_linear_layernorm_ex", "optimus_plan_linear_backward_ex",
    "optimus_plan_linear_act_backward_ex", "optimus_plan_split_op_cat_ex", "optimus_grouped_quantize_fp8_noalloc",
    "optimus_plan_execute", "optimus_plan_execute_mode", "optimus_plan_destroy", "optimus_plan_get_info",
    "optimus_validate_linear", "optimus_validate_linear_layernorm", "optimus_validate_layernorm",
    "optimus_validate_pointwise", "optimus_validate_split_op_cat", "optimus_validate_quantize_fp8",
    "optimus_validate_dequantize_fp8", "optimus_last_error", "optimus_version",
]


class OptimusError(RuntimeError):
    def __init__(self, status: int, message: str):
        super().__init__(f"{STATUS.get(status, status)}: {message}")
        self.status = status
        self.name = STATUS.get(status, str(status))


_lib = None


def lib() -> ctypes.CDLL:
    """The loaded liboptimus.so (raises if it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIBPATH):
            raise RuntimeError(f"{LIBPATH} is missing: build it with `python -m paper_2607_02945_amd.build`")
        L = ctypes.CDLL(LIBPATH)
        P = ctypes.POINTER
        st = ctypes.c_int
        sig = {
            "optimus_grouped_linear": (st, [P(LinearDesc), c_i32, ctypes.c_int, ctypes.c_int, c_vp]),
            "optimus_grouped_linear_layernorm": (st, [P(LinearDesc), P(c_vp), P(c_vp), c_i32, ctypes.c_int,
                                                      ctypes.c_float, ctypes.c_int, c_vp]),
            "optimus_grouped_layernorm": (st, [P(LayerNormDesc), c_i32, ctypes.c_int, ctypes.c_int, c_vp]),
            "optimus_grouped_pointwise": (st, [P(PointwiseDesc), c_i32, ctypes.c_int, ctypes.c_int, c_vp]),
            "optimus_split_op_cat": (st, [P(SplitOpCatDesc), ctypes.c_int, c_vp]),
            "optimus_plan_linear": (st, [P(LinearDesc), c_i32, ctypes.c_int, ctypes.c_int, P(c_vp)]),
            "optimus_plan_linear_layernorm": (st, [P(LinearDesc), P(c_vp), P(c_vp), c_i32, ctypes.c_int,
                                                   ctypes.c_float, ctypes.c_int, P(c_vp)]),
            "optimus_plan_layernorm": (st, [P(LayerNormDesc), c_i32, ctypes.c_int, ctypes.c_int, P(c_vp)]),
            "optimus_plan_pointwise": (st, [P(PointwiseDesc), c_i32, ctypes.c_int, ctypes.c_int, P(c_vp)]),
            "optimus_plan_split_op_cat": (st, [P(SplitOpCatDesc), ctypes.c_int, P(c_vp)]),
            "optimus_grouped_linear_backward": (st, [P(LinearGradDesc), c_i32, ctypes.c_int, c_vp]),
            "optimus_grouped_layernorm_backward": (st, [P(LayerNormGradDesc), c_i32, ctypes.c_int, c_vp]),
            "optimus_grouped_act_backward": (st, [P(ActGradDesc), c_i32, ctypes.c_int, ctypes.c_int, c_vp]),
            "optimus_grouped_layernorm_act_backward": (st, [P(LayerNormGradDesc), P(c_vp), c_i32, ctypes.c_int,
                                                            ctypes.c_int, c_vp]),
            "optimus_grouped_linear_act_backward": (st, [P(LinearGradDesc), P(c_vp), P(ctypes.c_int64), c_i32,
                                                         ctypes.c_int, ctypes.c_int, c_vp]),
            "optimus_plan_linear_act_backward": (st, [P(LinearGradDesc), P(c_vp), P(ctypes.c_int64), c_i32,
                                                      ctypes.c_int, ctypes.c_int, P(c_vp)]),
            "optimus_plan_layernorm_act_backward": (st, [P(LayerNormGradDesc), P(c_vp), c_i32, ctypes.c_int,
                                                         ctypes.c_int, P(c_vp)]),
            "optimus_plan_linear_backward": (st, [P(LinearGradDesc), c_i32, ctypes.c_int, P(c_vp)]),
            "optimus_plan_layernorm_backward": (st, [P(LayerNormGradDesc), c_i32, ctypes.c_int, P(c_vp)]),
            "optimus_plan_act_backward": (st, [P(ActGradDesc), c_i32, ctypes.c_int, ctypes.c_int, P(c_vp)]),
            "optimus_validate_linear_backward": (st, [P(LinearGradDesc), c_i32, ctypes.c_int]),
            "optimus_validate_layernorm_backward": (st, [P(LayerNormGradDesc), c_i32, ctypes.c_int]),
            "optimus_validate_act_backward": (st, [P(ActGradDesc), c_i32, ctypes.c_int, ctypes.c_int]),
            "optimus_grouped_quantize_fp8": (st, [P(Fp8QuantDesc), c_i32, ctypes.c_int, c_i32, c_vp]),
            "optimus_grouped_dequantize_fp8": (st, [P(Fp8DequantDesc), c_i32, ctypes.c_int, c_vp]),
            "optimus_grouped_quantize_fp8_noalloc": (st, [P(Fp8QuantDesc), c_i32, ctypes.c_int, c_i32, c_vp]),
            "optimus_plan_quantize_fp8": (st, [P(Fp8QuantDesc), c_i32, ctypes.c_int, c_i32, P(c_vp)]),
            "optimus_plan_dequantize_fp8": (st, [P(Fp8DequantDesc), c_i32, ctypes.c_int, P(c_vp)]),
            "optimus_validate_quantize_fp8": (st, [P(Fp8QuantDesc), c_i32, ctypes.c_int, c_i32]),
            "optimus_validate_dequantize_fp8": (st, [P(Fp8DequantDesc), c_i32, ctypes.c_int]),
            "optimus_plan_linear_ex": (st, [P(LinearDesc), c_i32, ctypes.c_int, ctypes.c_int, P(PlanOptions),
                                            P(c_vp)]),
            "optimus_plan_linear_layernorm_ex": (st, [P(LinearDesc), P(c_vp), P(c_vp), c_i32, ctypes.c_int,
                                                      ctypes.c_float, ctypes.c_int, P(PlanOptions), P(c_vp)]),
            "optimus_plan_linear_backward_ex": (st, [P(LinearGradDesc), c_i32, ctypes.c_int, P(PlanOptions),
                                                     P(c_vp)]),
            "optimus_plan_linear_act_backward_ex": (st, [P(LinearGradDesc), P(c_vp), P(ctypes.c_int64), c_i32,
                                                         ctypes.c_int, ctypes.c_int, P(PlanOptions), P(c_vp)]),
            "optimus_plan_split_op_cat_ex": (st, [P(SplitOpCatDesc), ctypes.c_int, P(PlanOptions), P(c_vp)]),
            "optimus_plan_execute": (st, [c_vp, c_vp]),
            "optimus_plan_execute_mode": (st, [c_vp, ctypes.c_int, c_vp]),
            "optimus_plan_destroy": (None, [c_vp]),
            "optimus_plan_get_info": (st, [c_vp, P(PlanInfo)]),
            "optimus_validate_linear": (st, [P(LinearDesc), c_i32, ctypes.c_int, ctypes.c_int]),
            "optimus_validate_linear_layernorm": (st, [P(LinearDesc), P(c_vp), P(c_vp), c_i32, ctypes.c_int,
                                                       ctypes.c_float, ctypes.c_int]),
            "optimus_validate_layernorm": (st, [P(LayerNormDesc), c_i32, ctypes.c_int, ctypes.c_int]),
            "optimus_validate_pointwise": (st, [P(PointwiseDesc), c_i32, ctypes.c_int, ctypes.c_int]),
            "optimus_validate_split_op_cat": (st, [P(SplitOpCatDesc), ctypes.c_int]),
            "optimus_last_error": (ctypes.c_char_p, []),
            "optimus_version": (ctypes.c_char_p, []),
        }
        for name, (res, args) in sig.items():
            f = getattr(L, name)
            f.restype = res
            f.argtypes = args
        _lib = L
    return _lib


def check(status: int) -> None:
    if status != 0:
        raise OptimusError(status, lib().optimus_last_error().decode())


# ------------------------------------------------------------------ marshalling
def dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return F32
    if t.dtype == torch.bfloat16:
        return BF16
    raise TypeError(f"unsupported dtype {t.dtype}")


def _act(a) -> int:
    return ACTS[a] if isinstance(a, str) else int(a)


def _mat(t: torch.Tensor, name: str):
    if t.dim() != 2 or (t.shape[1] > 1 and t.stride(1) != 1):
        raise ValueError(f"{name}: need a 2-D tensor with unit inner stride, got shape {tuple(t.shape)} "
                         f"strides {t.stride()}")
    return t.data_ptr(), max(t.stride(0), t.shape[1])


def _ptr(t: Optional[torch.Tensor]):
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        return torch.cuda.current_stream().cuda_stream
    return stream.cuda_stream if hasattr(stream, "cuda_stream") else int(stream)


def linear_descs(xs, ws, biases, ys) -> ctypes.Array:
    G = len(xs)
    arr = (LinearDesc * max(G, 1))()
    for g in range(G):
        x, ldx = _mat(xs[g], "x")
        w, ldw = _mat(ws[g], "w")
        y, ldy = _mat(ys[g], "y")
        arr[g] = LinearDesc(x, ldx, w, ldw, _ptr(biases[g] if biases is not None else None), y, ldy,
                            xs[g].shape[0], ws[g].shape[0], xs[g].shape[1])
    return arr


def layernorm_descs(xs, ys, gammas, betas, eps) -> ctypes.Array:
    G = len(xs)
    arr = (LayerNormDesc * max(G, 1))()
    for g in range(G):
        x, ldx = _mat(xs[g], "x")
        y, ldy = _mat(ys[g], "y")
        arr[g] = LayerNormDesc(x, ldx, y, ldy, _ptr(gammas[g] if gammas is not None else None),
                               _ptr(betas[g] if betas is not None else None), xs[g].shape[0], xs[g].shape[1],
                               float(eps))
    return arr


def pointwise_descs(xs, ys) -> ctypes.Array:
    G = len(xs)
    arr = (PointwiseDesc * max(G, 1))()
    for g in range(G):
        x, ldx = _mat(xs[g], "x")
        y, ldy = _mat(ys[g], "y")
        arr[g] = PointwiseDesc(x, ldx, y, ldy, xs[g].shape[0], xs[g].shape[1])
    return arr


def _opt_mat(t, name):
    return (None, 0) if t is None else _mat(t, name)


def linear_grad_descs(xs, ws, dys, dxs=None, dws=None, dbs=None) -> ctypes.Array:
    """Members of a Linear backward: forward X [M,K], W [N,K], dY [M,N]; the
    wanted gradients dX, dW, db (lists with None entries, or None)."""
    G = len(dys)
    arr = (LinearGradDesc * max(G, 1))()
    pick = lambda v, g: None if v is None else v[g]
    for g in range(G):
        dy, lddy = _mat(dys[g], "dy")
        x, ldx = _opt_mat(pick(xs, g), "x")
        w, ldw = _opt_mat(pick(ws, g), "w")
        dx, lddx = _opt_mat(pick(dxs, g), "dx")
        dw, lddw = _opt_mat(pick(dws, g), "dw")
        M, N = dys[g].shape
        K = (pick(xs, g) if pick(xs, g) is not None else pick(ws, g)).shape[1]
        arr[g] = LinearGradDesc(x, ldx, w, ldw, dy, lddy, dx, lddx, dw, lddw, _ptr(pick(dbs, g)), M, N, K)
    return arr


def layernorm_grad_descs(xs, dys, dxs, gammas=None, dgammas=None, dbetas=None, eps=1e-5) -> ctypes.Array:
    G = len(xs)
    arr = (LayerNormGradDesc * max(G, 1))()
    pick = lambda v, g: None if v is None else v[g]
    for g in range(G):
        x, ldx = _mat(xs[g], "x")
        dy, lddy = _mat(dys[g], "dy")
        dx, lddx = _mat(dxs[g], "dx")
        arr[g] = LayerNormGradDesc(x, ldx, _ptr(pick(gammas, g)), dy, lddy, dx, lddx, _ptr(pick(dgammas, g)),
                                   _ptr(pick(dbetas, g)), xs[g].shape[0], xs[g].shape[1], float(eps))
    return arr


def act_grad_descs(xs, dys, dxs) -> ctypes.Array:
    G = len(xs)
    arr = (ActGradDesc * max(G, 1))()
    for g in range(G):
        x, ldx = _mat(xs[g], "x")
        dy, lddy = _mat(dys[g], "dy")
        dx, lddx = _mat(dxs[g], "dx")
        arr[g] = ActGradDesc(x, ldx, dy, lddy, dx, lddx, xs[g].shape[0], xs[g].shape[1])
    return arr


def fp8_quant_descs(xs, qs, scales) -> ctypes.Array:
    """xs: values (bf16 / fp32), qs: uint8 codes of the same shapes, scales:
    one-element fp32 device tensors, or None (unscaled)."""
    G = len(xs)
    arr = (Fp8QuantDesc * max(G, 1))()
    for g in range(G):
        x, ldx = _mat(xs[g], "x")
        q, ldq = _mat(qs[g], "q")
        arr[g] = Fp8QuantDesc(x, ldx, q, ldq, _ptr(scales[g] if scales is not None else None), xs[g].shape[0],
                              xs[g].shape[1])
    return arr


def fp8_dequant_descs(qs, scales, ys) -> ctypes.Array:
    G = len(qs)
    arr = (Fp8DequantDesc * max(G, 1))()
    for g in range(G):
        q, ldq = _mat(qs[g], "q")
        y, ldy = _mat(ys[g], "y")
        arr[g] = Fp8DequantDesc(q, ldq, _ptr(scales[g] if scales is not None else None), y, ldy, qs[g].shape[0],
                                qs[g].shape[1])
    return arr


class _SocArgs:
    """Keeps the host arrays a split-op-cat descriptor points to alive."""

    def __init__(self, inp, out, widths, gammas, betas, apply_layernorm, eps, act):
        i, ldin = _mat(inp, "in")
        o, ldout = _mat(out, "out")
        n = len(widths)
        self.widths = (c_i64 * n)(*[int(w) for w in widths])
        self.gamma = None if gammas is None else (c_vp * n)(*[_ptr(g) for g in gammas])
        self.beta = None if betas is None else (c_vp * n)(*[_ptr(b) for b in betas])
        self.desc = SplitOpCatDesc(i, ldin, o, ldout, inp.shape[0], inp.shape[1], n, self.widths,
                                   self.gamma, self.beta, int(bool(apply_layernorm)), float(eps), _act(act))


# ------------------------------------------------------------------ one-shot entry points
def optimus_grouped_linear(xs: Sequence[torch.Tensor], ws, biases, ys, act="none", stream=None) -> None:
    """y_g = act(x_g w_g^T + b_g) for every member, one launch."""
    d = linear_descs(xs, ws, biases, ys)
    check(lib().optimus_grouped_linear(d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act), _stream(stream)))


def _ptrs(ts, G):
    """Host array of G device pointers (None entries -> NULL), or None."""
    return None if ts is None else (c_vp * max(G, 1))(*[_ptr(t) for t in ts])


def optimus_grouped_linear_layernorm(xs, ws, biases, ys, gammas=None, betas=None, eps=1e-5, act="none",
                                     stream=None) -> None:
    """y_g = act(LayerNorm_row(x_g w_g^T + b_g) * gamma_g + beta_g) for every member, one launch."""
    d = linear_descs(xs, ws, biases, ys)
    G = len(xs)
    check(lib().optimus_grouped_linear_layernorm(d, _ptrs(gammas, G), _ptrs(betas, G), G,
                                                 dtype_code(xs[0]) if xs else BF16, float(eps), _act(act),
                                                 _stream(stream)))


def optimus_grouped_layernorm(xs, ys, gammas=None, betas=None, eps=1e-5, act="none", stream=None) -> None:
    d = layernorm_descs(xs, ys, gammas, betas, eps)
    check(lib().optimus_grouped_layernorm(d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act), _stream(stream)))


def optimus_grouped_pointwise(xs, ys, act, stream=None) -> None:
    d = pointwise_descs(xs, ys)
    check(lib().optimus_grouped_pointwise(d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act), _stream(stream)))


def optimus_split_op_cat(inp, out, widths, gammas=None, betas=None, apply_layernorm=True, eps=1e-5, act="none",
                         stream=None) -> None:
    a = _SocArgs(inp, out, widths, gammas, betas, apply_layernorm, eps, act)
    check(lib().optimus_split_op_cat(ctypes.byref(a.desc), dtype_code(inp), _stream(stream)))


def optimus_grouped_quantize_fp8(xs, qs, scales=None, use_scaling=True, stream=None) -> None:
    """q_g = E4M3 codes of x_g (scaled: x_g * 448 / amax_g, with scale_g = amax_g / 448 written), one launch."""
    d = fp8_quant_descs(xs, qs, scales)
    check(lib().optimus_grouped_quantize_fp8(d, len(xs), dtype_code(xs[0]) if xs else BF16, int(use_scaling),
                                             _stream(stream)))


def optimus_grouped_quantize_fp8_noalloc(xs, qs, scales=None, use_scaling=True, stream=None) -> None:
    """optimus_grouped_quantize_fp8 with no device allocation: the table and amax
    partials live in the library's static per-GPU scratch array."""
    d = fp8_quant_descs(xs, qs, scales)
    check(lib().optimus_grouped_quantize_fp8_noalloc(d, len(xs), dtype_code(xs[0]) if xs else BF16,
                                                     int(use_scaling), _stream(stream)))


def optimus_grouped_dequantize_fp8(qs, scales, ys, stream=None) -> None:
    """y_g = value(q_g) * scale_g in the dtype of y_g, one launch; scales None (or None entries) mean 1."""
    d = fp8_dequant_descs(qs, scales, ys)
    check(lib().optimus_grouped_dequantize_fp8(d, len(qs), dtype_code(ys[0]) if ys else BF16, _stream(stream)))


def optimus_grouped_linear_backward(xs, ws, dys, dxs=None, dws=None, dbs=None, stream=None) -> None:
    """dX = dY W, dW = dY^T X, db = column sums of dY, for every member; two launches for the group."""
    d = linear_grad_descs(xs, ws, dys, dxs, dws, dbs)
    check(lib().optimus_grouped_linear_backward(d, len(dys), dtype_code(dys[0]) if dys else BF16, _stream(stream)))


def optimus_grouped_layernorm_backward(xs, dys, dxs, gammas=None, dgammas=None, dbetas=None, eps=1e-5,
                                       stream=None) -> None:
    d = layernorm_grad_descs(xs, dys, dxs, gammas, dgammas, dbetas, eps)
    check(lib().optimus_grouped_layernorm_backward(d, len(xs), dtype_code(xs[0]) if xs else BF16, _stream(stream)))


def _act_inputs(act_x, G):
    """Pointers and row strides of the activation inputs (entries may be None)."""
    ptrs = (c_vp * max(G, 1))(*[_ptr(a) for a in act_x])
    lds = (ctypes.c_int64 * max(G, 1))(*[(a.stride(0) if a is not None else 1) for a in act_x])
    return ptrs, lds


def optimus_grouped_linear_act_backward(xs, ws, dys, dxs, dws, dbs, act_x, act, stream=None) -> None:
    d = linear_grad_descs(xs, ws, dys, dxs, dws, dbs)
    ptrs, lds = _act_inputs(act_x, len(xs))
    check(lib().optimus_grouped_linear_act_backward(d, ptrs, lds, len(xs), dtype_code(xs[0]) if xs else BF16,
                                                    _act(act), _stream(stream)))


def optimus_plan_linear_act_backward(xs, ws, dys, dxs, dws, dbs, act_x, act) -> "Plan":
    d = linear_grad_descs(xs, ws, dys, dxs, dws, dbs)
    ptrs, lds = _act_inputs(act_x, len(xs))
    return _plan(lib().optimus_plan_linear_act_backward, d, ptrs, lds, len(xs), dtype_code(xs[0]) if xs else BF16,
                 _act(act), keep=(list(xs), list(ws), list(dys), dxs, dws, dbs, list(act_x)))


def optimus_grouped_layernorm_act_backward(xs, dys, dxs, gammas=None, betas=None, dgammas=None, dbetas=None,
                                           eps=1e-5, act="none", stream=None) -> None:
    d = layernorm_grad_descs(xs, dys, dxs, gammas, dgammas, dbetas, eps)
    G = len(xs)
    check(lib().optimus_grouped_layernorm_act_backward(d, _ptrs(betas, G), G, dtype_code(xs[0]) if xs else BF16,
                                                       _act(act), _stream(stream)))


def optimus_grouped_act_backward(xs, dys, dxs, act, stream=None) -> None:
    d = act_grad_descs(xs, dys, dxs)
    check(lib().optimus_grouped_act_backward(d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act),
                                             _stream(stream)))


# ------------------------------------------------------------------ plans
class Plan:
    """A validated group with its device table resident; execute() is one launch."""

    def __init__(self, handle: int, keep):
        self._h = ctypes.c_void_p(handle)
        self._keep = keep  # tensors the plan points to stay alive with it

    def execute(self, mode: str = "grouped", stream=None) -> None:
        check(lib().optimus_plan_execute_mode(self._h, EXEC_MODES[mode], _stream(stream)))

    def info(self) -> dict:
        pi = PlanInfo()
        check(lib().optimus_plan_get_info(self._h, ctypes.byref(pi)))
        return {"kind": pi.kind, "group_size": pi.group_size, "launches": pi.launches,
                "chain_launches": pi.chain_launches, "work_items": pi.work_items, "grid": pi.grid,
                "block": pi.block, "flops": pi.flops, "bytes": pi.bytes,
                "kernel": pi.kernel.decode() if pi.kernel else ""}

    def close(self) -> None:
        if self._h:
            lib().optimus_plan_destroy(self._h)
            self._h = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def _plan(fn, *args, keep=None) -> Plan:
    h = ctypes.c_void_p()
    check(fn(*args, ctypes.byref(h)))
    return Plan(h.value, keep)


def optimus_plan_linear(xs, ws, biases, ys, act="none") -> Plan:
    d = linear_descs(xs, ws, biases, ys)
    return _plan(lib().optimus_plan_linear, d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act),
                 keep=(list(xs), list(ws), biases, list(ys)))


def optimus_plan_linear_ex(xs, ws, biases, ys, act="none", options=None) -> Plan:
    """optimus_plan_linear with plan options (a PlanOptions, a dict of its fields, or None)."""
    d = linear_descs(xs, ws, biases, ys)
    return _plan(lib().optimus_plan_linear_ex, d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act),
                 _opts(options), keep=(list(xs), list(ws), biases, list(ys)))


def optimus_plan_linear_layernorm_ex(xs, ws, biases, ys, gammas=None, betas=None, eps=1e-5, act="none",
                                     options=None) -> Plan:
    d = linear_descs(xs, ws, biases, ys)
    G = len(xs)
    return _plan(lib().optimus_plan_linear_layernorm_ex, d, _ptrs(gammas, G), _ptrs(betas, G), G,
                 dtype_code(xs[0]) if xs else BF16, float(eps), _act(act), _opts(options),
                 keep=(list(xs), list(ws), biases, list(ys), gammas, betas))


def optimus_plan_linear_backward_ex(xs, ws, dys, dxs=None, dws=None, dbs=None, options=None) -> Plan:
    d = linear_grad_descs(xs, ws, dys, dxs, dws, dbs)
    return _plan(lib().optimus_plan_linear_backward_ex, d, len(dys), dtype_code(dys[0]) if dys else BF16,
                 _opts(options), keep=(xs, ws, list(dys), dxs, dws, dbs))


def optimus_plan_linear_act_backward_ex(xs, ws, dys, dxs, dws, dbs, act_x, act, options=None) -> Plan:
    d = linear_grad_descs(xs, ws, dys, dxs, dws, dbs)
    ptrs, lds = _act_inputs(act_x, len(xs))
    return _plan(lib().optimus_plan_linear_act_backward_ex, d, ptrs, lds, len(xs),
                 dtype_code(xs[0]) if xs else BF16, _act(act), _opts(options),
                 keep=(list(xs), list(ws), list(dys), dxs, dws, dbs, list(act_x)))


def optimus_plan_split_op_cat_ex(inp, out, widths, gammas=None, betas=None, apply_layernorm=True, eps=1e-5,
                                 act="none", options=None) -> Plan:
    a = _SocArgs(inp, out, widths, gammas, betas, apply_layernorm, eps, act)
    return _plan(lib().optimus_plan_split_op_cat_ex, ctypes.byref(a.desc), dtype_code(inp), _opts(options),
                 keep=(inp, out, gammas, betas))


def optimus_plan_linear_layernorm(xs, ws, biases, ys, gammas=None, betas=None, eps=1e-5, act="none") -> Plan:
    d = linear_descs(xs, ws, biases, ys)
    G = len(xs)
    return _plan(lib().optimus_plan_linear_layernorm, d, _ptrs(gammas, G), _ptrs(betas, G), G,
                 dtype_code(xs[0]) if xs else BF16, float(eps), _act(act),
                 keep=(list(xs), list(ws), biases, list(ys), gammas, betas))


def optimus_plan_layernorm(xs, ys, gammas=None, betas=None, eps=1e-5, act="none") -> Plan:
    d = layernorm_descs(xs, ys, gammas, betas, eps)
    return _plan(lib().optimus_plan_layernorm, d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act),
                 keep=(list(xs), list(ys), gammas, betas))


def optimus_plan_pointwise(xs, ys, act) -> Plan:
    d = pointwise_descs(xs, ys)
    return _plan(lib().optimus_plan_pointwise, d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act),
                 keep=(list(xs), list(ys)))


def optimus_plan_split_op_cat(inp, out, widths, gammas=None, betas=None, apply_layernorm=True, eps=1e-5,
                              act="none") -> Plan:
    a = _SocArgs(inp, out, widths, gammas, betas, apply_layernorm, eps, act)
    return _plan(lib().optimus_plan_split_op_cat, ctypes.byref(a.desc), dtype_code(inp),
                 keep=(inp, out, gammas, betas))


def optimus_plan_linear_backward(xs, ws, dys, dxs=None, dws=None, dbs=None) -> Plan:
    d = linear_grad_descs(xs, ws, dys, dxs, dws, dbs)
    return _plan(lib().optimus_plan_linear_backward, d, len(dys), dtype_code(dys[0]) if dys else BF16,
                 keep=(xs, ws, list(dys), dxs, dws, dbs))


def optimus_plan_layernorm_act_backward(xs, dys, dxs, gammas=None, betas=None, dgammas=None, dbetas=None, eps=1e-5,
                                        act="none") -> Plan:
    d = layernorm_grad_descs(xs, dys, dxs, gammas, dgammas, dbetas, eps)
    G = len(xs)
    return _plan(lib().optimus_plan_layernorm_act_backward, d, _ptrs(betas, G), G,
                 dtype_code(xs[0]) if xs else BF16, _act(act),
                 keep=(list(xs), list(dys), list(dxs), gammas, betas, dgammas, dbetas))


def optimus_plan_layernorm_backward(xs, dys, dxs, gammas=None, dgammas=None, dbetas=None, eps=1e-5) -> Plan:
    d = layernorm_grad_descs(xs, dys, dxs, gammas, dgammas, dbetas, eps)
    return _plan(lib().optimus_plan_layernorm_backward, d, len(xs), dtype_code(xs[0]) if xs else BF16,
                 keep=(list(xs), list(dys), list(dxs), gammas, dgammas, dbetas))


def optimus_plan_act_backward(xs, dys, dxs, act) -> Plan:
    d = act_grad_descs(xs, dys, dxs)
    return _plan(lib().optimus_plan_act_backward, d, len(xs), dtype_code(xs[0]) if xs else BF16, _act(act),
                 keep=(list(xs), list(dys), list(dxs)))


def optimus_plan_quantize_fp8(xs, qs, scales=None, use_scaling=True) -> Plan:
    d = fp8_quant_descs(xs, qs, scales)
    return _plan(lib().optimus_plan_quantize_fp8, d, len(xs), dtype_code(xs[0]) if xs else BF16, int(use_scaling),
                 keep=(list(xs), list(qs), scales))


def optimus_plan_dequantize_fp8(qs, scales, ys) -> Plan:
    d = fp8_dequant_descs(qs, scales, ys)
    return _plan(lib().optimus_plan_dequantize_fp8, d, len(qs), dtype_code(ys[0]) if ys else BF16,
                 keep=(list(qs), scales, list(ys)))


# ------------------------------------------------------------------ host-only validation
def optimus_validate_linear(descs: ctypes.Array, G: int, dtype: int, act="none") -> int:
    return lib().optimus_validate_linear(descs, G, dtype, _act(act))


def optimus_validate_linear_layernorm(descs: ctypes.Array, gammas, betas, G: int, dtype: int, eps=1e-5,
                                      act="none") -> int:
    """gammas / betas: host arrays of device pointers (ctypes c_void_p arrays) or None."""
    return lib().optimus_validate_linear_layernorm(descs, gammas, betas, G, dtype, float(eps), _act(act))


def optimus_validate_layernorm(descs: ctypes.Array, G: int, dtype: int, act="none") -> int:
    return lib().optimus_validate_layernorm(descs, G, dtype, _act(act))


def optimus_validate_pointwise(descs: ctypes.Array, G: int, dtype: int, act="none") -> int:
    return lib().optimus_validate_pointwise(descs, G, dtype, _act(act))


def optimus_validate_split_op_cat(desc: SplitOpCatDesc, dtype: int) -> int:
    return lib().optimus_validate_split_op_cat(ctypes.byref(desc), dtype)


def optimus_validate_linear_backward(descs: ctypes.Array, G: int, dtype: int) -> int:
    return lib().optimus_validate_linear_backward(descs, G, dtype)


def optimus_validate_layernorm_backward(descs: ctypes.Array, G: int, dtype: int) -> int:
    return lib().optimus_validate_layernorm_backward(descs, G, dtype)


def optimus_validate_act_backward(descs: ctypes.Array, G: int, dtype: int, act="none") -> int:
    return lib().optimus_validate_act_backward(descs, G, dtype, _act(act))


def optimus_validate_quantize_fp8(descs: ctypes.Array, G: int, dtype: int, use_scaling=1) -> int:
    return lib().optimus_validate_quantize_fp8(descs, G, dtype, int(use_scaling))


def optimus_validate_dequantize_fp8(descs: ctypes.Array, G: int, dtype: int) -> int:
    return lib().optimus_validate_dequantize_fp8(descs, G, dtype)


def optimus_last_error() -> str:
    return lib().optimus_last_error().decode()


def optimus_version() -> str:
    return lib().optimus_version().decode()
