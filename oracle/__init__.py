"""Optimus grouped-operator ORACLE -- test infrastructure only.

Python face of ``optimus_oracle.c``: the plain fp64 CPU definition of every
operator the GPU library groups. Only the test suite, ``__graft_entry__.smoke``
and the CPU-baseline leg of ``bench.py`` may import this package; the product
path (``paper_2607_02945_amd``) never does, and this package never imports it.

A group is checked one member at a time (paper Sec. 3.2, horizontal group
fusion: grouping changes launches, not results). Inputs are fp64 numpy arrays
holding the exact values the GPU reads (storage values widened exactly).

Parity pins: ``tests/test_oracle_pins.py`` checks every function here against
library routines (numpy BLAS, torch fp64), closed forms, invariants, brute
force on tiny integer inputs and the paper's appendix split-concat example;
``tests/test_oracle_mutants.py`` plants mistakes in copies of the C source and
checks that the pins catch them.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
import time
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
SOURCE = os.path.join(_HERE, "optimus_oracle.c")
LIBPATH = os.path.join(_HERE, "liboptimus_oracle.so")

ACT_NONE, ACT_RELU, ACT_SIGMOID, ACT_TANH, ACT_SILU = 0, 1, 2, 3, 4
ACTS = {"none": ACT_NONE, "relu": ACT_RELU, "sigmoid": ACT_SIGMOID, "tanh": ACT_TANH, "silu": ACT_SILU}

_dp = ctypes.POINTER(ctypes.c_double)
_i64p = ctypes.POINTER(ctypes.c_int64)


def compile_library(source: str = SOURCE, out: str = LIBPATH, extra_flags: Sequence[str] = ()) -> str:
    """Compile the C oracle with gcc (fp64, OpenMP over rows, no fast-math)."""
    cmd = ["gcc", "-O2", "-std=c11", "-fopenmp", "-fPIC", "-shared", "-fno-fast-math",
           *extra_flags, source, "-o", out + ".tmp", "-lm"]
    subprocess.run(cmd, check=True)
    os.replace(out + ".tmp", out)
    return out


def _act(act) -> int:
    return ACTS[act] if isinstance(act, str) else int(act)


def _c64(a: np.ndarray) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float64)


def _ptr(a: Optional[np.ndarray]):
    return None if a is None else a.ctypes.data_as(_dp)


class Oracle:
    """fp64 CPU oracle loaded from a compiled ``optimus_oracle.c``."""

    def __init__(self, libpath: str = LIBPATH):
        if libpath == LIBPATH and (not os.path.exists(libpath) or
                                   os.path.getmtime(libpath) < os.path.getmtime(SOURCE)):
            compile_library(out=libpath)
        self.lib = ctypes.CDLL(libpath)
        L = self.lib
        L.oracle_act_scalar.restype = ctypes.c_double
        L.oracle_act_scalar.argtypes = [ctypes.c_double, ctypes.c_int]
        L.oracle_linear.restype = None
        L.oracle_linear.argtypes = [_dp, ctypes.c_int64, _dp, ctypes.c_int64, _dp, _dp, ctypes.c_int64,
                                    ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int]
        L.oracle_linear_rows.restype = None
        L.oracle_linear_rows.argtypes = [_dp, ctypes.c_int64, _dp, ctypes.c_int64, _dp, _dp, ctypes.c_int64,
                                         _i64p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64, ctypes.c_int]
        L.oracle_layernorm.restype = None
        L.oracle_layernorm.argtypes = [_dp, ctypes.c_int64, _dp, ctypes.c_int64, ctypes.c_int64,
                                       ctypes.c_int64, _dp, _dp, ctypes.c_double, ctypes.c_int]
        L.oracle_pointwise.restype = None
        L.oracle_pointwise.argtypes = [_dp, ctypes.c_int64, _dp, ctypes.c_int64, ctypes.c_int64,
                                       ctypes.c_int64, ctypes.c_int]
        L.oracle_split_op_cat.restype = ctypes.c_int
        L.oracle_split_op_cat.argtypes = [_dp, ctypes.c_int64, _dp, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.c_int32, _i64p,
                                          ctypes.POINTER(_dp), ctypes.POINTER(_dp),
                                          ctypes.c_int32, ctypes.c_double, ctypes.c_int]
        L.oracle_fp8e4m3_decode.restype = ctypes.c_double
        L.oracle_fp8e4m3_decode.argtypes = [ctypes.c_int]
        L.oracle_fp8e4m3_encode.restype = ctypes.c_int
        L.oracle_fp8e4m3_encode.argtypes = [ctypes.c_double, ctypes.c_int]
        _u8p = ctypes.POINTER(ctypes.c_uint8)
        L.oracle_quantize_fp8.restype = None
        L.oracle_quantize_fp8.argtypes = [_dp, ctypes.c_int64, _u8p, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                          ctypes.c_int, ctypes.POINTER(ctypes.c_float)]
        L.oracle_dequantize_fp8.restype = None
        L.oracle_dequantize_fp8.argtypes = [_u8p, ctypes.c_int64, _dp, ctypes.c_int64, ctypes.c_int64, ctypes.c_int64,
                                            ctypes.c_float]
        L.oracle_linear_backward.restype = None
        L.oracle_linear_backward.argtypes = [_dp, ctypes.c_int64, _dp, ctypes.c_int64, _dp, ctypes.c_int64,
                                             _dp, ctypes.c_int64, _dp, ctypes.c_int64, _dp,
                                             ctypes.c_int64, ctypes.c_int64, ctypes.c_int64]
        L.oracle_act_grad_scalar.restype = ctypes.c_double
        L.oracle_act_grad_scalar.argtypes = [ctypes.c_double, ctypes.c_int]
        L.oracle_act_backward.restype = None
        L.oracle_act_backward.argtypes = [_dp, ctypes.c_int64, _dp, ctypes.c_int64, _dp, ctypes.c_int64,
                                          ctypes.c_int64, ctypes.c_int64, ctypes.c_int]
        L.oracle_layernorm_backward.restype = None
        L.oracle_layernorm_backward.argtypes = [_dp, ctypes.c_int64, _dp, _dp, ctypes.c_int64, _dp, ctypes.c_int64,
                                                _dp, _dp, ctypes.c_int64, ctypes.c_int64, ctypes.c_double]
        L.oracle_num_threads.restype = ctypes.c_int
        L.oracle_num_threads.argtypes = []
        L.oracle_set_num_threads.restype = None
        L.oracle_set_num_threads.argtypes = [ctypes.c_int]

    # ------------------------------------------------------------ one operator
    def act_scalar(self, x: float, act) -> float:
        return self.lib.oracle_act_scalar(float(x), _act(act))

    def linear(self, x, w, bias=None, act="none") -> np.ndarray:
        """Y = X W^T + bias, then act. x [M,K], w [N,K], bias [N] or None."""
        x, w = _c64(x), _c64(w)
        M, K = x.shape
        N, K2 = w.shape
        assert K == K2
        b = None if bias is None else _c64(bias)
        y = np.empty((M, N), dtype=np.float64)
        self.lib.oracle_linear(_ptr(x), K, _ptr(w), K, _ptr(b), _ptr(y), N, M, N, K, _act(act))
        return y

    def linear_rows(self, x, w, bias, rows, act="none") -> np.ndarray:
        """Rows ``rows`` of the same Linear; returns [len(rows), N]."""
        x, w = _c64(x), _c64(w)
        M, K = x.shape
        N = w.shape[0]
        rows = np.ascontiguousarray(rows, dtype=np.int64)
        assert rows.size == 0 or (rows.min() >= 0 and rows.max() < M)
        b = None if bias is None else _c64(bias)
        y = np.empty((rows.size, N), dtype=np.float64)
        self.lib.oracle_linear_rows(_ptr(x), K, _ptr(w), K, _ptr(b), _ptr(y), N,
                                    rows.ctypes.data_as(_i64p), rows.size, N, K, _act(act))
        return y

    def layernorm(self, x, gamma=None, beta=None, eps=1e-5, act="none") -> np.ndarray:
        """Row-wise LayerNorm over the last dim of x [rows, cols], then act."""
        x = _c64(x)
        rows, cols = x.shape
        g = None if gamma is None else _c64(gamma)
        b = None if beta is None else _c64(beta)
        y = np.empty_like(x)
        self.lib.oracle_layernorm(_ptr(x), cols, _ptr(y), cols, rows, cols, _ptr(g), _ptr(b),
                                  float(eps), _act(act))
        return y

    def pointwise(self, x, act) -> np.ndarray:
        x = _c64(x)
        rows, cols = x.shape
        y = np.empty_like(x)
        self.lib.oracle_pointwise(_ptr(x), cols, _ptr(y), cols, rows, cols, _act(act))
        return y

    def split_op_cat(self, x, widths, gammas=None, betas=None, apply_ln=True, eps=1e-5,
                     act="none") -> np.ndarray:
        """split x along dim 1 into ``widths``, LayerNorm_j (optional) + act per piece, cat."""
        x = _c64(x)
        rows, D = x.shape
        widths = np.ascontiguousarray(widths, dtype=np.int64)
        n = widths.size
        keep = []

        def ptr_array(arrs):
            if arrs is None:
                return None
            out = (_dp * n)()
            for j, a in enumerate(arrs):
                if a is None:
                    out[j] = _dp()
                else:
                    a = _c64(a)
                    keep.append(a)
                    out[j] = _ptr(a)
            return out

        gp, bp = ptr_array(gammas), ptr_array(betas)
        y = np.empty_like(x)
        rc = self.lib.oracle_split_op_cat(_ptr(x), D, _ptr(y), D, rows, D, n, widths.ctypes.data_as(_i64p),
                                          gp, bp, int(bool(apply_ln)), float(eps), _act(act))
        if rc != 0:
            raise ValueError("oracle_split_op_cat: widths do not sum to D")
        return y

    def linear_layernorm(self, x, w, bias, gamma=None, beta=None, eps=1e-5, act="none") -> np.ndarray:
        """A Linear and the row-wise LayerNorm that consumes its output, fused
        (paper Sec. 3.2, vertical optimization of consecutive operators): the
        plain composition LN(X W^T + bias) over each output row, then act, in
        fp64 with no rounding of the intermediate."""
        return self.layernorm(self.linear(x, w, bias, "none"), gamma, beta, eps, act)

    # ------------------------------------------------------------ fp8 codec
    def fp8_decode(self, code: int) -> float:
        """Value of an OCP E4M3 code."""
        return self.lib.oracle_fp8e4m3_decode(int(code))

    def fp8_encode(self, v: float, saturate: bool = False) -> int:
        """OCP E4M3 code of v (round to nearest even; overflow -> NaN or +-448)."""
        return self.lib.oracle_fp8e4m3_encode(float(v), int(bool(saturate)))

    def quantize_fp8(self, x, use_scaling=True):
        """(codes uint8 [rows, cols], fp32 scale) of one tensor of fp32-exact values."""
        x = _c64(x)
        rows, cols = x.shape
        q = np.empty((rows, cols), dtype=np.uint8)
        sc = ctypes.c_float(1.0)
        self.lib.oracle_quantize_fp8(_ptr(x), cols, q.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), cols, rows,
                                     cols, int(bool(use_scaling)), ctypes.byref(sc))
        return q, np.float32(sc.value)

    def dequantize_fp8(self, q, scale=1.0) -> np.ndarray:
        """fp32(decode(code) * scale), as fp64 values."""
        q = np.ascontiguousarray(q, dtype=np.uint8)
        rows, cols = q.shape
        y = np.empty((rows, cols), dtype=np.float64)
        self.lib.oracle_dequantize_fp8(q.ctypes.data_as(ctypes.POINTER(ctypes.c_uint8)), cols, _ptr(y), cols, rows,
                                       cols, float(np.float32(scale)))
        return y

    # ------------------------------------------------------------ backward
    def linear_backward(self, x, w, dy):
        """(dX [M,K], dW [N,K], db [N]) of Y = X W^T + b given dY [M,N]."""
        x, w, dy = _c64(x), _c64(w), _c64(dy)
        M, K = x.shape
        N = w.shape[0]
        assert w.shape[1] == K and dy.shape == (M, N)
        dx = np.empty((M, K)); dw = np.empty((N, K)); db = np.empty(N)
        self.lib.oracle_linear_backward(_ptr(x), K, _ptr(w), K, _ptr(dy), N, _ptr(dx), K, _ptr(dw), K, _ptr(db),
                                        M, N, K)
        return dx, dw, db

    def act_grad_scalar(self, x: float, act) -> float:
        return self.lib.oracle_act_grad_scalar(float(x), _act(act))

    def act_backward(self, x, dy, act) -> np.ndarray:
        """dX = dY * act'(X), X the activation's input."""
        x, dy = _c64(x), _c64(dy)
        rows, cols = x.shape
        dx = np.empty_like(x)
        self.lib.oracle_act_backward(_ptr(x), cols, _ptr(dy), cols, _ptr(dx), cols, rows, cols, _act(act))
        return dx

    def layernorm_backward(self, x, gamma, dy, eps=1e-5):
        """(dX, dgamma, dbeta) of the row LayerNorm (gamma None = 1)."""
        x, dy = _c64(x), _c64(dy)
        rows, cols = x.shape
        g = None if gamma is None else _c64(gamma)
        dx = np.empty_like(x); dg = np.empty(cols); dbt = np.empty(cols)
        self.lib.oracle_layernorm_backward(_ptr(x), cols, _ptr(g), _ptr(dy), cols, _ptr(dx), cols, _ptr(dg),
                                           _ptr(dbt), rows, cols, float(eps))
        return dx, dg, dbt

    def num_threads(self) -> int:
        return self.lib.oracle_num_threads()

    def set_num_threads(self, n: int) -> None:
        """OpenMP threads of the following calls (the CPU baseline's 1-thread run)."""
        self.lib.oracle_set_num_threads(int(n))

    # ------------------------------------------------------------ groups
    # A group is a list of members; grouping changes nothing in the math
    # (paper Sec. 3.2 group fusion), so each is a loop over members.
    def grouped_linear(self, xs, ws, biases, act="none"):
        return [self.linear(x, w, b, act) for x, w, b in zip(xs, ws, biases)]

    def grouped_layernorm(self, xs, gammas, betas, eps=1e-5, act="none"):
        return [self.layernorm(x, g, b, eps, act) for x, g, b in zip(xs, gammas, betas)]

    def grouped_linear_layernorm(self, xs, ws, biases, gammas, betas, eps=1e-5, act="none"):
        return [self.linear_layernorm(x, w, b, g, be, eps, act)
                for x, w, b, g, be in zip(xs, ws, biases, gammas, betas)]

    def grouped_pointwise(self, xs, act):
        return [self.pointwise(x, act) for x in xs]


_default: Optional[Oracle] = None


def get() -> Oracle:
    """The oracle built from ``optimus_oracle.c`` (compiled on first use)."""
    global _default
    if _default is None:
        _default = Oracle()
    return _default


def timed(fn, *args, **kw):
    """Run fn and return (result, wall seconds) -- for the CPU baseline."""
    t0 = time.perf_counter()
    r = fn(*args, **kw)
    return r, time.perf_counter() - t0
