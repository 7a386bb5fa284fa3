"""Pins for the fp64 oracle: every check compares the oracle with something other
than itself -- a library routine (numpy BLAS, torch fp64 ops), a closed form, an
invariant, brute force in exact integer arithmetic, or the paper's appendix
split-concat example. Each check raises AssertionError on a mismatch.

Kept as plain functions taking an ``Oracle`` so that the mutant test can run the
same checks against copies of the oracle with planted mistakes.
"""
from __future__ import annotations

import itertools
import json
import os

import numpy as np
import torch

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _rng(seed):
    return np.random.Generator(np.random.PCG64(seed))


def _nrm(a, b):
    """inf-normwise relative difference."""
    a, b = np.asarray(a, np.float64), np.asarray(b, np.float64)
    return np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300)


# ---------------------------------------------------------------- Linear
def linear_vs_blas(orc):
    """Y = X W^T + b against numpy's float64 matmul (BLAS dgemm) and torch's F.linear."""
    g = _rng(1)
    for (M, N, K) in [(7, 5, 3), (33, 17, 64), (64, 48, 16), (5, 129, 31)]:
        x, w, b = g.standard_normal((M, K)), g.standard_normal((N, K)), g.standard_normal(N)
        y = orc.linear(x, w, b)
        assert y.shape == (M, N)
        assert _nrm(y, x @ w.T + b) < 1e-13, (M, N, K)
        t = torch.nn.functional.linear(torch.from_numpy(x), torch.from_numpy(w), torch.from_numpy(b))
        assert _nrm(y, t.numpy()) < 1e-13
        assert _nrm(orc.linear(x, w, None), x @ w.T) < 1e-13


def linear_special_cases(orc):
    """Zero weights give the bias exactly; identity weights give the input exactly."""
    g = _rng(2)
    x, b = g.standard_normal((9, 6)), g.standard_normal(4)
    y = orc.linear(x, np.zeros((4, 6)), b)
    assert np.array_equal(y, np.broadcast_to(b, (9, 4)))
    x = g.standard_normal((11, 8))
    assert np.array_equal(orc.linear(x, np.eye(8), np.zeros(8)), x)
    assert np.array_equal(orc.linear(x, np.eye(8), None), x)


def linear_brute_force(orc):
    """Tiny groups of small integers: exact integer sums by brute force (every
    M, N, K in 1..4), so the oracle must match bit for bit."""
    g = _rng(3)
    for M, N, K in itertools.product(range(1, 5), repeat=3):
        x = g.integers(-4, 5, size=(M, K))
        w = g.integers(-4, 5, size=(N, K))
        b = g.integers(-8, 9, size=N)
        want = [[sum(int(x[m, k]) * int(w[n, k]) for k in range(K)) + int(b[n]) for n in range(N)]
                for m in range(M)]
        got = orc.linear(x.astype(np.float64), w.astype(np.float64), b.astype(np.float64))
        assert np.array_equal(got, np.array(want, dtype=np.float64)), (M, N, K)


def linear_epilogue(orc):
    """Linear followed by an activation equals the activation of the Linear."""
    g = _rng(4)
    x, w, b = g.standard_normal((13, 24)), g.standard_normal((10, 24)), g.standard_normal(10)
    z = x @ w.T + b
    want = {"relu": np.maximum(z, 0), "sigmoid": 1 / (1 + np.exp(-z)), "tanh": np.tanh(z),
            "silu": z / (1 + np.exp(-z)), "none": z}
    for a, v in want.items():
        assert _nrm(orc.linear(x, w, b, a), v) < 1e-13, a


def linear_rows_subset(orc):
    """Selected rows equal the same rows of the full Linear."""
    g = _rng(5)
    x, w, b = g.standard_normal((40, 20)), g.standard_normal((7, 20)), g.standard_normal(7)
    rows = np.array([39, 0, 17, 17, 3])
    assert np.array_equal(orc.linear_rows(x, w, b, rows, "tanh"), orc.linear(x, w, b, "tanh")[rows])
    assert _nrm(orc.linear_rows(x, w, b, rows), (x @ w.T + b)[rows]) < 1e-13


def linear_batch_fusion(orc):
    """Paper Sec. 3.2 batch fusion: equal-shape members stacked into one batched
    matmul (then unbound) give the grouped per-member results."""
    g = _rng(6)
    G, M, N, K = 5, 12, 8, 16
    xs, ws, bs = g.standard_normal((G, M, K)), g.standard_normal((G, N, K)), g.standard_normal((G, N))
    stacked = np.matmul(xs, np.transpose(ws, (0, 2, 1))) + bs[:, None, :]
    got = orc.grouped_linear(list(xs), list(ws), list(bs))
    for i in range(G):
        assert _nrm(got[i], stacked[i]) < 1e-13


def linear_shared_input(orc):
    """Paper Table 1 batch_linear_lhs: members that share one input equal a
    single matmul of that input with the members' weights concatenated along N
    (numpy BLAS), split back into the members' columns."""
    g = _rng(16)
    M, K, Ns = 14, 24, [3, 9, 1, 6]
    x = g.standard_normal((M, K))
    ws = [g.standard_normal((n, K)) for n in Ns]
    bs = [g.standard_normal(n) for n in Ns]
    whole = x @ np.concatenate(ws).T + np.concatenate(bs)
    got = orc.grouped_linear([x] * len(Ns), ws, bs)
    offs = np.cumsum([0] + Ns)
    for i in range(len(Ns)):
        assert _nrm(got[i], whole[:, offs[i]:offs[i + 1]]) < 1e-13


# ---------------------------------------------------------------- LayerNorm
def layernorm_vs_torch(orc):
    """Row LayerNorm against torch.nn.functional.layer_norm in fp64."""
    g = _rng(7)
    for rows, cols in [(5, 16), (9, 48), (3, 1000), (4, 1)]:
        x = g.standard_normal((rows, cols)) * 3 + 1
        gm, bt = g.uniform(0.5, 1.5, cols), g.standard_normal(cols)
        t = torch.nn.functional.layer_norm(torch.from_numpy(x), (cols,), torch.from_numpy(gm),
                                           torch.from_numpy(bt), eps=1e-5).numpy()
        assert _nrm(orc.layernorm(x, gm, bt, 1e-5), t) < 1e-12, (rows, cols)
        t0 = torch.nn.functional.layer_norm(torch.from_numpy(x), (cols,), eps=1e-3).numpy()
        assert _nrm(orc.layernorm(x, None, None, 1e-3), t0) < 1e-12


def layernorm_invariants(orc):
    """gamma=1, beta=0: per-row mean 0 and per-row (biased) variance equal to
    s2/(s2+eps) in closed form, where s2 is the row's biased variance."""
    g = _rng(8)
    x = g.standard_normal((20, 64)) * g.uniform(0.01, 10, (20, 1)) + g.standard_normal((20, 1))
    for eps in (1e-5, 0.5):
        y = orc.layernorm(x, np.ones(64), np.zeros(64), eps)
        s2 = x.var(axis=1)
        assert np.max(np.abs(y.mean(axis=1))) < 1e-12
        assert np.max(np.abs(y.var(axis=1) - s2 / (s2 + eps))) < 1e-12


def layernorm_constant_row(orc):
    """A constant row has zero variance, so the output is beta exactly, with no NaN."""
    bt = np.linspace(-2, 2, 32)
    x = np.full((3, 32), 0.75)
    y = orc.layernorm(x, np.full(32, 3.0), bt, 1e-5)
    assert np.array_equal(y, np.broadcast_to(bt, (3, 32)))


def layernorm_affine(orc):
    """The affine step is elementwise: LN(x; gamma, beta) = gamma * LN(x; 1, 0) + beta."""
    g = _rng(9)
    x = g.standard_normal((6, 40))
    gm, bt = g.uniform(-2, 2, 40), g.standard_normal(40)
    plain = orc.layernorm(x, None, None, 1e-5)
    assert _nrm(orc.layernorm(x, gm, bt, 1e-5), plain * gm + bt) < 1e-14


def layernorm_epilogue_and_batch(orc):
    """LN followed by an activation; equal-width members equal one LN over the stack."""
    g = _rng(10)
    x = g.standard_normal((4, 8, 24))
    stack = torch.nn.functional.layer_norm(torch.from_numpy(x), (24,), eps=1e-5).numpy()
    got = orc.grouped_layernorm(list(x), [None] * 4, [None] * 4, 1e-5, "tanh")
    for i in range(4):
        assert _nrm(got[i], np.tanh(stack[i])) < 1e-12


# ---------------------------------------------------------------- Linear + LayerNorm
def linear_layernorm_reductions(orc):
    """The fused Linear + LayerNorm reduces to a plain LayerNorm when W is the
    identity: with bias 0 it equals LN(x) (+ act), with a bias it equals
    LN(x + bias); the activation comes after the normalisation, not before."""
    g = _rng(17)
    x = g.standard_normal((12, 20)) * 2 + 0.5
    eye = np.eye(20)
    gm, bt = g.uniform(0.5, 1.5, 20), g.standard_normal(20)
    for act in ("none", "tanh", "silu"):
        got = orc.linear_layernorm(x, eye, np.zeros(20), gm, bt, 1e-5, act)
        assert _nrm(got, orc.layernorm(x, gm, bt, 1e-5, act)) < 1e-14, act
    b = g.standard_normal(20)
    assert _nrm(orc.linear_layernorm(x, eye, b, gm, bt, 1e-5), orc.layernorm(x + b, gm, bt, 1e-5)) < 1e-14
    t = torch.nn.functional.layer_norm(torch.from_numpy(x @ eye.T + b), (20,), torch.from_numpy(gm),
                                       torch.from_numpy(bt), eps=1e-5).numpy()
    assert _nrm(orc.linear_layernorm(x, eye, b, gm, bt, 1e-5), t) < 1e-12


def linear_layernorm_invariants(orc):
    """gamma=1, beta=0 over a real Linear: each output row has mean 0 and biased
    variance s2/(s2+eps), s2 the variance of the Linear's row (numpy BLAS);
    a weight matrix whose rows are all equal (and a constant bias) makes every
    output row constant, so the result is beta exactly."""
    g = _rng(18)
    x, w, b = g.standard_normal((9, 16)), g.standard_normal((24, 16)), g.standard_normal(24)
    y = orc.linear_layernorm(x, w, b, np.ones(24), np.zeros(24), 1e-5)
    s2 = (x @ w.T + b).var(axis=1)
    assert np.max(np.abs(y.mean(axis=1))) < 1e-12
    assert np.max(np.abs(y.var(axis=1) - s2 / (s2 + 1e-5))) < 1e-12
    # integer x and w: every dot product, sum and mean of a row is exact
    x = g.integers(-3, 4, (9, 16)).astype(np.float64)
    wc = np.broadcast_to(g.integers(-3, 4, 16).astype(np.float64), (24, 16))
    bt = np.linspace(-1, 1, 24)
    yc = orc.linear_layernorm(x, wc, np.full(24, 0.25), np.full(24, 2.0), bt, 1e-5)
    assert np.array_equal(yc, np.broadcast_to(bt, (9, 24)))


# ---------------------------------------------------------------- fp8 codec
def _torch_e4m3_value(codes):
    """Values of E4M3 codes through torch's own float8_e4m3fn type."""
    return torch.tensor(np.asarray(codes, np.uint8)).view(torch.float8_e4m3fn).to(torch.float64).numpy()


def _torch_e4m3_code(values):
    return torch.tensor(np.asarray(values, np.float32)).to(torch.float8_e4m3fn).view(torch.uint8).numpy()


def fp8_decode_all_codes(orc):
    """Every one of the 256 codes decodes to torch's float8_e4m3fn value (NaN
    at S.1111.111 only); the largest finite is 448 and the smallest subnormal 2^-9."""
    got = np.array([orc.fp8_decode(c) for c in range(256)])
    ref = _torch_e4m3_value(range(256))
    assert np.array_equal(np.isnan(got), np.isnan(ref)) and np.isnan(got).sum() == 2
    fin = ~np.isnan(ref)
    assert np.array_equal(got[fin], ref[fin]) and np.array_equal(np.signbit(got[fin]), np.signbit(ref[fin]))
    assert np.nanmax(got) == 448.0 and got[1] == 2.0 ** -9


def fp8_encode_round_trip_and_ties(orc):
    """encode(decode(c)) == c for every finite code (both modes), and every
    midpoint between adjacent codes of one sign goes to the even mantissa."""
    for sat in (False, True):
        for c in range(256):
            if c & 0x7F == 0x7F:
                continue
            assert orc.fp8_encode(orc.fp8_decode(c), sat) == c, (c, sat)
    for c in range(0, 0x7E):
        lo, hi = orc.fp8_decode(c), orc.fp8_decode(c + 1)
        mid = (lo + hi) / 2
        want = c if c % 2 == 0 else c + 1
        assert orc.fp8_encode(mid) == want and orc.fp8_encode(-mid) == want | 0x80, c
        assert orc.fp8_encode(np.nextafter(mid, 0)) == c and orc.fp8_encode(np.nextafter(mid, 1e9)) == c + 1


def fp8_encode_vs_torch(orc):
    """Every bf16 value (overflow, infinities and NaNs of both signs included)
    and 20000 random fp32 values of every magnitude encode, unsaturated, as
    torch's float8_e4m3fn conversion does; the fp32 neighbours of the overflow
    tie 464 too."""
    bits = np.arange(65536, dtype=np.uint32) << 16
    vals = bits.view(np.float32)
    g = _rng(19)
    rnd = (g.standard_normal(20000) * np.exp2(g.uniform(-14, 10, 20000))).astype(np.float32)
    edge = np.array([464.0, np.nextafter(np.float32(464), np.float32(0)), np.nextafter(np.float32(464), np.float32(1e9)),
                     447.99, 448.0, 456.0, 472.0, 479.99, 480.0], np.float32)
    for v in (vals, rnd, edge, -edge):
        got = np.array([orc.fp8_encode(float(t)) for t in v], dtype=np.uint8)
        assert np.array_equal(got, _torch_e4m3_code(v))


def fp8_overflow_and_scaling(orc):
    """Unscaled: |x| > 464 and infinities give NaN; the tie 464 itself rounds
    to the even mantissa, 448. Saturated: overflow and infinities give +-448,
    NaN stays NaN with its sign. Scaled: the largest magnitude lands exactly
    on +-448, every code is finite, and decode(code) * scale is within half a
    code step of x."""
    above = float(np.nextafter(464.0, 1e9))
    assert orc.fp8_encode(463.99) == 0x7E and orc.fp8_encode(464.0) == 0x7E and orc.fp8_encode(-464.0) == 0xFE
    assert orc.fp8_encode(above) == 0x7F and orc.fp8_encode(-above) == 0xFF
    assert orc.fp8_encode(float("inf")) == 0x7F and orc.fp8_encode(-float("inf")) == 0xFF
    assert orc.fp8_encode(float("nan")) == 0x7F and orc.fp8_encode(-float("nan")) == 0xFF
    assert orc.fp8_encode(1e6, True) == 0x7E and orc.fp8_encode(-1e6, True) == 0xFE
    assert orc.fp8_encode(above, True) == 0x7E and orc.fp8_encode(-float("inf"), True) == 0xFE
    assert orc.fp8_encode(float("nan"), True) == 0x7F and orc.fp8_encode(-float("nan"), True) == 0xFF
    g = _rng(20)
    x = (g.standard_normal((40, 33)) * 37.0).astype(np.float32).astype(np.float64)
    q, scale = orc.quantize_fp8(x, True)
    assert np.float32(scale) == np.float32(np.float32(np.abs(x).max()) / np.float32(448.0))
    i = np.unravel_index(np.argmax(np.abs(x)), x.shape)
    assert q[i] in (0x7E, 0xFE) and np.all((q & 0x7F) != 0x7F)
    y = orc.dequantize_fp8(q, scale)
    step = np.exp2(np.floor(np.log2(np.maximum(np.abs(x) / scale, 2.0 ** -6))) - 3) * scale
    assert np.all(np.abs(y - x) <= step / 2 * (1 + 1e-6))
    # torch: the same codes decode to the same values, times the fp32 scale
    ref = (torch.tensor(q).view(torch.float8_e4m3fn).to(torch.float32) * torch.tensor(scale)).to(torch.float64)
    assert np.array_equal(y, ref.numpy())
    # an infinite element makes amax infinite: inv = 0, finite values give
    # (signed) zero codes, the infinities NaN codes with their own sign
    xi = np.array([[1.5, -2.0, np.inf], [-np.inf, 0.0, 3.0]])
    qi, si = orc.quantize_fp8(xi, True)
    assert np.isinf(si) and qi.tolist() == [[0x00, 0x80, 0x7F], [0xFF, 0x00, 0x00]]
    # unscaled: in-range values keep torch's codes; 500 -> NaN
    x[0, 0] = 500.0
    qu, _ = orc.quantize_fp8(x, False)
    assert qu[0, 0] == 0x7F
    fin = np.abs(x) < 448
    assert np.array_equal(qu[fin], _torch_e4m3_code(x[fin].astype(np.float32)))


# ---------------------------------------------------------------- pointwise
def pointwise_closed_forms(orc):
    """Values at 0, symmetries, the tanh/sigmoid identity, saturation, numpy forms."""
    a = orc.act_scalar
    assert a(0.0, "sigmoid") == 0.5 and a(0.0, "tanh") == 0.0 and a(0.0, "silu") == 0.0
    assert a(-3.5, "relu") == 0.0 and a(2.25, "relu") == 2.25 and a(-7.0, "none") == -7.0
    assert abs(a(30.0, "sigmoid") - 1.0) < 1e-13 and 0.0 <= a(-30.0, "sigmoid") < 1e-13
    assert a(-800.0, "sigmoid") == 0.0 and a(800.0, "sigmoid") == 1.0   # no overflow
    assert a(-800.0, "silu") == 0.0
    x = np.linspace(-12, 12, 97)
    for v in x:
        s, t = a(v, "sigmoid"), a(v, "tanh")
        assert abs(a(-v, "sigmoid") - (1.0 - s)) < 1e-15
        assert a(-v, "tanh") == -t
        assert abs(t - (2.0 * a(2.0 * v, "sigmoid") - 1.0)) < 1e-14
        assert abs(a(v, "silu") - v * s) < 1e-14
    g = _rng(11)
    z = g.standard_normal((7, 33)) * 4
    assert _nrm(orc.pointwise(z, "tanh"), np.tanh(z)) < 1e-15
    assert _nrm(orc.pointwise(z, "sigmoid"), 1 / (1 + np.exp(-z))) < 1e-14
    assert _nrm(orc.pointwise(z, "silu"), z / (1 + np.exp(-z))) < 1e-14
    assert np.array_equal(orc.pointwise(z, "relu"), np.maximum(z, 0))
    assert np.array_equal(orc.pointwise(z, "none"), z)


# ---------------------------------------------------------------- split-op-cat
def split_concat_appendix_example(orc):
    """Appendix Sec. 8.1 listing: split [2,4] on dim 1, split the second piece
    [2,2], cat the three pieces on dim 1 -- the optimized program returns x."""
    with open(os.path.join(GOLDEN, "appendix_split_concat.json")) as f:
        ex = json.load(f)
    shape = tuple(ex["input_shape"])
    first = ex["first_split_sizes"]
    nested = ex["nested_split_sizes"]
    flat = first[:ex["nested_split_of_piece"]] + nested + first[ex["nested_split_of_piece"] + 1:]
    assert flat == ex["flattened_widths"]
    x = _rng(12).standard_normal(shape)
    y = orc.split_op_cat(x, flat, apply_ln=False, act="none")
    assert np.array_equal(y, x)
    # the same program written with torch on the CPU gives the same tensor
    t = torch.from_numpy(x)
    fs = torch.split(t, first, dim=1)
    pieces = [fs[0]] + list(fs[1].split(tuple(nested), 1))
    assert np.array_equal(torch.cat(pieces, dim=1).numpy(), y)


def split_concat_identity_random(orc):
    """split o cat is the identity for any widths (bit-exact)."""
    g = _rng(13)
    for D, n in [(64, 4), (4096, 32), (48, 3)]:
        cuts = np.sort(g.choice(np.arange(1, D), size=n - 1, replace=False))
        widths = np.diff(np.concatenate([[0], cuts, [D]]))
        x = g.standard_normal((5, D))
        assert np.array_equal(orc.split_op_cat(x, widths, apply_ln=False, act="none"), x)


def split_op_cat_pieces(orc):
    """Each output piece equals torch's LayerNorm + activation of that input piece,
    placed at its column offset; one piece of full width is a plain row LayerNorm;
    equal widths equal one LayerNorm over the stacked pieces (batch fusion)."""
    g = _rng(14)
    widths = [16, 48, 32, 160]
    D = sum(widths)
    x = g.standard_normal((6, D)) * 2 + 0.5
    gms = [g.uniform(0.5, 1.5, w) for w in widths]
    bts = [g.standard_normal(w) * 0.3 for w in widths]
    y = orc.split_op_cat(x, widths, gms, bts, True, 1e-5, "silu")
    o = 0
    for w, gm, bt in zip(widths, gms, bts):
        ref = torch.nn.functional.layer_norm(torch.from_numpy(x[:, o:o + w]), (w,), torch.from_numpy(gm),
                                             torch.from_numpy(bt), eps=1e-5)
        ref = torch.nn.functional.silu(ref).numpy()
        assert _nrm(y[:, o:o + w], ref) < 1e-12, (o, w)
        o += w
    one = orc.split_op_cat(x, [D], None, None, True, 1e-5, "none")
    assert _nrm(one, torch.nn.functional.layer_norm(torch.from_numpy(x), (D,), eps=1e-5).numpy()) < 1e-12
    xe = g.standard_normal((3, 8 * 16))
    ye = orc.split_op_cat(xe, [16] * 8, None, None, True, 1e-5, "tanh")
    st = torch.nn.functional.layer_norm(torch.from_numpy(xe.reshape(3, 8, 16)), (16,), eps=1e-5)
    assert _nrm(ye, torch.tanh(st).numpy().reshape(3, 128)) < 1e-12


def split_op_cat_tag(orc):
    """gamma_j = 0, beta_j = j: every element of piece j must equal j, so piece j
    lands exactly at its offset."""
    widths = [2, 5, 1, 8, 16]
    x = _rng(15).standard_normal((4, sum(widths)))
    y = orc.split_op_cat(x, widths, [np.zeros(w) for w in widths],
                         [np.full(w, float(j)) for j, w in enumerate(widths)], True, 1e-5, "none")
    want = np.concatenate([np.full((4, w), float(j)) for j, w in enumerate(widths)], axis=1)
    assert np.array_equal(y, want)


def split_op_cat_bad_widths(orc):
    try:
        orc.split_op_cat(np.zeros((2, 6)), [2, 2], apply_ln=False)
    except ValueError:
        return
    raise AssertionError("widths not summing to D must be rejected")


# ---------------------------------------------------------------- backward
def _autograd(fn, inputs, dy):
    """Gradients of sum(fn(*inputs) * dy) with torch autograd in fp64."""
    ts = [torch.tensor(a, dtype=torch.float64, requires_grad=True) for a in inputs]
    out = fn(*ts)
    out.backward(torch.tensor(dy, dtype=torch.float64))
    return [t.grad.numpy() for t in ts]


def linear_backward_vs_autograd(orc):
    """dX, dW, db of Y = X W^T + b against torch autograd (fp64) on ragged shapes."""
    g = _rng(40)
    for (M, N, K) in [(7, 5, 3), (33, 17, 64), (1, 9, 4), (65, 1, 2)]:
        x, w, b = g.standard_normal((M, K)), g.standard_normal((N, K)), g.standard_normal(N)
        dy = g.standard_normal((M, N))
        ref = _autograd(torch.nn.functional.linear, [x, w, b], dy)
        got = orc.linear_backward(x, w, dy)
        for a, r, name in zip(got, ref, ("dx", "dw", "db")):
            assert a.shape == r.shape and _nrm(a, r) < 1e-13, (M, N, K, name)


def linear_backward_integer_and_fd(orc):
    """Small integers: exact against numpy's int64 products; and a central
    difference of the oracle's own forward along a random direction matches
    the oracle's gradient (ties the backward to the forward definition)."""
    g = _rng(41)
    x = g.integers(-4, 5, (6, 3)); w = g.integers(-4, 5, (4, 3)); dy = g.integers(-3, 4, (6, 4))
    dx, dw, db = orc.linear_backward(x.astype(float), w.astype(float), dy.astype(float))
    assert np.array_equal(dx, (dy @ w).astype(float)) and np.array_equal(dw, (dy.T @ x).astype(float))
    assert np.array_equal(db, dy.sum(0).astype(float))
    x, w, b, dy = g.standard_normal((5, 4)), g.standard_normal((3, 4)), g.standard_normal(3), g.standard_normal((5, 3))
    vx, vw = g.standard_normal(x.shape), g.standard_normal(w.shape)
    L = lambda xx, ww: float(np.sum(orc.linear(xx, ww, b) * dy))
    h = 1e-6
    fd = (L(x + h * vx, w + h * vw) - L(x - h * vx, w - h * vw)) / (2 * h)
    dx, dw, _ = orc.linear_backward(x, w, dy)
    assert abs(fd - (np.sum(dx * vx) + np.sum(dw * vw))) < 1e-7


def act_backward_vs_autograd(orc):
    """act'(x) for every activation against torch autograd (fp64), including
    x = 0 exactly (relu passes no gradient there) and large |x|."""
    x = np.concatenate([np.linspace(-9, 9, 37), [0.0, -0.0, 30.0, -30.0, 1e-8]]).reshape(1, -1)
    dy = _rng(42).standard_normal(x.shape)
    fns = {"none": lambda t: t, "relu": torch.relu, "sigmoid": torch.sigmoid, "tanh": torch.tanh,
           "silu": torch.nn.functional.silu}
    for act, fn in fns.items():
        ref = _autograd(fn, [x], dy)[0]
        got = orc.act_backward(x, dy, act)
        assert np.max(np.abs(got - ref)) < 1e-14, act
    assert orc.act_grad_scalar(0.0, "sigmoid") == 0.25 and orc.act_grad_scalar(0.0, "tanh") == 1.0
    assert orc.act_grad_scalar(0.0, "silu") == 0.5 and orc.act_grad_scalar(0.0, "relu") == 0.0


def layernorm_backward_vs_autograd(orc):
    """dX, dgamma, dbeta of the row LayerNorm against torch autograd (fp64),
    with and without gamma, several eps."""
    g = _rng(43)
    for (R, C, eps) in [(5, 8, 1e-5), (17, 33, 1e-3), (1, 3, 0.0), (9, 64, 0.5)]:
        x, gm, bt = g.standard_normal((R, C)) * 3 + 1, g.uniform(0.5, 1.5, C), g.standard_normal(C)
        dy = g.standard_normal((R, C))
        fn = lambda xx, gg, bb: torch.nn.functional.layer_norm(xx, (C,), gg, bb, eps)
        ref = _autograd(fn, [x, gm, bt], dy)
        got = orc.layernorm_backward(x, gm, dy, eps)
        for a, r, name in zip(got, ref, ("dx", "dgamma", "dbeta")):
            assert _nrm(a, r) < 1e-12, (R, C, eps, name)
        ref1 = _autograd(lambda xx: torch.nn.functional.layer_norm(xx, (C,), None, None, eps), [x], dy)[0]
        assert _nrm(orc.layernorm_backward(x, None, dy, eps)[0], ref1) < 1e-12


def layernorm_backward_invariants(orc):
    """With eps = 0 the output is invariant to shifting and scaling an input
    row, so each row gradient is orthogonal to 1 and to x; dbeta = column
    sums of dY, dgamma = column sums of dY * xhat; a central difference of the
    oracle's forward (eps = 1e-5, with gamma)."""
    g = _rng(44)
    x, dy = g.standard_normal((12, 40)) * 2, g.standard_normal((12, 40))
    dx, dg, dbt = orc.layernorm_backward(x, None, dy, 0.0)
    xhat = orc.layernorm(x, None, None, 0.0)
    assert np.max(np.abs(dx.sum(1))) < 1e-12 and np.max(np.abs((dx * x).sum(1))) < 1e-11
    assert np.max(np.abs(dbt - dy.sum(0))) < 1e-12 and np.max(np.abs(dg - (dy * xhat).sum(0))) < 1e-12
    gm = g.uniform(0.5, 1.5, 40)
    v = g.standard_normal(x.shape)
    L = lambda xx: float(np.sum(orc.layernorm(xx, gm, None, 1e-5) * dy))
    h = 1e-6
    fd = (L(x + h * v) - L(x - h * v)) / (2 * h)
    assert abs(fd - np.sum(orc.layernorm_backward(x, gm, dy, 1e-5)[0] * v)) < 1e-6


ALL_PINS = [
    linear_vs_blas, linear_special_cases, linear_brute_force, linear_epilogue, linear_rows_subset,
    linear_batch_fusion, linear_shared_input, layernorm_vs_torch, layernorm_invariants, layernorm_constant_row,
    layernorm_affine, layernorm_epilogue_and_batch, linear_layernorm_reductions, linear_layernorm_invariants,
    fp8_decode_all_codes, fp8_encode_round_trip_and_ties, fp8_encode_vs_torch, fp8_overflow_and_scaling,
    linear_backward_vs_autograd, linear_backward_integer_and_fd, act_backward_vs_autograd,
    layernorm_backward_vs_autograd, layernorm_backward_invariants,
    pointwise_closed_forms,
    split_concat_appendix_example, split_concat_identity_random, split_op_cat_pieces, split_op_cat_tag,
    split_op_cat_bad_widths,
]
