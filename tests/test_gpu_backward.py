"""Backward of the grouped operators on the GPU against the fp64 oracle,
through the C ABI: Linear (dX, dW, db), activation, LayerNorm (dX, dgamma,
dbeta); inf-normwise relative error per member and output, 1e-5 for fp32 and
2e-2 for bf16 (fp32 sums, one rounding of each output)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_02945_amd import binding as B
from paper_2607_02945_amd import synth
from tests.gpu_util import assert_close, dev, host64, say

pytestmark = pytest.mark.gpu
ORC = oracle.get()
ACTS = ["none", "relu", "sigmoid", "tanh", "silu"]


def _t(a, dtype, pad=0, off=0):
    """Device tensor of the values (rounded once to the dtype), optionally a
    column slice of a wider buffer (row stride cols + pad + off, start off)."""
    st = synth.to_storage(a, dtype)
    if not pad and not off:
        return dev(st), synth.exact64(st)
    r, c = st.shape
    base = torch.zeros((r, c + pad + off), dtype=st.dtype)
    base[:, off:off + c] = st
    return dev(base)[:, off:off + c], synth.exact64(st)


def _empty(shape, dtype, pad=0):
    t = torch.full((shape[0], shape[1] + pad), float("nan"), dtype=synth.DTYPES[dtype], device="cuda")
    return t[:, :shape[1]] if pad else t


# ------------------------------------------------------------------ Linear
def _linear_members(shapes, dtype, seed, pad=0):
    g = synth.rng(seed)
    ms = []
    for M, N, K in shapes:
        x, x64 = _t(g.standard_normal((M, K)), dtype, pad)
        w, w64 = _t(g.standard_normal((N, K)) / np.sqrt(K), dtype, pad)
        dy, dy64 = _t(g.standard_normal((M, N)), dtype, pad)
        ms.append({"x": x, "w": w, "dy": dy, "x64": x64, "w64": w64, "dy64": dy64, "M": M, "N": N, "K": K})
    return ms


def _run_linear_bwd(ms, dtype, mode="oneshot", want=("dx", "dw", "db"), variant=None, pad=0, splits=0):
    """The one-shot call, or a plan executed in `mode`; a pinned tile variant
    (kernel-table index) or dW split count goes through the plan options."""
    for m in ms:
        m["dx"] = _empty((m["M"], m["K"]), dtype, pad) if "dx" in want else None
        m["dw"] = _empty((m["N"], m["K"]), dtype, pad) if "dw" in want else None
        m["db"] = torch.full((m["N"],), float("nan"), dtype=synth.DTYPES[dtype], device="cuda") if "db" in want else None
    args = ([m["x"] for m in ms], [m["w"] for m in ms], [m["dy"] for m in ms], [m["dx"] for m in ms],
            [m["dw"] for m in ms], [m["db"] for m in ms])
    opts = None
    if variant is not None or splits:
        opts = {"gemm_tile": 0 if variant is None else variant + 1, "wgrad_splits": splits}
    info = None
    if mode == "oneshot" and opts is None:
        B.optimus_grouped_linear_backward(*args)
    else:
        p = B.optimus_plan_linear_backward_ex(*args, options=opts)
        info = p.info()
        p.execute("grouped" if mode == "oneshot" else mode)
        torch.cuda.synchronize()
        p.close()
    torch.cuda.synchronize()
    return info


def _check_linear_bwd(ms, dtype, what, want=("dx", "dw", "db")):
    for i, m in enumerate(ms):
        rdx, rdw, rdb = ORC.linear_backward(m["x64"], m["w64"], m["dy64"])
        if "dx" in want:
            assert_close(host64(m["dx"]), rdx, dtype, f"{what} member {i} dx")
        if "dw" in want:
            assert_close(host64(m["dw"]), rdw, dtype, f"{what} member {i} dw")
        if "db" in want:
            assert_close(host64(m["db"][None, :])[0], rdb, dtype, f"{what} member {i} db")


SHAPES = [(1000, 256, 512), (300, 200, 136), (64, 17, 40), (513, 96, 8), (4097, 24, 64)]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("mode", ["oneshot", "grouped", "chain"])
def test_linear_backward(dtype, mode):
    """Ragged members (tails in every dimension, K and N not multiples of the
    16-byte chunk), every output."""
    say(f"[linear bwd] {dtype} {mode}")
    ms = _linear_members(SHAPES, dtype, seed=500)
    info = _run_linear_bwd(ms, dtype, mode)
    if info is not None:
        n = _launches(info)
        assert info["kind"] == 7 and info["launches"] == n and info["chain_launches"] == n * len(ms), info
    _check_linear_bwd(ms, dtype, f"{dtype} {mode}")


def _launches(info):
    """Launches of a Linear backward plan with dX and dW: the transpose of W
    (unless dX reads W as it lies), dX, dW and, when dW's batch is split,
    the reduction."""
    k = info["kernel"]
    return 1 + ("_dgrad_direct" not in k) + 1 + ("_split" in k)


def _wgrad_part(info):
    return [p for p in info["kernel"].split("+") if p.endswith("_wgrad") or "_wgrad_split" in p][0]


@pytest.mark.parametrize("variant", [1, 2, 3, 4, 5, 6])
def test_linear_backward_every_tile(variant):
    """Each tile shape of the backward GEMMs (bf16 128x128 and 256x256
    register-staged, the same two direct-to-LDS with transposing fragment
    reads, fp32 64x64 and 64x128), grouped and chain. The direct-to-LDS
    tiles take widths that are multiples of 8 values, still ragged against
    every tile and with batch tails."""
    dtype = "fp32" if variant in (3, 6) else "bf16"
    say(f"[linear bwd variant] {variant}")
    shapes = [(700, 296, 264), (129, 64, 32), (257, 8, 520)] if variant in (4, 5) else \
        [(700, 300, 260), (129, 64, 33), (257, 9, 520)]
    ms = _linear_members(shapes, dtype, seed=510 + variant)
    for mode in ["grouped", "chain"]:
        info = _run_linear_bwd(ms, dtype, mode, variant=variant)
        assert ("dma" in _wgrad_part(info)) == (variant in (4, 5)), info
        assert ("_dgrad_direct" in info["kernel"]) == (variant in (4, 5)), info   # W read as it lies
        _check_linear_bwd(ms, dtype, f"variant {variant} {mode}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("mode", ["oneshot", "grouped", "chain"])
@pytest.mark.parametrize("aligned", [False, True])
def test_linear_backward_split_reduction(dtype, mode, aligned):
    """Members with long batches only: dW (and db) reduce over the batch in
    fp32 splits summed by one more launch; ragged widths, one member without
    db beside members with it. Aligned widths (multiples of 8 values) take
    the direct-to-LDS dW tiles in bf16."""
    say(f"[linear bwd split] {dtype} {mode} aligned={aligned}")
    shapes = [(8192, 256, 512), (4096, 104, 72), (6000, 64, 136)] if aligned else \
        [(8192, 256, 512), (4096, 100, 72), (6000, 64, 136)]
    ms = _linear_members(shapes, dtype, seed=525)
    info = _run_linear_bwd(ms, dtype, mode)
    if info is not None:
        assert "_split" in info["kernel"] and info["launches"] == _launches(info), info
        assert ("dma" in _wgrad_part(info)) == (aligned and dtype == "bf16"), info
    _check_linear_bwd(ms, dtype, f"split {dtype} {mode}")
    for m in ms:
        m["db"] = None
    ms2 = _linear_members([(4096, 136, 264), (2500, 40, 8)], dtype, seed=526)   # 2 splits at most
    _run_linear_bwd(ms2, dtype, mode, want=("dx", "dw"))
    _check_linear_bwd(ms2, dtype, f"split, no db {dtype} {mode}", want=("dx", "dw"))


@pytest.mark.parametrize("splits", [1, 2, 3, 5, 7])
def test_linear_backward_pinned_split_counts(splits):
    """dW on the direct-to-LDS tiles with the batch split 1..7 ways (pinned),
    ragged batches so that the last split is shorter, db from the split row
    sums; the same results for every count."""
    say(f"[linear bwd splits={splits}]")
    ms = _linear_members([(5000, 256, 264), (3001, 64, 520)], "bf16", seed=600)
    info = _run_linear_bwd(ms, "bf16", "grouped", splits=splits)
    assert ("_split%d" % splits in info["kernel"]) == (splits > 1) and "dma" in _wgrad_part(info), info
    _check_linear_bwd(ms, "bf16", f"splits {splits}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("variant", [4, 5])
def test_direct_to_lds_backward_every_element_multi_tile(variant):
    """The backward's direct-to-LDS instances (dX reading W as it lies, dW
    with both operands reduction-major) with at least two tiles per
    persistent workgroup: a group of long batches and narrow outputs gives dX
    many tiles, a group of wide weights and a short batch gives dW many
    (its split pinned to 1, so every tile runs the plain epilogue); ragged
    batches; every element of dX, dW and db against the oracle."""
    say(f"[linear bwd dma multi-tile] variant {variant}")
    e = 1024 if variant == 4 else 512
    groups = {"dX": [(4096, 64, e)] * 7 + [(4000, 72, e - 8)],
              "dW": [(136, e, 1024)] * 31 + [(130, e - 8, 1016)]}
    for what, shapes in groups.items():
        ms = _linear_members(shapes, "bf16", seed=540 + variant + (1 if what == "dW" else 0))
        info = _run_linear_bwd(ms, "bf16", "grouped", variant=variant, splits=1)
        assert "_dgrad_direct" in info["kernel"] and "dma" in _wgrad_part(info), info
        _check_linear_bwd(ms, "bf16", f"variant {variant} multi-tile {what}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_linear_backward_strided_and_partial(dtype):
    """Row strides above the row lengths everywhere (the 16-byte paths), then
    only dX, only dW + db, dW without db."""
    say(f"[linear bwd strided] {dtype}")
    ms = _linear_members([(600, 128, 192), (77, 40, 56)], dtype, seed=520, pad=8)
    _run_linear_bwd(ms, dtype, "grouped", pad=8)
    _check_linear_bwd(ms, dtype, "strided")
    for want in [("dx",), ("dw", "db"), ("dw",)]:
        ms = _linear_members([(333, 64, 128), (65, 200, 8)], dtype, seed=521)
        _run_linear_bwd(ms, dtype, "grouped", want=want)
        _check_linear_bwd(ms, dtype, f"only {want}", want=want)


def test_linear_backward_unaligned():
    """A member starting one value off 16-byte alignment: every operand takes
    the per-value loads."""
    say("[linear bwd unaligned]")
    ms = _linear_members([(300, 72, 40)], "bf16", seed=530)
    g = synth.rng(531)
    for key, shape in [("x", (300, 40)), ("w", (72, 40)), ("dy", (300, 72))]:
        t, t64 = _t(g.standard_normal(shape) / (np.sqrt(40) if key == "w" else 1), "bf16", pad=3, off=1)
        ms[0][key], ms[0][key + "64"] = t, t64
    _run_linear_bwd(ms, "bf16", "grouped")
    _check_linear_bwd(ms, "bf16", "unaligned")


# ------------------------------------------------------------------ activation
@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_act_backward(act, dtype):
    say(f"[act bwd] {act} {dtype}")
    g = synth.rng(540)
    shapes = [(1000, 256), (300, 520), (17, 8), (64, 37)]
    xs, dys, refs = [], [], []
    for r, c in shapes:
        x, x64 = _t(g.standard_normal((r, c)) * 3, dtype)
        dy, dy64 = _t(g.standard_normal((r, c)), dtype)
        xs.append(x); dys.append(dy); refs.append(ORC.act_backward(x64, dy64, act))
    dxs = [_empty(x.shape, dtype) for x in xs]
    B.optimus_grouped_act_backward(xs, dys, dxs, act)
    for i, (dx, ref) in enumerate(zip(dxs, refs)):
        assert_close(host64(dx), ref, dtype, f"act {act} member {i}")
    # plan, chain, and in place (dx == dy)
    p = B.optimus_plan_act_backward(xs, dys, dys, act)
    p.execute("chain")
    torch.cuda.synchronize()
    p.close()
    for i, (dy, ref) in enumerate(zip(dys, refs)):
        assert_close(host64(dy), ref, dtype, f"act {act} in place member {i}")


# ------------------------------------------------------------------ LayerNorm
def _ln_members(shapes, dtype, seed, gamma=True, pad=0, off=0):
    g = synth.rng(seed)
    ms = []
    for r, c in shapes:
        x, x64 = _t(g.standard_normal((r, c)) * 2 + 0.5, dtype, pad, off)
        dy, dy64 = _t(g.standard_normal((r, c)), dtype, pad, off)
        gm, gm64 = _t(g.uniform(0.5, 1.5, (1, c)), dtype) if gamma else (None, None)
        ms.append({"x": x, "dy": dy, "x64": x64, "dy64": dy64, "gamma": None if gm is None else gm[0],
                   "g64": None if gm64 is None else gm64[0], "rows": r, "cols": c})
    return ms


def _run_ln_bwd(ms, dtype, mode="oneshot", params=True, inplace=False, eps=1e-5):
    for m in ms:
        m["dx"] = m["dy"] if inplace else _empty((m["rows"], m["cols"]), dtype)
        m["dg"] = torch.full((m["cols"],), float("nan"), dtype=synth.DTYPES[dtype], device="cuda") if params else None
        m["db"] = torch.full((m["cols"],), float("nan"), dtype=synth.DTYPES[dtype], device="cuda") if params else None
    args = ([m["x"] for m in ms], [m["dy"] for m in ms], [m["dx"] for m in ms], [m["gamma"] for m in ms],
            [m["dg"] for m in ms], [m["db"] for m in ms], eps)
    if mode == "oneshot":
        B.optimus_grouped_layernorm_backward(*args)
    else:
        p = B.optimus_plan_layernorm_backward(*args)
        info = p.info()
        assert info["kind"] == 8 and info["launches"] == (2 if params else 1)
        p.execute(mode)
        if not inplace:
            p.execute(mode)   # a second run over the same partial buffer (in place, dy is gone)
        torch.cuda.synchronize()
        p.close()
    torch.cuda.synchronize()


def _check_ln_bwd(ms, dtype, what, params=True, eps=1e-5):
    for i, m in enumerate(ms):
        rdx, rdg, rdb = ORC.layernorm_backward(m["x64"], m["g64"], m["dy64"], eps)
        assert_close(host64(m["dx"]), rdx, dtype, f"{what} member {i} dx")
        if params:
            assert_close(host64(m["dg"][None, :])[0], rdg, dtype, f"{what} member {i} dgamma")
            assert_close(host64(m["db"][None, :])[0], rdb, dtype, f"{what} member {i} dbeta")


LN_SHAPES = [(1000, 256), (300, 520), (4097, 24), (64, 1024), (3, 2000), (50, 37)]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("mode", ["oneshot", "grouped", "chain"])
def test_layernorm_backward(dtype, mode):
    """Rows held in registers (up to 1024 bf16 / 512 fp32 values) and wider or
    odd rows on the per-value path, in one group."""
    say(f"[ln bwd] {dtype} {mode}")
    ms = _ln_members(LN_SHAPES, dtype, seed=550)
    _run_ln_bwd(ms, dtype, mode)
    _check_ln_bwd(ms, dtype, f"{dtype} {mode}")


@pytest.mark.parametrize("act", ["none", "tanh"])
def test_layernorm_backward_bitwise_repeatable(act):
    """dgamma / dbeta are summed in a fixed order (per-wave slots added in
    wave order, then the partial rows in row order): repeated executes of one
    plan give bit-identical gradients, with and without the fused activation
    backward; the first execute against the oracle."""
    say(f"[ln bwd repeatable] {act}")
    ms = _ln_members([(4000, 256), (2000, 1024), (3000, 136)], "bf16", seed=560)
    for m in ms:
        m["dx"] = _empty((m["rows"], m["cols"]), "bf16")
        m["dg"] = torch.full((m["cols"],), float("nan"), dtype=torch.bfloat16, device="cuda")
        m["db"] = torch.full((m["cols"],), float("nan"), dtype=torch.bfloat16, device="cuda")
    args = ([m["x"] for m in ms], [m["dy"] for m in ms], [m["dx"] for m in ms], [m["gamma"] for m in ms])
    if act == "none":
        p = B.optimus_plan_layernorm_backward(*args, [m["dg"] for m in ms], [m["db"] for m in ms], 1e-5)
    else:
        betas = [torch.zeros_like(m["gamma"]) for m in ms]
        p = B.optimus_plan_layernorm_act_backward(*args, betas, [m["dg"] for m in ms], [m["db"] for m in ms],
                                                  1e-5, act)
    p.execute()
    torch.cuda.synchronize()
    first = [(m["dx"].clone(), m["dg"].clone(), m["db"].clone()) for m in ms]
    if act == "none":
        _check_ln_bwd(ms, "bf16", "repeatable")
    for _ in range(4):
        for m in ms:
            m["dg"].fill_(float("nan"))
            m["db"].fill_(float("nan"))
        p.execute()
        torch.cuda.synchronize()
        for m, (dx, dg, db) in zip(ms, first):
            assert torch.equal(m["dx"], dx) and torch.equal(m["dg"], dg) and torch.equal(m["db"], db)
    p.close()


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_layernorm_backward_variants(dtype):
    """No gamma, no dgamma/dbeta, in place (dx == dy), strided and unaligned rows, eps 0.5."""
    say(f"[ln bwd variants] {dtype}")
    ms = _ln_members(LN_SHAPES[:3], dtype, seed=560, gamma=False)
    _run_ln_bwd(ms, dtype, "grouped", eps=0.5)
    _check_ln_bwd(ms, dtype, "no gamma", eps=0.5)
    ms = _ln_members(LN_SHAPES[:3], dtype, seed=561)
    _run_ln_bwd(ms, dtype, "grouped", params=False, inplace=True)
    _check_ln_bwd(ms, dtype, "in place, no params", params=False)
    ms = _ln_members([(500, 256), (77, 128)], dtype, seed=562, pad=8)
    _run_ln_bwd(ms, dtype, "grouped")
    _check_ln_bwd(ms, dtype, "strided")
    ms = _ln_members([(500, 256), (77, 128)], dtype, seed=563, pad=3, off=1)
    _run_ln_bwd(ms, dtype, "grouped")
    _check_ln_bwd(ms, dtype, "unaligned")


# ------------------------------------------------------------------ fused dX activation backward
@pytest.mark.parametrize("act", ["relu", "tanh", "silu"])
@pytest.mark.parametrize("mode", ["oneshot", "grouped", "chain"])
@pytest.mark.parametrize("aligned", [True, False])
def test_linear_act_backward(act, mode, aligned):
    _linear_act_backward_case(act, mode, aligned, "bf16")


@pytest.mark.parametrize("act", ["sigmoid", "silu"])
@pytest.mark.parametrize("mode", ["grouped", "chain"])
def test_linear_act_backward_fp32(act, mode):
    """fp32 groups never take the direct-to-LDS dX: the plan adds the grouped
    activation-backward launch over dX."""
    _linear_act_backward_case(act, mode, False, "fp32")


def _linear_act_backward_case(act, mode, aligned, dtype):
    """dX with the activation backward of the layer below fused in: the
    input gradient times act'(a), a the activation's input [M][K]; against
    the oracle's Linear backward then activation backward. Aligned groups
    fuse it into the dX epilogue, others add one activation-backward launch."""
    say(f"[linear+act bwd] {act} {mode} aligned={aligned} {dtype}")
    shapes = [(700, 296, 264), (129, 64, 32), (257, 8, 520)] if aligned else [(300, 200, 136), (64, 17, 40)]
    ms = _linear_members(shapes, dtype, seed=590)
    g = synth.rng(591)
    acts = [_t(g.standard_normal((m["M"], m["K"])), dtype) for m in ms]
    for m in ms:
        m["dx"] = _empty((m["M"], m["K"]), dtype)
        m["dw"] = _empty((m["N"], m["K"]), dtype)
        m["db"] = torch.full((m["N"],), float("nan"), dtype=synth.DTYPES[dtype], device="cuda")
    args = ([m["x"] for m in ms], [m["w"] for m in ms], [m["dy"] for m in ms], [m["dx"] for m in ms],
            [m["dw"] for m in ms], [m["db"] for m in ms], [a[0] for a in acts], act)
    if mode == "oneshot":
        B.optimus_grouped_linear_act_backward(*args)
    else:
        p = B.optimus_plan_linear_act_backward(*args)
        info = p.info()
        n = _launches(info) + (0 if aligned else 1)
        assert ("_dgrad_direct_" + act in info["kernel"]) == aligned and info["launches"] == n, info
        p.execute(mode)
        torch.cuda.synchronize()
        p.close()
    torch.cuda.synchronize()
    for i, m in enumerate(ms):
        rdx, rdw, rdb = ORC.linear_backward(m["x64"], m["w64"], m["dy64"])
        assert_close(host64(m["dx"]), ORC.act_backward(acts[i][1], rdx, act), dtype, f"{act} member {i} dx")
        assert_close(host64(m["dw"]), rdw, dtype, f"{act} member {i} dw")
        assert_close(host64(m["db"][None, :])[0], rdb, dtype, f"{act} member {i} db")


def test_linear_act_backward_unaligned_activation_input():
    """Aligned dY / W / dX with the activation input starting one value off
    16-byte alignment (and a padded row stride): the fused epilogue's
    per-value path."""
    say("[linear+act bwd unaligned a]")
    ms = _linear_members([(700, 296, 264), (129, 64, 32)], "bf16", seed=595)
    g = synth.rng(596)
    acts = [_t(g.standard_normal((m["M"], m["K"])), "bf16", pad=3, off=1) for m in ms]
    for m in ms:
        m["dx"] = _empty((m["M"], m["K"]), "bf16")
    p = B.optimus_plan_linear_act_backward([m["x"] for m in ms], [m["w"] for m in ms], [m["dy"] for m in ms],
                                           [m["dx"] for m in ms], None, None, [a[0] for a in acts], "silu")
    assert "_dgrad_direct_silu" in p.info()["kernel"], p.info()
    p.execute("grouped")
    torch.cuda.synchronize()
    p.close()
    for i, m in enumerate(ms):
        rdx = ORC.linear_backward(m["x64"], m["w64"], m["dy64"])[0]
        assert_close(host64(m["dx"]), ORC.act_backward(acts[i][1], rdx, "silu"), "bf16", f"member {i} dx")


@pytest.mark.parametrize("dtype,aligned", [("fp32", False), ("bf16", False), ("bf16", True)])
@pytest.mark.parametrize("mode", ["oneshot", "grouped", "chain"])
def test_linear_act_backward_in_place(dtype, aligned, mode):
    """act_x is the member's dx itself (the activation input is overwritten by
    its gradient): fp32 and unaligned bf16 groups compute dY W into plan
    scratch before the activation backward reads it beside act_x; aligned
    bf16 groups read act_x in the dX epilogue. Against the oracle's Linear
    backward then activation backward on the original activation input."""
    say(f"[linear+act bwd in place] {dtype} aligned={aligned} {mode}")
    shapes = [(700, 296, 264), (129, 64, 32)] if aligned else [(300, 200, 136), (64, 17, 40), (513, 33, 9)]
    ms = _linear_members(shapes, dtype, seed=597)
    g = synth.rng(598)
    acts = [_t(g.standard_normal((m["M"], m["K"])), dtype) for m in ms]
    for m, a in zip(ms, acts):
        m["dx"] = a[0]  # the activation input's storage receives dL/da
        m["dw"] = _empty((m["N"], m["K"]), dtype)
    args = ([m["x"] for m in ms], [m["w"] for m in ms], [m["dy"] for m in ms], [m["dx"] for m in ms],
            [m["dw"] for m in ms], None, [m["dx"] for m in ms], "tanh")
    if mode == "oneshot":
        B.optimus_grouped_linear_act_backward(*args)
    else:
        p = B.optimus_plan_linear_act_backward(*args)
        assert ("_dgrad_direct_tanh" in p.info()["kernel"]) == aligned, p.info()
        p.execute(mode)
        torch.cuda.synchronize()
        p.close()
    torch.cuda.synchronize()
    for i, m in enumerate(ms):
        rdx, rdw, _ = ORC.linear_backward(m["x64"], m["w64"], m["dy64"])
        assert_close(host64(m["dx"]), ORC.act_backward(acts[i][1], rdx, "tanh"), dtype, f"member {i} dx in place")
        assert_close(host64(m["dw"]), rdw, dtype, f"member {i} dw")


# ------------------------------------------------------------------ fused LayerNorm + activation
def _ref_ln_act_bwd(m, beta64, act, eps):
    """The oracle composition: the activation's input z = LayerNorm(x) (fp64,
    from the stored x), dz = dout * act'(z), then the LayerNorm backward."""
    z = ORC.layernorm(m["x64"], m["g64"], beta64, eps)
    dz = ORC.act_backward(z, m["dy64"], act)
    return ORC.layernorm_backward(m["x64"], m["g64"], dz, eps)


@pytest.mark.parametrize("act", ACTS)
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("mode", ["oneshot", "grouped", "chain"])
def test_layernorm_act_backward(act, dtype, mode):
    """Backward of LayerNorm + activation in one pass (the activation's input
    recomputed from x) against the oracle's activation backward then
    LayerNorm backward; register and per-value rows, one member without beta."""
    say(f"[ln+act bwd] {act} {dtype} {mode}")
    eps = 1e-5
    ms = _ln_members(LN_SHAPES, dtype, seed=580)
    g = synth.rng(581)
    betas, b64s = [], []
    for i, m in enumerate(ms):
        if i == 2:
            betas.append(None); b64s.append(None)
            continue
        b, b64 = _t(g.normal(0.0, 0.3, (1, m["cols"])), dtype)
        betas.append(b[0]); b64s.append(b64[0])
    for m in ms:
        m["dx"] = _empty((m["rows"], m["cols"]), dtype)
        m["dg"] = torch.full((m["cols"],), float("nan"), dtype=synth.DTYPES[dtype], device="cuda")
        m["db"] = torch.full((m["cols"],), float("nan"), dtype=synth.DTYPES[dtype], device="cuda")
    args = ([m["x"] for m in ms], [m["dy"] for m in ms], [m["dx"] for m in ms], [m["gamma"] for m in ms], betas,
            [m["dg"] for m in ms], [m["db"] for m in ms], eps, act)
    if mode == "oneshot":
        B.optimus_grouped_layernorm_act_backward(*args)
    else:
        p = B.optimus_plan_layernorm_act_backward(*args)
        info = p.info()
        assert info["kind"] == 8 and info["launches"] == 2 and (act == "none") == ("_" + act not in info["kernel"])
        p.execute(mode)
        p.execute(mode)
        torch.cuda.synchronize()
        p.close()
    torch.cuda.synchronize()
    for i, m in enumerate(ms):
        rdx, rdg, rdb = _ref_ln_act_bwd(m, b64s[i], act, eps)
        assert_close(host64(m["dx"]), rdx, dtype, f"{act} member {i} dx")
        assert_close(host64(m["dg"][None, :])[0], rdg, dtype, f"{act} member {i} dgamma")
        assert_close(host64(m["db"][None, :])[0], rdb, dtype, f"{act} member {i} dbeta")


def test_layernorm_act_backward_in_place_no_params():
    """dx over dy (one pass reads the whole row first), no dgamma / dbeta, no gamma."""
    say("[ln+act bwd in place]")
    ms = _ln_members(LN_SHAPES[:3], "bf16", seed=585, gamma=False)
    refs = [_ref_ln_act_bwd(m, None, "silu", 1e-5)[0] for m in ms]
    B.optimus_grouped_layernorm_act_backward([m["x"] for m in ms], [m["dy"] for m in ms], [m["dy"] for m in ms],
                                             None, None, None, None, 1e-5, "silu")
    torch.cuda.synchronize()
    for i, m in enumerate(ms):
        assert_close(host64(m["dy"]), refs[i], "bf16", f"in place member {i} dx")


# ------------------------------------------------------------------ a training step's backward
def test_towers_backward_chain_of_groups():
    """The towers group's backward (LayerNorm, layer 2, relu, layer 1) as
    grouped launches, against the fp64 oracle composition fed the same
    stored intermediates: each operator per member within the bf16 bound."""
    say("[towers bwd]")
    wl = synth.towers(seed=3, G=6, M=512)
    g = synth.rng(570)
    T = wl.towers
    # forward intermediates from the oracle (stored in bf16 as the forward would)
    h_pre, h, o = [], [], []
    for t in T:
        hp = ORC.linear(synth.exact64(t.x), synth.exact64(t.w1), synth.exact64(t.b1))
        hp_t, hp64 = _t(hp, "bf16")
        h_t, h64 = _t(np.maximum(hp64, 0.0), "bf16")
        o_t, o64 = _t(ORC.linear(h64, synth.exact64(t.w2), synth.exact64(t.b2)), "bf16")
        h_pre.append((hp_t, hp64)); h.append((h_t, h64)); o.append((o_t, o64))
    dz = [_t(g.standard_normal((512, 256)), "bf16") for _ in T]
    gm = [dev(t.gamma) for t in T]
    # LayerNorm backward
    do = [_empty((512, 256), "bf16") for _ in T]
    dgm = [torch.empty(256, dtype=torch.bfloat16, device="cuda") for _ in T]
    dbt = [torch.empty(256, dtype=torch.bfloat16, device="cuda") for _ in T]
    B.optimus_grouped_layernorm_backward([v[0] for v in o], [v[0] for v in dz], do, gm, dgm, dbt, wl.eps)
    # layer 2 backward
    dh = [_empty((512, 512), "bf16") for _ in T]
    dw2 = [_empty((256, 512), "bf16") for _ in T]
    db2 = [torch.empty(256, dtype=torch.bfloat16, device="cuda") for _ in T]
    B.optimus_grouped_linear_backward([v[0] for v in h], [dev(t.w2) for t in T], do, dh, dw2, db2)
    # relu backward (in place) and layer 1 backward
    B.optimus_grouped_act_backward([v[0] for v in h_pre], dh, dh, "relu")
    dw1 = [_empty((512, t.x.shape[1]), "bf16") for t in T]
    db1 = [torch.empty(512, dtype=torch.bfloat16, device="cuda") for _ in T]
    B.optimus_grouped_linear_backward([dev(t.x) for t in T], [dev(t.w1) for t in T], dh, None, dw1, db1)
    torch.cuda.synchronize()
    for i, t in enumerate(T):
        r_do, r_dg, r_db = ORC.layernorm_backward(o[i][1], synth.exact64(t.gamma), dz[i][1], wl.eps)
        assert_close(host64(do[i]), r_do, "bf16", f"tower {i} d(layer 2 out)")
        assert_close(host64(dgm[i][None, :])[0], r_dg, "bf16", f"tower {i} dgamma")
        do64 = host64(do[i])
        r_dh, r_dw2, r_db2 = ORC.linear_backward(h[i][1], synth.exact64(t.w2), do64)
        assert_close(host64(dw2[i]), r_dw2, "bf16", f"tower {i} dW2")
        assert_close(host64(db2[i][None, :])[0], r_db2, "bf16", f"tower {i} db2")
        dh64 = host64(dh[i])   # after the in-place relu backward
        r_dhp = ORC.act_backward(h_pre[i][1], synth.exact64(synth.to_storage(r_dh, "bf16")), "relu")
        assert_close(dh64, r_dhp, "bf16", f"tower {i} d(layer 1 out)")
        _, r_dw1, r_db1 = ORC.linear_backward(synth.exact64(t.x), synth.exact64(t.w1), dh64)
        assert_close(host64(dw1[i]), r_dw1, "bf16", f"tower {i} dW1")
        assert_close(host64(db1[i][None, :])[0], r_db1, "bf16", f"tower {i} db1")


# ------------------------------------------------------------------ full-size backward op-groups
def _dw_sampled(x64, w64, dy64, ns):
    """dW rows ns and db[ns] of a whole batch: the oracle on dY's columns ns."""
    _, dw_s, db_s = ORC.linear_backward(x64, w64[ns], np.ascontiguousarray(dy64[:, ns]))
    return dw_s, db_s


def _sample(n, k, seed, block=256):
    """k random rows of n, both edge rows, and one random row of every
    `block`-row block (every M-block of the GEMM tiles)."""
    g = synth.rng(seed)
    per_block = [b + g.integers(0, min(block, n - b)) for b in range(0, n, block)]
    return np.unique(np.concatenate([[0, n - 1], per_block, g.choice(n, size=min(n, k), replace=False)])).astype(np.int64)


@pytest.mark.timeout(300)
def test_large_group_backward_full_size_sampled():
    """large_group's training backward at full size (32 members, batch 16384,
    K = 1024, N in {256, 512, 1024}) as the benchmark runs it: the LayerNorm +
    tanh backward in one pass, then the Linear backward. Per operator, the
    oracle is fed the GPU's stored inputs: the tanh input recomputed in fp64
    from y, then tanh and LayerNorm backward (dX on sampled rows, dgamma /
    dbeta over every row); the Linear's dX on sampled rows, dW / db on
    sampled output rows over the whole batch."""
    say("[large_group bwd] G=32 B=16384 K=1024 bf16")
    wl = synth.large_group(0)
    ms = wl.members
    bf = torch.bfloat16
    xs, ws, bs = [dev(m.x) for m in ms], [dev(m.w) for m in ms], [dev(m.b) for m in ms]
    gs, bes = [dev(g) for g in wl.gammas], [dev(b) for b in wl.betas]
    y = [torch.empty((m.M, m.N), dtype=bf, device="cuda") for m in ms]
    B.optimus_plan_linear(xs, ws, bs, y, "none").execute()
    gen = torch.Generator(device="cuda").manual_seed(2)
    dt_ = [torch.randn(v.shape, generator=gen, device="cuda").to(bf) for v in y]
    dy = [torch.empty_like(v) for v in y]
    dx, dw, db = [torch.empty_like(x) for x in xs], [torch.empty_like(w) for w in ws], [torch.empty_like(b) for b in bs]
    dgm, dbt = [torch.empty_like(g) for g in gs], [torch.empty_like(g) for g in gs]
    torch.cuda.synchronize()
    plans = [B.optimus_plan_layernorm_act_backward(y, dt_, dy, gs, bes, dgm, dbt, wl.eps, "tanh"),
             B.optimus_plan_linear_backward(xs, ws, dy, dx, dw, db)]
    lin_info = plans[1].info()
    say(f"  linear backward plan: {lin_info['kernel']} launches={lin_info['launches']}")
    for p in plans:
        p.execute("grouped")
    torch.cuda.synchronize()
    rows = _sample(16384, 40, seed=63)
    for i, m in enumerate(ms):
        say(f"  member {i} N={m.N}")
        y64, dt64 = host64(y[i]), host64(dt_[i])
        g64, b64 = synth.exact64(wl.gammas[i]), synth.exact64(wl.betas[i])
        dz64 = ORC.act_backward(ORC.layernorm(y64, g64, b64, wl.eps), dt64, "tanh")
        r_dy, r_dg, r_db = ORC.layernorm_backward(y64, g64, dz64, wl.eps)
        dy64 = host64(dy[i])
        assert_close(dy64[rows], r_dy[rows], "bf16", f"member {i} LayerNorm dX")
        assert_close(host64(dgm[i][None, :])[0], r_dg, "bf16", f"member {i} dgamma")
        assert_close(host64(dbt[i][None, :])[0], r_db, "bf16", f"member {i} dbeta")
        x64, w64 = synth.exact64(m.x), synth.exact64(m.w)
        r_dx = ORC.linear_backward(x64[rows], w64, dy64[rows])[0]
        assert_close(host64(dx[i])[rows], r_dx, "bf16", f"member {i} dX")
        ns = _sample(m.N, 6, seed=64 + i)
        r_dw, r_dbs = _dw_sampled(x64, w64, dy64, ns)
        assert_close(host64(dw[i])[ns], r_dw, "bf16", f"member {i} dW rows")
        assert_close(host64(db[i][None, :])[0][ns], r_dbs, "bf16", f"member {i} db")


@pytest.mark.timeout(300)
def test_towers_backward_full_size_sampled():
    """The towers group's training backward at full size (26 towers, batch
    4096) as the benchmark runs it: LayerNorm backward, layer 2 backward with
    the relu backward fused into its dX, layer 1 backward; per operator
    against the oracle fed the GPU's stored inputs, on sampled rows (dW / db:
    sampled output rows over the whole batch; dgamma: every row)."""
    say("[towers bwd] 26 towers B=4096 bf16")
    wl = synth.towers(0)
    T = wl.towers
    bf = torch.bfloat16
    xs = [dev(t.x) for t in T]
    w1, b1, w2, b2 = ([dev(getattr(t, a)) for t in T] for a in ("w1", "b1", "w2", "b2"))
    gm = [dev(t.gamma) for t in T]
    hp = [torch.empty((4096, 512), dtype=bf, device="cuda") for _ in T]
    h = [torch.empty_like(v) for v in hp]
    o = [torch.empty((4096, 256), dtype=bf, device="cuda") for _ in T]
    B.optimus_plan_linear(xs, w1, b1, hp, "none").execute()
    B.optimus_plan_pointwise(hp, h, "relu").execute()
    B.optimus_plan_linear(h, w2, b2, o, "none").execute()
    gen = torch.Generator(device="cuda").manual_seed(1)
    dz = [torch.randn(v.shape, generator=gen, device="cuda").to(bf) for v in o]
    do, dh = [torch.empty_like(v) for v in o], [torch.empty_like(v) for v in h]
    dx = [torch.empty_like(x) for x in xs]
    dw1, dw2 = [torch.empty_like(w) for w in w1], [torch.empty_like(w) for w in w2]
    db1, db2 = [torch.empty_like(b) for b in b1], [torch.empty_like(b) for b in b2]
    dgm, dbt = [torch.empty_like(g) for g in gm], [torch.empty_like(g) for g in gm]
    torch.cuda.synchronize()
    ln_b = B.optimus_plan_layernorm_backward(o, dz, do, gm, dgm, dbt, wl.eps)
    l2_b = B.optimus_plan_linear_act_backward(h, w2, do, dh, dw2, db2, hp, "relu")   # dX leaves as d(hp)
    l1_b = B.optimus_plan_linear_backward(xs, w1, dh, dx, dw1, db1)
    say(f"  layer 2: {l2_b.info()['kernel']}; layer 1: {l1_b.info()['kernel']}")
    for p in (ln_b, l2_b, l1_b):
        p.execute("grouped")
    torch.cuda.synchronize()
    rows = _sample(4096, 48, seed=65)
    for i, t in enumerate(T):
        o64, dz64 = host64(o[i]), host64(dz[i])
        r_do, r_dg, r_dbt = ORC.layernorm_backward(o64, synth.exact64(t.gamma), dz64, wl.eps)
        do64 = host64(do[i])
        assert_close(do64[rows], r_do[rows], "bf16", f"tower {i} LayerNorm dX")
        assert_close(host64(dgm[i][None, :])[0], r_dg, "bf16", f"tower {i} dgamma")
        assert_close(host64(dbt[i][None, :])[0], r_dbt, "bf16", f"tower {i} dbeta")
        h64, w2_64 = host64(h[i]), synth.exact64(t.w2)
        ns = _sample(256, 6, seed=66 + i)
        r_dw2, r_db2 = _dw_sampled(h64, w2_64, do64, ns)
        assert_close(host64(dw2[i])[ns], r_dw2, "bf16", f"tower {i} dW2 rows")
        assert_close(host64(db2[i][None, :])[0][ns], r_db2, "bf16", f"tower {i} db2")
        dhp64 = host64(dh[i])
        r_dh = ORC.linear_backward(h64[rows], w2_64, do64[rows])[0]
        assert_close(dhp64[rows], ORC.act_backward(host64(hp[i])[rows], r_dh, "relu"), "bf16",
                     f"tower {i} layer-2 dX with the relu backward")
        x64, w1_64 = synth.exact64(t.x), synth.exact64(t.w1)
        assert_close(host64(dx[i])[rows], ORC.linear_backward(x64[rows], w1_64, dhp64[rows])[0], "bf16",
                     f"tower {i} dX")
        ns = _sample(512, 6, seed=92 + i)
        r_dw1, r_db1 = _dw_sampled(x64, w1_64, dhp64, ns)
        assert_close(host64(dw1[i])[ns], r_dw1, "bf16", f"tower {i} dW1 rows")
        assert_close(host64(db1[i][None, :])[0][ns], r_db1, "bf16", f"tower {i} db1")
