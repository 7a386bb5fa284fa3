"""Grouped Linear with the row LayerNorm fused into the GEMM epilogue, on the
GPU against the fp64 oracle composition (through the C ABI)."""

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


def _members(shapes, dtype, seed, params=True, bias=True):
    """Linear members plus per-member gamma ~ U(0.5, 1.5), beta ~ N(0, 0.1)."""
    g = synth.rng(seed)
    ms = []
    for M, N, K in shapes:
        x = dev(synth.to_storage(g.standard_normal((M, K)), dtype))
        w = dev(synth.to_storage(g.standard_normal((N, K)) / np.sqrt(K), dtype))
        b = dev(synth.to_storage(g.standard_normal(N) * 0.3, dtype)) if bias else None
        gm = dev(synth.to_storage(g.uniform(0.5, 1.5, N), dtype)) if params else None
        be = dev(synth.to_storage(g.standard_normal(N) * 0.1, dtype)) if params else None
        ms.append((x, w, b, gm, be))
    return ms


def _run(ms, act, eps=1e-5, mode="oneshot", variant=None):
    """The one-shot call, or a plan executed in `mode`; a pinned tile variant
    (kernel-table index) goes through the plan options."""
    xs, ws, bs = [m[0] for m in ms], [m[1] for m in ms], [m[2] for m in ms]
    gs, es = [m[3] for m in ms], [m[4] for m in ms]
    ys = [torch.full((x.shape[0], w.shape[0]), float("nan"), dtype=x.dtype, device="cuda") for x, w, *_ in ms]
    if mode == "oneshot" and variant is None:
        B.optimus_grouped_linear_layernorm(xs, ws, bs, ys, gs, es, eps, act)
        kernel = None
    else:
        opts = None if variant is None else {"gemm_tile": variant + 1}
        p = B.optimus_plan_linear_layernorm_ex(xs, ws, bs, ys, gs, es, eps, act, options=opts)
        kernel = p.info()["kernel"]
        assert p.info()["kind"] == 4
        p.execute("grouped" if mode == "oneshot" else mode)
        torch.cuda.synchronize()
        p.close()
    return ys, kernel


def _check(ms, ys, dtype, act, what, eps=1e-5):
    for i, ((x, w, b, gm, be), y) in enumerate(zip(ms, ys)):
        ref = ORC.linear_layernorm(host64(x), host64(w), None if b is None else host64(b),
                                   None if gm is None else host64(gm), None if be is None else host64(be), eps, act)
        assert_close(host64(y), ref, dtype, f"{what} member {i}")


# (shapes, dtype, the kernel the planner is expected to pick)
CASES = {
    "bf16_rows_256_dma": ([(1000, 256, 512), (300, 256, 64), (513, 200, 136)], "bf16", "grouped_gemm_dma_bf16_256x256"),
    "bf16_rows_128_dma": ([(700, 128, 96), (257, 100, 64), (64, 17, 32)], "bf16", "grouped_gemm_dma_bf16_128x128"),
    "bf16_rows_64_one_step": ([(900, 64, 64), (130, 48, 16), (33, 16, 40)], "bf16", "grouped_gemm_bf16_128x64"),
    "bf16_unaligned_k": ([(400, 256, 100), (77, 250, 13)], "bf16", "grouped_gemm_bf16_256x256"),
    "bf16_unaligned_k_128": ([(400, 128, 100), (77, 90, 13)], "bf16", "grouped_gemm_bf16_128x128"),
    "fp32_rows_64": ([(8192, 64, 64), (4096, 64, 256), (100, 33, 40)], "fp32", "grouped_gemm_f32_64x64"),
    "fp32_rows_64_few_tiles": ([(512, 64, 64), (512, 64, 256), (100, 33, 40)], "fp32", "grouped_gemm_rows16_f32_16x128"),
    "fp32_rows_128_few_tiles": ([(512, 128, 128), (512, 64, 256), (150, 100, 24)], "fp32", "grouped_gemm_rows16_f32_16x128"),
    "fp32_rows_128": ([(8192, 128, 128), (8192, 64, 72), (150, 100, 24)], "fp32", "grouped_gemm_f32_64x128"),
}


@pytest.mark.parametrize("case", list(CASES))
@pytest.mark.parametrize("act", ["none", "tanh"])
def test_default_pick(case, act):
    shapes, dtype, kernel = CASES[case]
    say(f"[linear+ln default] {case} {act}")
    ms = _members(shapes, dtype, seed=40 + len(case))
    ys, name = _run(ms, act, mode="grouped")
    assert name.startswith(kernel) and name.endswith("_layernorm"), name
    _check(ms, ys, dtype, act, f"{case} {act}")
    ys, _ = _run(ms, act)
    _check(ms, ys, dtype, act, f"{case} {act} one-shot")


@pytest.mark.parametrize("act", ACTS)
def test_every_activation(act):
    say(f"[linear+ln act] {act}")
    ms = _members([(600, 256, 128), (200, 136, 72)], "bf16", seed=50)
    ys, _ = _run(ms, act, mode="grouped")
    _check(ms, ys, "bf16", act, f"act {act}")


@pytest.mark.parametrize("variant", [0, 1, 2, 4, 5])
def test_every_bf16_variant(variant):
    """Each tile variant that can hold the rows: 0 takes N <= 64 (and one K
    step), 1 and 5 N <= 128, 2 and 4 N <= 256."""
    bn = {0: 64, 1: 128, 2: 256, 4: 256, 5: 128}[variant]
    shapes = [(513, bn, 64 if variant == 0 else 136), (100, bn - 8, 40), (31, 16, 24)]
    say(f"[linear+ln variant] {variant}")
    ms = _members(shapes, "bf16", seed=60 + variant)
    for mode in ["grouped", "chain"]:
        ys, name = _run(ms, "silu", mode=mode, variant=variant)
        assert name.endswith("_layernorm")
        _check(ms, ys, "bf16", "silu", f"variant {variant} {mode}")


def test_no_gamma_beta_no_bias_and_eps():
    say("[linear+ln defaults]")
    ms = _members([(300, 256, 64), (300, 120, 64)], "bf16", seed=70, params=False, bias=False)
    ys, _ = _run(ms, "none", eps=0.25, mode="grouped")
    _check(ms, ys, "bf16", "none", "no gamma/beta/bias, eps 0.25", eps=0.25)


def test_chain_equals_grouped_bitwise():
    say("[linear+ln chain vs grouped]")
    ms = _members([(1000, 256, 512), (300, 200, 64), (64, 8, 16)], "bf16", seed=71)
    a, _ = _run(ms, "tanh", mode="grouped")
    c, _ = _run(ms, "tanh", mode="chain")
    for ya, yc in zip(a, c):
        assert torch.equal(ya, yc)


def test_constant_rows_give_beta():
    """Weights with equal rows and a constant bias make every pre-norm row
    constant: the output is beta up to the rounding of the row mean."""
    say("[linear+ln constant rows]")
    g = synth.rng(72)
    M, N, K = 256, 256, 64
    x = dev(synth.to_storage(g.standard_normal((M, K)), "bf16"))
    w = dev(synth.to_storage(np.broadcast_to(g.standard_normal(K) / 8, (N, K)).copy(), "bf16"))
    b = dev(synth.to_storage(np.full(N, 0.5), "bf16"))
    gm = dev(synth.to_storage(g.uniform(0.5, 1.5, N), "bf16"))
    be = dev(synth.to_storage(np.linspace(-1, 1, N), "bf16"))
    ys, _ = _run([(x, w, b, gm, be)], "none", mode="grouped")
    assert np.max(np.abs(host64(ys[0]) - host64(be)[None, :])) < 2e-2


def test_rows_too_wide_are_rejected():
    say("[linear+ln errors]")
    ms = _members([(64, 300, 32)], "bf16", seed=73)
    ys = [torch.zeros((64, 300), dtype=torch.bfloat16, device="cuda")]
    with pytest.raises(B.OptimusError) as ei:
        B.optimus_grouped_linear_layernorm([ms[0][0]], [ms[0][1]], [ms[0][2]], ys, [ms[0][3]], [ms[0][4]], 1e-5, "none")
    assert ei.value.name == "UNSUPPORTED"
    assert torch.count_nonzero(ys[0]) == 0
    B.optimus_grouped_linear_layernorm([], [], [], [], None, None, 1e-5, "none")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("variant", [4, 5])
def test_direct_to_lds_layernorm_every_element_multi_tile(variant):
    """The fused LayerNorm epilogue on each direct-to-LDS tile with at least
    two tiles per persistent workgroup (whole rows per tile: N <= the tile's
    width), a ragged row count and a narrower member; every element against
    the oracle's fused composition."""
    bn = {4: 256, 5: 128}[variant]
    shapes = [(16384, bn, 64)] * 8 + [(16000, bn - 8, 72), (15000, bn // 2, 136)]
    say(f"[linear+ln dma multi-tile] variant {variant}")
    ms = _members(shapes, "bf16", seed=160 + variant)
    xs, ws, bs = [m[0] for m in ms], [m[1] for m in ms], [m[2] for m in ms]
    gs, es = [m[3] for m in ms], [m[4] for m in ms]
    ys = [torch.full((x.shape[0], w.shape[0]), float("nan"), dtype=x.dtype, device="cuda") for x, w, *_ in ms]
    p = B.optimus_plan_linear_layernorm_ex(xs, ws, bs, ys, gs, es, 1e-5, "tanh", options={"gemm_tile": variant + 1})
    info = p.info()
    assert info["work_items"] >= 2 * info["grid"], info
    p.execute()
    torch.cuda.synchronize()
    p.close()
    _check(ms, ys, "bf16", "tanh", f"variant {variant} multi-tile")


@pytest.mark.parametrize("variant", [3, 6, 8, 10])
def test_every_fp32_variant(variant):
    """The fp32 tiles that can hold the rows (3: 64x64 for N <= 64; 6: 64x128;
    8: 32x128 with its K split over the wave pairs for members of N <= 64;
    10: 16x128 with register-direct operands, the planner's choice for groups
    of fewer 32-row tiles than CUs, its spare waves splitting K for members of
    N <= 64 or <= 32), grouped and chain, ragged rows and K, against the
    oracle's fused composition."""
    bn = {3: 64, 6: 128, 8: 128, 10: 128}[variant]
    shapes = [(513, bn, 136), (100, bn - 4, 40), (31, 16, 24), (257, bn // 2, 260), (300, 60, 200), (90, 33, 130),
              (40, bn - 28, 600)]
    say(f"[linear+ln fp32 variant] {variant}")
    ms = _members(shapes, "fp32", seed=170 + variant)
    for mode in ["grouped", "chain"]:
        ys, name = _run(ms, "tanh", mode=mode, variant=variant)
        assert name.startswith({3: "grouped_gemm_f32_64x64", 6: "grouped_gemm_f32_64x128",
                                8: "grouped_gemm_f32_32x128", 10: "grouped_gemm_rows16_f32_16x128"}[variant]), name
        _check(ms, ys, "fp32", "tanh", f"fp32 variant {variant} {mode}")
