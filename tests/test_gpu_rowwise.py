"""Grouped LayerNorm and grouped pointwise on the GPU against the fp64 oracle."""
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
# (rows, cols): lane-group sizes 1..64, ragged row tails, wide rows on the
# three-pass path, single column
SHAPES = [(33, 16), (129, 64), (300, 256), (17, 1024), (5, 2048), (64, 48), (9, 5000), (40, 1), (3, 520)]


def _ln_members(shapes, dtype, seed, affine=True):
    g = synth.rng(seed)
    out = []
    for r, c in shapes:
        x = dev(synth.to_storage(g.standard_normal((r, c)) * 2 + g.standard_normal((r, 1)), dtype))
        gm = dev(synth.to_storage(g.uniform(0.5, 1.5, c), dtype)) if affine else None
        bt = dev(synth.to_storage(g.standard_normal(c) * 0.3, dtype)) if affine else None
        out.append((x, gm, bt))
    return out


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("act", ACTS)
def test_grouped_layernorm(dtype, act):
    say(f"[layernorm] dtype={dtype} act={act}")
    ms = _ln_members(SHAPES, dtype, seed=20)
    ys = [torch.full_like(x, float("nan")) for x, _, _ in ms]
    B.optimus_grouped_layernorm([m[0] for m in ms], ys, [m[1] for m in ms], [m[2] for m in ms], 1e-5, act)
    for i, ((x, gm, bt), y) in enumerate(zip(ms, ys)):
        ref = ORC.layernorm(host64(x), host64(gm), host64(bt), 1e-5, act)
        assert_close(host64(y), ref, dtype, f"member {i} {x.shape}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_layernorm_plan_modes_and_edge_cases(dtype):
    say(f"[layernorm modes/edges] {dtype}")
    ms = _ln_members(SHAPES[:5], dtype, seed=21, affine=False)
    xs = [m[0] for m in ms]
    ya = [torch.empty_like(x) for x in xs]
    yc = [torch.empty_like(x) for x in xs]
    p = B.optimus_plan_layernorm(xs, ya, None, None, 1e-5, "tanh")
    p.execute("grouped")
    q = B.optimus_plan_layernorm(xs, yc, None, None, 1e-5, "tanh")
    q.execute("chain")
    torch.cuda.synchronize()
    assert p.info()["launches"] == 1 and p.info()["chain_launches"] == len(xs)
    for x, a, c in zip(xs, ya, yc):
        assert torch.equal(a, c)
        assert_close(host64(a), ORC.layernorm(host64(x), None, None, 1e-5, "tanh"), dtype, "plan")
    p.close()
    q.close()
    # constant rows: zero variance -> beta, never NaN
    x = torch.full((64, 256), 0.75, dtype=synth.DTYPES[dtype], device="cuda")
    bt = dev(synth.to_storage(np.linspace(-1, 1, 256), dtype))
    y = torch.empty_like(x)
    B.optimus_grouped_layernorm([x], [y], [None], [bt], 1e-5)
    assert np.array_equal(host64(y), np.broadcast_to(host64(bt), (64, 256)))
    # in place, and an unaligned (odd element offset) view on the per-element path
    ms = _ln_members([(100, 128)], dtype, seed=22)
    x, gm, bt = ms[0]
    ref = ORC.layernorm(host64(x), host64(gm), host64(bt), 1e-5, "silu")
    B.optimus_grouped_layernorm([x], [x], [gm], [bt], 1e-5, "silu")
    assert_close(host64(x), ref, dtype, "in place")
    buf = dev(synth.to_storage(synth.rng(23).standard_normal((50, 131)), dtype))
    xv = buf[:, 1:130]
    y = torch.empty((50, 129), dtype=buf.dtype, device="cuda")
    B.optimus_grouped_layernorm([xv], [y], None, None, 1e-5)
    assert_close(host64(y), ORC.layernorm(host64(xv), None, None, 1e-5), dtype, "unaligned view")


def test_layernorm_invariants_on_gpu():
    """gamma=1, beta=0, fp32: per-row mean ~0 and variance s2/(s2+eps)."""
    say("[layernorm invariants]")
    g = synth.rng(24)
    x = dev(synth.to_storage(g.standard_normal((256, 384)) * g.uniform(0.05, 5, (256, 1)), "fp32"))
    y = torch.empty_like(x)
    B.optimus_grouped_layernorm([x], [y], None, None, 0.1)
    yh, xh = host64(y), host64(x)
    s2 = xh.var(axis=1)
    assert np.max(np.abs(yh.mean(axis=1))) < 1e-5
    assert np.max(np.abs(yh.var(axis=1) - s2 / (s2 + 0.1))) < 1e-5


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("act", ACTS)
def test_grouped_pointwise(dtype, act):
    say(f"[pointwise] dtype={dtype} act={act}")
    g = synth.rng(30)
    xs = [dev(synth.to_storage(g.standard_normal((r, c)) * 4, dtype)) for r, c in SHAPES]
    ys = [torch.full_like(x, float("nan")) for x in xs]
    B.optimus_grouped_pointwise(xs, ys, act)
    for i, (x, y) in enumerate(zip(xs, ys)):
        assert_close(host64(y), ORC.pointwise(host64(x), act), dtype, f"member {i}")
    if act == "relu":  # exact
        for x, y in zip(xs, ys):
            assert np.array_equal(host64(y), np.maximum(host64(x), 0))
    if act == "none":
        for x, y in zip(xs, ys):
            assert torch.equal(x, y)


def test_pointwise_saturation_and_special_values():
    say("[pointwise saturation]")
    v = torch.tensor([[-1e4, -100.0, -30.0, -1.0, -0.0, 0.0, 1.0, 30.0, 100.0, 1e4, 0.5, -0.5, 2.0, -2.0, 7.0, -7.0]],
                     dtype=torch.float32, device="cuda")
    for act in ["sigmoid", "tanh", "silu"]:
        y = torch.empty_like(v)
        B.optimus_grouped_pointwise([v], [y], act)
        ref = ORC.pointwise(host64(v), act)
        yh = host64(y)
        assert np.all(np.isfinite(yh))
        assert np.all(np.abs(yh - ref) <= 2e-6 * np.maximum(1.0, np.abs(ref))), act
