"""Plans under HIP graph capture: an execution is a sequence of kernel launches
on the caller's stream with no host work, copies or fills, so it can be
recorded into a graph once and replayed. Each case captures one plan (grouped
and, where it has one, per-op chain mode), replays the graph several times
with eager work on the same outputs and synchronizations in between, and
checks every replay bit for bit against an eager execution of the same plan.
The kernels are the same either way, so the results must not differ at all."""
import numpy as np
import pytest
import torch

from paper_2607_02945_amd import binding as B
from paper_2607_02945_amd import synth
from tests.gpu_util import dev, say

pytestmark = pytest.mark.gpu
REPLAYS = 3


def _rand(g, shape, dtype, scale=1.0):
    return dev(synth.to_storage(g.standard_normal(shape) * scale, dtype))


def _check_replays(plan, outs, mode, what):
    """Eager reference, then REPLAYS replays of a captured execution, each
    preceded by eager work that overwrites the outputs."""
    plan.execute(mode)
    torch.cuda.synchronize()
    ref = [o.clone() for o in outs]
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph, stream=side):
        plan.execute(mode)
    torch.cuda.synchronize()
    for r in range(REPLAYS):
        for o in outs:
            o.fill_(7)  # eager work between the replays
        torch.cuda.synchronize()
        graph.replay()
        torch.cuda.synchronize()
        for i, (o, e) in enumerate(zip(outs, ref)):
            assert torch.equal(o, e), f"{what} {mode}: replay {r} output {i} differs from the eager execution"


def _linear_group(g, dtype, shapes):
    xs = [_rand(g, (M, K), dtype) for M, N, K in shapes]
    ws = [_rand(g, (N, K), dtype, 1.0 / np.sqrt(K)) for M, N, K in shapes]
    bs = [_rand(g, (N,), dtype, 0.1) for M, N, K in shapes]
    return xs, ws, bs


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_linear_and_fused_layernorm_plans_replay(dtype):
    say(f"[graph] linear / linear+layernorm {dtype}")
    g = synth.rng(401)
    shapes = [(512, 128, 256), (300, 64, 64), (513, 96, 136), (64, 16, 40)]
    xs, ws, bs = _linear_group(g, dtype, shapes)
    ys = [torch.empty((M, N), dtype=xs[0].dtype, device="cuda") for M, N, K in shapes]
    lin = B.optimus_plan_linear(xs, ws, bs, ys, "sigmoid")
    for mode in ("grouped", "chain"):
        _check_replays(lin, ys, mode, f"linear {dtype} ({lin.info()['kernel']})")
    gs = [_rand(g, (N,), dtype, 0.5) for M, N, K in shapes]
    be = [_rand(g, (N,), dtype, 0.1) for M, N, K in shapes]
    zs = [torch.empty_like(y) for y in ys]
    fused = B.optimus_plan_linear_layernorm(xs, ws, bs, zs, gs, be, 1e-5, "tanh")
    for mode in ("grouped", "chain"):
        _check_replays(fused, zs, mode, f"linear+layernorm {dtype} ({fused.info()['kernel']})")


def test_streaming_and_wide_gemm_plans_replay():
    say("[graph] streaming and 256x256 tiles")
    g = synth.rng(402)
    small = [(2048, 16 * (1 + i % 4), 16 * (1 + (i // 4) % 4)) for i in range(24)]
    xs, ws, bs = _linear_group(g, "bf16", small)
    ys = [torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for M, N, K in small]
    lin = B.optimus_plan_linear(xs, ws, bs, ys, "relu")
    _check_replays(lin, ys, "grouped", f"streaming linear ({lin.info()['kernel']})")
    wide = [(4096, 512, 512)] * 8
    xs, ws, bs = _linear_group(g, "bf16", wide)
    ys = [torch.empty((M, N), dtype=torch.bfloat16, device="cuda") for M, N, K in wide]
    lin = B.optimus_plan_linear(xs, ws, bs, ys, "none")
    _check_replays(lin, ys, "grouped", f"wide linear ({lin.info()['kernel']})")


@pytest.mark.parametrize("act", ["none", "silu"])
def test_rowwise_and_split_op_cat_plans_replay(act):
    say(f"[graph] layernorm / pointwise / split-op-cat {act}")
    g = synth.rng(403)
    rows = [(1000, 1024), (333, 200), (64, 4096)]
    xs = [_rand(g, s, "bf16") for s in rows]
    ys = [torch.empty_like(x) for x in xs]
    gs = [_rand(g, (c,), "bf16", 0.5) for r, c in rows]
    be = [_rand(g, (c,), "bf16", 0.1) for r, c in rows]
    ln = B.optimus_plan_layernorm(xs, ys, gs, be, 1e-5, act)
    for mode in ("grouped", "chain"):
        _check_replays(ln, ys, mode, f"layernorm {act}")
    pw = B.optimus_plan_pointwise(xs, ys, "tanh" if act == "none" else act)
    _check_replays(pw, ys, "grouped", f"pointwise {act}")
    widths = [64, 128, 16, 304, 512]
    x = _rand(g, (777, sum(widths)), "bf16")
    y = torch.empty_like(x)
    pg = [_rand(g, (w,), "bf16", 0.5) for w in widths]
    pb = [_rand(g, (w,), "bf16", 0.1) for w in widths]
    soc = B.optimus_plan_split_op_cat(x, y, widths, pg, pb, True, 1e-5, act)
    for mode in ("grouped", "horizontal", "chain"):
        _check_replays(soc, [y], mode, f"split-op-cat {act}")


def test_fp8_and_backward_plans_replay():
    say("[graph] fp8 codec and backward")
    g = synth.rng(404)
    xs = [_rand(g, (1000, c), "bf16", s) for c, s in ((256, 3.0), (512, 0.01), (96, 40.0))]
    qs = [torch.empty(x.shape, dtype=torch.uint8, device="cuda") for x in xs]
    sc = [torch.ones(1, dtype=torch.float32, device="cuda") for _ in xs]
    quant = B.optimus_plan_quantize_fp8(xs, qs, sc, True)
    _check_replays(quant, qs + sc, "grouped", "scaled quantize")
    ys = [torch.empty_like(x) for x in xs]
    deq = B.optimus_plan_dequantize_fp8(qs, sc, ys)
    _check_replays(deq, ys, "grouped", "dequantize")
    shapes = [(4096, 256, 512), (1000, 64, 96)]
    xs, ws, _ = _linear_group(g, "bf16", shapes)
    dys = [_rand(g, (M, N), "bf16") for M, N, K in shapes]
    dxs = [torch.empty_like(x) for x in xs]
    dws = [torch.empty_like(w) for w in ws]
    dbs = [torch.empty((N,), dtype=torch.bfloat16, device="cuda") for M, N, K in shapes]
    bwd = B.optimus_plan_linear_backward(xs, ws, dys, dxs, dws, dbs)
    _check_replays(bwd, dxs + dws + dbs, "grouped", "linear backward")
    lx = [_rand(g, (2000, c), "bf16") for c in (1024, 256)]
    ldy = [_rand(g, x.shape, "bf16") for x in lx]
    ldx = [torch.empty_like(x) for x in lx]
    lg = [_rand(g, (x.shape[1],), "bf16", 0.5) for x in lx]
    lb = [_rand(g, (x.shape[1],), "bf16", 0.1) for x in lx]
    dg = [torch.empty_like(v) for v in lg]
    db = [torch.empty_like(v) for v in lg]
    lnb = B.optimus_plan_layernorm_act_backward(lx, ldy, ldx, lg, lb, dg, db, 1e-5, "tanh")
    _check_replays(lnb, ldx + dg + db, "grouped", "layernorm + tanh backward")
