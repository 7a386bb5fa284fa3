"""Grouped Linear on the GPU against the fp64 oracle (through the C ABI)."""

import numpy as np
import pytest
import torch

import oracle
from paper_2607_02945_amd import binding as B
from paper_2607_02945_amd import synth
from tests.gpu_util import TOL, assert_close, dev, host64, say

pytestmark = pytest.mark.gpu
ORC = oracle.get()
ACTS = ["none", "relu", "sigmoid", "tanh", "silu"]


def _members(shapes, dtype, seed, integer=False, strided=False, bias=True):
    g = synth.rng(seed)
    ms = []
    for M, N, K in shapes:
        if integer:
            x = synth.to_storage(g.integers(-4, 5, size=(M, K)).astype(np.float64), dtype)
            w = synth.to_storage(g.integers(-4, 5, size=(N, K)).astype(np.float64), dtype)
            b = synth.to_storage(g.integers(-8, 9, size=N).astype(np.float64), dtype)
        else:
            x = synth.to_storage(g.standard_normal((M, K)), dtype)
            w = synth.to_storage(g.standard_normal((N, K)) / np.sqrt(K), dtype)
            b = synth.to_storage(g.standard_normal(N) * 0.1, dtype)
        xd = dev(x)
        if strided:  # x as a column view of a wider buffer
            big = torch.zeros((M, K + 24), dtype=x.dtype, device="cuda")
            big[:, 8:8 + K] = xd
            xd = big[:, 8:8 + K]
        ms.append((xd, dev(w), dev(b) if bias else None))
    return ms


def _run(ms, dtype, act, mode="oneshot", variant=None):
    """One group through the one-shot call, or a plan executed in `mode`; a
    pinned tile variant (kernel-table index) goes through the plan options."""
    ys = [torch.full((x.shape[0], w.shape[0]), float("nan"), dtype=x.dtype, device="cuda") for x, w, _ in ms]
    xs, ws, bs = [m[0] for m in ms], [m[1] for m in ms], [m[2] for m in ms]
    if mode == "oneshot" and variant is None:
        B.optimus_grouped_linear(xs, ws, bs, ys, act)
    else:
        opts = None if variant is None else {"gemm_tile": variant + 1}
        p = B.optimus_plan_linear_ex(xs, ws, bs, ys, act, options=opts)
        p.execute("grouped" if mode == "oneshot" else mode)
        torch.cuda.synchronize()
        p.close()
    return ys


def _check(ms, ys, dtype, act, what):
    for i, ((x, w, b), y) in enumerate(zip(ms, ys)):
        ref = ORC.linear(host64(x), host64(w), None if b is None else host64(b), act)
        assert_close(host64(y), ref, dtype, f"{what} member {i}")


RAGGED = [(1, 1, 8), (37, 16, 16), (130, 65, 48), (300, 200, 264), (64, 64, 64), (257, 129, 100)]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("act", ACTS)
def test_ragged_group_all_acts(dtype, act):
    say(f"[linear ragged] dtype={dtype} act={act}")
    ms = _members(RAGGED, dtype, seed=10)
    ys = _run(ms, dtype, act)
    _check(ms, ys, dtype, act, f"ragged {dtype} {act}")


@pytest.mark.parametrize("variant", [0, 1, 2, 4, 5])
def test_every_bf16_tile_variant(variant):
    say(f"[linear variant] {variant}")
    shapes = [(513, 300, 72), (256, 256, 1024), (31, 7, 40), (700, 520, 136)]
    ms = _members(shapes, "bf16", seed=11 + variant)
    for mode in ["grouped", "chain"]:
        ys = _run(ms, "bf16", "tanh", mode=mode, variant=variant)
        _check(ms, ys, "bf16", "tanh", f"variant {variant} {mode}")


@pytest.mark.parametrize("variant", [3, 6, 8, 10])
def test_every_fp32_tile_variant(variant):
    """The fp32 tiles, 64x64 (3), 64x128 (6), 32x128 (8: every K step's
    loads in flight at once when K <= 256, and the two wave pairs splitting K
    for members of N <= 64) and 16x128 (10: operands straight into MFMA
    registers in batches of 8 k-groups, spare waves splitting K two or four
    ways), grouped and chain, against the oracle: one to ten K steps (38
    k-groups: the 16-row kernel's batch loop turns over more than once),
    members of N <= 64 with even and odd step counts, a member wider than one
    tile."""
    say(f"[linear fp32 variant] {variant}")
    shapes = [(513, 120, 136), (300, 60, 200), (90, 33, 130), (257, 64, 260), (31, 7, 40), (130, 200, 64),
              (40, 100, 600)]
    ms = _members(shapes, "fp32", seed=15 + variant)
    for mode in ["grouped", "chain"]:
        ys = _run(ms, "fp32", "sigmoid", mode=mode, variant=variant)
        _check(ms, ys, "fp32", "sigmoid", f"fp32 variant {variant} {mode}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_unaligned_k_and_strided_input(dtype):
    say(f"[linear scalar path] {dtype}")
    ms = _members([(50, 33, 5), (70, 17, 13), (129, 40, 3)], dtype, seed=12)
    ys = _run(ms, dtype, "none")
    _check(ms, ys, dtype, "none", "K not a multiple of the vector width")
    ms = _members([(90, 48, 32), (65, 64, 56)], dtype, seed=13, strided=True)
    ys = _run(ms, dtype, "sigmoid")
    _check(ms, ys, dtype, "sigmoid", "strided x")
    ms = _members([(90, 48, 32)], dtype, seed=14, bias=False)
    ys = _run(ms, dtype, "relu")
    _check(ms, ys, dtype, "relu", "no bias")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_brute_force_integer_groups_bit_exact(dtype):
    """Small integers: every product and sum is exact in fp32 accumulation and the
    results (|y| <= 100) are exact in bf16, so the GPU must equal the oracle bit for bit."""
    say(f"[linear brute force] {dtype}")
    shapes = [(M, N, K) for M in (1, 2, 5) for N in (1, 3, 5) for K in (1, 2, 4, 5)]
    for s in range(0, len(shapes), 12):
        ms = _members(shapes[s:s + 12], dtype, seed=100 + s, integer=True)
        ys = _run(ms, dtype, "none")
        for (x, w, b), y in zip(ms, ys):
            ref = ORC.linear(host64(x), host64(w), host64(b))
            assert np.array_equal(host64(y), ref)


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_zero_and_identity_weights_bit_exact(dtype):
    say(f"[linear zero/identity] {dtype}")
    g = synth.rng(15)
    x = dev(synth.to_storage(g.standard_normal((200, 64)), dtype))
    b = dev(synth.to_storage(g.standard_normal(48), dtype))
    w0 = torch.zeros((48, 64), dtype=x.dtype, device="cuda")
    eye = torch.eye(64, dtype=x.dtype, device="cuda")
    z = torch.zeros(64, dtype=x.dtype, device="cuda")
    ys = _run([(x, w0, b), (x, eye, z)], dtype, "none")
    assert np.array_equal(host64(ys[0]), np.broadcast_to(host64(b), (200, 48)))
    assert np.array_equal(host64(ys[1]), host64(x))


def test_batch_fusion_identity_equal_shapes():
    """Equal-shape members (paper Sec. 3.2 batch fusion) against one batched
    matmul of the stacked operands, computed by the oracle member by member and
    by numpy on the stack."""
    say("[linear batch fusion]")
    ms = _members([(256, 64, 128)] * 6, "bf16", seed=16)
    ys = _run(ms, "bf16", "none")
    xs = np.stack([host64(m[0]) for m in ms])
    ws = np.stack([host64(m[1]) for m in ms])
    bs = np.stack([host64(m[2]) for m in ms])
    st = np.matmul(xs, np.transpose(ws, (0, 2, 1))) + bs[:, None, :]
    for i, y in enumerate(ys):
        assert_close(host64(y), st[i], "bf16", f"stacked member {i}")


def test_chain_equals_grouped_bitwise():
    """The per-member launch chain runs the same kernel per member, so it must give
    the grouped launch's bits exactly."""
    say("[linear chain vs grouped]")
    ms = _members(RAGGED, "bf16", seed=17)
    a = _run(ms, "bf16", "silu", mode="grouped")
    c = _run(ms, "bf16", "silu", mode="chain")
    for ya, yc in zip(a, c):
        assert torch.equal(ya, yc)


def test_empty_group_and_errors():
    say("[linear empty/errors]")
    B.optimus_grouped_linear([], [], [], [], "none")
    x = torch.zeros((8, 8), dtype=torch.bfloat16, device="cuda")
    w = torch.zeros((8, 8), dtype=torch.bfloat16, device="cuda")
    with pytest.raises(B.OptimusError) as ei:
        B.optimus_grouped_linear([x], [w], [None], [x], "none")
    assert ei.value.name == "ALIASING"
    assert torch.count_nonzero(x) == 0


def test_shared_input_members():
    """Members that share one input tensor (paper Table 1 batch_linear_lhs): the
    descriptors point at the same x; outputs against the oracle and against one
    matmul with the weights concatenated (inputs may alias each other)."""
    say("[linear shared input]")
    g = synth.rng(18)
    M, K, Ns = 1000, 256, [256, 512, 64, 256]
    x = dev(synth.to_storage(g.standard_normal((M, K)), "bf16"))
    ws = [dev(synth.to_storage(g.standard_normal((n, K)) / np.sqrt(K), "bf16")) for n in Ns]
    bs = [dev(synth.to_storage(g.standard_normal(n) * 0.1, "bf16")) for n in Ns]
    ms = [(x, w, b) for w, b in zip(ws, bs)]
    ys = _run(ms, "bf16", "relu")
    _check(ms, ys, "bf16", "relu", "shared input")
    whole = ORC.linear(host64(x), np.concatenate([host64(w) for w in ws]),
                       np.concatenate([host64(b) for b in bs]), "relu")
    offs = np.cumsum([0] + Ns)
    for i, y in enumerate(ys):
        assert_close(host64(y), whole[:, offs[i]:offs[i + 1]], "bf16", f"shared input member {i} vs concatenated W")


# Skinny members (every K, N <= 8: the decompose_mm shapes): the streaming
# kernel, one shape class per member, items of 1024 rows with a ragged last one.
SKINNY = [(1000, 8, 8), (1025, 2, 4), (5000, 4, 4), (300, 1, 3), (777, 5, 8), (64, 8, 7), (3, 3, 1), (2049, 6, 2), (4500, 8, 6), (6000, 2, 2)]


def _plan_kernel(ms, act):
    xs, ws, bs = [m[0] for m in ms], [m[1] for m in ms], [m[2] for m in ms]
    ys = [torch.empty((x.shape[0], w.shape[0]), dtype=x.dtype, device="cuda") for x, w, _ in ms]
    p = B.optimus_plan_linear(xs, ws, bs, ys, act)
    name = p.info()["kernel"]
    p.close()
    return name


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("act", ACTS)
def test_skinny_members(dtype, act):
    say(f"[linear skinny] {dtype} {act}")
    ms = _members(SKINNY, dtype, seed=30)
    assert _plan_kernel(ms, act) == "grouped_gemm_skinny"
    for mode in ["oneshot", "chain"]:
        ys = _run(ms, dtype, act, mode=mode)
        _check(ms, ys, dtype, act, f"skinny {dtype} {act} {mode}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_skinny_strided_rows_and_no_bias(dtype):
    """Rows that are not 16-byte pieces (x a column view of a wider buffer; K or
    N not the class size) take the element path."""
    say(f"[linear skinny strided] {dtype}")
    ms = _members([(900, 8, 8), (513, 2, 4), (300, 7, 5)], dtype, seed=31, strided=True)
    ys = _run(ms, dtype, "none")
    _check(ms, ys, dtype, "none", f"skinny strided {dtype}")
    ms = _members([(900, 8, 8), (513, 2, 4)], dtype, seed=32, bias=False)
    ys = _run(ms, dtype, "tanh")
    _check(ms, ys, dtype, "tanh", f"skinny no bias {dtype}")


def test_skinny_against_tiled_kernel():
    """The same fp32 group through the tiled MFMA kernel (variant 3) and the
    streaming kernel: both against the oracle."""
    say("[linear skinny vs tiled]")
    ms = _members([(4000, 8, 8), (3000, 4, 2)], "fp32", seed=33, bias=False)
    for v in (3, 7):
        ys = _run(ms, "fp32", "none", variant=v)
        _check(ms, ys, "fp32", "none", f"variant {v}")


@pytest.mark.timeout(300)
@pytest.mark.parametrize("variant", [4, 5])
def test_direct_to_lds_tiles_every_element_multi_tile(variant):
    """Each direct-to-LDS forward tile (256x256 8 waves, 128x128 4 waves) on a
    group with at least two tiles per persistent workgroup, so every
    workgroup prefetches a next tile's first K step during its last one and
    stages epilogues back to back; ragged tails in M and N, K of one to
    several steps; every output element against the oracle."""
    say(f"[linear dma multi-tile] variant {variant}")
    if variant == 4:
        shapes = [(4096, 1024, 64)] * 6 + [(4000, 1000, 72), (3900, 1016, 136)]
    else:
        shapes = [(4096, 512, 64)] * 7 + [(4000, 500, 72), (3900, 504, 136)]
    ms = _members(shapes, "bf16", seed=120 + variant)
    ys = [torch.full((x.shape[0], w.shape[0]), float("nan"), dtype=x.dtype, device="cuda") for x, w, _ in ms]
    p = B.optimus_plan_linear_ex([m[0] for m in ms], [m[1] for m in ms], [m[2] for m in ms], ys, "silu",
                                 options={"gemm_tile": variant + 1})
    info = p.info()
    assert info["work_items"] >= 2 * info["grid"], info
    p.execute()
    torch.cuda.synchronize()
    p.close()
    _check(ms, ys, "bf16", "silu", f"variant {variant} multi-tile")


@pytest.mark.parametrize("act", ACTS)
def test_streaming_small_members(act):
    """Members with K, N <= 64 (multiples of 8) on the streaming kernel (the
    planner's choice for such bf16 groups): ragged batches (1, tails inside a
    32-row slab and a 512-row item, several items), every K and N class, a
    member without bias; grouped and chain; every element against the oracle."""
    say(f"[linear streaming] {act}")
    shapes = [(1, 8, 8), (33, 16, 24), (511, 64, 64), (513, 48, 40), (1000, 24, 16), (2048, 56, 48), (70, 64, 8)]
    ms = _members(shapes, "bf16", seed=130)
    ms[1] = (ms[1][0], ms[1][1], None)
    for mode in ["grouped", "chain"]:
        xs, ws, bs = [m[0] for m in ms], [m[1] for m in ms], [m[2] for m in ms]
        ys = [torch.full((x.shape[0], w.shape[0]), float("nan"), dtype=x.dtype, device="cuda") for x, w, _ in ms]
        p = B.optimus_plan_linear(xs, ws, bs, ys, act)
        assert p.info()["kernel"] == "grouped_gemm_stream_bf16", p.info()
        p.execute(mode)
        torch.cuda.synchronize()
        p.close()
        _check(ms, ys, "bf16", act, f"streaming {mode}")


def test_streaming_reordered_item_list():
    """More streaming items than CUs: the planner orders them by bytes per row
    and reverses every other device-width of the list, so the grouped list is
    no longer member-major and the per-member chain launches walk their own
    copy. Both modes, every element against the oracle."""
    say("[linear streaming] reordered item list")
    g = synth.rng(131)
    dims = [8, 16, 24, 32, 40, 48, 56, 64]
    shapes = [(int(g.choice([300, 512, 700])), int(g.choice(dims)), int(g.choice(dims))) for _ in range(300)]
    ms = _members(shapes, "bf16", seed=132)
    xs, ws, bs = [m[0] for m in ms], [m[1] for m in ms], [m[2] for m in ms]
    for mode in ["grouped", "chain"]:
        ys = [torch.full((x.shape[0], w.shape[0]), float("nan"), dtype=x.dtype, device="cuda") for x, w, _ in ms]
        p = B.optimus_plan_linear(xs, ws, bs, ys, "sigmoid")
        info = p.info()
        assert info["kernel"] == "grouped_gemm_stream_bf16" and info["work_items"] > 256, info
        p.execute(mode)
        torch.cuda.synchronize()
        p.close()
        _check(ms, ys, "bf16", "sigmoid", f"streaming reordered {mode}")


def test_streaming_strided_and_fallback():
    """Row strides above the row lengths keep the streaming kernel (16-byte
    aligned rows); a member with K not a multiple of 8 sends the group to the
    register-staged 128x64 tile; both against the oracle."""
    say("[linear streaming strided / fallback]")
    g = synth.rng(131)
    x = dev(synth.to_storage(g.standard_normal((300, 72)), "bf16"))[:, 8:40]        # K = 32, ld 72
    w = dev(synth.to_storage(g.standard_normal((48, 40)) / 6, "bf16"))[:, :32]      # N = 48, ld 40
    b = dev(synth.to_storage(g.standard_normal(48) * 0.1, "bf16"))
    ybuf = torch.full((300, 56), float("nan"), dtype=torch.bfloat16, device="cuda")
    y = ybuf[:, :48]                                                                  # ld 56
    p = B.optimus_plan_linear([x], [w], [b], [y], "tanh")
    assert p.info()["kernel"] == "grouped_gemm_stream_bf16", p.info()
    p.execute()
    torch.cuda.synchronize()
    _check([(x, w, b)], [y], "bf16", "tanh", "streaming strided")
    ms = _members([(400, 32, 32), (200, 16, 12)], "bf16", seed=132)
    ys = [torch.full((m[0].shape[0], m[1].shape[0]), float("nan"), dtype=torch.bfloat16, device="cuda") for m in ms]
    p = B.optimus_plan_linear([m[0] for m in ms], [m[1] for m in ms], [m[2] for m in ms], ys, "relu")
    assert p.info()["kernel"].startswith("grouped_gemm_bf16_128x64"), p.info()
    p.execute()
    torch.cuda.synchronize()
    _check(ms, ys, "bf16", "relu", "K not a multiple of 8")
