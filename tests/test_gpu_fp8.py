"""The fp8 activation codec on the GPU against the oracle, through the C ABI:
codes and scales bit-exact, dequantized values bit-exact after the one
rounding to the storage dtype (both sides decide every code in fp32)."""
import numpy as np
import pytest
import torch

import oracle
from paper_2607_02945_amd import binding as B
from paper_2607_02945_amd import synth
from tests.gpu_util import dev, say

pytestmark = pytest.mark.gpu
ORC = oracle.get()
SENT = 0xA5  # code-buffer padding: must survive every call


def _member(values, dtype="bf16", padx=0, offx=0, padq=0, offq=0):
    """A member from fp64 values (or a storage tensor), placed at column
    offset offx of rows padded by padx values; its code buffer likewise."""
    st = values if isinstance(values, torch.Tensor) else synth.to_storage(values, dtype)
    rows, cols = st.shape
    base = torch.zeros((rows, cols + padx + offx), dtype=st.dtype)
    base[:, offx:offx + cols] = st
    xb = dev(base)
    qb = torch.full((rows, cols + padq + offq), SENT, dtype=torch.uint8, device="cuda")
    return {"x": xb[:, offx:offx + cols], "x64": synth.exact64(st), "qb": qb, "q": qb[:, offq:offq + cols],
            "offq": offq, "cols": cols}


def _quantize(ms, scaled, mode="oneshot", plan=None):
    xs, qs = [m["x"] for m in ms], [m["q"] for m in ms]
    scales = [torch.full((1,), float("nan"), dtype=torch.float32, device="cuda") for _ in ms] if scaled else None
    if mode == "oneshot":
        B.optimus_grouped_quantize_fp8(xs, qs, scales, scaled)
    else:
        p = B.optimus_plan_quantize_fp8(xs, qs, scales, scaled)
        info = p.info()
        launches = 2 if scaled else 1
        assert info["kind"] == 5 and info["launches"] == launches and info["chain_launches"] == launches * len(ms)
        assert info["kernel"].startswith("grouped_quantize_fp8_scaled" if scaled else "grouped_quantize_fp8_")
        p.execute(mode)
        torch.cuda.synchronize()
        p.close()
    torch.cuda.synchronize()
    return scales


def _check_codes(ms, scales, scaled, what):
    for i, m in enumerate(ms):
        ref_q, ref_s = ORC.quantize_fp8(m["x64"], scaled)
        got = m["q"].cpu().numpy()
        bad = np.argwhere(got != ref_q)
        if bad.size:
            r, c = bad[0]
            raise AssertionError(f"{what} member {i}: {len(bad)} codes differ; first at ({r}, {c}): x={m['x64'][r, c]!r} "
                                 f"gpu {got[r, c]:#04x} oracle {ref_q[r, c]:#04x}")
        if scaled:
            s = np.float32(scales[i].item())
            assert s.view(np.uint32) == np.float32(ref_s).view(np.uint32), f"{what} member {i}: scale {s} vs {ref_s}"
        qb = m["qb"].cpu().numpy()
        pad = np.ones(qb.shape, bool)
        pad[:, m["offq"]:m["offq"] + m["cols"]] = False
        assert np.all(qb[pad] == SENT), f"{what} member {i}: padding written"


def _bf16_all_values():
    bits = np.arange(65536, dtype=np.uint16).view(np.int16).reshape(256, 256)
    return torch.from_numpy(bits.copy()).view(torch.bfloat16)


# ------------------------------------------------------------------ every value
@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("layout", ["vector", "per_value"])
def test_every_bf16_value_unscaled(dtype, layout):
    """All 65536 bf16 bit patterns (zeros, subnormals, the overflow range,
    infinities, NaNs of both signs) as one member."""
    say(f"[fp8 all values] {dtype} {layout}")
    st = _bf16_all_values()
    if dtype == "fp32":
        st = st.float()
    kw = {} if layout == "vector" else {"offx": 1, "padq": 3, "offq": 1}
    ms = [_member(st, dtype, **kw)]
    _check_codes(ms, _quantize(ms, False), False, f"all values {dtype} {layout}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_every_finite_bf16_value_scaled(dtype):
    """Scaled: the finite bf16 values (amax = the largest bf16), once with the
    NaNs among them (the member takes the exact path, NaN skipped in amax) and
    once without."""
    say(f"[fp8 all finite values scaled] {dtype}")
    st = _bf16_all_values()
    f = torch.isfinite(st.float()).numpy()
    fin = st.flatten()[torch.from_numpy(f.flatten())][: 255 * 256].reshape(255, 256)
    nan_and_fin = st.clone()
    nan_and_fin[torch.from_numpy(np.isinf(st.float().numpy()))] = 0
    if dtype == "fp32":
        fin, nan_and_fin = fin.float(), nan_and_fin.float()
    ms = [_member(fin, dtype), _member(nan_and_fin, dtype)]
    for mode in ["oneshot", "grouped", "chain"]:
        _check_codes(ms, _quantize(ms, True, mode), True, f"finite values scaled {dtype} {mode}")


# ------------------------------------------------------------------ random groups
SHAPES = [(1000, 256, 1.0), (333, 520, 0.01), (64, 8, 100.0), (1, 4096, 3.0), (2, 40000, 0.5), (4097, 24, 50.0),
          (130, 1024, 2.0 ** -7), (2, 100000, 30.0)]


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("scaled", [True, False])
@pytest.mark.parametrize("mode", ["oneshot", "grouped", "chain"])
def test_ragged_group(dtype, scaled, mode):
    """Members of different shapes and scales in one launch: several tiles and
    ragged tails, a row wider than one item (row segments), a single row, a
    width of one 16-byte chunk; sigma 100 overflows E4M3 when unscaled."""
    say(f"[fp8 ragged] {dtype} scaled={scaled} {mode}")
    g = synth.rng(301)
    ms = [_member(g.standard_normal((r, c)) * s, dtype) for r, c, s in SHAPES]
    _check_codes(ms, _quantize(ms, scaled, mode), scaled, f"ragged {dtype} {scaled} {mode}")


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("scaled", [True, False])
def test_strided_and_unaligned(dtype, scaled):
    """Row strides above the width, a start one value off 16-byte alignment,
    widths that are not whole 16-byte chunks: the per-value path, and the
    16-byte path with padded strides."""
    say(f"[fp8 layouts] {dtype} scaled={scaled}")
    g = synth.rng(302)
    ms = [
        _member(g.standard_normal((300, 256)) * 4, dtype, padx=64, padq=16),        # 16-byte path, strided
        _member(g.standard_normal((257, 100)) * 4, dtype, padx=5, offx=1, padq=1),  # per-value path
        _member(g.standard_normal((50, 37)), dtype, padq=11, offq=3),               # odd width
        _member(g.standard_normal((3, 9000)) * 700, dtype, offx=1),                 # wide, per-value segments
    ]
    for mode in ["oneshot", "grouped"]:
        _check_codes(ms, _quantize(ms, scaled, mode), scaled, f"layouts {dtype} {scaled} {mode}")


def test_many_small_members():
    """300 small members, one amax slot each, in one launch pair."""
    say("[fp8 many members]")
    g = synth.rng(303)
    rows = g.integers(1, 200, size=300)
    cols = g.choice([8, 16, 40, 64, 136, 256], size=300)
    sig = np.exp2(g.uniform(-10, 10, size=300))
    ms = [_member(g.standard_normal((int(r), int(c))) * s, "bf16") for r, c, s in zip(rows, cols, sig)]
    _check_codes(ms, _quantize(ms, True, "grouped"), True, "many members")


def test_large_member_amax_tiles():
    """An 80 MB member: its amax tiles grow past the default so that a
    convert item reduces at most about 256 partials; a small member beside it."""
    say("[fp8 large member]")
    g = synth.rng(309)
    ms = [_member(g.standard_normal((40000, 1024)) * 3.0, "bf16"), _member(g.standard_normal((10, 64)), "bf16")]
    ms[0]["x"][12345, 678] = 1000.0   # the amax sits in one tile only
    ms[0]["x64"][12345, 678] = 1000.0
    for mode in ["grouped", "chain"]:
        _check_codes(ms, _quantize(ms, True, mode), True, f"large member {mode}")


def test_special_members():
    """amax 0 (zeros of both signs: scale 1, codes 0x00 / 0x80), an infinity
    (amax infinite: zero codes, NaN codes with the sign of x), NaNs skipped in
    amax, subnormal-only values (inv overflows to infinity)."""
    say("[fp8 special members]")
    z = np.zeros((40, 64))
    z[::2, ::3] = -0.0
    g = synth.rng(304)
    inf = g.standard_normal((40, 64))
    inf[3, 5], inf[7, 9] = np.inf, -np.inf
    nan = g.standard_normal((40, 64)) * 9
    nan[0, 0], nan[10, 10], nan[39, 63] = np.nan, -np.nan, np.nan
    tiny = g.standard_normal((40, 64)) * 1e-39
    for dtype in ["bf16", "fp32"]:
        ms = [_member(v, dtype) for v in (z, inf, nan, tiny)]
        for scaled in [True, False]:
            _check_codes(ms, _quantize(ms, scaled, "grouped"), scaled, f"special {dtype} {scaled}")


def test_plan_executes_again():
    """A scaled plan run several times, grouped and chain interleaved, with
    the inputs changed in place between runs: every run matches the oracle on
    the inputs it saw (no amax partial of an earlier run survives)."""
    say("[fp8 plan re-execution]")
    g = synth.rng(305)
    ms = [_member(g.standard_normal((r, c)) * s, "bf16") for r, c, s in SHAPES[:4]]
    xs, qs = [m["x"] for m in ms], [m["q"] for m in ms]
    scales = [torch.zeros(1, dtype=torch.float32, device="cuda") for _ in ms]
    p = B.optimus_plan_quantize_fp8(xs, qs, scales, True)
    for k, mode in enumerate(["grouped", "grouped", "chain", "grouped", "chain", "chain", "grouped"]):
        gk = synth.rng(310 + k)
        for m in ms:
            st = synth.to_storage(gk.standard_normal(tuple(m["x"].shape)) * float(np.exp2(gk.uniform(-8, 8))), "bf16")
            m["x"].copy_(dev(st))
            m["x64"] = synth.exact64(st)
        p.execute(mode)
        torch.cuda.synchronize()
        _check_codes(ms, scales, True, f"run {k} {mode}")
    p.close()


def test_empty_group_and_errors():
    say("[fp8 errors]")
    B.optimus_grouped_quantize_fp8([], [], None, True)
    B.optimus_grouped_dequantize_fp8([], None, [])
    x = torch.zeros((4, 16), dtype=torch.bfloat16, device="cuda")
    q = torch.full((4, 16), SENT, dtype=torch.uint8, device="cuda")
    with pytest.raises(B.OptimusError) as ei:
        B.optimus_grouped_quantize_fp8([x], [q], None, True)   # scaled needs a scale
    assert ei.value.name == "INVALID_ARG"
    assert torch.all(q == SENT)


# ------------------------------------------------------------------ dequantize
def _dequant_ref(codes, scale, dtype):
    y = ORC.dequantize_fp8(codes, 1.0 if scale is None else scale)
    return torch.from_numpy(y.astype(np.float32)).to(synth.DTYPES[dtype])


def _same_values(got: torch.Tensor, ref: torch.Tensor) -> bool:
    """Bitwise equality, NaN positions compared as positions."""
    a, b = got.float().numpy(), ref.float().numpy()
    na, nb = np.isnan(a), np.isnan(b)
    if not np.array_equal(na, nb):
        return False
    ib = got.view(torch.int16 if got.dtype == torch.bfloat16 else torch.int32).numpy()
    rb = ref.view(torch.int16 if ref.dtype == torch.bfloat16 else torch.int32).numpy()
    return bool(np.array_equal(ib[~na], rb[~na]))


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("mode", ["oneshot", "grouped", "chain"])
def test_dequantize_group(dtype, mode):
    """Every code (NaN codes included) times fp32 scales of very different
    magnitudes, a member without a scale, strided and unaligned layouts."""
    say(f"[fp8 dequant] {dtype} {mode}")
    g = synth.rng(306)
    spec = [(1000, 256, 0, 0, 0), (333, 520, 8, 0, 0), (2, 40000, 0, 0, 0), (257, 100, 3, 1, 5), (50, 37, 0, 0, 2)]
    scales_v = [float(np.float32(v)) for v in (0.0123, 3.5e-6, 17.25, 1.0e-30)]   # member 4: no scale (1)
    members, refs = [], []
    for i, (r, c, padq, offq, pady) in enumerate(spec):
        codes = synth.fp8_codes(400 + i, r, c)
        qb = torch.zeros((r, c + padq + offq), dtype=torch.uint8)
        qb[:, offq:offq + c] = codes
        qb = dev(qb)
        yb = torch.full((r, c + pady), float("nan"), dtype=synth.DTYPES[dtype], device="cuda")
        s = None if i == 4 else torch.tensor([scales_v[i]], dtype=torch.float32, device="cuda")
        members.append((qb[:, offq:offq + c], s, yb[:, :c], yb, c))
        refs.append(_dequant_ref(codes.numpy(), None if s is None else scales_v[i], dtype))
    qs, ss, ys = [m[0] for m in members], [m[1] for m in members], [m[2] for m in members]
    if mode == "oneshot":
        B.optimus_grouped_dequantize_fp8(qs, ss, ys)
    else:
        p = B.optimus_plan_dequantize_fp8(qs, ss, ys)
        assert p.info()["kind"] == 6
        p.execute(mode)
        p.close()
    torch.cuda.synchronize()
    for i, ((_, _, y, yb, c), ref) in enumerate(zip(members, refs)):
        assert _same_values(y.cpu(), ref), f"dequant {dtype} {mode} member {i}"
        assert torch.all(torch.isnan(yb[:, c:].float())), f"member {i}: padding written"


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
def test_round_trip(dtype):
    """GPU quantize then GPU dequantize equals the oracle's quantize then
    dequantize of the same inputs, value for value."""
    say(f"[fp8 round trip] {dtype}")
    g = synth.rng(307)
    ms = [_member(g.standard_normal((r, c)) * s, dtype) for r, c, s in SHAPES[:5]]
    scales = _quantize(ms, True, "grouped")
    ys = [torch.empty(m["x"].shape, dtype=synth.DTYPES[dtype], device="cuda") for m in ms]
    B.optimus_grouped_dequantize_fp8([m["q"] for m in ms], scales, ys)
    torch.cuda.synchronize()
    for i, (m, y) in enumerate(zip(ms, ys)):
        q, s = ORC.quantize_fp8(m["x64"], True)
        assert _same_values(y.cpu(), _dequant_ref(q, s, dtype)), f"round trip member {i}"


# ------------------------------------------------------------------ full size
def test_act_quant_full_size():
    """The 32 saved activations [16384, N_g] at full size, quantized by one
    grouped plan launch as the benchmark runs it: every scale and every code
    against the oracle, member by member; then dequantized, sampled rows."""
    say("[fp8 full size act_quant]")
    w = synth.act_quant()
    xs = [dev(x) for x in w.xs]
    qs = [torch.empty(x.shape, dtype=torch.uint8, device="cuda") for x in xs]
    scales = [torch.full((1,), float("nan"), dtype=torch.float32, device="cuda") for _ in xs]
    p = B.optimus_plan_quantize_fp8(xs, qs, scales, True)
    p.execute("grouped")
    p.execute("grouped")
    torch.cuda.synchronize()
    ys = [torch.empty(x.shape, dtype=torch.bfloat16, device="cuda") for x in xs]
    d = B.optimus_plan_dequantize_fp8(qs, scales, ys)
    d.execute("grouped")
    torch.cuda.synchronize()
    rows = synth.rng(308).integers(0, w.xs[0].shape[0], size=64)
    for i, x in enumerate(w.xs):
        ref_q, ref_s = ORC.quantize_fp8(synth.exact64(x), True)
        s = np.float32(scales[i].item())
        assert s.view(np.uint32) == np.float32(ref_s).view(np.uint32), f"member {i} scale"
        got = qs[i].cpu().numpy()
        assert np.array_equal(got, ref_q), f"member {i}: {int(np.sum(got != ref_q))} codes differ"
        assert _same_values(ys[i][rows].cpu(), _dequant_ref(ref_q[rows], ref_s, "bf16")), f"member {i} dequant"
    p.close()
    d.close()
