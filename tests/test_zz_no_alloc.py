"""The fp8 quantize entry point that allocates nothing
(optimus_grouped_quantize_fp8_noalloc: its table and amax partials live in
the library's static per-GPU scratch array) against the allocating
optimus_grouped_quantize_fp8, through the C ABI: codes and scales bit for
bit, on two calls in a row whose second group is smaller (the array keeps
the first call's contents), scaled and unscaled, bf16 and fp32; a group too
large for the array is refused with nothing written."""
import numpy as np
import pytest
import torch

from paper_2607_02945_amd import binding as B
from paper_2607_02945_amd import synth
from tests.gpu_util import dev, say

pytestmark = pytest.mark.gpu


def _group(shapes, dtype, seed):
    """Members of the given shapes, scales spread over 2^+-6, one member a
    strided column view, one starting one value off 16-byte alignment, and
    special values (NaN, +-inf, overflow range) in the first member."""
    g = synth.rng(seed)
    xs = []
    for i, (r, c) in enumerate(shapes):
        v = g.standard_normal((r, c)) * float(np.exp2(g.uniform(-6.0, 6.0)))
        if i == 0:
            v[0, :4] = [np.nan, np.inf, -np.inf, 600.0]
        t = dev(synth.to_storage(v, dtype))
        if i == 1:  # strided view of a wider buffer
            big = torch.zeros((r, c + 24), dtype=t.dtype, device="cuda")
            big[:, 8:8 + c] = t
            t = big[:, 8:8 + c]
        if i == 2:  # one value off alignment
            buf = torch.zeros(r * c + 1, dtype=t.dtype, device="cuda")
            buf[1:] = t.reshape(-1)
            t = buf[1:].view(r, c)
        xs.append(t)
    return xs


def _run(fn, xs, scaled):
    qs = [torch.full(x.shape, 0xA5, dtype=torch.uint8, device="cuda") for x in xs]
    sc = [torch.full((1,), -1.0, dtype=torch.float32, device="cuda") for _ in xs]
    fn(xs, qs, sc if scaled else None, scaled)
    return qs, sc


@pytest.mark.parametrize("dtype", ["bf16", "fp32"])
@pytest.mark.parametrize("scaled", [True, False])
def test_noalloc_quantize_equals_allocating_call(dtype, scaled):
    calls = [[(4096, 1024), (3000, 520), (777, 96), (2048, 4096), (5, 8), (1000, 1000)],
             [(1024, 512), (300, 64), (99, 40)]]
    for k, shapes in enumerate(calls):
        say(f"[fp8 noalloc] {dtype} scaled={scaled} call {k} shapes={shapes}")
        xs = _group(shapes, dtype, seed=900 + 10 * k + (1 if scaled else 0))
        q_ref, s_ref = _run(B.optimus_grouped_quantize_fp8, xs, scaled)
        q, s = _run(B.optimus_grouped_quantize_fp8_noalloc, xs, scaled)
        torch.cuda.synchronize()
        for i in range(len(xs)):
            assert torch.equal(q[i], q_ref[i]), f"call {k} member {i}: codes differ"
            if scaled:
                assert torch.equal(s[i], s_ref[i]), f"call {k} member {i}: scale {s[i].item()} vs {s_ref[i].item()}"


def test_noalloc_quantize_refuses_a_group_beyond_the_array():
    """40 000 one-row members need about 6.5 MB of table and partials, above
    the 4 MiB array: UNSUPPORTED, nothing launched (the codes keep their fill)."""
    say("[fp8 noalloc] oversize group refused")
    n = 40000
    x = dev(synth.to_storage(synth.rng(950).standard_normal((n, 8)), "bf16"))
    q = torch.full((n, 8), 0xA5, dtype=torch.uint8, device="cuda")
    sc = torch.full((n,), -1.0, dtype=torch.float32, device="cuda")
    xs, qs, ss = [x[i:i + 1] for i in range(n)], [q[i:i + 1] for i in range(n)], [sc[i:i + 1] for i in range(n)]
    with pytest.raises(B.OptimusError) as e:
        B.optimus_grouped_quantize_fp8_noalloc(xs, qs, ss, True)
    assert e.value.name == "UNSUPPORTED" and "limit" in str(e.value), str(e.value)
    torch.cuda.synchronize()
    assert bool((q == 0xA5).all()) and bool((sc == -1.0).all())
