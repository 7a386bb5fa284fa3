"""Seeded synthetic operator groups shaped like the paper's recommendation workloads.

This module only draws inputs: shapes, random values, and the one rounding of
each drawn fp64 value to its storage dtype. It holds none of the grouped
operators' arithmetic, and it is the only code the GPU path and the CPU oracle
share: tests draw a workload here, hand the storage tensors to the GPU and the
exact fp64 images of the same values to the oracle.

Every generator uses ``numpy.random.Generator(PCG64(seed))`` and a fixed draw
order: shapes first, then per member in the order (W, b, gamma, beta, X).
``N(mu, v)`` takes v as the VARIANCE. Sizes can be scaled down (for parity
tests) without changing the recipe.

The workload families (paper Sec. 5: DLRM-style recommendation models;
Sec. 5.2: many small bf16 operators; Sec. 3.2: split -> LayerNorm -> act -> cat):
  tiny_group        G=8 fp32 Linear members, shared batch 512, -> LayerNorm -> tanh
  launch_bound      G=256 tiny bf16 Linear members, batch 2048, -> sigmoid
  split_op_cat      [8192, 4096] bf16 split into 32 Dirichlet widths, LN_j -> silu, cat
  towers            26 bf16 MLP towers Linear(in_g->512)+relu+Linear(512->256)+LayerNorm, batch 4096
  large_group       G=32 bf16 Linear members, batch 16384, K=1024 -> LayerNorm -> tanh
  large_group_shared  the same with one input X shared by every member (batch_linear_lhs)
  decompose_mm      the four tall-skinny mm members of the appendix decompose_mm case
                    study ([~2e7, K] x [K, N], K, N in {(8, 8), (4, 2)}), fp32, no bias
  act_quant         G=32 bf16 saved activations [16384, N_g] (large_group's Linear outputs)
                    for the fp8 activation codec, per-member scale 2^U(-6, 6)
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import List, Optional

import numpy as np
import torch

DTYPES = {"fp32": torch.float32, "bf16": torch.bfloat16}


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def to_storage(a: np.ndarray, dtype: str) -> torch.Tensor:
    """Round an fp64 draw once to the storage dtype (CPU tensor)."""
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float64)).to(DTYPES[dtype]).contiguous()


def exact64(t: Optional[torch.Tensor]) -> Optional[np.ndarray]:
    """The exact fp64 image of a stored tensor (widening is exact)."""
    if t is None:
        return None
    return t.detach().to("cpu").to(torch.float64).numpy()


def _normal(g: np.random.Generator, shape, var: float) -> np.ndarray:
    return g.standard_normal(shape) * np.sqrt(var)


@dataclass
class LinearMember:
    x: torch.Tensor                 # [M, K]
    w: torch.Tensor                 # [N, K]
    b: Optional[torch.Tensor]       # [N]

    @property
    def M(self): return self.x.shape[0]

    @property
    def K(self): return self.x.shape[1]

    @property
    def N(self): return self.w.shape[0]


@dataclass
class LinearLNGroup:
    """Group of Linear members, each optionally followed by LayerNorm and an activation."""
    name: str
    dtype: str
    members: List[LinearMember]
    act: str                                     # activation after the last op
    ln: bool = False
    gammas: List[torch.Tensor] = field(default_factory=list)
    betas: List[torch.Tensor] = field(default_factory=list)
    eps: float = 1e-5

    @property
    def G(self): return len(self.members)


@dataclass
class SplitOpCatInput:
    name: str
    dtype: str
    x: torch.Tensor                              # [rows, D]
    widths: List[int]
    gammas: List[torch.Tensor]
    betas: List[torch.Tensor]
    eps: float
    act: str


@dataclass
class Tower:
    x: torch.Tensor       # [B, in_g]
    w1: torch.Tensor      # [512, in_g]
    b1: torch.Tensor
    w2: torch.Tensor      # [256, 512]
    b2: torch.Tensor
    gamma: torch.Tensor   # [256]
    beta: torch.Tensor


@dataclass
class TowersInput:
    name: str
    dtype: str
    towers: List[Tower]
    eps: float = 1e-5

    @property
    def G(self): return len(self.towers)


@dataclass
class ActQuantInput:
    """Saved activations handed to the fp8 activation codec."""
    name: str
    dtype: str
    xs: List[torch.Tensor]                       # [M, N_g] each
    sigmas: List[float]

    @property
    def G(self): return len(self.xs)


# ------------------------------------------------------------------ helpers
def dirichlet_widths(g: np.random.Generator, n_pieces: int, D: int, unit: int = 16) -> List[int]:
    """Widths that are multiples of ``unit`` summing to D, from a Dirichlet(1) draw.

    Each piece gets one unit; the remaining units are shared by largest remainder
    of (remaining * p), ties to the lower index.
    """
    total_units = D // unit
    assert total_units * unit == D and total_units >= n_pieces
    p = g.dirichlet(np.ones(n_pieces))
    spare = total_units - n_pieces
    q = spare * p
    base = np.floor(q).astype(np.int64)
    left = spare - int(base.sum())
    frac = q - base
    order = sorted(range(n_pieces), key=lambda i: (-frac[i], i))
    for i in order[:left]:
        base[i] += 1
    return [int(unit * (1 + b)) for b in base]


def xavier_uniform(g, n_out: int, n_in: int) -> np.ndarray:
    a = np.sqrt(6.0 / (n_in + n_out))
    return g.uniform(-a, a, size=(n_out, n_in))


def kaiming_normal_relu(g, n_out: int, n_in: int) -> np.ndarray:
    return _normal(g, (n_out, n_in), 2.0 / n_in)


# ------------------------------------------------------------------ workloads
def tiny_group(seed: int = 0, G: int = 8, M: int = 512) -> LinearLNGroup:
    """G fp32 Linear members on a shared batch M; K in {64,128,256}, N in {64,128};
    X, W ~ N(0, 1/K), b ~ N(0, 0.01); then LayerNorm(eps 1e-5, gamma 1, beta 0) and tanh."""
    g = rng(seed)
    Ks = g.choice([64, 128, 256], size=G)
    Ns = g.choice([64, 128], size=G)
    members, gammas, betas = [], [], []
    for K, N in zip(Ks.tolist(), Ns.tolist()):
        w = to_storage(_normal(g, (N, K), 1.0 / K), "fp32")
        b = to_storage(_normal(g, (N,), 0.01), "fp32")
        gammas.append(to_storage(np.ones(N), "fp32"))
        betas.append(to_storage(np.zeros(N), "fp32"))
        x = to_storage(_normal(g, (M, K), 1.0 / K), "fp32")
        members.append(LinearMember(x, w, b))
    return LinearLNGroup("tiny_group", "fp32", members, "tanh", True, gammas, betas, 1e-5)


def launch_bound(seed: int = 0, G: int = 256, M: int = 2048) -> LinearLNGroup:
    """G bf16 Linear members, batch M, K and N in {16,32,48,64}; X ~ N(0,1),
    W Xavier-uniform, b ~ N(0, 0.01); then sigmoid."""
    g = rng(seed)
    Ks = g.choice([16, 32, 48, 64], size=G)
    Ns = g.choice([16, 32, 48, 64], size=G)
    members = []
    for K, N in zip(Ks.tolist(), Ns.tolist()):
        w = to_storage(xavier_uniform(g, N, K), "bf16")
        b = to_storage(_normal(g, (N,), 0.01), "bf16")
        x = to_storage(g.standard_normal((M, K)), "bf16")
        members.append(LinearMember(x, w, b))
    return LinearLNGroup("launch_bound", "bf16", members, "sigmoid")


def split_op_cat(seed: int = 0, rows: int = 8192, D: int = 4096, n_pieces: int = 32) -> SplitOpCatInput:
    """[rows, D] bf16 ~ N(0,1) split along dim 1 into Dirichlet widths (multiples
    of 16); per piece LayerNorm(gamma ~ U(0.5,1.5), beta ~ N(0,0.1), eps 1e-5) then silu."""
    g = rng(seed)
    widths = dirichlet_widths(g, n_pieces, D)
    gammas, betas = [], []
    for w in widths:
        gammas.append(to_storage(g.uniform(0.5, 1.5, size=w), "bf16"))
        betas.append(to_storage(_normal(g, (w,), 0.1), "bf16"))
    x = to_storage(g.standard_normal((rows, D)), "bf16")
    return SplitOpCatInput("split_op_cat", "bf16", x, widths, gammas, betas, 1e-5, "silu")


def towers(seed: int = 0, G: int = 26, M: int = 4096, hidden: int = 512, out: int = 256) -> TowersInput:
    """G bf16 towers: Linear(in_g->hidden)+relu+Linear(hidden->out)+LayerNorm(gamma 1, beta 0);
    in_g in {64,128,256,512}; X ~ N(0,1); Kaiming-normal (fan_in, relu) weights; b ~ N(0, 0.01)."""
    g = rng(seed)
    ins = g.choice([64, 128, 256, 512], size=G)
    ts = []
    for K in ins.tolist():
        w1 = to_storage(kaiming_normal_relu(g, hidden, K), "bf16")
        b1 = to_storage(_normal(g, (hidden,), 0.01), "bf16")
        w2 = to_storage(kaiming_normal_relu(g, out, hidden), "bf16")
        b2 = to_storage(_normal(g, (out,), 0.01), "bf16")
        gamma = to_storage(np.ones(out), "bf16")
        beta = to_storage(np.zeros(out), "bf16")
        x = to_storage(g.standard_normal((M, K)), "bf16")
        ts.append(Tower(x, w1, b1, w2, b2, gamma, beta))
    return TowersInput("towers", "bf16", ts, 1e-5)


def large_group(seed: int = 0, G: int = 32, M: int = 16384, K: int = 1024) -> LinearLNGroup:
    """G bf16 Linear members, batch M, K in-features, N in {256,512,1024};
    X ~ N(0,1), W ~ N(0, 1/K), b ~ N(0, 0.01); then LayerNorm(gamma 1, beta 0) and tanh."""
    g = rng(seed)
    Ns = g.choice([256, 512, 1024], size=G)
    members, gammas, betas = [], [], []
    for N in Ns.tolist():
        w = to_storage(_normal(g, (N, K), 1.0 / K), "bf16")
        b = to_storage(_normal(g, (N,), 0.01), "bf16")
        gammas.append(to_storage(np.ones(N), "bf16"))
        betas.append(to_storage(np.zeros(N), "bf16"))
        x = to_storage(g.standard_normal((M, K)), "bf16")
        members.append(LinearMember(x, w, b))
    return LinearLNGroup("large_group", "bf16", members, "tanh", True, gammas, betas, 1e-5)


def large_group_shared(seed: int = 0, G: int = 32, M: int = 16384, K: int = 1024) -> LinearLNGroup:
    """large_group with ONE input X [M, K] shared by every member (Table 1's
    batch_linear_lhs: Linear members on a common left-hand side). Draws:
    shapes, per member (W, b, gamma, beta), then X once; distributions as
    large_group."""
    g = rng(seed)
    Ns = g.choice([256, 512, 1024], size=G)
    ws, gammas, betas = [], [], []
    for N in Ns.tolist():
        w = to_storage(_normal(g, (N, K), 1.0 / K), "bf16")
        b = to_storage(_normal(g, (N,), 0.01), "bf16")
        gammas.append(to_storage(np.ones(N), "bf16"))
        betas.append(to_storage(np.zeros(N), "bf16"))
        ws.append((w, b))
    x = to_storage(g.standard_normal((M, K)), "bf16")
    members = [LinearMember(x, w, b) for w, b in ws]
    return LinearLNGroup("large_group_shared", "bf16", members, "tanh", True, gammas, betas, 1e-5)


# The four aten.mm shapes of the decompose_mm case study (appendix Sec. 8.2):
# (M, K, N) of [M, K] x [K, N]; as Linear members the weight is W = [N, K].
DECOMPOSE_MM_SHAPES = [(18583840, 8, 8), (25247936, 4, 2), (22502112, 8, 8), (17980096, 4, 2)]


def decompose_mm(seed: int = 0, scale: float = 1.0, dtype: str = "fp32") -> LinearLNGroup:
    """The four tall-skinny mm members of the decompose_mm case study (no bias),
    M scaled by `scale` for parity tests; X ~ N(0, 1), W ~ N(0, 1/K). The paper
    states no dtype for them: fp32 (PyTorch's default) is the reading."""
    g = rng(seed)
    members = []
    for M, K, N in DECOMPOSE_MM_SHAPES:
        w = to_storage(_normal(g, (N, K), 1.0 / K), dtype)
        x = to_storage(g.standard_normal((max(1, int(round(M * scale))), K)), dtype)
        members.append(LinearMember(x, w, None))
    return LinearLNGroup("decompose_mm", dtype, members, "none")


def act_quant(seed: int = 0, G: int = 32, M: int = 16384, dtype: str = "bf16") -> ActQuantInput:
    """G activation tensors shaped like large_group's Linear outputs ([M, N_g],
    N_g in {256, 512, 1024}): the saved activations the activation-quantization
    rewrite stores in FP8 (paper Sec. 5, appendix Sec. 8.2). Member g ~ N(0,
    s_g^2) with log2 s_g ~ U(-6, 6), so the per-tensor scales span four orders
    of magnitude and, unscaled, the widest members overflow E4M3 (|x| > 464)."""
    g = rng(seed)
    Ns = g.choice([256, 512, 1024], size=G)
    sig = np.exp2(g.uniform(-6.0, 6.0, size=G))
    xs = [to_storage(g.standard_normal((M, int(N))) * float(s), dtype) for N, s in zip(Ns.tolist(), sig.tolist())]
    return ActQuantInput("act_quant", dtype, xs, sig.tolist())


def fp8_codes(seed: int, rows: int, cols: int) -> torch.Tensor:
    """Uniform random bytes: every E4M3 code, NaN codes included (uint8 [rows, cols])."""
    return torch.from_numpy(rng(seed).integers(0, 256, size=(rows, cols), dtype=np.uint8))


WORKLOADS = {
    "tiny_group": tiny_group,
    "launch_bound": launch_bound,
    "split_op_cat": split_op_cat,
    "towers": towers,
    "large_group": large_group,
    "large_group_shared": large_group_shared,
    "decompose_mm": decompose_mm,
    "act_quant": act_quant,
}
