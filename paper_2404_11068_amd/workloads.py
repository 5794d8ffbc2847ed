"""Seeded synthetic inputs for the Evoformer attention workloads.

This module only draws random numbers and stores them; it holds none of the
attention arithmetic.  Both the GPU path's tests/benchmark and the fp64
oracle consume exactly the arrays produced here, so the two sides see
identical bits.

The shapes stand in for the Evoformer attention calls of an AlphaFold
training step at the 256-residue crop (ScaleFold Section 2.1: four attention
modules per Evoformer block -- MSA row attention with pair bias, MSA column
attention, and triangle attention around the starting and ending node; the
extra-MSA stack runs the same row attention over many more sequences).  No
dataset is used: the OpenFold training data the paper trains on is replaced
by these seeded draws.

Recipe (one NumPy ``Generator(PCG64(seed))`` per workload; values drawn in
fp64, rounded to fp32, and for bf16 workloads rounded again to bf16 with
round-to-nearest-even).  Draw order: q, k, v, gate, bias, mask, dout.
"""
from __future__ import annotations

import dataclasses
import math
from typing import Dict, Optional

import numpy as np

__all__ = ["Workload", "WORKLOADS", "by_name", "generate", "as_float64", "f32_to_bf16_bits"]


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    n_rows: int          # N: independent attention rows (batch * rows)
    seq_len: int         # L: queries == keys
    n_heads: int         # H
    head_dim: int        # d
    dtype: str           # "f32" or "bf16"
    bias: bool           # pair bias [B,H,L,L] present
    rows_per_bias: int   # rows sharing one bias plane
    gate: bool = True
    mask: str = "none"   # none | bernoulli | tail_pad | length
    mask_p: float = 0.0  # drop probability for "bernoulli"
    pad_max: int = 0     # "tail_pad": pad the last U{0..pad_max} keys
    len_lo: int = 0      # "length": keep keys j < n, n ~ U{len_lo..len_hi}
    len_hi: int = 0
    qkv_scale: float = 1.0
    seed: int = 0
    description: str = ""

    @property
    def n_bias_planes(self) -> int:
        return self.n_rows // self.rows_per_bias if self.bias else 0

    @property
    def tokens(self) -> int:
        return self.n_rows * self.seq_len * self.n_heads * self.head_dim

    @property
    def score_elems(self) -> int:
        return self.n_rows * self.n_heads * self.seq_len * self.seq_len

    def flops_fwd(self) -> float:
        """Dense count: QK^T and PV, 2 flop per multiply-add."""
        return 4.0 * self.score_elems * self.head_dim

    def flops_bwd(self) -> float:
        """Dense count incl. the recomputed QK^T: QK^T, dP, dV, dQ, dK."""
        return 10.0 * self.score_elems * self.head_dim

    def with_rows(self, n_rows: int) -> "Workload":
        rpb = self.rows_per_bias if self.rows_per_bias <= n_rows else n_rows
        return dataclasses.replace(self, n_rows=n_rows, rows_per_bias=max(1, rpb))


WORKLOADS = [
    Workload("tri_tiny_f32", 32, 32, 4, 32, "f32", True, 32, mask="bernoulli", mask_p=0.10,
             seed=1000,
             description="tiny fp32 triangle-attention check: 32 rows x L=32, H=4, d=32, "
                         "pair bias [4,32,32], 10% random key drop"),
    Workload("msa_col_bf16", 256, 128, 8, 32, "bf16", False, 256, mask="tail_pad", pad_max=16,
             qkv_scale=1.0 / math.sqrt(32.0), seed=1001,
             description="MSA column attention: 256 residue columns x L=128 sequences, H=8, d=32, "
                         "no bias, last U{0..16} sequences padded"),
    Workload("msa_row_bias_bf16", 128, 256, 8, 32, "bf16", True, 128, mask="length",
             len_lo=224, len_hi=256, seed=1002,
             description="MSA row attention with pair bias: 128 rows x L=256 residues, H=8, d=32, "
                         "bias [8,256,256] shared by all rows, keys beyond U{224..256} padded"),
    Workload("tri_start_bf16", 256, 256, 4, 32, "bf16", True, 256, mask="length",
             len_lo=224, len_hi=256, seed=1003,
             description="triangle attention around the starting node: 256 rows x L=256, H=4, "
                         "d=32, bias [4,256,256], keys beyond U{224..256} padded"),
    Workload("extra_msa_bf16", 1024, 256, 8, 8, "bf16", True, 1024, mask="bernoulli",
             mask_p=0.05, seed=1004,
             description="extra-MSA row attention with pair bias: 1024 rows x L=256, H=8, d=8, "
                         "bias [8,256,256], 5% random key drop"),
    # one GPU's share when the rows of a call are split over 8 GPUs (each GPU
    # runs its rows with the whole bias plane): the kernels at their per-GPU
    # size
    Workload("msa_row_bias_bf16_share8", 16, 256, 8, 32, "bf16", True, 16, mask="length",
             len_lo=224, len_hi=256, seed=1005,
             description="one of 8 row shares of MSA row attention with pair bias: 16 rows x "
                         "L=256, H=8, d=32, bias [8,256,256], keys beyond U{224..256} padded"),
    Workload("extra_msa_bf16_share8", 128, 256, 8, 8, "bf16", True, 128, mask="bernoulli",
             mask_p=0.05, seed=1006,
             description="one of 8 row shares of extra-MSA row attention with pair bias: 128 rows "
                         "x L=256, H=8, d=8, bias [8,256,256], 5% random key drop"),
]


def by_name(name: str) -> Workload:
    for w in WORKLOADS:
        if w.name == name:
            return w
    raise KeyError(name)


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16 (round to nearest, ties to even); returns uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) >> 16
    return rounded.astype(np.uint16)


def as_float64(arr: np.ndarray, dtype: str) -> np.ndarray:
    """Exact fp64 value of an array stored as fp32 values or bf16 bits."""
    if dtype == "bf16":
        assert arr.dtype == np.uint16
        return (arr.astype(np.uint32) << 16).view(np.float32).astype(np.float64)
    return np.asarray(arr, dtype=np.float32).astype(np.float64)


def _store(x64: np.ndarray, dtype: str) -> np.ndarray:
    x32 = x64.astype(np.float32)
    return f32_to_bf16_bits(x32) if dtype == "bf16" else x32


def _mask(w: Workload, rng: np.random.Generator, n_rows: int, L: int) -> Optional[np.ndarray]:
    if w.mask == "none":
        return None
    if w.mask == "bernoulli":
        keep = (rng.random((n_rows, L)) >= w.mask_p).astype(np.uint8)
        empty = np.nonzero(keep.sum(axis=1) == 0)[0]
        fix = rng.integers(0, L, size=len(empty)) if len(empty) else []
        for r, j in zip(empty, fix):
            keep[r, j] = 1
        return keep
    if w.mask == "tail_pad":
        pad = int(rng.integers(0, w.pad_max + 1))
        keep = np.ones((n_rows, L), np.uint8)
        if pad:
            keep[:, L - pad:] = 0
        return keep
    if w.mask == "length":
        n = int(rng.integers(w.len_lo, w.len_hi + 1))
        keep = np.zeros((n_rows, L), np.uint8)
        keep[:, :n] = 1
        return keep
    raise ValueError(w.mask)


def generate(w: Workload, seed: Optional[int] = None, with_dout: bool = True) -> Dict[str, np.ndarray]:
    """Draw one input set.  Tensors q,k,v,gate,dout: [N,L,H,d]; bias: [B,H,L,L];
    mask: [N,L] uint8 (1 = keep).  Stored as float32, or uint16 bf16 bits."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    N, L, H, d = w.n_rows, w.seq_len, w.n_heads, w.head_dim
    shape = (N, L, H, d)
    out: Dict[str, np.ndarray] = {}
    for name in ("q", "k", "v"):
        out[name] = _store(rng.standard_normal(shape) * w.qkv_scale, w.dtype)
    out["gate"] = _store(rng.standard_normal(shape), w.dtype) if w.gate else None
    if w.bias:
        out["bias"] = _store(rng.standard_normal((w.n_bias_planes, H, L, L)), w.dtype)
    else:
        out["bias"] = None
    out["mask"] = _mask(w, rng, N, L)
    out["dout"] = _store(rng.standard_normal(shape), w.dtype) if with_dout else None
    return out


# ---------------------------------------------------------------------------
# LayerNorm workloads: the normalisations in front of the Evoformer blocks at
# the 256-residue crop (ScaleFold Section 3.3, "LayerNormalization": rows of
# 128 and 256 channels, plus the 64-channel extra-MSA stack).  x rows get a
# per-row offset and spread, as residual-stream activations do; the weight and
# bias sit near the identity transform, as trained LayerNorm parameters do.
# Draw order: row offset, row spread, x, weight, bias, dy.

@dataclasses.dataclass(frozen=True)
class LnWorkload:
    name: str
    n_rows: int
    n_cols: int
    dtype: str
    eps: float = 1e-5
    seed: int = 0
    description: str = ""

    def bytes_fwd(self) -> int:
        es = 2 if self.dtype == "bf16" else 4
        # x in, y out, mean and rstd out, weight and bias in
        return 2 * self.n_rows * self.n_cols * es + 8 * self.n_rows + 8 * self.n_cols

    def bytes_bwd(self) -> int:
        es = 2 if self.dtype == "bf16" else 4
        # x and dy in, dx out, mean and rstd in, weight in, dweight and dbias out
        return 3 * self.n_rows * self.n_cols * es + 8 * self.n_rows + 12 * self.n_cols


LN_WORKLOADS = [
    LnWorkload("ln_tiny_f32", 77, 64, "f32", seed=2000,
               description="tiny fp32 check: 77 rows x 64 channels"),
    LnWorkload("ln_msa_bf16", 128 * 256, 256, "bf16", seed=2001,
               description="MSA representation: 128 sequences x 256 residues, c_m = 256"),
    LnWorkload("ln_pair_bf16", 256 * 256, 128, "bf16", seed=2002,
               description="pair representation: 256 x 256 residue pairs, c_z = 128"),
    LnWorkload("ln_extra_msa_bf16", 1024 * 256, 64, "bf16", seed=2003,
               description="extra-MSA representation: 1024 sequences x 256 residues, c_e = 64"),
]


def ln_by_name(name: str) -> LnWorkload:
    for w in LN_WORKLOADS:
        if w.name == name:
            return w
    raise KeyError(name)


def generate_ln(w: LnWorkload, seed: Optional[int] = None, n_rows: Optional[int] = None
                ) -> Dict[str, np.ndarray]:
    """x, dy: [R, C]; weight, bias: [C] fp32.  x and dy are stored as fp32 or
    bf16 bits (w.dtype); the parameters are always fp32."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    R = w.n_rows if n_rows is None else n_rows
    C = w.n_cols
    offset = rng.standard_normal((R, 1)) * 2.0
    spread = rng.uniform(0.25, 4.0, size=(R, 1))
    x = rng.standard_normal((R, C)) * spread + offset
    weight = (1.0 + 0.2 * rng.standard_normal(C)).astype(np.float32)
    bias = (0.2 * rng.standard_normal(C)).astype(np.float32)
    dy = rng.standard_normal((R, C))
    return {"x": _store(x, w.dtype), "weight": weight, "bias": bias, "dy": _store(dy, w.dtype)}


# ---------------------------------------------------------------------------
# Fused LayerNorm + batched projections: the input side of each attention
# (ScaleFold Section 3.3, "GEMM Batching": query, key, value and gate linear
# layers over one normalised input).  Shapes of the three attention inputs at
# the 256-residue crop.  Weights ~ N(0, 1/C) (LeCun-normal scale), biases
# ~ N(0, 0.1^2), LayerNorm parameters near the identity.
# Draw order: row offset, row spread, x, ln weight, ln bias, weight, bias.

@dataclasses.dataclass(frozen=True)
class ProjWorkload:
    name: str
    n_rows: int      # R = N * L tokens
    c_in: int        # C
    proj_dim: int    # HD = H * d
    n_proj: int = 4
    bias: bool = True
    eps: float = 1e-5
    seed: int = 0
    description: str = ""

    def flops(self) -> float:
        return 2.0 * self.n_rows * self.c_in * self.n_proj * self.proj_dim

    def bytes(self) -> int:
        # x in, P outputs out (bf16), weight and parameters in
        return (2 * self.n_rows * self.c_in + 2 * self.n_rows * self.n_proj * self.proj_dim
                + 2 * self.n_proj * self.proj_dim * self.c_in + 8 * self.c_in
                + (4 * self.n_proj * self.proj_dim if self.bias else 0))


PROJ_WORKLOADS = [
    ProjWorkload("proj_msa_bf16", 128 * 256, 256, 8 * 32, seed=3001,
                 description="MSA row/column attention input: 128 x 256 tokens, c_m = 256 -> q,k,v,g [H=8, d=32]"),
    ProjWorkload("proj_tri_bf16", 256 * 256, 128, 4 * 32, seed=3002,
                 description="triangle attention input: 256 x 256 pairs, c_z = 128 -> q,k,v,g [H=4, d=32]"),
    ProjWorkload("proj_extra_msa_bf16", 1024 * 256, 64, 8 * 8, seed=3003,
                 description="extra-MSA attention input: 1024 x 256 tokens, c_e = 64 -> q,k,v,g [H=8, d=8]"),
]


def proj_by_name(name: str) -> ProjWorkload:
    for w in PROJ_WORKLOADS:
        if w.name == name:
            return w
    raise KeyError(name)


def generate_proj(w: ProjWorkload, seed: Optional[int] = None, n_rows: Optional[int] = None
                  ) -> Dict[str, np.ndarray]:
    """x [R, C] and weight [P*HD, C] as bf16 bits; ln_weight, ln_bias [C] and
    bias [P*HD] (or None) as fp32."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    R = w.n_rows if n_rows is None else n_rows
    C, F = w.c_in, w.n_proj * w.proj_dim
    offset = rng.standard_normal((R, 1)) * 2.0
    spread = rng.uniform(0.25, 4.0, size=(R, 1))
    x = rng.standard_normal((R, C)) * spread + offset
    lnw = (1.0 + 0.2 * rng.standard_normal(C)).astype(np.float32)
    lnb = (0.2 * rng.standard_normal(C)).astype(np.float32)
    W = rng.standard_normal((F, C)) / math.sqrt(C)
    b = (0.1 * rng.standard_normal(F)).astype(np.float32) if w.bias else None
    return {"x": _store(x, "bf16"), "ln_weight": lnw, "ln_bias": lnb, "weight": _store(W, "bf16"), "bias": b}


# ---------------------------------------------------------------------------
# Pair bias: LayerNorm(z) -> H logit biases per residue pair at the 256 crop
# (c_z = 128).  Weights ~ N(0, 1/C); the rest as in the other generators.
# Draw order: entry offset, entry spread, z, ln weight, ln bias, weight.

@dataclasses.dataclass(frozen=True)
class PairBiasWorkload:
    name: str
    n_batch: int
    seq_len: int
    c_in: int
    n_heads: int
    transpose: bool = False
    eps: float = 1e-5
    seed: int = 0
    description: str = ""

    def bytes(self) -> int:
        B, L, C, H = self.n_batch, self.seq_len, self.c_in, self.n_heads
        return 2 * B * L * L * C + 2 * B * H * L * L + 2 * H * C + 8 * C


PAIR_BIAS_WORKLOADS = [
    PairBiasWorkload("pb_msa_row_bf16", 1, 256, 128, 8, seed=4001,
                     description="MSA row attention pair bias: z [256, 256, 128] -> [8, 256, 256]"),
    PairBiasWorkload("pb_tri_start_bf16", 1, 256, 128, 4, seed=4002,
                     description="triangle attention (starting node) bias: z [256, 256, 128] -> [4, 256, 256]"),
    PairBiasWorkload("pb_tri_end_bf16", 1, 256, 128, 4, transpose=True, seed=4003,
                     description="triangle attention (ending node) bias, transposed layout"),
]


def pair_bias_by_name(name: str) -> PairBiasWorkload:
    for w in PAIR_BIAS_WORKLOADS:
        if w.name == name:
            return w
    raise KeyError(name)


def generate_pair_bias(w: PairBiasWorkload, seed: Optional[int] = None) -> Dict[str, np.ndarray]:
    """z [B, L, L, C] and weight [H, C] as bf16 bits; ln_weight, ln_bias fp32."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    B, L, C, H = w.n_batch, w.seq_len, w.c_in, w.n_heads
    offset = rng.standard_normal((B, L, L, 1)) * 2.0
    spread = rng.uniform(0.25, 4.0, size=(B, L, L, 1))
    z = rng.standard_normal((B, L, L, C)) * spread + offset
    lnw = (1.0 + 0.2 * rng.standard_normal(C)).astype(np.float32)
    lnb = (0.2 * rng.standard_normal(C)).astype(np.float32)
    W = rng.standard_normal((H, C)) / math.sqrt(C)
    return {"z": _store(z, "bf16"), "ln_weight": lnw, "ln_bias": lnb, "weight": _store(W, "bf16")}


# ---------------------------------------------------------------------------
# Optimizer step: the parameter tensors of an AlphaFold-sized model.  The
# paper trains a 97M-parameter model with over four thousand gradient tensors
# (ScaleFold Sections 2.2 and 3.3); the shapes below follow the Evoformer
# block at the standard widths (c_m = 256, c_z = 128, 8 MSA heads of 32,
# 4 pair heads of 32, transitions x4, outer product mean c = 32, triangle
# multiplication c = 128), repeated for 48 main blocks, 4 extra-MSA blocks
# (c_e = 64) and 2 template pair blocks (c_t = 64), plus embedding and
# structure-module sized extras.  Values: params ~ N(0, 0.02^2), grads ~
# N(0, 1e-3^2), Adam moments from a few earlier steps (m ~ N(0, 1e-4^2),
# v ~ |N(0, 1e-6^2)|), SWA copy = params + N(0, 1e-4^2).

def _evoformer_block_shapes(c_m: int, c_z: int, pair_only: bool = False):
    s = []

    def lin(cin, cout, bias=True):
        s.append((cout, cin))
        if bias:
            s.append((cout,))

    def ln(c):
        s.extend([(c,), (c,)])

    hm, dm, hz, dz = 8, 32, 4, 32
    if not pair_only:
        # MSA row attention with pair bias, MSA column attention, MSA transition, outer product mean
        ln(c_m); ln(c_z); lin(c_z, hm, bias=False)
        for _ in range(3):
            lin(c_m, hm * dm, bias=False)
        lin(c_m, hm * dm); lin(hm * dm, c_m)
        ln(c_m)
        for _ in range(3):
            lin(c_m, hm * dm, bias=False)
        lin(c_m, hm * dm); lin(hm * dm, c_m)
        ln(c_m); lin(c_m, 4 * c_m); lin(4 * c_m, c_m)
        ln(c_m); lin(c_m, 32); lin(c_m, 32); lin(32 * 32, c_z)
    # triangle multiplication (outgoing, incoming)
    for _ in range(2):
        ln(c_z)
        for _ in range(4):
            lin(c_z, 128)
        lin(c_z, c_z); ln(128); lin(128, c_z)
    # triangle attention (starting, ending node)
    for _ in range(2):
        ln(c_z); lin(c_z, hz, bias=False)
        for _ in range(3):
            lin(c_z, hz * dz, bias=False)
        lin(c_z, hz * dz); lin(hz * dz, c_z)
    # pair transition
    ln(c_z); lin(c_z, 4 * c_z); lin(4 * c_z, c_z)
    return s


def alphafold_param_shapes():
    shapes = []
    for _ in range(48):
        shapes += _evoformer_block_shapes(256, 128)
    for _ in range(4):
        shapes += _evoformer_block_shapes(64, 128)
    for _ in range(2):
        shapes += _evoformer_block_shapes(64, 64, pair_only=True)
    # embedders, recycling, structure module and heads (approximate sizes)
    extras = [(256, 49), (256,), (128, 22), (128,), (128, 22), (128,), (128, 65), (128,), (64, 25), (64,),
              (256, 256), (256,), (128, 15), (128,), (384, 256), (384,), (384, 384), (384,), (384, 384), (384,),
              (1152, 384), (1152,), (384, 1152), (384,), (128, 384), (128,), (50, 128), (50,), (64, 128), (64,),
              (23, 256), (23,), (37 * 14, 384), (256, 39), (128, 39)]
    for _ in range(8):
        extras += [(384, 384), (384,), (384,), (384,)]
    return shapes + extras


@dataclasses.dataclass(frozen=True)
class OptimWorkload:
    name: str
    subset: int = 0          # 0 = all tensors, else every subset-th tensor
    max_norm: float = 0.1
    lr: float = 1e-3
    betas: tuple = (0.9, 0.999)
    eps: float = 1e-6
    swa_decay: float = 0.999
    step: int = 10
    seed: int = 0
    description: str = ""

    def shapes(self):
        sh = alphafold_param_shapes()
        return sh if not self.subset else sh[::self.subset]

    def numel(self) -> int:
        return int(sum(int(np.prod(s)) for s in self.shapes()))

    def bytes_step(self) -> int:
        # read p, g, m, v, swa; write p, m, v, swa (fp32)
        return 36 * self.numel()

    def bytes_clip(self) -> int:
        return 4 * self.numel()


OPTIM_WORKLOADS = [
    OptimWorkload("adam_swa_alphafold", seed=5001,
                  description="all parameter tensors of an AlphaFold-sized model (fp32 master weights)"),
    OptimWorkload("adam_swa_small", subset=37, seed=5002,
                  description="every 37th tensor of the same model (a parity-test size)"),
]


def optim_by_name(name: str) -> OptimWorkload:
    for w in OPTIM_WORKLOADS:
        if w.name == name:
            return w
    raise KeyError(name)


def generate_optim(w: OptimWorkload, seed: Optional[int] = None):
    """Lists of fp32 arrays: params, grads, exp_avg, exp_avg_sq, swa (one per tensor)."""
    rng = np.random.Generator(np.random.PCG64(w.seed if seed is None else seed))
    out = {k: [] for k in ("params", "grads", "exp_avg", "exp_avg_sq", "swa")}
    for s in w.shapes():
        p = rng.standard_normal(s, dtype=np.float32) * np.float32(0.02)
        out["params"].append(p)
        out["grads"].append(rng.standard_normal(s, dtype=np.float32) * np.float32(1e-3))
        out["exp_avg"].append(rng.standard_normal(s, dtype=np.float32) * np.float32(1e-4))
        out["exp_avg_sq"].append(np.abs(rng.standard_normal(s, dtype=np.float32)) * np.float32(1e-6))
        out["swa"].append(p + rng.standard_normal(s, dtype=np.float32) * np.float32(1e-4))
    return out
