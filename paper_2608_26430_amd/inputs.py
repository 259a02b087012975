"""Seeded synthetic workloads for the FrameFT adapter path.

This module only draws random inputs and describes workload shapes; it holds
none of the method's arithmetic.  It is the one module that both the oracle
side (tests, CPU baseline) and the GPU side use, so that both consume the very
same numbers.

Workloads stand in for the paper's Llama-2-7B / Llama-70B / ViT-B adapter
layers (Sec. 4; throughput table "Tokens per second for different PEFT
methods"); no dataset or pretrained weight is involved:

* activations x and upstream gradients g are i.i.d. N(0, 1);
* coefficient values are N(0, 0.02) in fp32 (the adapter is kept in fp32,
  Sec. 3.4, "Storage efficiency");
* the support of C is uniform over the m x n coefficient grid, drawn without
  replacement (Sec. 3.3: random support, shared across layers);
* W0 ~ N(0, 1/n);
* bf16 tensors are fp32 draws rounded to nearest-even bf16 here, before either
  side sees them, so the oracle (which widens them to fp64) and the GPU read
  identical values;
* generator: numpy PCG64, seed 264300 + config number (+50 for the ViT
  layer of config 5, +100*layer + projection for the layer stack).
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np

SEED_BASE = 264300


@dataclass(frozen=True)
class Adapter:
    """One adapted linear layer W0 (d_out x d_in) and its two frames."""
    name: str
    d_in: int
    d_out: int
    rho_in: int
    rho_out: int
    nnz: int

    @property
    def k_in(self) -> int:
        return self.d_in // self.rho_in

    @property
    def k_out(self) -> int:
        return self.d_out // self.rho_out


@dataclass(frozen=True)
class Workload:
    """A configuration: adapters applied to `tokens` tokens in `dtype`."""
    name: str
    tokens: int
    dtype: str                # "f32" or "bf16"
    alpha: float              # scale s = alpha / sqrt(d_out * d_in)
    adapters: tuple = field(default_factory=tuple)
    layers: int = 1           # the stack repeats `adapters` per layer
    seed: int = SEED_BASE


def _q(d):
    return Adapter("q_proj", d, d, 64, 64, 10_000)


WORKLOADS = {
    # 256 x 256 fp32 layer, frame (16 subspaces of dim 16), 512 coefficients.
    "cfg1_256_fp32": Workload("cfg1_256_fp32", 64, "f32", 20.0,
                              (Adapter("linear", 256, 256, 16, 16, 512),), seed=SEED_BASE + 1),
    # Llama-2-7B q_proj 4096 x 4096, 64 subspaces of dim 64, 10k coefficients, 8 x 512 tokens.
    "cfg2_llama7b_qproj": Workload("cfg2_llama7b_qproj", 4096, "bf16", 200.0,
                                   (_q(4096),), seed=SEED_BASE + 2),
    # Llama-2-7B MLP up 4096 -> 11008 and down 11008 -> 4096, subspace dim 64, 50k coefficients.
    "cfg3_llama7b_mlp": Workload("cfg3_llama7b_mlp", 4096, "bf16", 200.0,
                                 (Adapter("up_proj", 4096, 11008, 64, 64, 50_000),
                                  Adapter("down_proj", 11008, 4096, 64, 64, 50_000)),
                                 seed=SEED_BASE + 3),
    # Full Llama-2-7B adapter stack: 32 layers x 7 projections, 10k coefficients each.
    "cfg4_llama7b_stack": Workload("cfg4_llama7b_stack", 2048, "bf16", 200.0,
                                   (Adapter("q_proj", 4096, 4096, 64, 64, 10_000),
                                    Adapter("k_proj", 4096, 4096, 64, 64, 10_000),
                                    Adapter("v_proj", 4096, 4096, 64, 64, 10_000),
                                    Adapter("o_proj", 4096, 4096, 64, 64, 10_000),
                                    Adapter("gate_proj", 4096, 11008, 64, 64, 10_000),
                                    Adapter("up_proj", 4096, 11008, 64, 64, 10_000),
                                    Adapter("down_proj", 11008, 4096, 64, 64, 10_000)),
                                   layers=32, seed=SEED_BASE + 4),
    # Llama-70B down_proj 28672 -> 8192, subspace dim 128, 200k coefficients, 8192 tokens.
    "cfg5_llama70b_down": Workload("cfg5_llama70b_down", 8192, "bf16", 200.0,
                                   (Adapter("down_proj", 28672, 8192, 128, 128, 200_000),),
                                   seed=SEED_BASE + 5),
    # ViT-B/16 qkv 768 -> 2304, 64 images x 197 tokens, 3k coefficients.
    "cfg5_vitb16_qkv": Workload("cfg5_vitb16_qkv", 64 * 197, "bf16", 250.0,
                                (Adapter("qkv", 768, 2304, 64, 64, 3_000),),
                                seed=SEED_BASE + 5 + 50),
    # The paper's own frames (Sec. 4.1, 4.2): subspace dimension 2, k rho = d, so each frame is
    # one realified DFT of size d/2.  Llama-2-7B q_proj with the instruction-tuning support of
    # 5000 coefficients, and a RoBERTa-large-sized 1024-wide query with 1000 coefficients.
    "rho2_llama7b_qproj": Workload("rho2_llama7b_qproj", 4096, "bf16", 200.0,
                                   (Adapter("q_proj", 4096, 4096, 2, 2, 5_000),), seed=SEED_BASE + 6),
    "rho2_roberta_large_query": Workload("rho2_roberta_large_query", 4096, "bf16", 20.0,
                                         (Adapter("query", 1024, 1024, 2, 2, 1_000),), seed=SEED_BASE + 7),
}


def scale_for(workload: Workload, adapter: Adapter) -> float:
    """s = alpha / sqrt(m n) with m = d_out, n = d_in."""
    return float(workload.alpha / np.sqrt(float(adapter.d_out) * float(adapter.d_in)))


def rng(seed: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed))


def bf16_round(a: np.ndarray) -> np.ndarray:
    """Round fp32 values to the nearest bf16 (ties to even); returns fp32 holding bf16 values."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounded = (u + 0x7FFF + ((u >> 16) & 1)) & 0xFFFF0000
    out = rounded.astype(np.uint32).view(np.float32)
    return np.where(np.isnan(a), a, out)


def bf16_bits(a: np.ndarray) -> np.ndarray:
    """The upper 16 bits of fp32 values that are already bf16-representable."""
    return (np.ascontiguousarray(a, dtype=np.float32).view(np.uint32) >> 16).astype(np.uint16)


def gaussian(g: np.random.Generator, shape, std: float = 1.0, dtype: str = "f32") -> np.ndarray:
    """N(0, std^2) fp32 draws, rounded to bf16 when dtype == 'bf16'."""
    x = (g.standard_normal(size=shape, dtype=np.float32) * np.float32(std)).astype(np.float32)
    return bf16_round(x) if dtype == "bf16" else x


def support(g: np.random.Generator, m: int, n: int, nnz: int):
    """nnz distinct positions drawn uniformly from the m x n grid (rows, cols as int32)."""
    if nnz > m * n:
        raise ValueError("nnz exceeds the grid")
    flat = g.choice(m * n, size=nnz, replace=False)
    return (flat // n).astype(np.int32), (flat % n).astype(np.int32)


def support_block_diagonal(g: np.random.Generator, k: int, rho_out: int, rho_in: int, nnz: int):
    """nnz distinct positions drawn uniformly from the diagonal blocks of C = diag(C_1..C_k).

    Sec. 3.1 writes C as block diagonal, block i (rho_out x rho_in) coupling output subspace i
    with input subspace i; Sec. 3.3 spreads the nonzeros uniformly across those blocks.  In the
    subspace-major coefficient order (P = [P_1 ... P_k]) block i covers rows
    [i rho_out, (i + 1) rho_out) and columns [i rho_in, (i + 1) rho_in).  Both frames must have
    the same number k of subspaces.
    """
    per = rho_out * rho_in
    if nnz > k * per:
        raise ValueError("nnz exceeds the diagonal blocks")
    flat = g.choice(k * per, size=nnz, replace=False)
    blk, within = flat // per, flat % per
    rows = blk * rho_out + within // rho_in
    cols = blk * rho_in + within % rho_in
    return rows.astype(np.int32), cols.astype(np.int32)


@dataclass
class AdapterData:
    """Host arrays for one adapter call: all fp32 (bf16-valued when dtype is bf16)."""
    adapter: Adapter
    scale: float
    rows: np.ndarray
    cols: np.ndarray
    vals: np.ndarray
    X: np.ndarray
    G: np.ndarray


def adapter_data(workload: Workload, adapter: Adapter, seed: int | None = None,
                 tokens: int | None = None, support_seed: int | None = None) -> AdapterData:
    """Draw support, coefficient values, X (T x d_in) and G (T x d_out) for one adapter."""
    seed = workload.seed if seed is None else seed
    T = workload.tokens if tokens is None else tokens
    gs = rng(seed if support_seed is None else support_seed)
    rows, cols = support(gs, adapter.d_out, adapter.d_in, adapter.nnz)
    g = rng(seed + 7919)
    vals = gaussian(g, (adapter.nnz,), std=0.02, dtype="f32")
    X = gaussian(g, (T, adapter.d_in), dtype=workload.dtype)
    G = gaussian(g, (T, adapter.d_out), dtype=workload.dtype)
    return AdapterData(adapter, scale_for(workload, adapter), rows, cols, vals, X, G)


def weight(g: np.random.Generator, d_out: int, d_in: int, dtype: str) -> np.ndarray:
    """Frozen weight W0 ~ N(0, 1/d_in), d_out x d_in row-major."""
    return gaussian(g, (d_out, d_in), std=1.0 / np.sqrt(d_in), dtype=dtype)
