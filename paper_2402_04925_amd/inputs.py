"""Seeded synthetic inputs for the TP-aware dequantization workloads.

This module only draws random numbers and lays them out in the storage format
the library consumes. It holds none of the method's arithmetic (no dequant, no
sort, no permutation of weights), so that the CPU oracle and the HIP path can
both take their inputs from it without sharing any computation.

Workloads (MLP problem sizes of the paper's experiments section):
  * Llama-70B MLP: hidden 8192, intermediate 28672 (single up_proj then
    down_proj, no gate).
  * Granite-20B MLP: hidden 6144, intermediate 24576.
Act-order is emulated as in Eq. 2-3: a seeded random permutation phi of the
K input channels and g_idx[i] = floor(phi(i) / G).

Storage format (the library's, fixed here):
  qweight int32 [K/8][N]   nibble j (bits 4j..4j+3) of word [r][n] = row 8r+j
  scales  fp16  [K/G][N]   (or bfloat16 values, held in float32 arrays)
  qzeros  int32 [K/G][N/8] nibble j of word [g][c] = column 8c+j
Uniform int4 codes packed eight to a word are exactly uniform 32-bit words, so
qweight and qzeros are drawn as random words.
"""
from __future__ import annotations

import dataclasses

import numpy as np

BASE_SEED = 20240207

# tensor ids for the per-tensor streams (T_*U: the up projection of a gated
# MLP, whose act-order permutation is W1's: both read the same input)
T_PHI1, T_PHI2, T_QW1, T_QW2, T_S1, T_S2, T_Z1, T_Z2, T_X = range(9)
T_QWU, T_SU, T_ZU = 9, 10, 11


@dataclasses.dataclass(frozen=True)
class Workload:
    """One MLP (or single GEMM) problem: global sizes plus the TP degree.

    K1 = hidden (input features of the column-parallel W1), N1 = intermediate
    (W1 output features = W2 input features K2), N2 = W2 output features.
    A workload with N2 == 0 is a single GEMM (only W1).
    """
    name: str
    cfg_id: int
    K1: int
    N1: int
    N2: int
    G: int
    tp: int
    Ms: tuple

    @property
    def K2(self) -> int:
        return self.N1


WORKLOADS = {
    "tiny_gemm": Workload("tiny_gemm", 0, 256, 128, 0, 32, 1, (4,)),
    "llama70b_tp8": Workload("llama70b_tp8", 1, 8192, 28672, 8192, 128, 8, (1, 4, 16)),
    "granite20b_tp4": Workload("granite20b_tp4", 2, 6144, 24576, 6144, 128, 4, (1, 8, 16)),
    "llama70b_tp1": Workload("llama70b_tp1", 3, 8192, 28672, 8192, 128, 1, (1, 16, 64)),
    "llama70b_tp2_prefill": Workload("llama70b_tp2_prefill", 4, 8192, 28672, 8192, 128, 2, (2048,)),
}


def rng_for(cfg_id: int, tensor_id: int, seed: int = BASE_SEED) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64([seed, cfg_id, tensor_id]))


def random_permutation(n: int, rng: np.random.Generator) -> np.ndarray:
    """phi of Eq. 2: a uniformly random permutation of 0..n-1 (int32)."""
    return rng.permutation(n).astype(np.int32)


def actorder_gidx(phi: np.ndarray, G: int) -> np.ndarray:
    """Input synthesis by Eq. 3: g_idx[i] = floor(phi(i) / G)."""
    return (phi // G).astype(np.int32)


def random_words(shape, rng: np.random.Generator) -> np.ndarray:
    """Uniform 32-bit words = eight uniform int4 codes each."""
    return rng.integers(0, 1 << 32, size=shape, dtype=np.uint64).astype(np.uint32).view(np.int32)


BF16 = "bf16"  # dtype tag: bfloat16 values held in float32 arrays


def _store(a: np.ndarray, dtype) -> np.ndarray:
    """The drawn values in the storage type: numpy's cast for fp16; for
    bfloat16, torch's CPU cast of the float32 values, kept in float32."""
    if dtype == BF16:
        import torch
        t = torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(torch.bfloat16)
        return t.to(torch.float32).numpy()
    return a.astype(dtype)


def random_scales(shape, rng: np.random.Generator, lo=0.002, hi=0.02, dtype=np.float16) -> np.ndarray:
    return _store(rng.uniform(lo, hi, size=shape), dtype)


def random_activations(M: int, K: int, rng: np.random.Generator, dtype=np.float16) -> np.ndarray:
    return _store(rng.standard_normal((M, K)), dtype)


@dataclasses.dataclass
class QuantLinear:
    """One GPTQ-style act-order layer in the library's storage format."""
    qweight: np.ndarray   # int32 [K/8][N]
    scales: np.ndarray    # fp16 [K/G][N] (bf16 layers: float32 holding bf16 values)
    qzeros: np.ndarray    # int32 [K/G][N/8]
    g_idx: np.ndarray     # int32 [K]
    phi: np.ndarray       # int32 [K], the emulated act-order permutation
    G: int

    @property
    def K(self) -> int:
        return self.qweight.shape[0] * 8

    @property
    def N(self) -> int:
        return self.qweight.shape[1]


def make_layer(K: int, N: int, G: int, cfg_id: int, t_phi: int, t_qw: int, t_s: int, t_z: int,
               seed: int = BASE_SEED, scale_dtype=np.float16) -> QuantLinear:
    """An act-order layer by Eq. 2-3; when G does not divide K the last of the
    ceil(K / G) groups is partial."""
    if K % 8 or N % 8 or G % 8 or G <= 0:
        raise ValueError(f"unsupported layer shape K={K} N={N} G={G}")
    ng = -(-K // G)
    phi = random_permutation(K, rng_for(cfg_id, t_phi, seed))
    return QuantLinear(
        qweight=random_words((K // 8, N), rng_for(cfg_id, t_qw, seed)),
        scales=random_scales((ng, N), rng_for(cfg_id, t_s, seed), dtype=scale_dtype),
        qzeros=random_words((ng, N // 8), rng_for(cfg_id, t_z, seed)),
        g_idx=actorder_gidx(phi, G),
        phi=phi,
        G=G,
    )


def unequal_gidx(phi: np.ndarray, sizes: np.ndarray) -> np.ndarray:
    """Input synthesis for groups of unequal size (a checkpoint's own
    grouping): row i belongs to group g when phi(i) lies in
    [sizes[0] + .. + sizes[g-1], sizes[0] + .. + sizes[g]), the unequal-size
    form of Eq. 3."""
    bounds = np.cumsum(np.asarray(sizes, dtype=np.int64))
    return np.searchsorted(bounds, np.asarray(phi, dtype=np.int64), side="right").astype(np.int32)


T_SIZES = 12  # stream of the group sizes of an unequal-group layer


def make_unequal_layer(K: int, N: int, ng: int, seed: int, cfg_id: int = 101, layer: int = 0,
                       scale_dtype=np.float16) -> QuantLinear:
    """An act-order layer whose ng groups have unequal sizes (multinomial over
    the groups, so some may be small or empty); G = 0 marks the grouping as
    given by g_idx alone."""
    if K % 8 or N % 8 or ng < 1:
        raise ValueError(f"unsupported layer shape K={K} N={N} ng={ng}")
    t = 16 * layer
    sizes = rng_for(cfg_id, t + T_SIZES, seed).multinomial(K, np.full(ng, 1.0 / ng))
    phi = random_permutation(K, rng_for(cfg_id, t + T_PHI1, seed))
    return QuantLinear(
        qweight=random_words((K // 8, N), rng_for(cfg_id, t + T_QW1, seed)),
        scales=random_scales((ng, N), rng_for(cfg_id, t + T_S1, seed), dtype=scale_dtype),
        qzeros=random_words((ng, N // 8), rng_for(cfg_id, t + T_Z1, seed)),
        g_idx=unequal_gidx(phi, sizes),
        phi=phi,
        G=0,
    )


def make_workload(w: Workload, seed: int = BASE_SEED, scale_dtype=np.float16):
    """Global (unsharded) layers of a workload: (W1, W2-or-None)."""
    w1 = make_layer(w.K1, w.N1, w.G, w.cfg_id, T_PHI1, T_QW1, T_S1, T_Z1, seed, scale_dtype)
    w2 = None
    if w.N2:
        w2 = make_layer(w.K2, w.N2, w.G, w.cfg_id, T_PHI2, T_QW2, T_S2, T_Z2, seed, scale_dtype)
    return w1, w2


def make_gated_workload(w: Workload, seed: int = BASE_SEED, scale_dtype=np.float16):
    """Global layers of the gated form of a workload: (gate, up, down). gate
    and down are make_workload's W1 and W2; up has gate's shape and act-order
    permutation (hence its g_idx) and codes, scales and zeros of its own."""
    gate, down = make_workload(w, seed, scale_dtype)
    up = make_layer(w.K1, w.N1, w.G, w.cfg_id, T_PHI1, T_QWU, T_SU, T_ZU, seed, scale_dtype)
    return gate, up, down


def make_x(w: Workload, M: int, seed: int = BASE_SEED, dtype=np.float16) -> np.ndarray:
    rng = np.random.Generator(np.random.PCG64([seed, w.cfg_id, T_X, M]))
    return random_activations(M, w.K1, rng, dtype)


def make_custom(K1: int, N1: int, N2: int, G: int, seed: int, cfg_id: int = 100, identity_phi=False,
                scale_dtype=np.float16):
    """Small ad-hoc layers for tests (ragged shapes, special cases)."""
    w1 = make_layer(K1, N1, G, cfg_id, T_PHI1, T_QW1, T_S1, T_Z1, seed, scale_dtype)
    w2 = make_layer(N1, N2, G, cfg_id, T_PHI2, T_QW2, T_S2, T_Z2, seed, scale_dtype) if N2 else None
    if identity_phi:
        for w in (w1, w2):
            if w is not None:
                w.phi = np.arange(w.K, dtype=np.int32)
                w.g_idx = actorder_gidx(w.phi, G)
    return w1, w2
