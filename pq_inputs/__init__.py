"""Seeded synthetic inputs for the product-quantized (PQ) linear layer.

This module is the only code shared by the CPU oracle and the HIP path's tests
and benchmark.  It draws inputs and encodes them into the packed storage format
that the library consumes; it holds none of the layer's arithmetic (no index
decoding, no codeword gather, no dot product).

What is drawn, and in which order (one generator per matrix):

1. codebook: ``C x d`` values from N(0, 0.02), rounded to fp16 (round to
   nearest even, numpy's ``astype``).  The paper stores centroids in FP16
   (Sec. 3.1.2 and the footprint equation of Sec. 3.2).
2. codeword ids: ``N x S`` integers drawn uniformly from ``[0, C)``, with
   ``S = K / d`` sub-vectors per weight row.  Trained k-means ids are skewed;
   uniform ids are the stand-in (the trained weights are not available).
3. activations x: ``M x K`` values from N(0, 1), rounded to fp16.

Each matrix gets its own generator
``default_rng(SeedSequence([seed, workload_id, layer, matrix_id]))`` so that a
single matrix can be regenerated without drawing the others.  The tiny
workload uses ``default_rng(seed)`` directly.

Packed index format (one row of ``R = ceil(S * idx_bits / 8)`` bytes per output
feature, rows back to back):

* ``idx_bits = 8``: byte ``s`` is id ``s``.
* ``idx_bits = 16``: id ``s`` is the little-endian pair of bytes ``2s, 2s+1``.
* ``idx_bits = 12``: a dense least-significant-bit-first stream: id ``s``
  occupies stream bits ``[12 s, 12 s + 12)``; stream bit ``b`` is bit
  ``b mod 8`` of byte ``b div 8``.  The pad nibble of an odd-length row is 0.

All three are the same rule (an LSB-first stream of ``idx_bits``-bit fields);
the encoder below writes 8/16 directly and 12 as byte triples per id pair.
"""

from __future__ import annotations

import dataclasses
from typing import Dict, Iterator, List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "SUPPORTED_IDX_BITS",
    "row_bytes",
    "pack_indices",
    "matrix_rng",
    "draw_codebook",
    "draw_ids",
    "draw_x",
    "PQProblem",
    "draw_problem",
    "MatrixSpec",
    "Workload",
    "WORKLOADS",
    "workload",
    "signed_one_hot_codebook",
    "scaled_signed_one_hot_codebook",
    "ternary_x",
    "subnormal_codebook",
    "subnormal_x",
    "FP16_SUBNORMAL_UNIT",
]

SUPPORTED_IDX_BITS = (8, 12, 16)


def row_bytes(S: int, idx_bits: int) -> int:
    """Bytes of one packed index row holding ``S`` ids of ``idx_bits`` bits."""
    if idx_bits not in SUPPORTED_IDX_BITS:
        raise ValueError(f"idx_bits must be one of {SUPPORTED_IDX_BITS}, got {idx_bits}")
    if S < 0:
        raise ValueError("S must be non-negative")
    return (S * idx_bits + 7) // 8


def pack_indices(ids: np.ndarray, idx_bits: int) -> np.ndarray:
    """Encode an ``[N, S]`` array of codeword ids into ``[N, R]`` uint8 rows."""
    ids = np.asarray(ids)
    if ids.ndim != 2:
        raise ValueError("ids must be 2-D [N, S]")
    if idx_bits not in SUPPORTED_IDX_BITS:
        raise ValueError(f"idx_bits must be one of {SUPPORTED_IDX_BITS}")
    if ids.size and (int(ids.min()) < 0 or int(ids.max()) >= (1 << idx_bits)):
        raise ValueError(f"ids do not fit in {idx_bits} bits")
    N, S = ids.shape
    R = row_bytes(S, idx_bits)
    if idx_bits == 8:
        return np.ascontiguousarray(ids.astype(np.uint8))
    if idx_bits == 16:
        return np.ascontiguousarray(ids.astype("<u2")).view(np.uint8).reshape(N, R)
    # 12 bits: two ids per three bytes.
    u = ids.astype(np.uint32)
    if S % 2:
        u = np.concatenate([u, np.zeros((N, 1), np.uint32)], axis=1)
    u0 = u[:, 0::2]
    u1 = u[:, 1::2]
    out = np.empty((N, u0.shape[1], 3), np.uint8)
    out[:, :, 0] = u0 & 0xFF
    out[:, :, 1] = ((u0 >> 8) & 0x0F) | ((u1 & 0x0F) << 4)
    out[:, :, 2] = (u1 >> 4) & 0xFF
    out = out.reshape(N, -1)
    return np.ascontiguousarray(out[:, :R])


def matrix_rng(seed: int, workload_id: int, layer: int, matrix_id: int) -> np.random.Generator:
    """Independent generator for one matrix of one workload."""
    return np.random.default_rng(np.random.SeedSequence([seed, workload_id, layer, matrix_id]))


def draw_codebook(rng: np.random.Generator, C: int, d: int, std: float = 0.02) -> np.ndarray:
    return rng.normal(0.0, std, size=(C, d)).astype(np.float16)


def draw_ids(rng: np.random.Generator, N: int, S: int, C: int) -> np.ndarray:
    dtype = np.uint16 if C <= (1 << 16) else np.uint32
    return rng.integers(0, C, size=(N, S), dtype=dtype)


def draw_x(rng: np.random.Generator, M: int, K: int) -> np.ndarray:
    return rng.normal(0.0, 1.0, size=(M, K)).astype(np.float16)


@dataclasses.dataclass
class PQProblem:
    """One PQ linear layer instance: ``y[M, N] = x[M, K] . W_hat^T``."""

    M: int
    K: int
    N: int
    d: int
    C: int
    idx_bits: int
    codebook: np.ndarray  # fp16 [C, d]
    ids: np.ndarray  # unsigned [N, S]
    idx: np.ndarray  # uint8 [N, R] packed
    x: np.ndarray  # fp16 [M, K]

    @property
    def S(self) -> int:
        return self.K // self.d

    @property
    def R(self) -> int:
        return self.idx.shape[1]


def draw_problem(
    rng: np.random.Generator,
    M: int,
    K: int,
    N: int,
    d: int,
    C: int,
    idx_bits: int,
    cb_std: float = 0.02,
) -> PQProblem:
    """Draw codebook, then ids, then x, and pack the ids."""
    if K % d:
        raise ValueError("K must be a multiple of d")
    if not (1 <= C <= (1 << idx_bits)):
        raise ValueError("C must lie in [1, 2**idx_bits]")
    S = K // d
    codebook = draw_codebook(rng, C, d, cb_std)
    ids = draw_ids(rng, N, S, C)
    x = draw_x(rng, M, K)
    return PQProblem(M, K, N, d, C, idx_bits, codebook, ids, pack_indices(ids, idx_bits), x)


# ---------------------------------------------------------------------------
# Named workloads: the Llama-3-8B / Qwen3-8B layer shapes the method is run on.
# ---------------------------------------------------------------------------

LLAMA3_8B = (
    ("q_proj", 4096, 4096),
    ("k_proj", 1024, 4096),
    ("v_proj", 1024, 4096),
    ("o_proj", 4096, 4096),
    ("gate_proj", 14336, 4096),
    ("up_proj", 14336, 4096),
    ("down_proj", 4096, 14336),
)

QWEN3_8B = (
    ("q_proj", 4096, 4096),
    ("k_proj", 1024, 4096),
    ("v_proj", 1024, 4096),
    ("o_proj", 4096, 4096),
    ("gate_proj", 12288, 4096),
    ("up_proj", 12288, 4096),
    ("down_proj", 4096, 12288),
)


@dataclasses.dataclass(frozen=True)
class MatrixSpec:
    name: str
    N: int
    K: int


@dataclasses.dataclass(frozen=True)
class Workload:
    name: str
    workload_id: int
    d: int
    C: int
    idx_bits: int
    Ms: Tuple[int, ...]
    matrices: Tuple[MatrixSpec, ...]
    layers: int = 1
    description: str = ""

    def problem(self, matrix: int, M: Optional[int] = None, seed: int = 0, layer: int = 0) -> PQProblem:
        spec = self.matrices[matrix]
        M = self.Ms[0] if M is None else M
        if self.name == "tiny":
            rng = np.random.default_rng(seed)
        else:
            rng = matrix_rng(seed, self.workload_id, layer, matrix)
        return draw_problem(rng, M, spec.K, spec.N, self.d, self.C, self.idx_bits)


def _specs(rows) -> Tuple[MatrixSpec, ...]:
    return tuple(MatrixSpec(n, N, K) for (n, N, K) in rows)


WORKLOADS: Dict[str, Workload] = {
    "tiny": Workload(
        "tiny", 0, d=4, C=256, idx_bits=8, Ms=(1,),
        matrices=(MatrixSpec("tiny", 128, 256),),
        description="M=1, K=256, N=128, d=4, C=256, uint8 ids, seed 0",
    ),
    "llama3_8b_4bit": Workload(
        "llama3_8b_4bit", 1, d=2, C=256, idx_bits=8, Ms=(1,),
        matrices=_specs(LLAMA3_8B),
        description="Llama-3-8B decoder layer, effective 4-bit (d=2, C=256, 8-bit ids), M=1",
    ),
    "llama3_8b_3bit": Workload(
        "llama3_8b_3bit", 2, d=4, C=4096, idx_bits=12, Ms=(1,),
        matrices=_specs(LLAMA3_8B) + (MatrixSpec("lm_head", 128256, 4096),),
        description="Llama-3-8B decoder layer + lm_head, effective 3-bit (d=4, C=4096, 12-bit ids), M=1",
    ),
    "prefill": Workload(
        "prefill", 3, d=4, C=256, idx_bits=8, Ms=(128, 512, 2048),
        matrices=_specs((("q_proj", 4096, 4096), ("gate_proj", 14336, 4096), ("down_proj", 4096, 14336))),
        description="Llama-3-8B prefill shapes, d=4, C=256, 8-bit ids, M in {128, 512, 2048}",
    ),
    "qwen3_8b_sweep": Workload(
        "qwen3_8b_sweep", 4, d=4, C=65536, idx_bits=16, Ms=(1, 4, 16),
        matrices=_specs(QWEN3_8B), layers=36,
        description="Qwen3-8B decoder layers, d=4, C=65536 (512 KiB codebook), 16-bit ids, M in {1, 4, 16}",
    ),
}


def workload(name: str) -> Workload:
    return WORKLOADS[name]


# ---------------------------------------------------------------------------
# Structured inputs whose layer output has a closed form.
# ---------------------------------------------------------------------------

def signed_one_hot_codebook(C: int, d: int, rng: Optional[np.random.Generator] = None) -> np.ndarray:
    """Codeword k is +-e_(k mod d) (a signed unit vector), as fp16.

    Signs are random when ``rng`` is given, else alternate with ``k div d``.
    """
    cb = np.zeros((C, d), np.float16)
    k = np.arange(C)
    if rng is None:
        sign = np.where((k // d) % 2 == 0, 1.0, -1.0)
    else:
        sign = rng.choice([-1.0, 1.0], size=C)
    cb[k, k % d] = sign.astype(np.float16)
    return cb


def scaled_signed_one_hot_codebook(C: int, d: int, rng: np.random.Generator) -> Tuple[np.ndarray, np.ndarray]:
    """Codeword k is sign_k * 2**-((k div d) mod 4) * e_(k mod d), fp16.

    Returns the codebook and the per-codeword signs (+-1, float64).
    """
    k = np.arange(C)
    sign = rng.choice([-1.0, 1.0], size=C)
    scale = 2.0 ** (-((k // d) % 4))
    cb = np.zeros((C, d), np.float16)
    cb[k, k % d] = (sign * scale).astype(np.float16)
    return cb, sign


def ternary_x(rng: np.random.Generator, M: int, K: int) -> np.ndarray:
    """Activations drawn uniformly from {-1, 0, 1}, fp16."""
    return rng.integers(-1, 2, size=(M, K)).astype(np.float16)


# The smallest positive fp16 subnormal, 2**-24.  Every fp16 subnormal is an
# integer k (1 <= k <= 1023) times it.
FP16_SUBNORMAL_UNIT = 2.0 ** -24


def _signed_subnormal_bits(rng: np.random.Generator, shape, large_frac: float) -> np.ndarray:
    """fp16 bit patterns of +-k * 2**-24 with k in {0, 1, 2, 3} (k = 0 gives
    +0 or -0), a `large_frac` share of them replaced by k in {512, 1023} (the
    largest subnormal).  Every value is an fp16 subnormal or a signed zero."""
    k = rng.integers(0, 4, size=shape).astype(np.uint16)
    if large_frac > 0.0:
        big = rng.random(size=shape) < large_frac
        k = np.where(big, rng.choice(np.array([512, 1023], np.uint16), size=shape), k)
    sign = rng.integers(0, 2, size=shape).astype(np.uint16) << np.uint16(15)
    return (k | sign).astype(np.uint16)


def subnormal_codebook(rng: np.random.Generator, C: int, d: int, large_frac: float = 0.0) -> np.ndarray:
    """A ``C x d`` fp16 codebook made only of subnormals and signed zeros
    (+-k * 2**-24, see ``_signed_subnormal_bits``), for checking that no
    kernel flushes fp16 subnormal codewords."""
    return _signed_subnormal_bits(rng, (C, d), large_frac).view(np.float16)


def subnormal_x(rng: np.random.Generator, M: int, K: int, large_frac: float = 0.0) -> np.ndarray:
    """``M x K`` fp16 activations made only of subnormals and signed zeros."""
    return _signed_subnormal_bits(rng, (M, K), large_frac).view(np.float16)


# ---------------------------------------------------------------------------
# Encoder inputs: a dense fp16 weight matrix and the starting codebook.  The
# starting points are random numbers the encoder would otherwise draw, so both
# the CPU oracle and the GPU encoder receive them as inputs.
# ---------------------------------------------------------------------------

def draw_weights(rng: np.random.Generator, N: int, K: int, std: float = 0.02) -> np.ndarray:
    """Dense weights ``N x K`` from N(0, std), rounded to fp16 (a stand-in for a
    trained layer, whose weights are not available)."""
    return (rng.standard_normal((N, K)) * std).astype(np.float16)


def init_point_ids(rng: np.random.Generator, n_points: int, C: int) -> np.ndarray:
    """``C`` distinct sub-vector indices in ``[0, n_points)`` (sorted): where
    k-means starts."""
    if C > n_points:
        raise ValueError("more codewords than sub-vectors")
    return np.sort(rng.choice(n_points, size=C, replace=False)).astype(np.int64)


def subvectors_at(w: np.ndarray, d: int, point_ids: np.ndarray) -> np.ndarray:
    """Sub-vectors ``point_ids`` of ``w`` (point ``n * (K / d) + s`` is
    ``w[n, s*d:(s+1)*d]``), as an fp16 ``[len(point_ids), d]`` array (a copy)."""
    N, K = w.shape
    return np.ascontiguousarray(w.reshape(N * (K // d), d)[point_ids])
