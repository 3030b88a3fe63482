"""Byte and launch-size arithmetic stated in the paper, written out plainly.

TEST INFRASTRUCTURE ONLY (see ``oracle/pq_oracle.py``).  These helpers restate
the paper's storage formula and its GPU auto-tuner rules so that the tests can
check them against the numbers the paper prints; the library makes its own
launch choices for a different GPU and does not use them.
"""

from __future__ import annotations

import math

__all__ = [
    "id_bits",
    "layer_footprint_bits",
    "effective_bits",
    "index_table_bytes",
    "subspace_codebook_bytes",
    "gemv_ksplit",
    "gemm_splits",
    "lut_waste_fraction",
    "double_buffered_lut_bytes",
]


def id_bits(k_s: int) -> int:
    """Storage bits of one id: ceil(log2 K_s) (Sec. 3.2)."""
    if k_s < 1:
        raise ValueError("K_s must be >= 1")
    return math.ceil(math.log2(k_s)) if k_s > 1 else 0


def layer_footprint_bits(k_s: int, n_ss: int, sz_ss: int, dim_dp: int) -> int:
    """Eq. reduced-model-size: per-subspace codebooks plus the index table.

    ``16 * K_s * dim_ss`` bits of fp16 centroids (``N_ss`` tables of ``K_s``
    centroids of ``SZ_ss`` values, ``dim_ss = N_ss * SZ_ss``) plus
    ``ceil(log2 K_s) * N_ss * dim_dp`` bits of ids.
    """
    dim_ss = n_ss * sz_ss
    return 16 * k_s * dim_ss + id_bits(k_s) * n_ss * dim_dp


def effective_bits(k_s: int, sz_ss: int) -> float:
    """#W: index bits per weight, ceil(log2 K_s) / SZ_ss (Sec. 3.2)."""
    return id_bits(k_s) / sz_ss


def index_table_bytes(n_ss: int, f_out: int, bits: int = 8) -> int:
    """Bytes of T_index with ``bits``-bit ids (Sec. 4.1, Sec. 4.4)."""
    return n_ss * f_out * bits // 8


def subspace_codebook_bytes(k_s: int, sz_ss: int) -> int:
    """Bytes of one subspace's fp16 centroid table (Sec. 4.1)."""
    return k_s * sz_ss * 2


def gemv_ksplit(n_sm: int, batch: int, f_out: int, blocks_per_sm: int = 8, block_threads: int = 128) -> int:
    """Decode split-K count from the paper's auto-tuner (Sec. 4.1).

    ``ceil(N_SM * 8 / (B_s * ceil(F_out / 128)))``: enough splits of the
    subspace loop that the grid holds about 8 blocks per SM.
    """
    return math.ceil(n_sm * blocks_per_sm / (batch * math.ceil(f_out / block_threads)))


def gemm_splits(n_sm: int, seq_len: int, blocks_per_sm: int = 6) -> int:
    """Prefill split count for about 6 blocks per SM (Sec. 4.2).

    The paper gives the target (about 6 blocks per SM, one block row per
    token) and the outcome at L = 128 (about 4 splits, 512 blocks) but not the
    rounding; this reading rounds up.
    """
    return max(1, math.ceil(n_sm * blocks_per_sm / seq_len))


def lut_waste_fraction(k_s: int) -> float:
    """Share of a K_s-entry LUT left unused when one token reads one entry (Sec. 4.1)."""
    return 1.0 - 1.0 / k_s


def double_buffered_lut_bytes(k_s: int) -> int:
    """Two fp32 LUT slots padded to K_s + 1 entries (Sec. 4.2)."""
    return 2 * (k_s + 1) * 4
