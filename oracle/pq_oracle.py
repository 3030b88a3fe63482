"""CPU oracle for the FASQ product-quantized linear layer (fp64, NumPy).

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports, links or calls this
module; only the tests, the smoke check and the benchmark's CPU-baseline leg
use it.  It shares no code with the HIP path: it decodes the packed indices,
gathers codewords and multiplies with code written here and nowhere else.

What it computes (paper: Sec. 3.1.2, Eq. lut-accumulate; Sec. 2.2):

A PQ-compressed weight matrix ``W_hat`` with ``N`` output features and ``K``
input features is split along K into ``S = K / d`` sub-vectors of length ``d``
per output row.  Sub-vector ``s`` of row ``n`` is replaced by the id
``u(n, s)`` of one of ``C`` fp16 codewords, so

    W_hat[n, s*d + i] = codebook[u(n, s), i]                     (reconstruct)
    y[m, n]           = sum_k x[m, k] * W_hat[n, k]              (dense matmul)
                      = sum_s dot(x[m, s*d:(s+1)*d], codebook[u(n, s)])

The last line is Eq. lut-accumulate with every subspace using the same
codebook; it is an exact rewrite of the dense product, so the oracle uses the
plain definition (reconstruct, then an fp64 matmul) and, separately, the
paper's per-subspace form (``lut_accumulate``), which also accepts one
codebook per subspace.

Readings of the paper used here (the paper is silent or ambiguous):

* sub-vectors run along the reduction axis K, one id per (output row,
  subspace), as Eq. lut-accumulate and the decode algorithm index them;
* ids are stored row-major per output feature (``N`` rows of packed ids);
* one fp16 codebook per matrix (the shared form), unless a per-subspace
  table is passed to ``lut_accumulate``;
* ids must be ``< C``; the oracle rejects anything else.

Pins (checked in the CPU test-suite): brute-force loops on tiny shapes, the
closed form for a signed one-hot codebook, linearity in x, the identity
codebook (d = 1, C = 65536) that turns the layer into a plain fp16 matmul,
full vector quantization (d = K), and a hand-worked byte example of the
12-bit stream.
"""

from __future__ import annotations

from typing import Optional, Sequence

import numpy as np

__all__ = [
    "unpack_indices",
    "reconstruct_bits",
    "reconstruct",
    "pq_linear",
    "lut_accumulate",
    "relative_l2",
    "max_abs_over_rms",
]


def unpack_indices(idx: np.ndarray, S: int, idx_bits: int, C: Optional[int] = None,
                   rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """Decode packed id rows into an ``[N, S]`` uint32 array.

    The storage rule is one least-significant-bit-first bit stream per row:
    id ``s`` occupies stream bits ``[b*s, b*s + b)`` (``b = idx_bits``) and
    stream bit ``t`` is bit ``t mod 8`` of byte ``t div 8``.  For b = 8 this is
    one byte per id, for b = 16 a little-endian byte pair, for b = 12 three
    bytes per pair of ids.  The decoder applies the rule literally, one bit of
    every id at a time.

    ``rows`` restricts decoding to a subset of output rows.  When ``C`` is
    given, every id must be ``< C``.
    """
    if idx_bits not in (8, 12, 16):
        raise ValueError("idx_bits must be 8, 12 or 16")
    idx = np.asarray(idx)
    if idx.dtype != np.uint8 or idx.ndim != 2:
        raise ValueError("idx must be a 2-D uint8 array [N, R]")
    if rows is not None:
        idx = idx[np.asarray(rows, dtype=np.int64)]
    n_rows, R = idx.shape
    if R * 8 < S * idx_bits:
        raise ValueError(f"row of {R} bytes is too short for {S} ids of {idx_bits} bits")
    u = np.zeros((n_rows, S), dtype=np.uint32)
    first_bit = np.arange(S, dtype=np.int64) * idx_bits
    for t in range(idx_bits):
        pos = first_bit + t
        byte = pos // 8
        bit = (pos % 8).astype(np.uint32)
        u |= ((idx[:, byte].astype(np.uint32) >> bit) & np.uint32(1)) << np.uint32(t)
    if C is not None and u.size and int(u.max()) >= C:
        raise ValueError(f"id {int(u.max())} is out of range for C = {C}")
    return u


def reconstruct_bits(u: np.ndarray, codebook: np.ndarray) -> np.ndarray:
    """Bit patterns of ``W_hat``: ``[N, S*d]`` uint16, a pure codeword gather."""
    cb = np.ascontiguousarray(np.asarray(codebook, dtype=np.float16))
    if cb.ndim != 2:
        raise ValueError("codebook must be [C, d]")
    C, d = cb.shape
    u = np.asarray(u)
    if u.size and int(u.max()) >= C:
        raise ValueError("id out of range")
    cb_bits = cb.view(np.uint16)
    n_rows, S = u.shape
    return cb_bits[u.astype(np.int64)].reshape(n_rows, S * d)


def reconstruct(idx: np.ndarray, K: int, idx_bits: int, d: int, codebook: np.ndarray,
                rows: Optional[Sequence[int]] = None) -> np.ndarray:
    """``W_hat`` as fp16 ``[N, K]`` (or the requested rows)."""
    if K % d:
        raise ValueError("K must be a multiple of d")
    C = np.asarray(codebook).shape[0]
    u = unpack_indices(idx, K // d, idx_bits, C=C, rows=rows)
    return reconstruct_bits(u, codebook).view(np.float16)


def pq_linear(x: np.ndarray, idx: np.ndarray, idx_bits: int, d: int, codebook: np.ndarray,
              rows: Optional[Sequence[int]] = None, chunk: int = 4096) -> np.ndarray:
    """``y = x . W_hat^T`` in fp64, ``[M, N]`` (or ``[M, len(rows)]``).

    ``x`` may be fp16 (the layer's input type) or any float type (fp64 for the
    linearity check).  ``W_hat`` is decoded ``chunk`` rows at a time so that
    large matrices (an lm_head) never exist densely in fp64.
    """
    x = np.asarray(x)
    if x.ndim == 1:
        x = x[None, :]
    M, K = x.shape
    x64 = x.astype(np.float64)
    all_rows = np.arange(np.asarray(idx).shape[0]) if rows is None else np.asarray(rows, dtype=np.int64)
    out = np.empty((M, all_rows.size), dtype=np.float64)
    for lo in range(0, all_rows.size, chunk):
        sel = all_rows[lo:lo + chunk]
        w = reconstruct(idx, K, idx_bits, d, codebook, rows=sel).astype(np.float64)
        out[:, lo:lo + sel.size] = x64 @ w.T
    return out


def lut_accumulate(x: np.ndarray, t_cluster: np.ndarray, t_index: np.ndarray) -> np.ndarray:
    """Eq. lut-accumulate in the paper's own layout, fp64.

    ``t_cluster``: ``[N_ss, K_s, SZ]`` centroids (one table per subspace).
    ``t_index``: ``[N_ss, F_out]`` ids, subspace-major.
    ``x``: ``[M, N_ss * SZ]``.
    Returns ``o[m, j] = sum_ss dot(x[m, ss*SZ:(ss+1)*SZ], t_cluster[ss, t_index[ss, j]])``.
    """
    x = np.asarray(x)
    if x.ndim == 1:
        x = x[None, :]
    t_cluster = np.asarray(t_cluster)
    t_index = np.asarray(t_index)
    n_ss, k_s, sz = t_cluster.shape
    if x.shape[1] != n_ss * sz or t_index.shape[0] != n_ss:
        raise ValueError("shape mismatch")
    if t_index.size and int(t_index.max()) >= k_s:
        raise ValueError("id out of range")
    x64 = x.astype(np.float64)
    o = np.zeros((x.shape[0], t_index.shape[1]), dtype=np.float64)
    for ss in range(n_ss):
        x_ss = x64[:, ss * sz:(ss + 1) * sz]                      # [M, SZ]
        cent = t_cluster[ss].astype(np.float64)[t_index[ss].astype(np.int64)]  # [F_out, SZ]
        o += x_ss @ cent.T
    return o


def relative_l2(y: np.ndarray, y_ref: np.ndarray) -> float:
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    den = float(np.linalg.norm(y_ref))
    num = float(np.linalg.norm(y - y_ref))
    if den == 0.0:
        return 0.0 if num == 0.0 else float("inf")
    return num / den


def max_abs_over_rms(y: np.ndarray, y_ref: np.ndarray) -> float:
    y = np.asarray(y, dtype=np.float64)
    y_ref = np.asarray(y_ref, dtype=np.float64)
    rms = float(np.sqrt(np.mean(y_ref * y_ref))) if y_ref.size else 0.0
    err = float(np.max(np.abs(y - y_ref))) if y_ref.size else 0.0
    if rms == 0.0:
        return 0.0 if err == 0.0 else float("inf")
    return err / rms
