"""CPU oracle for calibration-free PQ encoding: k-means over weight sub-vectors.

TEST INFRASTRUCTURE ONLY.  Nothing in the library imports, links or calls this
module; only the tests, the smoke check and the benchmark's CPU-baseline leg
use it.  It shares no code with the HIP encoder.

What it computes (paper: Sec. 3.1.1 and Alg. 1, calibration-free k-means):

A weight matrix ``W`` with ``N`` output rows and ``K`` input columns is cut
along K into ``S = K / d`` sub-vectors of length ``d`` per row; sub-vector
``s`` of row ``n`` is data point ``p = n * S + s``.  Lloyd's k-means with ``C``
clusters then alternates

    assignment:  u(p)  = the index k of the codeword nearest to point p
    update:      c_k   = the mean of the points with u(p) = k

``iters`` times, starting from a given fp16 codebook, and a last assignment
against the final codebook gives the ids.  Alg. 1 runs one k-means per
subspace; the kernels of this project consume one codebook shared by every
subspace, so the encoder clusters the sub-vectors of all subspaces together.

Readings of the paper, which fixes none of these details:

* starting codebook: given by the caller (the tests and the binding take C
  distinct sub-vectors of W chosen by a seeded generator);
* number of iterations: given by the caller;
* distance: the squared Euclidean distance, evaluated in fp32 from the fp16
  values as ``acc = 0; acc = acc + (w_i - c_i) * (w_i - c_i)`` for
  i = 0 .. d-1, every operation rounded to fp32 (no fused multiply-add);
* ties: the lowest codeword index wins;
* the mean: the sum of a cluster's values is formed exactly (each fp16 value
  is an integer multiple of 2^-24), converted to fp64, scaled by 2^-24,
  divided by the count in fp64, and rounded to fp16 (round to nearest even);
* an empty cluster keeps its codeword;
* inputs are finite with |w| < 128 (so the exact sums fit in 64 bits).
"""

from __future__ import annotations

import numpy as np

__all__ = ["points_of", "assign", "update", "kmeans_encode", "objective", "Q_SCALE"]

Q_SCALE = 2 ** 24  # fp16 values are integer multiples of 2^-24


def points_of(w: np.ndarray, d: int) -> np.ndarray:
    """The ``N * (K / d)`` sub-vectors of ``w`` (fp16 ``[N, K]``) as ``[P, d]``
    fp16, point ``n * S + s`` being ``w[n, s*d:(s+1)*d]``."""
    w = np.asarray(w)
    if w.dtype != np.float16 or w.ndim != 2:
        raise ValueError("w must be a 2-D fp16 array")
    N, K = w.shape
    if d < 1 or K % d:
        raise ValueError("K must be a multiple of d")
    if not np.all(np.isfinite(w)) or np.abs(w.astype(np.float32)).max(initial=0.0) >= 128.0:
        raise ValueError("weights must be finite with |w| < 128")
    return w.reshape(N * (K // d), d)


def assign(points: np.ndarray, codebook: np.ndarray) -> np.ndarray:
    """Nearest codeword of every point (fp32 squared distance, lowest index on
    ties), as uint32 ``[P]``."""
    pts = np.asarray(points).astype(np.float32)
    cb = np.asarray(codebook).astype(np.float32)
    P, d = pts.shape
    C = cb.shape[0]
    block = max(1, (1 << 24) // C)  # points per block: bounds the [block, C] distance table
    out = np.empty(P, dtype=np.uint32)
    for b0 in range(0, P, block):
        p = pts[b0:b0 + block]
        acc = np.zeros((p.shape[0], C), dtype=np.float32)
        for i in range(d):  # fixed order, one fp32 rounding per operation
            diff = p[:, i:i + 1] - cb[None, :, i]
            acc = acc + diff * diff
        out[b0:b0 + block] = np.argmin(acc, axis=1)  # first minimum: lowest index
    return out


def _f64_to_f16(v: np.ndarray) -> np.ndarray:
    return np.asarray(v, dtype=np.float64).astype(np.float16)


def update(points: np.ndarray, u: np.ndarray, codebook: np.ndarray) -> np.ndarray:
    """New fp16 codebook: each non-empty cluster's mean (exact integer sum,
    fp64 division, fp16 rounding); empty clusters keep their codeword."""
    pts = np.asarray(points)
    C, d = codebook.shape
    q = (pts.astype(np.float64) * Q_SCALE).astype(np.int64)  # exact: fp16 * 2^24 is an integer
    sums = np.zeros((C, d), dtype=np.int64)
    np.add.at(sums, u.astype(np.int64), q)
    counts = np.bincount(u.astype(np.int64), minlength=C).astype(np.int64)
    new = np.array(codebook, dtype=np.float16, copy=True)
    live = counts > 0
    mean = (sums[live].astype(np.float64) * (1.0 / Q_SCALE)) / counts[live].astype(np.float64)[:, None]
    new[live] = _f64_to_f16(mean)
    return new


def objective(points: np.ndarray, u: np.ndarray, codebook: np.ndarray) -> float:
    """Sum of squared distances of the points to their codewords, in fp64."""
    diff = np.asarray(points).astype(np.float64) - np.asarray(codebook).astype(np.float64)[u.astype(np.int64)]
    return float(np.sum(diff * diff))


def kmeans_encode(w: np.ndarray, d: int, init_codebook: np.ndarray, iters: int, history: bool = False):
    """Encode ``w`` (fp16 ``[N, K]``): ``iters`` Lloyd iterations from
    ``init_codebook`` (fp16 ``[C, d]``), then the final assignment.

    Returns ``(codebook fp16 [C, d], ids uint32 [N, K/d])``, and with
    ``history`` also the list of objectives before each update and after the
    final assignment.
    """
    pts = points_of(w, d)
    cb = np.asarray(init_codebook)
    if cb.dtype != np.float16 or cb.ndim != 2 or cb.shape[1] != d:
        raise ValueError("init_codebook must be fp16 [C, d]")
    if not np.all(np.isfinite(cb)):
        raise ValueError("init_codebook must be finite")
    if iters < 0:
        raise ValueError("iters must be >= 0")
    objs = []
    for _ in range(iters):
        u = assign(pts, cb)
        objs.append(objective(pts, u, cb))
        cb = update(pts, u, cb)
    u = assign(pts, cb)
    objs.append(objective(pts, u, cb))
    ids = u.reshape(w.shape[0], w.shape[1] // d)
    return (cb, ids, objs) if history else (cb, ids)
