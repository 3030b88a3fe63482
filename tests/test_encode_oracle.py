"""Pins for the k-means encoder oracle (Alg. 1): each check rests on something
other than the oracle itself.

* exact rational arithmetic (fractions) for the nearest codeword and the mean;
* planted clusters that a correct Lloyd iteration recovers exactly;
* SciPy's k-means (kmeans2 with a given starting codebook) on well-separated
  data;
* the closed form of a one-dimensional two-cluster example;
* the Lloyd invariant that the objective never increases (up to the fp16
  rounding of the means);
* planted mistakes in the oracle, which these pins must catch.
"""

from fractions import Fraction

import numpy as np
import pytest

import pq_inputs as pi
from oracle import pq_encode as enc


def exact_sq_dist(p, c):
    return sum((Fraction(float(a)) - Fraction(float(b))) ** 2 for a, b in zip(p, c))


def fp16_nearest(q: Fraction) -> np.float16:
    """Round an exact rational to fp16, nearest, ties to even (by search over
    the two fp16 neighbours)."""
    lo = np.float16(float(q))  # a neighbour (float() rounds once, then fp16 once)
    cands = set()
    for v in (lo, np.nextafter(lo, np.float16(np.inf)), np.nextafter(lo, np.float16(-np.inf))):
        cands.add(v)
    best = None
    for v in sorted(cands, key=float):
        err = abs(Fraction(float(v)) - q)
        if best is None or err < best[0] or (err == best[0] and int(v.view(np.uint16)) % 2 == 0):
            best = (err, v)
    return best[1]


# ---------------------------------------------------------------------------
# Assignment
# ---------------------------------------------------------------------------

def test_assignment_is_the_exact_nearest_codeword():
    rng = np.random.default_rng(0)
    for d, C in ((1, 7), (2, 16), (4, 9), (8, 5)):
        pts = pi.draw_weights(rng, 60, d, std=0.5)
        cb = pi.draw_weights(rng, C, d, std=0.5)
        u = enc.assign(pts, cb)
        checked = 0
        for p, k in zip(pts, u):
            dists = [exact_sq_dist(p, c) for c in cb]
            best = min(dists)
            second = min(x for j, x in enumerate(dists) if j != dists.index(best)) if C > 1 else best + 1
            if second - best > Fraction(1, 10 ** 6) * (best + Fraction(1, 10 ** 6)):
                assert dists[int(k)] == best
                checked += 1
        assert checked > 50


def test_ties_go_to_the_lowest_index():
    # duplicate codewords: the lower index takes every point
    cb = np.array([[0.5, 0.5], [0.25, -1.0], [0.5, 0.5], [0.25, -1.0]], dtype=np.float16)
    pts = np.array([[0.5, 0.5], [0.3, 0.4], [0.25, -1.0], [0.2, -0.9]], dtype=np.float16)
    assert enc.assign(pts, cb).tolist() == [0, 0, 1, 1]
    # a point exactly halfway between two codewords (d = 1)
    cb1 = np.array([[2.0], [0.0]], dtype=np.float16)
    assert enc.assign(np.array([[1.0]], dtype=np.float16), cb1).tolist() == [0]


# ---------------------------------------------------------------------------
# Update
# ---------------------------------------------------------------------------

def test_update_is_the_exact_mean_rounded_to_fp16():
    rng = np.random.default_rng(1)
    pts = pi.draw_weights(rng, 500, 4, std=0.3)
    C = 12
    u = rng.integers(0, C, size=500).astype(np.uint32)
    cb0 = pi.draw_weights(rng, C, 4)
    new = enc.update(pts, u, cb0)
    for k in range(C):
        members = pts[u == k]
        for i in range(4):
            mean = sum(Fraction(float(v)) for v in members[:, i]) / len(members)
            assert new[k, i].view(np.uint16) == fp16_nearest(mean).view(np.uint16), (k, i)


def test_halfway_means_round_to_even():
    # the mean of two neighbouring fp16 values lies exactly halfway between them
    a = np.float16(1.0)
    b = np.nextafter(a, np.float16(2.0))  # 1 + 2^-10: odd mantissa
    c = np.nextafter(b, np.float16(2.0))  # even mantissa
    pts = np.array([[a], [b], [b], [c]], dtype=np.float16)
    u = np.array([0, 0, 1, 1], dtype=np.uint32)
    new = enc.update(pts, u, np.zeros((2, 1), np.float16))
    assert new[0, 0] == a  # halfway between a (even) and b (odd): a
    assert new[1, 0] == c  # halfway between b (odd) and c (even): c


def test_empty_cluster_keeps_its_codeword():
    pts = np.array([[0.0], [0.5], [1.0]], dtype=np.float16)
    cb = np.array([[0.25], [100.0]], dtype=np.float16)
    cb2, ids = enc.kmeans_encode(pts.reshape(3, 1), 1, cb, iters=3)
    assert cb2[1, 0] == np.float16(100.0)
    assert ids.ravel().tolist() == [0, 0, 0]


# ---------------------------------------------------------------------------
# Whole iterations
# ---------------------------------------------------------------------------

def test_one_dimensional_two_cluster_closed_form():
    w = np.array([[0.0, 1.0, 10.0, 11.0]], dtype=np.float16)
    cb, ids = enc.kmeans_encode(w, 1, np.array([[0.0], [11.0]], dtype=np.float16), iters=1)
    assert cb.ravel().tolist() == [0.5, 10.5]
    assert ids.ravel().tolist() == [0, 0, 1, 1]


def test_recovers_planted_clusters_exactly():
    rng = np.random.default_rng(2)
    C, d, N, K = 32, 4, 64, 64
    centers = (rng.integers(-40, 40, size=(C, d)) / 4).astype(np.float16)
    centers[:, 0] = (np.arange(C) * 4 - 64).astype(np.float16)  # distinct, far apart
    labels = rng.integers(0, C, size=N * K // d)
    w = centers[labels].reshape(N, K)
    perm = rng.permutation(C)
    cb, ids, objs = enc.kmeans_encode(w, d, centers[perm], iters=1, history=True)
    inv = np.argsort(perm)
    assert np.array_equal(cb.view(np.uint16), centers[perm].view(np.uint16))
    assert np.array_equal(ids.ravel(), inv[labels])
    assert objs[-1] == 0.0


def test_matches_scipy_kmeans_on_separated_clusters():
    vq = pytest.importorskip("scipy.cluster.vq")
    rng = np.random.default_rng(3)
    C, d = 8, 2
    centers = np.stack([np.arange(C) * 3.0, (np.arange(C) % 3) * 5.0], axis=1)
    labels = rng.integers(0, C, size=4000)
    pts = (centers[labels] + rng.normal(0, 0.3, size=(4000, d))).astype(np.float16)
    init = (centers + 0.7).astype(np.float16)
    cb, ids = enc.kmeans_encode(pts.reshape(100, 40 * d), d, init, iters=4)
    data = pts.astype(np.float64)
    ref_cb, _ = vq.kmeans2(data, init.astype(np.float64), iter=4, minit="matrix", missing="raise")
    ref_ids = vq.vq(data, ref_cb)[0]
    assert np.array_equal(ids.ravel(), ref_ids)
    ulp = np.spacing(np.abs(ref_cb).astype(np.float16)).astype(np.float64)
    assert np.all(np.abs(cb.astype(np.float64) - ref_cb) <= ulp)


def test_objective_on_a_hand_worked_example():
    """Three 2-D points, two codewords, worked by hand:
    p0 = (1, 2)  -> c0 = (0, 0): 1^2 + 2^2     = 5
    p1 = (3, -1) -> c1 = (1, 1): 2^2 + (-2)^2  = 8
    p2 = (0.5, 0) -> c0:         0.5^2 + 0^2   = 0.25
    sum of squared distances = 13.25 (an unsquared sum, 3 + 4 + 0.5 after
    |.| per coordinate, gives 7.5; Euclidean lengths give sqrt(5) + sqrt(8)
    + 0.5)."""
    pts = np.array([[1.0, 2.0], [3.0, -1.0], [0.5, 0.0]], np.float16)
    cb = np.array([[0.0, 0.0], [1.0, 1.0]], np.float16)
    u = np.array([0, 1, 0])
    assert enc.objective(pts, u, cb) == 13.25
    # the nearest codewords move p0 to c1 ((1-1)^2 + (2-1)^2 = 1): 1 + 8 + 0.25
    assert np.array_equal(enc.assign(pts, cb), [1, 1, 0])
    assert enc.objective(pts, enc.assign(pts, cb), cb) == 9.25


def test_objective_never_increases():
    rng = np.random.default_rng(4)
    w = pi.draw_weights(rng, 64, 256)
    d, C = 2, 16
    ids0 = pi.init_point_ids(rng, 64 * 256 // d, C)
    init = pi.subvectors_at(w, d, ids0)
    _, _, objs = enc.kmeans_encode(w, d, init, iters=8, history=True)
    # rounding a mean to fp16 moves it by at most half an ulp of |w| <= 0.125
    slack = (64 * 256) * (2.0 ** -14) ** 2
    assert objs[-1] < objs[0]
    for a, b in zip(objs, objs[1:]):
        assert b <= a + slack


def test_rejects_out_of_range_weights():
    cb = np.zeros((2, 2), np.float16)
    with pytest.raises(ValueError):
        enc.kmeans_encode(np.full((2, 4), 200.0, np.float16), 2, cb, 1)
    with pytest.raises(ValueError):
        enc.kmeans_encode(np.full((2, 4), np.inf, np.float16), 2, cb, 1)


# ---------------------------------------------------------------------------
# Planted mistakes: a broken oracle must fail the pins above
# ---------------------------------------------------------------------------

def _ties_to_highest(points, codebook):
    pts = np.asarray(points).astype(np.float32)
    cb = np.asarray(codebook).astype(np.float32)
    acc = np.zeros((pts.shape[0], cb.shape[0]), np.float32)
    for i in range(pts.shape[1]):
        diff = pts[:, i:i + 1] - cb[None, :, i]
        acc = acc + diff * diff
    return (cb.shape[0] - 1 - np.argmin(acc[:, ::-1], axis=1)).astype(np.uint32)


def _mean_not_rounded(points, u, codebook):
    C, d = codebook.shape
    new = np.array(codebook, dtype=np.float64)
    for k in range(C):
        m = np.asarray(points)[u == k]
        if len(m):
            new[k] = m.astype(np.float64).mean(axis=0) * (1 + 2 ** -9)  # off by a fraction of an ulp
    return new.astype(np.float16)


def test_planted_tie_mistake_is_caught(monkeypatch):
    monkeypatch.setattr(enc, "assign", _ties_to_highest)
    with pytest.raises(AssertionError):
        test_ties_go_to_the_lowest_index()


def test_planted_mean_mistake_is_caught(monkeypatch):
    monkeypatch.setattr(enc, "update", _mean_not_rounded)
    with pytest.raises(AssertionError):
        test_update_is_the_exact_mean_rounded_to_fp16()
