"""Pins for the CPU oracle: each check rests on something other than the oracle.

* hand-worked bytes of the packed index stream (golden file);
* arbitrary-precision integer bit extraction (Python ints) for the decoder;
* pure-Python loops for the codeword gather and the dot products;
* the closed form of a signed, power-of-two scaled one-hot codebook;
* linearity of the layer in x;
* the identity codebook (d = 1, C = 65536), where the layer is a plain fp16
  matmul, and full vector quantization (d = K);
* planted mistakes in a copy of the oracle, which the pins above must catch.
"""

import math

import numpy as np
import pytest

import pq_inputs as pi
from oracle import pq_oracle as orc
from conftest import read_golden_table


# --------------------------------------------------------------------------
# Pure-Python references (no NumPy arithmetic)
# --------------------------------------------------------------------------

def py_unpack_row(row_bytes, S, bits):
    """Ids of one row via one big little-endian integer."""
    stream = int.from_bytes(bytes(row_bytes), "little")
    mask = (1 << bits) - 1
    return [(stream >> (bits * s)) & mask for s in range(S)]


def py_reconstruct(ids, codebook_f):
    """W_hat rows as Python floats from ids [N][S] and codebook [C][d]."""
    W = []
    for row in ids:
        w = []
        for u in row:
            w.extend(codebook_f[u])
        W.append(w)
    return W


def py_matmul_nt(x, W):
    """y[m][n] = sum_k x[m][k] * W[n][k] with math.fsum (exactly rounded sums)."""
    return [[math.fsum(a * b for a, b in zip(xr, wr)) for wr in W] for xr in x]


def as_pylist(a):
    return np.asarray(a, dtype=np.float64).tolist()


# --------------------------------------------------------------------------
# Index decoding
# --------------------------------------------------------------------------

def test_unpack_matches_hand_worked_bytes():
    rows = read_golden_table("packed_index_examples.txt")
    assert len(rows) >= 6
    for bits_s, ids_s, bytes_s in rows:
        bits = int(bits_s)
        ids = [int(t, 16) for t in ids_s.split()]
        raw = np.array([[int(t, 16) for t in bytes_s.split()]], dtype=np.uint8)
        got = orc.unpack_indices(raw, len(ids), bits)
        assert got.tolist() == [ids], (bits, ids_s)
        # The shared encoder must produce exactly the hand-worked bytes.
        enc = pi.pack_indices(np.array([ids]), bits)
        assert enc.tolist() == raw.tolist(), (bits, ids_s)


@pytest.mark.parametrize("bits", [8, 12, 16])
@pytest.mark.parametrize("S", [1, 2, 3, 7, 16, 33])
def test_unpack_matches_bigint_extraction(bits, S):
    rng = np.random.default_rng(1000 + bits * 100 + S)
    R = pi.row_bytes(S, bits)
    raw = rng.integers(0, 256, size=(5, R), dtype=np.uint8)
    if (S * bits) % 8:  # the pad bits of the last byte are zero in valid rows
        keep = (S * bits) % 8
        raw[:, -1] &= (1 << keep) - 1
    got = orc.unpack_indices(raw, S, bits)
    for n in range(raw.shape[0]):
        assert got[n].tolist() == py_unpack_row(raw[n], S, bits)


@pytest.mark.parametrize("bits", [8, 12, 16])
@pytest.mark.parametrize("S", [1, 5, 64, 129])
def test_pack_unpack_roundtrip(bits, S):
    rng = np.random.default_rng(7 * bits + S)
    C = 1 << bits
    ids = rng.integers(0, C, size=(9, S))
    packed = pi.pack_indices(ids, bits)
    assert packed.shape == (9, pi.row_bytes(S, bits))
    assert np.array_equal(orc.unpack_indices(packed, S, bits), ids.astype(np.uint32))


def test_unpack_rejects_out_of_range_and_short_rows():
    packed = pi.pack_indices(np.array([[0, 5, 255]]), 8)
    with pytest.raises(ValueError):
        orc.unpack_indices(packed, 3, 8, C=200)
    with pytest.raises(ValueError):
        orc.unpack_indices(packed, 4, 8)
    with pytest.raises(ValueError):
        orc.unpack_indices(packed, 3, 10)


def test_unpack_row_subset():
    rng = np.random.default_rng(3)
    ids = rng.integers(0, 4096, size=(10, 11))
    packed = pi.pack_indices(ids, 12)
    rows = [7, 2, 9]
    assert np.array_equal(orc.unpack_indices(packed, 11, 12, rows=rows), ids[rows].astype(np.uint32))


# --------------------------------------------------------------------------
# Reconstruction (bit-exact gather)
# --------------------------------------------------------------------------

def test_reconstruct_tiny_workload_bruteforce():
    p = pi.workload("tiny").problem(0)
    assert (p.M, p.K, p.N, p.d, p.C, p.idx_bits) == (1, 256, 128, 4, 256, 8)
    bits = orc.reconstruct(p.idx, p.K, p.idx_bits, p.d, p.codebook).view(np.uint16)
    cb_bits = p.codebook.view(np.uint16).tolist()
    for n in range(p.N):
        row = py_unpack_row(p.idx[n], p.S, 8)
        expect = []
        for u in row:
            expect.extend(cb_bits[u])
        assert bits[n].tolist() == expect


def test_reconstruct_preserves_subnormals_and_signed_zero():
    specials = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x03FF, 0x83FF, 0x0400, 0x7BFF],
                        dtype=np.uint16)
    cb = specials.view(np.float16).reshape(4, 2)
    ids = np.array([[3, 0, 1, 2], [0, 0, 3, 1]])
    w = orc.reconstruct(pi.pack_indices(ids, 8), 8, 8, 2, cb)
    expect = np.concatenate([specials.reshape(4, 2)[r] for r in ids.ravel()]).reshape(2, 8)
    assert np.array_equal(w.view(np.uint16), expect)


# --------------------------------------------------------------------------
# Layer output y
# --------------------------------------------------------------------------

BRUTE_CASES = [
    # M, K, N, d, C, bits
    (1, 256, 128, 4, 256, 8),   # the tiny workload's shape
    (3, 12, 5, 3, 7, 8),
    (2, 16, 7, 1, 300, 12),
    (4, 24, 6, 8, 4096, 12),
    (2, 18, 3, 2, 65536, 16),
    (5, 10, 4, 10, 9, 16),      # full VQ: d = K
]


@pytest.mark.parametrize("case", BRUTE_CASES)
def test_pq_linear_matches_pure_python(case):
    M, K, N, d, C, bits = case
    rng = np.random.default_rng(sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    y = orc.pq_linear(p.x, p.idx, bits, d, p.codebook)
    assert y.shape == (M, N)
    ids = [py_unpack_row(p.idx[n], p.S, bits) for n in range(N)]
    W = py_reconstruct(ids, as_pylist(p.codebook))
    ref = py_matmul_nt(as_pylist(p.x), W)
    ref = np.array(ref)
    assert np.allclose(y, ref, rtol=1e-12, atol=1e-15 * max(1.0, float(np.abs(ref).max())))


@pytest.mark.parametrize("case", BRUTE_CASES)
def test_lut_accumulate_shared_codebook_matches_pure_python(case):
    M, K, N, d, C, bits = case
    rng = np.random.default_rng(100 + sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    S = K // d
    t_cluster = np.broadcast_to(p.codebook, (S, C, d))
    t_index = p.ids.T  # subspace-major [N_ss, F_out]
    o = orc.lut_accumulate(p.x, t_cluster, t_index)
    cb = as_pylist(p.codebook)
    xs = as_pylist(p.x)
    for m in range(M):
        for n in range(N):
            terms = []
            for s in range(S):
                cent = cb[int(p.ids[n, s])]
                terms.extend(xs[m][s * d + i] * cent[i] for i in range(d))
            assert o[m, n] == pytest.approx(math.fsum(terms), rel=1e-12, abs=1e-14)


def test_lut_accumulate_per_subspace_codebooks_pure_python():
    rng = np.random.default_rng(11)
    n_ss, k_s, sz, f_out, M = 6, 5, 3, 4, 2
    t_cluster = rng.normal(0, 0.02, size=(n_ss, k_s, sz)).astype(np.float16)
    t_index = rng.integers(0, k_s, size=(n_ss, f_out))
    x = rng.normal(size=(M, n_ss * sz)).astype(np.float16)
    o = orc.lut_accumulate(x, t_cluster, t_index)
    tc = np.asarray(t_cluster, np.float64).tolist()
    xs = as_pylist(x)
    for m in range(M):
        for j in range(f_out):
            terms = [xs[m][ss * sz + i] * tc[ss][int(t_index[ss, j])][i]
                     for ss in range(n_ss) for i in range(sz)]
            assert o[m, j] == pytest.approx(math.fsum(terms), rel=1e-12, abs=1e-15)


@pytest.mark.parametrize("d,C,bits", [(1, 2, 8), (2, 256, 8), (4, 4096, 12), (8, 64, 16), (4, 65536, 16)])
def test_scaled_one_hot_codebook_closed_form(d, C, bits):
    """codebook[k] = sign_k * 2^-((k div d) mod 4) * e_(k mod d) gives
    y[m, n] = sum_s sign_u * 2^-((u div d) mod 4) * x[m, s*d + (u mod d)], u = u(n, s)."""
    rng = np.random.default_rng(d * 1000 + C)
    M, S, N = 3, 37, 11
    K = S * d
    cb, sign = pi.scaled_signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, S))
    x = pi.draw_x(rng, M, K)
    y = orc.pq_linear(x, pi.pack_indices(ids, bits), bits, d, cb)
    xs = as_pylist(x)
    for m in range(M):
        for n in range(N):
            total = 0.0
            for s in range(S):
                u = int(ids[n, s])
                total += sign[u] * 2.0 ** (-((u // d) % 4)) * xs[m][s * d + (u % d)]
            # every term is an fp16 value times a power of two: exact in fp64
            assert y[m, n] == total


def test_linearity_in_x():
    rng = np.random.default_rng(5)
    p = pi.draw_problem(rng, 2, 64, 9, 4, 256, 8)
    x1 = rng.normal(size=(2, 64))
    x2 = rng.normal(size=(2, 64))
    a, b = rng.normal(), rng.normal()
    lhs = orc.pq_linear(a * x1 + b * x2, p.idx, 8, 4, p.codebook)
    rhs = a * orc.pq_linear(x1, p.idx, 8, 4, p.codebook) + b * orc.pq_linear(x2, p.idx, 8, 4, p.codebook)
    assert np.allclose(lhs, rhs, rtol=1e-12, atol=1e-13)


def test_identity_codebook_is_plain_fp16_matmul():
    """d = 1, C = 65536, codebook[k] = the fp16 whose bit pattern is k: W_hat is
    the id array viewed as fp16, and the layer is an ordinary matmul."""
    rng = np.random.default_rng(9)
    cb = np.arange(65536, dtype=np.uint16).view(np.float16).reshape(65536, 1)
    M, K, N = 3, 40, 17
    # finite, moderate values only: exponent field below 0x1E (|w| < 2^15)
    ids = rng.integers(0, 0x7800, size=(N, K)).astype(np.uint16)
    ids |= (rng.integers(0, 2, size=(N, K)).astype(np.uint16) << 15)
    x = pi.draw_x(rng, M, K)
    y = orc.pq_linear(x, pi.pack_indices(ids, 16), 16, 1, cb)
    w = ids.view(np.float16).astype(np.float64)
    ref = np.array(py_matmul_nt(as_pylist(x), w.tolist()))
    assert np.allclose(y, ref, rtol=1e-12, atol=0)


def test_full_vector_quantization():
    """d = K (one sub-vector per row): y = x . codebook[u(n)]^T."""
    rng = np.random.default_rng(12)
    M, K, N, C = 2, 24, 6, 50
    cb = pi.draw_codebook(rng, C, K)
    ids = rng.integers(0, C, size=(N, 1))
    x = pi.draw_x(rng, M, K)
    y = orc.pq_linear(x, pi.pack_indices(ids, 8), 8, K, cb)
    ref = as_pylist(x)
    cbl = as_pylist(cb)
    for m in range(M):
        for n in range(N):
            assert y[m, n] == pytest.approx(math.fsum(a * b for a, b in zip(ref[m], cbl[int(ids[n, 0])])),
                                            rel=1e-12, abs=1e-15)


def test_chunked_rows_equal_unchunked():
    rng = np.random.default_rng(13)
    p = pi.draw_problem(rng, 2, 32, 37, 2, 256, 8)
    a = orc.pq_linear(p.x, p.idx, 8, 2, p.codebook, chunk=5)
    b = orc.pq_linear(p.x, p.idx, 8, 2, p.codebook, chunk=4096)
    c = orc.pq_linear(p.x, p.idx, 8, 2, p.codebook, rows=[36, 0, 5])
    assert np.array_equal(a, b)
    assert np.array_equal(c, b[:, [36, 0, 5]])


def test_statistical_scale_of_outputs():
    """rms(y) is near 0.02 * sqrt(K) for x ~ N(0,1) and N(0, 0.02) codewords."""
    rng = np.random.default_rng(14)
    p = pi.draw_problem(rng, 1, 4096, 2048, 2, 256, 8)
    y = orc.pq_linear(p.x, p.idx, 8, 2, p.codebook)
    rms = float(np.sqrt(np.mean(y ** 2)))
    assert 0.8 * 0.02 * 64 < rms < 1.2 * 0.02 * 64


def test_comparison_metrics():
    y_ref = np.array([1.0, -2.0, 2.0])
    assert orc.relative_l2(y_ref, y_ref) == 0.0
    assert orc.relative_l2(y_ref + np.array([0.0, 0.0, 0.3]), y_ref) == pytest.approx(0.1)
    assert orc.max_abs_over_rms(y_ref + np.array([0.0, 0.0, 0.3]), y_ref) == pytest.approx(0.3 / math.sqrt(3.0))


# --------------------------------------------------------------------------
# Planted mistakes: plausible bugs in a copy of the oracle must fail a pin.
# --------------------------------------------------------------------------

def _mutant_dropped_last_subspace(x, idx, bits, d, cb):
    K = x.shape[1]
    w = orc.reconstruct(idx, K, bits, d, cb).astype(np.float64)
    w[:, -d:] = 0.0
    return x.astype(np.float64) @ w.T


def _mutant_transposed_subvector(x, idx, bits, d, cb):
    K = x.shape[1]
    u = orc.unpack_indices(idx, K // d, bits)
    w = np.asarray(cb, np.float16)[u.astype(np.int64)][:, :, ::-1].reshape(idx.shape[0], K)
    return x.astype(np.float64) @ w.astype(np.float64).T


def _mutant_12bit_wrong_shift(x, idx, bits, d, cb):
    K = x.shape[1]
    S = K // d
    u = orc.unpack_indices(idx, S, bits)
    if bits == 12:
        u = u[:, ::-1]  # ids read in the wrong order within the row
    w = np.asarray(cb, np.float16)[u.astype(np.int64)].reshape(idx.shape[0], K)
    return x.astype(np.float64) @ w.astype(np.float64).T


def _mutant_sign(x, idx, bits, d, cb):
    return -orc.pq_linear(x, idx, bits, d, cb)


@pytest.mark.parametrize("mutant", [_mutant_dropped_last_subspace, _mutant_transposed_subvector,
                                    _mutant_12bit_wrong_shift, _mutant_sign])
def test_planted_mistakes_are_caught(mutant):
    rng = np.random.default_rng(21)
    M, K, N, d, C, bits = 2, 24, 5, 4, 4096, 12
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    ids = [py_unpack_row(p.idx[n], p.S, bits) for n in range(N)]
    ref = np.array(py_matmul_nt(as_pylist(p.x), py_reconstruct(ids, as_pylist(p.codebook))))
    bad = mutant(p.x, p.idx, bits, d, p.codebook)
    assert not np.allclose(bad, ref, rtol=1e-6, atol=1e-9)
