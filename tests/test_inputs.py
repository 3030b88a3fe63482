"""Seeded input generator: determinism, shapes, distributions, named workloads."""

import numpy as np
import pytest

import pq_inputs as pi


def test_tiny_workload_shapes_and_determinism():
    w = pi.workload("tiny")
    a = w.problem(0)
    b = w.problem(0)
    assert a.codebook.shape == (256, 4) and a.codebook.dtype == np.float16
    assert a.idx.shape == (128, 64) and a.idx.dtype == np.uint8
    assert a.x.shape == (1, 256) and a.x.dtype == np.float16
    for f in ("codebook", "ids", "idx", "x"):
        assert np.array_equal(getattr(a, f), getattr(b, f))


def test_matrices_get_independent_streams():
    w = pi.workload("llama3_8b_4bit")
    rng_a = pi.matrix_rng(0, w.workload_id, 0, 1)
    rng_b = pi.matrix_rng(0, w.workload_id, 0, 2)
    assert not np.array_equal(rng_a.integers(0, 256, 64), rng_b.integers(0, 256, 64))


def test_distributions():
    rng = np.random.default_rng(0)
    p = pi.draw_problem(rng, 4, 4096, 512, 2, 256, 8)
    cb = p.codebook.astype(np.float64)
    assert abs(cb.std() - 0.02) < 0.003
    x = p.x.astype(np.float64)
    assert abs(x.std() - 1.0) < 0.03
    counts = np.bincount(p.ids.ravel(), minlength=256)
    assert counts.min() > 0.8 * counts.mean()


def test_row_bytes():
    assert pi.row_bytes(2048, 8) == 2048
    assert pi.row_bytes(1024, 12) == 1536
    assert pi.row_bytes(3, 12) == 5
    assert pi.row_bytes(3072, 16) == 6144
    with pytest.raises(ValueError):
        pi.row_bytes(4, 10)


def test_workload_catalogue():
    assert [m.N for m in pi.workload("llama3_8b_4bit").matrices] == [4096, 1024, 1024, 4096, 14336, 14336, 4096]
    assert pi.workload("llama3_8b_3bit").matrices[-1].N == 128256
    q = pi.workload("qwen3_8b_sweep")
    assert (q.C, q.idx_bits, q.d, q.layers) == (65536, 16, 4, 36)
    assert pi.workload("prefill").Ms == (128, 512, 2048)


def test_pack_rejects_wide_ids():
    with pytest.raises(ValueError):
        pi.pack_indices(np.array([[256]]), 8)
    with pytest.raises(ValueError):
        pi.pack_indices(np.array([[4096]]), 12)


def test_draw_problem_validation():
    rng = np.random.default_rng(0)
    with pytest.raises(ValueError):
        pi.draw_problem(rng, 1, 10, 4, 4, 16, 8)      # K % d != 0
    with pytest.raises(ValueError):
        pi.draw_problem(rng, 1, 8, 4, 2, 300, 8)      # C > 2^bits


def test_subnormal_generators_draw_only_subnormals_and_signed_zeros():
    """Every value is +-k * 2**-24 with k in {0, 1, 2, 3} (or 512, 1023 in
    the wide variant): an fp16 exponent field of zero, both zero signs
    present."""
    rng = np.random.default_rng(0)
    for arr in (pi.subnormal_codebook(rng, 4096, 4), pi.subnormal_x(rng, 3, 4096),
                pi.subnormal_codebook(rng, 4096, 4, large_frac=0.05)):
        bits = arr.view(np.uint16)
        assert arr.dtype == np.float16
        assert np.all((bits & 0x7C00) == 0)               # exponent field 0: subnormal or zero
        k = bits & 0x03FF
        assert set(np.unique(k).tolist()) <= {0, 1, 2, 3, 512, 1023}
        assert np.any(bits == 0x8000) and np.any(bits == 0x0000)
        units = arr.astype(np.float64) / pi.FP16_SUBNORMAL_UNIT
        assert np.array_equal(np.abs(units), k.astype(np.float64))
    wide = pi.subnormal_codebook(rng, 4096, 4, large_frac=0.05).view(np.uint16) & 0x03FF
    assert np.any(wide == 1023) and np.any(wide == 512)
