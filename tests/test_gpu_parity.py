"""GPU parity: libfasq (through the C ABI) against the CPU oracle.

Index decoding and reconstruction must match bit for bit; y must satisfy
rel_L2 <= 1e-3 and max|err| <= 1e-2 * rms(y_ref); structured inputs whose
exact result fits fp16 must match bit for bit.  Full-size workloads are
checked on sampled output rows.
"""

import os

import numpy as np
import pytest

import pq_inputs as pi
from oracle import pq_oracle as orc
from gpu_util import assert_close, sample_rows, to_dev, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
fasq = pytest.importorskip("paper_2605_04084_amd")


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fasq.lib()
    yield
    torch.cuda.synchronize()


def run(entry, p, x=None):
    fn = fasq.pq_gemv if entry == "gemv" else fasq.pq_gemm
    x = p.x if x is None else x
    y = fn(to_dev(x), to_dev(p.idx), p.idx_bits, p.d, to_dev(p.codebook))
    return to_np(y).astype(np.float64)


# ---------------------------------------------------------------------------
# Reconstruction: bit-exact
# ---------------------------------------------------------------------------

RECON_CASES = [
    # N, K, d, C, bits
    (37, 64, 1, 256, 8),
    (129, 256, 2, 256, 8),
    (5, 12, 3, 7, 8),
    (64, 96, 4, 4096, 12),
    (33, 36, 4, 4096, 12),   # S = 9: odd 12-bit rows with a pad nibble
    (70, 56, 8, 100, 12),
    (17, 40, 4, 65536, 16),
    (300, 128, 2, 3000, 16),
]


@pytest.mark.parametrize("case", RECON_CASES)
def test_reconstruct_bit_exact(case):
    N, K, d, C, bits = case
    print(f"[case] reconstruct {case}", flush=True)
    rng = np.random.default_rng(sum(case))
    p = pi.draw_problem(rng, 1, K, N, d, C, bits)
    w = fasq.pq_reconstruct(to_dev(p.idx), K, bits, d, to_dev(p.codebook))
    ref = orc.reconstruct(p.idx, K, bits, d, p.codebook)
    assert np.array_equal(to_np(w).view(np.uint16), ref.view(np.uint16))


def test_reconstruct_preserves_special_values():
    specials = np.array([0x0000, 0x8000, 0x0001, 0x8001, 0x03FF, 0x83FF, 0x7C00, 0xFC00,
                         0x7E01, 0xFE55, 0x3C00, 0xBC00, 0x0200, 0x8200, 0x7BFF, 0xFBFF], dtype=np.uint16)
    cb = specials.view(np.float16).reshape(4, 4)
    rng = np.random.default_rng(5)
    ids = rng.integers(0, 4, size=(50, 24))
    for bits in (8, 12, 16):
        idx = pi.pack_indices(ids, bits)
        w = fasq.pq_reconstruct(to_dev(idx), 96, bits, 4, to_dev(cb))
        ref = orc.reconstruct(idx, 96, bits, 4, cb)
        assert np.array_equal(to_np(w).view(np.uint16), ref.view(np.uint16))


@pytest.mark.parametrize("wl,mat", [("llama3_8b_4bit", 4), ("llama3_8b_3bit", 7), ("qwen3_8b_sweep", 6)])
def test_reconstruct_full_size_sampled(wl, mat):
    print(f"[case] reconstruct full {wl} matrix {mat}", flush=True)
    p = pi.workload(wl).problem(mat)
    w = fasq.pq_reconstruct(to_dev(p.idx), p.K, p.idx_bits, p.d, to_dev(p.codebook))
    rows = sample_rows(p.N, 64)
    got = to_np(w[torch.from_numpy(rows).to(w.device)]).view(np.uint16)
    ref = orc.reconstruct(p.idx, p.K, p.idx_bits, p.d, p.codebook, rows=rows).view(np.uint16)
    assert np.array_equal(got, ref)


# ---------------------------------------------------------------------------
# y on the named workloads (full size, sampled rows)
# ---------------------------------------------------------------------------

def test_gemv_tiny_workload():
    p = pi.workload("tiny").problem(0)
    y = run("gemv", p)
    assert_close(y, orc.pq_linear(p.x, p.idx, 8, 4, p.codebook), "tiny")


@pytest.mark.parametrize("mat", range(7))
def test_gemv_llama3_8b_4bit(mat):
    w = pi.workload("llama3_8b_4bit")
    print(f"[case] gemv 4bit {w.matrices[mat]}", flush=True)
    p = w.problem(mat)
    y = run("gemv", p)
    rows = sample_rows(p.N)
    assert_close(y[:, rows], orc.pq_linear(p.x, p.idx, p.idx_bits, p.d, p.codebook, rows=rows),
                 f"4bit {w.matrices[mat].name}")


@pytest.mark.parametrize("mat", range(8))
def test_gemv_llama3_8b_3bit(mat):
    w = pi.workload("llama3_8b_3bit")
    print(f"[case] gemv 3bit {w.matrices[mat]}", flush=True)
    p = w.problem(mat)
    y = run("gemv", p)
    rows = sample_rows(p.N)
    assert_close(y[:, rows], orc.pq_linear(p.x, p.idx, p.idx_bits, p.d, p.codebook, rows=rows),
                 f"3bit {w.matrices[mat].name}")


@pytest.mark.parametrize("M", [1, 4, 16])
@pytest.mark.parametrize("mat", [0, 1, 4, 6])
def test_gemv_qwen3_8b_sweep(M, mat):
    w = pi.workload("qwen3_8b_sweep")
    print(f"[case] gemv qwen M={M} {w.matrices[mat]}", flush=True)
    p = w.problem(mat, M=M)
    y = run("gemv", p)
    rows = sample_rows(p.N)
    assert_close(y[:, rows], orc.pq_linear(p.x, p.idx, p.idx_bits, p.d, p.codebook, rows=rows),
                 f"qwen M={M} {w.matrices[mat].name}")


@pytest.mark.parametrize("M", [128, 512, 2048])
@pytest.mark.parametrize("mat", range(3))
def test_gemm_prefill(M, mat):
    w = pi.workload("prefill")
    print(f"[case] gemm prefill M={M} {w.matrices[mat]}", flush=True)
    p = w.problem(mat, M=M)
    y = run("gemm", p)
    rows = sample_rows(p.N, 128)
    assert_close(y[:, rows], orc.pq_linear(p.x, p.idx, p.idx_bits, p.d, p.codebook, rows=rows),
                 f"prefill M={M} {w.matrices[mat].name}")


WIDE_TILE = [
    # M, K, N, d, C, bits: enough output tiles for the 128 x 256 GEMM tile, ragged M and N
    (1030, 256, 16400, 2, 256, 8),
    (1030, 384, 16400, 4, 4096, 12),
    (1100, 256, 16500, 4, 65536, 16),
    (1025, 128, 16390, 8, 256, 8),
    (1030, 320, 16400, 4, 256, 8),      # the 256 x 256 tile (half-row codebook, 16 copies)
]


def test_gemm_tile_choice():
    """Enough 256 x 256 tiles to fill the CUs: the big tile with the half-row
    codebook (one copy for 4096 entries); fewer: 128 x 256 with the
    replicated codebook."""
    assert fasq.plan("gemm", 2048, 4096, 14336, 8, 4, 256).startswith("k_gemm_mfma<8, 4, 5, 256, 256, 2, 4, ")
    assert fasq.plan("gemm", 2048, 4096, 14336, 8, 8, 256).startswith("k_gemm_mfma<8, 8, 5, 256, 256, 2, 4, ")
    assert fasq.plan("gemm", 2048, 4096, 14336, 12, 4, 4096).startswith("k_gemm_mfma<12, 4, 1, 256, 256, 2, 4, ")
    assert fasq.plan("gemm", 2048, 4096, 4096, 8, 4, 256).startswith("k_gemm_mfma<8, 4, 0, 128, 256, 2, 4, ")
    assert fasq.plan("gemm", 512, 4096, 14336, 8, 4, 256).startswith("k_gemm_mfma<8, 4, 0, 128, 256, 2, 4, ")
    # sub-vectors of 1 or 2, or 16-bit ids, would spill in the big tile
    assert fasq.plan("gemm", 2048, 4096, 14336, 8, 2, 256).startswith("k_gemm_mfma<8, 2, 0, 128, 256, ")
    assert fasq.plan("gemm", 2048, 4096, 14336, 16, 4, 65536).startswith("k_gemm_mfma<16, 4, 2, 128, 256, ")


@pytest.mark.parametrize("case", [(777, 448, 12345, 4, 256, 8), (600, 384, 16400, 4, 4096, 12)])
def test_gemm_big_tile_one_hot_bit_exact(case):
    """Exact small-integer results on the 256 x 256 tile with ragged M, N and
    an odd number of K chunks."""
    M, K, N, d, C, bits = case
    print(f"[case] gemm big tile {case}", flush=True)
    assert ", 256, 256, " in fasq.plan("gemm", M, K, N, bits, d, C)
    rng = np.random.default_rng(5 + sum(case))
    cb = pi.signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, K // d))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    assert np.abs(ref).max() <= 2048
    y = to_np(fasq.pq_gemm(to_dev(x), to_dev(idx), bits, d, to_dev(cb))).astype(np.float64)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("case", WIDE_TILE)
def test_gemm_wide_tiles(case):
    M, K, N, d, C, bits = case
    print(f"[case] gemm wide tile {case}", flush=True)
    rng = np.random.default_rng(sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    y = run("gemm", p)
    rows = np.unique(np.concatenate([sample_rows(N, 96), np.arange(N - 40, N)]))
    assert_close(y[:, rows], orc.pq_linear(p.x, p.idx, bits, d, p.codebook, rows=rows), f"wide {case}")


# ---------------------------------------------------------------------------
# Ragged and small shapes, every id width and sub-vector length
# ---------------------------------------------------------------------------

RAGGED = [
    # M, K, N, d, C, bits
    (1, 256, 129, 2, 256, 8),
    (1, 4096 + 512, 1000, 2, 256, 8),   # row not a multiple of the per-wave span
    (1, 320, 77, 4, 256, 8),
    (1, 1024, 33, 1, 256, 8),
    (1, 2048, 50, 8, 256, 8),
    (1, 128 * 12, 260, 4, 4096, 12),
    (1, 4096, 31, 2, 4096, 12),
    (1, 4096, 45, 4, 65536, 16),
    (1, 512, 64, 2, 1000, 16),
    (1, 36, 5, 4, 9, 12),               # odd 12-bit rows: general kernel
    (1, 30, 7, 3, 11, 8),               # d = 3: general kernel
    (1, 24, 9, 24, 40, 8),              # full vector quantization, d = K
    (2, 4096, 1000, 2, 256, 8),         # two tokens: the row-streaming kernel
    (2, 320, 77, 4, 256, 8),            # two tokens, masked chunk tail
    (2, 128 * 12, 260, 4, 4096, 12),    # two tokens, one codebook copy in LDS
    (2, 4096, 45, 4, 65536, 16),        # two tokens, codebook larger than LDS: the M <= 16 kernel
    (3, 256, 100, 4, 256, 8),
    (5, 192, 70, 2, 256, 8),
    (17, 640, 200, 4, 256, 8),
    (37, 320, 130, 2, 300, 16),
    (64, 128, 64, 8, 256, 8),
    (130, 256, 257, 4, 4096, 12),
    (33, 64, 50, 1, 256, 8),
    (16, 4096, 200, 2, 256, 8),         # 16 rows of x leave no room for the replicated table
    (1, 320, 20000, 4, 256, 8),         # enough rows per workgroup for the replicated table, masked tail
    (1, 1024, 9000, 1, 256, 8),
]


@pytest.mark.parametrize("entry", ["gemv", "gemm"])
@pytest.mark.parametrize("case", RAGGED)
def test_ragged_shapes(entry, case):
    M, K, N, d, C, bits = case
    print(f"[case] {entry} ragged {case}", flush=True)
    rng = np.random.default_rng(sum(case) + (entry == "gemm"))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    y = run(entry, p)
    assert_close(y, orc.pq_linear(p.x, p.idx, bits, d, p.codebook), f"{entry} {case}")


# ---------------------------------------------------------------------------
# Exact cases, determinism, path invariance, alignment, linearity
# ---------------------------------------------------------------------------

ONE_HOT = [
    (1, 4096, 300, 2, 256, 8),
    (1, 4096, 100, 4, 4096, 12),
    (1, 2048, 64, 4, 65536, 16),
    (1, 1024, 70, 1, 256, 8),
    (1, 2048, 40, 8, 256, 8),
    (16, 4096, 64, 4, 65536, 16),
    (200, 1024, 150, 4, 256, 8),
]


@pytest.mark.parametrize("entry", ["gemv", "gemm"])
@pytest.mark.parametrize("case", ONE_HOT)
def test_signed_one_hot_is_bit_exact(entry, case):
    """Codewords in {0, +-1} and x in {-1, 0, 1}: every partial sum is a small
    integer, so the kernels must reproduce the oracle exactly."""
    M, K, N, d, C, bits = case
    rng = np.random.default_rng(77 + sum(case))
    cb = pi.signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, K // d))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    assert np.abs(ref).max() <= 2048
    fn = fasq.pq_gemv if entry == "gemv" else fasq.pq_gemm
    y = to_np(fn(to_dev(x), to_dev(idx), bits, d, to_dev(cb))).astype(np.float64)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("entry", ["gemv", "gemm"])
def test_repeated_launches_are_bitwise_identical(entry):
    p = pi.workload("llama3_8b_4bit").problem(4) if entry == "gemv" else pi.workload("prefill").problem(0, M=128)
    x, idx, cb = to_dev(p.x), to_dev(p.idx), to_dev(p.codebook)
    fn = fasq.pq_gemv if entry == "gemv" else fasq.pq_gemm
    a = fn(x, idx, p.idx_bits, p.d, cb)
    b = fn(x, idx, p.idx_bits, p.d, cb)
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


@pytest.mark.parametrize("case", [(1, 4096, 1024, 2, 256, 8), (1, 4096, 512, 4, 4096, 12),
                                  (4, 4096, 300, 4, 65536, 16), (96, 512, 200, 4, 256, 8)])
def test_tuned_kernels_match_general_kernel(case, monkeypatch):
    M, K, N, d, C, bits = case
    rng = np.random.default_rng(3 + sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    fast = run("gemv", p)
    monkeypatch.setenv("FASQ_FORCE_PATH", "generic")
    slow = run("gemv", p)
    ref = orc.pq_linear(p.x, p.idx, bits, d, p.codebook)
    assert_close(fast, ref, "tuned")
    assert_close(slow, ref, "general")


@pytest.mark.parametrize("entry", ["gemv", "gemm"])
def test_unaligned_buffers_take_a_correct_path(entry):
    rng = np.random.default_rng(8)
    M, K, N, d, C, bits = (1 if entry == "gemv" else 40), 1024, 96, 2, 256, 8
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    # offset every buffer by a few bytes inside a larger allocation
    xb = torch.zeros(M * K + 1, dtype=torch.float16, device="cuda:0")
    xb[1:].copy_(to_dev(p.x).view(-1))
    ib = torch.zeros(p.idx.size + 3, dtype=torch.uint8, device="cuda:0")
    ib[3:].copy_(to_dev(p.idx).view(-1))
    cbb = torch.zeros(C * d + 1, dtype=torch.float16, device="cuda:0")
    cbb[1:].copy_(to_dev(p.codebook).view(-1))
    yb = torch.zeros(M * N + 1, dtype=torch.float16, device="cuda:0")
    fn = fasq.gemv_raw if entry == "gemv" else fasq.gemm_raw
    st = fn(xb.data_ptr() + 2, M, K, N, ib.data_ptr() + 3, bits, d, cbb.data_ptr() + 2, C,
            yb.data_ptr() + 2, torch.cuda.current_stream().cuda_stream)
    assert st == fasq.FASQ_OK
    y = to_np(yb[1:]).astype(np.float64).reshape(M, N)
    assert_close(y, orc.pq_linear(p.x, p.idx, bits, d, p.codebook), f"unaligned {entry}")


def test_linearity_in_x_on_gpu():
    rng = np.random.default_rng(9)
    p = pi.draw_problem(rng, 1, 4096, 512, 2, 256, 8)
    x1 = (rng.integers(-8, 9, size=(1, 4096)) / 8).astype(np.float16)
    x2 = (rng.integers(-8, 9, size=(1, 4096)) / 8).astype(np.float16)
    y1 = run("gemv", p, x1)
    y2 = run("gemv", p, x2)
    y12 = run("gemv", p, (x1.astype(np.float64) + x2).astype(np.float16))
    ref = orc.pq_linear(x1.astype(np.float64) + x2, p.idx, 8, 2, p.codebook)
    assert_close(y12, ref, "x1+x2")
    assert_close(y1 + y2, ref, "y(x1)+y(x2)")


def test_errors_surface_as_exceptions():
    x = torch.zeros((1, 16), dtype=torch.float16, device="cuda:0")
    idx = torch.zeros((4, 8), dtype=torch.uint8, device="cuda:0")
    cb = torch.zeros((256, 2), dtype=torch.float16, device="cuda:0")
    with pytest.raises(ValueError):
        fasq.pq_gemv(x, idx[:, :4], 8, 2, cb)          # wrong row bytes
    with pytest.raises(TypeError):
        fasq.pq_gemv(x.float(), idx, 8, 2, cb)
    with pytest.raises(ValueError):
        fasq.pq_gemv(torch.zeros((16, 2), dtype=torch.float16, device="cuda:0").t(), idx, 8, 2, cb)
    st = fasq.gemv_raw(x.data_ptr(), 1, 16, 4, idx.data_ptr(), 8, 2, cb.data_ptr(), 300, x.data_ptr(), 0)
    assert st == fasq.FASQ_ERR_INVALID_ARG


# ---------------------------------------------------------------------------
# Several matrices sharing x in one call (fasq_pq_gemv_batched)
# ---------------------------------------------------------------------------

def _batched(x, probs, bits, d):
    ys = fasq.pq_gemv_batched(to_dev(x), [to_dev(p.idx) for p in probs], bits, d,
                              [to_dev(p.codebook) for p in probs])
    return [to_np(y) for y in ys]


BATCH_CASES = [
    # M, K, d, bits, [(N, C), ...]
    (1, 4096, 2, 8, [(4096, 256), (1024, 256), (1024, 256)]),      # q, k, v shapes
    (1, 4096, 2, 8, [(14336, 256), (14336, 256)]),                 # gate, up shapes
    (1, 256, 2, 8, [(1, 256), (300, 256), (17, 64), (129, 8)]),    # ragged N, mixed C
    (1, 512, 4, 12, [(100, 4096), (33, 4096), (257, 1000)]),
    (1, 320, 4, 16, [(64, 65536), (65, 300)]),
    (1, 256, 2, 8, [(40 + 7 * i, 256) for i in range(11)]),        # more than one launch's worth
    (1, 1024, 2, 8, [(5000, 256), (3, 256)]),                      # a large matrix cut in uneven parts
    (1, 640, 4, 12, [(2049, 4096), (700, 4096), (1, 4096)]),       # parts of several sizes, one 1-row matrix
    (2, 4096, 2, 8, [(4096, 256), (1024, 256), (1024, 256)]),      # two tokens, one launch
    (2, 512, 4, 12, [(300, 4096), (129, 1000)]),                   # two tokens, ragged N, mixed C
    (3, 256, 2, 8, [(70, 256), (130, 256)]),                       # M > 2: the 16-row-tile kernel, one launch
    (4, 4096, 2, 8, [(4096, 256), (1024, 256), (1024, 256)]),      # q, k, v shapes, four tokens
    (16, 1024, 2, 8, [(5000, 256), (3, 256)]),                     # sixteen tokens, uneven parts
    (8, 512, 4, 12, [(300, 4096), (129, 1000), (1, 4096)]),        # ragged N, mixed C, a 1-row matrix
    (7, 640, 4, 12, [(2049, 4096), (700, 4096), (1, 4096)]),       # rows not a whole number of wave spans
    (5, 320, 4, 16, [(64, 65536), (65, 300)]),                     # codebook gathered from global memory
    (2, 320, 4, 16, [(64, 65536), (65, 300)]),                     # two tokens, codebook too large for LDS
    (2, 4096, 4, 16, [(4096, 65536), (1024, 300)]),                # the same mix at full row count
    (4, 256, 2, 8, [(40 + 7 * i, 256) for i in range(11)]),        # more than one launch's worth
    (1, 96, 3, 8, [(20, 7), (9, 5)]),                              # d = 3: general kernel
    (4, 96, 3, 8, [(20, 7), (9, 5)]),                              # d = 3, four tokens
]


@pytest.mark.parametrize("case", BATCH_CASES)
def test_batched_matches_single_calls_and_oracle(case):
    M, K, d, bits, mats = case
    print(f"[case] batched {case}", flush=True)
    rng = np.random.default_rng(len(mats) * 1000 + K)
    probs = [pi.draw_problem(rng, M, K, N, d, C, bits) for N, C in mats]
    x = probs[0].x
    got = _batched(x, probs, bits, d)
    for i, p in enumerate(probs):
        single = to_np(fasq.pq_gemv(to_dev(x), to_dev(p.idx), bits, d, to_dev(p.codebook)))
        assert np.array_equal(got[i].view(np.uint16), single.view(np.uint16)), f"matrix {i}"
        rows = sample_rows(p.N)
        ref = orc.pq_linear(x, p.idx, bits, d, p.codebook, rows=rows)
        assert_close(got[i].astype(np.float64)[:, rows], ref, f"batched matrix {i}")


@pytest.mark.parametrize("wl", ["llama3_8b_4bit", "llama3_8b_3bit"])
def test_batched_layer_groups_full_size(wl):
    """q/k/v and gate/up of the effective-4-bit and effective-3-bit layers as
    grouped launches, every output row against the oracle."""
    w = pi.workload(wl)
    for group in ((0, 1, 2), (4, 5)):
        print(f"[case] batched full {wl} {group}", flush=True)
        probs = [w.problem(i) for i in group]
        x = probs[0].x
        got = _batched(x, probs, probs[0].idx_bits, probs[0].d)
        for g, p in zip(got, probs):
            assert np.isfinite(g).all()
            ref = orc.pq_linear(x, p.idx, p.idx_bits, p.d, p.codebook)
            assert_close(g.astype(np.float64), ref, f"{wl} group {group} (all rows)")


def test_batched_one_hot_bit_exact():
    """Signed one-hot codebooks with ternary x: every partial sum is an exact
    integer, so each grouped output equals the oracle bit for bit."""
    rng = np.random.default_rng(77)
    K, d = 1024, 2
    x = pi.ternary_x(rng, 1, K)
    probs = []
    for N in (513, 64, 1000):
        cb = pi.signed_one_hot_codebook(256, d, rng)
        ids = rng.integers(0, 256, size=(N, K // d))
        probs.append(pi.PQProblem(M=1, K=K, N=N, d=d, C=256, idx_bits=8, codebook=cb, ids=ids,
                                  idx=pi.pack_indices(ids, 8), x=x))
    got = _batched(x, probs, 8, d)
    for g, p in zip(got, probs):
        ref = orc.pq_linear(x, p.idx, 8, d, p.codebook)
        assert np.array_equal(g.astype(np.float64), ref)


# ---------------------------------------------------------------------------
# Codebooks larger than LDS, staged slice by slice (one pass per slice)
# ---------------------------------------------------------------------------

SLICED = [
    # M, K, N, d, C, bits: the decode kernels take the codebook in LDS slices
    (1, 4096, 300, 4, 40000, 16),    # 3 slices of 16384 entries, the last one partial
    (1, 2048, 100, 2, 65536, 16),    # 2 slices of 32768
    (1, 1024, 200, 8, 65536, 16),    # 8 slices of 8192
    (1, 4096, 64, 1, 65536, 16),     # 1 slice: the whole 128 KB codebook
    (1, 12288, 70, 4, 65536, 16),    # wide x beside the slice
    (2, 2048, 100, 1, 65536, 16),    # several tokens: one slice beside x and the partials
    (4, 1024, 64, 1, 60000, 16),
]


@pytest.mark.parametrize("case", SLICED)
def test_sliced_codebook(case):
    M, K, N, d, C, bits = case
    print(f"[case] gemv sliced codebook {case}", flush=True)
    assert ", 3, " in fasq.plan("gemv", M, K, N, bits, d, C)  # CB_SLICE
    rng = np.random.default_rng(sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    assert_close(run("gemv", p), orc.pq_linear(p.x, p.idx, bits, d, p.codebook), f"sliced {case}")


@pytest.mark.parametrize("case", SLICED)
def test_sliced_codebook_boundaries_bit_exact(case):
    """Ids on both sides of every slice boundary, and the last id, with
    signed one-hot codewords: exact integers, so bit-exact."""
    M, K, N, d, C, bits = case
    print(f"[case] gemv sliced boundaries {case}", flush=True)
    rng = np.random.default_rng(5 + sum(case))
    cb = pi.signed_one_hot_codebook(C, d, rng)
    edges = []
    for shift in (13, 14, 15, 16):
        for b in range(1 << shift, C, 1 << shift):
            edges += [b - 1, b]
    edges = np.unique(np.array(edges + [0, C - 1]))
    ids = rng.choice(edges, size=(N, K // d))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    assert np.abs(ref).max() <= 2048
    y = to_np(fasq.pq_gemv(to_dev(x), to_dev(idx), bits, d, to_dev(cb))).astype(np.float64)
    assert np.array_equal(y, ref)


def test_wide_x_in_registers_keeps_the_replicated_codebook():
    """M = 16 at K = 4096 keeps the decode kernel: x goes from global memory
    straight to registers and takes no LDS, so the replicated codebook
    (mode 0) still fits; with x in LDS (a masked row) it drops to one copy
    (mode 1)."""
    assert fasq.plan("gemv", 16, 4096, 4096, 8, 2, 256) == "k_gemv<8, 2, 2, 0, 16, 0>"
    assert ", 1, 16, 1>" in fasq.plan("gemv", 16, 4096 + 64, 4096, 8, 2, 256)


# ---------------------------------------------------------------------------
# Prefill GEMM with K split over two groups of waves inside the workgroup
# ---------------------------------------------------------------------------

K_GROUPS = [
    # M, K, N, d, C, bits: small grids (64-row tiles, two K groups); an odd
    # number of 64-wide K chunks leaves the second group one chunk short
    (8, 192, 64, 2, 256, 8),
    (40, 320, 100, 4, 256, 8),
    (64, 4096 + 64, 130, 4, 4096, 12),
    (100, 1088, 70, 4, 65536, 16),
]


@pytest.mark.parametrize("case", K_GROUPS)
def test_gemm_k_groups_one_hot_bit_exact(case):
    """Exact small-integer results: a chunk summed twice or dropped by a
    group would show as an exact mismatch."""
    M, K, N, d, C, bits = case
    print(f"[case] gemm k groups {case}", flush=True)
    assert fasq.plan("gemm", M, K, N, bits, d, C).endswith(", 2>")
    rng = np.random.default_rng(11 + sum(case))
    cb = pi.signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, K // d))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    assert np.abs(ref).max() <= 2048
    y = to_np(fasq.pq_gemm(to_dev(x), to_dev(idx), bits, d, to_dev(cb))).astype(np.float64)
    assert np.array_equal(y, ref)


# ---------------------------------------------------------------------------
# The paper's lookup-table GEMM (Alg. 3), kept for comparison
# ---------------------------------------------------------------------------

LUT_CASES = [
    # M, K, N, d, C, bits
    (5, 256, 300, 2, 256, 8),      # ragged tokens and features
    (128, 512, 256, 4, 256, 8),
    (9, 320, 77, 1, 64, 8),
    (16, 512, 130, 8, 256, 16),
    (12, 384, 90, 4, 2048, 12),    # one subspace per table batch
    (3, 36, 20, 4, 9, 12),         # odd 12-bit rows, batch past the last subspace
]


@pytest.mark.parametrize("case", LUT_CASES)
def test_lut_gemm_matches_oracle(case):
    M, K, N, d, C, bits = case
    print(f"[case] lut gemm {case}", flush=True)
    rng = np.random.default_rng(31 + sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    y = to_np(fasq.pq_gemm_lut(to_dev(p.x), to_dev(p.idx), bits, d, to_dev(p.codebook))).astype(np.float64)
    assert_close(y, orc.pq_linear(p.x, p.idx, bits, d, p.codebook), f"lut {case}")


def test_lut_gemm_one_hot_is_bit_exact():
    M, K, N, d, C, bits = 20, 1024, 200, 2, 256, 8
    rng = np.random.default_rng(41)
    cb = pi.signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, K // d))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    y = to_np(fasq.pq_gemm_lut(to_dev(x), to_dev(idx), bits, d, to_dev(cb))).astype(np.float64)
    assert np.array_equal(y, ref)


def test_lut_gemm_rejects_tables_larger_than_lds():
    x = torch.zeros((2, 64), dtype=torch.float16, device="cuda:0")
    idx = torch.zeros((4, 64 * 12 // 8 // 4), dtype=torch.uint8, device="cuda:0")
    cb = torch.zeros((4096, 4), dtype=torch.float16, device="cuda:0")
    y = torch.empty((2, 4), dtype=torch.float16, device="cuda:0")
    st = fasq.gemm_lut_raw(x.data_ptr(), 2, 64, 4, idx.data_ptr(), 12, 4, cb.data_ptr(), 4096, y.data_ptr(), 0)
    assert st == fasq.FASQ_ERR_UNSUPPORTED
    assert "C <= 2048" in fasq.last_error()


def test_codebook_placement_follows_the_work_per_workgroup():
    """Few ids per workgroup: one LDS copy of the codebook (mode 1); many: the
    replicated table (mode 0)."""
    assert fasq.plan("gemv", 1, 256, 128, 8, 4, 256) == "k_gemv_m1<8, 4, 1, 1, 1>"
    assert fasq.plan("gemv", 1, 4096, 4096, 8, 2, 256) == "k_gemv_m1<8, 2, 2, 0, 0>"
    assert fasq.plan("gemv_batched", 1, 4096, 4096, 8, 2, 256) == "k_gemv_m1<8, 2, 2, 0, 0>"
    assert fasq.plan("gemv_batched", 2, 4096, 4096, 8, 2, 256).startswith("k_gemv_mt<8, 2, ")
    assert fasq.plan("gemv", 2, 4096, 4096, 8, 2, 256).startswith("k_gemv_mt<8, 2, ")
    assert fasq.plan("gemv_batched", 4, 4096, 4096, 8, 2, 256).startswith("k_gemv<")
    # two tokens with a codebook too large for LDS: the 16-row-tile kernel, the codebook's first
    # entries in LDS and the rest gathered from global memory (mode 4)
    assert fasq.plan("gemv_batched", 2, 320, 64, 16, 4, 65536) == "k_gemv<16, 4, 1, 4, 16, 1>"
    assert fasq.plan("gemv", 1, 320, 20000, 8, 4, 256).startswith("k_gemv_m1<8, 4, 1, 0, ")


# ---------------------------------------------------------------------------
# Prefill with K split over workgroups (fasq_pq_gemm_ex and its workspace)
# ---------------------------------------------------------------------------

SPLIT_K = [
    # M, K, N, d, C, bits: grids that leave CUs idle
    (8, 4096, 512, 4, 256, 8),           # 8 tiles: eight K ranges
    (128, 4096, 4096, 4, 256, 8),        # the prefill q_proj shape at M = 128
    (130, 4096 + 64 * 3, 700, 2, 256, 8),
    (40, 14336, 200, 4, 4096, 12),
    (33, 2048, 100, 4, 65536, 16),
]


def _gemm_ex(x, idx, bits, d, cb, ws_bytes=None):
    need = fasq.gemm_ex_workspace_bytes(x.shape[0], x.shape[1], idx.shape[0], bits, d, cb.shape[0])
    n = need if ws_bytes is None else ws_bytes
    ws = torch.zeros(max(n, 4), dtype=torch.uint8, device="cuda:0")
    y = torch.empty((x.shape[0], idx.shape[0]), dtype=torch.float16, device="cuda:0")
    xd, idd, cbd = to_dev(x), to_dev(idx), to_dev(cb)  # held until the call has run
    st = fasq.gemm_ex_raw(xd.data_ptr(), x.shape[0], x.shape[1], idx.shape[0], idd.data_ptr(), bits, d,
                          cbd.data_ptr(), cb.shape[0], y.data_ptr(), ws.data_ptr(), n, 0)
    assert st == fasq.FASQ_OK, fasq.last_error()
    torch.cuda.synchronize()
    return to_np(y), need


@pytest.mark.parametrize("case", SPLIT_K)
def test_gemm_split_k_one_hot_bit_exact(case):
    """Exact small-integer results: a K range summed twice or dropped would
    show as an exact mismatch."""
    M, K, N, d, C, bits = case
    print(f"[case] gemm split k {case}", flush=True)
    rng = np.random.default_rng(23 + sum(case))
    cb = pi.signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, K // d))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    assert np.abs(ref).max() <= 2048
    y, need = _gemm_ex(x, idx, bits, d, cb)
    assert need > 0  # the call does split
    assert np.array_equal(y.astype(np.float64), ref)


@pytest.mark.parametrize("case", SPLIT_K[:3])
def test_gemm_split_k_random_against_oracle(case):
    M, K, N, d, C, bits = case
    print(f"[case] gemm split k random {case}", flush=True)
    rng = np.random.default_rng(29 + sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    y, need = _gemm_ex(p.x, p.idx, bits, d, p.codebook)
    assert need > 0
    assert_close(y, orc.pq_linear(p.x, p.idx, bits, d, p.codebook), f"split k {case}")
    # deterministic: the same call gives the same bits
    y2, _ = _gemm_ex(p.x, p.idx, bits, d, p.codebook)
    assert np.array_equal(y.view(np.uint16), y2.view(np.uint16))


def test_gemm_ex_small_workspace_is_the_plain_gemm():
    M, K, N, d, C, bits = SPLIT_K[1]
    rng = np.random.default_rng(31)
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    y_small, need = _gemm_ex(p.x, p.idx, bits, d, p.codebook, ws_bytes=16)
    assert need > 16
    y_plain = to_np(fasq.pq_gemm(to_dev(p.x), to_dev(p.idx), bits, d, to_dev(p.codebook)))
    assert np.array_equal(y_small.view(np.uint16), y_plain.view(np.uint16))


def test_gemm_ex_no_split_for_full_grids():
    assert fasq.gemm_ex_workspace_bytes(2048, 4096, 14336, 8, 4, 256) == 0
    assert fasq.gemm_ex_workspace_bytes(128, 4096, 4096, 8, 4, 256) == 2 * 128 * 4096 * 4


def test_gemv_ex_shared_codebook_gemm_fallback_splits_k():
    """fasq_pq_gemv_ex with one shared codebook hands M > 16 to the GEMM, which
    splits K with the workspace; exact on small-integer data."""
    M, K, N, d, C, bits = 20, 2048, 300, 4, 256, 8
    assert fasq.gemv_ex_workspace_bytes(1, K, N, bits, d, C, 0) == 0
    need = fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, 0)
    assert need > 0
    rng = np.random.default_rng(37)
    cb = pi.signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, K // d))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    xd, idd, cbd = to_dev(x), to_dev(idx), to_dev(cb)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda:0")
    y = torch.empty((M, N), dtype=torch.float16, device="cuda:0")
    st = fasq.gemv_ex_raw(xd.data_ptr(), M, K, N, idd.data_ptr(), bits, d, cbd.data_ptr(), C, 0, y.data_ptr(),
                          ws.data_ptr(), need, 0)
    assert st == fasq.FASQ_OK, fasq.last_error()
    assert np.array_equal(to_np(y).astype(np.float64), ref)


# ---------------------------------------------------------------------------
# Codebooks larger than LDS at 2 to 16 tokens: the first entries in LDS, the
# rest gathered from global memory, in one pass
# ---------------------------------------------------------------------------

SPLIT_BOOK = [
    # M, K, N, d, C, bits
    (4, 4096, 300, 4, 65536, 16),       # Qwen3-8B-like rows at four tokens, ragged N
    (7, 2048, 129, 4, 40000, 16),       # C not a power of two
    (3, 512, 4100, 8, 30000, 16),       # d = 8
    (2, 1024, 1000, 2, 65536, 16),      # d = 2, two tokens
]


@pytest.mark.parametrize("case", SPLIT_BOOK)
def test_split_codebook_one_hot_bit_exact(case):
    """Exact small-integer results: an id read from the wrong place (LDS for
    an entry past the staged ones, or the wrong entry) shows as a mismatch."""
    M, K, N, d, C, bits = case
    print(f"[case] split codebook one-hot {case}", flush=True)
    assert fasq.plan("gemv", M, K, N, bits, d, C).split(", ")[3] == "4"
    rng = np.random.default_rng(47 + sum(case))
    cb = pi.signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, K // d))
    ids[:, 0] = C - 1   # the last entry, from global memory
    ids[:, 1] = 0       # the first entry, from LDS
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    y = to_np(fasq.pq_gemv(to_dev(x), to_dev(idx), bits, d, to_dev(cb)))
    assert np.array_equal(y.astype(np.float64), ref)


@pytest.mark.parametrize("case", SPLIT_BOOK[:2])
def test_split_codebook_random_against_oracle(case):
    M, K, N, d, C, bits = case
    print(f"[case] split codebook random {case}", flush=True)
    rng = np.random.default_rng(53 + sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    y = run("gemv", p)
    assert_close(y, orc.pq_linear(p.x, p.idx, bits, d, p.codebook), f"split codebook {case}")


# ---------------------------------------------------------------------------
# The 16-row-tile decode kernel with x staged in K slabs (rows of x too long
# for LDS)
# ---------------------------------------------------------------------------

SLAB_DECODE = [
    # M, K, N, d, C, bits
    (8, 14336, 300, 2, 256, 8),        # down_proj rows at 8 tokens
    (16, 12288, 200, 4, 65536, 16),    # Qwen3-8B down_proj rows at 16 tokens, codebook head in LDS
    (12, 14336 + 128, 70, 2, 256, 8),  # slabs of unequal length
    (6, 28672, 90, 2, 256, 8),
    (16, 14336, 130, 4, 4096, 12),
    (10, 16384, 64, 1, 256, 8),
]


@pytest.mark.parametrize("case", SLAB_DECODE)
def test_decode_kernel_x_slabs(case):
    M, K, N, d, C, bits = case
    print(f"[case] gemv x slabs {case}", flush=True)
    assert fasq.plan("gemv", M, K, N, bits, d, C).startswith("k_gemv<"), fasq.plan("gemv", M, K, N, bits, d, C)
    rng = np.random.default_rng(71 + sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    y = run("gemv", p)
    assert np.isfinite(y).all()
    assert_close(y, orc.pq_linear(p.x, p.idx, bits, d, p.codebook), f"x slabs {case}")


@pytest.mark.parametrize("case", SLAB_DECODE)
def test_decode_kernel_x_slabs_one_hot_bit_exact(case):
    """Exact small-integer results: a slab summed twice or skipped shows as
    an exact mismatch."""
    M, K, N, d, C, bits = case
    print(f"[case] gemv x slabs one-hot {case}", flush=True)
    rng = np.random.default_rng(73 + sum(case))
    cb = pi.signed_one_hot_codebook(C, d, rng)
    ids = rng.integers(0, C, size=(N, K // d))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = orc.pq_linear(x, idx, bits, d, cb)
    assert np.abs(ref).max() <= 2048
    y = to_np(fasq.pq_gemv(to_dev(x), to_dev(idx), bits, d, to_dev(cb))).astype(np.float64)
    assert np.array_equal(y, ref)


@pytest.mark.parametrize("M", [8, 12, 16])
def test_batched_x_slabs(M):
    """Grouped launches with x in slabs equal single calls bit for bit."""
    rng = np.random.default_rng(79 + M)
    K, d, bits = 14336, 2, 8
    probs = [pi.draw_problem(rng, M, K, N, d, C, bits) for N, C in ((500, 256), (130, 256), (33, 200))]
    x = probs[0].x
    got = _batched(x, probs, bits, d)
    for i, p in enumerate(probs):
        single = to_np(fasq.pq_gemv(to_dev(x), to_dev(p.idx), bits, d, to_dev(p.codebook)))
        assert np.array_equal(got[i].view(np.uint16), single.view(np.uint16)), f"matrix {i}"
        assert_close(got[i].astype(np.float64), orc.pq_linear(x, p.idx, bits, d, p.codebook), f"batched M={M} {i}")


@pytest.mark.parametrize("case", [(12, 14336, 300, 2, 256, 8), (16, 14336, 130, 4, 4096, 12)])
def test_decode_with_workspace_takes_the_gemm_past_the_crossover(case):
    """From 12 tokens on, a decode call whose x needs slabs goes to the GEMM
    with its K split when it has a workspace (the measured crossover); it
    then equals fasq_pq_gemm_ex bit for bit, while fasq_pq_gemv (no
    workspace) keeps the decode kernel."""
    M, K, N, d, C, bits = case
    print(f"[case] crossover dispatch {case}", flush=True)
    assert fasq.plan("gemv", M, K, N, bits, d, C).startswith("k_gemv<")
    need = fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, 0)
    assert need > 0 and need == fasq.gemm_ex_workspace_bytes(M, K, N, bits, d, C)
    rng = np.random.default_rng(83 + sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    ws = torch.empty(need, dtype=torch.uint8, device="cuda:0")
    y_ex = to_np(fasq.pq_gemv_ex(to_dev(p.x), to_dev(p.idx), bits, d, to_dev(p.codebook), workspace=ws))
    y_gemm, _ = _gemm_ex(p.x, p.idx, bits, d, p.codebook)
    assert np.array_equal(y_ex.view(np.uint16), y_gemm.view(np.uint16))
    ref = orc.pq_linear(p.x, p.idx, bits, d, p.codebook)
    assert_close(y_ex.astype(np.float64), ref, f"gemv_ex past the crossover {case}")
    assert_close(run("gemv", p), ref, f"gemv below the crossover {case}")


def test_decode_with_workspace_keeps_the_decode_kernel_elsewhere():
    # x whole in registers (q_proj rows at 16 tokens): no workspace
    assert fasq.gemv_ex_workspace_bytes(16, 4096, 4096, 8, 2, 256, 0) == 0
    # a codebook the GEMM would gather from global memory (Qwen3-8B down_proj
    # rows at 16 tokens), and below 12 tokens (down_proj rows at 8): the decode
    # kernel, which splits K with the workspace (8 and 4 segments)
    for (M, K, N, bits, d, C), nseg in (((16, 12288, 4096, 16, 4, 65536), 8), ((8, 14336, 4096, 8, 2, 256), 4)):
        assert fasq.plan("gemv", M, K, N, bits, d, C).startswith("k_gemv<")
        assert fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, 0) == nseg * M * N * 4


@pytest.mark.parametrize("case", [(3, 14336, 333, 2, 256, 8), (4, 14336, 1000, 2, 256, 8),
                                  (8, 14336, 4096, 2, 256, 8), (5, 14336, 130, 4, 4096, 12),
                                  (16, 12288, 700, 4, 65536, 16), (4, 12288, 4096, 4, 65536, 16),
                                  (4, 12288, 500, 4, 8192, 16), (7, 8192, 257, 1, 256, 8),
                                  (11, 14336, 500, 2, 256, 8), (12, 12288, 333, 4, 65536, 16)])
def test_decode_k_split_with_workspace(case):
    """Where x outweighs a workgroup's share of the ids, fasq_pq_gemv_ex's
    workspace lets the 16-row-tile decode kernel split K over workgroups.
    Every output is written, matches the oracle, and repeats bit for bit;
    fasq_pq_gemv (no workspace) keeps the unsplit kernel."""
    M, K, N, d, C, bits = case
    print(f"[case] decode K split {case}", flush=True)
    need = fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, 0)
    assert need > 0 and need % (M * N * 4) == 0 and 2 <= need // (M * N * 4) <= 8, need
    rng = np.random.default_rng(97 + sum(case))
    p = pi.draw_problem(rng, M, K, N, d, C, bits)
    ws = torch.full((need,), 0xFF, dtype=torch.uint8, device="cuda:0")  # NaN partials before the call
    xd, idd, cbd = to_dev(p.x), to_dev(p.idx), to_dev(p.codebook)
    y1 = to_np(fasq.pq_gemv_ex(xd, idd, bits, d, cbd, workspace=ws))
    y2 = to_np(fasq.pq_gemv_ex(xd, idd, bits, d, cbd, workspace=ws))
    assert np.isfinite(y1).all()
    assert np.array_equal(y1.view(np.uint16), y2.view(np.uint16))
    ref = orc.pq_linear(p.x, p.idx, bits, d, p.codebook)
    assert_close(y1.astype(np.float64), ref, f"gemv_ex decode K split {case}")
    assert_close(run("gemv", p), ref, f"gemv without the split {case}")
