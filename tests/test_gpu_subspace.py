"""GPU parity of the per-subspace codebook path (fasq_pq_gemv_ex) against the
oracle's Eq. lut-accumulate with one table per subspace."""

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


def draw(rng, M, K, N, d, C, bits):
    S = K // d
    books = pi.draw_codebook(rng, S * C, d).reshape(S, C, d)
    ids = pi.draw_ids(rng, N, S, C)
    x = pi.draw_x(rng, M, K)
    return x, books, ids, pi.pack_indices(ids, bits)


def reference(x, books, idx, bits, rows=None):
    S = books.shape[0]
    ids = orc.unpack_indices(idx, S, bits, books.shape[1], rows=rows)
    return orc.lut_accumulate(x, books, ids.T)


CASES = [
    # M, K, N, d, C, bits
    (1, 4096, 300, 2, 256, 8),        # 8 chunks of 16 ids per segment, 16 segments
    (1, 4096 + 128, 200, 2, 256, 8),  # last segment half empty
    (1, 1024, 100, 4, 256, 8),
    (1, 512, 64, 1, 16, 8),
    (1, 768, 70, 4, 1024, 12),
    (1, 512, 50, 8, 256, 16),
    (3, 256, 40, 2, 256, 8),          # several tokens: x slices staged in LDS
    (2, 4096, 300, 2, 256, 8),
    (4, 4096 + 128, 200, 2, 256, 8),  # several tokens, last segment half empty
    (16, 2048, 130, 2, 256, 8),       # the most tokens the tuned kernel takes
    (5, 1024, 100, 4, 256, 8),
    (3, 512, 64, 1, 16, 8),
    (7, 768, 70, 4, 1024, 12),
    (2, 512, 50, 2, 256, 16),
    (2, 512, 50, 8, 256, 16),         # several tokens at d = 8: general kernel
    (17, 256, 40, 2, 256, 8),         # more than 16 tokens: general kernel
    (1, 36, 5, 4, 9, 12),             # odd 12-bit rows: general kernel
]


@pytest.mark.parametrize("case", CASES)
def test_per_subspace_books_match_oracle(case):
    M, K, N, d, C, bits = case
    print(f"[case] gemv_ex per-subspace {case}", flush=True)
    rng = np.random.default_rng(sum(case))
    x, books, ids, idx = draw(rng, M, K, N, d, C, bits)
    y = to_np(fasq.pq_gemv_ex(to_dev(x), to_dev(idx), bits, d, to_dev(books))).astype(np.float64)
    assert_close(y, reference(x, books, idx, bits), f"per-subspace {case}")


def test_tuned_path_takes_up_to_16_tokens():
    # fp32 partials of 16 segments per token
    assert fasq.gemv_ex_workspace_bytes(1, 4096, 4096, 8, 2, 256, 512) == 16 * 4096 * 4
    assert fasq.gemv_ex_workspace_bytes(3, 4096, 4096, 8, 2, 256, 512) == 16 * 3 * 4096 * 4
    assert fasq.gemv_ex_workspace_bytes(16, 4096, 4096, 8, 2, 256, 512) == 16 * 16 * 4096 * 4
    # more tokens, or several tokens at d = 8: the general kernel, no workspace
    assert fasq.gemv_ex_workspace_bytes(17, 4096, 4096, 8, 2, 256, 512) == 0
    assert fasq.gemv_ex_workspace_bytes(2, 4096, 4096, 8, 8, 256, 2048) == 0
    assert fasq.gemv_ex_workspace_bytes(1, 4096, 4096, 8, 2, 256, 0) == 0
    assert fasq.gemv_ex_workspace_bytes(1, 4096, 4096, 8, 2, 256, 7) == -1


@pytest.mark.parametrize("case", [(1, 2048, 128, 2, 256, 8), (1, 1024, 96, 4, 4096, 12),
                                  (4, 2048, 128, 2, 256, 8), (3, 1024, 96, 4, 4096, 12), (16, 512, 64, 1, 16, 8)])
def test_per_subspace_one_hot_is_bit_exact(case):
    M, K, N, d, C, bits = case
    rng = np.random.default_rng(3 + sum(case))
    S = K // d
    books = np.stack([pi.signed_one_hot_codebook(C, d, rng) for _ in range(S)])
    ids = rng.integers(0, C, size=(N, S))
    x = pi.ternary_x(rng, M, K)
    idx = pi.pack_indices(ids, bits)
    ref = reference(x, books, idx, bits)
    assert np.abs(ref).max() <= 2048
    y = to_np(fasq.pq_gemv_ex(to_dev(x), to_dev(idx), bits, d, to_dev(books))).astype(np.float64)
    assert np.array_equal(y, ref)


def test_shared_stride_is_fasq_pq_gemv():
    rng = np.random.default_rng(5)
    p = pi.draw_problem(rng, 1, 4096, 1000, 2, 256, 8)
    a = fasq.pq_gemv(to_dev(p.x), to_dev(p.idx), 8, 2, to_dev(p.codebook))
    b = fasq.pq_gemv_ex(to_dev(p.x), to_dev(p.idx), 8, 2, to_dev(p.codebook))
    assert torch.equal(a.view(torch.int16), b.view(torch.int16))


def test_equal_books_agree_with_the_shared_codebook():
    rng = np.random.default_rng(6)
    p = pi.draw_problem(rng, 1, 2048, 500, 2, 256, 8)
    books = np.broadcast_to(p.codebook, (1024, 256, 2)).copy()
    y = to_np(fasq.pq_gemv_ex(to_dev(p.x), to_dev(p.idx), 8, 2, to_dev(books))).astype(np.float64)
    assert_close(y, orc.pq_linear(p.x, p.idx, 8, 2, p.codebook), "equal books")


def test_small_workspace_takes_the_general_kernel():
    rng = np.random.default_rng(7)
    x, books, ids, idx = draw(rng, 1, 1024, 200, 2, 256, 8)
    y = torch.empty((1, 200), dtype=torch.float16, device="cuda:0")
    ws = torch.empty(64, dtype=torch.uint8, device="cuda:0")
    xd, idd, bd = to_dev(x), to_dev(idx), to_dev(books)
    st = fasq.gemv_ex_raw(xd.data_ptr(), 1, 1024, 200, idd.data_ptr(), 8, 2, bd.data_ptr(), 256, 512, y.data_ptr(),
                          ws.data_ptr(), 64, torch.cuda.current_stream().cuda_stream)
    assert st == 0, fasq.last_error()
    assert_close(to_np(y).astype(np.float64), reference(x, books, idx, 8), "general kernel")


def test_one_workspace_serves_consecutive_calls_of_different_shapes():
    """One workspace serves calls of different shapes back to back."""
    rng = np.random.default_rng(12)
    need = max(fasq.gemv_ex_workspace_bytes(1, K, N, 8, 2, 256, 512) for K, N in ((4096, 700), (2048, 3000)))
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda:0")
    for rep in range(3):
        for K, N in ((4096, 700), (2048, 3000)):
            x, books, ids, idx = draw(rng, 1, K, N, 2, 256, 8)
            y = fasq.pq_gemv_ex(to_dev(x), to_dev(idx), 8, 2, to_dev(books), workspace=ws)
            assert_close(to_np(y).astype(np.float64), reference(x, books, idx, 8), f"reuse {rep} {K}x{N}")


def test_several_tokens_match_single_token_calls():
    """Each token of a multi-token call gives the bits of a call with that
    token alone: the same segments, added in the same order."""
    rng = np.random.default_rng(13)
    M, K, N = 6, 4096, 700
    x, books, ids, idx = draw(rng, M, K, N, 2, 256, 8)
    idd, bd = to_dev(idx), to_dev(books)
    y = fasq.pq_gemv_ex(to_dev(x), idd, 8, 2, bd)
    for m in range(M):
        ym = fasq.pq_gemv_ex(to_dev(np.ascontiguousarray(x[m:m + 1])), idd, 8, 2, bd)
        assert torch.equal(y[m:m + 1].view(torch.int16), ym.view(torch.int16)), m


def test_paper_layer_4096_2_256_sampled():
    """The paper's sensitivity layer (4096 x 4096, d = 2, K_s = 256, one
    codebook per subspace), checked on sampled rows; repeated calls are
    bit-identical."""
    rng = np.random.default_rng(8)
    x, books, ids, idx = draw(rng, 1, 4096, 4096, 2, 256, 8)
    xd, idd, bd = to_dev(x), to_dev(idx), to_dev(books)
    y1 = fasq.pq_gemv_ex(xd, idd, 8, 2, bd)
    y2 = fasq.pq_gemv_ex(xd, idd, 8, 2, bd)
    assert torch.equal(y1.view(torch.int16), y2.view(torch.int16))
    rows = sample_rows(4096, 128)
    assert_close(to_np(y1)[:, rows].astype(np.float64), reference(x, books, idx, 8, rows=rows), "paper layer")
