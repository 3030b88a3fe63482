"""fasq_pq_gemv_ex_noalloc: the entry point that allocates nothing.

Through the C ABI, its output must equal fasq_pq_gemv_ex's with a caller
workspace bit for bit (the same kernels run; only the scratch memory
differs), and lie within the oracle's tolerance, on two calls in a row, the
second with a smaller input (the scratch keeps the first call's contents).
Sizes whose scratch exceeds the library's array are rejected before any
launch.
"""

import numpy as np
import pytest

import pq_inputs as pi
from oracle import pq_oracle as orc
from gpu_util import assert_close, to_dev, to_np

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


def _draw(rng, M, K, N, d, C, bits, per_subspace):
    S = K // d
    if per_subspace:
        books = pi.draw_codebook(rng, S * C, d).reshape(S, C, d)
    else:
        books = pi.draw_codebook(rng, C, d)
    ids = pi.draw_ids(rng, N, S, C)
    return pi.draw_x(rng, M, K), books, pi.pack_indices(ids, bits)


def _reference(x, books, idx, bits, d, per_subspace):
    if per_subspace:
        S = books.shape[0]
        return orc.lut_accumulate(x, books, orc.unpack_indices(idx, S, bits, books.shape[1]).T)
    return orc.pq_linear(x, idx, bits, d, books)


def _run_both(x, books, idx, M, K, N, d, C, bits, per_subspace):
    """y of fasq_pq_gemv_ex_noalloc and of fasq_pq_gemv_ex (with a workspace
    of the size it asks for), through the C ABI on one stream."""
    stride = C * d if per_subspace else 0
    need = fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, stride)
    assert 0 <= need <= fasq.noalloc_scratch_bytes()
    xd, idd, bd = to_dev(x), to_dev(idx), to_dev(books)
    y_na = torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda:0")
    y_ex = torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda:0")
    ws = torch.empty(max(need, 4), dtype=torch.uint8, device="cuda:0")
    stream = torch.cuda.current_stream().cuda_stream
    st = fasq.gemv_ex_noalloc_raw(xd.data_ptr(), M, K, N, idd.data_ptr(), bits, d, bd.data_ptr(), C, stride,
                                  y_na.data_ptr(), stream)
    assert st == fasq.FASQ_OK, fasq.last_error()
    st = fasq.gemv_ex_raw(xd.data_ptr(), M, K, N, idd.data_ptr(), bits, d, bd.data_ptr(), C, stride,
                          y_ex.data_ptr(), ws.data_ptr(), need, stream)
    assert st == fasq.FASQ_OK, fasq.last_error()
    return to_np(y_na), to_np(y_ex), need


# (label, per-subspace books, first call (M, K, N, d, C, bits), second, smaller call)
CASES = [
    ("per-subspace books, K split over workgroups", True,
     (1, 4096, 4096, 2, 256, 8), (1, 1024, 300, 2, 256, 8)),
    ("per-subspace books, several tokens", True,
     (8, 2048, 1000, 2, 256, 8), (3, 1024, 300, 2, 256, 8)),
    ("shared codebook, GEMM fallback with K split", False,
     (20, 2048, 300, 4, 256, 8), (17, 1024, 100, 4, 256, 8)),
    ("shared codebook, decode kernel splitting K", False,
     (8, 14336, 700, 2, 256, 8), (4, 14336, 300, 2, 256, 8)),
    ("shared codebook, decode kernel (no scratch)", False,
     (1, 4096, 1024, 2, 256, 8), (1, 512, 64, 2, 256, 8)),
]


@pytest.mark.parametrize("case", CASES, ids=[c[0] for c in CASES])
def test_noalloc_matches_workspace_call_twice(case):
    label, per_subspace, first, second = case
    rng = np.random.default_rng(61)
    for call, (M, K, N, d, C, bits) in enumerate((first, second)):
        print(f"[case] noalloc {label} call {call}: {(M, K, N, d, C, bits)}", flush=True)
        x, books, idx = _draw(rng, M, K, N, d, C, bits, per_subspace)
        y_na, y_ex, need = _run_both(x, books, idx, M, K, N, d, C, bits, per_subspace)
        if "no scratch" not in label:
            assert need > 0, label
        assert np.isfinite(y_na).all()
        assert np.array_equal(y_na.view(np.uint16), y_ex.view(np.uint16)), (label, call)
        assert_close(y_na.astype(np.float64), _reference(x, books, idx, bits, d, per_subspace),
                     f"noalloc {label} call {call}")


def test_noalloc_rejects_scratch_beyond_the_array():
    """Per-subspace books on 270000 rows need 16 segments x 270000 x 4 bytes of
    partials, more than the array holds: rejected, nothing launched (y keeps
    its NaNs)."""
    M, K, N, d, C, bits = 1, 4096, 270000, 2, 256, 8
    stride = C * d
    need = fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, stride)
    assert need > fasq.noalloc_scratch_bytes()
    x = torch.zeros((M, K), dtype=torch.float16, device="cuda:0")
    idx = torch.zeros((N, fasq.idx_row_bytes(K, d, bits)), dtype=torch.uint8, device="cuda:0")
    books = torch.zeros((K // d, C, d), dtype=torch.float16, device="cuda:0")
    y = torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda:0")
    st = fasq.gemv_ex_noalloc_raw(x.data_ptr(), M, K, N, idx.data_ptr(), bits, d, books.data_ptr(), C, stride,
                                  y.data_ptr(), torch.cuda.current_stream().cuda_stream)
    assert st == fasq.FASQ_ERR_INVALID_ARG
    msg = fasq.last_error()
    assert str(need) in msg and str(fasq.noalloc_scratch_bytes()) in msg
    torch.cuda.synchronize()
    assert torch.isnan(y).all()


def test_noalloc_argument_checks_launch_nothing():
    x = torch.zeros((1, 64), dtype=torch.float16, device="cuda:0")
    idx = torch.zeros((4, 32), dtype=torch.uint8, device="cuda:0")
    cb = torch.zeros((256, 2), dtype=torch.float16, device="cuda:0")
    y = torch.full((1, 4), float("nan"), dtype=torch.float16, device="cuda:0")
    # K not a multiple of d, a NULL pointer, a codebook stride that is neither 0 nor C * d
    assert fasq.gemv_ex_noalloc_raw(x.data_ptr(), 1, 63, 4, idx.data_ptr(), 8, 2, cb.data_ptr(), 256, 0,
                                    y.data_ptr(), 0) == fasq.FASQ_ERR_INVALID_ARG
    assert fasq.gemv_ex_noalloc_raw(x.data_ptr(), 1, 64, 4, 0, 8, 2, cb.data_ptr(), 256, 0,
                                    y.data_ptr(), 0) == fasq.FASQ_ERR_INVALID_ARG
    assert fasq.gemv_ex_noalloc_raw(x.data_ptr(), 1, 64, 4, idx.data_ptr(), 8, 2, cb.data_ptr(), 256, 3,
                                    y.data_ptr(), 0) == fasq.FASQ_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert torch.isnan(y).all()
