"""Launch lists (fasq_launch_list_*): record the launches of a sequence of
calls, queue them again later.

Through the C ABI: recording launches nothing; a run writes, bit for bit,
what the same calls made directly write (decode kernels one-token, grouped
and 16-row-tile, the prefill GEMM with its K-split reduction, the
per-subspace decode with its reduction, the no-allocation entry point, the
reconstruction), and within the oracle's tolerance; a later run reads the
inputs as they are then; a run on another stream works; misuse is rejected.
"""

import ctypes

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


def _nan(M, N):
    return torch.full((M, N), float("nan"), dtype=torch.float16, device="cuda:0")


class _Case:
    """One call with its inputs, one set of outputs for direct calls and one
    for the list (``outs[k]`` is a list of tensors), and the oracle results."""

    def __init__(self, name, call, outs, refs):
        self.name, self.call, self.outs, self.refs = name, call, outs, refs


def _one(name, call, M, N, ref):
    return _Case(name, lambda ys, s: call(ys[0], s), [[_nan(M, N)], [_nan(M, N)]], [ref])


def _cases(seed=0):
    rng = np.random.default_rng(seed)
    cases = []

    # one token, shared codebook: the row-streaming kernel (ragged N)
    M, K, N, d, C, bits = 1, 1024, 3000, 2, 256, 8
    x, cb = pi.draw_x(rng, M, K), pi.draw_codebook(rng, C, d)
    idx = pi.pack_indices(pi.draw_ids(rng, N, K // d, C), bits)
    xd, cbd, idd = to_dev(x), to_dev(cb), to_dev(idx)
    cases.append(_one("gemv M=1", lambda y, s: fasq.gemv_raw(
        xd.data_ptr(), 1, 1024, 3000, idd.data_ptr(), 8, 2, cbd.data_ptr(), 256, y.data_ptr(), s),
        M, N, orc.pq_linear(x, idx, bits, d, cb)))
    first = (x, xd, idx, cb, M, K, N, d, C, bits)

    # three matrices sharing x: one grouped launch
    Ns = [1000, 256, 256]
    x2 = pi.draw_x(rng, 1, 1024)
    books = [pi.draw_codebook(rng, 256, 2) for _ in Ns]
    idxs = [pi.pack_indices(pi.draw_ids(rng, n, 512, 256), 8) for n in Ns]
    x2d, bd, ixd = to_dev(x2), [to_dev(b) for b in books], [to_dev(i) for i in idxs]
    cases.append(_Case("batched", lambda ys, s: fasq.gemv_batched_raw(
        x2d.data_ptr(), 1, 1024, [t.data_ptr() for t in ixd], Ns, [t.data_ptr() for t in bd], [256] * 3,
        [t.data_ptr() for t in ys], 8, 2, s), [[_nan(1, n) for n in Ns], [_nan(1, n) for n in Ns]],
        [orc.pq_linear(x2, i, 8, 2, b) for i, b in zip(idxs, books)]))

    # four tokens, 12-bit ids, a 4096-entry codebook: the 16-row-tile kernel
    M, K, N, d, C, bits = 4, 1024, 700, 4, 4096, 12
    x3, cb3 = pi.draw_x(rng, M, K), pi.draw_codebook(rng, C, d)
    idx3 = pi.pack_indices(pi.draw_ids(rng, N, K // d, C), bits)
    a3 = (to_dev(x3), to_dev(idx3), to_dev(cb3))
    cases.append(_one("gemv M=4", lambda y, s, a=a3: fasq.gemv_raw(
        a[0].data_ptr(), 4, 1024, 700, a[1].data_ptr(), 12, 4, a[2].data_ptr(), 4096, y.data_ptr(), s),
        M, N, orc.pq_linear(x3, idx3, bits, d, cb3)))

    # prefill GEMM with a workspace: K split, then the reduction kernel
    M, K, N, d, C, bits = 128, 4096, 1024, 4, 256, 8
    x4, cb4 = pi.draw_x(rng, M, K), pi.draw_codebook(rng, C, d)
    idx4 = pi.pack_indices(pi.draw_ids(rng, N, K // d, C), bits)
    a4 = (to_dev(x4), to_dev(idx4), to_dev(cb4))
    need = fasq.gemm_ex_workspace_bytes(M, K, N, bits, d, C)
    assert need > 0, "this shape is meant to split K"
    ws4 = torch.empty(need, dtype=torch.uint8, device="cuda:0")
    cases.append(_one("gemm_ex K split", lambda y, s, a=a4: fasq.gemm_ex_raw(
        a[0].data_ptr(), 128, 4096, 1024, a[1].data_ptr(), 8, 4, a[2].data_ptr(), 256, y.data_ptr(),
        ws4.data_ptr(), need, s), M, N, orc.pq_linear(x4, idx4, bits, d, cb4)))

    # per-subspace codebooks: the K-split decode kernel and its reduction
    M, K, N, d, C, bits = 1, 512, 700, 2, 64, 8
    S = K // d
    x5, books5 = pi.draw_x(rng, M, K), pi.draw_codebook(rng, S * C, d).reshape(S, C, d)
    ids5 = pi.draw_ids(rng, N, S, C)
    idx5 = pi.pack_indices(ids5, bits)
    a5 = (to_dev(x5), to_dev(idx5), to_dev(books5))
    need5 = fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, C * d)
    assert need5 > 0
    ws5 = torch.empty(need5, dtype=torch.uint8, device="cuda:0")
    cases.append(_one("gemv_ex per-subspace", lambda y, s, a=a5: fasq.gemv_ex_raw(
        a[0].data_ptr(), 1, 512, 700, a[1].data_ptr(), 8, 2, a[2].data_ptr(), 64, 128, y.data_ptr(),
        ws5.data_ptr(), need5, s), M, N, orc.lut_accumulate(x5, books5, ids5.T)))

    # the entry point that allocates nothing (two tokens)
    M, K, N, d, C, bits = 2, 1024, 500, 2, 256, 8
    x6, cb6 = pi.draw_x(rng, M, K), pi.draw_codebook(rng, C, d)
    idx6 = pi.pack_indices(pi.draw_ids(rng, N, K // d, C), bits)
    a6 = (to_dev(x6), to_dev(idx6), to_dev(cb6))
    cases.append(_one("gemv_ex_noalloc M=2", lambda y, s, a=a6: fasq.gemv_ex_noalloc_raw(
        a[0].data_ptr(), 2, 1024, 500, a[1].data_ptr(), 8, 2, a[2].data_ptr(), 256, 0, y.data_ptr(), s),
        M, N, orc.pq_linear(x6, idx6, bits, d, cb6)))

    # the reconstruction (every element a codebook entry)
    N7, K7, d7, C7 = 100, 256, 4, 256
    cb7 = pi.draw_codebook(rng, C7, d7)
    idx7 = pi.pack_indices(pi.draw_ids(rng, N7, K7 // d7, C7), 8)
    a7 = (to_dev(idx7), to_dev(cb7))
    cases.append(_one("reconstruct", lambda y, s, a=a7: fasq.reconstruct_raw(
        a[0].data_ptr(), 100, 256, 8, 4, a[1].data_ptr(), 256, y.data_ptr(), s),
        N7, K7, orc.reconstruct(idx7, K7, 8, d7, cb7)))
    return cases, first


def _bits(t):
    return to_np(t).view(np.uint16)


def test_recorded_launches_reproduce_the_calls():
    cases, first = _cases()
    stream = torch.cuda.current_stream().cuda_stream
    for c in cases:
        assert c.call(c.outs[0], stream) == fasq.FASQ_OK, (c.name, fasq.last_error())
    torch.cuda.synchronize()
    lst = fasq.LaunchList()
    with lst:
        for c in cases:
            assert c.call(c.outs[1], stream) == fasq.FASQ_OK, (c.name, fasq.last_error())
    torch.cuda.synchronize()
    print(f"[launch list] {len(lst)} launches recorded for {len(cases)} calls", flush=True)
    # one launch per call, plus the reductions of the two K splits
    assert len(lst) == len(cases) + 2
    for c in cases:  # recording queued nothing
        for t in c.outs[1]:
            assert np.isnan(to_np(t).astype(np.float32)).all(), c.name
    lst.run(stream)
    torch.cuda.synchronize()
    for c in cases:
        for j, (t_list, t_direct, ref) in enumerate(zip(c.outs[1], c.outs[0], c.refs)):
            assert np.array_equal(_bits(t_list), _bits(t_direct)), (c.name, j)
            if c.name == "reconstruct":
                assert np.array_equal(_bits(t_list), ref.view(np.uint16)), c.name
            else:
                assert_close(to_np(t_list), ref, f"launch list {c.name} {j}")

    # a later run reads the inputs as they are then, on any stream
    x, xd, idx, cb, M, K, N, d, C, bits = first
    x_new = pi.draw_x(np.random.default_rng(7), M, K)
    xd.copy_(torch.from_numpy(x_new).to(xd.device))
    side = torch.cuda.Stream()
    side.wait_stream(torch.cuda.current_stream())
    lst.run(side)
    side.synchronize()
    y_direct = [_nan(M, N)]
    assert cases[0].call(y_direct, stream) == fasq.FASQ_OK
    torch.cuda.synchronize()
    assert np.array_equal(_bits(cases[0].outs[1][0]), _bits(y_direct[0]))
    assert_close(to_np(cases[0].outs[1][0]), orc.pq_linear(x_new, idx, bits, d, cb), "launch list rerun")
    lst.close()


def test_recording_rejects_misuse():
    L = fasq.lib()
    rng = np.random.default_rng(3)
    M, K, N, d, C, bits = 1, 256, 64, 2, 16, 8
    xd = to_dev(pi.draw_x(rng, M, K))
    cbd = to_dev(pi.draw_codebook(rng, C, d))
    idd = to_dev(pi.pack_indices(pi.draw_ids(rng, N, K // d, C), bits))
    y = _nan(M, N)
    lst, other = fasq.LaunchList(), fasq.LaunchList()
    h, ho = ctypes.c_void_p(lst.handle), ctypes.c_void_p(other.handle)
    stream = torch.cuda.current_stream().cuda_stream
    assert L.fasq_launch_list_begin(h) == fasq.FASQ_OK
    try:
        # a second begin on this thread, for this or another list
        assert L.fasq_launch_list_begin(h) == fasq.FASQ_ERR_INVALID_ARG
        assert L.fasq_launch_list_begin(ho) == fasq.FASQ_ERR_INVALID_ARG
        # no run while recording
        assert L.fasq_launch_list_run(h, stream) == fasq.FASQ_ERR_INVALID_ARG
        assert L.fasq_launch_list_run(ho, stream) == fasq.FASQ_ERR_INVALID_ARG
        # an invalid call records nothing
        assert fasq.gemv_raw(xd.data_ptr(), M, K, N, idd.data_ptr(), 10, d, cbd.data_ptr(), C, y.data_ptr(),
                             stream) == fasq.FASQ_ERR_INVALID_ARG
        assert len(lst) == 0
        assert fasq.gemv_raw(xd.data_ptr(), M, K, N, idd.data_ptr(), bits, d, cbd.data_ptr(), C, y.data_ptr(),
                             stream) == fasq.FASQ_OK
        assert len(lst) == 1
        assert L.fasq_launch_list_end(ho) == fasq.FASQ_ERR_INVALID_ARG
    finally:
        assert L.fasq_launch_list_end(h) == fasq.FASQ_OK
    assert L.fasq_launch_list_end(h) == fasq.FASQ_ERR_INVALID_ARG
    torch.cuda.synchronize()
    assert np.isnan(to_np(y).astype(np.float32)).all()
    # a list extends over several recordings
    with lst:
        assert fasq.gemv_raw(xd.data_ptr(), M, K, N, idd.data_ptr(), bits, d, cbd.data_ptr(), C, y.data_ptr(),
                             stream) == fasq.FASQ_OK
    assert len(lst) == 2
    lst.run(stream)
    # an empty list runs and queues nothing
    other.run(stream)
    torch.cuda.synchronize()
    ref = orc.pq_linear(to_np(xd), to_np(idd), bits, d, to_np(cbd))
    assert_close(to_np(y), ref, "launch list, two recordings")
    lst.close()
    other.close()
