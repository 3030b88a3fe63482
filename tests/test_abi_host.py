"""Host-side checks of the C ABI: the library loads, exports every declared
symbol, and rejects bad arguments before touching the GPU."""

import ctypes
import os
import re

import pytest

import paper_2605_04084_amd as fasq
from conftest import ROOT

HEADER = os.path.join(ROOT, "include", "fasq.h")


@pytest.fixture(scope="module")
def L():
    if not os.path.exists(fasq.LIB_PATH):
        from paper_2605_04084_amd import _build

        _build.build()
    return fasq.lib()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(fasq_[a-z0-9_]+)\s*\(", text)))


def test_header_declares_the_binding_symbols():
    assert declared_functions() == sorted(fasq.EXPORTED_SYMBOLS)


def test_every_declared_symbol_is_exported(L):
    for name in declared_functions():
        assert hasattr(L, name), name
        assert ctypes.cast(getattr(L, name), ctypes.c_void_p).value


def test_abi_version(L):
    assert fasq.abi_version() == fasq.ABI_VERSION
    m = re.search(r"#define FASQ_ABI_VERSION (\d+)", open(HEADER).read())
    assert int(m.group(1)) == fasq.ABI_VERSION


def test_status_strings(L):
    assert fasq.status_string(0) == "FASQ_OK"
    assert fasq.status_string(1) == "FASQ_ERR_INVALID_ARG"
    assert fasq.status_string(2) == "FASQ_ERR_UNSUPPORTED"
    assert fasq.status_string(3) == "FASQ_ERR_HIP"
    assert fasq.status_string(4) == "FASQ_ERR_HOST_MEMORY"
    assert fasq.status_string(99) == "FASQ_UNKNOWN_STATUS"


@pytest.mark.parametrize("K,d,bits,R", [(4096, 2, 8, 2048), (4096, 4, 12, 1536), (4096, 4, 16, 2048),
                                        (14336, 2, 8, 7168), (12, 4, 12, 5), (256, 4, 8, 64), (7, 7, 8, 1),
                                        (10, 3, 8, -1), (0, 1, 8, -1), (8, 0, 8, -1), (8, 2, 10, -1)])
def test_idx_row_bytes(L, K, d, bits, R):
    assert fasq.idx_row_bytes(K, d, bits) == R


DUMMY = 0x1000  # never dereferenced: validation fails first


@pytest.mark.parametrize("entry", ["gemv", "gemm"])
@pytest.mark.parametrize("args,why", [
    (dict(M=0), "M, K and N"),
    (dict(K=0), "M, K and N"),
    (dict(N=-1), "M, K and N"),
    (dict(d=0), "d must"),
    (dict(K=10, d=4), "multiple of d"),
    (dict(idx_bits=10), "idx_bits"),
    (dict(C=0), "C must"),
    (dict(C=257), "C must"),
    (dict(idx_bits=12, C=4097), "C must"),
    (dict(x=0), "NULL"),
    (dict(idx=0), "NULL"),
    (dict(codebook=0), "NULL"),
    (dict(y=0), "NULL"),
])
def test_invalid_arguments_rejected_without_launch(L, entry, args, why):
    a = dict(x=DUMMY, M=1, K=16, N=4, idx=DUMMY, idx_bits=8, d=2, codebook=DUMMY, C=256, y=DUMMY)
    a.update(args)
    fn = fasq.gemv_raw if entry == "gemv" else fasq.gemm_raw
    st = fn(a["x"], a["M"], a["K"], a["N"], a["idx"], a["idx_bits"], a["d"], a["codebook"], a["C"], a["y"], 0)
    assert st == fasq.FASQ_ERR_INVALID_ARG
    assert why in fasq.last_error()


def test_reconstruct_validation(L):
    st = fasq.reconstruct_raw(DUMMY, 4, 10, 8, 4, DUMMY, 16, DUMMY, 0)
    assert st == fasq.FASQ_ERR_INVALID_ARG
    st = fasq.reconstruct_raw(0, 4, 8, 8, 4, DUMMY, 16, DUMMY, 0)
    assert st == fasq.FASQ_ERR_INVALID_ARG
    st = fasq.reconstruct_raw(DUMMY, 4, 8, 16, 4, DUMMY, 70000, DUMMY, 0)
    assert st == fasq.FASQ_ERR_INVALID_ARG


def test_python_binding_rejects_host_tensors(L):
    torch = pytest.importorskip("torch")
    x = torch.zeros((1, 16), dtype=torch.float16)
    idx = torch.zeros((4, 8), dtype=torch.uint8)
    cb = torch.zeros((256, 2), dtype=torch.float16)
    with pytest.raises(ValueError):
        fasq.pq_gemv(x, idx, 8, 2, cb)


def test_binding_has_no_cpu_compute_path():
    """The binding module must not import or reference the oracle."""
    src = open(os.path.join(ROOT, "paper_2605_04084_amd", "__init__.py")).read()
    assert "oracle" not in src.replace("Oracle", "")
    for f in os.listdir(os.path.join(ROOT, "paper_2605_04084_amd", "csrc")):
        text = open(os.path.join(ROOT, "paper_2605_04084_amd", "csrc", f)).read()
        assert "oracle" not in text.lower(), f


def _batched(**kw):
    a = dict(x=DUMMY, M=1, K=16, idx=[DUMMY, DUMMY], N=[4, 8], codebook=[DUMMY, DUMMY], C=[256, 16],
             y=[DUMMY + 64, DUMMY + 128], idx_bits=8, d=2)
    a.update(kw)
    return fasq.gemv_batched_raw(a["x"], a["M"], a["K"], a["idx"], a["N"], a["codebook"], a["C"], a["y"],
                                 a["idx_bits"], a["d"], 0)


@pytest.mark.parametrize("args,why", [
    (dict(idx=[], N=[], codebook=[], C=[], y=[]), "count"),
    (dict(N=[4, 0]), "matrix 1: M, K and N"),
    (dict(C=[256, 257]), "matrix 1: C must"),
    (dict(idx=[0, DUMMY]), "matrix 0: a buffer pointer is NULL"),
    (dict(y=[DUMMY, 0]), "matrix 1: a buffer pointer is NULL"),
    (dict(x=0), "matrix 0: a buffer pointer is NULL"),
    (dict(K=10, d=4), "matrix 0: K must be a multiple of d"),
])
def test_batched_invalid_arguments_rejected_without_launch(L, args, why):
    assert _batched(**args) == fasq.FASQ_ERR_INVALID_ARG
    assert why in fasq.last_error()


def test_batched_null_arrays_rejected(L):
    st = L.fasq_pq_gemv_batched(DUMMY, 1, 16, 2, None, None, None, None, None, 8, 2, None)
    assert st == fasq.FASQ_ERR_INVALID_ARG
    assert "array is NULL" in fasq.last_error()


def test_batched_binding_checks_lengths(L):
    with pytest.raises(ValueError):
        fasq.gemv_batched_raw(DUMMY, 1, 16, [DUMMY], [4, 4], [DUMMY], [16], [DUMMY], 8, 2)


# ---------------------------------------------------------------------------
# Encoder entry points: validation before any HIP call
# ---------------------------------------------------------------------------

def test_encode_workspace_bytes(L):
    # [C x d] int64 sums and [C] int64 counts (256-byte aligned), then one uint32 id per sub-vector
    assert fasq.encode_workspace_bytes(4, 16, 2, 256) == 256 * 3 * 8 + 4 * 8 * 4
    assert fasq.encode_workspace_bytes(4, 16, 3, 4) == -1
    assert fasq.encode_workspace_bytes(0, 16, 2, 4) == -1
    assert fasq.encode_workspace_bytes(4, 16, 2, 70000) == -1


@pytest.mark.parametrize("args,why,status", [
    (dict(N=0), "N and K", 1),
    (dict(d=0), "d must", 1),
    (dict(K=10, d=4), "multiple of d", 1),
    (dict(idx_bits=9), "idx_bits", 1),
    (dict(C=257), "C must", 1),
    (dict(iters=-1), "iters", 1),
    (dict(w=0), "NULL", 1),
    (dict(init=0), "NULL", 1),
    (dict(cb=0), "NULL", 1),
    (dict(idx=0), "NULL", 1),
    (dict(ws=0), "NULL", 1),
    (dict(w=DUMMY + 1), "aligned", 1),
    (dict(ws=DUMMY + 4), "aligned", 1),
    (dict(ws_bytes=16), "workspace smaller", 1),
    (dict(K=34, d=17, ws_bytes=1 << 20), "d <= 16", 2),
])
def test_encode_invalid_arguments_rejected_without_launch(L, args, why, status):
    a = dict(w=DUMMY, N=4, K=16, d=2, C=256, idx_bits=8, init=DUMMY, iters=2, cb=DUMMY, idx=DUMMY, ws=DUMMY,
             ws_bytes=1 << 20)
    a.update(args)
    st = fasq.encode_raw(a["w"], a["N"], a["K"], a["d"], a["C"], a["idx_bits"], a["init"], a["iters"], a["cb"],
                         a["idx"], a["ws"], a["ws_bytes"], 0)
    assert st == status
    assert why in fasq.last_error()


# ---------------------------------------------------------------------------
# Prefill with a workspace (K split over workgroups): validation before any
# HIP call
# ---------------------------------------------------------------------------

@pytest.mark.parametrize("args,why", [
    (dict(M=0), "M, K and N"),
    (dict(K=10, d=4), "multiple of d"),
    (dict(idx_bits=10), "idx_bits"),
    (dict(C=257), "C must"),
    (dict(y=0), "NULL"),
    (dict(ws_bytes=-1), "workspace_bytes"),
])
def test_gemm_ex_invalid_arguments_rejected_without_launch(L, args, why):
    a = dict(x=DUMMY, M=1, K=16, N=4, idx=DUMMY, idx_bits=8, d=2, codebook=DUMMY, C=256, y=DUMMY, ws=DUMMY,
             ws_bytes=1 << 20)
    a.update(args)
    st = fasq.gemm_ex_raw(a["x"], a["M"], a["K"], a["N"], a["idx"], a["idx_bits"], a["d"], a["codebook"], a["C"],
                          a["y"], a["ws"], a["ws_bytes"], 0)
    assert st == fasq.FASQ_ERR_INVALID_ARG
    assert why in fasq.last_error()


def test_gemm_ex_workspace_bytes_invalid_sizes(L):
    assert fasq.gemm_ex_workspace_bytes(0, 16, 4, 8, 2, 256) == -1
    assert fasq.gemm_ex_workspace_bytes(1, 10, 4, 8, 4, 256) == -1
    assert fasq.gemm_ex_workspace_bytes(1, 16, 4, 8, 2, 300) == -1


def test_launch_list_host_paths(L):
    """Launch lists: creation, size, misuse and the empty run need no GPU."""
    h = ctypes.c_void_p()
    assert L.fasq_launch_list_create(ctypes.byref(h)) == fasq.FASQ_OK and h.value
    try:
        assert L.fasq_launch_list_size(h) == 0
        assert L.fasq_launch_list_end(h) == fasq.FASQ_ERR_INVALID_ARG  # not recording
        assert "not recording" in fasq.last_error()
        assert L.fasq_launch_list_run(h, None) == fasq.FASQ_OK  # empty: queues nothing
        st = L.fasq_launch_list_begin(h)
        if st == fasq.FASQ_OK:  # a GPU is present: recording started, end it
            assert L.fasq_launch_list_end(h) == fasq.FASQ_OK
        else:
            assert st == fasq.FASQ_ERR_HIP and "device" in fasq.last_error()
        assert L.fasq_launch_list_size(h) == 0
    finally:
        L.fasq_launch_list_destroy(h)
    assert L.fasq_launch_list_create(None) == fasq.FASQ_ERR_INVALID_ARG
    assert L.fasq_launch_list_begin(None) == fasq.FASQ_ERR_INVALID_ARG
    assert L.fasq_launch_list_end(None) == fasq.FASQ_ERR_INVALID_ARG
    assert L.fasq_launch_list_run(None, None) == fasq.FASQ_ERR_INVALID_ARG
    assert L.fasq_launch_list_size(None) == -1
    L.fasq_launch_list_destroy(None)
    lst = fasq.LaunchList()
    assert len(lst) == 0 and lst.handle
    lst.close()
    assert lst.handle == 0
    with pytest.raises(ValueError):
        len(lst)
