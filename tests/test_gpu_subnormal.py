"""fp16 subnormals and signed zeros through every kernel that computes y.

The codebooks of the paper are fp16 (Sec. 3.2) and nothing in the method
flushes small values, so a codeword or an activation that is an fp16
subnormal must reach the fp32 accumulator unchanged.  These tests make that
exact and checkable bit for bit:

* codebook kind: every codeword is +-k * 2**-24 (k in {0, 1, 2, 3}, with +0
  and -0; the "wide" variant also has k = 512 and 1023, the largest
  subnormal), and x is ternary;
* activation kind: every x is +-k * 2**-24 and the codebook is signed
  one-hot (codewords in {0, +-1}).

Every product is then an integer multiple of 2**-24, and so is every partial
sum, of magnitude below 2**24 units: fp32 holds each one exactly, in any
summation order.  The kernel's single fp16 rounding of that exact sum must
therefore equal the round-to-nearest-even of the oracle's fp64 value, bit for
bit (a zero's sign depends on the summation order, so zeros compare by
value).  In the narrow kinds every |y| is at most 2047 * 2**-24, which fp16
represents exactly, and many outputs are themselves subnormal, so the fp16
store of a subnormal result is covered too.  A kernel that flushed subnormal
inputs would return zeros.

Each case first checks with fasq_pq_plan (or the workspace query) that the
call takes the kernel and codebook placement it is listed under.
"""

import numpy as np
import pytest

import pq_inputs as pi
from oracle import pq_oracle as orc
from gpu_util import to_dev, to_np

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
fasq = pytest.importorskip("paper_2605_04084_amd")

UNIT = pi.FP16_SUBNORMAL_UNIT


@pytest.fixture(scope="module", autouse=True)
def _gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    fasq.lib()
    yield
    torch.cuda.synchronize()


def parse_plan(name):
    """("k_gemv_m1", [8, 2, 2, 0, 0]) from "k_gemv_m1<8, 2, 2, 0, 0>"."""
    assert name, "no kernel planned"
    base, rest = name.split("<", 1)
    return base, [int(v) for v in rest.rstrip(">").split(",")]


def draw(kind, M, K, N, d, C, seed):
    """x, codebook and ids of one case of the given kind."""
    rng = np.random.default_rng(seed)
    if kind == "x":
        x = pi.subnormal_x(rng, M, K, large_frac=0.05)
        cb = pi.signed_one_hot_codebook(C, d, rng)
    else:
        x = pi.ternary_x(rng, M, K)
        cb = pi.subnormal_codebook(rng, C, d, large_frac=0.05 if kind == "wide" else 0.0)
    ids = rng.integers(0, C, size=(N, K // d))
    return x, cb, ids


def check_exact(y_gpu, y_ref, kind, label):
    """y_gpu (fp16) against the oracle's exact fp64 value, rounded once."""
    y_ref = np.asarray(y_ref, dtype=np.float64)
    units = np.abs(y_ref) / UNIT
    # the precondition that makes every partial sum exact in fp32
    assert np.all(units == np.round(units)) and units.max() < 2 ** 24, label
    nz = np.count_nonzero(y_ref)
    assert nz >= 0.5 * y_ref.size, f"{label}: the case is nearly all zeros"
    if kind == "codebook":
        assert units.max() <= 2047, label          # fp16 holds every y exactly
        assert np.count_nonzero((units > 0) & (units < 1024)) > 0, label  # subnormal outputs
    expect = y_ref.astype(np.float16).astype(np.float64)
    got = np.asarray(y_gpu).astype(np.float64)
    bad = np.flatnonzero(got.ravel() != expect.ravel())
    print(f"[subnormal] {label}: {y_ref.size} outputs, max |y| = {units.max():.0f} units, "
          f"{bad.size} mismatches", flush=True)
    assert bad.size == 0, (label, bad[:8], got.ravel()[bad[:8]], expect.ravel()[bad[:8]])


KINDS = ["codebook", "wide", "x"]

# fasq_pq_gemv paths: (kernel, codebook placement or None, (M, K, N, d, C, bits)).
# Placements: 0 replicated in LDS, 1 one LDS copy, 2 global memory,
# 3 LDS slices (one pass per slice), 4 head in LDS and the rest global.
GEMV_PATHS = [
    ("k_gemv_m1", 0, (1, 4096, 1000, 2, 256, 8)),
    ("k_gemv_m1", 1, (1, 4096, 100, 4, 4096, 12)),
    ("k_gemv_m1", 2, (1, 512, 64, 2, 250, 8)),
    ("k_gemv_m1", 3, (1, 2048, 100, 2, 65536, 16)),
    ("k_gemv_m1", 0, (1, 4096 + 512, 600, 2, 256, 8)),   # masked chunk tail
    ("k_gemv_mt", None, (2, 4096, 1000, 2, 256, 8)),
    ("k_gemv_mt", 0, (2, 4096, 16500, 2, 256, 8)),        # many rows per CU: two loads per row part, x in registers
    ("k_gemv_mt", 1, (2, 1536, 260, 4, 4096, 12)),
    ("k_gemv", 0, (4, 4096, 500, 2, 256, 8)),
    ("k_gemv", 1, (8, 1024, 200, 4, 4096, 12)),
    ("k_gemv", 2, (4, 512, 64, 2, 250, 8)),
    ("k_gemv", 3, (2, 2048, 100, 1, 65536, 16)),
    ("k_gemv", 4, (4, 4096, 300, 4, 65536, 16)),
    ("k_gemv", 1, (16, 4096 + 64, 300, 2, 256, 8)),       # x staged in LDS, masked tail
]


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("path", GEMV_PATHS, ids=lambda p: f"{p[0]}-mode{p[1]}-{p[2]}")
def test_gemv_paths(path, kind):
    kernel, mode, (M, K, N, d, C, bits) = path
    label = f"gemv {kernel} mode {mode} {path[2]} {kind}"
    print(f"[case] {label}", flush=True)
    base, params = parse_plan(fasq.plan("gemv", M, K, N, bits, d, C))
    assert base == kernel, (label, base)
    if mode is not None:
        assert params[3] == mode, (label, params)
    x, cb, ids = draw(kind, M, K, N, d, C, seed=M * 7 + K + N + C)
    idx = pi.pack_indices(ids, bits)
    y = to_np(fasq.pq_gemv(to_dev(x), to_dev(idx), bits, d, to_dev(cb)))
    check_exact(y, orc.pq_linear(x, idx, bits, d, cb), kind, label)


# fasq_pq_gemm tiles: (rows, columns) of the output tile, (M, K, N, d, C, bits)
GEMM_PATHS = [
    ((256, 256), (777, 448, 12345, 4, 256, 8)),   # half-row codebook
    ((256, 256), (600, 256, 16400, 4, 4096, 12)),  # one codebook copy
    ((128, 256), (1030, 256, 16400, 2, 256, 8)),
    ((128, 128), (1000, 256, 3000, 4, 256, 8)),
    ((64, 128), (500, 256, 3000, 4, 256, 8)),
    ((64, 64), (40, 320, 100, 4, 256, 8)),
    ((64, 128), (130, 256, 257, 4, 4096, 12)),   # 12-bit ids: the 64 x 64 tile cannot split its id copies evenly
    ((64, 64), (100, 1088, 70, 4, 65536, 16)),
]


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("path", GEMM_PATHS, ids=lambda p: f"{p[0][0]}x{p[0][1]}-{p[1]}")
def test_gemm_tiles(path, kind):
    tile, (M, K, N, d, C, bits) = path
    label = f"gemm tile {tile} {path[1]} {kind}"
    print(f"[case] {label}", flush=True)
    base, params = parse_plan(fasq.plan("gemm", M, K, N, bits, d, C))
    assert base == "k_gemm_mfma" and tuple(params[3:5]) == tile, (label, params)
    x, cb, ids = draw(kind, M, K, N, d, C, seed=M + K + N + C + 1)
    idx = pi.pack_indices(ids, bits)
    y = to_np(fasq.pq_gemm(to_dev(x), to_dev(idx), bits, d, to_dev(cb)))
    check_exact(y, orc.pq_linear(x, idx, bits, d, cb), kind, label)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("case", [(128, 4096, 4096, 4, 256, 8), (40, 14336, 200, 4, 4096, 12),
                                  (37, 8192, 211, 4, 256, 8)])  # M * N odd: the scalar reduce
def test_gemm_k_split(case, kind):
    """fasq_pq_gemm_ex splitting K over workgroups (fp32 partials in the
    workspace, then the fixed-order sum)."""
    M, K, N, d, C, bits = case
    label = f"gemm_ex K split {case} {kind}"
    print(f"[case] {label}", flush=True)
    need = fasq.gemm_ex_workspace_bytes(M, K, N, bits, d, C)
    assert need > 0, label
    x, cb, ids = draw(kind, M, K, N, d, C, seed=sum(case) + 3)
    idx = pi.pack_indices(ids, bits)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda:0")
    y = to_np(fasq.pq_gemm_ex(to_dev(x), to_dev(idx), bits, d, to_dev(cb), workspace=ws))
    check_exact(y, orc.pq_linear(x, idx, bits, d, cb), kind, label)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("case", [(4, 14336, 300, 2, 256, 8), (8, 14336, 140, 4, 4096, 12),
                                  (11, 14336, 200, 2, 256, 8), (16, 12288, 100, 4, 65536, 16)])
def test_gemv_k_split(case, kind):
    """fasq_pq_gemv_ex with one shared codebook where the 16-row-tile decode
    kernel splits K over workgroups (each stages its segment of x; fp32
    partials in the workspace, then the fixed-order sum)."""
    M, K, N, d, C, bits = case
    label = f"gemv_ex decode K split {case} {kind}"
    print(f"[case] {label}", flush=True)
    assert fasq.plan("gemv", M, K, N, bits, d, C).startswith("k_gemv<"), label
    need = fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, 0)
    assert need > 0 and need % (M * N * 4) == 0 and need // (M * N * 4) >= 2, (label, need)
    x, cb, ids = draw(kind, M, K, N, d, C, seed=sum(case) + 5)
    idx = pi.pack_indices(ids, bits)
    ws = torch.zeros(need, dtype=torch.uint8, device="cuda:0")
    y = to_np(fasq.pq_gemv_ex(to_dev(x), to_dev(idx), bits, d, to_dev(cb), workspace=ws))
    check_exact(y, orc.pq_linear(x, idx, bits, d, cb), kind, label)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("case", [(1, 4096, 300, 2, 256, 8), (1, 768, 70, 4, 1024, 12),
                                  (4, 1024, 300, 2, 256, 8), (16, 768, 70, 4, 1024, 12)])
def test_per_subspace_books(case, kind):
    """fasq_pq_gemv_ex with one codebook per subspace (the K-split kernel
    with its books in LDS and v_dot2 products; several tokens with their x
    slices staged in LDS)."""
    M, K, N, d, C, bits = case
    S = K // d
    label = f"gemv_ex per-subspace {case} {kind}"
    print(f"[case] {label}", flush=True)
    assert fasq.gemv_ex_workspace_bytes(M, K, N, bits, d, C, C * d) > 0, label  # the tuned kernel
    x, _, ids = draw(kind, M, K, N, d, C, seed=sum(case) + 5)
    rng = np.random.default_rng(sum(case) + 6)
    if kind == "x":
        books = np.stack([pi.signed_one_hot_codebook(C, d, rng) for _ in range(S)])
    else:
        books = pi.subnormal_codebook(rng, S * C, d, large_frac=0.05 if kind == "wide" else 0.0).reshape(S, C, d)
    idx = pi.pack_indices(ids, bits)
    y = to_np(fasq.pq_gemv_ex(to_dev(x), to_dev(idx), bits, d, to_dev(books)))
    ref = orc.lut_accumulate(x, books, orc.unpack_indices(idx, S, bits, C).T)
    check_exact(y, ref, kind, label)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("case", [(5, 256, 300, 2, 256, 8), (12, 384, 90, 4, 2048, 12)])
def test_lookup_table_gemm(case, kind):
    """The paper's lookup-table GEMM (fp32 tables in LDS)."""
    M, K, N, d, C, bits = case
    label = f"gemm_lut {case} {kind}"
    print(f"[case] {label}", flush=True)
    x, cb, ids = draw(kind, M, K, N, d, C, seed=sum(case) + 7)
    idx = pi.pack_indices(ids, bits)
    y = to_np(fasq.pq_gemm_lut(to_dev(x), to_dev(idx), bits, d, to_dev(cb)))
    check_exact(y, orc.pq_linear(x, idx, bits, d, cb), kind, label)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("case", [(1, 4096, 100, 2, 256, 8), (3, 96, 20, 3, 7, 8), (1, 36, 5, 4, 9, 12)])
def test_general_kernel(case, kind, monkeypatch):
    """The general kernel (any d, any alignment), forced for every call."""
    M, K, N, d, C, bits = case
    label = f"general {case} {kind}"
    print(f"[case] {label}", flush=True)
    monkeypatch.setenv("FASQ_FORCE_PATH", "generic")
    assert fasq.plan("gemv", M, K, N, bits, d, C).startswith("k_pq_generic")
    x, cb, ids = draw(kind, M, K, N, d, C, seed=sum(case) + 9)
    idx = pi.pack_indices(ids, bits)
    y = to_np(fasq.pq_gemv(to_dev(x), to_dev(idx), bits, d, to_dev(cb)))
    check_exact(y, orc.pq_linear(x, idx, bits, d, cb), kind, label)


@pytest.mark.parametrize("kind", KINDS)
@pytest.mark.parametrize("M", [1, 2, 4])
def test_grouped_launch(M, kind):
    """q, k and v shapes (scaled down in K) as one grouped call."""
    K, d, C, bits = 4096, 2, 256, 8
    mats = [(4096, 11), (1024, 12), (1024, 13)]
    label = f"batched M={M} {kind}"
    print(f"[case] {label}", flush=True)
    x, _, _ = draw(kind, M, K, 1, d, C, seed=100 + M)
    probs = []
    for N, seed in mats:
        _, cb, ids = draw(kind, M, K, N, d, C, seed=seed)
        probs.append((cb, pi.pack_indices(ids, bits)))
    ys = fasq.pq_gemv_batched(to_dev(x), [to_dev(i) for _, i in probs], bits, d, [to_dev(c) for c, _ in probs])
    for (cb, idx), y in zip(probs, ys):
        check_exact(to_np(y), orc.pq_linear(x, idx, bits, d, cb), kind, label)
