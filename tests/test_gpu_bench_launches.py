"""The decode layers exactly as bench.py launches and times them, at full size.

Each workload's matrices go out in bench.py's launch groups (q+k+v and
gate+up as one grouped call, the others alone, a workspace where the call
takes one), first eagerly, then from a launch list (the timed form) run
several times and from a captured HIP graph replayed several times.  Every output element must be written (the buffers start as NaN).  The
single-token effective-4-bit and effective-3-bit layers, lm_head included,
are compared with the oracle on every output row; the others on sampled rows
that include the rows at every possible part boundary of a grouped launch.
Every run and replay must equal the eager result bit for bit.
"""

import numpy as np
import pytest

import bench
import pq_inputs as pi
from oracle import pq_oracle as orc
from gpu_util import assert_close, sample_rows

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


LAYERS = [
    ("llama3_8b_4bit", 1),
    ("llama3_8b_4bit", 2),
    ("llama3_8b_3bit", 1),
    ("qwen3_8b_sweep", 1),
    ("qwen3_8b_sweep", 4),
    ("qwen3_8b_sweep", 16),
]
# layers compared on every output row (the oracle works in row chunks)
FULL_OUTPUT = {("llama3_8b_4bit", 1), ("llama3_8b_3bit", 1)}


@pytest.mark.parametrize("wl_name,M", LAYERS)
def test_decode_layer_as_timed(wl_name, M):
    print(f"[case] bench layer {wl_name} M={M}", flush=True)
    wl = pi.workload(wl_name)
    problems = [wl.problem(i, M=M) for i in range(len(wl.matrices))]
    names = [m.name for m in wl.matrices]
    ms = bench.MatrixSet(torch, fasq, problems, names, bench.launch_groups(names), min_copies=1,
                         rotation_bytes=0)
    assert ms.copies == 1
    ys = [s["y"] for s in ms.sets[0]]
    stream = torch.cuda.current_stream().cuda_stream

    # eager launches, checked against the oracle on sampled rows; a grouped
    # call reads the x of its first matrix for every member
    x_of = {i: problems[g[0]].x for g in ms.groups for i in g}
    for y in ys:
        y.fill_(float("nan"))
    ms.launch_all(0, stream)
    torch.cuda.synchronize()
    eager = [y.cpu().numpy() for y in ys]
    full = (wl_name, M) in FULL_OUTPUT
    for i, (p, name, got) in enumerate(zip(problems, names, eager)):
        assert np.isfinite(got).all(), f"{wl_name} M={M} {name}: an output was not written"
        rows = np.arange(p.N) if full else sample_rows(p.N, 128)
        ref = orc.pq_linear(x_of[i], p.idx, p.idx_bits, p.d, p.codebook, rows=rows)
        assert_close(got.astype(np.float64)[:, rows], ref,
                     f"{wl_name} M={M} {name} ({'all' if full else len(rows)} rows)")

    # the same launches recorded into a launch list, as bench.py times them
    lst = fasq.LaunchList()
    with lst:
        ms.launch_all(0, stream)
    assert len(lst) >= len(ms.groups)
    for rep in range(3):
        for y in ys:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        lst.run(stream)
        torch.cuda.synchronize()
        for name, y, e in zip(names, ys, eager):
            assert np.array_equal(y.cpu().numpy().view(np.uint16), e.view(np.uint16)), f"list run {rep} {name}"
    lst.close()

    # the same launches from a graph (capture_graphs warms up eagerly first)
    graphs = ms.capture_graphs(1)
    for rep in range(3):
        for y in ys:
            y.fill_(float("nan"))
        torch.cuda.synchronize()
        graphs[0].replay()
        torch.cuda.synchronize()
        for name, y, e in zip(names, ys, eager):
            assert np.array_equal(y.cpu().numpy().view(np.uint16), e.view(np.uint16)), f"replay {rep} {name}"
    del graphs


@pytest.mark.parametrize("M", [128, 512, 2048])
@pytest.mark.parametrize("mat", range(3))
def test_prefill_as_timed(mat, M):
    """fasq_pq_gemm_ex with the workspace bench.py gives it (K split where the
    grid leaves CUs idle), at the prefill shapes."""
    wl = pi.workload("prefill")
    spec = wl.matrices[mat]
    print(f"[case] bench prefill {spec.name} M={M}", flush=True)
    p = wl.problem(mat, M=M)
    dev = torch.device("cuda:0")
    x, idx, cb = (torch.from_numpy(a).to(dev) for a in (p.x, p.idx, p.codebook))
    y = torch.full((M, p.N), float("nan"), dtype=torch.float16, device=dev)
    need = fasq.gemm_ex_workspace_bytes(M, p.K, p.N, p.idx_bits, p.d, p.C)
    ws = torch.empty(max(need, 4), dtype=torch.uint8, device=dev)
    st = fasq.gemm_ex_raw(x.data_ptr(), M, p.K, p.N, idx.data_ptr(), p.idx_bits, p.d, cb.data_ptr(), p.C,
                          y.data_ptr(), ws.data_ptr(), need, torch.cuda.current_stream().cuda_stream)
    assert st == fasq.FASQ_OK, fasq.last_error()
    torch.cuda.synchronize()
    got = y.cpu().numpy()
    assert np.isfinite(got).all(), f"prefill {spec.name} M={M}: an output was not written"
    rows = sample_rows(p.N, 128)
    ref = orc.pq_linear(p.x, p.idx, p.idx_bits, p.d, p.codebook, rows=rows)
    assert_close(got.astype(np.float64)[:, rows], ref, f"prefill {spec.name} M={M} (workspace {need} B)")
