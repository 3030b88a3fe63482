"""GPU parity of the k-means encoder (fasq_pq_encode) against the CPU oracle.

The encoder's arithmetic is fully defined (fp32 distances without fused
multiply-add, lowest index on ties, exact cluster sums, fp64 division, one
fp16 rounding), so the codebook and the ids must match the oracle bit for bit.
"""

import numpy as np
import pytest

import pq_inputs as pi
from oracle import pq_encode as enc
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


def gpu_encode(w, d, bits, init, iters):
    cb, idx = fasq.pq_encode(to_dev(w), d, bits, to_dev(init), iters)
    return to_np(cb), to_np(idx)


def check_encode(w, d, C, bits, init, iters, label):
    cb_ref, ids_ref = enc.kmeans_encode(w, d, init, iters)
    cb, idx = gpu_encode(w, d, bits, init, iters)
    assert np.array_equal(cb.view(np.uint16), cb_ref.view(np.uint16)), f"{label}: codebook"
    ids = orc.unpack_indices(idx, w.shape[1] // d, bits, C)
    assert np.array_equal(ids, ids_ref), f"{label}: ids ({int((ids != ids_ref).sum())} differ)"
    return cb, idx


CASES = [
    # N, K, d, C, bits, iters
    (256, 512, 2, 256, 8, 5),     # cluster sums gathered in LDS per workgroup
    (128, 512, 4, 4096, 12, 3),   # sums straight to global atomics
    (256, 512, 4, 20000, 16, 2),  # codebook in five LDS tiles
    (64, 256, 8, 256, 8, 4),
    (100, 300, 3, 50, 8, 3),      # d = 3: the general-d kernel
    (33, 64, 1, 16, 8, 6),
    (50, 36, 4, 9, 12, 4),        # odd 12-bit rows (pad nibble)
    (40, 64, 2, 64, 8, 0),        # no update: ids against the starting codebook
]


@pytest.mark.parametrize("case", CASES)
def test_encode_matches_oracle_bit_exact(case):
    N, K, d, C, bits, iters = case
    print(f"[case] encode {case}", flush=True)
    rng = np.random.default_rng(sum(case))
    w = pi.draw_weights(rng, N, K)
    init = pi.subvectors_at(w, d, pi.init_point_ids(rng, N * K // d, C))
    check_encode(w, d, C, bits, init, iters, str(case))


def test_encode_is_deterministic_and_accepts_in_place_init():
    rng = np.random.default_rng(7)
    N, K, d, C, bits = 512, 1024, 2, 256, 8
    w = to_dev(pi.draw_weights(rng, N, K))
    init = to_dev(pi.subvectors_at(to_np(w), d, pi.init_point_ids(rng, N * K // d, C)))
    a_cb, a_idx = fasq.pq_encode(w, d, bits, init, 4)
    b_cb, b_idx = fasq.pq_encode(w, d, bits, init, 4)
    assert torch.equal(a_cb.view(torch.int16), b_cb.view(torch.int16))
    assert torch.equal(a_idx, b_idx)
    # init_codebook == codebook: the encoder updates the buffer in place
    buf = init.clone()
    idx = torch.empty_like(a_idx)
    ws = torch.empty(fasq.encode_workspace_bytes(N, K, d, C), dtype=torch.uint8, device=w.device)
    st = fasq.encode_raw(w.data_ptr(), N, K, d, C, bits, buf.data_ptr(), 4, buf.data_ptr(), idx.data_ptr(),
                         ws.data_ptr(), ws.numel(), torch.cuda.current_stream().cuda_stream)
    assert st == 0, fasq.last_error()
    assert torch.equal(buf.view(torch.int16), a_cb.view(torch.int16))
    assert torch.equal(idx, a_idx)


def test_means_on_fp16_halfway_points_and_subnormals():
    """Cluster means that fall exactly halfway between fp16 neighbours (ties
    to even) and means in the fp16 subnormal range."""
    rng = np.random.default_rng(9)
    d, C, bits = 1, 64, 8
    vals = []
    for k in range(C // 2):
        a = np.float16(1.0 + k / 64)
        b = np.nextafter(a, np.float16(4.0))
        vals += [a, b]                       # mean halfway between a and b
    for k in range(C // 2):
        vals += [np.float16((k + 1) * 2.0 ** -24), np.float16((k + 2) * 2.0 ** -24)]  # subnormal means
    pts = np.array(vals, dtype=np.float16)
    w = np.repeat(pts, 4).reshape(-1, 8)     # each value four times: same means
    init = np.unique(pts)[:C].reshape(-1, 1)
    init = np.concatenate([init, np.full((C - len(init), 1), 100.0, np.float16)]).astype(np.float16)
    check_encode(w, d, C, bits, init, 3, "halfway")


def test_encoded_layer_runs_through_the_matmul():
    """Encode dense weights, then y = x . W_hat^T from the encoding agrees with
    the oracle on the oracle's encoding (they are the same bits)."""
    rng = np.random.default_rng(10)
    N, K, d, C, bits = 512, 2048, 2, 256, 8
    w = pi.draw_weights(rng, N, K)
    init = pi.subvectors_at(w, d, pi.init_point_ids(rng, N * K // d, C))
    cb, idx = check_encode(w, d, C, bits, init, 6, "layer")
    x = pi.draw_x(rng, 1, K)
    y = to_np(fasq.pq_gemv(to_dev(x), to_dev(idx), bits, d, to_dev(cb))).astype(np.float64)
    assert_close(y, orc.pq_linear(x, idx, bits, d, cb), "encoded layer")
    # quantization error of the layer output against the dense fp16 weights, for the record
    dense = x.astype(np.float64) @ w.astype(np.float64).T
    print(f"[encode] layer rel error vs dense weights: {orc.relative_l2(y, dense):.3f}", flush=True)
