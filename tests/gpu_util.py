"""Helpers for the GPU parity tests (device transfer, sampling, tolerances)."""

import numpy as np

from oracle import pq_oracle as orc

# Tolerances for y: fp32 accumulation, one fp16 rounding of each output.
REL_L2_TOL = 1e-3
MAX_ERR_OVER_RMS_TOL = 1e-2


def torch_mod():
    import torch

    return torch


def dev():
    return torch_mod().device("cuda:0")


def to_dev(a):
    torch = torch_mod()
    return torch.from_numpy(np.ascontiguousarray(a)).to(dev())


def to_np(t):
    torch = torch_mod()
    torch.cuda.synchronize()
    return t.cpu().numpy()


def sample_rows(N, k=256, seed=0):
    """Sorted sample of output rows, always including the first and last."""
    rng = np.random.default_rng(seed + N)
    if N <= k:
        return np.arange(N)
    rows = set(rng.choice(N, size=k - 2, replace=False).tolist())
    rows.update([0, N - 1])
    return np.array(sorted(rows))


def assert_close(y, y_ref, label=""):
    y = np.asarray(y, dtype=np.float64)
    rel = orc.relative_l2(y, y_ref)
    mx = orc.max_abs_over_rms(y, y_ref)
    print(f"[parity] {label} rel_l2={rel:.3e} max_err/rms={mx:.3e}", flush=True)
    assert rel <= REL_L2_TOL, (label, rel)
    assert mx <= MAX_ERR_OVER_RMS_TOL, (label, mx)
    return rel, mx
