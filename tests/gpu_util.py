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


def part_boundary_rows(N, max_parts=8, tile=16):
    """Rows on both sides of every place a launch may cut a matrix into parts.

    A grouped decode launch cuts a matrix into at most ``max_parts`` parts of
    near-equal size: ranges of rows (the row-streaming kernels) or of whole
    ``tile``-row tiles (the 16-row-tile kernel).  Every such cut, for every
    part count, contributes the last row before it and the first row after.
    """
    rows = set()
    for c in range(1, max_parts + 1):
        for units, scale in ((N, 1), ((N + tile - 1) // tile, tile)):
            base, extra = divmod(units, c)
            start = 0
            for i in range(c):
                start += (base + (1 if i < extra else 0)) * scale
                rows.update(r for r in (start - 1, start) if 0 <= r < N)
    return rows


def sample_rows(N, k=256, seed=0):
    """Sorted sample of output rows: k random rows plus the first and last
    row and the rows at every possible part boundary of a grouped launch."""
    rng = np.random.default_rng(seed + N)
    if N <= k:
        return np.arange(N)
    rows = set(rng.choice(N, size=k - 2, replace=False).tolist())
    rows.update([0, N - 1])
    rows.update(part_boundary_rows(N))
    return np.array(sorted(rows))


def assert_close(y, y_ref, label=""):
    y = np.asarray(y, dtype=np.float64)
    rel = orc.relative_l2(y, y_ref)
    mx = orc.max_abs_over_rms(y, y_ref)
    print(f"[parity] {label} rel_l2={rel:.3e} max_err/rms={mx:.3e}", flush=True)
    assert rel <= REL_L2_TOL, (label, rel)
    assert mx <= MAX_ERR_OVER_RMS_TOL, (label, mx)
    return rel, mx
