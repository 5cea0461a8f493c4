"""Shared helpers of the GPU parity tests (imported by tests marked gpu)."""
import sys

import numpy as np

# Tolerance on fp32 table values after a step, against the double-precision
# oracle: |gpu - oracle| <= ABS + REL |oracle|.
ABS_TOL = 1e-6
REL_TOL = 1e-5


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def assert_close(gpu, ref, what, abs_tol=ABS_TOL, rel_tol=REL_TOL):
    g = np.asarray(gpu, np.float64)
    r = np.asarray(ref, np.float64)
    assert g.shape == r.shape, (what, g.shape, r.shape)
    diff = np.abs(g - r)
    bound = abs_tol + rel_tol * np.abs(r)
    bad = ~(diff <= bound)
    if bad.any():
        idx = np.argwhere(bad)[:5]
        raise AssertionError(
            f"{what}: {int(bad.sum())} of {bad.size} elements outside tolerance; "
            f"max |diff| {np.nanmax(diff):.3e}; first {idx.tolist()} "
            f"gpu {g[tuple(idx[0])]!r} oracle {r[tuple(idx[0])]!r}")


def dev(a, torch):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()
