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


def bf16_values(bits):
    """Exact float64 values of bf16 bit patterns (uint16)."""
    return (np.asarray(bits, np.uint16).astype(np.uint32) << 16).view(np.float32).astype(np.float64)


def assert_bf16_close(got, want, what, abs_tol=ABS_TOL, max_mismatch=2e-3):
    """bf16 tables (uint16 bit patterns) after a step against the oracle's.

    Each element within one bf16 step (|x| 2^-7 bounds it) plus abs_tol,
    the fp32 step's absolute tolerance: the kernels' fp32 arithmetic errs by
    a few fp32 ulps of the operands, which spans more than one bf16 step only
    where the result is much smaller than the operands (cancellation near
    zero).  And nearly all elements equal."""
    got = np.asarray(got, np.uint16)
    want = np.asarray(want, np.uint16)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    g, w = bf16_values(got), bf16_values(want)
    err = np.abs(g - w)
    bound = np.maximum(np.abs(g), np.abs(w)) * 2.0 ** -7 + abs_tol
    bad = np.count_nonzero(got != want)
    say(f"  {what}: {bad} of {got.size} elements differ, max error / bound "
        f"{(err / bound).max() if got.size else 0.0:.3f}")
    assert np.all(err <= bound), what
    assert bad <= max_mismatch * got.size, what


def dev(a, torch):
    return torch.from_numpy(np.ascontiguousarray(a)).cuda()
