"""huge_eval_summary_static -- the summary on the library's own static device
scratch, for callers that cannot allocate -- against huge_eval_summary on a
caller workspace, through the C ABI: bit-identical outputs (the same kernels)
on consecutive calls whose inputs shrink and grow, up to the largest count
the scratch holds, and HUGE_ERR_WORKSPACE one above it, returned before any
launch."""
import ctypes

import numpy as np
import pytest

torch = pytest.importorskip("torch")

import paper_2307_14490_amd as P  # noqa: E402
from paper_2307_14490_amd import binding as B  # noqa: E402
from gpu_common import say  # noqa: E402

pytestmark = pytest.mark.gpu

MAX_STATIC = 3_726_784  # largest n_edge + n_non the 32 MiB scratch holds
QUANTILES = (0.0, 1.0, 10.0, 25.0, 50.0, 75.0, 90.0, 99.0, 100.0)


@pytest.fixture(autouse=True)
def _need_gpu():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    yield
    torch.cuda.synchronize()


def _distances(rng, n_edge, n_non):
    """Edge distances below the non-edge ones on average, a few NaNs (failed
    non-edge draws), ties, zeros and subnormals."""
    e = rng.gamma(2.0, 0.3, n_edge).astype(np.float32)
    x = rng.gamma(4.0, 0.3, n_non).astype(np.float32)
    d = np.concatenate([e, x])
    if d.size:
        idx = rng.choice(d.size, size=min(d.size, 1 + d.size // 50), replace=False)
        d[idx[0::3]] = np.nan
        d[idx[1::3]] = 0.0
        d[idx[2::3]] = np.float32(1e-40)
        d[rng.choice(d.size, size=min(d.size, 7), replace=False)] = np.float32(0.75)
    return d


def _static(dist, n_edge, n_non):
    nq = len(QUANTILES)
    q = (ctypes.c_double * nq)(*QUANTILES)
    out = torch.full((5 + 2 * nq,), -7.0, dtype=torch.float64, device="cuda")
    st = P.load().huge_eval_summary_static(ctypes.c_void_p(dist.data_ptr()), n_edge, n_non, q,
                                           nq, ctypes.c_void_p(out.data_ptr()), None)
    torch.cuda.synchronize()
    return st, out.cpu().numpy()


def _reference(dist, n_edge, n_non):
    nq = len(QUANTILES)
    q = (ctypes.c_double * nq)(*QUANTILES)
    ws_bytes = P.load().huge_eval_workspace_bytes(max(n_edge + n_non, 1), 16, 16, 1)
    assert ws_bytes > 0
    ws = torch.empty(ws_bytes + 256, dtype=torch.uint8, device="cuda")
    ptr = ws.data_ptr() + ((-ws.data_ptr()) % 256)
    out = torch.full((5 + 2 * nq,), -9.0, dtype=torch.float64, device="cuda")
    st = P.load().huge_eval_summary(ctypes.c_void_p(dist.data_ptr()), n_edge, n_non, q, nq,
                                    ctypes.c_void_p(out.data_ptr()), ctypes.c_void_p(ptr),
                                    ws_bytes, None)
    torch.cuda.synchronize()
    assert st == B.HUGE_OK
    return out.cpu().numpy()


def test_static_summary_equals_workspace_summary():
    rng = np.random.default_rng(355)
    # two calls in a row, the second smaller; then the largest; then small again
    for n_edge, n_non in ((150_000, 90_001), (3_001, 1_999), (MAX_STATIC - 1_000_000, 1_000_000),
                          (0, 777), (12, 0)):
        say(f"static summary: n_edge={n_edge} n_non={n_non}")
        d = torch.from_numpy(_distances(rng, n_edge, n_non)).cuda()
        st, got = _static(d, n_edge, n_non)
        assert st == B.HUGE_OK
        ref = _reference(d, n_edge, n_non)
        np.testing.assert_array_equal(got, ref)
        valid_edge = int(np.count_nonzero(~np.isnan(d[:n_edge].cpu().numpy())))
        assert got[0] == valid_edge


def test_static_summary_rejects_more_than_its_scratch():
    d = torch.zeros(MAX_STATIC + 1, dtype=torch.float32, device="cuda")
    st, got = _static(d, MAX_STATIC + 1 - 10, 10)
    assert st == B.HUGE_ERR_WORKSPACE
    assert (got == -7.0).all()  # nothing was launched
    st, got = _static(d, -1, 10)
    assert st == B.HUGE_ERR_INVALID_ARG
