"""Host-side checks of the C ABI (no GPU): the library loads, exports every
function declared in include/huge.h, sizes its workspace, builds alias tables
identical to the oracle's, and rejects bad arguments before any launch."""
import ctypes
import os
import re

import numpy as np
import pytest

import paper_2307_14490_amd as P
from paper_2307_14490_amd import binding as B
from oracle import oracle as orc

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))


def _declared():
    text = open(os.path.join(ROOT, "include", "huge.h")).read()
    decl = r"^(?:size_t|huge_status|void|const char\*)\s+(huge_[a-z_]+)\s*\("
    return sorted(set(re.findall(decl, text, flags=re.M)))


def test_library_exports_every_declared_symbol():
    L = P.load()
    names = _declared()
    assert len(names) >= 12
    for n in names:
        assert hasattr(L, n), n
    assert sorted(B.EXPORTED) == names


def test_library_exports_only_declared_symbols():
    """The dynamic symbol table of libhuge.so holds exactly the functions of
    include/huge.h: no helper, kernel stub or template instantiation that
    another library in the process could collide with."""
    import shutil
    import subprocess
    nm = shutil.which("nm")
    if nm is None:
        pytest.skip("nm is not installed")
    out = subprocess.run([nm, "-D", "--defined-only", B.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = sorted(line.split()[-1] for line in out.splitlines() if line.strip())
    assert exported == _declared()


def _bad_tables():
    import torch
    N, D = 64, 8
    f32 = torch.float32
    good = torch.zeros((N, D), dtype=f32)
    yield "shape", (torch.zeros((N - 1, D), dtype=f32), good)
    yield "shape", (good, torch.zeros((N, D + 4), dtype=f32))
    yield "dtype", (torch.zeros((N, D), dtype=torch.float64), good)
    yield "dtype", (good, torch.zeros((N, D), dtype=torch.bfloat16))
    yield "contiguous", (torch.zeros((D, N), dtype=f32).t(), good)
    yield "on cpu", (good, good)
    yield "pair", (good,)


@pytest.mark.parametrize("case", list(range(7)))
def test_trainer_rejects_bad_tables_before_any_launch(case):
    """Caller tables are checked for shape, dtype, contiguity and device
    before any pointer reaches the library: every step writes rows at offsets
    computed from (num_nodes, dim)."""
    what, tables = list(_bad_tables())[case]
    with pytest.raises((ValueError, TypeError)):
        B.Trainer(64, 8, 2, 16, tables=tables, device="cuda:0")


def test_evaluator_rejects_mismatched_lengths():
    """Lengths the kernels index by are checked on the host (no GPU: the
    checks run before any device allocation or launch)."""
    import torch
    ev = B.Evaluator.__new__(B.Evaluator)  # no workspace: the checks come first
    ev.device = "cpu"
    ev.k = 10
    off = torch.zeros(11, dtype=torch.int64)
    nbr = torch.zeros(5, dtype=torch.int32)
    with pytest.raises(ValueError):
        ev.pairs(off, nbr, 12, 0, 4, 4)           # offsets must be num_nodes + 1
    with pytest.raises(ValueError):
        ev.recall(off, nbr, 12, torch.zeros(3, dtype=torch.int32),
                  torch.zeros((3, 2), dtype=torch.int32))
    with pytest.raises(ValueError):
        ev.recall(off, nbr, 10, torch.zeros(3, dtype=torch.int32),
                  torch.zeros((4, 2), dtype=torch.int32))  # one id row per query
    tab = torch.zeros((10, 8), dtype=torch.float32)
    with pytest.raises(ValueError):
        ev.distances(tab, torch.zeros(3, dtype=torch.int32), torch.zeros(4, dtype=torch.int32))
    with pytest.raises(ValueError):
        ev.distances(tab.view(-1), torch.zeros(3, dtype=torch.int32),
                     torch.zeros(3, dtype=torch.int32))
    with pytest.raises(ValueError):
        ev.summary(torch.zeros(5, dtype=torch.float32), 3, 3)  # 6 pairs, 5 distances
    with pytest.raises(ValueError):
        ev.knn(tab.view(-1), torch.zeros(2, dtype=torch.int32), 1)


def test_status_strings_cover_every_code():
    seen = set()
    for code in (0, -1, -2, -3, -4, -5):
        s = B.status_string(code)
        assert s and s != "unknown status"
        seen.add(s)
    assert len(seen) == 6
    assert B.status_string(-99) == "unknown status"


@pytest.mark.parametrize("kw", [
    dict(num_nodes=0), dict(num_nodes=2**31), dict(dim=6), dict(dim=0), dict(dim=1028),
    dict(num_neg=0), dict(num_neg=65), dict(max_batch=0), dict(max_batch=2**31 // 7 + 1),
])
def test_invalid_configs_have_no_workspace(kw):
    base = dict(num_nodes=1000, dim=32, num_neg=5, max_batch=100)
    base.update(kw)
    assert P.workspace_bytes(P.make_config(**base)) == 0


def test_bad_kind_and_width():
    c = P.make_config(1000, 32, 5, 100)
    c.neg_kind = 7
    assert P.workspace_bytes(c) == 0
    c = P.make_config(1000, 32, 5, 100)
    c.scatter_kind = 2
    assert P.workspace_bytes(c) == 0
    c = P.make_config(1000, 32, 5, 100, init_half_width=-1.0)
    assert P.workspace_bytes(c) == 0
    c = P.make_config(1000, 32, 5, 100, init_half_width=float("inf"))
    assert P.workspace_bytes(c) == 0


def test_table_dtype_config():
    f32 = P.workspace_bytes(P.make_config(10**5, 64, 5, 1000))
    bf16 = P.workspace_bytes(P.make_config(10**5, 64, 5, 1000, table_dtype=P.binding.HUGE_DTYPE_BF16))
    # the workspace (fp32 contributions of repeated rows) does not depend on it
    assert bf16 == f32 > 0
    # bf16 tables take the sorted scatter only
    assert P.workspace_bytes(P.make_config(10**5, 64, 5, 1000, scatter_kind=1, table_dtype=1)) == 0
    c = P.make_config(10**5, 64, 5, 1000)
    c.table_dtype = 2
    assert P.workspace_bytes(c) == 0


def test_workspace_grows_with_batch_and_holds_duplicate_buffer():
    small = P.workspace_bytes(P.make_config(10**6, 128, 5, 1000))
    big = P.workspace_bytes(P.make_config(10**6, 128, 5, 100_000))
    assert big > small > 0
    # sorted scatter keeps one D-float slot per occurrence
    M = 100_000 * 7
    assert big >= M * 128 * 4
    atomic = P.workspace_bytes(P.make_config(10**6, 128, 5, 100_000, scatter_kind=1))
    assert 0 < atomic < big


def test_host_alias_table_equals_oracle_bitwise():
    rng = np.random.default_rng(0)
    for w in (rng.pareto(1.2, 50_000) + 1e-3,
              np.concatenate([np.zeros(10), rng.integers(1, 100, 1000).astype(float)]),
              np.ones(33), np.array([0.0, 0.0, 2.5])):
        t1, a1 = P.build_alias(w)
        t2, a2 = orc.build_alias(w)
        assert np.array_equal(t1, t2) and np.array_equal(a1, a2)


def test_host_alias_rejects_bad_weights():
    for w in (np.zeros(3), np.array([1.0, -2.0]), np.array([np.inf]), np.array([])):
        with pytest.raises(B.HugeError) as e:
            P.build_alias(w)
        assert e.value.status == B.HUGE_ERR_INVALID_ARG


def test_calls_reject_bad_arguments_before_any_launch():
    L = P.load()
    vp = ctypes.c_void_p
    # null handle
    assert L.huge_train_step(None, None, None, None, 0, 0, 0.1, None, None) == -1
    assert L.huge_eval_loss(None, None, None, None, 0, 0, None, None) == -1
    assert L.huge_get_rows(None, 0, None, 1, None, None) == -1
    assert L.huge_sample_negatives(None, 1, 0, None, None) == -1
    assert L.huge_probe_rows(None, None, None, 1, 0, None) == -1
    assert L.huge_check(None, None) == -1
    assert L.huge_step_stats(None, None, None, None, None) == -1
    L.huge_destroy(None)
    # invalid config or null pointers: rejected on the host
    h = vp()
    cfg = P.make_config(1000, 6, 5, 10)
    assert L.huge_init_tables(ctypes.byref(cfg), 4096, 8192, None, None, 1 << 20, 1 << 30,
                              None, ctypes.byref(h)) == -1
    cfg = P.make_config(1000, 32, 5, 10)
    assert L.huge_init_tables(ctypes.byref(cfg), None, 8192, None, None, 1 << 20, 1 << 30,
                              None, ctypes.byref(h)) == -1
    assert L.huge_init_tables(ctypes.byref(cfg), 4096, 8192, None, None, None, 1 << 30,
                              None, ctypes.byref(h)) == -1
    # alias sampling without tables
    cfg = P.make_config(1000, 32, 5, 10, neg_kind=1)
    assert L.huge_init_tables(ctypes.byref(cfg), 4096, 8192, None, None, 1 << 20, 1 << 30,
                              None, ctypes.byref(h)) == -1
    # misaligned workspace
    cfg = P.make_config(1000, 32, 5, 10)
    assert L.huge_init_tables(ctypes.byref(cfg), 4096, 8192, None, None, (1 << 20) + 8,
                              1 << 30, None, ctypes.byref(h)) == -1
    # workspace too small
    need = P.workspace_bytes(cfg)
    assert L.huge_init_tables(ctypes.byref(cfg), 4096, 8192, None, None, 1 << 20, need - 1,
                              None, ctypes.byref(h)) == -4
    assert L.huge_attach_tables(ctypes.byref(cfg), 4096, 8192, None, None, 1 << 20, need - 1,
                                ctypes.byref(h)) == -4
    assert not h.value


def test_host_tensors_are_refused_before_any_device_work():
    """The C calls take raw device pointers: the binding refuses tensors of
    another type or on the host instead of passing their memory on."""
    torch = pytest.importorskip("torch")
    with pytest.raises(TypeError, match="GPU tensor of int32"):
        P.cocount_weights(torch.zeros((3, 2), dtype=torch.int32), [1.0, 0.5])
    with pytest.raises(TypeError, match="int64"):
        P.sample_walks(torch.zeros(4, dtype=torch.int64), torch.zeros(3, dtype=torch.int32),
                       3, 1, 2, 1)


def test_bench_refuses_several_gpus():
    """The benchmark measures one GPU and says so for --gpus above 1."""
    import subprocess
    import sys
    root = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
    r = subprocess.run([sys.executable, os.path.join(root, "bench.py"), "--gpus", "2"],
                       capture_output=True, text=True, timeout=120, cwd=root)
    assert r.returncode == 2 and "one GPU" in r.stderr
