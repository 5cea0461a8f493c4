"""ctypes binding of libhuge (argument marshalling only).

Every call maps one-to-one onto a function of ``include/huge.h``; all work
happens in the library's HIP kernels.  PyTorch provides device memory and the
current HIP stream.  If ``libhuge.so`` has not been built, importing this
module raises: there is no fallback path.
"""
from __future__ import annotations

import ctypes
import os

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhuge.so")

HUGE_OK = 0
HUGE_ERR_INVALID_ARG = -1
HUGE_ERR_ID_OUT_OF_RANGE = -2
HUGE_ERR_BAD_COUNT = -3
HUGE_ERR_WORKSPACE = -4
HUGE_ERR_HIP = -5

HUGE_NEG_UNIFORM = 0
HUGE_NEG_ALIAS = 1
HUGE_SCATTER_SORTED = 0
HUGE_SCATTER_ATOMIC = 1
HUGE_DTYPE_F32 = 0
HUGE_DTYPE_BF16 = 1

EXPORTED = [
    "huge_workspace_bytes", "huge_build_alias", "huge_init_tables", "huge_attach_tables",
    "huge_train_step", "huge_prepare_step", "huge_train_prepared", "huge_eval_loss",
    "huge_get_rows", "huge_sample_negatives", "huge_probe_rows", "huge_check", "huge_step_stats", "huge_profile_begin", "huge_profile_end",
    "huge_destroy", "huge_status_string", "huge_walk_workspace_bytes", "huge_sample_walks",
    "huge_eval_workspace_bytes", "huge_eval_pairs", "huge_eval_distances", "huge_eval_summary",
    "huge_eval_summary_static",
    "huge_eval_knn", "huge_eval_knn_lists", "huge_eval_recall", "huge_train_step_weighted", "huge_prepare_step_weighted",
    "huge_eval_loss_weighted", "huge_cocount_weights",
]
HUGE_PHASES = 6


class HugeConfig(ctypes.Structure):
    _fields_ = [
        ("num_nodes", ctypes.c_int64),
        ("dim", ctypes.c_int32),
        ("num_neg_per_pos", ctypes.c_int32),
        ("max_batch", ctypes.c_int64),
        ("seed", ctypes.c_uint64),
        ("init_half_width", ctypes.c_float),
        ("neg_kind", ctypes.c_int32),
        ("scatter_kind", ctypes.c_int32),
        ("table_dtype", ctypes.c_int32),
    ]


class HugeWalkConfig(ctypes.Structure):
    _fields_ = [
        ("num_nodes", ctypes.c_int64),
        ("walks_per_node", ctypes.c_int32),
        ("walk_steps", ctypes.c_int32),
        ("window", ctypes.c_int32),
        ("seed_pairs_only", ctypes.c_int32),
        ("seed", ctypes.c_uint64),
    ]


class HugeError(RuntimeError):
    def __init__(self, status: int, what: str):
        super().__init__(f"{what}: {status_string(status)} ({status})")
        self.status = status


_vp = ctypes.c_void_p
_lib = None


def load() -> ctypes.CDLL:
    """Load libhuge.so; raise if it is missing (build it first)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run python -m paper_2307_14490_amd.build")
    L = ctypes.CDLL(LIB_PATH)
    cfgp = ctypes.POINTER(HugeConfig)
    L.huge_workspace_bytes.argtypes = [cfgp]
    L.huge_workspace_bytes.restype = ctypes.c_size_t
    L.huge_build_alias.argtypes = [_vp, ctypes.c_int64, _vp, _vp]
    L.huge_init_tables.argtypes = [cfgp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t, _vp,
                                   ctypes.POINTER(_vp)]
    L.huge_attach_tables.argtypes = [cfgp, _vp, _vp, _vp, _vp, _vp, ctypes.c_size_t,
                                     ctypes.POINTER(_vp)]
    L.huge_train_step.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_uint64,
                                  ctypes.c_float, _vp, _vp]
    L.huge_prepare_step.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_uint64, _vp]
    L.huge_train_prepared.argtypes = [_vp, ctypes.c_float, _vp, _vp]
    L.huge_eval_loss.argtypes = [_vp, _vp, _vp, _vp, ctypes.c_int64, ctypes.c_uint64, _vp, _vp]
    L.huge_get_rows.argtypes = [_vp, ctypes.c_int32, _vp, ctypes.c_int64, _vp, _vp]
    L.huge_sample_negatives.argtypes = [_vp, ctypes.c_int64, ctypes.c_uint64, _vp, _vp]
    L.huge_probe_rows.argtypes = [_vp, _vp, _vp, ctypes.c_int64, ctypes.c_uint64, _vp]
    L.huge_check.argtypes = [_vp, _vp]
    L.huge_step_stats.argtypes = [_vp, _vp, ctypes.POINTER(ctypes.c_int64),
                                  ctypes.POINTER(ctypes.c_int64), ctypes.POINTER(ctypes.c_int64)]
    L.huge_profile_begin.argtypes = [_vp, ctypes.c_int32, ctypes.c_int32, ctypes.c_int32]
    L.huge_profile_end.argtypes = [_vp, _vp, ctypes.POINTER(ctypes.c_double),
                                   ctypes.POINTER(ctypes.c_int32)]
    wcfgp = ctypes.POINTER(HugeWalkConfig)
    L.huge_walk_workspace_bytes.argtypes = [wcfgp, ctypes.c_int64]
    L.huge_walk_workspace_bytes.restype = ctypes.c_size_t
    L.huge_sample_walks.argtypes = [wcfgp, _vp, _vp, ctypes.c_int64, ctypes.c_int64,
                                    ctypes.c_int64, _vp, _vp, _vp, _vp, ctypes.c_int64, _vp, _vp,
                                    _vp, ctypes.c_size_t, _vp]
    L.huge_sample_walks.restype = ctypes.c_int32
    i64, i32, u64, szt = ctypes.c_int64, ctypes.c_int32, ctypes.c_uint64, ctypes.c_size_t
    L.huge_eval_workspace_bytes.argtypes = [i64, i64, i32, i32]
    L.huge_eval_workspace_bytes.restype = szt
    L.huge_eval_pairs.argtypes = [_vp, _vp, i64, i64, u64, i64, i64, i32, _vp, _vp, _vp, _vp]
    L.huge_eval_distances.argtypes = [_vp, i64, i32, _vp, _vp, i64, _vp, _vp, _vp]
    L.huge_eval_summary.argtypes = [_vp, i64, i64, ctypes.POINTER(ctypes.c_double), i32, _vp,
                                    _vp, szt, _vp]
    L.huge_eval_summary_static.argtypes = [_vp, i64, i64, ctypes.POINTER(ctypes.c_double), i32,
                                           _vp, _vp]
    L.huge_eval_knn.argtypes = [_vp, i64, i32, _vp, i32, i32, _vp, _vp, _vp, szt, _vp, _vp]
    L.huge_eval_knn_lists.argtypes = L.huge_eval_knn.argtypes
    L.huge_eval_recall.argtypes = [_vp, _vp, i64, i64, _vp, i32, _vp, i32, _vp, _vp, _vp]
    for name in ("huge_eval_pairs", "huge_eval_distances", "huge_eval_summary", "huge_eval_knn",
                 "huge_eval_knn_lists", "huge_eval_recall"):
        getattr(L, name).restype = ctypes.c_int32
    L.huge_train_step_weighted.argtypes = [_vp, _vp, _vp, _vp, i64, ctypes.c_uint64,
                                           ctypes.c_float, _vp, _vp]
    L.huge_prepare_step_weighted.argtypes = [_vp, _vp, _vp, _vp, i64, ctypes.c_uint64, _vp]
    L.huge_eval_loss_weighted.argtypes = [_vp, _vp, _vp, _vp, i64, ctypes.c_uint64, _vp, _vp]
    L.huge_cocount_weights.argtypes = [_vp, i64, i32, ctypes.POINTER(ctypes.c_float), _vp, _vp]
    for name in ("huge_train_step_weighted", "huge_prepare_step_weighted",
                 "huge_eval_loss_weighted", "huge_cocount_weights"):
        getattr(L, name).restype = ctypes.c_int32
    L.huge_destroy.argtypes = [_vp]
    L.huge_destroy.restype = None
    L.huge_status_string.argtypes = [ctypes.c_int32]
    L.huge_status_string.restype = ctypes.c_char_p
    for name in ("huge_build_alias", "huge_init_tables", "huge_attach_tables", "huge_train_step",
                 "huge_prepare_step", "huge_train_prepared",
                 "huge_eval_loss", "huge_get_rows", "huge_sample_negatives", "huge_probe_rows",
                 "huge_check",
                 "huge_step_stats", "huge_profile_begin", "huge_profile_end"):
        getattr(L, name).restype = ctypes.c_int32
    _lib = L
    return L


def status_string(st: int) -> str:
    return load().huge_status_string(st).decode()


def _ok(st: int, what: str):
    if st != HUGE_OK:
        raise HugeError(st, what)


def make_config(num_nodes, dim, num_neg, max_batch, seed=0, init_half_width=0.0,
                neg_kind=HUGE_NEG_UNIFORM, scatter_kind=HUGE_SCATTER_SORTED,
                table_dtype=HUGE_DTYPE_F32) -> HugeConfig:
    return HugeConfig(int(num_nodes), int(dim), int(num_neg), int(max_batch), int(seed),
                      float(init_half_width), int(neg_kind), int(scatter_kind),
                      int(table_dtype))


def workspace_bytes(cfg: HugeConfig) -> int:
    return int(load().huge_workspace_bytes(ctypes.byref(cfg)))


def build_alias(weights):
    """Host alias table: returns (thr uint32[n], alias int32[n]) numpy arrays."""
    w = np.ascontiguousarray(weights, dtype=np.float64)
    thr = np.empty(w.size, np.uint32)
    alias = np.empty(w.size, np.int32)
    _ok(load().huge_build_alias(w.ctypes.data, w.size, thr.ctypes.data, alias.ctypes.data),
        "huge_build_alias")
    return thr, alias


def _stream_ptr(stream=None):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return s.cuda_stream


def _dptr(t):
    return None if t is None else t.data_ptr()


def _arg(t, dtypes, what):
    """Device pointer of `t`, which must be a contiguous GPU tensor of one of
    `dtypes` (torch dtype names): the C calls take raw pointers, so a tensor
    of another type would be read as the wrong type."""
    import torch
    ok = (isinstance(t, torch.Tensor) and t.is_cuda and t.is_contiguous()
          and any(t.dtype == getattr(torch, d) for d in dtypes))
    if not ok:
        got = (f"{t.dtype} on {t.device}{'' if t.is_contiguous() else ', not contiguous'}"
               if isinstance(t, torch.Tensor) else type(t).__name__)
        raise TypeError(f"{what}: expected a contiguous GPU tensor of {' or '.join(dtypes)}, "
                        f"got {got}")
    return t.data_ptr()


def _batch(src, dst, cc, what):
    """Pointers of a batch: int32 ids, int32 co_counts or float32 weights."""
    if src.numel() != dst.numel() or src.numel() != cc.numel():
        raise ValueError(f"{what}: src, dst and counts differ in length")
    return (_arg(src, ("int32",), what + " src"), _arg(dst, ("int32",), what + " dst"),
            _arg(cc, ("int32", "float32"), what + " counts"))


def _is_float(t):
    import torch
    return t is not None and t.dtype == torch.float32


def cocount_weights(hist, dist_weights, stream=None):
    """float32 weight per triple from its distance histogram (device int32,
    n x window) and per-distance weights (host sequence), by
    huge_cocount_weights."""
    import torch
    n, window = hist.shape
    wd = (ctypes.c_float * window)(*[float(x) for x in dist_weights])
    out = torch.empty(n, dtype=torch.float32, device=hist.device)
    _ok(load().huge_cocount_weights(_arg(hist, ("int32",), "cocount_weights hist"), int(n),
                                    int(window), wd, _dptr(out),
                                    _stream_ptr(stream)), "huge_cocount_weights")
    return out


def _check_tables(tables, num_nodes, dim, dtype, device):
    """Caller-supplied (S, T): each must be a contiguous (num_nodes, dim)
    tensor of `dtype` on `device`; every step writes rows of both at offsets
    computed from num_nodes and dim, so a smaller, strided or host table would
    be written out of bounds.  Checked before anything is allocated."""
    import torch
    if not (isinstance(tables, (tuple, list)) and len(tables) == 2):
        raise TypeError("tables: expected a pair (S, T) of tensors")
    for name, t in zip(("S", "T"), tables):
        if not isinstance(t, torch.Tensor):
            raise TypeError(f"table {name}: expected a tensor, got {type(t).__name__}")
        if tuple(t.shape) != (num_nodes, dim):
            raise ValueError(f"table {name}: shape {tuple(t.shape)}, expected ({num_nodes}, {dim})")
        if t.dtype != dtype:
            raise ValueError(f"table {name}: dtype {t.dtype}, expected {dtype}")
        if not t.is_contiguous():
            raise ValueError(f"table {name}: not contiguous")
        if t.device.type != "cuda" or (device.index is not None and t.device != device):
            raise ValueError(f"table {name}: on {t.device}, expected {device}")


class Trainer:
    """Tables, workspace and a libhuge handle on one GPU.

    S and T are float32 (or, with dtype="bf16", bfloat16) torch tensors
    (N x D) on the device; the workspace is a uint8 torch tensor.  Batches are
    int32 device tensors.
    """

    def __init__(self, num_nodes, dim, num_neg, max_batch, seed=0, init_half_width=0.0,
                 alias_weights=None, scatter="sorted", device="cuda", tables=None,
                 init=True, dtype="f32"):
        import torch
        load()
        self.device = torch.device(device)
        kind = HUGE_NEG_ALIAS if alias_weights is not None else HUGE_NEG_UNIFORM
        sk = {"sorted": HUGE_SCATTER_SORTED, "atomic": HUGE_SCATTER_ATOMIC}[scatter]
        td = {"f32": HUGE_DTYPE_F32, "bf16": HUGE_DTYPE_BF16}[dtype]
        tdt = torch.bfloat16 if td == HUGE_DTYPE_BF16 else torch.float32
        self.cfg = make_config(num_nodes, dim, num_neg, max_batch, seed, init_half_width, kind, sk,
                               td)
        ws = workspace_bytes(self.cfg)
        if ws == 0:
            raise HugeError(HUGE_ERR_INVALID_ARG, "huge_workspace_bytes")
        if tables is not None:
            _check_tables(tables, int(num_nodes), int(dim), tdt, self.device)
            self.S, self.T = tables
        else:
            self.S = torch.empty((num_nodes, dim), dtype=tdt, device=self.device)
            self.T = torch.empty((num_nodes, dim), dtype=tdt, device=self.device)
        self.workspace = torch.empty(ws, dtype=torch.uint8, device=self.device)
        if kind == HUGE_NEG_ALIAS:
            thr, alias = build_alias(alias_weights)
            self.alias_thr = torch.from_numpy(thr.view(np.int32)).to(self.device)
            self.alias = torch.from_numpy(alias).to(self.device)
        else:
            self.alias_thr = self.alias = None
        self.loss_buf = torch.zeros(1, dtype=torch.float64, device=self.device)
        h = _vp()
        if init:
            st = load().huge_init_tables(ctypes.byref(self.cfg), _dptr(self.S), _dptr(self.T),
                                         _dptr(self.alias_thr), _dptr(self.alias),
                                         _dptr(self.workspace), ws, _stream_ptr(), ctypes.byref(h))
        else:
            st = load().huge_attach_tables(ctypes.byref(self.cfg), _dptr(self.S), _dptr(self.T),
                                           _dptr(self.alias_thr), _dptr(self.alias),
                                           _dptr(self.workspace), ws, ctypes.byref(h))
        _ok(st, "huge_init_tables" if init else "huge_attach_tables")
        self._h = h

    # -- calls ------------------------------------------------------------
    # cc: int32 co_counts, or float32 weights (the *_weighted calls)
    def step(self, src, dst, cc, first_pos, lr, loss_out=None, stream=None):
        loss = self.loss_buf if loss_out is None else loss_out
        fn = "huge_train_step_weighted" if _is_float(cc) else "huge_train_step"
        ps, pd, pc = _batch(src, dst, cc, fn)
        _ok(getattr(load(), fn)(self._h, ps, pd, pc, src.numel(), int(first_pos), float(lr),
                                _arg(loss, ("float64",), fn + " loss"), _stream_ptr(stream)), fn)
        return loss

    def step_no_loss(self, src, dst, cc, first_pos, lr, stream=None):
        fn = "huge_train_step_weighted" if _is_float(cc) else "huge_train_step"
        ps, pd, pc = _batch(src, dst, cc, fn)
        _ok(getattr(load(), fn)(self._h, ps, pd, pc, src.numel(), int(first_pos), float(lr),
                                None, _stream_ptr(stream)), fn)

    def prepare(self, src, dst, cc, first_pos, stream=None):
        """Group a batch (validation, negatives, de-duplication) into a slot."""
        fn = "huge_prepare_step_weighted" if _is_float(cc) else "huge_prepare_step"
        ps, pd, pc = _batch(src, dst, cc, fn)
        _ok(getattr(load(), fn)(self._h, ps, pd, pc, src.numel(), int(first_pos),
                                _stream_ptr(stream)), fn)

    def train_prepared(self, lr, loss_out=None, with_loss=True, stream=None):
        """Apply the oldest prepared batch; returns the loss tensor (or None)."""
        loss = (self.loss_buf if loss_out is None else loss_out) if with_loss else None
        pl = None if loss is None else _arg(loss, ("float64",), "huge_train_prepared loss")
        _ok(load().huge_train_prepared(self._h, float(lr), pl, _stream_ptr(stream)),
            "huge_train_prepared")
        return loss

    def eval_loss(self, src, dst, cc, first_pos, loss_out=None, stream=None):
        loss = self.loss_buf if loss_out is None else loss_out
        fn = "huge_eval_loss_weighted" if _is_float(cc) else "huge_eval_loss"
        ps, pd, pc = _batch(src, dst, cc, fn)
        _ok(getattr(load(), fn)(self._h, ps, pd, pc, src.numel(), int(first_pos),
                                _arg(loss, ("float64",), fn + " loss"), _stream_ptr(stream)), fn)
        return loss

    def get_rows(self, table, ids, stream=None):
        import torch
        ids = ids.to(device=self.device, dtype=torch.int64).contiguous()
        out = torch.empty((ids.numel(), self.cfg.dim), dtype=torch.float32, device=self.device)
        _ok(load().huge_get_rows(self._h, int(table), _dptr(ids), ids.numel(), _dptr(out),
                                 _stream_ptr(stream)), "huge_get_rows")
        return out

    def sample_negatives(self, n, first_pos, stream=None):
        import torch
        out = torch.empty((n, self.cfg.num_neg_per_pos), dtype=torch.int32, device=self.device)
        _ok(load().huge_sample_negatives(self._h, int(n), int(first_pos), _dptr(out),
                                         _stream_ptr(stream)), "huge_sample_negatives")
        return out

    def probe_rows(self, src, dst, first_pos, stream=None):
        """Read and write back, unchanged, every row a step over this batch
        would touch (the bandwidth ceiling of the step's row traffic)."""
        n = src.numel()
        if dst.numel() != n:
            raise ValueError("src and dst must have the same length")
        _ok(load().huge_probe_rows(self._h, _arg(src, ("int32",), "probe_rows src"),
                                   _arg(dst, ("int32",), "probe_rows dst"), n, int(first_pos),
                                   _stream_ptr(stream)), "huge_probe_rows")

    def check(self, stream=None) -> int:
        return int(load().huge_check(self._h, _stream_ptr(stream)))

    def stats(self, stream=None):
        a, b, c = ctypes.c_int64(), ctypes.c_int64(), ctypes.c_int64()
        _ok(load().huge_step_stats(self._h, _stream_ptr(stream), ctypes.byref(a), ctypes.byref(b),
                                   ctypes.byref(c)), "huge_step_stats")
        return a.value, b.value, c.value

    def profile_begin(self, max_steps, all_phases=False, every=1):
        """Events on every `every`-th one of the next batches, max_steps of them."""
        _ok(load().huge_profile_begin(self._h, int(max_steps), int(bool(all_phases)), int(every)),
            "huge_profile_begin")

    def profile_end(self, stream=None):
        """Summed phase durations (ms, list of HUGE_PHASES) and the step count."""
        arr = (ctypes.c_double * HUGE_PHASES)()
        n = ctypes.c_int32()
        _ok(load().huge_profile_end(self._h, _stream_ptr(stream), arr, ctypes.byref(n)),
            "huge_profile_end")
        return list(arr), n.value

    def close(self):
        if getattr(self, "_h", None) is not None and self._h.value:
            load().huge_destroy(self._h)
            self._h = _vp()

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def walk_config(num_nodes, walks_per_node, walk_steps, window, seed_pairs_only=True, seed=0):
    return HugeWalkConfig(int(num_nodes), int(walks_per_node), int(walk_steps), int(window),
                          int(bool(seed_pairs_only)), int(seed))


def sample_walks(offsets, neighbors, num_nodes, walks_per_node, walk_steps, window,
                 seed_pairs_only=True, seed=0, first_seed=0, num_seeds=None, capacity=None,
                 with_hist=True, stream=None):
    """Co-occurrence triples of random walks on a device CSR graph (int64
    offsets, int32 neighbours), computed by huge_sample_walks.  With
    capacity=None the triples are counted first (one extra pass) and the
    outputs sized to fit.  Returns (src, dst, cc, hist or None) on the device."""
    import torch
    L = load()
    p_off = _arg(offsets, ("int64",), "sample_walks offsets")
    p_nbr = _arg(neighbors, ("int32",), "sample_walks neighbors")
    cfg = walk_config(num_nodes, walks_per_node, walk_steps, window, seed_pairs_only, seed)
    if num_seeds is None:
        num_seeds = int(num_nodes) - int(first_seed)
    dev = offsets.device
    ws_bytes = L.huge_walk_workspace_bytes(ctypes.byref(cfg), int(num_seeds))
    if ws_bytes == 0:
        raise HugeError(HUGE_ERR_INVALID_ARG, "huge_walk_workspace_bytes")
    ws = torch.empty(ws_bytes + 256, dtype=torch.uint8, device=dev)
    ws_off = (-ws.data_ptr()) % 256
    count = torch.zeros(1, dtype=torch.int64, device=dev)
    status = torch.zeros(1, dtype=torch.int32, device=dev)
    empty = torch.empty(0, dtype=torch.int32, device=dev)

    def run(cap, src, dst, cc, hist):
        _ok(L.huge_sample_walks(ctypes.byref(cfg), p_off, p_nbr,
                                neighbors.numel(), int(first_seed), int(num_seeds),
                                _dptr(src) if cap else None, _dptr(dst) if cap else None,
                                _dptr(cc) if cap else None,
                                _dptr(hist) if (cap and hist is not None) else None, int(cap),
                                _dptr(count), _dptr(status), ws.data_ptr() + ws_off, ws_bytes,
                                _stream_ptr(stream)), "huge_sample_walks")

    if capacity is None:
        run(0, empty, empty, empty, None)
        st = int(status.item())
        if st not in (0, -4):
            raise HugeError(st, "huge_sample_walks (device)")
        capacity = int(count.item())
    n = int(capacity)
    src = torch.empty(n, dtype=torch.int32, device=dev)
    dst = torch.empty(n, dtype=torch.int32, device=dev)
    cc = torch.empty(n, dtype=torch.int32, device=dev)
    hist = torch.empty((n, int(window)), dtype=torch.int32, device=dev) if with_hist else None
    run(n, src, dst, cc, hist)
    st = int(status.item())
    if st != 0:
        raise HugeError(st, "huge_sample_walks (device)")
    got = int(count.item())
    return src[:got], dst[:got], cc[:got], (hist[:got] if hist is not None else None)


# --------------------------------------------------------------------------- #
# Embedding evaluation (argument marshalling for the huge_eval_* calls)
# --------------------------------------------------------------------------- #
def _check_csr(offsets, neighbors, num_nodes, what):
    """A CSR graph of num_nodes nodes: num_nodes + 1 offsets (the kernels read
    offsets[u] and offsets[u + 1] for every node u)."""
    if offsets.dim() != 1 or offsets.numel() != int(num_nodes) + 1:
        raise ValueError(f"{what}: {offsets.numel()} offsets for {int(num_nodes)} nodes "
                         f"(expected num_nodes + 1)")
    if neighbors.dim() != 1:
        raise ValueError(f"{what}: neighbors must be one-dimensional")


def _check_table2d(table, what):
    if table.dim() != 2:
        raise ValueError(f"{what}: table must be two-dimensional, got shape {tuple(table.shape)}")


class Evaluator:
    """Workspace and status word for the huge_eval_* calls on one table shape.
    Each method checks the device status word after its call (synchronising
    the stream) and raises HugeError on a device-detected error."""

    def __init__(self, num_rows, dim, max_pairs, k=10, device="cuda"):
        import torch
        L = load()
        self.num_rows, self.dim, self.k = int(num_rows), int(dim), int(k)
        self.ws_bytes = L.huge_eval_workspace_bytes(int(max_pairs), self.num_rows, self.dim,
                                                    self.k)
        if self.ws_bytes == 0:
            raise HugeError(HUGE_ERR_INVALID_ARG, "huge_eval_workspace_bytes")
        self._ws = torch.empty(self.ws_bytes + 256, dtype=torch.uint8, device=device)
        self._ws_ptr = self._ws.data_ptr() + ((-self._ws.data_ptr()) % 256)
        self.status = torch.zeros(1, dtype=torch.int32, device=device)
        self.device = device

    def _check(self, what):
        st = int(self.status.item())
        if st != 0:
            raise HugeError(st, what + " (device)")

    def pairs(self, offsets, neighbors, num_nodes, seed, n_edge, n_non, max_tries=64,
              stream=None):
        """(u, v) int32 device tensors: n_edge edge pairs, then n_non non-edges."""
        import torch
        _check_csr(offsets, neighbors, num_nodes, "Evaluator.pairs")
        n = int(n_edge) + int(n_non)
        u = torch.empty(n, dtype=torch.int32, device=self.device)
        v = torch.empty(n, dtype=torch.int32, device=self.device)
        _ok(load().huge_eval_pairs(_arg(offsets, ("int64",), "Evaluator.pairs offsets"),
                                   _arg(neighbors, ("int32",), "Evaluator.pairs neighbors"),
                                   int(num_nodes),
                                   int(neighbors.numel()), int(seed), int(n_edge), int(n_non),
                                   int(max_tries), _dptr(u), _dptr(v), _dptr(self.status),
                                   _stream_ptr(stream)), "huge_eval_pairs")
        self._check("huge_eval_pairs")
        return u, v

    def distances(self, table, u, v, stream=None):
        import torch
        _check_table2d(table, "Evaluator.distances")
        if u.numel() != v.numel():
            raise ValueError("Evaluator.distances: u and v differ in length")
        d = torch.empty(u.numel(), dtype=torch.float32, device=self.device)
        _ok(load().huge_eval_distances(_arg(table, ("float32",), "Evaluator.distances table"),
                                       table.shape[0], table.shape[1],
                                       _arg(u, ("int32",), "Evaluator.distances u"),
                                       _arg(v, ("int32",), "Evaluator.distances v"), u.numel(),
                                       _dptr(d), _dptr(self.status),
                                       _stream_ptr(stream)), "huge_eval_distances")
        self._check("huge_eval_distances")
        return d

    def summary(self, dist, n_edge, n_non, quantiles=(0, 10, 25, 50, 75, 90, 100), stream=None,
                static=False):
        """dict: count_edge, count_non, mean_edge, mean_non, snr, pct_edge, pct_non.
        static=True: through huge_eval_summary_static (the library's own
        device scratch, no workspace)."""
        import torch
        if int(n_edge) < 0 or int(n_non) < 0 or dist.numel() < int(n_edge) + int(n_non):
            raise ValueError(f"Evaluator.summary: {dist.numel()} distances for "
                             f"{int(n_edge)} + {int(n_non)} pairs")
        q = (ctypes.c_double * len(quantiles))(*[float(x) for x in quantiles])
        nq = len(quantiles)
        out = torch.empty(5 + 2 * nq, dtype=torch.float64, device=self.device)
        if static:
            _ok(load().huge_eval_summary_static(
                _arg(dist, ("float32",), "Evaluator.summary dist"), int(n_edge), int(n_non), q,
                nq, _dptr(out), _stream_ptr(stream)), "huge_eval_summary_static")
        else:
            _ok(load().huge_eval_summary(_arg(dist, ("float32",), "Evaluator.summary dist"),
                                         int(n_edge), int(n_non), q, nq, _dptr(out),
                                         self._ws_ptr, self.ws_bytes, _stream_ptr(stream)),
                "huge_eval_summary")
        o = out.cpu().tolist()
        return {"count_edge": int(o[0]), "count_non": int(o[1]), "mean_edge": o[2],
                "mean_non": o[3], "snr": o[4], "pct_edge": o[5:5 + nq],
                "pct_non": o[5 + nq:5 + 2 * nq]}

    def knn(self, table, queries, k=None, stream=None, lists=False):
        """(ids int32 [nq, k], dist float32 [nq, k]) of the nearest rows
        (lists=True: by huge_eval_knn_lists, the per-wave list search)."""
        import torch
        k = self.k if k is None else int(k)
        if k > self.k:
            raise HugeError(HUGE_ERR_INVALID_ARG, "Evaluator.knn: k above the workspace's")
        _check_table2d(table, "Evaluator.knn")
        nq = queries.numel()
        ids = torch.empty((nq, k), dtype=torch.int32, device=self.device)
        dist = torch.empty((nq, k), dtype=torch.float32, device=self.device)
        name = "huge_eval_knn_lists" if lists else "huge_eval_knn"
        _ok(getattr(load(), name)(_arg(table, ("float32",), "Evaluator.knn table"),
                                  table.shape[0], table.shape[1],
                                  _arg(queries, ("int32",), "Evaluator.knn queries"),
                                  nq, k, _dptr(ids), _dptr(dist), self._ws_ptr, self.ws_bytes,
                                  _dptr(self.status), _stream_ptr(stream)), name)
        self._check(name)
        return ids, dist

    def recall(self, offsets, neighbors, num_nodes, queries, ids, stream=None):
        import torch
        _check_csr(offsets, neighbors, num_nodes, "Evaluator.recall")
        if ids.dim() != 2 or ids.shape[0] != queries.numel():
            raise ValueError(f"Evaluator.recall: ids of shape {tuple(ids.shape)} for "
                             f"{queries.numel()} queries")
        nq, k = ids.shape
        out = torch.empty(nq, dtype=torch.float64, device=self.device)
        _ok(load().huge_eval_recall(_arg(offsets, ("int64",), "Evaluator.recall offsets"),
                                    _arg(neighbors, ("int32",), "Evaluator.recall neighbors"),
                                    int(num_nodes), int(neighbors.numel()),
                                    _arg(queries, ("int32",), "Evaluator.recall queries"),
                                    int(nq), _arg(ids, ("int32",), "Evaluator.recall ids"),
                                    int(k), _dptr(out), _dptr(self.status),
                                    _stream_ptr(stream)), "huge_eval_recall")
        self._check("huge_eval_recall")
        return out
