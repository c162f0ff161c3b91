"""ctypes binding of libgt (C ABI in include/gt.h).

Argument marshalling only: every wrapper checks tensor shapes/dtypes/devices,
allocates outputs and workspace with torch on the tensors' device, and calls
the C entry point of the same name on torch's current HIP stream.  Nothing
here computes any part of the method.  The library must be built
(``python -m paper_2407_14106_amd.build``); loading fails loudly otherwise.
"""

from __future__ import annotations

import ctypes
import math
import os
import threading
from dataclasses import dataclass

import torch

LIB_PATH = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libgt.so")

GT_OK = 0
GT_ERR_INVALID_ARG = -1
GT_ERR_UNSUPPORTED = -2
GT_ERR_UNSORTED = -3
GT_ERR_DUPLICATE = -4
GT_ERR_OUT_OF_RANGE = -5
GT_ERR_WORKSPACE = -6
GT_ERR_HIP = -7
GT_F32 = 0
GT_BF16 = 1
GT_LONG_ROW = 256

_i32, _i64, _u32, _u64 = ctypes.c_int32, ctypes.c_int64, ctypes.c_uint32, ctypes.c_uint64
_vp, _sz, _f32 = ctypes.c_void_p, ctypes.c_size_t, ctypes.c_float


class GtTiles(ctypes.Structure):
    _fields_ = [
        ("n", _i64), ("T", _i32), ("reserved", _i32), ("n_row_tiles", _i64), ("n_dense", _i64),
        ("nnz_sparse", _i64), ("n_long_rows", _i64), ("n_long_cols", _i64),
        ("tile_rowptr", _vp), ("tile_col", _vp), ("tile_nnz", _vp), ("tile_mask", _vp),
        ("sp_rowptr", _vp), ("sp_col", _vp), ("sp_colptr", _vp), ("sp_row", _vp),
        ("tileT_ptr", _vp), ("tileT_idx", _vp), ("long_rows", _vp), ("long_cols", _vp),
        ("sp_pos", _vp), ("tile_pos", _vp),
    ]


GT_AUTOTUNER_RUNGS = 7
GT_AUTOTUNER_HISTORY = 64
_f64 = ctypes.c_double


class GtAutotuner(ctypes.Structure):
    _fields_ = [
        ("F", _f64), ("ldr", _f64 * GT_AUTOTUNER_HISTORY), ("t", _i64), ("last_change", _i64), ("level", _i32),
        ("delta", _i32), ("num", _u64 * GT_AUTOTUNER_RUNGS), ("den", _u64 * GT_AUTOTUNER_RUNGS),
    ]


class GtInterleaveReport(ctypes.Structure):
    _fields_ = [
        ("n", _i64), ("missing_self_loops", _i64), ("min_degree", _i64), ("reached", _i64), ("ecc_root", _i32),
        ("ecc_far", _i32), ("c1", _i32), ("c2", _i32), ("c3", _i32), ("use_sparse", _i32),
    ]


_P = ctypes.POINTER
SIGNATURES = {
    "gt_abi_version": (_i32, []),
    "gt_status_string": (ctypes.c_char_p, [_i32]),
    "gt_last_error": (ctypes.c_char_p, []),
    "gt_validate_csr_workspace_size": (_sz, []),
    "gt_validate_csr": (_i32, [_i64, _i64, _vp, _vp, _vp, _sz, _vp]),
    "gt_reorder_workspace_size": (_sz, [_i64, _i64]),
    "gt_reorder": (_i32, [_i64, _i64, _vp, _vp, _i32, _u64, _vp, _vp, _vp, _P(_i32), _vp, _sz, _vp]),
    "gt_reorder_streams": (_i32, [_i64, _i64, _vp, _vp, _i32, _u64, _vp, _vp, _vp, _P(_i32), _vp, _sz, _vp,
                                  _vp, _vp, _i32]),
    "gt_permute_workspace_size": (_sz, [_i64, _i64]),
    "gt_permute_csr": (_i32, [_i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "gt_permute_edges_workspace_size": (_sz, [_i64, _i64]),
    "gt_permute_csr_edges": (_i32, [_i64, _i64, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "gt_gather_rows": (_i32, [_i64, _i64, _vp, _vp, _vp, _vp]),
    "gt_scatter_rows": (_i32, [_i64, _i64, _vp, _vp, _vp, _vp]),
    "gt_tiles_workspace_size": (_sz, [_i64, _i64, _i32]),
    "gt_tiles_count": (_i32, [_i64, _i64, _vp, _vp, _i32, _u32, _P(GtTiles), _vp, _sz, _vp]),
    "gt_build_tiles": (_i32, [_i64, _i64, _vp, _vp, _i32, _u32, _P(GtTiles), _vp, _sz, _vp]),
    "gt_sparse_attn_fwd_workspace_size": (_sz, [_P(GtTiles), _i32, _i32, _i32]),
    "gt_sparse_attn_fwd": (_i32, [_P(GtTiles), _i32, _i32, _i32, _vp, _vp, _vp, _f32, _vp, _vp, _vp, _sz, _vp]),
    "gt_sparse_attn_bwd_workspace_size": (_sz, [_P(GtTiles), _i32, _i32, _i32]),
    "gt_sparse_attn_bwd": (_i32, [_P(GtTiles), _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _f32, _vp, _vp, _vp,
                                  _vp, _sz, _vp]),
    "gt_sparse_attn_bwd_rows_workspace_size": (_sz, [_P(GtTiles), _i32, _i32, _i32]),
    "gt_sparse_attn_bwd_rows": (_i32, [_P(GtTiles), _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _f32, _vp, _vp,
                                       _vp, _sz, _vp]),
    "gt_sparse_attn_bwd_cols_workspace_size": (_sz, [_P(GtTiles), _i32, _i32, _i32]),
    "gt_sparse_attn_bwd_cols": (_i32, [_P(GtTiles), _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _f32, _vp,
                                       _vp, _vp, _sz, _vp]),
    "gt_edge_map_workspace_size": (_sz, [_P(GtTiles)]),
    "gt_edge_map": (_i32, [_P(GtTiles), _vp, _vp, _sz, _vp]),
    "gt_sparse_attn_fwd_bias_workspace_size": (_sz, [_P(GtTiles), _i32, _i32, _i32]),
    "gt_sparse_attn_bwd_bias_workspace_size": (_sz, [_P(GtTiles), _i32, _i32, _i32]),
    "gt_sparse_attn_fwd_bias": (_i32, [_P(GtTiles), _i32, _i32, _i32, _vp, _vp, _vp, _vp, _f32, _vp, _vp, _vp,
                                       _sz, _vp]),
    "gt_sparse_attn_bwd_bias": (_i32, [_P(GtTiles), _vp, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _f32,
                                       _vp, _vp, _vp, _vp, _vp, _sz, _vp]),
    "gt_gather_probe": (_i32, [_P(GtTiles), _i32, _i32, _i32, _vp, _vp, _vp, _vp]),
    "gt_ecr_max_nnz": (_i64, [_i64, _i32, _i32]),
    "gt_ecr_workspace_size": (_sz, [_i64, _i64, _i32, _i32]),
    "gt_ecr_compact": (_i32, [_i64, _i64, _vp, _vp, _i32, _i32, _u64, _u64, _vp, _vp, _i64, _P(_i64), _P(_i32), _vp,
                              _sz, _vp]),
    "gt_autotuner_init": (_i32, [_P(GtAutotuner), _i64, _i64, _i32]),
    "gt_autotuner_step": (_i32, [_P(GtAutotuner), _f64, _f64, _P(_i32), _P(_u64), _P(_u64)]),
    "gt_interleave_workspace_size": (_sz, [_i64]),
    "gt_interleave_check": (_i32, [_i64, _i64, _vp, _vp, _i32, _P(GtInterleaveReport), _vp, _vp, _sz, _vp]),
    "gt_dense_attn_fwd": (_i32, [_i64, _i32, _i32, _i32, _vp, _vp, _vp, _f32, _vp, _vp, _vp]),
    "gt_dense_attn_bwd_workspace_size": (_sz, [_i64, _i32, _i32, _i32]),
    "gt_dense_attn_bwd": (_i32, [_i64, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _f32, _vp, _vp, _vp, _vp,
                                 _sz, _vp]),
    "gt_dense_attn_bwd_noalloc_max_bytes": (_sz, []),
    "gt_dense_attn_bwd_noalloc": (_i32, [_i64, _i32, _i32, _i32, _vp, _vp, _vp, _vp, _vp, _vp, _f32, _vp, _vp,
                                         _vp, _vp]),
}

_LIB = None


class GtError(RuntimeError):
    def __init__(self, status: int, where: str, text: str):
        super().__init__(f"{where}: status {status} ({text})")
        self.status = status


def load_library(path: str = LIB_PATH) -> ctypes.CDLL:
    """Load libgt.so and declare its signatures; raises if it is missing."""
    global _LIB
    if _LIB is not None:
        return _LIB
    if not os.path.exists(path):
        raise RuntimeError(f"libgt.so not found at {path}: build it with `python -m paper_2407_14106_amd.build`")
    lib = ctypes.CDLL(path)
    for name, (res, args) in SIGNATURES.items():
        fn = getattr(lib, name)
        fn.restype = res
        fn.argtypes = args
    _LIB = lib
    return lib


def _check(status: int, where: str):
    if status != GT_OK:
        lib = load_library()
        raise GtError(status, where, lib.gt_last_error().decode() or lib.gt_status_string(status).decode())


def _ptr(t: torch.Tensor | None):
    return None if t is None else ctypes.c_void_p(t.data_ptr())


def _stream(device: torch.device):
    return ctypes.c_void_p(torch.cuda.current_stream(device).cuda_stream)


def _workspace(nbytes: int, device) -> torch.Tensor:
    return torch.empty(max(int(nbytes), 256), dtype=torch.uint8, device=device)


def _need(cond: bool, msg: str):
    if not cond:
        raise ValueError(msg)


def _check_csr(rowptr: torch.Tensor, col: torch.Tensor):
    _need(rowptr.is_cuda and col.is_cuda, "CSR must be on the GPU")
    _need(rowptr.dtype == torch.int64 and col.dtype == torch.int32, "rowptr int64 and col int32 expected")
    _need(rowptr.is_contiguous() and col.is_contiguous(), "CSR must be contiguous")
    _need(rowptr.dim() == 1 and rowptr.numel() >= 1, "rowptr must be 1-D with n+1 entries")


# ------------------------------------------------------------------------ integer stages

def validate_csr(rowptr: torch.Tensor, col: torch.Tensor) -> None:
    lib = load_library()
    _check_csr(rowptr, col)
    ws = _workspace(lib.gt_validate_csr_workspace_size(), rowptr.device)
    _check(lib.gt_validate_csr(rowptr.numel() - 1, col.numel(), _ptr(rowptr), _ptr(col), _ptr(ws), ws.numel(),
                               _stream(rowptr.device)), "gt_validate_csr")


_SIDE = threading.local()


def side_streams(dev: torch.device):
    """(streams, events) for the calls that spread independent work beside the current stream: two streams of
    the device (default priority) and three events, made once per host thread and kept by this module (a
    call records the events, so two threads never share them)."""
    idx = dev.index if dev.index is not None else torch.cuda.current_device()
    per = getattr(_SIDE, "per_device", None)
    if per is None:
        per = _SIDE.per_device = {}
    got = per.get(idx)
    if got is None:
        streams = [torch.cuda.Stream(device=idx) for _ in range(2)]
        events = [torch.cuda.Event() for _ in range(3)]
        with torch.cuda.device(idx):
            for e in events:
                e.record(torch.cuda.current_stream(idx))  # makes the event
        got = per[idx] = (streams, events)
    return got


def reorder(rowptr: torch.Tensor, col: torch.Tensor, iters: int = 20, seed: int = 0, want_sweeps: bool = False,
            n_side: int = 2):
    """(perm, iperm, labels[, sweeps]) of the cluster reordering.  n_side (0 to 2) side streams run each
    sweep's row classes beside the current stream (the same result with any n_side)."""
    lib = load_library()
    _check_csr(rowptr, col)
    n, nnz = rowptr.numel() - 1, col.numel()
    dev = rowptr.device
    perm = torch.empty(n, dtype=torch.int32, device=dev)
    iperm = torch.empty(n, dtype=torch.int32, device=dev)
    labels = torch.empty(n, dtype=torch.int32, device=dev)
    ws = _workspace(lib.gt_reorder_workspace_size(n, nnz), dev)
    sweeps = ctypes.c_int32(-1)
    side = events = None
    if n_side > 0:
        streams, evs = side_streams(dev)
        side = (ctypes.c_void_p * 2)(*[s.cuda_stream for s in streams])
        events = (ctypes.c_void_p * 3)(*[e.cuda_event for e in evs])
    _check(lib.gt_reorder_streams(n, nnz, _ptr(rowptr), _ptr(col), iters, ctypes.c_uint64(seed % (1 << 64)),
                                  _ptr(perm), _ptr(iperm), _ptr(labels),
                                  ctypes.byref(sweeps) if want_sweeps else None, _ptr(ws), ws.numel(),
                                  _stream(dev), side, events, n_side), "gt_reorder")
    return (perm, iperm, labels, sweeps.value) if want_sweeps else (perm, iperm, labels)


def permute_csr(rowptr: torch.Tensor, col: torch.Tensor, perm: torch.Tensor, iperm: torch.Tensor):
    lib = load_library()
    _check_csr(rowptr, col)
    n, nnz = rowptr.numel() - 1, col.numel()
    _need(perm.dtype == torch.int32 and iperm.dtype == torch.int32 and perm.numel() == n == iperm.numel(),
          "perm/iperm must be int32[n]")
    dev = rowptr.device
    rp = torch.empty(n + 1, dtype=torch.int64, device=dev)
    cl = torch.empty(nnz, dtype=torch.int32, device=dev)
    ws = _workspace(lib.gt_permute_workspace_size(n, nnz), dev)
    _check(lib.gt_permute_csr(n, nnz, _ptr(rowptr), _ptr(col), _ptr(perm), _ptr(iperm), _ptr(rp), _ptr(cl),
                              _ptr(ws), ws.numel(), _stream(dev)), "gt_permute_csr")
    return rp, cl


def permute_csr_edges(rowptr: torch.Tensor, col: torch.Tensor, perm: torch.Tensor, iperm: torch.Tensor):
    """(rowptr_out, col_out, src_pos): the relabelled CSR and, per new edge, its old CSR position."""
    lib = load_library()
    _check_csr(rowptr, col)
    n, nnz = rowptr.numel() - 1, col.numel()
    _need(perm.dtype == torch.int32 and iperm.dtype == torch.int32 and perm.numel() == n == iperm.numel(),
          "perm/iperm must be int32[n]")
    dev = rowptr.device
    rp = torch.empty(n + 1, dtype=torch.int64, device=dev)
    cl = torch.empty(nnz, dtype=torch.int32, device=dev)
    src = torch.empty(nnz, dtype=torch.int32, device=dev)
    ws = _workspace(lib.gt_permute_edges_workspace_size(n, nnz), dev)
    _check(lib.gt_permute_csr_edges(n, nnz, _ptr(rowptr), _ptr(col), _ptr(perm), _ptr(iperm), _ptr(rp), _ptr(cl),
                                    _ptr(src), _ptr(ws), ws.numel(), _stream(dev)), "gt_permute_csr_edges")
    return rp, cl, src


def _row_bytes(x: torch.Tensor) -> int:
    return x[0].numel() * x.element_size() if x.shape[0] else 0


def gather_rows(x: torch.Tensor, perm: torch.Tensor) -> torch.Tensor:
    """out[r] = x[perm[r]] (row gather along dim 0)."""
    lib = load_library()
    _need(x.is_contiguous() and perm.dtype == torch.int32 and perm.numel() == x.shape[0], "bad gather arguments")
    out = torch.empty_like(x)
    _check(lib.gt_gather_rows(x.shape[0], _row_bytes(x), _ptr(x), _ptr(perm), _ptr(out), _stream(x.device)),
           "gt_gather_rows")
    return out


def scatter_rows(x: torch.Tensor, perm: torch.Tensor) -> torch.Tensor:
    """out[perm[r]] = x[r] (inverse of gather_rows)."""
    lib = load_library()
    _need(x.is_contiguous() and perm.dtype == torch.int32 and perm.numel() == x.shape[0], "bad scatter arguments")
    out = torch.empty_like(x)
    _check(lib.gt_scatter_rows(x.shape[0], _row_bytes(x), _ptr(x), _ptr(perm), _ptr(out), _stream(x.device)),
           "gt_scatter_rows")
    return out


def ecr_compact(rowptr: torch.Tensor, col: torch.Tensor, k: int, d_b: int, num: int, den: int):
    """(rowptr', col', n_transferred): the graph after the lossy cluster reformation at threshold num/den."""
    lib = load_library()
    _check_csr(rowptr, col)
    n, nnz = rowptr.numel() - 1, col.numel()
    dev = rowptr.device
    cap = lib.gt_ecr_max_nnz(nnz, k, d_b)
    _need(cap >= 0, "k must be in [1, 64] and d_b in [1, 256]")
    rp = torch.empty(n + 1, dtype=torch.int64, device=dev)
    cl = torch.empty(max(cap, 1), dtype=torch.int32, device=dev)
    ws = _workspace(lib.gt_ecr_workspace_size(n, nnz, k, d_b), dev)
    out = ctypes.c_int64(0)
    moved = ctypes.c_int32(0)
    _check(lib.gt_ecr_compact(n, nnz, _ptr(rowptr), _ptr(col), k, d_b, ctypes.c_uint64(num), ctypes.c_uint64(den),
                              _ptr(rp), _ptr(cl), cap, ctypes.byref(out), ctypes.byref(moved), _ptr(ws), ws.numel(),
                              _stream(dev)), "gt_ecr_compact")
    return rp, cl[:out.value].clone(), moved.value


def interleave_check(rowptr: torch.Tensor, col: torch.Tensor, L: int, want_levels: bool = False):
    """The C1-C3 report of the interleave decision as a dict (and the first search's depths if asked)."""
    lib = load_library()
    _check_csr(rowptr, col)
    n, nnz = rowptr.numel() - 1, col.numel()
    dev = rowptr.device
    ws = _workspace(lib.gt_interleave_workspace_size(n), dev)
    rep = GtInterleaveReport()
    lev = torch.empty(n, dtype=torch.int32, device=dev) if want_levels else None
    _check(lib.gt_interleave_check(n, nnz, _ptr(rowptr), _ptr(col), int(L), ctypes.byref(rep), _ptr(lev), _ptr(ws),
                                   ws.numel(), _stream(dev)), "gt_interleave_check")
    out = {name: getattr(rep, name) for name, _ in GtInterleaveReport._fields_}
    return (out, lev) if want_levels else out


class AutoTuner:
    """The transfer-threshold controller of the lossy reformation (state held in the C struct)."""

    def __init__(self, n: int, nnz: int, delta: int = 10):
        self.lib = load_library()
        self.c = GtAutotuner()
        _check(self.lib.gt_autotuner_init(ctypes.byref(self.c), n, nnz, delta), "gt_autotuner_init")

    def step(self, loss: float, epoch_seconds: float):
        """Returns (level, num, den) for the next epoch."""
        lv, num, den = ctypes.c_int32(0), ctypes.c_uint64(0), ctypes.c_uint64(0)
        _check(self.lib.gt_autotuner_step(ctypes.byref(self.c), float(loss), float(epoch_seconds), ctypes.byref(lv),
                                          ctypes.byref(num), ctypes.byref(den)), "gt_autotuner_step")
        return lv.value, num.value, den.value


_ITEMSIZE = {torch.int64: 8, torch.int32: 4}


@dataclass
class Plan:
    """A tile plan: the device arrays and the C struct pointing at them.  The arrays live in one device buffer;
    `arrays` gives tensor views of them (made on first use)."""

    c: GtTiles
    buffer: torch.Tensor
    layout: dict  # name -> (byte offset, elements, dtype)
    nnz: int = -1  # edges of the input CSR (remainder plus dense tiles)
    _views: dict | None = None

    @property
    def arrays(self) -> dict:
        if self._views is None:
            self._views = {k: self.buffer[o:o + cnt * _ITEMSIZE[dt]].view(dt)
                           for k, (o, cnt, dt) in self.layout.items()}
        return self._views

    @property
    def n(self):
        return self.c.n

    @property
    def T(self):
        return self.c.T

    @property
    def n_dense(self):
        return self.c.n_dense

    @property
    def nnz_sparse(self):
        return self.c.nnz_sparse

    def to_numpy(self) -> dict:
        out = {k: v.cpu().numpy() for k, v in self.arrays.items()}
        out["T"] = self.c.T
        out["n_row_tiles"] = self.c.n_row_tiles
        return out


def tau_to_ppm(tau: float) -> int:
    return int(round(float(tau) * 1e6))


# Default density threshold: the break-even density measured on MI355X for bf16
# features (a 128 x 128 tile, forward and backward, costs about what 6.6% (d=32)
# to 12% (d=64, partial sums merged by the edge kernels included) of its pairs
# cost as edges), so a tile the plan makes dense is not slower than its edges.
# The paper's lower thresholds remain available through tau_ppm.
BREAK_EVEN_TAU_PPM = 120_000


def build_tiles(rowptr: torch.Tensor, col: torch.Tensor, T: int = 128, tau_ppm: int = BREAK_EVEN_TAU_PPM, *,
                build_ws: torch.Tensor | None = None, between=None, edge_positions: bool = False) -> Plan:
    """Tile plan of the CSR at tile edge T and density threshold tau_ppm (parts per million; by default
    the measured break-even density, BREAK_EVEN_TAU_PPM).

    gt_tiles_count and gt_build_tiles share one workspace, so the build takes the counts from it.  build_ws
    gives the build call a workspace of its own instead, and between(ws) runs between the two calls; with
    either, the build counts again (the library checks the workspace).  edge_positions: also fill sp_pos and
    tile_pos (the input-CSR positions a per-edge bias needs on a plan with dense tiles)."""
    lib = load_library()
    _check_csr(rowptr, col)
    n, nnz = rowptr.numel() - 1, col.numel()
    dev = rowptr.device
    ws = _workspace(lib.gt_tiles_workspace_size(n, nnz, T), dev)
    c = GtTiles()
    st = _stream(dev)
    _check(lib.gt_tiles_count(n, nnz, _ptr(rowptr), _ptr(col), T, tau_ppm, ctypes.byref(c), _ptr(ws), ws.numel(), st),
           "gt_tiles_count")
    R, nd, ns = c.n_row_tiles, c.n_dense, c.nnz_sparse
    i64, i32 = torch.int64, torch.int32
    sizes = [("tile_rowptr", R + 1, i64), ("tile_col", nd, i32), ("tile_nnz", nd, i32),
             ("tile_mask", nd * T * T // 32, i32), ("sp_rowptr", n + 1, i64), ("sp_col", ns, i32),
             ("sp_colptr", n + 1, i64), ("sp_row", ns, i32), ("tileT_ptr", R + 1, i64), ("tileT_idx", nd, i32),
             ("long_rows", c.n_long_rows, i32), ("long_cols", c.n_long_cols, i32)]
    if edge_positions:
        sizes += [("sp_pos", ns, i32), ("tile_pos", nd * T, i32)]
    # one allocation for all of them, each array at a 256-byte boundary
    layout, at = {}, 0
    for name, cnt, dt in sizes:
        layout[name] = (at, cnt, dt)
        at += (cnt * _ITEMSIZE[dt] + 255) & ~255
    buf = torch.empty(max(at, 256), dtype=torch.uint8, device=dev)
    base = buf.data_ptr()
    for name, (off, _, _) in layout.items():
        setattr(c, name, base + off)
    if between is not None:
        between(ws)
    if build_ws is not None:
        _need(build_ws.numel() >= ws.numel() and build_ws.device == ws.device, "build_ws too small")
        ws = build_ws
    _check(lib.gt_build_tiles(n, nnz, _ptr(rowptr), _ptr(col), T, tau_ppm, ctypes.byref(c), _ptr(ws), ws.numel(), st),
           "gt_build_tiles")
    return Plan(c=c, buffer=buf, layout=layout, nnz=nnz)


# ------------------------------------------------------------------------------ attention

def _dtype_code(t: torch.Tensor) -> int:
    if t.dtype == torch.float32:
        return GT_F32
    if t.dtype == torch.bfloat16:
        return GT_BF16
    raise ValueError(f"unsupported dtype {t.dtype}")


def _check_feats(n: int, *ts: torch.Tensor):
    ref = ts[0]
    _need(ref.dim() == 3 and ref.shape[0] == n, "features must be [n, H, d]")
    for t in ts:
        _need(t.shape == ref.shape and t.dtype == ref.dtype and t.is_cuda and t.is_contiguous(),
              "feature tensors must share shape/dtype and be contiguous GPU tensors")


def sparse_attn_fwd(plan: Plan, Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, scale: float | None = None):
    """(O, LSE) of neighbourhood softmax attention over the plan's graph."""
    lib = load_library()
    _check_feats(plan.n, Q, K, V)
    n, H, d = Q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dt = _dtype_code(Q)
    O = torch.empty_like(Q)
    LSE = torch.empty((n, H), dtype=torch.float32, device=Q.device)
    ws = _workspace(lib.gt_sparse_attn_fwd_workspace_size(ctypes.byref(plan.c), H, d, dt), Q.device)
    _check(lib.gt_sparse_attn_fwd(ctypes.byref(plan.c), H, d, dt, _ptr(Q), _ptr(K), _ptr(V), scale, _ptr(O),
                                  _ptr(LSE), _ptr(ws), ws.numel(), _stream(Q.device)), "gt_sparse_attn_fwd")
    return O, LSE


def sparse_attn_bwd(plan: Plan, Q, K, V, dO, LSE, scale: float | None = None):
    """(dQ, dK, dV) of neighbourhood softmax attention."""
    lib = load_library()
    _check_feats(plan.n, Q, K, V, dO)
    n, H, d = Q.shape
    _need(LSE.dtype == torch.float32 and LSE.shape == (n, H) and LSE.is_contiguous(), "LSE must be fp32 [n, H]")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dt = _dtype_code(Q)
    dQ, dK, dV = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
    ws = _workspace(lib.gt_sparse_attn_bwd_workspace_size(ctypes.byref(plan.c), H, d, dt), Q.device)
    _check(lib.gt_sparse_attn_bwd(ctypes.byref(plan.c), H, d, dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(dO), _ptr(LSE),
                                  scale, _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(ws), ws.numel(), _stream(Q.device)),
           "gt_sparse_attn_bwd")
    return dQ, dK, dV


def sparse_attn_bwd_rows(plan: Plan, Q, K, V, dO, LSE, scale: float | None = None):
    """(dQ, Dstat) - the row-owned half of the backward."""
    lib = load_library()
    _check_feats(plan.n, Q, K, V, dO)
    n, H, d = Q.shape
    _need(LSE.dtype == torch.float32 and LSE.shape == (n, H) and LSE.is_contiguous(), "LSE must be fp32 [n, H]")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dt = _dtype_code(Q)
    dQ = torch.empty_like(Q)
    Dstat = torch.empty((n, H), dtype=torch.float32, device=Q.device)
    ws = _workspace(lib.gt_sparse_attn_bwd_rows_workspace_size(ctypes.byref(plan.c), H, d, dt), Q.device)
    _check(lib.gt_sparse_attn_bwd_rows(ctypes.byref(plan.c), H, d, dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(dO),
                                       _ptr(LSE), scale, _ptr(dQ), _ptr(Dstat), _ptr(ws), ws.numel(),
                                       _stream(Q.device)), "gt_sparse_attn_bwd_rows")
    return dQ, Dstat


def sparse_attn_bwd_cols(plan: Plan, Q, K, V, dO, LSE, Dstat, scale: float | None = None):
    """(dK, dV) - the column-owned half of the backward."""
    lib = load_library()
    _check_feats(plan.n, Q, K, V, dO)
    n, H, d = Q.shape
    _need(LSE.dtype == torch.float32 and LSE.shape == (n, H) and LSE.is_contiguous(), "LSE must be fp32 [n, H]")
    _need(Dstat.dtype == torch.float32 and Dstat.shape == (n, H) and Dstat.is_contiguous(), "Dstat must be fp32 [n, H]")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dt = _dtype_code(Q)
    dK, dV = torch.empty_like(K), torch.empty_like(V)
    ws = _workspace(lib.gt_sparse_attn_bwd_cols_workspace_size(ctypes.byref(plan.c), H, d, dt), Q.device)
    _check(lib.gt_sparse_attn_bwd_cols(ctypes.byref(plan.c), H, d, dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(dO), _ptr(LSE),
                                       _ptr(Dstat), scale, _ptr(dK), _ptr(dV), _ptr(ws), ws.numel(),
                                       _stream(Q.device)), "gt_sparse_attn_bwd_cols")
    return dK, dV


def gather_probe(plan: Plan, A: torch.Tensor, B: torch.Tensor, sink: torch.Tensor | None = None) -> torch.Tensor:
    """Measurement only: the forward's partner-row gathers of A and B over the plan, no arithmetic."""
    lib = load_library()
    _check_feats(plan.n, A, B)
    n, H, d = A.shape
    sink = torch.zeros(1, dtype=torch.int32, device=A.device) if sink is None else sink
    _check(lib.gt_gather_probe(ctypes.byref(plan.c), H, d, _dtype_code(A), _ptr(A), _ptr(B), _ptr(sink),
                               _stream(A.device)), "gt_gather_probe")
    return sink


def edge_map(plan: Plan) -> torch.Tensor:
    """csc_pos[c]: the input-CSR position of the c-th entry of the plan's transpose (sp_row)."""
    lib = load_library()
    dev = plan.arrays["sp_rowptr"].device
    out = torch.empty(plan.nnz_sparse, dtype=torch.int32, device=dev)
    ws = _workspace(lib.gt_edge_map_workspace_size(ctypes.byref(plan.c)), dev)
    _check(lib.gt_edge_map(ctypes.byref(plan.c), _ptr(out), _ptr(ws), ws.numel(), _stream(dev)), "gt_edge_map")
    return out


def _check_bias(plan: Plan, bias: torch.Tensor, H: int):
    _need(bias.dtype == torch.float32 and bias.shape == (plan.nnz, H) and bias.is_contiguous()
          and bias.is_cuda, "bias must be a contiguous fp32 GPU tensor [nnz, H] in the input CSR's order")


def sparse_attn_fwd_bias(plan: Plan, Q, K, V, bias, scale: float | None = None):
    """(O, LSE) with the per-edge additive bias (the input CSR's edge order, fp32 [nnz, H])."""
    lib = load_library()
    _check_feats(plan.n, Q, K, V)
    n, H, d = Q.shape
    _check_bias(plan, bias, H)
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dt = _dtype_code(Q)
    O = torch.empty_like(Q)
    LSE = torch.empty((n, H), dtype=torch.float32, device=Q.device)
    ws = _workspace(lib.gt_sparse_attn_fwd_bias_workspace_size(ctypes.byref(plan.c), H, d, dt), Q.device)
    _check(lib.gt_sparse_attn_fwd_bias(ctypes.byref(plan.c), H, d, dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(bias), scale,
                                       _ptr(O), _ptr(LSE), _ptr(ws), ws.numel(), _stream(Q.device)),
           "gt_sparse_attn_fwd_bias")
    return O, LSE


def sparse_attn_bwd_bias(plan: Plan, csc_pos, Q, K, V, bias, dO, LSE, scale: float | None = None):
    """(dQ, dK, dV, dbias) with the per-edge additive bias; csc_pos from edge_map(plan)."""
    lib = load_library()
    _check_feats(plan.n, Q, K, V, dO)
    n, H, d = Q.shape
    _check_bias(plan, bias, H)
    _need(csc_pos.dtype == torch.int32 and csc_pos.numel() == plan.nnz_sparse, "csc_pos must be int32[nnz_sparse]")
    _need(LSE.dtype == torch.float32 and LSE.shape == (n, H) and LSE.is_contiguous(), "LSE must be fp32 [n, H]")
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dt = _dtype_code(Q)
    dQ, dK, dV = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
    dB = torch.empty_like(bias)
    ws = _workspace(lib.gt_sparse_attn_bwd_bias_workspace_size(ctypes.byref(plan.c), H, d, dt), Q.device)
    _check(lib.gt_sparse_attn_bwd_bias(ctypes.byref(plan.c), _ptr(csc_pos), H, d, dt, _ptr(Q), _ptr(K), _ptr(V),
                                       _ptr(bias), _ptr(dO), _ptr(LSE), scale, _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(dB),
                                       _ptr(ws), ws.numel(), _stream(Q.device)), "gt_sparse_attn_bwd_bias")
    return dQ, dK, dV, dB


def dense_attn_fwd(Q: torch.Tensor, K: torch.Tensor, V: torch.Tensor, scale: float | None = None):
    """(O, LSE) of full softmax attention over all n nodes."""
    lib = load_library()
    _check_feats(Q.shape[0], Q, K, V)
    n, H, d = Q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    O = torch.empty_like(Q)
    LSE = torch.empty((n, H), dtype=torch.float32, device=Q.device)
    _check(lib.gt_dense_attn_fwd(n, H, d, _dtype_code(Q), _ptr(Q), _ptr(K), _ptr(V), scale, _ptr(O), _ptr(LSE),
                                 _stream(Q.device)), "gt_dense_attn_fwd")
    return O, LSE


def dense_attn_bwd(Q, K, V, O, dO, LSE, scale: float | None = None):
    """(dQ, dK, dV) of full softmax attention."""
    lib = load_library()
    _check_feats(Q.shape[0], Q, K, V, O, dO)
    n, H, d = Q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dt = _dtype_code(Q)
    dQ, dK, dV = torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V)
    ws = _workspace(lib.gt_dense_attn_bwd_workspace_size(n, H, d, dt), Q.device)
    _check(lib.gt_dense_attn_bwd(n, H, d, dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(dO), _ptr(LSE), scale,
                                 _ptr(dQ), _ptr(dK), _ptr(dV), _ptr(ws), ws.numel(), _stream(Q.device)),
           "gt_dense_attn_bwd")
    return dQ, dK, dV


def dense_attn_bwd_noalloc(Q, K, V, O, dO, LSE, scale: float | None = None, out=None):
    """(dQ, dK, dV) of full softmax attention through the entry point that allocates nothing: its scratch is the
    library's own device array (n * H <= 16,777,216).  ``out``: optional (dQ, dK, dV) to write into."""
    lib = load_library()
    _check_feats(Q.shape[0], Q, K, V, O, dO)
    n, H, d = Q.shape
    scale = 1.0 / math.sqrt(d) if scale is None else float(scale)
    dt = _dtype_code(Q)
    dQ, dK, dV = out if out is not None else (torch.empty_like(Q), torch.empty_like(K), torch.empty_like(V))
    _check(lib.gt_dense_attn_bwd_noalloc(n, H, d, dt, _ptr(Q), _ptr(K), _ptr(V), _ptr(O), _ptr(dO), _ptr(LSE),
                                         scale, _ptr(dQ), _ptr(dK), _ptr(dV), _stream(Q.device)),
           "gt_dense_attn_bwd_noalloc")
    return dQ, dK, dV
