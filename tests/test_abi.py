"""The C-ABI library loads, exports every symbol that include/gt.h declares, and
rejects bad arguments on the host before touching any device (no GPU needed)."""

import ctypes
import os
import re

import pytest

from paper_2407_14106_amd import gt

HEADER = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "include", "gt.h")
FAKE = ctypes.c_void_p(0x1000)  # never dereferenced: every call below fails its host-side checks first


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(gt.LIB_PATH):
        from paper_2407_14106_amd import build

        build.build()
    return gt.load_library()


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(gt_[a-z0-9_]+)\s*\(", text)))


def test_every_declared_symbol_is_exported(lib):
    names = declared_functions()
    assert "gt_sparse_attn_fwd" in names and "gt_reorder" in names and len(names) >= 20
    for name in names:
        assert hasattr(lib, name), name
    assert set(names) == set(gt.SIGNATURES), "binding signatures out of sync with the header"


def test_library_creates_no_runtime_objects(lib):
    # The library keeps no state between calls and owns no device memory: it imports no HIP call that creates
    # streams or events or that allocates or frees memory (the symbol table of the built library).
    import subprocess

    out = subprocess.run(["nm", "-D", "--undefined-only", gt.LIB_PATH], capture_output=True, text=True, check=True)
    imported = {line.split()[-1].split("@")[0] for line in out.stdout.splitlines() if line.strip()}
    hip = {name for name in imported if name.startswith("hip")}
    forbidden = re.compile(r"^hip(Stream|Event|Graph)Create|^hip(Ext)?Malloc|^hipFree|^hipHost(Malloc|Register)"
                           r"|^hipMemset|^hipMallocManaged")
    assert "hipLaunchKernel" in hip
    assert not sorted(n for n in hip if forbidden.search(n)), hip


def test_version_and_status_strings(lib):
    assert lib.gt_abi_version() == 2
    assert lib.gt_status_string(gt.GT_OK) == b"ok"
    assert lib.gt_status_string(gt.GT_ERR_WORKSPACE) == b"workspace too small"
    assert lib.gt_status_string(-99) == b"unknown status"


def test_struct_layout_matches_header():
    assert ctypes.sizeof(gt.GtTiles) == 8 * 6 + 4 * 2 + 8 * 14


def test_workspace_queries_are_host_only(lib):
    assert lib.gt_reorder_workspace_size(1000, 5000) > lib.gt_reorder_workspace_size(10, 50) > 0
    assert lib.gt_permute_workspace_size(1000, 5000) > 0
    assert lib.gt_tiles_workspace_size(1000, 5000, 128) > 0
    c = gt.GtTiles(n=1000, T=128, n_row_tiles=8, n_dense=0)
    assert lib.gt_sparse_attn_fwd_workspace_size(ctypes.byref(c), 8, 32, gt.GT_BF16) > 0
    c.n_dense = 5
    with_tiles = lib.gt_sparse_attn_fwd_workspace_size(ctypes.byref(c), 8, 32, gt.GT_BF16)
    assert with_tiles >= 1000 * 8 * 34 * 4
    assert lib.gt_sparse_attn_fwd_workspace_size(ctypes.byref(c), 8, 48, gt.GT_BF16) == 0  # unsupported d


def test_argument_errors_without_device(lib):
    stream = None
    # null plan
    assert lib.gt_sparse_attn_fwd(None, 8, 32, gt.GT_BF16, FAKE, FAKE, FAKE, 1.0, FAKE, FAKE, FAKE, 1 << 30,
                                  stream) == gt.GT_ERR_INVALID_ARG
    c = gt.GtTiles(n=100, T=128, n_row_tiles=1)
    for name in ("tile_rowptr", "sp_rowptr", "sp_colptr", "tileT_ptr"):
        setattr(c, name, 0x1000)
    # unsupported head width and head count
    assert lib.gt_sparse_attn_fwd(ctypes.byref(c), 8, 48, gt.GT_BF16, FAKE, FAKE, FAKE, 1.0, FAKE, FAKE, FAKE,
                                  1 << 30, stream) == gt.GT_ERR_UNSUPPORTED
    assert lib.gt_sparse_attn_bwd(ctypes.byref(c), 3, 32, gt.GT_F32, FAKE, FAKE, FAKE, FAKE, FAKE, 1.0, FAKE,
                                  FAKE, FAKE, FAKE, 1 << 30, stream) == gt.GT_ERR_UNSUPPORTED
    # workspace too small
    assert lib.gt_sparse_attn_fwd(ctypes.byref(c), 8, 32, gt.GT_BF16, FAKE, FAKE, FAKE, 1.0, FAKE, FAKE, FAKE, 0,
                                  stream) == gt.GT_ERR_WORKSPACE
    # null feature pointer
    assert lib.gt_sparse_attn_fwd(ctypes.byref(c), 8, 32, gt.GT_BF16, None, FAKE, FAKE, 1.0, FAKE, FAKE, FAKE,
                                  1 << 30, stream) == gt.GT_ERR_INVALID_ARG
    assert b"null" in lib.gt_last_error()
    # tiles: unsupported T, too many tile rows, workspace
    t = gt.GtTiles()
    assert lib.gt_tiles_count(1000, 10, FAKE, FAKE, 96, 100, ctypes.byref(t), FAKE, 1 << 30,
                              stream) == gt.GT_ERR_UNSUPPORTED
    assert lib.gt_tiles_count(64 * 20000, 10, FAKE, FAKE, 64, 100, ctypes.byref(t), FAKE, 1 << 40,
                              stream) == gt.GT_ERR_UNSUPPORTED
    assert lib.gt_tiles_count(1000, 10, FAKE, FAKE, 64, 100, ctypes.byref(t), FAKE, 16, stream) == gt.GT_ERR_WORKSPACE
    # reorder / permute / validate
    assert lib.gt_reorder(-1, 0, FAKE, FAKE, 10, 0, FAKE, FAKE, None, None, FAKE, 1 << 30,
                          stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_reorder(100, 10, FAKE, FAKE, 5000, 0, FAKE, FAKE, None, None, FAKE, 1 << 30,
                          stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_reorder(100, 10, FAKE, FAKE, 10, 0, FAKE, FAKE, None, None, FAKE, 8, stream) == gt.GT_ERR_WORKSPACE
    # side streams and events: at most two streams, given, non-null, distinct and not the call's own stream;
    # one event more, non-null and distinct (host checks, before any device query)
    two = (ctypes.c_void_p * 2)(FAKE, FAKE)
    s2 = (ctypes.c_void_p * 2)(0x1000, 0x2000)
    e3 = (ctypes.c_void_p * 3)(0x3000, 0x4000, 0x5000)
    e3_null = (ctypes.c_void_p * 3)(0x3000, 0, 0x5000)
    e3_rep = (ctypes.c_void_p * 3)(0x3000, 0x4000, 0x3000)
    for side, events, n_side in ((None, e3, 1), (s2, None, 1), (s2, e3, 3), (s2, e3, -1), (two, e3, 2),
                                 (s2, e3_null, 2), (s2, e3_rep, 2)):
        assert lib.gt_reorder_streams(100, 10, FAKE, FAKE, 10, 0, FAKE, FAKE, None, None, FAKE, 1 << 30, stream,
                                      side, events, n_side) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_reorder_streams(100, 10, FAKE, FAKE, 10, 0, FAKE, FAKE, None, None, FAKE, 8, stream, s2, e3,
                                  1) == gt.GT_ERR_WORKSPACE
    assert lib.gt_permute_csr(100, 10, None, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, 1 << 30,
                              stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_validate_csr(10, 10, FAKE, FAKE, FAKE, 0, stream) == gt.GT_ERR_WORKSPACE
    assert lib.gt_gather_rows(10, 6, FAKE, FAKE, FAKE, stream) == gt.GT_ERR_INVALID_ARG
    # dense layer: bad pointers / sizes
    assert lib.gt_dense_attn_fwd(100, 8, 64, gt.GT_BF16, None, FAKE, FAKE, 1.0, FAKE, FAKE,
                                 stream) == gt.GT_ERR_INVALID_ARG


def test_python_binding_rejects_cpu_tensors(lib):
    import torch

    rp = torch.zeros(5, dtype=torch.int64)
    cl = torch.zeros(0, dtype=torch.int32)
    with pytest.raises(ValueError):
        gt.build_tiles(rp, cl)


def test_extension_entry_points_reject_bad_arguments(lib):
    stream = None
    c = gt.GtTiles(n=100, T=128, n_row_tiles=1, nnz_sparse=50)
    for name in ("tile_rowptr", "sp_rowptr", "sp_colptr", "tileT_ptr", "sp_col", "sp_row"):
        setattr(c, name, 0x1000)
    ws = 1 << 30
    # bias calls: a plan with dense tiles but no edge positions is refused, a null bias too
    c.n_dense = 3
    c.tile_col = c.tile_mask = c.tileT_idx = 0x1000
    assert lib.gt_sparse_attn_fwd_bias(ctypes.byref(c), 8, 32, gt.GT_BF16, FAKE, FAKE, FAKE, FAKE, 1.0, FAKE, FAKE,
                                       FAKE, ws, stream) == gt.GT_ERR_INVALID_ARG
    assert b"sp_pos and tile_pos" in lib.gt_last_error()
    assert (lib.gt_sparse_attn_bwd_bias_workspace_size(ctypes.byref(c), 8, 32, gt.GT_BF16)
            >= lib.gt_sparse_attn_bwd_workspace_size(ctypes.byref(c), 8, 32, gt.GT_BF16) + 2 * 3 * 8 * 128 * 128 * 4)
    c.n_dense = 0
    assert lib.gt_sparse_attn_fwd_bias(ctypes.byref(c), 8, 32, gt.GT_BF16, FAKE, FAKE, FAKE, None, 1.0, FAKE, FAKE,
                                       FAKE, ws, stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_sparse_attn_bwd_bias(ctypes.byref(c), None, 8, 32, gt.GT_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                       1.0, FAKE, FAKE, FAKE, FAKE, FAKE, ws, stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_sparse_attn_bwd_bias(ctypes.byref(c), FAKE, 8, 32, gt.GT_BF16, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE,
                                       1.0, FAKE, FAKE, FAKE, None, FAKE, ws, stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_sparse_attn_fwd_bias(ctypes.byref(c), 8, 32, gt.GT_BF16, FAKE, FAKE, FAKE, FAKE, 1.0, FAKE, FAKE,
                                       FAKE, 0, stream) == gt.GT_ERR_WORKSPACE
    # edge map / probe / relabel with edge positions
    assert lib.gt_edge_map(None, FAKE, FAKE, ws, stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_edge_map(ctypes.byref(c), FAKE, FAKE, 0, stream) == gt.GT_ERR_WORKSPACE
    assert lib.gt_gather_probe(ctypes.byref(c), 8, 48, gt.GT_BF16, FAKE, FAKE, FAKE, stream) == gt.GT_ERR_UNSUPPORTED
    assert lib.gt_gather_probe(ctypes.byref(c), 8, 32, gt.GT_BF16, FAKE, None, FAKE, stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_permute_csr_edges(100, 10, FAKE, FAKE, FAKE, FAKE, FAKE, FAKE, None, FAKE, ws,
                                    stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_permute_edges_workspace_size(100, 10) > lib.gt_permute_workspace_size(100, 10)
    # interleave check
    rep = gt.GtInterleaveReport()
    assert lib.gt_interleave_check(100, 10, FAKE, FAKE, -1, ctypes.byref(rep), None, FAKE, ws,
                                   stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_interleave_check(100, 10, FAKE, FAKE, 4, None, None, FAKE, ws, stream) == gt.GT_ERR_INVALID_ARG
    assert lib.gt_interleave_check(100, 10, FAKE, FAKE, 4, ctypes.byref(rep), None, FAKE, 0,
                                   stream) == gt.GT_ERR_WORKSPACE
    assert lib.gt_interleave_workspace_size(100) > 0


def test_report_and_tuner_layouts_match_header():
    assert ctypes.sizeof(gt.GtInterleaveReport) == 8 * 4 + 4 * 6
    assert ctypes.sizeof(gt.GtAutotuner) == 8 + 8 * gt.GT_AUTOTUNER_HISTORY + 8 + 8 + 4 + 4 + 2 * 8 * gt.GT_AUTOTUNER_RUNGS
