"""GPU integer stages vs the oracle, bit for bit: CSR validation, cluster
reordering (§3.3), relabelling, tile plan (§3.4)."""

import sys

import numpy as np
import pytest
import torch

from oracle import plan as OP
from oracle import reorder as OR
from synth import csr_from_pairs, make_workload
from tests.helpers import dev_csr

pytestmark = pytest.mark.gpu


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def small_graphs():
    rng = np.random.default_rng(7)
    out = []
    out.append(("single", *csr_from_pairs(1, [], [])))
    out.append(("empty_rows", *csr_from_pairs(130, [0, 5, 9, 129], [1, 6, 120, 3], symmetric=False, self_loops=False)))
    m = rng.random((257, 257)) < 0.05
    u, v = np.nonzero(m)
    out.append(("random_directed_257", *csr_from_pairs(257, u, v, symmetric=False, self_loops=True)))
    # a star whose center has > 4096 neighbours (workspace count table) and a 100-leaf star (LDS table)
    n = 6000
    u = np.concatenate([np.zeros(5000, np.int64), np.full(100, 5500)])
    v = np.concatenate([np.arange(1, 5001), np.arange(5401, 5501)])
    u2, v2 = np.nonzero(np.random.default_rng(3).random((n, 8)) < 0.5)
    out.append(("hubs_6000", *csr_from_pairs(n, np.concatenate([u, u2 % n]),
                                             np.concatenate([v, (u2 * 7 + v2 * 131) % n]))))
    # several rows above 4096 entries at once (each spread over the whole grid), of different table sizes
    n = 30000
    hubs = [(0, 4500), (7, 9000), (29999, 20000)]
    u = np.concatenate([np.full(d, h, np.int64) for h, d in hubs])
    v = np.concatenate([(np.arange(1, d + 1) * 13 + h) % n for h, d in hubs])
    u2 = rng.integers(0, n, 60000)
    v2 = (u2 + rng.integers(1, 50, 60000)) % n
    out.append(("three_hubs_30000", *csr_from_pairs(n, np.concatenate([u, u2]), np.concatenate([v, v2]))))
    # b1 at 10%: the global token's row (about 98,000 entries) takes the whole-grid path (rows above 2^16)
    for name, sc in (("c1", 1.0), ("c2", 0.05), ("c3", 0.02), ("c4", 0.02), ("c5", 0.1), ("b1", 0.02), ("b1", 0.1)):
        g = make_workload(name, sc).graph
        out.append((f"{name}@{sc}", g.rowptr, g.col))
    return out


GRAPHS = small_graphs()


@pytest.mark.parametrize("name,rowptr,col", GRAPHS, ids=[g[0] for g in GRAPHS])
def test_reorder_bit_exact(gt, name, rowptr, col):
    say("reorder", name, len(rowptr) - 1, len(col))
    rp, cl = dev_csr(rowptr, col)
    perm, iperm, labels, sweeps = gt.reorder(rp, cl, iters=20, seed=5, want_sweeps=True)
    lab_ref, done = OR.lp_labels(rowptr, col, iters=20, seed=5)
    perm_ref, iperm_ref = OR.cluster_order(rowptr, col, lab_ref)
    np.testing.assert_array_equal(labels.cpu().numpy(), lab_ref)
    np.testing.assert_array_equal(perm.cpu().numpy(), perm_ref)
    np.testing.assert_array_equal(iperm.cpu().numpy(), iperm_ref)
    assert sweeps == done


def test_reorder_concurrent_calls(gt):
    # two host threads reordering at once, each on a stream of its own (default priority), both get the oracle's
    # order, call after call (the library keeps nothing between or across calls)
    import threading

    cases = [g for g in GRAPHS if g[0] in ("three_hubs_30000", "b1@0.1")]
    refs = {}
    for name, rowptr, col in cases:
        lab_ref, _ = OR.lp_labels(rowptr, col, iters=20, seed=5)
        refs[name] = OR.cluster_order(rowptr, col, lab_ref)
    dev_graphs = {name: dev_csr(rowptr, col) for name, rowptr, col in cases}
    torch.cuda.synchronize()
    results, errors = {}, []

    def work(name):
        try:
            s = torch.cuda.Stream()
            with torch.cuda.stream(s):
                rp, cl = dev_graphs[name]
                for _ in range(3):
                    perm, iperm, _lab = gt.reorder(rp, cl, iters=20, seed=5)
                    results.setdefault(name, []).append((perm.cpu().numpy(), iperm.cpu().numpy()))
        except Exception as e:  # reported below, in the test's own thread
            errors.append(e)

    say("reorder concurrent", ", ".join(dev_graphs))
    threads = [threading.Thread(target=work, args=(name,)) for name in dev_graphs]
    for t in threads:
        t.start()
    for t in threads:
        t.join()
    assert not errors, errors
    for name, (perm_ref, iperm_ref) in refs.items():
        assert len(results[name]) == 3
        for perm, iperm in results[name]:
            np.testing.assert_array_equal(perm, perm_ref)
            np.testing.assert_array_equal(iperm, iperm_ref)


def mixed_classes_graph():
    # most entries in rows of more than 64 (so a sweep's classes run on the side streams): 4,000 nodes with
    # about 120 neighbours among themselves, 20 rows of about 1,500 and two of 6,000, the rest short rows
    rng = np.random.default_rng(23)
    n = 20000
    u = [np.repeat(np.arange(4000), 60), np.repeat(np.arange(4000, 4020), 1500), np.repeat([4020, 4021], 6000)]
    v = [rng.integers(0, 4000, 240000), rng.integers(0, n, 30000), rng.integers(0, n, 12000)]
    short = np.arange(4022, n)
    u.append(np.repeat(short, 2))
    v.append(rng.integers(4022, n, 2 * len(short)))
    return csr_from_pairs(n, np.concatenate(u), np.concatenate(v))


@pytest.mark.parametrize("name", ["mixed_classes_20000", "hubs_6000", "c3@0.02", "b1@0.1"])
def test_reorder_side_streams_same_result(gt, name):
    # the sweeps spread over zero, one or two side streams give one result, call after call with the same
    # streams and events; on the first graph the rows of more than 64 entries hold most entries, so the side
    # streams are used (the others stay on one stream), and it is checked against the oracle too
    if name == "mixed_classes_20000":
        rowptr, col = mixed_classes_graph()
        deg = np.diff(rowptr)
        assert 4 * deg[deg > 64].sum() >= len(col)
    else:
        rowptr, col = next((g[1], g[2]) for g in GRAPHS if g[0] == name)
    rp, cl = dev_csr(rowptr, col)
    ref = [x.cpu().numpy() for x in gt.reorder(rp, cl, iters=20, seed=5, n_side=0)]
    if name == "mixed_classes_20000":
        lab_ref, _ = OR.lp_labels(rowptr, col, iters=20, seed=5)
        perm_ref, _ = OR.cluster_order(rowptr, col, lab_ref)
        np.testing.assert_array_equal(ref[2], lab_ref)
        np.testing.assert_array_equal(ref[0], perm_ref)
    for n_side in (1, 2, 1, 2):
        say("reorder side streams", name, n_side)
        got = gt.reorder(rp, cl, iters=20, seed=5, n_side=n_side)
        for a, b in zip(got, ref):
            np.testing.assert_array_equal(a.cpu().numpy(), b)


@pytest.mark.parametrize("name,rowptr,col", GRAPHS, ids=[g[0] for g in GRAPHS])
def test_permute_bit_exact(gt, name, rowptr, col):
    say("permute", name)
    n = len(rowptr) - 1
    perm = np.random.default_rng(11).permutation(n).astype(np.int32)
    iperm = np.empty(n, np.int32)
    iperm[perm] = np.arange(n)
    rp, cl = dev_csr(rowptr, col)
    rp2, cl2 = gt.permute_csr(rp, cl, torch.from_numpy(perm).cuda(), torch.from_numpy(iperm).cuda())
    ref_rp, ref_cl = OP.permute_csr(rowptr, col, perm, iperm)
    np.testing.assert_array_equal(rp2.cpu().numpy(), ref_rp)
    np.testing.assert_array_equal(cl2.cpu().numpy(), ref_cl)


def test_permute_every_row_size(gt):
    # rows of 65 to 512 entries are sorted by one wavefront (2, 4 or 8 entries a lane), 513 to 2,048 and longer
    # ones by the keyed radix sort: star rows at each boundary of those classes, plus short rows; with and
    # without the edge map, against the oracle (the map: each new edge's old position holds the same edge)
    sizes = [65, 100, 128, 129, 200, 256, 257, 400, 511, 512, 513, 1000, 2048, 2049, 5000]
    n = 12000
    rng = np.random.default_rng(31)
    u = [np.full(d, 100 + 37 * k, np.int64) for k, d in enumerate(sizes)]
    v = [rng.choice(n, d, replace=False) for d in sizes]
    u.append(rng.integers(1000, n, 3 * n))  # short rows, away from the stars' centres
    v.append(rng.integers(0, n, 3 * n))
    rowptr, col = csr_from_pairs(n, np.concatenate(u), np.concatenate(v), symmetric=False, self_loops=False)
    deg = np.diff(rowptr)
    assert all((deg == d).any() for d in sizes)
    perm = np.random.default_rng(12).permutation(n).astype(np.int32)
    iperm = np.empty(n, np.int32)
    iperm[perm] = np.arange(n)
    rp, cl = dev_csr(rowptr, col)
    pt, it = torch.from_numpy(perm).cuda(), torch.from_numpy(iperm).cuda()
    ref_rp, ref_cl = OP.permute_csr(rowptr, col, perm, iperm)
    say("permute row sizes", n, len(col))
    rp2, cl2 = gt.permute_csr(rp, cl, pt, it)
    np.testing.assert_array_equal(rp2.cpu().numpy(), ref_rp)
    np.testing.assert_array_equal(cl2.cpu().numpy(), ref_cl)
    rp3, cl3, src = gt.permute_csr_edges(rp, cl, pt, it)
    np.testing.assert_array_equal(rp3.cpu().numpy(), ref_rp)
    np.testing.assert_array_equal(cl3.cpu().numpy(), ref_cl)
    src = src.cpu().numpy().astype(np.int64)
    rows_old = np.repeat(np.arange(n), deg)
    new_rows = np.repeat(np.arange(n), np.diff(ref_rp))
    np.testing.assert_array_equal(iperm[rows_old[src]], new_rows)
    np.testing.assert_array_equal(iperm[col[src]], ref_cl)


def compare_plan(got: dict, ref: dict):
    for key in ("tile_rowptr", "tile_col", "tile_nnz", "sp_rowptr", "sp_col", "sp_colptr", "sp_row", "tileT_ptr",
                "tileT_idx"):
        np.testing.assert_array_equal(got[key], ref[key], err_msg=key)
    np.testing.assert_array_equal(got["tile_mask"].view(np.uint32), ref["tile_mask"], err_msg="tile_mask")
    deg = np.diff(ref["sp_rowptr"])
    np.testing.assert_array_equal(got["long_rows"], np.flatnonzero(deg > 256))
    cdeg = np.diff(ref["sp_colptr"])
    np.testing.assert_array_equal(got["long_cols"], np.flatnonzero(cdeg > 256))


@pytest.mark.parametrize("name,rowptr,col", GRAPHS, ids=[g[0] for g in GRAPHS])
@pytest.mark.parametrize("T", [64, 128])
def test_tiles_bit_exact(gt, name, rowptr, col, T):
    rp, cl = dev_csr(rowptr, col)
    n = len(rowptr) - 1
    for tau in (0, 5000, 10000, 50000, 200000, 1_000_001):
        say("tiles", name, T, tau)
        plan = gt.build_tiles(rp, cl, T, tau)
        ref = OP.build_tiles(rowptr, col, T, tau)
        assert plan.n_dense == len(ref["tile_col"]) and plan.nnz_sparse == len(ref["sp_col"])
        compare_plan(plan.to_numpy(), ref)
    assert n >= 1


@pytest.mark.parametrize("tile_rows,small", [(2048, True), (4096, False)])
def test_tile_transpose_both_paths(gt, tile_rows, small):
    # plans of up to 8192 dense tiles group their tiles by column in one workgroup, larger ones by radix sort.
    # Three tiles per tile row at threshold 0 (every tile with an edge is dense): the diagonal, ten tile
    # columns to the right, and one of the first seven columns, so those seven columns hold hundreds of tiles
    # each.  Checked against the definitions: the dense tiles are the occupied (I, J) in (I, J) order, and
    # the transpose is their stable order by J.
    T = 64
    n = T * tile_rows
    i = np.arange(n, dtype=np.int64)
    u = np.concatenate([i, i, i])
    v = np.concatenate([i, (i + 10 * T) % n, i % T + T * ((i // T) % 7)])
    rowptr, col = csr_from_pairs(n, u, v, symmetric=False, self_loops=False)
    say("tile transpose", tile_rows, len(col))
    rp, cl = dev_csr(rowptr, col)
    plan = gt.build_tiles(rp, cl, T, 0)
    got = plan.to_numpy()
    rows = np.repeat(np.arange(n, dtype=np.int64), np.diff(rowptr))
    occupied = np.unique((rows // T) * tile_rows + col.astype(np.int64) // T)
    assert (plan.n_dense <= 8192) == small
    np.testing.assert_array_equal(got["tile_col"], occupied % tile_rows)
    np.testing.assert_array_equal(got["tile_rowptr"],
                                  np.concatenate([[0], np.cumsum(np.bincount(occupied // tile_rows,
                                                                             minlength=tile_rows))]))
    np.testing.assert_array_equal(got["tileT_idx"], np.argsort(occupied % tile_rows, kind="stable"))
    np.testing.assert_array_equal(got["tileT_ptr"],
                                  np.concatenate([[0], np.cumsum(np.bincount(occupied % tile_rows,
                                                                             minlength=tile_rows))]))


@pytest.mark.parametrize("name", ["hubs_6000", "three_hubs_30000", "c3@0.02", "b1@0.1"])
def test_tiles_counts_taken_or_recounted(gt, name):
    # gt_build_tiles takes gt_tiles_count's counts from the shared workspace only while they are unchanged
    # there: a workspace of its own, or one overwritten in between, makes it count again; every way gives the
    # oracle's plan
    rowptr, col = next((g[1], g[2]) for g in GRAPHS if g[0] == name)
    rp, cl = dev_csr(rowptr, col)
    for T, tau in ((64, 10000), (128, 50000)):
        ref = OP.build_tiles(rowptr, col, T, tau)
        ws_bytes = gt.load_library().gt_tiles_workspace_size(len(rowptr) - 1, len(col), T)
        ways = {
            "shared": {},
            "own workspace": {"build_ws": torch.full((max(ws_bytes, 256),), 0x5A, dtype=torch.uint8,
                                                     device=rp.device)},
            "overwritten": {"between": lambda ws: ws.fill_(0xA5)},
            "one byte changed": {"between": lambda ws: ws[ws.numel() // 3].add_(1)},
            # the count record's last word (whether a row exceeds 2,048 entries), flipped: the record check
            # (the flag is folded into the stored checksum) must send the build back to counting
            "record flag flipped": {"between": lambda ws: ws[256 + 7 * 8].bitwise_xor_(1)},
        }
        for way, kw in ways.items():
            say("tiles counts", name, T, tau, way)
            plan = gt.build_tiles(rp, cl, T, tau, **kw)
            compare_plan(plan.to_numpy(), ref)


def test_tiles_threshold_equality(gt):
    # a 64x64 tile with exactly 64 edges (density 1/64 = 15625 ppm): dense at 15625, sparse at 15626
    u = np.arange(64)
    v = (np.arange(64) * 5) % 64
    rowptr, col = csr_from_pairs(64, u, v, symmetric=False, self_loops=False)
    rp, cl = dev_csr(rowptr, col)
    assert gt.build_tiles(rp, cl, 64, 15625).n_dense == 1
    assert gt.build_tiles(rp, cl, 64, 15626).n_dense == 0


def test_full_size_tile_plan_c4(gt):
    w = make_workload("c4")
    g = w.graph
    say("full-size c4 tiles", g.n, g.nnz)
    perm = np.lexsort((np.arange(g.n), g.block))
    iperm = np.empty(g.n, np.int64)
    iperm[perm] = np.arange(g.n)
    rp_h, cl_h = OP.permute_csr(g.rowptr, g.col, perm, iperm)
    rp, cl = dev_csr(rp_h, cl_h)
    plan = gt.build_tiles(rp, cl, 128, 10000)
    ref = OP.build_tiles(rp_h, cl_h, 128, 10000)
    compare_plan(plan.to_numpy(), ref)


def test_validation_errors(gt):
    good_rp = np.array([0, 2, 3, 3], np.int64)
    cases = [
        (np.array([1, 0, 2], np.int32), gt.GT_ERR_UNSORTED),
        (np.array([1, 1, 2], np.int32), gt.GT_ERR_DUPLICATE),
        (np.array([0, 1, 7], np.int32), gt.GT_ERR_OUT_OF_RANGE),
    ]
    for col, code in cases:
        rp, cl = dev_csr(good_rp, col)
        with pytest.raises(gt.GtError) as e:
            gt.validate_csr(rp, cl)
        assert e.value.status == code
        with pytest.raises(gt.GtError) as e:
            gt.build_tiles(rp, cl, 64, 100)
        assert e.value.status == code
        with pytest.raises(gt.GtError) as e:
            gt.reorder(rp, cl)
        assert e.value.status == code
    rp, cl = dev_csr(np.array([0, 2, 1, 3], np.int64), np.array([0, 1, 2], np.int32))
    with pytest.raises(gt.GtError) as e:
        gt.validate_csr(rp, cl)
    assert e.value.status == gt.GT_ERR_UNSORTED
    rp, cl = dev_csr(good_rp, np.array([0, 1, 2], np.int32))
    gt.validate_csr(rp, cl)


def test_validation_errors_in_long_rows(gt):
    # rows above 2,048 entries are checked chunk by chunk over the grid: plant each error at a chunk boundary
    # (entries 2047/2048 of the CSR) or inside a long row that starts in the middle of a chunk
    n = 6000
    deg = np.zeros(n, np.int64)
    deg[0], deg[1], deg[2] = 5000, 7, 3000
    rowptr = np.concatenate([[0], np.cumsum(deg)])
    good = np.concatenate([np.arange(5000), np.arange(7) * 3, np.arange(3000) * 2]).astype(np.int32)
    rp, cl = dev_csr(rowptr, good)
    gt.validate_csr(rp, cl)
    b = int(rowptr[2])  # row 2 starts at entry 5007, inside the third chunk
    cases = []
    bad = good.copy(); bad[2047], bad[2048] = bad[2048], bad[2047]; cases.append((bad, gt.GT_ERR_UNSORTED))
    bad = good.copy(); bad[2048] = bad[2047]; cases.append((bad, gt.GT_ERR_DUPLICATE))
    bad = good.copy(); bad[b + 1] = bad[b]; cases.append((bad, gt.GT_ERR_DUPLICATE))
    bad = good.copy(); bad[b + 2999] = 1; cases.append((bad, gt.GT_ERR_UNSORTED))
    bad = good.copy(); bad[4999] = n + 5; cases.append((bad, gt.GT_ERR_OUT_OF_RANGE))
    for col, code in cases:
        rp, cl = dev_csr(rowptr, col)
        with pytest.raises(gt.GtError) as e:
            gt.validate_csr(rp, cl)
        assert e.value.status == code


def test_gather_scatter_rows(gt):
    x = torch.randn(1000, 8, 32, device="cuda").to(torch.bfloat16)
    perm = torch.randperm(1000, device="cuda").to(torch.int32)
    y = gt.gather_rows(x, perm)
    assert torch.equal(y, x[perm.long()])
    assert torch.equal(gt.scatter_rows(y, perm), x)


def test_validation_errors_in_short_rows(gt):
    # rows of up to 256 entries are checked by one thread in batches of 8 loads: plant each error on either side
    # of a batch boundary and at the ends of rows of several lengths, next to rows that are valid
    lens = [1, 7, 8, 9, 15, 16, 17, 100, 256]
    rp = np.concatenate([[0], np.cumsum(lens)]).astype(np.int64)
    n = 300
    good = np.concatenate([np.arange(L, dtype=np.int32) * 1 + (i % 5) for i, L in enumerate(lens)])
    rp_n = np.concatenate([rp, np.full(n - len(lens), rp[-1])]).astype(np.int64)  # n rows, the last ones empty
    gt.validate_csr(*dev_csr(rp_n, good))
    for r, L in enumerate(lens):
        a = int(rp[r])
        for k in sorted({0, 6, 7, 8, 9, 15, 16, L - 1}):
            if k >= L:
                continue
            cases = [(n + 3, gt.GT_ERR_OUT_OF_RANGE), (-1, gt.GT_ERR_OUT_OF_RANGE)]
            if k > 0:
                cases.append((int(good[a + k - 1]), gt.GT_ERR_DUPLICATE))
                cases.append((int(good[a + k - 1]) - 1, gt.GT_ERR_UNSORTED))
            for val, code in cases:
                bad = good.copy()
                bad[a + k] = val
                if code == gt.GT_ERR_UNSORTED and val < 0:
                    continue
                say("validate short", L, k, val)
                rp_d, cl_d = dev_csr(rp_n, bad)
                with pytest.raises(gt.GtError) as e:
                    gt.validate_csr(rp_d, cl_d)
                assert e.value.status == code, (L, k, val)
