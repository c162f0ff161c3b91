"""Pins of the lossy reformation and Auto Tuner oracle (§3.4, cluster sparsity, transfer strategy,
hyperparameter modeling): a hand-worked example, a dense-matrix brute force on tiny graphs, the threshold's
end points, and a hand-computed tuner trace."""

from fractions import Fraction

import numpy as np
import pytest

from oracle import ecr as OE
from synth import csr_from_pairs


def dense_of(rowptr, col, n):
    A = np.zeros((n, n), dtype=bool)
    A[np.repeat(np.arange(n), np.diff(rowptr)), col] = True
    return A


def brute(A, k, d_b, num, den):
    """The same definition over a dense boolean matrix, cluster by cluster and block by block."""
    n = A.shape[0]
    c = -(-n // k) if n else 1
    B = A.copy()
    for I in range(k):
        for J in range(k):
            r0, c0 = I * c, J * c
            r1, c1 = min(n, r0 + c), min(n, c0 + c)
            if r1 <= r0 or c1 <= c0:
                continue
            sub = A[r0:r1, c0:c1]
            cnt = int(sub.sum())
            if not (cnt >= 1 and cnt * den < num * sub.size):
                continue
            diag = np.zeros_like(sub)
            for i in range(r0, r1):
                if c0 <= i < c1:
                    diag[i - r0, i - c0] = True
            moved = sub & ~diag
            m = -(-int(moved.sum()) // (d_b * d_b))
            cand = []
            for a in range(-(-(r1 - r0) // d_b)):
                for b in range(-(-(c1 - c0) // d_b)):
                    cand.append((-int(moved[a * d_b:(a + 1) * d_b, b * d_b:(b + 1) * d_b].sum()), a, b))
            cand.sort()
            new = sub & diag
            for cneg, a, b in cand[:m]:
                assert cneg < 0
                new[a * d_b:(a + 1) * d_b, b * d_b:(b + 1) * d_b] = True
            B[r0:r1, c0:c1] = new
    return B


def test_hand_worked_example():
    # N = 8, k = 2 (clusters of 4), d_b = 2, threshold 1/4.  Off-diagonal cluster (0, 1) holds (0,5), (2,7),
    # (3,4): density 3/16 < 1/4, one sub-block (ceil(3/4)); its blocks (0,0), (1,1), (1,0) hold one edge each,
    # so the tie goes to (0,0): rows 0-1, columns 4-5.  Cluster (1, 0) mirrors it: rows 4-5, columns 0-1.
    # Diagonal cluster (0, 0) holds 4 self-loops + (0,1), (1,0): 6/16 is not below 1/4, kept.  Cluster (1, 1)
    # holds its 4 self-loops: 4/16 is not below 1/4 (equality), kept.
    u = [0, 2, 3, 5, 7, 4, 0, 1]
    v = [5, 7, 4, 0, 2, 3, 1, 0]
    rowptr, col = csr_from_pairs(8, np.array(u), np.array(v), symmetric=False, self_loops=True)
    rp, cl, info = OE.ecr_compact(rowptr, col, 2, 2, 1, 4)
    assert list(info["transfer"]) == [False, True, True, False]
    assert info["chosen"] == {1: [(0, 0)], 2: [(0, 0)]}
    got = sorted(zip(np.repeat(np.arange(8), np.diff(rp)).tolist(), cl.tolist()))
    want = sorted({(i, i) for i in range(8)} | {(0, 1), (1, 0)} | {(0, 4), (0, 5), (1, 4), (1, 5)}
                  | {(4, 0), (4, 1), (5, 0), (5, 1)})
    assert got == want


@pytest.mark.parametrize("seed", range(40))
def test_matches_dense_brute_force(seed):
    rng = np.random.default_rng(seed)
    n = int(rng.integers(1, 41))
    m = int(rng.integers(0, 3 * n + 1))
    u, v = rng.integers(0, n, m), rng.integers(0, n, m)
    rowptr, col = csr_from_pairs(n, u, v, symmetric=bool(seed % 2), self_loops=bool(seed % 3))
    k = int(rng.integers(1, 6))
    d_b = int(rng.integers(1, 5))
    num, den = int(rng.integers(0, 9)), int(rng.integers(1, 9))
    rp, cl, _ = OE.ecr_compact(rowptr, col, k, d_b, num, den)
    assert np.array_equal(dense_of(rp, cl, n), brute(dense_of(rowptr, col, n), k, d_b, num, den))
    assert np.all(np.diff(rp) >= 0) and len(cl) == rp[-1] <= OE.max_nnz(len(col), k, d_b)


def test_threshold_end_points_and_invariants():
    rng = np.random.default_rng(5)
    n = 300
    u, v = rng.integers(0, n, 900), rng.integers(0, n, 900)
    rowptr, col = csr_from_pairs(n, u, v, symmetric=True, self_loops=True)
    # threshold 0: nothing is below it, E' = E
    rp, cl, info = OE.ecr_compact(rowptr, col, 8, 4, 0, 1)
    assert not info["transfer"].any() and np.array_equal(rp, rowptr) and np.array_equal(cl, col)
    # threshold 1: every non-full cluster is transferred; self-loops survive; each transferred cluster holds its
    # self-loops plus exactly m whole sub-blocks (blocks never overlap)
    rp, cl, info = OE.ecr_compact(rowptr, col, 8, 4, 1, 1)
    assert info["transfer"].all()
    rows = np.repeat(np.arange(n), np.diff(rp))
    assert np.all(np.isin(np.arange(n), rows[rows == cl]))
    c = info["c"]
    A = dense_of(rp, cl, n)
    for x, blocks in info["chosen"].items():
        I, J = divmod(x, 8)
        assert len(blocks) == info["m"][x]
        sub = A[I * c:(I + 1) * c, J * c:(J + 1) * c]
        cells = 0
        for a, b in blocks:
            blk = sub[a * 4:(a + 1) * 4, b * 4:(b + 1) * 4]
            assert blk.all()
            cells += blk.size
        if I != J:
            assert sub.sum() == cells
    # the indolent rule (beta_G = nnz / N^2) leaves the dense diagonal clusters alone
    rp, cl, info = OE.ecr_compact(rowptr, col, 8, 4, len(col), n * n)
    diag = [x for x in range(64) if x // 8 == x % 8]
    assert not info["transfer"][diag].any()


def test_ladder_values_and_cap():
    assert OE.ladder(30, 100) == [0, Fraction(3, 1000), Fraction(9, 2000), Fraction(15, 1000), Fraction(21, 1000),
                                  Fraction(3, 100), 1]
    assert OE.ladder(5000, 100)[3:] == [1, 1, 1, 1]  # 5 bG = 2.5 is capped at 1


def test_auto_tuner_hand_trace():
    # delta = 2.  F: 10, 9, 8.1, 7.29, 6.561, 5.9049 (losses 0 after the first), epoch time 1:
    # LDR_1..5 = -1, -0.9, -0.81, -0.729, -0.6561.  t=3: LDR_3 >= LDR_1 -> up (level 2).  t=4: one epoch since
    # the change, no decision.  t=5: LDR_5 >= LDR_3 -> up (3).  Then epoch time 0.1: LDR_6 = -5.9049,
    # LDR_7 = -5.31441.  t=7: LDR_7 < LDR_5 -> down (2).
    tu = OE.AutoTuner(nnz=30, n=100, delta=2)
    levels = [tu.step(10.0 if t == 0 else 0.0, 1.0 if t < 6 else 0.1) for t in range(8)]
    assert levels == [1, 1, 1, 2, 2, 3, 3, 2]
    assert tu.ldr[:5] == pytest.approx([-1, -0.9, -0.81, -0.729, -0.6561])
    assert tu.threshold == Fraction(9, 2000)


def test_auto_tuner_clamps():
    up = OE.AutoTuner(nnz=30, n=100, delta=1)
    for t in range(20):  # a steadily slowing descent: LDR rises every epoch
        up.step(10.0 / (t + 1), 1.0)
    assert up.level == 6 and up.threshold == 1
    down = OE.AutoTuner(nnz=30, n=100, delta=1)
    for t in range(20):  # a descent that keeps steepening
        down.step(-float(t * t), 1.0)
    assert down.level == 0 and down.threshold == 0
