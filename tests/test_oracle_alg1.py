"""Pins of the oracle's Algorithm 1 (§6, iterative bubble-aware tuning): the branch as printed,
the bubble split it decides on (a timeline worked by hand), a partitioning run that must end
balanced at the closed-form makespan, the neighbourhood shapes, and properties of every search
(the makespan never grows and falls exactly at kept moves; a converged record has no better
neighbour in any phase)."""
import numpy as np
import pytest

from oracle import alg1 as A
from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

NTHREADS = 4


def test_branch_as_printed():
    """Partitioning iff Δb > t_layer; else placement iff b_bd > b_res; else scheduling; an
    exhausted phase falls to the first remaining one in priority order."""
    assert A.choose_phase(11, 10, 0, 5, set()) == 0
    assert A.choose_phase(10, 10, 6, 5, set()) == 1
    assert A.choose_phase(10, 10, 5, 5, set()) == 2
    assert A.choose_phase(11, 10, 6, 5, {0}) == 1
    assert A.choose_phase(0, 10, 6, 5, {1}) == 0
    assert A.choose_phase(0, 10, 0, 5, {2, 0}) == 1
    assert A.choose_phase(0, 10, 0, 5, {0, 1, 2}) is None


def test_bubble_split_of_a_known_timeline():
    """The §3.2 two-stage example (1F1B, S0 2T, S1 4T per workload, no transfer cost). By hand:
    device 0 runs F0 [0,2], F1 [2,4], B0 [14,18], B1 [26,30]; device 1 runs F0 [2,6],
    B0 [6,14], F1 [14,18], B1 [18,26]. So device 1 idles 2T before and 4T after its ops and none
    between; device 0 idles only between its ops."""
    T = 1000
    recs = I.pack_records(2, 1, 0, [I.POLICY["1F1B"]], [1], [[1]], [[0, 1]])
    prob = R.problem(2, 2, 1, 2, recs.shape[1], 0)
    costs = np.array([[2, 2, 2], [4, 4, 4]], np.int64) * T
    ms, bub, bounds = R.sim_batch_bounds(prob, costs, I.link_matrix(2, 0), recs)
    assert ms[0] == 30 * T and bub[0].tolist() == [18 * T, 6 * T]
    assert bounds[0].tolist() == [[0, 30 * T], [2 * T, 26 * T]]
    delta_b, b_bd, b_res, busy, resid = A.bubble_split(int(ms[0]), bub[0].tolist(), bounds[0])
    assert (delta_b, b_bd, b_res) == (12 * T, 6 * T, 18 * T)
    assert busy == [12 * T, 24 * T] and resid == [18 * T, 0]


def test_partitioning_balances_two_devices():
    """Eight equal layers split 1 | 7 over two devices (v_max = 1, so no dispersion): the
    imbalance exceeds one layer's time, so partitioning migrates one layer per iteration from
    the loaded device until 4 | 4, where 1F1B with fused backward ends at (M + 1)(f + b) for the
    stage costs f = 4t, b = 8t."""
    t, M = 1000, 8
    recs = I.pack_records(2, 1, 0, [I.POLICY["1F1B"]], [1], [[1]], [[0, 1]])
    prob = R.problem(8, 2, 1, M, recs.shape[1], 0)
    costs = np.tile(np.array([[t, t, t]], np.int64), (8, 1))
    trace = []
    out, ms, _, acc, _ = A.tune(prob, costs, I.link_matrix(2, 0), recs, 3, trace=trace)
    assert [s[:2] for s in trace[0]] == [(0, True)] * 3
    assert int(out[0][4]) == 4 and ms[0] == (M + 1) * (4 * t + 8 * t)


def test_neighbourhood_shapes():
    P, v, M, L = 4, 2, 8, 24
    rng = np.random.default_rng(2)
    recs = I.random_candidates(rng, L, P, v, M, 40, policies=(3,))
    lay = A.Layout(P, v, 3, I.record_stride(P, v, 3))
    recs = np.concatenate([recs, np.zeros((len(recs), lay.stride - recs.shape[1]), np.uint8)], 1)
    busy, bub, resid = [5, 9, 1, 3], [4, 0, 8, 6], [1, 0, 3, 3]
    for rec in recs:
        c = lay.read(rec)
        vv = c["v"]
        S = P * vv
        part = A.neighbours(lay, rec, 0, L, M, busy, bub, resid)
        src = [s for s in range(S) if c["dev"][s] == 1]  # most loaded device
        bnd = c["b"] + [L]
        assert len(part) == vv * sum(bnd[a + 1] - bnd[a] >= 2 for a in src)
        for n in part:  # one layer leaves a stage of device 1 for one of device 2
            cn = lay.read(n)
            size = np.diff(cn["b"] + [L]) - np.diff(bnd)
            assert sorted(size[size != 0].tolist()) == [-1, 1]
            assert c["dev"][int(np.nonzero(size < 0)[0][0])] == 1
            assert c["dev"][int(np.nonzero(size > 0)[0][0])] == 2
        place = A.neighbours(lay, rec, 1, L, M, busy, bub, resid)
        disp = 2 * vv <= v and all(bnd[s + 1] - bnd[s] >= 2 for s in range(S))
        assert len(place) == vv * vv * (P - 1) + disp
        sched = A.neighbours(lay, rec, 2, L, M, busy, bub, resid)
        assert len(sched) == 3 + 3 * vv * M - 1
        assert all(lay.read(n)["pert"][-1][0] == 2 for n in sched[3:])


def test_search_properties():
    """Random searches: the makespan never grows and falls exactly at kept moves; a search that
    stops early has no better neighbour left in any phase."""
    rng = np.random.default_rng(3)
    L, P, v, M, mp = 24, 4, 2, 8, 6
    recs = I.random_candidates(rng, L, P, v, M, 12, policies=(1, 2, 3))
    lay = A.Layout(P, v, mp, I.record_stride(P, v, mp))
    recs = np.concatenate([recs, np.zeros((len(recs), lay.stride - recs.shape[1]), np.uint8)], 1)
    prob = R.problem(L, P, v, M, lay.stride, mp)
    costs = rng.integers(100_000, 3_000_000, size=(L, 3)).astype(np.int64)
    link = I.link_matrix(P, 200_000)
    ms0, _ = R.sim_batch(prob, costs, link, recs)
    iters = 40
    trace = []
    out, ms, bub, acc, used = A.tune(prob, costs, link, recs, iters, NTHREADS, trace=trace)
    assert (ms <= ms0).all() and (acc.sum(axis=1) > 0).all()
    for i, steps in enumerate(trace):
        last = ms0[i]
        for phase, kept, after in steps:
            assert after <= last and (after < last) == kept
            last = after
        if used[i] < iters:  # converged: every phase exhausted at the final record
            r = out[i]
            m1, b1, bd = R.sim_batch_bounds(prob, costs, link, r[None])
            _, _, _, busy, resid = A.bubble_split(int(m1[0]), b1[0].tolist(), bd[0])
            for ph in range(3):
                nb = A.neighbours(lay, r, ph, L, M, busy, b1[0].tolist(), resid)
                if nb:
                    nms, _ = R.sim_batch(prob, costs, link, np.array(nb))
                    assert not ((nms >= 0) & (nms < m1[0])).any()
    assert (used < iters).sum() >= 3
