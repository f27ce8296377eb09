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


def _insertion_example():
    from conftest import read_golden
    kv, _ = read_golden("overlap_insertion_example.txt")
    T = int(kv["T_ns"])
    recs = I.pack_records(2, 1, 2, [I.POLICY["ZB"]], [1], [[1]], [[0, 1]])
    prob = R.problem(2, 2, 1, 3, recs.shape[1], 2)
    costs = np.array([[1, 4, 1], [2, 4, 2]], np.int64) * T
    link = I.link_matrix(2, int(kv["transfer_T"]) * T)
    return kv, T, recs, prob, costs, link


def test_overlap_insertion_worked_example():
    """§6's overlap-aware insertion on a hand-worked timeline: the one insertion of device 0
    (the device with the larger residual bubble), and the makespan after it."""
    kv, T, recs, prob, costs, link = _insertion_example()
    lay = A.Layout(prob.P, prob.v_max, prob.max_pert, prob.cand_stride)
    ms, bub, bounds = R.sim_batch_bounds(prob, costs, link, recs)
    assert ms[0] == int(kv["before_makespan_T"]) * T
    resid = A.bubble_split(int(ms[0]), bub[0].tolist(), bounds[0])[4]
    assert A.first_arg(resid, True) == int(kv["device"])
    ins = A.insertions(prob, costs, link, recs[0], lay, 0)
    assert ins == [tuple(int(x) for x in kv["insertion"].split())]
    assert A.insertions(prob, costs, link, recs[0], lay, 1) == \
        [tuple(int(x) for x in kv["device1_insertion"].split())]
    nb = lay.write(dict(lay.read(recs[0]), pert=list(ins)), recs[0])
    assert R.sim_batch(prob, costs, link, nb[None])[0][0] == int(kv["after_makespan_T"]) * T


def test_scheduling_phase_takes_the_insertion():
    """On that record Algorithm 1 searches the scheduling phase; no other policy nor adjacent
    swap reaches 30T, so the kept move is the insertion; without insertions the phase keeps the
    adjacent swap at 31T."""
    kv, T, recs, prob, costs, link = _insertion_example()
    lay = A.Layout(prob.P, prob.v_max, prob.max_pert, prob.cand_stride)
    trace = []
    out, ms, _, acc, _ = A.tune(prob, costs, link, recs, 1, trace=trace)
    assert trace[0] == [(2, True, int(kv["after_makespan_T"]) * T)]
    assert lay.read(out[0])["pert"] == [tuple(int(x) for x in kv["insertion"].split())]
    trace = []
    out0, ms0, _, _, _ = A.tune(prob, costs, link, recs, 1, insert=False, trace=trace)
    assert trace[0] == [(2, True, int(kv["without_insertion_T"]) * T)]
    assert lay.read(out0[0])["pert"] == [tuple(int(x) for x in
                                               kv["without_insertion_move"].split())]


def test_insertions_follow_their_rule_on_random_records():
    """Every insertion the oracle proposes, re-derived from the timeline by the rule's
    definition (idle before B, a communication not overlappable, the first later op ready when
    A ends), and no neighbour built from one deadlocks."""
    rng = np.random.default_rng(61)
    found = 0
    for trial in range(40):
        P, v_max, M = int(rng.integers(2, 5)), int(rng.integers(1, 3)), int(rng.integers(2, 6))
        L = P * v_max + 2
        recs = I.random_candidates(rng, L, P, v_max, M, 6, max_pert=2, pert_rate=0.3)
        prob = R.problem(L, P, v_max, M, recs.shape[1], 2)
        lay = A.Layout(P, v_max, 2, prob.cand_stride)
        costs = rng.integers(1, 6, size=(L, 3)).astype(np.int64)
        link = rng.integers(0, 8, size=(P, P)).astype(np.int64)
        for r in recs:
            c = lay.read(r)
            q = R.dump_queues(prob, r)
            if q is None or c["n_pert"] >= 2:
                continue
            S = P * c["v"]
            split = c["policy"] == A.POL_ZB
            F, B, W = A.stage_costs(c, costs, L)
            rc, _, _, start, _ = R.sim_queues(P, S, M, split, c["dev"], F, B, W, link, q, True)
            if rc != 0:
                continue
            node = lambda op: (op[0] * S + op[1]) * M + op[2]
            dur = lambda op: [F, [B[s] + (0 if split else W[s]) for s in range(S)], W][op[0]][op[1]]
            st = lambda op: int(start[node(op)])
            fin = lambda op: st(op) + dur(op)
            for d in range(P):
                ins = A.insertions(prob, costs, link, r, lay, d)
                Q = q[d]
                for (dd, j, k) in ins:
                    assert dd == d and j > k >= 1 and st(Q[k]) > fin(Q[k - 1])
                    for jj in range(k + 1, j):   # no earlier op was ready
                        rdy = max([fin(p) + (0 if c["dev"][p[1]] == d else
                                             int(link[c["dev"][p[1]]][d]))
                                   for p in A.producers(Q[jj], S)], default=0)
                        assert rdy > fin(Q[k - 1])
                if ins:
                    nbs = np.array([lay.write(dict(c, pert=c["pert"] + [mv]), r) for mv in ins])
                    assert (R.sim_batch(prob, costs, link, nbs)[0] > 0).all()
                    found += len(ins)
    assert found > 20


def test_random_phase_follows_philox():
    """The random-search variant: each searched iteration's phase is the (u mod n)-th open phase,
    u from Philox4x64-10 at counter (record, iteration, 1, 0) and key (seed, 0), computed here
    with numpy's own Philox; the per-phase iteration counts add up."""
    rng = np.random.default_rng(62)
    P, v_max, M, L = 4, 2, 4, 12
    recs = I.random_candidates(rng, L, P, v_max, M, 6, max_pert=2, pert_rate=0.0,
                               policies=(I.POLICY["1F1B"], I.POLICY["ZB"]))
    prob = R.problem(L, P, v_max, M, recs.shape[1], 2)
    costs = rng.integers(1, 6, size=(L, 3)).astype(np.int64) * 1000
    link = I.link_matrix(P, 700)
    seed = 777
    trace = []
    pit = np.zeros((len(recs), 3), np.int64)
    _, _, _, acc, used = A.tune(prob, costs, link, recs, 12, trace=trace, random_search=True,
                                seed=seed, phase_iters=pit)
    for i, steps in enumerate(trace):
        exhausted = set()
        for it, (phase, kept, _) in enumerate(steps):
            open_ = [p for p in range(3) if p not in exhausted]
            ctr = [i, it, 1, 0]
            bg = np.random.Philox(key=np.array([seed, 0], dtype=np.uint64),
                                  counter=np.array([ctr[0] - 1 if i else 2**64 - 1,
                                                    it if i else it - 1 if it else 2**64 - 1,
                                                    1 if (i or it) else 0, 0], dtype=np.uint64))
            u = int(bg.random_raw(1)[0])
            assert phase == open_[u % len(open_)], (i, it)
            exhausted = set() if kept else exhausted | {phase}
        assert pit[i].sum() == used[i] == len(steps)
