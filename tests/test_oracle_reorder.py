"""Pins of the oracle's reordering of the communication (§7, "Unified Pipeline Executor": the
three steps of its deadlock-free, overlap-aware reordering) under handshake transfers: a worked
example, the removed §3.3 deadlocks, programs built independently in Python (tick-by-tick
asynchronous run, levels by fixpoint iteration, the three steps) and executed tick by tick, and
invariants."""
import numpy as np
import pytest

import bruteforce as BF
from conftest import read_golden
from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

NTHREADS = 4


def test_worked_example():
    kv, _ = read_golden("reorder_worked_example.txt")
    T = int(kv["T_ns"])
    recs = I.pack_records(2, 1, 0, [I.POLICY["1F1B"], I.POLICY["AFAB"]], [1, 1], [[1], [1]],
                          [[0, 1], [0, 1]])
    prob = R.problem(2, 2, 1, 2, recs.shape[1], 0)
    costs = np.array([[2, 2, 2], [4, 4, 4]], np.int64) * T
    link = I.link_matrix(2, int(kv["transfer_T"]) * T)
    assert R.sim_batch_rdv(prob, costs, link, recs)[0][0] == -1
    ms, bub, st = R.sim_batch_reorder(prob, costs, link, recs)
    assert ms[0] == int(kv["reorder_1f1b_makespan_T"]) * T
    assert bub[0].tolist() == [int(kv["reorder_1f1b_bubble0_T"]) * T,
                               int(kv["reorder_1f1b_bubble1_T"]) * T]
    assert st[0].tolist() == [int(kv["reorder_1f1b_transfers"]),
                              int(kv["reorder_1f1b_mismatched"])]
    assert ms[1] == int(kv["reorder_gpipe_makespan_T"]) * T
    assert bub[1].tolist() == [int(kv["reorder_gpipe_bubble0_T"]) * T,
                               int(kv["reorder_gpipe_bubble1_T"]) * T]
    assert st[1, 1] == int(kv["reorder_gpipe_mismatched"])


@pytest.mark.parametrize("P,M", [(2, 2), (2, 5), (3, 2), (4, 8), (8, 8)])
@pytest.mark.parametrize("pol", ["1F1B", "ZB"])
def test_removes_the_naive_deadlock(P, M, pol):
    """Where the naive coordination deadlocks (§3.3: 1F1B's crossing sends), the reordered
    programs run, never faster than asynchronous transfers, with mismatched receives found."""
    recs = I.pack_records(P, 1, 0, [I.POLICY[pol]], [1], [np.arange(1, P)], [np.arange(P)])
    prob = R.problem(P, P, 1, M, recs.shape[1], 0)
    costs = np.tile(np.array([[1000, 2000, 500]], np.int64), (P, 1))
    link = I.link_matrix(P, 300)
    assert R.sim_batch_rdv(prob, costs, link, recs)[0][0] == -1
    plain = R.sim_batch(prob, costs, link, recs)[0][0]
    ms, _, st = R.sim_batch_reorder(prob, costs, link, recs)
    assert ms[0] >= plain > 0
    assert st[0, 0] == 2 * (P - 1) * M and st[0, 1] > 0


def _stage_costs(c, costs, L):
    b = c["b"] + [L]
    S = len(c["dev"])
    return ([int(costs[b[s]:b[s + 1], k].sum()) for s in range(S)] for k in range(3))


@pytest.mark.parametrize("seed", [51, 52])
def test_independent_programs_and_tick_execution(seed):
    """Random tiny candidates (every policy and placement, moves, some cyclic): programs built
    independently in Python by the three steps, executed tick by tick with handshake transfers;
    makespan, bubbles and the two counts against the oracle (links may cost nothing)."""
    rng = np.random.default_rng(seed)
    checked = moved = 0
    for trial in range(60):
        P = int(rng.integers(1, 5))
        v_max = int(rng.integers(1, 3))
        M = int(rng.integers(1, 5))
        L = P * v_max + int(rng.integers(0, 3))
        recs = I.random_candidates(rng, L, P, v_max, M, 8, max_pert=2, pert_rate=0.5)
        prob = R.problem(L, P, v_max, M, recs.shape[1], 2)
        costs = rng.integers(1, 5, size=(L, 3)).astype(np.int64)
        link = rng.integers(0, 6, size=(P, P)).astype(np.int64)
        ms, bub, st = R.sim_batch_reorder(prob, costs, link, recs)
        for i in range(len(recs)):
            q = R.dump_queues(prob, recs[i])
            if q is None:
                assert ms[i] == -2
                continue
            c = I.unpack_record(recs[i], P, v_max, 2)
            S = len(c["dev"])
            Fs, Bs, Ws = _stage_costs(c, costs, L)
            split = c["policy"] == I.POLICY["ZB"]
            starts = {}
            ams, _ = BF.tick_simulate(P, S, M, split, c["dev"], Fs, Bs, Ws, link.tolist(), q,
                                      starts=starts)
            if ams == -1:
                assert ms[i] == -1
                continue
            lvl = BF.levels(S, split, c["dev"], q)
            progs, ntr, nmis = BF.reorder_programs(S, M, split, c["dev"], Fs, Bs, Ws,
                                                   link.tolist(), q, starts, lvl)
            tms, tbub = BF.handshake_tick_simulate(P, S, M, split, c["dev"], Fs, Bs, Ws,
                                                   link.tolist(), q, progs)
            assert tms > 0, (trial, i)
            assert ms[i] == tms and list(bub[i]) == tbub, (trial, i, ms[i], tms)
            assert st[i].tolist() == [ntr, nmis], (trial, i)
            checked += 1
            moved += nmis > 0
    assert checked > 250 and moved > 30


def test_zero_costs_tie_keys():
    """Zero-length ops and free links tie the transfers' producer ends; the level breaks the
    ties, so nothing deadlocks and the makespan is 0 or the plain one."""
    rng = np.random.default_rng(53)
    for (L, P, v, M) in [(8, 4, 2, 4), (6, 3, 1, 5), (16, 8, 2, 3)]:
        recs = I.random_candidates(rng, L, P, v, M, 200, max_pert=2, pert_rate=0.4)
        prob = R.problem(L, P, v, M, recs.shape[1], 2)
        costs = rng.integers(0, 2, size=(L, 3)).astype(np.int64)
        link = np.zeros((P, P), np.int64)
        ms, _ = R.sim_batch(prob, costs, link, recs, NTHREADS)
        rs, _, _ = R.sim_batch_reorder(prob, costs, link, recs, NTHREADS)
        assert ((ms == -1) == (rs == -1)).all() and ((ms == -2) == (rs == -2)).all()


def test_never_deadlocks_and_bounds():
    """Every device meets its transfers in key order, so the reordered programs deadlock only
    where the compute orders themselves do; handshakes never beat asynchronous transfers, and
    never lose to blocking ones on the same programs' naive form where that runs."""
    rng = np.random.default_rng(54)
    for (L, P, v, M) in [(20, 4, 2, 8), (24, 8, 1, 16), (30, 3, 3, 6), (40, 16, 2, 8)]:
        recs = I.random_candidates(rng, L, P, v, M, 300, max_pert=3, pert_rate=0.4)
        prob = R.problem(L, P, v, M, recs.shape[1], 3)
        costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
        link = rng.integers(0, 2_000_000, size=(P, P)).astype(np.int64)
        ms, _ = R.sim_batch(prob, costs, link, recs, NTHREADS)
        rs, rb, st = R.sim_batch_reorder(prob, costs, link, recs, NTHREADS)
        nv, _ = R.sim_batch_rdv(prob, costs, link, recs, NTHREADS)
        assert ((ms < 0) == (rs < 0)).all() and (rs[ms < 0] == ms[ms < 0]).all()
        ok = ms > 0
        assert (rs[ok] >= ms[ok]).all() and (rb[ok] >= 0).all() and ok.sum() > 100
        both = ok & (nv > 0) & (st[:, 1] == 0)
        assert (rs[both] <= nv[both]).all()
        assert ((st[ok, 1] >= 0) & (st[ok, 1] <= st[ok, 0])).all()
