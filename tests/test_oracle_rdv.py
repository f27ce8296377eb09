"""Pins of the oracle's blocking rendezvous transfers (the naive coordination of §3.3: receive
right before the consumer, send right after the producer, a transfer holding both devices until
it ends): a worked example, a closed form, the deadlock the paper describes, an independent
tick-by-tick execution of the device programs on tiny instances, and invariants."""
import numpy as np
import pytest

import bruteforce as BF
from conftest import read_golden
from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

NTHREADS = 4


def chain(P, M, pol, f, b, c, w=0):
    recs = I.pack_records(P, 1, 0, [pol], [1], [np.arange(1, P)], [np.arange(P)])
    prob = R.problem(P, P, 1, M, recs.shape[1], 0)
    costs = np.tile(np.array([[f, b, w]], np.int64), (P, 1))
    link = I.link_matrix(P, c)
    return (R.sim_batch(prob, costs, link, recs)[0][0],
            R.sim_batch_rdv(prob, costs, link, recs))


def test_worked_example():
    kv, _ = read_golden("rdv_worked_example.txt")
    T = int(kv["T_ns"])
    recs = I.pack_records(2, 1, 0, [I.POLICY["AFAB"], I.POLICY["1F1B"]], [1, 1], [[1], [1]],
                          [[0, 1], [0, 1]])
    prob = R.problem(2, 2, 1, 2, recs.shape[1], 0)
    costs = np.array([[2, 2, 2], [4, 4, 4]], np.int64) * T
    link = I.link_matrix(2, int(kv["transfer_T"]) * T)
    ms, bub = R.sim_batch_rdv(prob, costs, link, recs)
    assert ms[0] == int(kv["gpipe_makespan_T"]) * T
    assert bub[0].tolist() == [int(kv["gpipe_bubble0_T"]) * T, int(kv["gpipe_bubble1_T"]) * T]
    assert R.sim_batch(prob, costs, link, recs)[0][0] == int(kv["async_gpipe_makespan_T"]) * T
    assert ms[1] == int(kv["one_f_one_b"]) and (bub[1] == -1).all()


@pytest.mark.parametrize("M,f,b,c", [(1, 100, 200, 300), (4, 1000, 2000, 3000),
                                     (8, 1000, 1000, 1), (16, 700, 900, 0), (5, 3, 11, 7)])
def test_gpipe_two_devices_closed_form(M, f, b, c):
    """GPipe on two devices: the two arrive at every transfer together, so each forward step
    costs f + c and each backward step b + c: (M + 1)(f + b) + 2Mc, against (M + 1)(f + b) + 2c
    with asynchronous transfers."""
    plain, (ms, bub) = chain(2, M, I.POLICY["AFAB"], f, b, c)
    assert ms[0] == (M + 1) * (f + b) + 2 * M * c
    assert plain == (M + 1) * (f + b) + 2 * c
    assert bub[0].tolist() == [ms[0] - M * (f + b)] * 2


@pytest.mark.parametrize("P,M", [(2, 2), (2, 5), (3, 2), (4, 8), (8, 8)])
@pytest.mark.parametrize("pol", ["1F1B", "ZB"])
def test_one_f_one_b_deadlocks(P, M, pol):
    """The paper's naive-coordination deadlock (§3.3): in 1F1B's steady state the last two
    stages send to each other at once (a forward's output up, a backward's output down), each
    blocked until the other receives. One micro-batch never crosses."""
    _, (ms, _) = chain(P, M, I.POLICY[pol], 1000, 2000, 300, 500)
    assert ms[0] == -1
    _, (ms1, _) = chain(P, 1, I.POLICY[pol], 1000, 2000, 300, 500)
    assert ms1[0] > 0


def test_tick_execution_tiny():
    """Random tiny candidates (all policies and placements, random moves) against a tick-by-tick
    execution of the device programs with blocking transfers."""
    rng = np.random.default_rng(31)
    checked = dead = alive = 0
    for trial in range(70):
        P = int(rng.integers(1, 4))
        v_max = int(rng.integers(1, 3))
        M = int(rng.integers(1, 4))
        L = P * v_max + int(rng.integers(0, 3))
        recs = I.random_candidates(rng, L, P, v_max, M, 8, max_pert=2, pert_rate=0.5)
        prob = R.problem(L, P, v_max, M, recs.shape[1], 2)
        costs = rng.integers(0, 5, size=(L, 3)).astype(np.int64)
        link = rng.integers(0, 6, size=(P, P)).astype(np.int64)
        ms, bub = R.sim_batch_rdv(prob, costs, link, recs)
        for i in range(len(recs)):
            q = R.dump_queues(prob, recs[i])
            if q is None:
                assert ms[i] == -2
                continue
            c = I.unpack_record(recs[i], P, v_max, 2)
            b = c["b"] + [L]
            S = len(c["dev"])
            Fs = [int(costs[b[s]:b[s + 1], 0].sum()) for s in range(S)]
            Bs = [int(costs[b[s]:b[s + 1], 1].sum()) for s in range(S)]
            Ws = [int(costs[b[s]:b[s + 1], 2].sum()) for s in range(S)]
            split = c["policy"] == I.POLICY["ZB"]
            tms, tbub = BF.rdv_tick_simulate(P, S, M, split, c["dev"], Fs, Bs, Ws,
                                             link.tolist(), q)
            assert ms[i] == tms and list(bub[i]) == tbub, (trial, i)
            checked += 1
            dead += tms == -1
            alive += tms > 0
    assert checked > 300 and dead > 30 and alive > 100


def test_invariants():
    """Blocking only adds waiting: rendezvous >= asynchronous, and a deadlock of the plain model
    stays one; with every stage on one device there is no transfer, so the two agree."""
    rng = np.random.default_rng(37)
    L, P, v, M = 20, 4, 2, 8
    recs = I.random_candidates(rng, L, P, v, M, 400, max_pert=2, pert_rate=0.3,
                               invalid_rate=0.1)
    prob = R.problem(L, P, v, M, recs.shape[1], 2)
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 2_000_000, size=(P, P)).astype(np.int64)
    ms, _ = R.sim_batch(prob, costs, link, recs, NTHREADS)
    rs, rb = R.sim_batch_rdv(prob, costs, link, recs, NTHREADS)
    assert ((ms == -2) == (rs == -2)).all() and (rs[ms == -1] == -1).all()
    both = (ms > 0) & (rs > 0)
    assert (rs[both] >= ms[both]).all() and both.sum() > 20 and (rs == -1).sum() > 50
    assert (rb[rs > 0] >= 0).all()
    one = I.pack_records(1, 3, 0, [0, 1, 3], [3, 3, 3], [[4, 9], [4, 9], [4, 9]],
                         [[0, 0, 0]] * 3)
    p1 = R.problem(20, 1, 3, 8, one.shape[1], 0)
    l1 = np.zeros((1, 1), np.int64)
    assert (R.sim_batch(p1, costs, l1, one)[0] == R.sim_batch_rdv(p1, costs, l1, one)[0]).all()


# ---------------------------------------------------------------------------------------------
# The reordered coordination (deadlock-free, overlap-aware reordering of the communication,
# §7 "Unified Pipeline Executor"): each transfer at its ideal start in the asynchronous schedule.
# ---------------------------------------------------------------------------------------------

def test_ordered_worked_example():
    kv, _ = read_golden("rdv_worked_example.txt")
    T = int(kv["T_ns"])
    recs = I.pack_records(2, 1, 0, [I.POLICY["AFAB"], I.POLICY["1F1B"]], [1, 1], [[1], [1]],
                          [[0, 1], [0, 1]])
    prob = R.problem(2, 2, 1, 2, recs.shape[1], 0)
    costs = np.array([[2, 2, 2], [4, 4, 4]], np.int64) * T
    link = I.link_matrix(2, int(kv["transfer_T"]) * T)
    ms, bub = R.sim_batch_ordered(prob, costs, link, recs)
    assert ms[0] == int(kv["ordered_gpipe_makespan_T"]) * T
    assert ms[1] == int(kv["ordered_1f1b_makespan_T"]) * T
    assert bub[1].tolist() == [int(kv["ordered_1f1b_bubble0_T"]) * T,
                               int(kv["ordered_1f1b_bubble1_T"]) * T]


@pytest.mark.parametrize("P,M", [(2, 2), (2, 5), (3, 2), (4, 8), (8, 8), (8, 64)])
@pytest.mark.parametrize("pol", ["1F1B", "ZB", "I1F1B"])
def test_ordered_removes_the_deadlock(P, M, pol):
    """Where the naive coordination deadlocks (1F1B's crossing sends), the reordered one runs,
    and no faster than the asynchronous schedule."""
    plain, (naive, _) = chain(P, M, I.POLICY[pol], 1000, 2000, 300, 500)
    recs = I.pack_records(P, 1, 0, [I.POLICY[pol]], [1], [np.arange(1, P)], [np.arange(P)])
    prob = R.problem(P, P, 1, M, recs.shape[1], 0)
    costs = np.tile(np.array([[1000, 2000, 500]], np.int64), (P, 1))
    ms, _ = R.sim_batch_ordered(prob, costs, I.link_matrix(P, 300), recs)
    assert naive[0] == -1 and ms[0] >= plain > 0


def test_ordered_tick_execution_tiny():
    """Random tiny candidates: reordered programs built independently (from a tick-by-tick
    asynchronous run) and executed tick by tick with blocking transfers, against the oracle
    (links may cost nothing)."""
    rng = np.random.default_rng(41)
    checked = alive = 0
    for trial in range(70):
        P = int(rng.integers(1, 4))
        v_max = int(rng.integers(1, 3))
        M = int(rng.integers(1, 4))
        L = P * v_max + int(rng.integers(0, 3))
        recs = I.random_candidates(rng, L, P, v_max, M, 8, max_pert=2, pert_rate=0.5)
        prob = R.problem(L, P, v_max, M, recs.shape[1], 2)
        # ops of at least one tick: the asynchronous tick run is exact only for those
        costs = rng.integers(1, 5, size=(L, 3)).astype(np.int64)
        link = rng.integers(0, 6, size=(P, P)).astype(np.int64)
        ms, bub = R.sim_batch_ordered(prob, costs, link, recs)
        for i in range(len(recs)):
            q = R.dump_queues(prob, recs[i])
            if q is None:
                assert ms[i] == -2
                continue
            c = I.unpack_record(recs[i], P, v_max, 2)
            b = c["b"] + [L]
            S = len(c["dev"])
            Fs = [int(costs[b[s]:b[s + 1], 0].sum()) for s in range(S)]
            Bs = [int(costs[b[s]:b[s + 1], 1].sum()) for s in range(S)]
            Ws = [int(costs[b[s]:b[s + 1], 2].sum()) for s in range(S)]
            split = c["policy"] == I.POLICY["ZB"]
            starts = {}
            ams, _ = BF.tick_simulate(P, S, M, split, c["dev"], Fs, Bs, Ws, link.tolist(), q,
                                      starts=starts)
            if ams == -1:
                assert ms[i] == -1
                continue
            progs = BF.ordered_programs(S, M, split, c["dev"], Fs, Bs, Ws, q, starts)
            tms, tbub = BF.rdv_tick_simulate(P, S, M, split, c["dev"], Fs, Bs, Ws,
                                             link.tolist(), q, progs)
            assert ms[i] == tms and list(bub[i]) == tbub, (trial, i)
            checked += 1
            alive += tms > 0
    assert checked > 250 and alive > 200


def test_ordered_never_deadlocks_with_positive_costs():
    """With every op and transfer taking time, every dependency strictly increases the global
    key, so the reordered programs never deadlock unless the compute orders themselves do; and
    blocking transfers never beat asynchronous ones."""
    rng = np.random.default_rng(43)
    for (L, P, v, M) in [(20, 4, 2, 8), (24, 8, 1, 16), (30, 3, 3, 6)]:
        recs = I.random_candidates(rng, L, P, v, M, 300, max_pert=3, pert_rate=0.4)
        prob = R.problem(L, P, v, M, recs.shape[1], 3)
        costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
        link = rng.integers(1, 2_000_000, size=(P, P)).astype(np.int64)
        ms, _ = R.sim_batch(prob, costs, link, recs, NTHREADS)
        os_, ob = R.sim_batch_ordered(prob, costs, link, recs, NTHREADS)
        assert ((ms < 0) == (os_ < 0)).all() and (os_[ms < 0] == ms[ms < 0]).all()
        ok = ms > 0
        assert (os_[ok] >= ms[ok]).all() and (ob[ok] >= 0).all() and ok.sum() > 100
