"""Pins of the oracle's serialised links (a variant of §5's communication nodes: a directed link
carries one transfer at a time, first come first served): a closed form, the cases where nothing
queues, an independent tick simulation on tiny instances, and invariants."""
import numpy as np
import pytest

import bruteforce as BF
from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

NTHREADS = 4


def chain(P, M, pol, f, b, c):
    recs = I.pack_records(P, 1, 0, [pol], [1], [np.arange(1, P)], [np.arange(P)])
    prob = R.problem(P, P, 1, M, recs.shape[1], 0)
    costs = np.tile(np.array([[f, b, 0]], np.int64), (P, 1))
    link = I.link_matrix(P, c)
    return R.sim_batch(prob, costs, link, recs)[0][0], R.sim_batch_serial(prob, costs, link,
                                                                         recs)[0][0]


@pytest.mark.parametrize("M,f,b,c", [(1, 100, 200, 300), (4, 1000, 2000, 3000),
                                     (8, 1000, 1000, 1000), (16, 700, 900, 901)])
def test_gpipe_two_devices_closed_form(M, f, b, c):
    """GPipe on two devices with c >= max(f, b): forwards reach the second device every c
    (arrival of m at f + (m+1) c, which it keeps up with), its backwards return every c as well,
    so the last backward ends at 2f + 2b + 2Mc (without the queue: (M+1)(f+b) + 2c)."""
    plain, serial = chain(2, M, I.POLICY["AFAB"], f, b, c)
    assert serial == 2 * f + 2 * b + 2 * M * c
    assert plain == (M + 1) * (f + b) + 2 * c


@pytest.mark.parametrize("P,M,pol", [(4, 8, "AFAB"), (3, 5, "AFAB"), (4, 8, "1F1B"),
                                     (6, 6, "1F1B")])
def test_nothing_queues_when_transfers_are_short(P, M, pol):
    """One stage per device and c <= min(f, b): a device sends at most once per op on each
    link, and each transfer ends before the next one is issued."""
    plain, serial = chain(P, M, I.POLICY[pol], 1000, 1500, 1000)
    assert serial == plain


def test_tick_simulation_tiny():
    """Random tiny candidates (all policies and placements, random moves, many deadlocks) against
    a tick-by-tick execution with per-link transfer queues."""
    rng = np.random.default_rng(12)
    checked = dead = 0
    for trial in range(60):
        P = int(rng.integers(1, 4))
        v_max = int(rng.integers(1, 3))
        M = int(rng.integers(1, 4))
        L = P * v_max + int(rng.integers(0, 3))
        recs = I.random_candidates(rng, L, P, v_max, M, 8, max_pert=2, pert_rate=0.5)
        prob = R.problem(L, P, v_max, M, recs.shape[1], 2)
        costs = rng.integers(1, 5, size=(L, 3)).astype(np.int64)
        link = rng.integers(0, 7, size=(P, P)).astype(np.int64)
        ms, bub = R.sim_batch_serial(prob, costs, link, recs)
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
            tms, tbub = BF.tick_simulate(P, S, M, split, c["dev"], Fs, Bs, Ws, link.tolist(), q,
                                         serial=True)
            assert ms[i] == tms and list(bub[i]) == tbub, (trial, i)
            checked += 1
            dead += tms == -1
    assert checked > 300 and dead > 10


def test_invariants():
    """Queued transfers only delay: serial >= plain; deadlock and validity are structural, so the
    sentinels agree; free links queue nothing."""
    rng = np.random.default_rng(19)
    L, P, v, M = 20, 4, 2, 8
    recs = I.random_candidates(rng, L, P, v, M, 400, max_pert=2, pert_rate=0.3,
                               invalid_rate=0.1)
    prob = R.problem(L, P, v, M, recs.shape[1], 2)
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 12_000_000, size=(P, P)).astype(np.int64)
    ms, _ = R.sim_batch(prob, costs, link, recs, NTHREADS)
    ss, _ = R.sim_batch_serial(prob, costs, link, recs, NTHREADS)
    ok = ms > 0
    assert ((ms < 0) == (ss < 0)).all() and (ms[~ok] == ss[~ok]).all()
    assert (ss[ok] >= ms[ok]).all() and (ss[ok] > ms[ok]).sum() > 50
    z = np.zeros((P, P), np.int64)
    assert (R.sim_batch(prob, costs, z, recs, NTHREADS)[0] ==
            R.sim_batch_serial(prob, costs, z, recs, NTHREADS)[0]).all()


def test_xgmi_link_matrix_and_queues_across_nodes():
    """The MI355X link recipe: xGMI inside a node of eight GPUs, the NIC between nodes. With
    large activations on a two-node pipeline the slower node-crossing link queues transfers."""
    m = I.xgmi_link_matrix(16, 32 << 20)
    assert (np.diag(m) == 0).all() and (m == m.T).all()
    assert m[0, 1] == I.link_cost_ns(32 << 20, 5_000, 153) and m[0, 8] == I.link_cost_ns(
        32 << 20, 20_000, 50)
    assert m[3, 7] < m[7, 8]
    P, M = 16, 16
    recs = I.pack_records(P, 1, 0, [I.POLICY["1F1B"]], [1], [np.arange(1, P)], [np.arange(P)])
    prob = R.problem(P, P, 1, M, recs.shape[1], 0)
    costs = np.full((P, 3), 1_000_000, np.int64)
    link = I.xgmi_link_matrix(P, 1 << 30)
    plain, serial = R.sim_batch(prob, costs, link, recs)[0][0], \
        R.sim_batch_serial(prob, costs, link, recs)[0][0]
    assert serial > plain
