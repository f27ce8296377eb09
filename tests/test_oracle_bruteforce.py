"""The oracle against independent brute force on tiny instances, deadlock constructions and
invariants of the time model (§5, §6 Eq. 1)."""
import itertools

import numpy as np
import pytest

import bruteforce as BF
from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

F, B, W = 0, 1, 2


def stage_costs(rec_fields, costs):
    b = rec_fields["b"] + [costs.shape[0]]
    S = len(rec_fields["dev"])
    Fs = [int(costs[b[s]:b[s + 1], 0].sum()) for s in range(S)]
    Bs = [int(costs[b[s]:b[s + 1], 1].sum()) for s in range(S)]
    Ws = [int(costs[b[s]:b[s + 1], 2].sum()) for s in range(S)]
    return Fs, Bs, Ws


def test_all_orders_two_stages_two_microbatches():
    """P = 2, M = 2: every pair of per-device permutations (24 x 24, of which 6 x 6 respect
    F-before-B). Oracle vs tick simulation vs DFS cycle check, with a transfer cost."""
    P = S = M = 2
    dev = [0, 1]
    Fs, Bs, Ws = [2, 3], [1, 4], [2, 1]
    link = [[0, 3], [2, 0]]
    lk = np.array(link, dtype=np.int64)
    ops = [[(k, s, m) for k in (F, B) for m in range(M)] for s in range(S)]
    n_ok = 0
    for q0 in itertools.permutations(ops[0]):
        for q1 in itertools.permutations(ops[1]):
            queues = [list(q0), list(q1)]
            rc, ms, bub, _, _ = R.sim_queues(P, S, M, False, dev, Fs, Bs, Ws, lk, queues)
            tms, tbub = BF.tick_simulate(P, S, M, False, dev, Fs, Bs, Ws, link, queues)
            cyc = BF.has_cycle(P, S, M, False, dev, queues)
            assert (rc == 1) == cyc == (tms == -1)
            if rc == 0:
                n_ok += 1
                assert ms == tms and list(bub) == tbub
    # 36 of the order combinations respecting F-before-B can still deadlock across devices;
    # the count of deadlock-free combinations is what the three methods agree on.
    assert n_ok > 0


def test_valid_orders_split_backward():
    """Split backward, P = 2, M = 2: all orders of each device's F/B/W ops with F(m) < B(m) <
    W(m) per micro-batch (6!/(3!)^2 = 20 per device, 400 combinations), oracle vs tick
    simulation vs DFS."""
    P = S = M = 2
    dev = [0, 1]
    Fs, Bs, Ws = [1, 2], [2, 1], [1, 3]
    link = [[0, 1], [2, 0]]
    lk = np.array(link, dtype=np.int64)

    def orders(s):
        ops = [(k, s, m) for k in (F, B, W) for m in range(M)]
        for perm in itertools.permutations(ops):
            pos = {o: i for i, o in enumerate(perm)}
            if all(pos[(F, s, m)] < pos[(B, s, m)] < pos[(W, s, m)] for m in range(M)):
                yield list(perm)

    o0, o1 = list(orders(0)), list(orders(1))
    assert len(o0) == len(o1) == 20
    for q0, q1 in itertools.product(o0, o1):
        queues = [q0, q1]
        rc, ms, bub, _, _ = R.sim_queues(P, S, M, True, dev, Fs, Bs, Ws, lk, queues)
        tms, tbub = BF.tick_simulate(P, S, M, True, dev, Fs, Bs, Ws, link, queues)
        assert (rc == 1) == BF.has_cycle(P, S, M, True, dev, queues) == (tms == -1)
        if rc == 0:
            assert ms == tms and list(bub) == tbub


@pytest.mark.parametrize("seed", range(6))
def test_policies_against_tick_simulation(seed):
    """Random tiny candidates of every policy, placement and v, with random moves: the oracle's
    makespan/bubbles (or deadlock) equal the tick simulation of the same queues."""
    rng = np.random.default_rng(100 + seed)
    for _ in range(40):
        P = int(rng.integers(1, 4))
        v_max = int(rng.integers(1, 3))
        M = int(rng.integers(1, 5))
        if rng.random() < 0.5:
            M = P * int(rng.integers(1, 3))
        L = P * v_max + int(rng.integers(0, 3))
        costs = rng.integers(1, 5, size=(L, 3)).astype(np.int64)
        link = rng.integers(0, 4, size=(P, P)).astype(np.int64)
        np.fill_diagonal(link, 0)
        max_pert = 2
        recs = I.random_candidates(rng, L, P, v_max, M, 8, max_pert=max_pert, pert_rate=0.4)
        prob = R.problem(L, P, v_max, M, recs.shape[1], max_pert)
        ms, bub = R.sim_batch(prob, costs, link, recs)
        for i in range(len(recs)):
            queues = R.dump_queues(prob, recs[i])
            if queues is None:
                assert ms[i] == -2 and (bub[i] == -2).all()
                continue
            fields = I.unpack_record(recs[i], P, v_max, max_pert)
            S = P * fields["v"]
            Fs, Bs, Ws = stage_costs(fields, costs)
            split = fields["policy"] == I.POLICY["ZB"]
            tms, tbub = BF.tick_simulate(P, S, M, split, fields["dev"], Fs, Bs, Ws,
                                         link.tolist(), queues)
            assert BF.has_cycle(P, S, M, split, fields["dev"], queues) == (tms == -1)
            assert ms[i] == tms and list(bub[i]) == tbub


def test_generated_queues_are_deadlock_free():
    """Every policy's queues on every balanced placement kind are free of cycles (tiny sizes,
    checked by DFS on the queues the oracle generates)."""
    rng = np.random.default_rng(5)
    for P, v_max, M in [(2, 2, 2), (2, 2, 4), (3, 2, 3), (4, 2, 4), (2, 3, 2), (4, 1, 3)]:
        L = P * v_max + 2
        recs = I.random_candidates(rng, L, P, v_max, M, 60)
        prob = R.problem(L, P, v_max, M, recs.shape[1], 0)
        for rec in recs:
            q = R.dump_queues(prob, rec)
            if q is None:
                continue
            f = I.unpack_record(rec, P, v_max, 0)
            assert not BF.has_cycle(P, P * f["v"], M, f["policy"] == 3, f["dev"], q)


def test_deadlock_backward_before_own_forward():
    """A backward placed ahead of its own forward can never run (§3.3)."""
    P, v, M, L = 4, 1, 4, 8
    costs = np.full((L, 3), 10, dtype=np.int64)
    link = I.link_matrix(P, 3)
    base = I.pack_records(P, v, 1, [1], [1], [[2, 4, 6]], [[0, 1, 2, 3]])
    prob = R.problem(L, P, v, M, base.shape[1], 1)
    q = R.dump_queues(prob, base[0])
    d = 2
    i_b = q[d].index((B, 2, 1))
    i_f = q[d].index((F, 2, 1))
    rec = I.pack_records(P, v, 1, [1], [1], [[2, 4, 6]], [[0, 1, 2, 3]],
                         perts=[[[d, i_b, i_f]]], n_pert=[1])
    ms, bub = R.sim_batch(prob, costs, link, rec)
    assert ms[0] == -1 and (bub[0] == -1).all()
    # and the "last op to the front" move used for deliberately cyclic workload candidates
    for pol in (0, 1, 2, 3):
        n_ops = (3 if pol == 3 else 2) * v * M
        rec = I.pack_records(P, v, 1, [pol], [1], [[2, 4, 6]], [[0, 1, 2, 3]],
                             perts=[[[1, n_ops - 1, 0]]], n_pert=[1])
        ms, _ = R.sim_batch(prob, costs, link, rec)
        assert ms[0] == -1


def test_deadlock_cross_device_two_cycle():
    """Device 0 runs B(0,m) before F(0,m'), while device 1 runs F(1,m') before B(1,m): each waits
    on the other (the cyclic wait of §3.3 / §7)."""
    P = S = 2
    M = 2
    ones = np.ones(2, dtype=np.int64)
    lk = I.link_matrix(2, 1)
    q0 = [(F, 0, 0), (B, 0, 0), (F, 0, 1), (B, 0, 1)]
    q1 = [(F, 1, 1), (F, 1, 0), (B, 1, 0), (B, 1, 1)]
    rc, *_ = R.sim_queues(P, S, M, False, [0, 1], ones, ones, ones, lk, [q0, q1])
    assert rc == 1
    assert BF.has_cycle(P, S, M, False, [0, 1], [q0, q1])


def test_interleaved_order_on_vshape_deadlocks():
    """The interleaved order written out for P = 2, v = 2, M = 2 (rank 0: warm-up 4, rank 1:
    warm-up 2) runs on the looped placement but deadlocks on the V-shape one, which is why
    non-looped placements use the MERGE order."""
    P, M, S = 2, 2, 4
    rank0 = [(F, 0, 0), (F, 0, 1), (F, 1, 0), (F, 1, 1), (B, 1, 0), (B, 1, 1), (B, 0, 0), (B, 0, 1)]
    rank1 = [(F, 0, 0), (F, 0, 1), (F, 1, 0), (B, 1, 0), (F, 1, 1), (B, 1, 1), (B, 0, 0), (B, 0, 1)]
    ones = np.ones(S, dtype=np.int64)
    lk = I.link_matrix(P, 1)

    def on(placement):
        dev = I.placement(placement, P, 2)
        A = [[s for s in range(S) if dev[s] == d] for d in range(P)]
        pat = [rank0, rank1] if A[0][0] == 0 else [rank1, rank0]
        qs = [[(k, A[d][c], m) for (k, c, m) in pat[d]] for d in range(P)]
        return R.sim_queues(P, S, M, False, dev, ones, ones, ones, lk, qs)[0], dev, qs

    rc, dev, qs = on("looped")
    assert rc == 0 and not BF.has_cycle(P, S, M, False, dev, qs)
    rc, dev, qs = on("vshape")
    assert rc == 1 and BF.has_cycle(P, S, M, False, dev, qs)
    # the oracle's own generator for looped I1F1B matches the hand-written order
    prob = R.problem(S, P, 2, M, I.record_stride(P, 2, 0), 0)
    rec = I.pack_records(P, 2, 0, [2], [2], [[1, 2, 3]], [I.placement("looped", P, 2)])
    q = R.dump_queues(prob, rec[0])
    assert q == [[(k, c * 2 + 0, m) for (k, c, m) in rank0], [(k, c * 2 + 1, m) for (k, c, m) in rank1]]


def test_merge_ideal_times_and_order():
    """MERGE: the ideal start times are the earliest-start times of the stage-level pipeline
    (checked by tick simulation), and each device queue is sorted by (tau, stage)."""
    for S, M, split in [(4, 3, False), (4, 3, True), (6, 5, False), (3, 4, True)]:
        tau = R.merge_tau(S, M, split)
        # stage-level queues from the v = 1 generator (one device per stage)
        L = S
        prob = R.problem(L, S, 1, M, I.record_stride(S, 1, 0), 0)
        pol = I.POLICY["ZB"] if split else I.POLICY["1F1B"]
        rec = I.pack_records(S, 1, 0, [pol], [1], [list(range(1, S))], [list(range(S))])
        queues = R.dump_queues(prob, rec[0])
        fin = {}
        ones = [1] * S
        # tick simulation records start = finish - duration
        ms, _ = BF.tick_simulate(S, S, M, split, list(range(S)), ones, ones, ones,
                                 [[0] * S for _ in range(S)], queues)
        # recompute start times by an independent ASAP walk to compare op by op
        start = {}
        done = {}
        clock = [0] * S
        ptr = [0] * S
        progress = True
        while progress:
            progress = False
            for d in range(S):
                while ptr[d] < len(queues[d]):
                    k, s, m = queues[d][ptr[d]]
                    prods = BF._producers((k, s, m), S, split, list(range(S)), [[0] * S] * S)
                    if not all(p in done for p, _ in prods):
                        break
                    st = max([clock[d]] + [done[p] for p, _ in prods])
                    dur = 1 if (k != B or split) else 2
                    start[(k, s, m)] = st
                    done[(k, s, m)] = st + dur
                    clock[d] = st + dur
                    ptr[d] += 1
                    progress = True
        assert max(done.values()) == ms
        for (k, s, m), st in start.items():
            assert tau[k, s, m] == st
        # device queues of a MERGE candidate are sorted by (tau, stage)
        P, v = 2, S // 2 if S % 2 == 0 else None
        if v is None:
            continue
        prob2 = R.problem(S, P, v, M, I.record_stride(P, v, 0), 0)
        dev = I.placement("vshape", P, v)
        rec2 = I.pack_records(P, v, 0, [pol], [v], [list(range(1, S))], [dev])
        q2 = R.dump_queues(prob2, rec2[0])
        for d in range(P):
            keys = [(int(tau[k, s, m]), s) for (k, s, m) in q2[d]]
            assert keys == sorted(keys)
            assert len(q2[d]) == (3 if split else 2) * v * M


@pytest.mark.parametrize("seed", range(3))
def test_invariants(seed):
    """Bubbles >= 0; makespan >= every device's busy time and >= one micro-batch's critical path;
    makespan <= total work plus all transfers; scaling every cost and link by k scales the
    makespan by k; P = 1 gives the total work (§6 Eq. 1; max-plus algebra)."""
    rng = np.random.default_rng(seed)
    P, v_max, M, L = 4, 2, 8, 20
    costs = rng.integers(1000, 5000, size=(L, 3)).astype(np.int64)
    link = I.link_matrix(P, 700)
    recs = I.random_candidates(rng, L, P, v_max, M, 200)
    prob = R.problem(L, P, v_max, M, recs.shape[1], 0)
    ms, bub = R.sim_batch(prob, costs, link, recs)
    assert (ms > 0).all()
    assert (bub >= 0).all()
    for i in range(len(recs)):
        f = I.unpack_record(recs[i], P, v_max, 0)
        Fs, Bs, Ws = stage_costs(f, costs)
        busy = ms[i] - bub[i]
        assert ms[i] >= busy.max()
        crit = sum(Fs) + sum(Bs)  # forward chain then input-gradient chain of one micro-batch
        assert ms[i] >= crit
        S = len(Fs)
        assert ms[i] <= M * (sum(Fs) + sum(Bs) + sum(Ws)) + 2 * (S - 1) * M * 700
    ms3, bub3 = R.sim_batch(prob, 3 * costs, 3 * link, recs)
    assert (ms3 == 3 * ms).all() and (bub3 == 3 * bub).all()
    # one device: everything serial
    prob1 = R.problem(L, 1, 1, M, I.record_stride(1, 1, 0), 0)
    for pol in range(4):
        r1 = I.pack_records(1, 1, 0, [pol], [1], np.zeros((1, 0)), [[0]])
        m1, b1 = R.sim_batch(prob1, costs, I.link_matrix(1, 0), r1)
        assert m1[0] == M * costs.sum() and b1[0, 0] == 0


def test_monotone_in_costs_and_relabel_invariant():
    """Raising any layer cost never shortens the pipeline; relabelling devices under uniform
    links leaves the makespan unchanged and permutes the bubbles."""
    rng = np.random.default_rng(11)
    P, v_max, M, L = 4, 2, 6, 16
    costs = rng.integers(1000, 5000, size=(L, 3)).astype(np.int64)
    link = I.link_matrix(P, 900)
    recs = I.random_candidates(rng, L, P, v_max, M, 120, policies=(0, 1, 2, 3))
    prob = R.problem(L, P, v_max, M, recs.shape[1], 0)
    ms, bub = R.sim_batch(prob, costs, link, recs)
    for _ in range(5):
        c2 = costs.copy()
        c2[int(rng.integers(0, L)), int(rng.integers(0, 3))] += int(rng.integers(1, 3000))
        ms2, _ = R.sim_batch(prob, c2, link, recs)
        assert (ms2 >= ms).all()
    s_max = P * v_max
    pi = rng.permutation(P)
    rel = recs.copy()
    rel[:, 3 + s_max:3 + 2 * s_max] = pi[rel[:, 3 + s_max:3 + 2 * s_max].astype(np.int64)]
    ms_r, bub_r = R.sim_batch(prob, costs, link, rel)
    assert (ms_r == ms).all()
    assert (bub_r[:, pi] == bub).all()
