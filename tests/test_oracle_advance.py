"""Pins of the oracle's selective W advancing and memory-constrained local search (§6
"Scheduling Tuning", third policy; §6 Eq. 2: peak memory per device within its capacity).

The policy: while a device's peak exceeds its capacity, advance a deferred W of that device to
the queue position at which the peak is first reached (its stage's activations are then
released before that allocation), preferring a W whose advance does not lengthen the makespan,
else the earliest eligible one. These tests pin it to an order forced by the capacity (derived
below by hand), to the plain simulator and search it reduces to, and to properties every result
must have, checked with the plain (already pinned) simulator and an order walk of the queues.
"""
import numpy as np
import pytest

from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

NTHREADS = 4
KF, KB, KW = 0, 1, 2


def one_stage_per_device(P, M, pol, max_pert):
    recs = I.pack_records(P, 1, max_pert, [pol], [1], [np.arange(1, P)], [np.arange(P)])
    return R.problem(P, P, 1, M, recs.shape[1], max_pert), recs


def walk(queue, act, split):
    """Running activation total along one queue: (largest total, first position reaching it)."""
    cur = hi = 0
    at = -1
    for i, (k, s, m) in enumerate(queue):
        if k == KF:
            cur += act[s]
            if cur > hi:
                hi, at = cur, i
        elif (k == KB and not split) or k == KW:
            cur -= act[s]
    return hi, at


def eager_zb_queue(S, s, M):
    """The 1F1B order of stage s (warm-up min(S-1-s, M)) with every W right after its B."""
    w = min(S - 1 - s, M)
    q = [(KF, s, m) for m in range(w)]
    for i in range(M - w):
        q += [(KF, s, w + i), (KB, s, i), (KW, s, i)]
    for m in range(M - w, M):
        q += [(KB, s, m), (KW, s, m)]
    return q


@pytest.mark.parametrize("P,M", [(3, 6), (4, 8), (2, 5), (5, 12)])
def test_capacity_of_1f1b_forces_eager_w(P, M):
    """ZB defers W by the device's rank r and holds min(S, M) micro-batches; a capacity of the
    1F1B footprint min(S - s, M) forces each W that precedes a later forward into the one slot
    between its B and that forward, which is the eager order until the last forward. The W after
    the last forward never precede an allocation and stay where the policy put them."""
    A, Z = 1000, 77
    prob, recs = one_stage_per_device(P, M, I.POLICY["ZB"], 200)
    costs = np.tile(np.array([[300, 500, 200]], np.int64), (P, 1))
    mem = np.tile(np.array([[A, Z]], np.int64), (P, 1))
    cap = Z + A * np.minimum(P - np.arange(P), M)
    link = I.link_matrix(P, 40)
    out, ms, bub, peak = R.advance_w(prob, costs, mem, cap, link, recs)
    assert (peak[0] == cap).all()
    q = R.dump_queues(prob, out[0])
    base = R.dump_queues(prob, recs[0])
    for s in range(P):
        w = min(P - 1 - s, M)
        last_f = max(i for i, o in enumerate(q[s]) if o[0] == KF)
        eager = eager_zb_queue(P, s, M)
        assert q[s][:last_f + 2] == eager[:last_f + 2], s
        # after the last forward: the policy's own order, untouched
        assert [o for o in q[s][last_f + 2:]] == [o for o in base[s] if o not in q[s][:last_f + 2]]
        assert [o for o in q[s] if o[0] == KW and o[2] >= M - w - 1] == \
            [o for o in base[s] if o[0] == KW and o[2] >= M - w - 1]
    # the outputs describe the output record, as the plain simulator sees it
    ms2, bub2, peak2 = R.sim_batch_mem(prob, costs, mem, link, out)
    assert ms2[0] == ms[0] and (bub2 == bub).all() and (peak2 == peak).all()
    st, ms3, _, _, _ = R.sim_queues(P, P, M, True, np.arange(P), costs[:, 0], costs[:, 1],
                                    costs[:, 2], link, q)
    assert st == 0 and ms3 == ms[0]


def test_enough_capacity_changes_nothing():
    rng = np.random.default_rng(5)
    L, P, v, M = 16, 4, 2, 8
    recs = I.random_candidates(rng, L, P, v, M, 200, max_pert=6, pert_rate=0.3,
                               invalid_rate=0.1)
    prob = R.problem(L, P, v, M, recs.shape[1], 6)
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    mem = np.stack([rng.integers(0, 1 << 30, L), rng.integers(0, 1 << 34, L)], axis=1)
    link = rng.integers(0, 900_000, size=(P, P)).astype(np.int64)
    cap = np.full(P, 1 << 62, np.int64)
    out, ms, bub, peak = R.advance_w(prob, costs, mem, cap, link, recs, NTHREADS)
    assert (out == recs).all()
    ms2, bub2, peak2 = R.sim_batch_mem(prob, costs, mem, link, recs, NTHREADS)
    assert (ms == ms2).all() and (bub == bub2).all() and (peak == peak2).all()


def _eligible(q, p, act, split):
    """W entries after position p whose B precedes p, in queue order (their stages hold
    activations)."""
    posB = {(s, m): i for i, (k, s, m) in enumerate(q) if k == KB}
    return [j for j in range(p + 1, len(q))
            if q[j][0] == KW and act[q[j][1]] > 0 and posB[(q[j][1], q[j][2])] < p]


def _stage_mem(rec, P, v_max, max_pert, mem, L):
    c = I.unpack_record(rec, P, v_max, max_pert)
    b = c["b"] + [L]
    S = P * c["v"]
    act = [int(mem[b[s]:b[s + 1], 0].sum()) for s in range(S)]
    stat = [int(mem[b[s]:b[s + 1], 1].sum()) for s in range(S)]
    return c, act, stat


def test_every_advance_follows_the_rule():
    """Replays each output record's appended moves one by one: each move takes the first W
    (queue order) at the first-peak position of the lowest over-capacity device whose advance
    does not lengthen the makespan, else the first eligible W; the search stops only when all
    devices fit, nothing is eligible, or the record has no free perturbation slot."""
    rng = np.random.default_rng(11)
    L, P, v_max, M, mp = 14, 3, 2, 6, 24
    recs = I.random_candidates(rng, L, P, v_max, M, 80, max_pert=2, pert_rate=0.3,
                               policies=(3, 3, 3, 1))
    stride = I.record_stride(P, v_max, mp)
    recs = np.concatenate([recs, np.zeros((len(recs), stride - recs.shape[1]), np.uint8)], axis=1)
    prob = R.problem(L, P, v_max, M, stride, mp)
    costs = rng.integers(1, 5, size=(L, 3)).astype(np.int64) * 1000
    mem = np.stack([rng.integers(1, 100, L), rng.integers(0, 50, L)], axis=1)
    link = rng.integers(0, 3000, size=(P, P)).astype(np.int64)
    ms0, _, peak0 = R.sim_batch_mem(prob, costs, mem, link, recs)
    cap = np.percentile(peak0[ms0 > 0], 30, axis=0).astype(np.int64)
    out, ms, bub, peak = R.advance_w(prob, costs, mem, cap, link, recs, NTHREADS)
    moved = choices = 0
    for i in range(len(recs)):
        if ms0[i] < 0:
            assert (out[i] == recs[i]).all() and ms[i] == ms0[i]
            continue
        c0 = I.unpack_record(recs[i], P, v_max, mp)
        c1, act, stat = _stage_mem(out[i], P, v_max, mp, mem, L)
        split = c1["policy"] == I.POLICY["ZB"]
        assert c1["pert"][:c0["n_pert"]] == c0["pert"]
        extra = c1["pert"][c0["n_pert"]:]
        cur = recs[i].copy()
        for k, (d, j, p) in enumerate(extra):
            q = R.dump_queues(prob, cur)
            dm = [sum(stat[s] for s in range(len(stat)) if c1["dev"][s] == e) for e in range(P)]
            hi = [walk(q[e], act, split) for e in range(P)]
            over = [e for e in range(P) if dm[e] + hi[e][0] > cap[e]]
            assert over and over[0] == d and hi[d][1] == p
            el = _eligible(q[d], p, act, split)
            assert j in el
            base_ms = R.sim_batch(prob, costs, link, cur[None])[0][0]
            trial = []
            for jj in el:
                r2 = cur.copy()
                r2[2] += 1
                n = int(r2[2]) - 1
                po = I.pert_offset(P, v_max) + 6 * n
                r2[po:po + 6] = np.array([d, jj, p], np.uint16).view(np.uint8)
                trial.append(R.sim_batch(prob, costs, link, r2[None])[0][0])
                if jj == j:
                    nxt = r2
            ok = [t <= base_ms for t in trial]
            want = el[ok.index(True)] if any(ok) else el[0]
            assert j == want
            choices += len(el) > 1
            cur = nxt
            moved += 1
        assert (cur == out[i]).all()
        q = R.dump_queues(prob, cur)
        dm = [sum(stat[s] for s in range(len(stat)) if c1["dev"][s] == e) for e in range(P)]
        hi = [walk(q[e], act, split) for e in range(P)]
        assert [dm[e] + hi[e][0] for e in range(P)] == list(peak[i])
        over = [e for e in range(P) if peak[i][e] > cap[e]]
        if over and c1["n_pert"] < mp:
            assert not _eligible(q[over[0]], hi[over[0]][1], act, split)
    assert moved > 30 and choices > 5


def test_fused_schedules_and_static_overflow():
    """Fused backward frees activations at B: there is no W to advance. A device whose capacity
    is below its static bytes gets every advance that lowers its peak (it ends in the eager
    order, one micro-batch held) and stays over; a device with nothing eligible stops the
    search."""
    P, M = 4, 8
    prob, recs = one_stage_per_device(P, M, I.POLICY["1F1B"], 10)
    costs = np.tile(np.array([[300, 500, 200]], np.int64), (P, 1))
    mem = np.tile(np.array([[1000, 50]], np.int64), (P, 1))
    link = I.link_matrix(P, 40)
    out, ms, _, peak = R.advance_w(prob, costs, mem, np.full(P, 1050), link, recs)
    assert (out == recs).all() and (peak[0] == 50 + 1000 * np.minimum(P - np.arange(P), M)).all()
    prob, recs = one_stage_per_device(P, M, I.POLICY["ZB"], 40)
    big = 1 << 40
    out, ms, _, peak = R.advance_w(prob, costs, mem, np.array([big, big, big, 10]), link, recs)
    q = R.dump_queues(prob, out[0])
    assert peak[0].tolist() == [50 + 1000 * min(P, M)] * 3 + [50 + 1000]
    assert q[3] == eager_zb_queue(P, 3, M)
    assert q[:3] == R.dump_queues(prob, recs[0])[:3]
    # the lowest over-capacity device has nothing eligible (rank 0 already releases eagerly)
    out, ms, _, peak = R.advance_w(prob, costs, mem, np.full(P, 10), link, recs)
    assert (out == recs).all() and (peak[0] == 50 + 1000 * min(P, M)).all()


def test_tune_with_room_is_the_plain_search():
    """With capacity to spare, the memory-constrained search makes the plain search's moves."""
    w = I.WORKLOADS[5]
    P, v, M, L = 4, 2, 8, 24
    rng = np.random.default_rng(3)
    recs = I.random_candidates(rng, L, P, v, M, 60, policies=(2, 3))
    prob = R.problem(L, P, v, M, recs.shape[1], 0)
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    mem = np.stack([rng.integers(0, 1 << 30, L), rng.integers(0, 1 << 34, L)], axis=1)
    link = I.link_matrix(P, w.link_ns)
    a = R.tune(prob, costs, link, recs, 9, 30, NTHREADS, want_queues=True)
    b = R.tune_mem(prob, costs, mem, np.full(P, 1 << 62), 50, link, recs, 9, 30, NTHREADS,
                   want_queues=True)
    assert (a[0] == b[0]).all() and (a[1] == b[1]).all() and (a[2] == b[2]).all()
    assert (a[3] == b[4]).all() and (a[4] == b[5]).all()
    assert (a[1] > 0).sum() > 20 and a[3].sum() > 50


def test_tune_keeps_states_within_capacity():
    """Every accepted state fits; its peaks are those of its final queues (order walk)."""
    P, v, M, L = 4, 2, 8, 24
    rng = np.random.default_rng(4)
    recs = I.random_candidates(rng, L, P, v, M, 60, policies=(3,))
    recs = recs[[I.unpack_record(r, P, v, 0)["v"] == 2 for r in recs]]
    prob = R.problem(L, P, v, M, recs.shape[1], 0)
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    mem = np.stack([rng.integers(1, 1000, L), rng.integers(0, 100, L)], axis=1)
    link = I.link_matrix(P, 50_000)
    _, _, pk0 = R.sim_batch_mem(prob, costs, mem, link, recs)
    cap = np.percentile(pk0, 50, axis=0).astype(np.int64)
    out, ms, bub, peak, acc, qs = R.tune_mem(prob, costs, mem, cap, 64, link, recs, 21, 40,
                                             NTHREADS, want_queues=True)
    fit = (ms > 0) & (peak <= cap).all(axis=1)
    # a state is only ever replaced by one that fits
    assert (fit[acc > 0]).all() and fit.sum() > 10 and acc.sum() > 50
    for i in np.nonzero(ms > 0)[0]:
        c, act, stat = _stage_mem(out[i], P, v, 0, mem, L)
        S = P * c["v"]
        split = c["policy"] == I.POLICY["ZB"]
        for d in range(P):
            st = [s for s in range(S) if c["dev"][s] == d]
            q = [(x >> 14, st[(x >> 11) & 7], x & 2047) for x in qs[i, d, :(3 if split else 2) * c["v"] * M]]
            hi, _ = walk(q, act, split)
            assert peak[i, d] == sum(stat[s] for s in st) + hi
