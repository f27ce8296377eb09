"""Pins of the oracle's memory model (§5 memory nodes, §6 Eq. 2 peak memory per device).

Each forward F(s,m) allocates stage s's activations for micro-batch m when it starts; the last
backward op of (s,m) (B fused, W split) releases them when it ends; static bytes stay resident.
The oracle replays these events in time order from its simulated start times. These tests pin
it to closed forms of the textbook schedules and to properties that hold for any schedule.
"""
import numpy as np
import pytest

from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

NTHREADS = 4


def one_stage_per_device(P, M, pol, act, stat, costs=None, rng=None):
    """P devices, one layer per stage (identity placement), per-layer memory act/stat."""
    L = P
    costs = np.full((L, 3), 1000, np.int64) if costs is None else costs
    mem = np.stack([np.asarray(act, np.int64), np.asarray(stat, np.int64)], axis=1)
    recs = I.pack_records(P, 1, 0, [pol], [1], [np.arange(1, P)], [np.arange(P)])
    prob = R.problem(L, P, 1, M, recs.shape[1], 0)
    return R.sim_batch_mem(prob, costs, mem, I.link_matrix(P, 50_000), recs, 1)


@pytest.mark.parametrize("P,M", [(1, 3), (2, 2), (4, 8), (4, 3), (8, 16), (5, 5)])
def test_gpipe_holds_every_microbatch(P, M):
    """AFAB runs all forwards before any backward: each device holds all M micro-batches."""
    act = np.arange(1, P + 1) * 1000
    stat = np.arange(P) * 7 + 3
    _, _, peak = one_stage_per_device(P, M, I.POLICY["AFAB"], act, stat)
    assert (peak[0] == stat + M * act).all()


@pytest.mark.parametrize("P,M", [(1, 3), (2, 2), (4, 8), (4, 3), (8, 16), (8, 5)])
def test_1f1b_holds_stages_to_go(P, M):
    """1F1B: the device of stage s warms up with S-1-s forwards, so it holds min(S - s, M)
    micro-batches at its peak (the first stage the most)."""
    act = np.full(P, 4096)
    stat = np.zeros(P, np.int64)
    _, _, peak = one_stage_per_device(P, M, I.POLICY["1F1B"], act, stat)
    s = np.arange(P)
    assert (peak[0] == act * np.minimum(P - s, M)).all()


@pytest.mark.parametrize("P,M", [(2, 2), (4, 8), (4, 3), (8, 16)])
def test_zero_bubble_w_lag_holds_S(P, M):
    """Split backward with W deferred by the device's rank r: activations wait for W, which
    trails B by r ops; with warm-up S-1-r every device holds min(S, M) micro-batches."""
    act = np.full(P, 64)
    _, _, peak = one_stage_per_device(P, M, I.POLICY["ZB"], act, np.zeros(P, np.int64))
    assert (peak[0] == 64 * min(P, M)).all()


def test_memory_does_not_depend_on_times():
    """Ops of one device never overlap, so its memory follows its queue order: random costs and
    link weights change the makespan, never the peak."""
    rng = np.random.default_rng(3)
    L, P, v, M = 20, 4, 2, 8
    recs = I.random_candidates(rng, L, P, v, M, 150, max_pert=1, pert_rate=0.3)
    prob = R.problem(L, P, v, M, recs.shape[1], 1)
    mem = np.stack([rng.integers(0, 10_000, L), rng.integers(0, 500, L)], axis=1)
    out = []
    for k in range(3):
        costs = rng.integers(0, 3_000_000, size=(L, 3)).astype(np.int64)
        link = rng.integers(0, 900_000, size=(P, P)).astype(np.int64)
        out.append(R.sim_batch_mem(prob, costs, mem, link, recs, NTHREADS))
    assert (out[0][0] != out[1][0]).any()
    assert (out[0][2] == out[1][2]).all() and (out[0][2] == out[2][2]).all()


def _order_walk(queues, act, stat, dev, split):
    """Peak per device from queue order alone (an independent formulation)."""
    P = len(queues)
    out = []
    for d in range(P):
        cur = hi = 0
        for k, s, m in queues[d]:
            if k == 0:
                cur += act[s]
            elif (k == 1 and not split) or k == 2:
                cur -= act[s]
            hi = max(hi, cur)
        out.append(hi + sum(stat[s] for s in range(len(dev)) if dev[s] == d))
    return out


def test_time_replay_equals_queue_walk():
    """The oracle replays events by time; walking each final queue in order must agree (zero
    costs included, where events share instants)."""
    rng = np.random.default_rng(8)
    L, P, v, M = 14, 3, 2, 4
    recs = I.random_candidates(rng, L, P, v, M, 120, max_pert=2, pert_rate=0.4)
    prob = R.problem(L, P, v, M, recs.shape[1], 2)
    costs = rng.integers(0, 3, size=(L, 3)).astype(np.int64) * 1000
    mem = np.stack([rng.integers(1, 100, L), rng.integers(0, 9, L)], axis=1)
    ms, _, peak = R.sim_batch_mem(prob, costs, mem, I.link_matrix(P, 0), recs, NTHREADS)
    checked = 0
    for i in range(len(recs)):
        if ms[i] < 0:
            continue
        c = I.unpack_record(recs[i], P, v, 2)
        S = P * c["v"]
        b = c["b"] + [L]
        act = [int(mem[b[s]:b[s + 1], 0].sum()) for s in range(S)]
        stat = [int(mem[b[s]:b[s + 1], 1].sum()) for s in range(S)]
        q = R.dump_queues(prob, recs[i])
        want = _order_walk(q, act, stat, list(c["dev"][:S]), c["policy"] == I.POLICY["ZB"])
        assert list(peak[i]) == want, i
        checked += 1
    assert checked > 60


def test_bounds_and_sentinels():
    """static + the largest stage footprint <= peak <= static + M x all its stages' activations;
    deadlocked candidates report -1, invalid ones -2."""
    w = I.WORKLOADS[4]
    recs = I.candidates(w, 3000)
    rng = np.random.default_rng(1)
    mem = np.stack([rng.integers(1, 1 << 30, w.L), rng.integers(0, 1 << 32, w.L)], axis=1)
    prob = R.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], w.max_pert)
    ms, _, peak = R.sim_batch_mem(prob, I.layer_costs(w), mem, I.link_matrix(w.P, w.link_ns),
                                  recs, NTHREADS)
    assert (peak[ms == -1] == -1).all() and (ms == -1).sum() > 10
    for i in np.nonzero(ms > 0)[0][:300]:
        c = I.unpack_record(recs[i], w.P, w.v_max, w.max_pert)
        S = w.P * c["v"]
        b = c["b"] + [w.L]
        for d in range(w.P):
            st = [s for s in range(S) if c["dev"][s] == d]
            a = [int(mem[b[s]:b[s + 1], 0].sum()) for s in st]
            base = sum(int(mem[b[s]:b[s + 1], 1].sum()) for s in st)
            assert base + max(a) <= peak[i, d] <= base + w.M * sum(a)
    bad = recs[:5].copy()
    bad[:, 3] = 1  # flags must be 0
    _, _, pk = R.sim_batch_mem(prob, I.layer_costs(w), mem, I.link_matrix(w.P, w.link_ns), bad, 1)
    assert (pk == -2).all()
