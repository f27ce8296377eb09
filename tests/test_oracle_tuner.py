"""Properties of the oracle's local search (§6: every move is re-simulated; a move is kept
only if it does not lengthen the pipeline)."""
import numpy as np

from oracle import octoref as R
from paper_2509_23722_amd import inputs as I


def test_tuner_is_monotone_and_consistent():
    rng = np.random.default_rng(2)
    P, v, M, L = 4, 2, 8, 16
    costs = rng.integers(100_000, 3_000_000, size=(L, 3)).astype(np.int64)
    link = I.link_matrix(P, 250_000)
    recs = I.random_candidates(rng, L, P, v, M, 60, policies=(1, 2, 3))
    prob = R.problem(L, P, v, M, recs.shape[1], 0)
    init_ms, _ = R.sim_batch(prob, costs, link, recs)
    prev = init_ms
    for steps in (5, 15, 40):
        recs_f, ms, bub, acc, queues = R.tune(prob, costs, link, recs, 99, steps, want_queues=True)
        assert (ms <= prev).all()          # acceptance never lengthens the pipeline
        assert (acc <= steps).all()
        prev = ms
    # the final state re-simulates to the reported makespan and bubbles: record + queues
    for i in range(len(recs)):
        f = I.unpack_record(recs_f[i], P, v, 0)
        S = P * f["v"]
        b = f["b"] + [L]
        Fs = [int(costs[b[s]:b[s + 1], 0].sum()) for s in range(S)]
        Bs = [int(costs[b[s]:b[s + 1], 1].sum()) for s in range(S)]
        Ws = [int(costs[b[s]:b[s + 1], 2].sum()) for s in range(S)]
        A = [[s for s in range(S) if f["dev"][s] == d] for d in range(P)]
        split = f["policy"] == 3
        qlen = (3 if split else 2) * f["v"] * M
        qs = [[(int(e) >> 14, A[d][(int(e) >> 11) & 7], int(e) & 0x7FF)
               for e in queues[i, d, :qlen]] for d in range(P)]
        rc, m2, b2, _, _ = R.sim_queues(P, S, M, split, f["dev"], Fs, Bs, Ws, link, qs)
        assert rc == 0 and m2 == ms[i] and list(b2) == list(bub[i])


def test_tuner_moves_follow_philox_draws():
    """Step 1 of a chain applies exactly the move its Philox draw selects."""
    P, v, M, L = 4, 1, 4, 8
    costs = np.full((L, 3), 1000, dtype=np.int64)
    link = I.link_matrix(P, 0)
    rec = I.pack_records(P, v, 0, [1], [1], [[2, 4, 6]], [[0, 1, 2, 3]])
    prob = R.problem(L, P, v, M, rec.shape[1], 0)
    seed = 1234
    for chain in range(6):
        recs = np.repeat(rec, chain + 1, axis=0)
        out, ms, _, acc, q = R.tune(prob, costs, link, recs, seed, 1, want_queues=True)
        u = R.philox4x64_10([chain, 1, 0, 0], [seed, 0])
        kind = u[0] % 3
        f = I.unpack_record(out[chain], P, v, 0)
        if kind == 0:
            i = 1 + u[1] % (P * v - 1)
            moved = f["b"][i] != [0, 2, 4, 6][i]
            assert moved == bool(acc[chain])
        elif kind == 1:
            assert sorted(f["dev"]) == [0, 1, 2, 3]
        else:
            assert acc[chain] in (0, 1)


# ---------------------------------------------------------------------------------------------
# Hand-worked pins of move kinds 1 and 2 on the two-stage example of §3.2 (Fig. 3)
# ---------------------------------------------------------------------------------------------

def _numpy_draw(seed, chain, step):
    """(u0, u1, u2, u3) for counter (chain, step, 0, 0), key (seed, 0) from numpy's own
    Philox4x64-10, which produces the block after the counter it holds."""
    if chain:
        ctr = [chain - 1, step, 0, 0]
    else:
        ctr = [2**64 - 1, step - 1, 0, 0]
    bg = np.random.Philox(key=np.array([seed, 0], dtype=np.uint64),
                          counter=np.array(ctr, dtype=np.uint64))
    return [int(x) for x in bg.random_raw(4)]


def _seed_for(want):
    """The smallest seed whose step-1 draw of chain 0 satisfies want(u)."""
    for seed in range(1, 100_000):
        if want(_numpy_draw(seed, 0, 1)):
            return seed
    raise AssertionError("no seed found")


def _fig3_chain():
    from conftest import read_golden
    kv, _ = read_golden("tuner_moves_fig3.txt")
    T = int(kv["T_ns"])
    rec = I.pack_records(2, 1, 0, [I.POLICY["1F1B"]], [1], [[1]], [[0, 1]])
    prob = R.problem(2, 2, 1, 2, rec.shape[1], 0)
    costs = np.array([[2, 2, 2], [4, 4, 4]], np.int64) * T
    return kv, T, rec, prob, costs, I.link_matrix(2, 0)


def _qrow(queues, d, n=4):
    return [((int(e) >> 14), (int(e) >> 11) & 7, int(e) & 0x7FF) for e in queues[0, d, :n]]


def test_start_state_of_fig3():
    kv, T, rec, prob, costs, link = _fig3_chain()
    out, ms, bub, acc, q = R.tune(prob, costs, link, rec, 1, 0, want_queues=True)
    assert ms[0] == int(kv["start_makespan_T"]) * T and acc[0] == 0
    assert _qrow(q, 0) == [(0, 0, 0), (0, 0, 1), (1, 0, 0), (1, 0, 1)]
    assert _qrow(q, 1) == [(0, 0, 0), (1, 0, 0), (0, 0, 1), (1, 0, 1)]


def test_placement_swap_keeps_each_devices_slot_pattern():
    """Move 1 exchanges the two devices' stage sets; each keeps its queue slot pattern, so the
    proposal deadlocks and is rejected. Swapping the queues too would be a relabelling that is
    accepted with the devices exchanged — the result this pin rules out."""
    kv, T, rec, prob, costs, link = _fig3_chain()
    seed = _seed_for(lambda u: u[0] % 3 == 1)
    out, ms, bub, acc, q = R.tune(prob, costs, link, rec, seed, 1, want_queues=True)
    f = I.unpack_record(out[0], 2, 1, 0)
    assert ms[0] == int(kv["swap_makespan_T"]) * T
    assert acc[0] == int(kv["swap_accepted"])
    assert f["dev"] == [int(x) for x in kv["swap_dev"].split()]
    assert f["dev"] != [int(x) for x in kv["relabel_dev"].split()]
    # the proposal itself, evaluated directly: stage 1 on device 0 with device 0's pattern
    qs = [[(0, 1, 0), (0, 1, 1), (1, 1, 0), (1, 1, 1)], [(0, 0, 0), (1, 0, 0), (0, 0, 1), (1, 0, 1)]]
    rc, *_ = R.sim_queues(2, 2, 2, False, [1, 0], [2 * T, 4 * T], [4 * T, 8 * T], [0, 0], link, qs)
    assert rc == 1  # deadlock


def test_adjacent_swap_accepted_on_equal_makespan():
    """Move 2 on device 1 at index 1: F0 B0 F1 B1 -> F0 F1 B0 B1, makespan 30T again, kept."""
    kv, T, rec, prob, costs, link = _fig3_chain()
    seed = _seed_for(lambda u: u[0] % 3 == 2 and u[1] % 2 == 1 and u[2] % 3 == 1)
    out, ms, bub, acc, q = R.tune(prob, costs, link, rec, seed, 1, want_queues=True)
    assert ms[0] == int(kv["adj_d1_i1_makespan_T"]) * T
    assert acc[0] == int(kv["adj_d1_i1_accepted"])
    assert bub[0].tolist() == [int(x) * T for x in kv["adj_d1_i1_bubble_T"].split()]
    assert _qrow(q, 1) == [(0, 0, 0), (0, 0, 1), (1, 0, 0), (1, 0, 1)]
    assert _qrow(q, 0) == [(0, 0, 0), (0, 0, 1), (1, 0, 0), (1, 0, 1)]


def test_adjacent_swap_rejected_when_longer():
    """Move 2 on device 0 at index 0: F1 F0 B0 B1 runs 32T > 30T, so it is not kept."""
    kv, T, rec, prob, costs, link = _fig3_chain()
    seed = _seed_for(lambda u: u[0] % 3 == 2 and u[1] % 2 == 0 and u[2] % 3 == 0)
    out, ms, bub, acc, q = R.tune(prob, costs, link, rec, seed, 1, want_queues=True)
    assert ms[0] == int(kv["start_makespan_T"]) * T and acc[0] == int(kv["adj_d0_i0_accepted"])
    assert _qrow(q, 0) == [(0, 0, 0), (0, 0, 1), (1, 0, 0), (1, 0, 1)]
    qs = [[(0, 0, 1), (0, 0, 0), (1, 0, 0), (1, 0, 1)], [(0, 1, 0), (1, 1, 0), (0, 1, 1), (1, 1, 1)]]
    rc, m2, *_ = R.sim_queues(2, 2, 2, False, [0, 1], [2 * T, 4 * T], [4 * T, 8 * T], [0, 0],
                              link, qs)
    assert rc == 0 and m2 == int(kv["adj_d0_i0_proposal_T"]) * T
