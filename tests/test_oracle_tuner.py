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
