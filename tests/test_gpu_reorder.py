"""octo_sim_batch_reorder (the executor's three-step reordering of the communication, handshake
transfers) vs the CPU oracle: makespan, bubbles and the two counts element by element (bit-exact
int64), through the C ABI."""
import os

import numpy as np
import pytest

from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

pytestmark = pytest.mark.gpu
NTHREADS = min(16, os.cpu_count() or 1)


@pytest.fixture(scope="module")
def gpu():
    import torch
    from paper_2509_23722_amd import _lib
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    _lib.lib()
    return torch.device("cuda:0")


def log(msg):
    print(msg, flush=True)


def run_gpu(dev, L, P, v_max, M, max_pert, costs, link, recs, fn="sim_batch_reorder"):
    import torch
    from paper_2509_23722_amd import _lib
    prob = _lib.problem(L, P, v_max, M, recs.shape[1], max_pert)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    out = getattr(_lib, fn)(prob, t(costs), t(link), t(recs))
    torch.cuda.synchronize()
    return tuple(x.cpu().numpy() for x in out)


def run_oracle(L, P, v_max, M, max_pert, costs, link, recs):
    prob = R.problem(L, P, v_max, M, recs.shape[1], max_pert)
    return R.sim_batch_reorder(prob, costs, link, recs, nthreads=NTHREADS)


def assert_same(g, r, label):
    bad = np.nonzero((g[0] != r[0]) | (g[1] != r[1]).any(axis=1) | (g[2] != r[2]).any(axis=1))[0]
    if len(bad):
        i = int(bad[0])
        raise AssertionError(f"{label}: {len(bad)}/{len(g[0])} differ; first {i}: gpu ms "
                             f"{g[0][i]} stats {g[2][i].tolist()} oracle ms {r[0][i]} stats "
                             f"{r[2][i].tolist()}")


def test_workload1_all_candidates(gpu):
    """Every candidate of the tiny exhaustive batch (the naive coordination deadlocks all 1F1B
    ones): every one runs, no faster than asynchronous transfers."""
    w = I.WORKLOADS[1]
    log("reorder: workload 1")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w)
    args = (w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    g = run_gpu(gpu, *args)
    assert_same(g, run_oracle(*args), "workload 1")
    plain = run_gpu(gpu, *args, fn="sim_batch")
    assert (g[0] >= plain[0]).all() and (g[0] > 0).all() and (g[2][:, 1] > 0).any()


@pytest.mark.parametrize("P,v_max,M,L,pert", [
    (1, 1, 1, 1, 0), (2, 2, 2, 5, 2), (4, 2, 8, 12, 3), (4, 3, 4, 14, 2), (5, 1, 7, 9, 2),
    (8, 2, 16, 20, 2), (8, 4, 8, 40, 2), (16, 2, 16, 40, 2), (12, 1, 24, 20, 2),
    (4, 1, 5, 8, 1), (2, 2, 33, 8, 1), (8, 2, 17, 20, 1), (8, 1, 32, 20, 1), (4, 2, 64, 16, 1),
    (3, 8, 4, 30, 1), (2, 1, 1, 4, 2), (3, 2, 1, 9, 2), (32, 2, 8, 70, 1),
    (64, 1, 64, 255, 1), (32, 2, 37, 255, 1),
])
def test_random_structures(gpu, P, v_max, M, L, pert):
    """Every policy, placement kind and v, moves (some cyclic), invalid records, zero-cost
    links and zero-length ops (ties of the producer ends, broken by the level)."""
    rng = np.random.default_rng(9900 + 1000 * P + 10 * v_max + M)
    log(f"reorder: random P={P} v_max={v_max} M={M} L={L}")
    costs = rng.integers(0, 3_000_000, size=(L, 3)).astype(np.int64)
    costs[rng.random(L) < 0.1] = 0
    link = rng.integers(0, 2_000_000, size=(P, P)).astype(np.int64)
    link[rng.random((P, P)) < 0.2] = 0
    recs = I.random_candidates(rng, L, P, v_max, M, 300, max_pert=pert, pert_rate=0.3,
                               invalid_rate=0.1)
    args = (L, P, v_max, M, pert, costs, link, recs)
    assert_same(run_gpu(gpu, *args), run_oracle(*args), f"P={P} v_max={v_max} M={M}")


def test_workload3_every_candidate(gpu):
    """The 1,048,576-candidate P = 8, M = 64 batch, every candidate against the oracle; every
    candidate runs, no faster than asynchronous transfers."""
    w = I.WORKLOADS[3]
    log("reorder: workload 3")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w)
    g = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    plain = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs, fn="sim_batch")
    assert (g[0] > 0).all() and (g[0] >= plain[0]).all()
    r = run_oracle(w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(g, r, "workload 3, every candidate")


def test_workload4_and_huge(gpu):
    """The whole P = 16, M = 128 batch (cyclic moves deadlock on both sides), and times beyond
    40 bits."""
    w = I.WORKLOADS[4]
    log("reorder: workload 4")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w)
    g = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    r = run_oracle(w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(g, r, "workload 4, every candidate")
    for M in (8, 32):
        rng = np.random.default_rng(226 + M)
        P, v_max, L = 4, 2, 12
        costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
        costs[5] = [40_000_000_000, 30_000_000_000, 20_000_000_000]
        link = I.link_matrix(P, 20_000_000_000)
        recs = I.random_candidates(rng, L, P, v_max, M, 300, max_pert=1, pert_rate=0.1)
        args = (L, P, v_max, M, 1, costs, link, recs)
        g = run_gpu(gpu, *args)
        assert_same(g, run_oracle(*args), f"huge M={M}")
        assert (g[0] > (1 << 37)).sum() > 10
