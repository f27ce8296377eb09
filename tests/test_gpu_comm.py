"""octo_sim_batch_comm (communication nodes and their overlap) vs the CPU oracle: makespan,
bubbles and the four communication figures, element by element (bit-exact int64), through the
C ABI."""
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


def run_gpu(dev, L, P, v_max, M, max_pert, costs, link, recs):
    import torch
    from paper_2509_23722_amd import _lib
    prob = _lib.problem(L, P, v_max, M, recs.shape[1], max_pert)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    ms, bub, comm = _lib.sim_batch_comm(prob, t(costs), t(link), t(recs))
    torch.cuda.synchronize()
    return ms.cpu().numpy(), bub.cpu().numpy(), comm.cpu().numpy()


def run_oracle(L, P, v_max, M, max_pert, costs, link, recs):
    prob = R.problem(L, P, v_max, M, recs.shape[1], max_pert)
    return R.sim_batch_comm(prob, costs, link, recs, nthreads=NTHREADS)


def assert_same(g, r, label):
    bad = np.nonzero((g[0] != r[0]) | (g[1] != r[1]).any(axis=1) | (g[2] != r[2]).any(axis=1))[0]
    if len(bad):
        i = int(bad[0])
        raise AssertionError(f"{label}: {len(bad)}/{len(g[0])} differ; first {i}: gpu ms {g[0][i]} "
                             f"comm {g[2][i].tolist()} oracle ms {r[0][i]} comm {r[2][i].tolist()}")


def test_workload1_all_candidates(gpu):
    w = I.WORKLOADS[1]
    log("comm: workload 1")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w)
    args = (w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    g = run_gpu(gpu, *args)
    assert_same(g, run_oracle(*args), "workload 1")
    assert (g[2][:, 1] > 0).all()


@pytest.mark.parametrize("P,v_max,M,L,pert", [
    (1, 1, 1, 1, 0), (2, 2, 2, 5, 2), (4, 2, 8, 12, 3), (4, 3, 4, 14, 2), (5, 1, 7, 9, 2),
    (8, 2, 16, 20, 2), (8, 4, 8, 40, 2), (16, 2, 16, 40, 2), (12, 1, 24, 20, 2),
    (4, 1, 5, 8, 1), (2, 2, 33, 8, 1), (8, 2, 17, 20, 1), (8, 1, 32, 20, 1), (4, 2, 64, 16, 1),
    (64, 1, 64, 255, 1), (64, 1, 45, 255, 1), (32, 2, 37, 255, 1),
])
def test_random_structures(gpu, P, v_max, M, L, pert):
    """Every policy, placement kind and v (table-driven, generated, GPipe and materialised
    paths), moves (some cyclic), invalid records, links with zeros."""
    rng = np.random.default_rng(8000 + 1000 * P + 10 * v_max + M)
    log(f"comm: random P={P} v_max={v_max} M={M} L={L}")
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 800_000, size=(P, P)).astype(np.int64)
    link[rng.random((P, P)) < 0.2] = 0
    recs = I.random_candidates(rng, L, P, v_max, M, 300, max_pert=pert, pert_rate=0.3,
                               invalid_rate=0.1)
    args = (L, P, v_max, M, pert, costs, link, recs)
    assert_same(run_gpu(gpu, *args), run_oracle(*args), f"P={P} v_max={v_max} M={M}")


def test_same_times_as_plain_call(gpu):
    import torch
    from paper_2509_23722_amd import _lib
    w = I.WORKLOADS[2]
    log("comm: workload 2, times vs plain call")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w, 20000)
    g = run_gpu(gpu, w.L, w.P, w.v_max, w.M, 0, costs, link, recs)
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], 0)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(gpu)
    ms, bub = _lib.sim_batch(prob, t(costs), t(link), t(recs))
    assert (ms.cpu().numpy() == g[0]).all() and (bub.cpu().numpy() == g[1]).all()
    r = run_oracle(w.L, w.P, w.v_max, w.M, 0, costs, link, recs)
    assert_same(g, r, "workload 2, every candidate")


def test_workload3_full_size(gpu):
    """The 1,048,576-candidate batch: every candidate against the oracle; for all of them the
    node count is 4 M per cross-device stage boundary and overlaps are bounded by the nodes."""
    w = I.WORKLOADS[3]
    log("comm: workload 3")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w)
    g = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    v = recs[:, 1].astype(np.int64)
    S = w.P * v
    dev = recs[:, 3 + w.s_max:3 + 2 * w.s_max].astype(np.int64)
    idx = np.arange(w.s_max - 1)
    cross = ((dev[:, :-1] != dev[:, 1:]) & (idx[None, :] < (S - 1)[:, None])).sum(axis=1)
    assert (g[2][:, 0] == 4 * w.M * cross).all()
    assert (g[2][:, 2] == 4 * w.M * cross * w.link_ns).all()
    assert (g[2][:, 1] <= g[2][:, 0]).all() and (g[2][:, 3] <= g[2][:, 2]).all()
    r = run_oracle(w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(g, r, "workload 3, every candidate")


def test_workload4_every_candidate(gpu):
    w = I.WORKLOADS[4]
    log("comm: workload 4")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w)
    g = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    cyc = recs[:, 2] > 0
    assert (g[2][cyc] == -1).all() and (g[2][~cyc, 0] > 0).all()
    r = run_oracle(w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(g, r, "workload 4, every candidate")


def test_beyond_32_and_40_bits(gpu):
    """Transfers longer than 2^32 ns (table streams are 32-bit) and times beyond the 40-bit
    slots are recomputed on the 64-bit path with their tallies."""
    rng = np.random.default_rng(122)
    P, v_max, M, L = 4, 2, 8, 12
    log("comm: huge costs and links")
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    costs[5] = [40_000_000_000, 30_000_000_000, 20_000_000_000]
    link = I.link_matrix(P, 1000)
    link[1, 2] = 5_000_000_000
    recs = I.random_candidates(rng, L, P, v_max, M, 300, max_pert=1, pert_rate=0.1)
    args = (L, P, v_max, M, 1, costs, link, recs)
    assert_same(run_gpu(gpu, *args), run_oracle(*args), "huge")
