"""octo_alg1_tune (Algorithm 1 of §6, iterative bubble-aware tuning) vs the oracle's search
(oracle/alg1.py): every record's final bytes, makespan, bubbles, kept moves per phase and
searched iterations, element by element, through the C ABI."""
import os

import numpy as np
import pytest

from oracle import alg1 as A
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


def restride(recs, P, v_max, max_pert):
    """Records widened to hold max_pert moves (the new bytes zero)."""
    out = np.zeros((len(recs), I.record_stride(P, v_max, max_pert)), np.uint8)
    k = min(recs.shape[1], out.shape[1])
    out[:, :k] = recs[:, :k]
    return out


def run_gpu(dev, L, P, v_max, M, max_pert, costs, link, recs, iters):
    import torch
    from paper_2509_23722_amd import _lib
    prob = _lib.problem(L, P, v_max, M, recs.shape[1], max_pert)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    r = t(recs)
    ms, bub, stats = _lib.alg1_tune(prob, t(costs), t(link), r, iters)
    torch.cuda.synchronize()
    return r.cpu().numpy(), ms.cpu().numpy(), bub.cpu().numpy(), stats.cpu().numpy()


def run_oracle(L, P, v_max, M, max_pert, costs, link, recs, iters):
    prob = R.problem(L, P, v_max, M, recs.shape[1], max_pert)
    out, ms, bub, acc, used = A.tune(prob, costs, link, recs, iters, nthreads=NTHREADS)
    return out, ms, bub, np.concatenate([acc, used[:, None]], axis=1)


def assert_same(g, r, label):
    bad = np.nonzero((g[0] != r[0]).any(axis=1) | (g[1] != r[1]) | (g[2] != r[2]).any(axis=1) |
                     (g[3] != r[3]).any(axis=1))[0]
    if len(bad):
        i = int(bad[0])
        raise AssertionError(
            f"{label}: {len(bad)}/{len(g[1])} records differ; first {i}: gpu ms {g[1][i]} "
            f"stats {g[3][i].tolist()} oracle ms {r[1][i]} stats {r[3][i].tolist()}; records "
            f"equal: {bool((g[0][i] == r[0][i]).all())}")


def check(dev, L, P, v_max, M, max_pert, costs, link, recs, iters, label):
    args = (L, P, v_max, M, max_pert, costs, link, recs, iters)
    g = run_gpu(dev, *args)
    r = run_oracle(*args)
    assert_same(g, r, label)
    return g


@pytest.mark.parametrize("P,v_max,M,L,max_pert,iters", [
    (4, 2, 8, 24, 6, 40), (2, 2, 4, 9, 3, 30), (4, 1, 6, 11, 2, 25), (3, 2, 5, 13, 4, 30),
    (8, 2, 16, 40, 2, 12), (1, 2, 4, 6, 2, 10), (4, 4, 8, 40, 2, 15), (5, 1, 7, 9, 0, 20),
    (16, 2, 16, 60, 2, 10), (32, 2, 8, 255, 2, 6), (64, 1, 8, 255, 2, 4),
])
def test_random_searches(gpu, P, v_max, M, L, max_pert, iters):
    """Random candidates of every policy, placement kind and v, some with moves or invalid, on
    heterogeneous costs and non-uniform links: the same search step for step."""
    rng = np.random.default_rng(9100 + 100 * P + 10 * v_max + M)
    log(f"alg1: random P={P} v_max={v_max} M={M} L={L} max_pert={max_pert} iters={iters}")
    costs = rng.integers(100_000, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 600_000, size=(P, P)).astype(np.int64)
    recs = I.random_candidates(rng, L, P, v_max, M, 40, max_pert=max_pert, pert_rate=0.2,
                               invalid_rate=0.1)
    g = check(gpu, L, P, v_max, M, max_pert, costs, link, recs, iters, f"P={P} v_max={v_max}")
    ms0 = R.sim_batch(R.problem(L, P, v_max, M, recs.shape[1], max_pert), costs, link, recs)[0]
    ok = ms0 >= 0
    assert (g[1][ok] <= ms0[ok]).all() and (g[1][~ok] == ms0[~ok]).all()
    assert (g[3][~ok] == 0).all() and (g[0][~ok] == recs[~ok]).all()


def test_reserved_bytes_and_trailing_bytes(gpu):
    """Garbage in the reserved boundary / placement bytes and after the moves: neighbours read
    the reserved bytes as zero and copy the rest, so the final records match byte for byte."""
    rng = np.random.default_rng(9201)
    P, v_max, M, L, mp = 4, 2, 8, 24, 3
    log("alg1: reserved bytes")
    costs = rng.integers(100_000, 3_000_000, size=(L, 3)).astype(np.int64)
    link = I.link_matrix(P, 150_000)
    recs = I.random_candidates(rng, L, P, v_max, M, 30, max_pert=mp, policies=(0, 1, 2, 3))
    s_max, po = P * v_max, I.pert_offset(P, v_max)
    for rec in recs:
        S = P * int(rec[1])
        rec[3 + S:3 + s_max] = rng.integers(1, 256, size=s_max - S)
        rec[3 + s_max + S:3 + 2 * s_max] = rng.integers(1, 256, size=s_max - S)
        rec[po + 6 * int(rec[2]):] = rng.integers(0, 256, size=len(rec) - po - 6 * int(rec[2]))
    check(gpu, L, P, v_max, M, mp, costs, link, recs, 25, "reserved bytes")


def test_zero_iterations_and_sentinels(gpu):
    """iters = 0 only evaluates; invalid and deadlocked records never search."""
    rng = np.random.default_rng(9202)
    P, v_max, M, L, mp = 4, 2, 8, 16, 2
    log("alg1: zero iterations, sentinels")
    costs = rng.integers(100_000, 3_000_000, size=(L, 3)).astype(np.int64)
    link = I.link_matrix(P, 100_000)
    recs = I.random_candidates(rng, L, P, v_max, M, 60, max_pert=mp, pert_rate=0.5,
                               invalid_rate=0.3)
    g0 = check(gpu, L, P, v_max, M, mp, costs, link, recs, 0, "iters 0")
    assert (g0[0] == recs).all() and (g0[3] == 0).all()
    g = check(gpu, L, P, v_max, M, mp, costs, link, recs, 30, "sentinels")
    bad = g0[1] < 0
    assert bad.any() and (g[1][bad] == g0[1][bad]).all() and (g[3][bad] == 0).all()


def test_benchmark_shape(gpu):
    """Records of the 1,048,576-candidate P = 8, M = 64 workload (52 layers, v <= 2), widened to
    four move slots: the search on the GPU equals the oracle's on 16 records of every stratum."""
    w = I.WORKLOADS[3]
    log("alg1: workload 3, 256 records")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w)
    rng = np.random.default_rng(9203)
    strata = recs[:, 1].astype(np.int64) * 4 + recs[:, 0]
    pick = np.concatenate([rng.choice(np.nonzero(strata == s)[0], size=16, replace=False)
                           for s in np.unique(strata)])
    sub = restride(recs[pick], w.P, w.v_max, 4)
    g = check(gpu, w.L, w.P, w.v_max, w.M, 4, costs, link, sub, 30, "workload 3")
    assert (g[3][:, :3].sum(axis=1) > 0).all()


def test_empty_batch(gpu):
    import torch
    from paper_2509_23722_amd import _lib
    prob = _lib.problem(8, 2, 1, 4, I.record_stride(2, 1, 0), 0)
    z = torch.zeros((0, prob.cand_stride), dtype=torch.uint8, device=gpu)
    c = torch.ones((8, 3), dtype=torch.int64, device=gpu)
    ms, bub, st = _lib.alg1_tune(prob, c, torch.zeros((2, 2), dtype=torch.int64, device=gpu), z, 5)
    torch.cuda.synchronize()
    assert ms.numel() == 0 and st.numel() == 0


@pytest.mark.parametrize("flags", [0, 2, 3])
def test_options_random_phase_and_no_insertion(gpu, flags):
    """octo_alg1_tune_ex: insertions off (0), random phases without (2) and with (3)
    insertions: the same search step for step as the oracle with those options, per-phase
    iteration counts included."""
    import torch
    from paper_2509_23722_amd import _lib
    rng = np.random.default_rng(9300 + flags)
    P, v_max, M, L, mp, iters, seed = 4, 2, 8, 24, 4, 30, 4242 + flags
    log(f"alg1: options flags={flags}")
    costs = rng.integers(100_000, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 900_000, size=(P, P)).astype(np.int64)
    recs = I.random_candidates(rng, L, P, v_max, M, 48, max_pert=mp, pert_rate=0.2,
                               invalid_rate=0.05)
    prob = _lib.problem(L, P, v_max, M, recs.shape[1], mp)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(gpu)
    r = t(recs)
    ms, bub, stats, pit = _lib.alg1_tune_ex(prob, t(costs), t(link), r, iters, flags, seed)
    torch.cuda.synchronize()
    g = (r.cpu().numpy(), ms.cpu().numpy(), bub.cpu().numpy(), stats.cpu().numpy())
    rprob = R.problem(L, P, v_max, M, recs.shape[1], mp)
    opit = np.zeros((len(recs), 3), np.int64)
    out, oms, obub, acc, used = A.tune(rprob, costs, link, recs, iters, nthreads=NTHREADS,
                                      random_search=bool(flags & 2), seed=seed,
                                      insert=bool(flags & 1), phase_iters=opit)
    assert_same(g, (out, oms, obub, np.concatenate([acc, used[:, None]], axis=1)),
                f"flags={flags}")
    assert (pit.cpu().numpy() == opit).all()


def test_insertion_worked_example_on_gpu(gpu):
    """The hand-worked insertion (tests/golden/overlap_insertion_example.txt): one iteration
    keeps the move (0, 4, 2) at 30T."""
    import torch
    from paper_2509_23722_amd import _lib
    from conftest import read_golden
    kv, _ = read_golden("overlap_insertion_example.txt")
    T = int(kv["T_ns"])
    recs = I.pack_records(2, 1, 2, [I.POLICY["ZB"]], [1], [[1]], [[0, 1]])
    prob = _lib.problem(2, 2, 1, 3, recs.shape[1], 2)
    costs = np.array([[1, 4, 1], [2, 4, 2]], np.int64) * T
    link = I.link_matrix(2, int(kv["transfer_T"]) * T)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(gpu)
    r = t(recs)
    ms, _, stats = _lib.alg1_tune(prob, t(costs), t(link), r, 1)
    torch.cuda.synchronize()
    rec = r.cpu().numpy()[0]
    po = I.pert_offset(2, 1)
    assert int(ms[0]) == int(kv["after_makespan_T"]) * T and int(rec[2]) == 1
    assert np.frombuffer(bytes(rec[po:po + 6]), np.uint16).tolist() == \
        [int(x) for x in kv["insertion"].split()]
