"""HIP path vs the CPU oracle, element by element (bit-exact int64), through the C ABI."""
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


def run_gpu(dev, L, P, v_max, M, max_pert, costs, link, recs):
    import torch
    from paper_2509_23722_amd import _lib
    prob = _lib.problem(L, P, v_max, M, recs.shape[1], max_pert)
    ms, bub = _lib.sim_batch(prob, torch.from_numpy(np.ascontiguousarray(costs)).to(dev),
                             torch.from_numpy(np.ascontiguousarray(link)).to(dev),
                             torch.from_numpy(np.ascontiguousarray(recs)).to(dev))
    torch.cuda.synchronize()
    return ms.cpu().numpy(), bub.cpu().numpy()


def run_oracle(L, P, v_max, M, max_pert, costs, link, recs):
    prob = R.problem(L, P, v_max, M, recs.shape[1], max_pert)
    return R.sim_batch(prob, costs, link, recs, nthreads=NTHREADS)


def assert_same(gms, gbub, rms, rbub, label):
    bad = np.nonzero((gms != rms) | (gbub != rbub).any(axis=1))[0]
    if len(bad):
        i = int(bad[0])
        raise AssertionError(f"{label}: {len(bad)}/{len(gms)} differ; first index {i}: gpu "
                             f"{gms[i]} {gbub[i].tolist()} oracle {rms[i]} {rbub[i].tolist()}")


def log(msg):
    print(msg, flush=True)


def test_workload1_all_candidates(gpu):
    w = I.WORKLOADS[1]
    log(f"workload 1 {w.name}: 910 candidates")
    costs, link, recs = I.layer_costs(w), I.link_matrix(w.P, w.link_ns), I.candidates(w)
    g = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    r = run_oracle(w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(*g, *r, "workload 1")
    assert (g[0] > 0).all()


@pytest.mark.parametrize("P,v_max,M,L,pert", [
    (1, 1, 1, 1, 0), (1, 3, 5, 4, 2), (2, 2, 2, 5, 2), (3, 2, 6, 9, 2), (4, 2, 8, 12, 3),
    (4, 3, 4, 14, 2), (5, 1, 7, 9, 2), (6, 2, 12, 15, 2), (8, 2, 16, 20, 2), (8, 4, 8, 40, 2),
    (7, 3, 14, 30, 1), (16, 2, 16, 40, 2), (16, 4, 4, 64, 1), (32, 2, 8, 70, 1),
    (12, 1, 24, 20, 2), (33, 1, 3, 40, 1), (64, 1, 2, 64, 1), (8, 8, 3, 64, 1),
    # finish-table rows as rings of R = next power of two >= P v slots: M = R + 1, M not a
    # multiple of R, non-power-of-two P, long wraps
    (4, 1, 5, 8, 1), (4, 2, 9, 12, 1), (2, 2, 33, 8, 1), (3, 1, 40, 9, 2), (8, 2, 17, 20, 1),
    (5, 2, 23, 14, 1), (2, 1, 64, 3, 1),
])
def test_random_structures(gpu, P, v_max, M, L, pert):
    """Every policy, placement kind, v, ragged P / M, random moves (some cyclic) and invalid
    records, over many bins and both the generated and the materialised paths."""
    rng = np.random.default_rng(1000 * P + 10 * v_max + M)
    n = 300
    log(f"random structures P={P} v_max={v_max} M={M} L={L} n={n}")
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 800_000, size=(P, P)).astype(np.int64)
    recs = I.random_candidates(rng, L, P, v_max, M, n, max_pert=pert, pert_rate=0.3,
                               invalid_rate=0.1)
    g = run_gpu(gpu, L, P, v_max, M, pert, costs, link, recs)
    r = run_oracle(L, P, v_max, M, pert, costs, link, recs)
    assert_same(*g, *r, f"P={P} v_max={v_max} M={M}")


def test_workload2_all_candidates(gpu):
    w = I.WORKLOADS[2]
    log(f"workload 2 {w.name}: {w.n} candidates")
    costs, link, recs = I.layer_costs(w), I.link_matrix(w.P, w.link_ns), I.candidates(w)
    g = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    r = run_oracle(w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(*g, *r, "workload 2")


def test_workload3_full_size(gpu):
    """The headline workload at full size (1,048,576 candidates, P = 8, M = 64, v in {1, 2}),
    in the launch configuration the benchmark times: every candidate against the oracle, and
    properties that hold for every candidate."""
    w = I.WORKLOADS[3]
    log(f"workload 3 {w.name}: {w.n} candidates")
    costs, link, recs = I.layer_costs(w), I.link_matrix(w.P, w.link_ns), I.candidates(w)
    gms, gbub = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    # every candidate is valid and deadlock-free (policies only)
    assert (gms > 0).all() and (gbub >= 0).all()
    assert (gms[:, None] - gbub > 0).all()
    rms, rbub = run_oracle(w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(gms, gbub, rms, rbub, "workload 3, every candidate")


def test_workload4_full_size(gpu):
    """DeepSeek-V3-like workload at full size: every candidate against the oracle, and exactly
    the 1% deliberately cyclic candidates flagged as deadlocked."""
    w = I.WORKLOADS[4]
    log(f"workload 4 {w.name}: {w.n} candidates")
    costs, link, recs = I.layer_costs(w), I.link_matrix(w.P, w.link_ns), I.candidates(w)
    gms, gbub = run_gpu(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    cyc = recs[:, 2] > 0
    assert cyc.sum() == w.n // 100
    assert (gms[cyc] == -1).all() and (gbub[cyc] == -1).all()
    assert (gms[~cyc] > 0).all() and (gbub[~cyc] >= 0).all()
    rms, rbub = run_oracle(w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(gms, gbub, rms, rbub, "workload 4, every candidate")


def test_edge_cases(gpu):
    """Empty batch, one device, one micro-batch, one layer per stage, zero costs, the largest M
    that fits LDS, S = 64 stages."""
    import torch
    from paper_2509_23722_amd import _lib
    # empty batch: nothing launched, nothing written
    prob = _lib.problem(4, 2, 1, 2, I.record_stride(2, 1, 0), 0)
    z = torch.zeros((0, prob.cand_stride), dtype=torch.uint8, device=gpu)
    ms, bub = _lib.sim_batch(prob, torch.ones((4, 3), dtype=torch.int64, device=gpu),
                             torch.zeros((2, 2), dtype=torch.int64, device=gpu), z)
    assert ms.numel() == 0
    cases = [
        dict(P=1, v_max=1, M=1, L=1), dict(P=2, v_max=1, M=1, L=2), dict(P=4, v_max=2, M=1, L=8),
        dict(P=8, v_max=1, M=2047, L=8), dict(P=8, v_max=8, M=4, L=64),
        dict(P=32, v_max=2, M=32, L=64), dict(P=64, v_max=1, M=16, L=64),
    ]
    for c in cases:
        rng = np.random.default_rng(c["M"] * 7 + c["P"])
        log(f"edge case {c}")
        costs = rng.integers(0, 2, size=(c["L"], 3)).astype(np.int64) * 1000
        link = I.link_matrix(c["P"], 50)
        recs = I.random_candidates(rng, c["L"], c["P"], c["v_max"], c["M"], 40, max_pert=1,
                                   pert_rate=0.2)
        g = run_gpu(gpu, c["L"], c["P"], c["v_max"], c["M"], 1, costs, link, recs)
        r = run_oracle(c["L"], c["P"], c["v_max"], c["M"], 1, costs, link, recs)
        assert_same(*g, *r, f"edge {c}")


@pytest.mark.parametrize("M", [8, 32])
def test_times_beyond_40bit_slots(gpu, M):
    """Layer costs so large that finish times pass 2^37 ns: those candidates are recomputed with
    64-bit finish tables and must still match the oracle exactly; small ones stay fast. At M = 32
    the candidates with moves start on 40-bit rings."""
    rng = np.random.default_rng(21 + M)
    P, v_max, L = 4, 2, 12
    log(f"huge costs P=4 v_max=2 M={M}")
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    costs[5] = [40_000_000_000, 30_000_000_000, 20_000_000_000]  # ~ 2^35 per op of that layer
    link = I.link_matrix(P, 1000)
    recs = I.random_candidates(rng, L, P, v_max, M, 400, max_pert=1, pert_rate=0.1)
    g = run_gpu(gpu, L, P, v_max, M, 1, costs, link, recs)
    r = run_oracle(L, P, v_max, M, 1, costs, link, recs)
    assert_same(*g, *r, "huge costs")
    assert (r[0] >= 2 ** 37).sum() > 50


def test_interleaved_problems_keep_results(gpu):
    """Calls on one stream alternate between problems of different sizes (and v_max, so the
    library's cached MERGE tables must survive calls that do not use them)."""
    rng = np.random.default_rng(31)
    cases = [(4, 2, 8, 12), (8, 1, 32, 40), (4, 2, 8, 30), (6, 2, 6, 20), (4, 2, 8, 16)]
    for P, v_max, M, L in cases * 2:
        log(f"interleaved P={P} v_max={v_max} M={M} L={L}")
        costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
        link = I.link_matrix(P, 300_000)
        recs = I.random_candidates(rng, L, P, v_max, M, 2000 if v_max == 1 else 300)
        g = run_gpu(gpu, L, P, v_max, M, 0, costs, link, recs)
        r = run_oracle(L, P, v_max, M, 0, costs, link, recs)
        assert_same(*g, *r, f"interleaved P={P} v_max={v_max} M={M} L={L}")


def test_repeatable_and_stream_independent(gpu):
    import torch
    w = I.WORKLOADS[2]
    costs, link, recs = I.layer_costs(w), I.link_matrix(w.P, w.link_ns), I.candidates(w, 5000)
    a = run_gpu(gpu, w.L, w.P, w.v_max, w.M, 0, costs, link, recs)
    s = torch.cuda.Stream()
    with torch.cuda.stream(s):
        b = run_gpu(gpu, w.L, w.P, w.v_max, w.M, 0, costs, link, recs)
    assert (a[0] == b[0]).all() and (a[1] == b[1]).all()
