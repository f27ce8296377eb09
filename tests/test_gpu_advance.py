"""Selective W advancing under per-device capacities on the GPU (octo_advance_w) and the
memory-constrained local search (octo_tune_step_mem) vs the CPU oracle, through the C ABI:
output records byte for byte, makespans, bubbles, peaks, accepted moves and queues, bit-exact."""
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


def t_(x, dev):
    import torch
    return torch.from_numpy(np.ascontiguousarray(x)).to(dev)


def widen(recs, P, v_max, max_pert):
    """Records re-strided to hold max_pert moves (existing moves kept)."""
    stride = I.record_stride(P, v_max, max_pert)
    out = np.zeros((len(recs), stride), np.uint8)
    out[:, :recs.shape[1]] = recs
    return out


def run_advance(dev, L, P, v_max, M, mp, costs, mem, cap, link, recs, in_place=False):
    import torch
    from paper_2509_23722_amd import _lib
    prob = _lib.problem(L, P, v_max, M, recs.shape[1], mp)
    src = t_(recs, dev)
    out = src if in_place else torch.full_like(src, 0xA5)
    o = _lib.advance_w(prob, t_(costs, dev), t_(mem, dev), t_(cap, dev), t_(link, dev), src,
                       out_candidates=out)
    torch.cuda.synchronize()
    return tuple(x.cpu().numpy() for x in o)


def check_advance(g, r, label):
    bad = np.nonzero((g[1] != r[1]) | (g[2] != r[2]).any(axis=1) | (g[3] != r[3]).any(axis=1) |
                     (g[0] != r[0]).any(axis=1))[0]
    if len(bad):
        i = int(bad[0])
        raise AssertionError(
            f"{label}: {len(bad)}/{len(g[1])} differ; first {i}: gpu ms {g[1][i]} peak "
            f"{g[3][i].tolist()} n_pert {g[0][i][2]} oracle ms {r[1][i]} peak {r[3][i].tolist()} "
            f"n_pert {r[0][i][2]} record bytes differ at {np.nonzero(g[0][i] != r[0][i])[0][:8]}")


@pytest.mark.parametrize("P,M", [(3, 6), (4, 8), (2, 5), (5, 12)])
def test_capacity_of_1f1b(gpu, P, M):
    """ZB with the 1F1B footprint as capacity: the advances that make W eager."""
    log(f"advance: 1F1B capacity P={P} M={M}")
    A, Z = 1000, 77
    recs = I.pack_records(P, 1, 200, [I.POLICY["ZB"]], [1], [np.arange(1, P)], [np.arange(P)])
    costs = np.tile(np.array([[300, 500, 200]], np.int64), (P, 1))
    mem = np.tile(np.array([[A, Z]], np.int64), (P, 1))
    cap = (Z + A * np.minimum(P - np.arange(P), M)).astype(np.int64)
    link = I.link_matrix(P, 40)
    args = (P, P, 1, M, 200, costs, mem, cap, link, recs)
    g = run_advance(gpu, *args)
    r = R.advance_w(R.problem(P, P, 1, M, recs.shape[1], 200), costs, mem, cap, link, recs)
    check_advance(g, r, f"P={P} M={M}")
    assert g[0][0][2] > 0 and (g[3][0] == cap).all()


@pytest.mark.parametrize("P,v_max,M,L,mp,pct", [
    (1, 1, 4, 3, 8, 30), (2, 2, 4, 6, 16, 30), (3, 2, 6, 14, 24, 30), (4, 2, 8, 16, 40, 20),
    (4, 3, 4, 14, 24, 30), (5, 1, 7, 9, 20, 40), (8, 2, 16, 24, 60, 30), (16, 1, 8, 20, 40, 30),
    (8, 1, 32, 20, 80, 10), (4, 2, 64, 16, 120, 20), (4, 2, 32, 16, 80, 20),
    (3, 1, 16, 10, 40, 30), (6, 2, 24, 20, 60, 25), (32, 2, 8, 255, 60, 30),
    (64, 1, 24, 255, 80, 10),
])
def test_random_structures(gpu, P, v_max, M, L, mp, pct):
    """Every policy and placement kind, records with moves already (some deadlocked), invalid
    records, capacities at a low percentile of the unadvanced peaks."""
    rng = np.random.default_rng(900 + 100 * P + 10 * v_max + M)
    log(f"advance: random P={P} v_max={v_max} M={M} L={L} max_pert={mp}")
    costs = rng.integers(1, 6, size=(L, 3)).astype(np.int64) * 100_000
    link = rng.integers(0, 300_000, size=(P, P)).astype(np.int64)
    mem = np.stack([rng.integers(0, 1 << 26, L), rng.integers(0, 1 << 30, L)], axis=1)
    recs = I.random_candidates(rng, L, P, v_max, M, 240, max_pert=2, pert_rate=0.2,
                               invalid_rate=0.05, policies=(3, 3, 3, 0, 1, 2))
    recs = widen(recs, P, v_max, mp)
    prob = R.problem(L, P, v_max, M, recs.shape[1], mp)
    ms0, _, pk0 = R.sim_batch_mem(prob, costs, mem, link, recs, NTHREADS)
    cap = np.percentile(pk0[ms0 > 0], pct, axis=0).astype(np.int64)
    args = (L, P, v_max, M, mp, costs, mem, cap, link, recs)
    g = run_advance(gpu, *args)
    r = R.advance_w(prob, costs, mem, cap, link, recs, NTHREADS)
    check_advance(g, r, f"P={P} v_max={v_max} M={M}")
    if P > 1:
        assert (g[0][:, 2] > recs[:, 2]).sum() > 10


def test_in_place_and_huge_costs(gpu):
    """Output records may be the input buffer; times beyond 2^37 ns (64-bit tables)."""
    rng = np.random.default_rng(31)
    P, v_max, M, L, mp = 4, 2, 8, 12, 40
    log("advance: in place, huge costs")
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    costs[5] = [40_000_000_000, 30_000_000_000, 20_000_000_000]
    mem = np.stack([rng.integers(1, 1 << 20, L), rng.integers(0, 1 << 24, L)], axis=1)
    link = I.link_matrix(P, 5000)
    recs = widen(I.random_candidates(rng, L, P, v_max, M, 200, policies=(3,)), P, v_max, mp)
    prob = R.problem(L, P, v_max, M, recs.shape[1], mp)
    _, _, pk0 = R.sim_batch_mem(prob, costs, mem, link, recs, NTHREADS)
    cap = np.percentile(pk0, 25, axis=0).astype(np.int64)
    g = run_advance(gpu, L, P, v_max, M, mp, costs, mem, cap, link, recs, in_place=True)
    r = R.advance_w(prob, costs, mem, cap, link, recs, NTHREADS)
    check_advance(g, r, "in place")


@pytest.mark.parametrize("M", [8, 32])
def test_huge_costs_ring_and_full_rows(gpu, M):
    """Times beyond 2^37 ns, in place, on a shape whose search runs on 40-bit ring tables (M = 32:
    such candidates are searched again on 64-bit rows, from the input record the ring pass left
    as it was) and on one that uses 64-bit rows only (M = 8); the same records under ordinary
    costs stay on the rings."""
    rng = np.random.default_rng(47 + M)
    P, v_max, L, mp = 4, 2, 12, 60
    log(f"advance: huge costs M={M}")
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    huge = costs.copy()
    huge[3] = [40_000_000_000, 30_000_000_000, 20_000_000_000]
    mem = np.stack([rng.integers(1, 1 << 20, L), rng.integers(0, 1 << 24, L)], axis=1)
    link = I.link_matrix(P, 5000)
    recs = widen(I.random_candidates(rng, L, P, v_max, M, 200, policies=(3,)), P, v_max, mp)
    prob = R.problem(L, P, v_max, M, recs.shape[1], mp)
    _, _, pk0 = R.sim_batch_mem(prob, costs, mem, link, recs, NTHREADS)
    cap = np.percentile(pk0, 25, axis=0).astype(np.int64)
    for cs, label in ((costs, "ordinary"), (huge, "huge")):
        g = run_advance(gpu, L, P, v_max, M, mp, cs, mem, cap, link, recs, in_place=True)
        r = R.advance_w(prob, cs, mem, cap, link, recs, NTHREADS)
        check_advance(g, r, f"{label} M={M}")
        assert (g[0][:, 2] > recs[:, 2]).sum() > 20
        if label == "huge":
            assert (g[1] > (1 << 37)).sum() > 50


def test_workload3_candidates(gpu):
    """The 52-layer, P = 8, M = 64 batch with its memory recipe: 4,096 of its candidates
    (every stratum), 255 move slots, one capacity for all devices at the 40th percentile of the
    candidates' largest peaks; every one of them against the oracle."""
    w = I.WORKLOADS[3]
    log("advance: workload 3, 4096 candidates")
    costs, mem, link = I.layer_costs(w), I.layer_mem(w), I.link_matrix(w.P, w.link_ns)
    rng = np.random.default_rng(303)
    recs = I.candidates(w)
    recs = widen(recs[np.sort(rng.choice(len(recs), 4096, replace=False))], w.P, w.v_max, 255)
    prob = R.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], 255)
    ms0, _, pk0 = R.sim_batch_mem(prob, costs, mem, link, recs, NTHREADS)
    cap = np.full(w.P, int(np.percentile(pk0.max(axis=1)[ms0 > 0], 40)), np.int64)
    g = run_advance(gpu, w.L, w.P, w.v_max, w.M, 255, costs, mem, cap, link, recs)
    r = R.advance_w(prob, costs, mem, cap, link, recs, NTHREADS)
    check_advance(g, r, "workload 3")
    fit0 = (pk0 <= cap).all(axis=1) & (ms0 > 0)
    fit1 = (g[3] <= cap).all(axis=1) & (g[1] > 0)
    assert (g[0][:, 2] > 0).sum() > 400 and fit1.sum() > fit0.sum() and (fit1 >= fit0).all()


# ---------------------------------------------------------------------------------------------
# memory-constrained local search
# ---------------------------------------------------------------------------------------------

def run_tune_mem(dev, prob, costs, mem, cap, max_adv, link, recs, seed, steps, plain=False):
    import torch
    from paper_2509_23722_amd import _lib
    stride = _lib.chain_stride(prob)
    n = recs.shape[0]
    chains = np.zeros((n, stride), dtype=np.uint8)
    chains[:, :recs.shape[1]] = recs
    chains = t_(chains, dev)
    queues = torch.zeros((n, prob.P, _lib.queue_capacity(prob)), dtype=torch.int16, device=dev)
    c_t, m_t, k_t, l_t = t_(costs, dev), t_(mem, dev), t_(cap, dev), t_(link, dev)
    for t in range(steps + 1):
        if plain:
            _lib.tune_step(prob, c_t, l_t, chains, queues, seed, t)
        else:
            _lib.tune_step_mem(prob, c_t, m_t, k_t, max_adv, l_t, chains, queues, seed, t)
    torch.cuda.synchronize()
    ms, acc, bub, peak = _lib.chain_state(chains, prob, with_peak=True)
    return (chains.cpu().numpy()[:, :recs.shape[1]], ms.numpy(), bub.numpy(), peak.numpy(),
            acc.numpy(), queues.cpu().numpy().view(np.uint16))


def check_tune(g, r, label, rec_bytes, peaks=True):
    grec, gms, gbub, gpk, gacc, gq = g
    rrec, rms, rbub, rpk, racc, rq = r
    bad = (gms != rms) | (gbub != rbub).any(axis=1) | (gacc != racc)
    if peaks:
        bad |= (gpk != rpk).any(axis=1)
    bad = np.nonzero(bad)[0]
    if len(bad):
        i = int(bad[0])
        raise AssertionError(f"{label}: {len(bad)}/{len(gms)} chains differ; first {i}: gpu ms "
                             f"{gms[i]} acc {gacc[i]} peak {gpk[i].tolist()} oracle ms {rms[i]} "
                             f"acc {racc[i]} peak {rpk[i].tolist()}")
    assert (grec[:, :rec_bytes] == rrec[:, :rec_bytes]).all(), f"{label}: final records differ"
    if rq is not None:
        ok = rms != -2
        gq = gq[..., :rq.shape[-1]]
        assert (gq[ok].astype(np.int64) == rq[ok]).all(), f"{label}: final queues differ"


@pytest.mark.parametrize("P,v,M,L,pct,max_adv", [
    (4, 2, 8, 16, 40, 64), (3, 2, 6, 12, 30, 64), (8, 1, 8, 20, 40, 64), (4, 1, 5, 9, 50, 8),
    (2, 3, 4, 10, 40, 64), (4, 2, 8, 16, 50, 0),
])
def test_tune_mem_small(gpu, P, v, M, L, pct, max_adv):
    from paper_2509_23722_amd import _lib
    rng = np.random.default_rng(P * 100 + v * 10 + M + pct)
    n, steps, seed = 96, 30, 5 + P
    log(f"tune_mem P={P} v={v} M={M} L={L} cap pct={pct} max_adv={max_adv}")
    costs = rng.integers(100_000, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 500_000, size=(P, P)).astype(np.int64)
    mem = np.stack([rng.integers(1, 1 << 26, L), rng.integers(0, 1 << 28, L)], axis=1)
    recs = I.random_candidates(rng, L, P, v, M, n, policies=(0, 1, 2, 3, 3, 3))
    rprob = R.problem(L, P, v, M, recs.shape[1], 0)
    ms0, _, pk0 = R.sim_batch_mem(rprob, costs, mem, link, recs, NTHREADS)
    cap = np.full(P, int(np.percentile(pk0.max(axis=1)[ms0 > 0], pct)), np.int64)
    prob = _lib.problem(L, P, v, M, recs.shape[1], 0)
    g = run_tune_mem(gpu, prob, costs, mem, cap, max_adv, link, recs, seed, steps)
    r = R.tune_mem(rprob, costs, mem, cap, max_adv, link, recs, seed, steps, NTHREADS,
                   want_queues=True)
    check_tune(g, r, f"P={P} v={v} M={M}", 3 + 2 * P * v)
    assert (g[4] > 0).sum() > 30


def test_tune_mem_with_room_is_the_plain_search(gpu):
    from paper_2509_23722_amd import _lib
    rng = np.random.default_rng(77)
    P, v, M, L = 4, 2, 8, 16
    log("tune_mem: ample capacity vs plain search")
    costs = rng.integers(100_000, 3_000_000, size=(L, 3)).astype(np.int64)
    mem = np.stack([rng.integers(1, 1 << 26, L), rng.integers(0, 1 << 28, L)], axis=1)
    link = I.link_matrix(P, 200_000)
    recs = I.random_candidates(rng, L, P, v, M, 128, policies=(2, 3))
    prob = _lib.problem(L, P, v, M, recs.shape[1], 0)
    cap = np.full(P, 1 << 62, np.int64)
    a = run_tune_mem(gpu, prob, costs, mem, cap, 32, link, recs, 4, 25)
    b = run_tune_mem(gpu, prob, costs, mem, cap, 32, link, recs, 4, 25, plain=True)
    check_tune(a, b, "ample capacity", 3 + 2 * P * v, peaks=False)


def test_tune_mem_workload5_chains(gpu):
    """The 96-layer, P = 32, M = 256 chains with layer memory, one capacity for all devices at
    the median of the chains' largest initial peaks: 64 chains x 6 steps on the GPU, every one
    replayed by the oracle."""
    from paper_2509_23722_amd import _lib
    w = I.WORKLOADS[5]
    log("tune_mem: workload 5, 64 chains")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    mem = I.layer_mem(w)
    recs = I.tuner_chains(w, 64)
    rprob = R.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], 0)
    _, _, pk0 = R.sim_batch_mem(rprob, costs, mem, link, recs, NTHREADS)
    cap = np.full(w.P, int(np.percentile(pk0.max(axis=1), 50)), np.int64)
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], 0)
    g = run_tune_mem(gpu, prob, costs, mem, cap, 64, link, recs, w.seed, 6)
    r = R.tune_mem(rprob, costs, mem, cap, 64, link, recs, w.seed, 6, NTHREADS)
    check_tune(tuple(g[:5]) + (None,), r[:5] + (None,), "workload 5", 3 + 2 * w.s_max)
    assert (g[4] > 0).sum() > 20
