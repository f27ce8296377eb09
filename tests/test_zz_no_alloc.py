"""octo_sim_batch_noalloc (every buffer in the library's static device scratch) against
octo_sim_batch, bit for bit, through the C ABI: two calls in a row, the second smaller, and a
batch too large for the scratch rejected before any launch."""
import numpy as np
import pytest

from paper_2509_23722_amd import inputs as I

pytestmark = pytest.mark.gpu


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


def both(dev, L, P, v_max, M, max_pert, costs, link, recs):
    import torch
    from paper_2509_23722_amd import _lib
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    prob = _lib.problem(L, P, v_max, M, recs.shape[1], max_pert)
    c, lk, r = t(costs), t(link), t(recs)
    n = recs.shape[0]
    ms = torch.full((n,), 7, dtype=torch.int64, device=dev)
    bub = torch.full((n, P), 7, dtype=torch.int64, device=dev)
    _lib.sim_batch_noalloc(prob, c, lk, r, ms, bub)
    ref_ms, ref_bub = _lib.sim_batch(prob, c, lk, r)
    torch.cuda.synchronize()
    return ms.cpu().numpy(), bub.cpu().numpy(), ref_ms.cpu().numpy(), ref_bub.cpu().numpy()


def assert_same(gms, gbub, rms, rbub, label):
    bad = np.nonzero((gms != rms) | (gbub != rbub).any(axis=1))[0]
    assert len(bad) == 0, (f"{label}: {len(bad)}/{len(gms)} differ; first {int(bad[0])}: noalloc "
                           f"{gms[bad[0]]} octo_sim_batch {rms[bad[0]]}")


def test_two_calls_second_smaller(gpu):
    w = I.WORKLOADS[3]
    log(f"noalloc: {w.name}, {w.n} candidates")
    costs, link, recs = I.layer_costs(w), I.link_matrix(w.P, w.link_ns), I.candidates(w)
    out = both(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(*out, "P=8 M=64 batch")
    assert (out[0] > 0).all()
    # smaller, another shape, with moves (materialised queues), cyclic and invalid records
    rng = np.random.default_rng(77)
    L, P, v_max, M = 20, 4, 2, 16
    log(f"noalloc: random P={P} v_max={v_max} M={M}, 3000 candidates with moves")
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 800_000, size=(P, P)).astype(np.int64)
    recs = I.random_candidates(rng, L, P, v_max, M, 3000, max_pert=2, pert_rate=0.4,
                               invalid_rate=0.1)
    out = both(gpu, L, P, v_max, M, 2, costs, link, recs)
    assert_same(*out, "small batch with moves")
    assert (out[0] == -1).sum() > 10 and (out[0] == -2).sum() > 10
    # the headline batch again after the other shape (the cached tables are rebuilt)
    w = I.WORKLOADS[2]
    log(f"noalloc: {w.name}, {w.n} candidates")
    costs, link, recs = I.layer_costs(w), I.link_matrix(w.P, w.link_ns), I.candidates(w)
    out = both(gpu, w.L, w.P, w.v_max, w.M, w.max_pert, costs, link, recs)
    assert_same(*out, "P=8 M=32 batch")


def test_deeper_interleaving(gpu):
    """v up to 4 (one generated-queue launch per v, each with its own work counter in the
    scratch's control block), with moves and invalid records."""
    rng = np.random.default_rng(78)
    L, P, v_max, M = 24, 4, 4, 24
    log(f"noalloc: random P={P} v_max={v_max} M={M}, 2000 candidates")
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 800_000, size=(P, P)).astype(np.int64)
    recs = I.random_candidates(rng, L, P, v_max, M, 2000, max_pert=2, pert_rate=0.2,
                               invalid_rate=0.05)
    out = both(gpu, L, P, v_max, M, 2, costs, link, recs)
    assert_same(*out, "v_max = 4 batch")
    assert (recs[:, 1] >= 3).sum() > 500


def test_too_large_for_the_scratch(gpu):
    import ctypes
    import torch
    from paper_2509_23722_amd import _lib
    w = I.WORKLOADS[3]
    n = 3_000_000  # 13 bytes of lists per candidate: more than 32 MiB
    log(f"noalloc: {n} records, expecting OCTO_ESCRATCH")
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, I.record_stride(w.P, w.v_max, 0), 0)
    recs = torch.zeros((n, prob.cand_stride), dtype=torch.uint8, device=gpu)
    costs = torch.ones((w.L, 3), dtype=torch.int64, device=gpu)
    link = torch.zeros((w.P, w.P), dtype=torch.int64, device=gpu)
    ms = torch.zeros(n, dtype=torch.int64, device=gpu)
    bub = torch.zeros((n, w.P), dtype=torch.int64, device=gpu)
    with pytest.raises(RuntimeError, match="static scratch"):
        _lib.sim_batch_noalloc(prob, costs, link, recs, ms, bub)
    torch.cuda.synchronize()
    assert int(ms.abs().sum()) == 0  # nothing was launched
