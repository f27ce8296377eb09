"""Workspace growth on a fresh stream: calls queued back to back, with batches that grow (and
an entry point with buffers of its own between them), give the oracle's results with no host
wait between the calls; the workspace of a stream grows in stream order."""
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


def test_growing_batches_on_a_fresh_stream(gpu):
    import torch
    from paper_2509_23722_amd import _lib
    w = I.WORKLOADS[3]
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    recs = I.candidates(w)[:131072]
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], w.max_pert)
    c = torch.from_numpy(costs).to(gpu)
    lk = torch.from_numpy(link).to(gpu)
    r = torch.from_numpy(recs).to(gpu)
    torch.cuda.synchronize()
    plan = [("sim", 64), ("sim", 8192), ("ordered", 1024), ("sim", 131072), ("ordered", 4096),
            ("sim", 1000)]
    s = torch.cuda.Stream()
    outs = []
    print("workspace: queueing", plan, flush=True)
    with torch.cuda.stream(s):
        for kind, n in plan:
            fn = _lib.sim_batch if kind == "sim" else _lib.sim_batch_ordered
            outs.append(fn(prob, c, lk, r[:n])[:2])
    s.synchronize()
    rp = R.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], w.max_pert)
    ref = {"sim": R.sim_batch(rp, costs, link, recs, nthreads=NTHREADS),
           "ordered": R.sim_batch_ordered(rp, costs, link, recs[:4096], nthreads=NTHREADS)}
    for (kind, n), (ms, bub) in zip(plan, outs):
        ms, bub = ms.cpu().numpy(), bub.cpu().numpy()
        rms, rbub = ref[kind][0][:n], ref[kind][1][:n]
        bad = np.nonzero((ms != rms) | (bub != rbub).any(axis=1))[0]
        assert len(bad) == 0, f"{kind} n={n}: {len(bad)} differ, first {int(bad[0])}"


def test_binding_rejects_wrong_extents(gpu):
    """The library takes plain pointers: the binding refuses a buffer whose element count is
    not the one the call reads or writes, before anything is launched."""
    import torch
    from paper_2509_23722_amd import _lib
    w = I.WORKLOADS[3]
    recs = I.candidates(w)[:256]
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], w.max_pert)
    c = torch.from_numpy(I.layer_costs(w)).to(gpu)
    lk = torch.from_numpy(I.link_matrix(w.P, w.link_ns)).to(gpu)
    r = torch.from_numpy(recs).to(gpu)
    n = r.shape[0]
    ms = torch.empty(n, dtype=torch.int64, device=gpu)
    with pytest.raises(ValueError, match="out_bubble"):
        _lib.sim_batch(prob, c, lk, r, ms, torch.empty(n, dtype=torch.int64, device=gpu))
    with pytest.raises(ValueError, match="out_comm"):
        _lib.sim_batch_comm(prob, c, lk, r, ms, None, torch.empty((n, 2), dtype=torch.int64,
                                                                   device=gpu))
    with pytest.raises(ValueError, match="candidates"):
        _lib.sim_batch(prob, c, lk, r[:, :-16].contiguous())
    with pytest.raises(ValueError, match="link"):
        _lib.sim_batch(prob, c, lk[:-1].contiguous(), r)
    ms_ok, _ = _lib.sim_batch(prob, c, lk, r)
    torch.cuda.synchronize()
    assert ms_ok.shape == (n,)
