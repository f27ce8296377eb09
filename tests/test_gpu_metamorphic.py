"""Metamorphic properties of the GPU simulator on the full 1,048,576-candidate P = 8, M = 64
batch — properties of the time model (§5, §6 Eq. 1) that hold at any size, checked on every
candidate rather than on a sample:

* scaling every layer cost and every link by k scales every makespan and bubble by k (the
  relaxation is max-plus: max and + commute with a positive factor);
* relabelling the devices under uniform links permutes the bubbles and keeps the makespan (a
  device's queue depends only on the stages it hosts, and every transfer costs the same);
* raising one layer's cost never shortens a schedule (every start is a max of sums of costs);
* the same scaling holds with blocking rendezvous transfers and the reordered coordination.
"""
import numpy as np
import pytest

from paper_2509_23722_amd import inputs as I

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module")
def batch():
    import torch
    from paper_2509_23722_amd import _lib
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    _lib.lib()
    dev = torch.device("cuda:0")
    w = I.WORKLOADS[3]
    recs = I.candidates(w)
    return dev, w, recs


def run(dev, w, recs, costs, link, fn="sim_batch"):
    import torch
    from paper_2509_23722_amd import _lib
    prob = _lib.problem(w.L, w.P, w.v_max, w.M, recs.shape[1], w.max_pert)
    t = lambda x: torch.from_numpy(np.ascontiguousarray(x)).to(dev)
    ms, bub = getattr(_lib, fn)(prob, t(costs), t(link), t(recs))[:2]
    torch.cuda.synchronize()
    return ms.cpu().numpy(), bub.cpu().numpy()


def log(msg):
    print(msg, flush=True)


def test_scaling(batch):
    dev, w, recs = batch
    log("metamorphic: scaling")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    ms, bub = run(dev, w, recs, costs, link)
    ms3, bub3 = run(dev, w, recs, 3 * costs, 3 * link)
    ok = ms > 0
    assert ok.sum() == len(recs)
    assert (ms3 == 3 * ms).all() and (bub3 == 3 * bub).all()


def test_device_relabel(batch):
    dev, w, recs = batch
    log("metamorphic: device relabel")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    perm = np.array([3, 7, 0, 5, 1, 6, 2, 4])
    re = recs.copy()
    s_max = w.P * w.v_max
    S = w.P * re[:, 1].astype(np.int64)
    dv = re[:, 3 + s_max:3 + 2 * s_max]
    cols = np.arange(s_max)[None, :] < S[:, None]
    dv[cols] = perm[dv[cols]]
    ms, bub = run(dev, w, recs, costs, link)
    ms2, bub2 = run(dev, w, re, costs, link)
    assert (ms2 == ms).all()
    assert (bub2[:, perm] == bub).all()


def test_monotone_in_a_layer_cost(batch):
    dev, w, recs = batch
    log("metamorphic: monotone")
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    ms, _ = run(dev, w, recs, costs, link)
    up = costs.copy()
    up[17] += [700_000, 300_000, 900_000]
    ms2, _ = run(dev, w, recs, up, link)
    assert (ms2 >= ms).all() and (ms2 > ms).sum() > len(recs) // 2


@pytest.mark.parametrize("fn", ["sim_batch_rdv", "sim_batch_ordered"])
def test_scaling_blocking_transfers(batch, fn):
    dev, w, recs = batch
    log(f"metamorphic: scaling, {fn}")
    sub = recs[::16]
    costs, link = I.layer_costs(w), I.link_matrix(w.P, w.link_ns)
    ms, bub = run(dev, w, sub, costs, link, fn)
    ms3, bub3 = run(dev, w, sub, 2 * costs, 2 * link, fn)
    live = ms > 0
    assert live.sum() > 1000
    assert (ms3[live] == 2 * ms[live]).all() and (bub3[live] == 2 * bub[live]).all()
    assert (ms3[~live] == ms[~live]).all()
