"""ctypes wrapper around the CPU oracle ``liboctoref.so``.

Test infrastructure only: tests, the smoke check and the benchmark's CPU-baseline leg load it;
the product path never does. Build it with ``oracle/build.py`` (``__graft_entry__.build()`` does).
"""
import ctypes
import os

import numpy as np

HERE = os.path.dirname(os.path.abspath(__file__))
# OCTOREF_LIB may name another build of the same source (the sanitizer build)
LIB_PATH = os.environ.get("OCTOREF_LIB") or os.path.join(HERE, "liboctoref.so")


class RefProblem(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("P", ctypes.c_int32), ("v_max", ctypes.c_int32),
                ("M", ctypes.c_int32), ("cand_stride", ctypes.c_int32),
                ("max_pert", ctypes.c_int32)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            from . import build as _b  # noqa: F401  (oracle/build.py)
            _b.build()
        L = ctypes.CDLL(LIB_PATH)
        p = ctypes.c_void_p
        L.oracle_sim_batch.argtypes = [ctypes.POINTER(RefProblem), p, p, p, ctypes.c_int64, p, p,
                                       ctypes.c_int]
        L.oracle_sim_batch.restype = ctypes.c_int
        L.oracle_sim_batch_mem.argtypes = [ctypes.POINTER(RefProblem), p, p, p, p,
                                           ctypes.c_int64, p, p, p, ctypes.c_int]
        L.oracle_sim_batch_mem.restype = ctypes.c_int
        L.oracle_sim_batch_serial.argtypes = [ctypes.POINTER(RefProblem), p, p, p,
                                              ctypes.c_int64, p, p, ctypes.c_int]
        L.oracle_sim_batch_serial.restype = ctypes.c_int
        L.oracle_sim_batch_rdv.argtypes = [ctypes.POINTER(RefProblem), p, p, p,
                                           ctypes.c_int64, p, p, ctypes.c_int]
        L.oracle_sim_batch_rdv.restype = ctypes.c_int
        L.oracle_sim_batch_ordered.argtypes = [ctypes.POINTER(RefProblem), p, p, p,
                                               ctypes.c_int64, p, p, ctypes.c_int]
        L.oracle_sim_batch_ordered.restype = ctypes.c_int
        L.oracle_sim_batch_reorder.argtypes = [ctypes.POINTER(RefProblem), p, p, p,
                                               ctypes.c_int64, p, p, p, ctypes.c_int]
        L.oracle_sim_batch_reorder.restype = ctypes.c_int
        L.oracle_sim_batch_bounds.argtypes = [ctypes.POINTER(RefProblem), p, p, p,
                                              ctypes.c_int64, p, p, p, ctypes.c_int]
        L.oracle_sim_batch_bounds.restype = ctypes.c_int
        L.oracle_sim_batch_comm.argtypes = [ctypes.POINTER(RefProblem), p, p, p, ctypes.c_int64,
                                            p, p, p, ctypes.c_int]
        L.oracle_sim_batch_comm.restype = ctypes.c_int
        L.oracle_dump_queues.argtypes = [ctypes.POINTER(RefProblem), p, p, ctypes.c_int32, p]
        L.oracle_dump_queues.restype = ctypes.c_int
        L.oracle_sim_queues.argtypes = [ctypes.c_int32] * 4 + [p] * 9 + [p, p]
        L.oracle_sim_queues.restype = ctypes.c_int
        L.oracle_merge_tau.argtypes = [ctypes.c_int32] * 3 + [p]
        L.oracle_merge_tau.restype = ctypes.c_int
        L.oracle_philox4x64_10.argtypes = [p, p, p]
        L.oracle_philox4x64_10.restype = None
        L.oracle_tune.argtypes = [ctypes.POINTER(RefProblem), p, p, p, ctypes.c_int64,
                                  ctypes.c_uint64, ctypes.c_int32, p, p, p, p, p, ctypes.c_int]
        L.oracle_tune.restype = ctypes.c_int
        L.oracle_tune_mem.argtypes = [ctypes.POINTER(RefProblem), p, p, p, ctypes.c_int32, p, p,
                                      ctypes.c_int64, ctypes.c_uint64, ctypes.c_int32, p, p, p,
                                      p, p, p, ctypes.c_int]
        L.oracle_tune_mem.restype = ctypes.c_int
        L.oracle_advance_w.argtypes = [ctypes.POINTER(RefProblem), p, p, p, p, p,
                                       ctypes.c_int64, p, p, p, p, ctypes.c_int]
        L.oracle_advance_w.restype = ctypes.c_int
        _lib = L
    return _lib


def _ptr(a):
    return a.ctypes.data_as(ctypes.c_void_p) if a is not None else None


def problem(L, P, v_max, M, cand_stride, max_pert):
    return RefProblem(L, P, v_max, M, cand_stride, max_pert)


def sim_batch(prob, costs, link, cands, nthreads=1):
    """Evaluate candidate records (uint8 [n, stride]). Returns (makespan[n], bubble[n, P])."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    rc = lib().oracle_sim_batch(ctypes.byref(prob), _ptr(costs), _ptr(link), _ptr(cands), n,
                                _ptr(ms), _ptr(bub), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_sim_batch rejected the arguments (rc={rc})")
    return ms, bub


def sim_batch_mem(prob, costs, mem, link, cands, nthreads=1):
    """Evaluate candidate records with the memory model: mem int64 [L, 2] = {activation bytes
    per micro-batch, static bytes} per layer. Returns (makespan[n], bubble[n, P], peak[n, P])."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    mem = np.ascontiguousarray(mem, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    peak = np.zeros((n, prob.P), dtype=np.int64)
    rc = lib().oracle_sim_batch_mem(ctypes.byref(prob), _ptr(costs), _ptr(mem), _ptr(link),
                                    _ptr(cands), n, _ptr(ms), _ptr(bub), _ptr(peak), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_sim_batch_mem rejected the arguments (rc={rc})")
    return ms, bub, peak


def sim_batch_rdv(prob, costs, link, cands, nthreads=1):
    """Evaluate candidate records with blocking rendezvous transfers (receive right before the
    consumer, send right after the producer; a transfer holds both devices until it ends).
    Returns (makespan[n], bubble[n, P])."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    rc = lib().oracle_sim_batch_rdv(ctypes.byref(prob), _ptr(costs), _ptr(link), _ptr(cands), n,
                                    _ptr(ms), _ptr(bub), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_sim_batch_rdv rejected the arguments (rc={rc})")
    return ms, bub


def sim_batch_ordered(prob, costs, link, cands, nthreads=1):
    """Evaluate candidate records with blocking rendezvous transfers in the reordered
    coordination (every transfer at its ideal start in the asynchronous schedule, one global
    order per device). Returns (makespan[n], bubble[n, P])."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    rc = lib().oracle_sim_batch_ordered(ctypes.byref(prob), _ptr(costs), _ptr(link), _ptr(cands),
                                        n, _ptr(ms), _ptr(bub), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_sim_batch_ordered rejected the arguments (rc={rc})")
    return ms, bub


def sim_batch_reorder(prob, costs, link, cands, nthreads=1):
    """Evaluate candidate records under the executor's three-step reordering of the
    communication (mismatched pairs, feasible windows, greedy minimum of span - overlap) with
    handshake transfers. Returns (makespan[n], bubble[n, P], stats[n, 2] = {transfers,
    mismatched receives})."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    st = np.zeros((n, 2), dtype=np.int64)
    rc = lib().oracle_sim_batch_reorder(ctypes.byref(prob), _ptr(costs), _ptr(link), _ptr(cands),
                                        n, _ptr(ms), _ptr(bub), _ptr(st), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_sim_batch_reorder rejected the arguments (rc={rc})")
    return ms, bub, st


def sim_batch_serial(prob, costs, link, cands, nthreads=1):
    """Evaluate candidate records with serialised links (one transfer at a time per directed
    link, in issue order). Returns (makespan[n], bubble[n, P])."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    rc = lib().oracle_sim_batch_serial(ctypes.byref(prob), _ptr(costs), _ptr(link), _ptr(cands),
                                       n, _ptr(ms), _ptr(bub), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_sim_batch_serial rejected the arguments (rc={rc})")
    return ms, bub


def sim_batch_bounds(prob, costs, link, cands, nthreads=1):
    """Evaluate candidate records plus each device's first start and last finish. Returns
    (makespan[n], bubble[n, P], bounds[n, P, 2])."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    bounds = np.zeros((n, prob.P, 2), dtype=np.int64)
    rc = lib().oracle_sim_batch_bounds(ctypes.byref(prob), _ptr(costs), _ptr(link), _ptr(cands),
                                       n, _ptr(ms), _ptr(bub), _ptr(bounds), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_sim_batch_bounds rejected the arguments (rc={rc})")
    return ms, bub, bounds


def sim_batch_comm(prob, costs, link, cands, nthreads=1):
    """Evaluate candidate records with communication accounting. Returns (makespan[n],
    bubble[n, P], comm[n, 4]) with comm = {comm nodes, overlappable nodes, comm node time,
    overlap time}."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    comm = np.zeros((n, 4), dtype=np.int64)
    rc = lib().oracle_sim_batch_comm(ctypes.byref(prob), _ptr(costs), _ptr(link), _ptr(cands), n,
                                     _ptr(ms), _ptr(bub), _ptr(comm), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_sim_batch_comm rejected the arguments (rc={rc})")
    return ms, bub, comm


def advance_w(prob, costs, mem, cap, link, cands, nthreads=1):
    """Selective W advancing on candidate records: each record gains at most max_pert - n_pert
    perturbations that advance W ops until every device's peak is within cap (int64 [P]).

    Returns (records, makespan[n], bubble[n, P], peak[n, P]) of the output records."""
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    mem = np.ascontiguousarray(mem, dtype=np.int64)
    cap = np.ascontiguousarray(cap, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    cands = np.ascontiguousarray(cands, dtype=np.uint8)
    n = cands.shape[0]
    out = np.zeros_like(cands)
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    peak = np.zeros((n, prob.P), dtype=np.int64)
    rc = lib().oracle_advance_w(ctypes.byref(prob), _ptr(costs), _ptr(mem), _ptr(cap),
                                _ptr(link), _ptr(cands), n, _ptr(out), _ptr(ms), _ptr(bub),
                                _ptr(peak), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_advance_w rejected the arguments (rc={rc})")
    return out, ms, bub, peak


def dump_queues(prob, rec):
    """Final queues of one candidate as a list (per device) of (kind, stage, m) tuples,
    or None if the candidate is invalid."""
    qcap = 3 * prob.v_max * prob.M
    ops = np.zeros((prob.P, qcap), dtype=np.int32)
    qlen = np.zeros(prob.P, dtype=np.int32)
    rec = np.ascontiguousarray(rec, dtype=np.uint8)
    rc = lib().oracle_dump_queues(ctypes.byref(prob), _ptr(rec), _ptr(ops), qcap, _ptr(qlen))
    if rc == -2:
        return None
    if rc != 0:
        raise ValueError(f"oracle_dump_queues failed (rc={rc})")
    out = []
    for d in range(prob.P):
        row = ops[d, :qlen[d]]
        out.append([(int(x) >> 24, (int(x) >> 16) & 0xFF, int(x) & 0xFFFF) for x in row])
    return out


def sim_queues(P, S, M, split, dev, F, B, W, link, queues, want_start=False):
    """Evaluate explicit queues (list per device of (kind, stage, m)).

    Returns (status, makespan, bubble[P], start or None, n_cross) where status is 0 (ok),
    1 (deadlock) or 2 (queues are not exactly the op set)."""
    ops = np.array([(k << 24) | (s << 16) | m for q in queues for (k, s, m) in q] or [0],
                   dtype=np.int32)
    qlen = np.array([len(q) for q in queues], dtype=np.int32)
    dev = np.ascontiguousarray(dev, dtype=np.int32)
    F = np.ascontiguousarray(F, dtype=np.int64)
    B = np.ascontiguousarray(B, dtype=np.int64)
    W = np.ascontiguousarray(W, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    ms = np.zeros(1, dtype=np.int64)
    bub = np.zeros(P, dtype=np.int64)
    nk = 3 if split else 2
    start = np.zeros(nk * S * M, dtype=np.int64) if want_start else None
    ncross = np.zeros(1, dtype=np.int64)
    rc = lib().oracle_sim_queues(P, S, M, int(bool(split)), _ptr(dev), _ptr(F), _ptr(B), _ptr(W),
                                 _ptr(link), _ptr(ops), _ptr(qlen), _ptr(ms), _ptr(bub),
                                 _ptr(start), _ptr(ncross))
    if rc < 0:
        raise ValueError(f"oracle_sim_queues rejected the arguments (rc={rc})")
    return rc, int(ms[0]), bub, start, int(ncross[0])


def merge_tau(S, M, split):
    nk = 3 if split else 2
    tau = np.zeros(nk * S * M, dtype=np.int64)
    rc = lib().oracle_merge_tau(S, M, int(bool(split)), _ptr(tau))
    if rc != 0:
        raise ValueError(f"oracle_merge_tau failed (rc={rc})")
    return tau.reshape(nk, S, M)


def philox4x64_10(counter, key):
    ctr = np.array(counter, dtype=np.uint64)
    k = np.array(key, dtype=np.uint64)
    out = np.zeros(4, dtype=np.uint64)
    lib().oracle_philox4x64_10(_ptr(ctr), _ptr(k), _ptr(out))
    return [int(x) for x in out]


def tune(prob, costs, link, recs, seed, n_steps, nthreads=1, want_queues=False, chain_ids=None):
    """Run the local search (steps 0..n_steps) on every chain record (chain index = position,
    or chain_ids[i]).

    Returns (final_records, makespan[n], bubble[n, P], accepted[n], queues or None)."""
    recs = np.array(recs, dtype=np.uint8, copy=True, order="C")
    ids = None if chain_ids is None else np.ascontiguousarray(chain_ids, dtype=np.int64)
    n = recs.shape[0]
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    acc = np.zeros(n, dtype=np.int64)
    qcap = 3 * prob.v_max * prob.M
    queues = np.zeros((n, prob.P, qcap), dtype=np.int32) if want_queues else None
    rc = lib().oracle_tune(ctypes.byref(prob), _ptr(costs), _ptr(link), _ptr(recs), n,
                           ctypes.c_uint64(seed), int(n_steps), _ptr(ms), _ptr(bub), _ptr(acc),
                           _ptr(queues), _ptr(ids), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_tune rejected the arguments (rc={rc})")
    return recs, ms, bub, acc, queues


def tune_mem(prob, costs, mem, cap, max_adv, link, recs, seed, n_steps, nthreads=1,
             want_queues=False, chain_ids=None):
    """The local search under the memory constraint (cap int64 [P]) with selective W advancing
    (at most max_adv advances per evaluation).

    Returns (final_records, makespan[n], bubble[n, P], peak[n, P], accepted[n], queues or
    None)."""
    recs = np.array(recs, dtype=np.uint8, copy=True, order="C")
    ids = None if chain_ids is None else np.ascontiguousarray(chain_ids, dtype=np.int64)
    n = recs.shape[0]
    costs = np.ascontiguousarray(costs, dtype=np.int64)
    mem = np.ascontiguousarray(mem, dtype=np.int64)
    cap = np.ascontiguousarray(cap, dtype=np.int64)
    link = np.ascontiguousarray(link, dtype=np.int64)
    ms = np.zeros(n, dtype=np.int64)
    bub = np.zeros((n, prob.P), dtype=np.int64)
    peak = np.zeros((n, prob.P), dtype=np.int64)
    acc = np.zeros(n, dtype=np.int64)
    qcap = 3 * prob.v_max * prob.M
    queues = np.zeros((n, prob.P, qcap), dtype=np.int32) if want_queues else None
    rc = lib().oracle_tune_mem(ctypes.byref(prob), _ptr(costs), _ptr(mem), _ptr(cap),
                               int(max_adv), _ptr(link), _ptr(recs), n, ctypes.c_uint64(seed),
                               int(n_steps), _ptr(ms), _ptr(bub), _ptr(peak), _ptr(acc),
                               _ptr(queues), _ptr(ids), int(nthreads))
    if rc != 0:
        raise ValueError(f"oracle_tune_mem rejected the arguments (rc={rc})")
    return recs, ms, bub, peak, acc, queues


def tune_chains(prob, costs, link, all_recs, chain_ids, seed, n_steps, nthreads=1):
    """Replay only the chains chain_ids of a larger set; returns (records, ms, bub, acc)."""
    recs, ms, bub, acc, _ = tune(prob, costs, link, np.asarray(all_recs)[chain_ids], seed,
                                 n_steps, nthreads=nthreads, chain_ids=chain_ids)
    return recs, ms, bub, acc
