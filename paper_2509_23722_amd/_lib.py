"""ctypes binding of libocto.so (argument marshalling only; every step runs in HIP kernels).

Arrays are torch tensors on the GPU; the call is enqueued on torch's current stream of the
tensors' device. Raises if the library is missing or a call returns an error status.
"""
import ctypes
import os

import torch

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libocto.so")

OCTO_MS_DEADLOCK = -1
OCTO_MS_INVALID = -2
AFAB, ONEF1B, I1F1B, ZB = 0, 1, 2, 3


class OctoProblem(ctypes.Structure):
    _fields_ = [("L", ctypes.c_int32), ("P", ctypes.c_int32), ("v_max", ctypes.c_int32),
                ("M", ctypes.c_int32), ("cand_stride", ctypes.c_int32),
                ("max_pert", ctypes.c_int32)]


_lib = None


def lib():
    """Load libocto.so (fails loudly when it has not been built)."""
    global _lib
    if _lib is None:
        if not os.path.exists(LIB_PATH):
            raise RuntimeError(f"{LIB_PATH} is missing: build it with "
                               "`python -c 'import __graft_entry__ as g; g.build()'`")
        L = ctypes.CDLL(LIB_PATH)
        vp, i32, i64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64
        pp = ctypes.POINTER(OctoProblem)
        L.octo_record_pert_offset.argtypes = [i32, i32]
        L.octo_record_pert_offset.restype = i32
        L.octo_record_stride.argtypes = [i32, i32, i32]
        L.octo_record_stride.restype = i32
        L.octo_chain_stride.argtypes = [pp]
        L.octo_chain_stride.restype = i32
        L.octo_queue_capacity.argtypes = [pp]
        L.octo_queue_capacity.restype = i32
        L.octo_sim_batch.argtypes = [pp, vp, vp, vp, i64, vp, vp, vp]
        L.octo_sim_batch.restype = ctypes.c_int
        L.octo_sim_batch_noalloc.argtypes = [pp, vp, vp, vp, i64, vp, vp, vp]
        L.octo_sim_batch_noalloc.restype = ctypes.c_int
        L.octo_sim_batch_mem.argtypes = [pp, vp, vp, vp, vp, i64, vp, vp, vp, vp]
        L.octo_sim_batch_comm.argtypes = [pp, vp, vp, vp, i64, vp, vp, vp, vp]
        L.octo_sim_batch_serial.argtypes = [pp, vp, vp, vp, i64, vp, vp, vp]
        L.octo_sim_batch_rdv.argtypes = [pp, vp, vp, vp, i64, vp, vp, vp]
        L.octo_sim_batch_ordered.argtypes = [pp, vp, vp, vp, i64, vp, vp, vp]
        L.octo_sim_batch_reorder.argtypes = [pp, vp, vp, vp, i64, vp, vp, vp, vp]
        L.octo_sim_batch_bounds.argtypes = [pp, vp, vp, vp, i64, vp, vp, vp, vp]
        L.octo_sim_batch_mem.restype = ctypes.c_int
        L.octo_tune_step.argtypes = [pp, vp, vp, vp, vp, i64, ctypes.c_uint64, i32, vp]
        L.octo_tune_step_mem.argtypes = [pp, vp, vp, vp, i32, vp, vp, vp, i64, ctypes.c_uint64,
                                         i32, vp]
        L.octo_advance_w.argtypes = [pp, vp, vp, vp, vp, vp, i64, vp, vp, vp, vp, vp]
        L.octo_tune_step.restype = ctypes.c_int
        L.octo_alg1_tune.argtypes = [pp, vp, vp, vp, i64, i32, vp, vp, vp, vp]
        L.octo_alg1_tune_ex.argtypes = [pp, vp, vp, vp, i64, i32, i32, ctypes.c_uint64, vp, vp,
                                        vp, vp, vp]
        L.octo_alg1_tune.restype = ctypes.c_int
        L.octo_profile_events.argtypes = [ctypes.POINTER(ctypes.c_void_p), i32]
        L.octo_profile_events.restype = ctypes.c_int
        L.octo_strerror.argtypes = [ctypes.c_int]
        L.octo_strerror.restype = ctypes.c_char_p
        _lib = L
    return _lib


def problem(L, P, v_max, M, cand_stride, max_pert=0):
    return OctoProblem(L, P, v_max, M, cand_stride, max_pert)


def _check(rc, what):
    if rc != 0:
        raise RuntimeError(f"{what} failed: {lib().octo_strerror(rc).decode()} (status {rc})")


def _dev_ptr(t, dtype, name, numel):
    """The device address of a contiguous tensor of `dtype` holding exactly `numel` elements
    (the library takes plain pointers and cannot check the extents itself)."""
    if not isinstance(t, torch.Tensor) or not t.is_cuda:
        raise TypeError(f"{name} must be a CUDA (HIP) tensor")
    if t.dtype != dtype or not t.is_contiguous():
        raise TypeError(f"{name} must be a contiguous {dtype} tensor")
    if t.numel() != numel:
        raise ValueError(f"{name} must hold {numel} elements, not {t.numel()} "
                         f"(shape {tuple(t.shape)})")
    return ctypes.c_void_p(t.data_ptr())


def _stream(t, stream):
    s = stream if stream is not None else torch.cuda.current_stream(t.device)
    return ctypes.c_void_p(s.cuda_stream)


def record_stride(P, v_max, max_pert):
    return lib().octo_record_stride(P, v_max, max_pert)


def chain_stride(prob):
    return lib().octo_chain_stride(ctypes.byref(prob))


def queue_capacity(prob):
    return lib().octo_queue_capacity(ctypes.byref(prob))


def sim_batch(prob, layer_costs, link, candidates, out_makespan=None, out_bubble=None,
              stream=None):
    """octo_sim_batch: candidates uint8 [n, stride] -> (makespan int64 [n], bubble int64 [n, P])."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    rc = lib().octo_sim_batch(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P), _stream(candidates, stream))
    _check(rc, "octo_sim_batch")
    return out_makespan, out_bubble


def sim_batch_noalloc(prob, layer_costs, link, candidates, out_makespan, out_bubble,
                      stream=None):
    """octo_sim_batch_noalloc: as sim_batch, with caller-allocated outputs and every other
    buffer in the library's static device scratch (nothing is allocated by the call)."""
    n = candidates.shape[0]
    rc = lib().octo_sim_batch_noalloc(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P), _stream(candidates, stream))
    _check(rc, "octo_sim_batch_noalloc")
    return out_makespan, out_bubble


def sim_batch_mem(prob, layer_costs, layer_mem, link, candidates, out_makespan=None,
                  out_bubble=None, out_peak=None, stream=None):
    """octo_sim_batch_mem: as sim_batch, plus layer_mem int64 [L, 2] -> peak int64 [n, P].
    Returns (makespan, bubble, peak)."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    if out_peak is None:
        out_peak = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    rc = lib().octo_sim_batch_mem(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(layer_mem, torch.int64, "layer_mem", 2 * prob.L), _dev_ptr(link, torch.int64, "link", prob.P * prob.P),
        _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P),
        _dev_ptr(out_peak, torch.int64, "out_peak", n * prob.P), _stream(candidates, stream))
    _check(rc, "octo_sim_batch_mem")
    return out_makespan, out_bubble, out_peak


def sim_batch_serial(prob, layer_costs, link, candidates, out_makespan=None, out_bubble=None,
                     stream=None):
    """octo_sim_batch_serial: as sim_batch, with serialised links (one transfer at a time per
    directed link, in issue order)."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    rc = lib().octo_sim_batch_serial(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P), _stream(candidates, stream))
    _check(rc, "octo_sim_batch_serial")
    return out_makespan, out_bubble


def sim_batch_rdv(prob, layer_costs, link, candidates, out_makespan=None, out_bubble=None,
                  stream=None):
    """octo_sim_batch_rdv: as sim_batch, with blocking rendezvous transfers (receive right before
    the consumer, send right after the producer, both devices held until the transfer ends)."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    rc = lib().octo_sim_batch_rdv(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P), _stream(candidates, stream))
    _check(rc, "octo_sim_batch_rdv")
    return out_makespan, out_bubble


def sim_batch_ordered(prob, layer_costs, link, candidates, out_makespan=None, out_bubble=None,
                      stream=None):
    """octo_sim_batch_ordered: blocking rendezvous transfers in the reordered coordination
    (every transfer at its ideal start in the asynchronous schedule)."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    rc = lib().octo_sim_batch_ordered(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P), _stream(candidates, stream))
    _check(rc, "octo_sim_batch_ordered")
    return out_makespan, out_bubble


def sim_batch_reorder(prob, layer_costs, link, candidates, out_makespan=None, out_bubble=None,
                      out_stats=None, stream=None):
    """octo_sim_batch_reorder: the executor's three-step reordering of the communication with
    handshake transfers. Returns (makespan, bubble, stats int64 [n, 2] = {transfers,
    mismatched receives})."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    if out_stats is None:
        out_stats = torch.empty((n, 2), dtype=torch.int64, device=dev)
    rc = lib().octo_sim_batch_reorder(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P),
        _dev_ptr(out_stats, torch.int64, "out_stats", 2 * n), _stream(candidates, stream))
    _check(rc, "octo_sim_batch_reorder")
    return out_makespan, out_bubble, out_stats


def sim_batch_bounds(prob, layer_costs, link, candidates, out_makespan=None, out_bubble=None,
                     out_bounds=None, stream=None):
    """octo_sim_batch_bounds: as sim_batch, plus bounds int64 [n, P, 2] = {first start, last
    finish} per device. Returns (makespan, bubble, bounds)."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    if out_bounds is None:
        out_bounds = torch.empty((n, prob.P, 2), dtype=torch.int64, device=dev)
    rc = lib().octo_sim_batch_bounds(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P),
        _dev_ptr(out_bounds, torch.int64, "out_bounds", 2 * n * prob.P), _stream(candidates, stream))
    _check(rc, "octo_sim_batch_bounds")
    return out_makespan, out_bubble, out_bounds


def sim_batch_comm(prob, layer_costs, link, candidates, out_makespan=None, out_bubble=None,
                   out_comm=None, stream=None):
    """octo_sim_batch_comm: as sim_batch, plus comm int64 [n, 4] = {comm nodes, overlappable
    nodes, comm node time, overlap time}. Returns (makespan, bubble, comm)."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    if out_comm is None:
        out_comm = torch.empty((n, 4), dtype=torch.int64, device=dev)
    rc = lib().octo_sim_batch_comm(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P),
        _dev_ptr(out_comm, torch.int64, "out_comm", 4 * n), _stream(candidates, stream))
    _check(rc, "octo_sim_batch_comm")
    return out_makespan, out_bubble, out_comm


def tune_step(prob, layer_costs, link, chains, queues, seed, step, stream=None):
    """octo_tune_step on chain states (uint8 [n, chain_stride]) and queues (int16/uint16)."""
    n = chains.shape[0]
    q = queues
    if q.dtype not in (torch.int16, torch.uint16):
        raise TypeError("queues must be a 16-bit tensor")
    rc = lib().octo_tune_step(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(chains, torch.uint8, "chains", n * chain_stride(prob)),
        _dev_ptr(q, q.dtype, "queues", n * prob.P * queue_capacity(prob)), n, ctypes.c_uint64(seed & (2**64 - 1)), int(step),
        _stream(chains, stream))
    _check(rc, "octo_tune_step")


def tune_step_mem(prob, layer_costs, layer_mem, capacity, max_advance, link, chains, queues,
                  seed, step, stream=None):
    """octo_tune_step_mem: the local-search step under per-device capacities (int64 [P]) with
    selective W advancing (at most max_advance advances per evaluation)."""
    n = chains.shape[0]
    q = queues
    if q.dtype not in (torch.int16, torch.uint16):
        raise TypeError("queues must be a 16-bit tensor")
    rc = lib().octo_tune_step_mem(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(layer_mem, torch.int64, "layer_mem", 2 * prob.L),
        _dev_ptr(capacity, torch.int64, "capacity", prob.P), int(max_advance),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(chains, torch.uint8, "chains", n * chain_stride(prob)),
        _dev_ptr(q, q.dtype, "queues", n * prob.P * queue_capacity(prob)), n, ctypes.c_uint64(seed & (2**64 - 1)), int(step),
        _stream(chains, stream))
    _check(rc, "octo_tune_step_mem")


def advance_w(prob, layer_costs, layer_mem, capacity, link, candidates, out_candidates=None,
              out_makespan=None, out_bubble=None, out_peak=None, stream=None):
    """octo_advance_w: selective W advancing on candidate records under capacity (int64 [P]).
    Returns (records, makespan, bubble, peak) of the output records."""
    n = candidates.shape[0]
    dev = candidates.device
    if out_candidates is None:
        out_candidates = torch.empty_like(candidates)
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    if out_peak is None:
        out_peak = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    rc = lib().octo_advance_w(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(layer_mem, torch.int64, "layer_mem", 2 * prob.L),
        _dev_ptr(capacity, torch.int64, "capacity", prob.P), _dev_ptr(link, torch.int64, "link", prob.P * prob.P),
        _dev_ptr(candidates, torch.uint8, "candidates", n * prob.cand_stride), n,
        _dev_ptr(out_candidates, torch.uint8, "out_candidates", n * prob.cand_stride),
        _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P),
        _dev_ptr(out_peak, torch.int64, "out_peak", n * prob.P), _stream(candidates, stream))
    _check(rc, "octo_advance_w")
    return out_candidates, out_makespan, out_bubble, out_peak


def alg1_tune(prob, layer_costs, link, records, iters, out_makespan=None, out_bubble=None,
              out_stats=None, stream=None):
    """octo_alg1_tune: Algorithm 1 on every record (uint8 [n, stride], updated in place) for
    `iters` iterations. Returns (makespan [n], bubble [n, P], stats [n, 4] = kept moves per
    phase (partitioning, placement, scheduling) and iterations that searched)."""
    n = records.shape[0]
    dev = records.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    if out_stats is None:
        out_stats = torch.empty((n, 4), dtype=torch.int64, device=dev)
    rc = lib().octo_alg1_tune(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(records, torch.uint8, "records", n * prob.cand_stride), n,
        int(iters), _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P),
        _dev_ptr(out_stats, torch.int64, "out_stats", 4 * n), _stream(records, stream))
    _check(rc, "octo_alg1_tune")
    return out_makespan, out_bubble, out_stats


A1_INSERT, A1_RANDOM = 1, 2


def alg1_tune_ex(prob, layer_costs, link, records, iters, flags, seed=0, out_makespan=None,
                 out_bubble=None, out_stats=None, out_phase_iters=None, stream=None):
    """octo_alg1_tune_ex: alg1_tune with flags (A1_INSERT: overlap-aware insertions in the
    scheduling phase; A1_RANDOM: phases drawn at random with `seed`). Returns (makespan,
    bubble, stats [n, 4], phase iterations [n, 3])."""
    n = records.shape[0]
    dev = records.device
    if out_makespan is None:
        out_makespan = torch.empty(n, dtype=torch.int64, device=dev)
    if out_bubble is None:
        out_bubble = torch.empty((n, prob.P), dtype=torch.int64, device=dev)
    if out_stats is None:
        out_stats = torch.empty((n, 4), dtype=torch.int64, device=dev)
    if out_phase_iters is None:
        out_phase_iters = torch.empty((n, 3), dtype=torch.int64, device=dev)
    rc = lib().octo_alg1_tune_ex(
        ctypes.byref(prob), _dev_ptr(layer_costs, torch.int64, "layer_costs", 3 * prob.L),
        _dev_ptr(link, torch.int64, "link", prob.P * prob.P), _dev_ptr(records, torch.uint8, "records", n * prob.cand_stride), n,
        int(iters), int(flags), int(seed), _dev_ptr(out_makespan, torch.int64, "out_makespan", n),
        _dev_ptr(out_bubble, torch.int64, "out_bubble", n * prob.P),
        _dev_ptr(out_stats, torch.int64, "out_stats", 4 * n),
        _dev_ptr(out_phase_iters, torch.int64, "out_phase_iters", 3 * n), _stream(records, stream))
    _check(rc, "octo_alg1_tune_ex")
    return out_makespan, out_bubble, out_stats, out_phase_iters


def profile_events(events):
    """Record hipEvent_t handles (ints) at the simulation-kernel boundaries of later calls
    (see include/octo.h); an empty list turns it off."""
    arr = (ctypes.c_void_p * max(len(events), 1))(*events)
    _check(lib().octo_profile_events(arr, len(events)), "octo_profile_events")


def chain_state(chains, prob, with_peak=False):
    """Decode (makespan [n], accepted [n], bubble [n, P]) from chain-state bytes (host copy);
    with_peak: also the peak bytes [n, P] stored by tune_step_mem."""
    c = chains.cpu() if isinstance(chains, torch.Tensor) else torch.as_tensor(chains)
    off = prob.cand_stride
    tail = c[:, off:off + 16 + 16 * prob.P].contiguous().view(torch.int64)
    out = (tail[:, 0], tail[:, 1], tail[:, 2:2 + prob.P])
    return out + (tail[:, 2 + prob.P:2 + 2 * prob.P],) if with_peak else out
