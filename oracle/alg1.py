"""Algorithm 1 of §6 ("Iterative and Bubble-Aware Tuning"), the CPU oracle.

TEST INFRASTRUCTURE ONLY: tests, the smoke check and the benchmark's CPU-baseline leg may use
it; the product path never does. Plain Python over candidate records; every evaluation is the
oracle's simulator (``octoref``). It shares nothing with the HIP path but the record format.

One search per record, all independent. Each iteration (Algorithm 1's loop body):

1. Evaluate the current record: makespan, bubble per device, first start and last finish per
   device. Derived: the gap ``Δb = max_d bubble_d − min_d bubble_d``; the boundary bubble
   ``b_bd = Σ_d (first start_d + makespan − last finish_d)``; the residual bubble
   ``b_res = Σ_d bubble_d − b_bd``; ``t_layer = M · min_l (F_l + B_l + W_l)``, the smallest
   computation one layer adds to a device in an iteration.
2. Pick the phase: partitioning if ``Δb > t_layer``, else placement if ``b_bd > b_res``, else
   scheduling (the priority order of §6). A phase whose last search found nothing better is
   exhausted until some phase improves; an exhausted pick falls to the first non-exhausted
   phase in the order partitioning, placement, scheduling; with all three exhausted the search
   has converged. The random-search variant of §8 ("Pipeline Search Cost": the same iterative
   framework, phases picked at random without regard to the bubbles) takes instead the
   ``u mod n``-th of the n open phases (in that order), u the first word of
   Philox4x64-10(counter = (record, iteration, 1, 0), key = (seed, 0)).
3. ``argmin`` over the phase's neighbourhood (below): the first record, in neighbourhood order,
   of the smallest makespan among those that neither deadlock nor are invalid. It replaces the
   current record iff its makespan is strictly smaller; otherwise the phase is exhausted.

Neighbourhoods (§6 Partitioning / Placement / Scheduling Tuning):

* partitioning — migrate one layer from a stage of the most loaded device (largest busy time,
  lowest index on ties) to a stage of the least loaded one: for each pair (a, b), a of the
  first device's stages and b of the second's, ascending: the stages between them pass one
  layer along (a < b: boundaries b[a+1..b] − 1; a > b: boundaries b[b+1..a] + 1); only where
  stage a keeps a layer.
* placement — layer exchange: the device with the largest bubble (d1) swaps one of its stages
  with one of another device's (d2 ascending, then d1's stages, then d2's stages ascending);
  then stage dispersion when ``2v ≤ v_max`` and every stage has two layers or more: each stage
  splits at its middle layer into two, the 2S stages placed looped over the old device order
  (stage k on the device of old stage k mod S), moves cleared.
* scheduling — each other policy (moves cleared), then, if the record has a free move slot, every
  adjacent swap ``(d, i, i+1)`` appended as a move on the device with the largest residual bubble
  (bubble minus its leading and trailing idle), then that device's overlap-aware insertions
  (§6 "Scheduling Tuning", the second policy), appended as moves ``(d, j, k)``.

Overlap-aware insertion. On the current schedule (§5's times: every op's start and finish), for
each position k >= 1 of device d's queue, with A = Q[k-1] and B = Q[k]: if the device idles
between them (B starts after A finishes) and a communication there is not overlappable in §5's
sense — A's output goes to another device and B does not run during that transfer
[end A, end A + c], or B's input comes from another device and A does not run during that
transfer — then the first later op Z = Q[j] (j > k) that is ready when A finishes (each of its
producers finished, plus the transfer time for one on another device, by the end of A) moves to
index k, between A and B, where it computes while the communication is in flight. Z cannot
depend on the pending communication, nor on any op it moves ahead of (those start after A
ends), so the move adds no cycle. One insertion per such position, in position order.
"""
import numpy as np

from . import octoref as R

PHASES = ("partition", "placement", "schedule")
POL_ZB = 3


class Layout:
    """Byte layout of candidate records for (P, v_max, max_pert)."""

    def __init__(self, P, v_max, max_pert, stride):
        self.P, self.v_max, self.max_pert, self.stride = P, v_max, max_pert, stride
        self.s_max = P * v_max
        self.po = (3 + 2 * self.s_max + 1) & ~1

    def read(self, rec):
        v = int(rec[1])
        S = self.P * v
        return {
            "policy": int(rec[0]), "v": v, "n_pert": int(rec[2]),
            "b": [0] + [int(x) for x in rec[4:4 + S - 1]],
            "dev": [int(x) for x in rec[3 + self.s_max:3 + self.s_max + S]],
            "pert": [tuple(int(x) for x in np.frombuffer(
                bytes(rec[self.po + 6 * i:self.po + 6 * i + 6]), dtype=np.uint16))
                for i in range(int(rec[2]))],
        }

    def write(self, c, like):
        out = np.array(like, dtype=np.uint8, copy=True)
        S = self.P * c["v"]
        out[0], out[1], out[2] = c["policy"], c["v"], len(c["pert"])
        out[4:4 + self.s_max - 1] = 0
        out[4:4 + S - 1] = c["b"][1:S]
        out[3 + self.s_max:3 + 2 * self.s_max] = 0
        out[3 + self.s_max:3 + self.s_max + S] = c["dev"]
        for i, p in enumerate(c["pert"]):
            out[self.po + 6 * i:self.po + 6 * i + 6] = np.array(p, np.uint16).view(np.uint8)
        return out


def first_arg(x, largest):
    """Index of the largest (or smallest) value, lowest index on ties."""
    best = 0
    for i in range(1, len(x)):
        if (x[i] > x[best]) if largest else (x[i] < x[best]):
            best = i
    return best


def stage_costs(c, costs, L):
    """Per-stage forward, input-gradient and weight-gradient durations of record c."""
    b = c["b"] + [L]
    S = len(c["dev"])
    return ([int(costs[b[s]:b[s + 1], k].sum()) for s in range(S)] for k in range(3))


def producers(op, S):
    """The ops whose outputs op takes (kind 0 F, 1 B, 2 W)."""
    kind, s, m = op
    if kind == 0:
        return [(0, s - 1, m)] if s > 0 else []
    if kind == 1:
        return [(0, s, m)] + ([(1, s + 1, m)] if s < S - 1 else [])
    return [(1, s, m)]


def insertions(prob, costs, link, rec, lay, d):
    """Overlap-aware insertions on device d of record rec: moves (d, j, k), in k order."""
    c = lay.read(rec)
    q = R.dump_queues(prob, rec)
    if q is None:
        return []
    S, M = prob.P * c["v"], prob.M
    split = c["policy"] == POL_ZB
    F, B, W = stage_costs(c, costs, prob.L)
    rc, _, _, start, _ = R.sim_queues(prob.P, S, M, split, c["dev"], F, B, W, link, q,
                                      want_start=True)
    if rc != 0:
        return []
    dev = c["dev"]
    node = lambda op: (op[0] * S + op[1]) * M + op[2]
    dur = lambda op: F[op[1]] if op[0] == 0 else (B[op[1]] + (0 if split else W[op[1]])
                                                    if op[0] == 1 else W[op[1]])
    st = lambda op: int(start[node(op)])
    fin = lambda op: st(op) + dur(op)
    w = lambda p, op: 0 if dev[p[1]] == dev[op[1]] else int(link[dev[p[1]]][dev[op[1]]])
    ready = lambda op: max([fin(p) + w(p, op) for p in producers(op, S)], default=0)

    def out_of(op):  # the consumer on another device and the transfer time, or None
        kind, s, m = op
        t = s + 1 if kind == 0 else s - 1 if kind == 1 else None
        if t is None or t < 0 or t >= S or dev[t] == dev[s]:
            return None
        return int(link[dev[s]][dev[t]])

    def into(op):  # the producer on another device and the transfer time, or None
        for p in producers(op, S):
            if dev[p[1]] != dev[op[1]]:
                return p, int(link[dev[p[1]]][dev[op[1]]])
        return None

    def meets(op, lo, hi):  # op runs during [lo, hi] for a positive length
        return min(fin(op), hi) - max(st(op), lo) > 0

    Q = q[d]
    out = []
    for k in range(1, len(Q)):
        A, Bo = Q[k - 1], Q[k]
        if st(Bo) <= fin(A):
            continue
        co = out_of(A)
        send_alone = co is not None and not meets(Bo, fin(A), fin(A) + co)
        xi = into(Bo)
        recv_alone = xi is not None and not meets(A, fin(xi[0]), fin(xi[0]) + xi[1])
        if not (send_alone or recv_alone):
            continue
        for j in range(k + 1, len(Q)):
            if ready(Q[j]) <= fin(A):
                out.append((d, j, k))
                break
    return out


def neighbours(lay, rec, phase, L, M, busy, bub, resid, ins=()):
    """Records of the phase's neighbourhood, in order (ins: the scheduling phase's insertion
    moves)."""
    c = lay.read(rec)
    P, S = lay.P, lay.P * c["v"]
    stages = [[s for s in range(S) if c["dev"][s] == d] for d in range(P)]
    out = []
    if phase == 0:
        dmax, dmin = first_arg(busy, True), first_arg(busy, False)
        if dmax == dmin:
            return out
        bnd = c["b"] + [L]
        for a in stages[dmax]:
            for b in stages[dmin]:
                if bnd[a + 1] - bnd[a] < 2:
                    continue
                nb = list(c["b"])
                if a < b:
                    for k in range(a + 1, b + 1):
                        nb[k] -= 1
                else:
                    for k in range(b + 1, a + 1):
                        nb[k] += 1
                out.append(lay.write(dict(c, b=nb), rec))
    elif phase == 1:
        d1 = first_arg(bub, True)
        for d2 in range(P):
            if d2 == d1:
                continue
            for s1 in stages[d1]:
                for s2 in stages[d2]:
                    dv = list(c["dev"])
                    dv[s1], dv[s2] = dv[s2], dv[s1]
                    out.append(lay.write(dict(c, dev=dv), rec))
        bnd = c["b"] + [L]
        if 2 * c["v"] <= lay.v_max and all(bnd[s + 1] - bnd[s] >= 2 for s in range(S)):
            nb = []
            for s in range(S):
                nb += [bnd[s], bnd[s] + (bnd[s + 1] - bnd[s]) // 2]
            dv = [c["dev"][k % S] for k in range(2 * S)]
            out.append(lay.write(dict(c, v=2 * c["v"], b=nb, dev=dv, pert=[]), rec))
    else:
        for pol in range(4):
            if pol != c["policy"]:
                out.append(lay.write(dict(c, policy=pol, pert=[]), rec))
        if c["n_pert"] < lay.max_pert:
            d = first_arg(resid, True)
            qlen = (3 if c["policy"] == POL_ZB else 2) * c["v"] * M
            for i in range(qlen - 1):
                out.append(lay.write(dict(c, pert=c["pert"] + [(d, i, i + 1)]), rec))
            for mv in ins:
                out.append(lay.write(dict(c, pert=c["pert"] + [mv]), rec))
    return out


def choose_phase(delta_b, t_layer, b_bd, b_res, exhausted):
    """Algorithm 1's branch: partitioning if Δb > t_layer, else placement if b_bd > b_res, else
    scheduling; an exhausted pick falls to the first phase not exhausted; None: converged."""
    pref = 0 if delta_b > t_layer else 1 if b_bd > b_res else 2
    if pref not in exhausted:
        return pref
    return next((p for p in range(3) if p not in exhausted), None)


def random_phase(record, iteration, seed, exhausted):
    """The random-search variant's pick: the (u mod n)-th of the n open phases; None: all
    exhausted."""
    open_ = [p for p in range(3) if p not in exhausted]
    if not open_:
        return None
    u = R.philox4x64_10([record, iteration, 1, 0], [seed, 0])[0]
    return open_[u % len(open_)]


def bubble_split(ms, bub, bounds):
    """(Δb, b_bd, b_res, busy per device, residual bubble per device) of one evaluation."""
    P = len(bub)
    busy = [ms - b for b in bub]
    lead_trail = [int(bounds[d][0]) + ms - int(bounds[d][1]) for d in range(P)]
    resid = [bub[d] - lead_trail[d] for d in range(P)]
    b_bd = sum(lead_trail)
    return max(bub) - min(bub), b_bd, sum(bub) - b_bd, busy, resid


def tune(prob, costs, link, recs, iters, nthreads=1, trace=None, random_search=False, seed=0,
         insert=True, phase_iters=None):
    """Run `iters` iterations of Algorithm 1 on every record. Returns (final records, makespan,
    bubbles, accepted moves per phase [n, 3], iterations that searched a phase [n] — the rest
    idle after convergence). trace (a list, optional) receives per record a list of
    (phase, kept, makespan after) per searching iteration. random_search: the phase is drawn at
    random (seed) instead of by the bubbles; insert: the scheduling phase includes the
    overlap-aware insertions; phase_iters (an [n, 3] array, optional) receives the iterations
    that searched each phase."""
    lay = Layout(prob.P, prob.v_max, prob.max_pert, prob.cand_stride)
    costs = np.asarray(costs, dtype=np.int64)
    t_layer = prob.M * int(costs.sum(axis=1).min())
    recs = np.array(recs, dtype=np.uint8, copy=True)
    n = len(recs)
    acc = np.zeros((n, 3), dtype=np.int64)
    used = np.zeros(n, dtype=np.int64)
    for i in range(n):
        exhausted = set()
        steps = []
        for it in range(iters):
            ms, bub, bounds = R.sim_batch_bounds(prob, costs, link, recs[i:i + 1])
            ms, bub, bounds = int(ms[0]), [int(x) for x in bub[0]], bounds[0]
            if ms < 0:
                break
            delta_b, b_bd, b_res, busy, resid = bubble_split(ms, bub, bounds)
            if random_search:
                phase = random_phase(i, it, seed, exhausted)
            else:
                phase = choose_phase(delta_b, t_layer, b_bd, b_res, exhausted)
            if phase is None:
                break
            used[i] += 1
            if phase_iters is not None:
                phase_iters[i, phase] += 1
            ins = ()
            if phase == 2 and insert and lay.read(recs[i])["n_pert"] < lay.max_pert:
                ins = insertions(prob, costs, link, recs[i], lay, first_arg(resid, True))
            nb = neighbours(lay, recs[i], phase, prob.L, prob.M, busy, bub, resid, ins)
            best = None
            if nb:
                nms, _ = R.sim_batch(prob, costs, link, np.array(nb), nthreads=nthreads)
                for j, x in enumerate(nms):
                    if x >= 0 and (best is None or x < nms[best]):
                        best = j
            if best is not None and nms[best] < ms:
                recs[i] = nb[best]
                acc[i, phase] += 1
                exhausted = set()
                steps.append((phase, True, int(nms[best])))
            else:
                exhausted.add(phase)
                steps.append((phase, False, ms))
        if trace is not None:
            trace.append(steps)
    ms, bub = R.sim_batch(prob, costs, link, recs, nthreads=nthreads)
    return recs, ms, bub, acc, used
