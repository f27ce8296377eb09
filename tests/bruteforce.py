"""Independent pure-Python checkers for tiny instances (test infrastructure).

These recompute the time model of §5 by different means than the C oracle, so that the oracle
is pinned to something other than itself:

* ``tick_simulate`` advances an integer clock one tick at a time; at every tick each idle device
  starts its next op if all producers have delivered (finish + transfer <= now). This is the
  as-soon-as-possible execution the paper's traversal records (§5 "Estimating Pipeline
  Performance"), obtained without any graph algorithm. Durations must be small integers.
  With ``serial``, a directed link carries one transfer at a time: when an op ends, each of its
  transfers joins its link's queue and starts once the link is free.
* ``rdv_tick_simulate`` executes device programs with blocking rendezvous transfers (the naive
  coordination of §3.3): each device receives an op's cross-device input right before the op and
  sends its cross-device output right after it; a device that reaches a send or receive waits
  there, and once both ends have arrived the transfer runs for the link time, holding both.
  Tick by tick, with no graph: a program that can never move again is a deadlock.
* ``reorder_programs`` builds the executor's reordered programs (§7's three steps: mismatched
  receives, their feasible windows, the greedy cheapest gap by span minus overlap) from a
  tick-by-tick asynchronous run and levels found by fixpoint iteration; ``handshake_tick_simulate``
  executes programs tick by tick with handshake transfers (a device waits at a send or receive
  until the other end is reached; the data arrives the link time later while both compute).
* ``has_cycle`` builds the dependency graph from its definition (§5, §6 "Scheduling Tuning") and
  runs an iterative three-colour DFS.

Queues are lists (per device) of (kind, stage, m) with kind 0 = F, 1 = B, 2 = W.
"""
import itertools

F, B, W = 0, 1, 2


def _dur(kind, s, split, Fs, Bs, Ws):
    if kind == F:
        return Fs[s]
    if kind == B:
        return Bs[s] if split else Bs[s] + Ws[s]
    return Ws[s]


def _producers(op, S, split, dev, link):
    """(producer op, transfer cost) pairs of op, from the dependency rules."""
    kind, s, m = op
    out = []
    if kind == F and s > 0:
        out.append(((F, s - 1, m), 0 if dev[s - 1] == dev[s] else link[dev[s - 1]][dev[s]]))
    if kind == B:
        out.append(((F, s, m), 0))
        if s < S - 1:
            out.append(((B, s + 1, m), 0 if dev[s + 1] == dev[s] else link[dev[s + 1]][dev[s]]))
    if kind == W:
        out.append(((B, s, m), 0))
    return out


def _consumers(op, S, dev):
    """Ops on other devices that take op's output."""
    kind, s, m = op
    if kind == F and s < S - 1 and dev[s + 1] != dev[s]:
        return [(F, s + 1, m)]
    if kind == B and s > 0 and dev[s - 1] != dev[s]:
        return [(B, s - 1, m)]
    return []


def tick_simulate(P, S, M, split, dev, Fs, Bs, Ws, link, queues, max_ticks=None, serial=False,
                  starts=None):
    """Returns (makespan, bubbles) or (-1, [-1]*P) on deadlock. starts (a dict, optional)
    receives each op's start tick."""
    total = sum(_dur(k, s, split, Fs, Bs, Ws) for q in queues for (k, s, m) in q)
    if max_ticks is None:
        max_ticks = total + 2 * S * M * (max(max(r) for r in link) if P > 0 else 0) + 2
    arrive = {}                        # (producer, consumer) -> arrival tick (serial links)
    link_free = {}                     # (p, q) -> tick the link is free again

    def sent(op, t):
        for c in _consumers(op, S, dev):
            key = (dev[op[1]], dev[c[1]])
            go = max(t, link_free.get(key, 0))
            arrive[(op, c)] = go + link[key[0]][key[1]]
            link_free[key] = arrive[(op, c)]

    def delivered(p, w, op, t):
        if serial and (p, op) in arrive:
            return arrive[(p, op)] <= t
        return p in fin and fin[p] + w <= t

    fin = {}
    ptr = [0] * P
    busy_until = [0] * P
    running = [None] * P
    t = 0
    while t <= max_ticks:
        for d in range(P):
            if running[d] is not None and busy_until[d] <= t:
                fin[running[d]] = busy_until[d]
                sent(running[d], busy_until[d])
                running[d] = None
        for d in range(P):
            if running[d] is None and ptr[d] < len(queues[d]):
                op = queues[d][ptr[d]]
                ok = all(delivered(p, w, op, t) for p, w in _producers(op, S, split, dev, link))
                if ok:
                    running[d] = op
                    if starts is not None:
                        starts[op] = t
                    busy_until[d] = t + _dur(op[0], op[1], split, Fs, Bs, Ws)
                    ptr[d] += 1
                    if busy_until[d] == t:  # zero-length op finishes immediately
                        fin[op] = t
                        sent(op, t)
                        running[d] = None
        if all(ptr[d] == len(queues[d]) and running[d] is None for d in range(P)):
            break
        t += 1
    if not all(ptr[d] == len(queues[d]) and running[d] is None for d in range(P)):
        return -1, [-1] * P
    ms = max(fin.values()) if fin else 0
    bub = [ms - sum(_dur(k, s, split, Fs, Bs, Ws) for (k, s, m) in queues[d]) for d in range(P)]
    return ms, bub


def rdv_programs(S, dev, queues):
    """Per device: ("r", producer op) before an op with a cross-device input, ("c", op), and
    ("s", op) after an op with a cross-device output. A transfer is named by its producer."""
    progs = []
    for d, q in enumerate(queues):
        prog = []
        for op in q:
            kind, s, m = op
            if kind == F and s > 0 and dev[s - 1] != d:
                prog.append(("r", (F, s - 1, m)))
            if kind == B and s < S - 1 and dev[s + 1] != d:
                prog.append(("r", (B, s + 1, m)))
            prog.append(("c", op))
            if _consumers(op, S, dev):
                prog.append(("s", op))
        progs.append(prog)
    return progs


def ordered_programs(S, M, split, dev, Fs, Bs, Ws, queues, starts):
    """The reordered coordination: a device keeps its compute order and places each transfer at
    the end of its producer in the asynchronous schedule (starts: op -> start); its items are
    sorted by (time, communication first, then the producer's node id (kind S + stage) M + m
    for a transfer or the queue position for a computation)."""
    node = lambda op: (op[0] * S + op[1]) * M + op[2]
    end = lambda op: starts[op] + _dur(op[0], op[1], split, Fs, Bs, Ws)
    progs = []
    for d, q in enumerate(queues):
        items = []
        for i, op in enumerate(q):
            kind, s, m = op
            items.append(((starts[op], 1, i), ("c", op)))
            src = None
            if kind == F and s > 0 and dev[s - 1] != d:
                src = (F, s - 1, m)
            if kind == B and s < S - 1 and dev[s + 1] != d:
                src = (B, s + 1, m)
            if src is not None:
                items.append(((end(src), 0, node(src)), ("r", src)))
            if _consumers(op, S, dev):
                items.append(((end(op), 0, node(op)), ("s", op)))
        progs.append([it for _, it in sorted(items)])
    return progs


def rdv_tick_simulate(P, S, M, split, dev, Fs, Bs, Ws, link, queues, progs=None):
    """Returns (makespan, bubbles) or (-1, [-1]*P) on deadlock. progs: the device programs
    (default: the naive coordination)."""
    if progs is None:
        progs = rdv_programs(S, dev, queues)
    total = sum(_dur(k, s, split, Fs, Bs, Ws) for q in queues for (k, s, m) in q)
    max_ticks = total + sum(max(r) for r in link) * 2 * S * M + 2
    ptr = [0] * P
    running = [None] * P               # ("c", op) or ("x", transfer) until busy_until
    busy_until = [0] * P
    arrived = {}                       # transfer -> the ends ("s", "r") waiting at it
    fin = {}
    t = 0
    while t <= max_ticks:
        changed = True
        while changed:
            changed = False
            for d in range(P):
                if running[d] is not None and busy_until[d] <= t:
                    if running[d][0] == "c":
                        fin[running[d][1]] = busy_until[d]
                    running[d] = None
                    ptr[d] += 1
                    changed = True
            for d in range(P):
                if running[d] is not None or ptr[d] >= len(progs[d]):
                    continue
                what, x = progs[d][ptr[d]]
                if what == "c":
                    local = [p for p, _ in _producers(x, S, split, dev, link) if dev[p[1]] == d]
                    if all(p in fin and fin[p] <= t for p in local):
                        running[d] = ("c", x)
                        busy_until[d] = t + _dur(x[0], x[1], split, Fs, Bs, Ws)
                        changed = True
                elif what == "s" and not (x in fin and fin[x] <= t):
                    pass                       # a send waits for its producer
                elif what not in arrived.setdefault(x, set()):
                    arrived[x].add(what)
                    if arrived[x] == {"s", "r"}:
                        p = dev[x[1]]
                        q = dev[_consumers(x, S, dev)[0][1]]
                        for e in (p, q):
                            running[e] = ("x", x)
                            busy_until[e] = t + link[p][q]
                    changed = True
        if all(ptr[d] == len(progs[d]) for d in range(P)):
            break
        t += 1
    if not all(ptr[d] == len(progs[d]) for d in range(P)):
        return -1, [-1] * P
    ms = max(max(fin.values(), default=0), max(busy_until, default=0))
    bub = [ms - sum(_dur(k, s, split, Fs, Bs, Ws) for (k, s, m) in queues[d]) for d in range(P)]
    return ms, bub


def levels(S, split, dev, queues):
    """Number of ops on the longest dependency chain before each op (queue order and data
    dependencies), by iterating lvl(op) = max(lvl(pred) + 1) to a fixpoint."""
    lvl = {op: 0 for q in queues for op in q}
    preds = {}
    for q in queues:
        for i, op in enumerate(q):
            ps = [p for p, _ in _producers(op, S, split, dev, [[0] * len(queues)] * len(queues))]
            if i > 0:
                ps.append(q[i - 1])
            preds[op] = ps
    changed = True
    while changed:
        changed = False
        for op, ps in preds.items():
            v = max([lvl[p] + 1 for p in ps], default=0)
            if v != lvl[op]:
                lvl[op], changed = v, True
    return lvl


def reorder_programs(S, M, split, dev, Fs, Bs, Ws, link, queues, starts, lvl):
    """The executor's reordering (see the module docstring). Returns (programs, transfers,
    mismatched receives)."""
    node = lambda op: (op[0] * S + op[1]) * M + op[2]
    dur = lambda op: _dur(op[0], op[1], split, Fs, Bs, Ws)
    end = lambda op: starts[op] + dur(op)
    progs, ntr, nmis = [], 0, 0
    for d, q in enumerate(queues):
        post = [0] + [end(op) for op in q]
        items = []                                   # [key, gap, item]
        for i, op in enumerate(q):
            kind, s, m = op
            src = None
            if kind == F and s > 0 and dev[s - 1] != d:
                src = (F, s - 1, m)
            if kind == B and s < S - 1 and dev[s + 1] != d:
                src = (B, s + 1, m)
            if src is not None:
                items.append([(end(src), lvl[src], node(src)), i, ("r", src)])
                ntr += 1
            if _consumers(op, S, dev):
                items.append([(end(op), lvl[op], node(op)), i + 1, ("s", op)])
        rec, flagged = [], []
        for it in items:
            if not rec or it[0] > rec[-1][0]:
                rec.append(it)
            else:
                flagged.append(it)
        nmis += len(flagged)
        lastg = 0
        for f in sorted(flagged, key=lambda it: it[0]):
            assert f[2][0] == "r"
            lo = max([lastg] + [r[1] for r in rec if r[0] < f[0]])
            hi = min(r[1] for r in rec if r[0] > f[0])
            X, iY = f[2][1], f[1]
            c = link[dev[X[1]]][d]
            gx = next((g for g in range(len(q) + 1) if post[g] >= starts[X]), len(q) + 1)
            first = min(max(lo, gx), hi)
            best = None
            for g in range(hi, first - 1, -1):
                cost = abs(end(X) - post[g]) - min(c, sum(dur(q[j]) for j in range(g, iY)))
                if best is None or cost < best[0]:
                    best = (cost, g)
            f[1] = lastg = best[1]
        allc = sorted(items, key=lambda it: it[0])
        assert all(allc[j][1] <= allc[j + 1][1] for j in range(len(allc) - 1))
        prog, j = [], 0
        for i, op in enumerate(q):
            while j < len(allc) and allc[j][1] <= i:
                prog.append(allc[j][2])
                j += 1
            prog.append(("c", op))
        prog += [it[2] for it in allc[j:]]
        progs.append(prog)
    return progs, ntr, nmis


def handshake_tick_simulate(P, S, M, split, dev, Fs, Bs, Ws, link, queues, progs):
    """Returns (makespan, bubbles) or (-1, [-1]*P) on deadlock."""
    total = sum(_dur(k, s, split, Fs, Bs, Ws) for q in queues for (k, s, m) in q)
    max_ticks = total + sum(max(r) for r in link) * 2 * S * M + 2
    ptr = [0] * P
    running = [None] * P
    busy_until = [0] * P
    waiting = {}                       # transfer -> the device waiting at its other end
    arrival = {}                       # transfer -> tick its data arrives
    fin = {}
    t = 0
    while t <= max_ticks:
        changed = True
        while changed:
            changed = False
            for d in range(P):
                if running[d] is not None and busy_until[d] <= t:
                    fin[running[d]] = busy_until[d]
                    running[d] = None
                    ptr[d] += 1
                    changed = True
            for d in range(P):
                if running[d] is not None or ptr[d] >= len(progs[d]):
                    continue
                what, x = progs[d][ptr[d]]
                if what == "c":
                    ok = True
                    for p, _ in _producers(x, S, split, dev, link):
                        if dev[p[1]] == d:
                            ok = ok and p in fin and fin[p] <= t
                        else:
                            ok = ok and p in arrival and arrival[p] <= t
                    if ok:
                        running[d] = x
                        busy_until[d] = t + _dur(x[0], x[1], split, Fs, Bs, Ws)
                        changed = True
                elif what == "s" and not (x in fin and fin[x] <= t):
                    pass                               # a send waits for its producer
                elif x in waiting and waiting[x] != d:
                    other = waiting.pop(x)
                    p = dev[x[1]]
                    q = dev[_consumers(x, S, dev)[0][1]]
                    arrival[x] = t + link[p][q]
                    ptr[other] += 1
                    ptr[d] += 1
                    changed = True
                elif x not in waiting:
                    waiting[x] = d
                    changed = True
        if all(ptr[d] == len(progs[d]) and running[d] is None for d in range(P)):
            break
        t += 1
    if not all(ptr[d] == len(progs[d]) for d in range(P)):
        return -1, [-1] * P
    ms = max(fin.values(), default=0)
    bub = [ms - sum(_dur(k, s, split, Fs, Bs, Ws) for (k, s, m) in queues[d]) for d in range(P)]
    return ms, bub


def has_cycle(P, S, M, split, dev, queues):
    nodes = [(k, s, m) for k in range(3 if split else 2) for s in range(S) for m in range(M)]
    succ = {n: [] for n in nodes}
    for q in queues:
        for a, b in zip(q, q[1:]):
            succ[a].append(b)
    for n in nodes:
        for p, _ in _producers(n, S, split, dev, [[0] * P for _ in range(P)]):
            succ[p].append(n)
    color = {n: 0 for n in nodes}
    for root in nodes:
        if color[root]:
            continue
        stack = [(root, iter(succ[root]))]
        color[root] = 1
        while stack:
            node, it = stack[-1]
            nxt = next(it, None)
            if nxt is None:
                color[node] = 2
                stack.pop()
            elif color[nxt] == 1:
                return True
            elif color[nxt] == 0:
                color[nxt] = 1
                stack.append((nxt, iter(succ[nxt])))
    return False


def valid_stage_orders(s, M):
    """All orders of one stage's F/B ops in which each B(m) follows F(m) ((2M)!/2^M of them)."""
    ops = [(F, s, m) for m in range(M)] + [(B, s, m) for m in range(M)]
    for perm in itertools.permutations(ops):
        pos = {op: i for i, op in enumerate(perm)}
        if all(pos[(F, s, m)] < pos[(B, s, m)] for m in range(M)):
            yield list(perm)
