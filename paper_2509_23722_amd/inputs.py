"""Seeded synthetic inputs: layer-cost tables, link matrices and candidate records.

This module holds no part of the simulator's arithmetic (no queue generation, no timing). It
only draws random numbers and packs the candidate-record byte format that the C ABI defines, so
that the CPU oracle and the HIP path can be fed identical inputs.

The workloads stand in for the paper's profiled layer costs of LLaMA / Jamba / Nemotron-H
(§8, model table), which are not available: per-layer forward costs are drawn per layer type
(uniform or lognormal around a type mean) and the backward halves cost one forward each
(``{F, B, W} = {f, f, f}``; a fused backward therefore costs 2f).
"""
from dataclasses import dataclass
import itertools

import numpy as np

# ---------------------------------------------------------------------------------------------
# Candidate record byte layout (the ABI's format; see include/octo.h)
# ---------------------------------------------------------------------------------------------

POLICY = {"AFAB": 0, "1F1B": 1, "I1F1B": 2, "ZB": 3}
KIND_F, KIND_B, KIND_W = 0, 1, 2


def pert_offset(P, v_max):
    s_max = P * v_max
    return (3 + 2 * s_max + 1) & ~1


def record_stride(P, v_max, max_pert):
    """Smallest record stride (multiple of 16 bytes) holding max_pert perturbations."""
    need = pert_offset(P, v_max) + 6 * max_pert
    return (need + 15) // 16 * 16


def pack_records(P, v_max, max_pert, policy, v, bounds, dev, perts=None, n_pert=None,
                 flags=None):
    """Pack candidate records.

    policy, v: int [n]; bounds: int [n, S_max-1] (b[1..S-1] first, rest ignored);
    dev: int [n, S_max] (first S used); perts: int [n, max_pert, 3] (device, from, to) or None;
    n_pert: int [n] or None. Returns uint8 [n, stride].
    """
    s_max = P * v_max
    n = len(policy)
    stride = record_stride(P, v_max, max_pert)
    rec = np.zeros((n, stride), dtype=np.uint8)
    rec[:, 0] = np.asarray(policy, dtype=np.uint8)
    rec[:, 1] = np.asarray(v, dtype=np.uint8)
    rec[:, 2] = 0 if n_pert is None else np.asarray(n_pert, dtype=np.uint8)
    rec[:, 3] = 0 if flags is None else np.asarray(flags, dtype=np.uint8)
    if s_max > 1:
        rec[:, 4:4 + s_max - 1] = np.asarray(bounds, dtype=np.uint8)[:, :s_max - 1]
    rec[:, 3 + s_max:3 + 2 * s_max] = np.asarray(dev, dtype=np.uint8)[:, :s_max]
    if perts is not None and max_pert > 0:
        po = pert_offset(P, v_max)
        p16 = np.asarray(perts, dtype=np.uint16).reshape(n, max_pert * 3)
        rec[:, po:po + 6 * max_pert] = p16.view(np.uint8).reshape(n, 6 * max_pert)
    return rec


def unpack_record(rec, P, v_max, max_pert):
    """Inverse of pack_records for one record (dict of fields)."""
    s_max = P * v_max
    v = int(rec[1])
    S = P * v
    po = pert_offset(P, v_max)
    npert = int(rec[2])
    p16 = np.frombuffer(bytes(rec[po:po + 6 * max_pert]), dtype=np.uint16).reshape(max_pert, 3) \
        if max_pert else np.zeros((0, 3), dtype=np.uint16)
    return {
        "policy": int(rec[0]), "v": v, "n_pert": npert, "flags": int(rec[3]),
        "b": [0] + [int(x) for x in rec[4:4 + S - 1]],
        "dev": [int(x) for x in rec[3 + s_max:3 + s_max + S]],
        "pert": [tuple(int(x) for x in p16[i]) for i in range(min(npert, max_pert))],
    }


# ---------------------------------------------------------------------------------------------
# Cost tables and links
# ---------------------------------------------------------------------------------------------

MEAN_NS = {"attention": 2_000_000, "mamba": 1_200_000, "moe": 2_400_000, "dense": 1_000_000}


def link_cost_ns(nbytes, latency_ns=20_000, gb_per_s=50):
    """20 us + bytes / (50 GB/s), GB = 1e9 bytes, rounded to the nearest ns."""
    num = nbytes * 1_000_000_000 + 0  # bytes * 1e9 ns/s
    den = gb_per_s * 1_000_000_000
    return latency_ns + (2 * num + den) // (2 * den)


def link_matrix(P, cost):
    m = np.full((P, P), cost, dtype=np.int64)
    np.fill_diagonal(m, 0)
    return m


# MI355X platform links: eight GPUs per node, each pair joined by one xGMI link (seven per GPU)
# of about 153 GB/s per direction; nodes joined by one 400 Gb/s NIC per GPU (50 GB/s). The
# latencies are assumptions of this recipe: 5 us on xGMI, 20 us across nodes (as the paper's
# own link model).
XGMI_GPUS_PER_NODE = 8
XGMI_GB_PER_S, XGMI_LATENCY_NS = 153, 5_000
NIC_GB_PER_S, NIC_LATENCY_NS = 50, 20_000


def xgmi_link_matrix(P, nbytes):
    """Transfer cost (ns) of nbytes between pipeline devices 0..P-1 placed on consecutive GPUs
    of MI355X nodes: xGMI within a node, the NIC between nodes; diagonal 0."""
    intra = link_cost_ns(nbytes, XGMI_LATENCY_NS, XGMI_GB_PER_S)
    inter = link_cost_ns(nbytes, NIC_LATENCY_NS, NIC_GB_PER_S)
    node = np.arange(P) // XGMI_GPUS_PER_NODE
    m = np.where(node[:, None] == node[None, :], intra, inter).astype(np.int64)
    np.fill_diagonal(m, 0)
    return m


def _lognormal_ns(rng, mean_ns, sigma, size=None):
    z = rng.standard_normal(size)
    return np.rint(mean_ns * np.exp(sigma * z)).astype(np.int64)


def _fbw(f):
    f = np.asarray(f, dtype=np.int64)
    return np.stack([f, f, f], axis=1)


# ---------------------------------------------------------------------------------------------
# Workload configurations (synthetic stand-ins; sizes as stated per workload)
# ---------------------------------------------------------------------------------------------

@dataclass(frozen=True)
class Workload:
    key: int
    name: str
    L: int
    P: int
    M: int
    v_max: int
    n: int              # candidates (or chains for the tuner workload)
    max_pert: int
    act_bytes: int
    steps: int = 0      # tuner steps
    seed: int = 0

    @property
    def s_max(self):
        return self.P * self.v_max

    @property
    def stride(self):
        return record_stride(self.P, self.v_max, self.max_pert)

    @property
    def link_ns(self):
        return link_cost_ns(self.act_bytes)


MIB = 1 << 20
WORKLOADS = {
    1: Workload(1, "tiny-exhaustive-16L-P4-M8", 16, 4, 8, 1, 910, 0, 16 * MIB, seed=20250924),
    2: Workload(2, "jamba-like-32L-P8-M32", 32, 8, 32, 1, 65536, 0, 32 * MIB, seed=20250925),
    3: Workload(3, "nemotron-h-like-52L-P8-M64", 52, 8, 64, 2, 1 << 20, 0, 32 * MIB,
                seed=20250926),
    4: Workload(4, "deepseek-v3-like-61L-P16-M128", 61, 16, 128, 2, 262144, 2, 32 * MIB,
                seed=20250927),
    5: Workload(5, "tuner-96L-P32-M256", 96, 32, 256, 2, 4096, 0, 32 * MIB, steps=64,
                seed=20250928),
}


def layer_costs(w: Workload, with_types=False):
    """int64 [L, 3] = {F, B, W} per layer for workload w (and the layer types, if asked)."""
    f, types = _layer_draws(w)
    return (_fbw(f), types) if with_types else _fbw(f)


def _layer_draws(w: Workload):
    rng = np.random.default_rng(w.seed)
    L = w.L
    if w.key == 1:
        f = np.empty(L, dtype=np.int64)
        for i in range(L):
            lo, hi = (800, 1200) if i % 2 == 0 else (1500, 2500)
            f[i] = int(rng.integers(lo, hi, endpoint=True)) * 1000
        return f, ["dense" if i % 2 == 0 else "moe" for i in range(L)]
    if w.key == 2:
        sig = 0.15
        f = np.empty(L, dtype=np.int64)
        types = []
        for i in range(L):
            mixer = "attention" if i % 8 == 0 else "mamba"
            ffn = "moe" if i % 2 == 1 else "dense"
            f[i] = _lognormal_ns(rng, MEAN_NS[mixer], sig) + _lognormal_ns(rng, MEAN_NS[ffn], sig)
            types.append(mixer + "+" + ffn)
        return f, types
    if w.key == 3:
        sig = 0.15
        n_attn = int(round(0.08 * L))
        attn = set(int(x) for x in rng.choice(L, size=n_attn, replace=False))
        types, alt = [], 0
        for i in range(L):
            if i in attn:
                types.append("attention")
            else:
                types.append("mamba" if alt % 2 == 0 else "dense")
                alt += 1
        f = np.array([_lognormal_ns(rng, MEAN_NS[t], sig) for t in types], dtype=np.int64)
        return f, types
    if w.key == 4:
        sig = 0.2
        types = ["dense"] * 3 + ["moe"] * (L - 3)
        f = np.array([_lognormal_ns(rng, MEAN_NS[t], sig) for t in types], dtype=np.int64)
        f[0] += 3 * _lognormal_ns(rng, MEAN_NS["dense"], sig)      # embedding
        f[L - 1] += 3 * _lognormal_ns(rng, MEAN_NS["dense"], sig)  # LM head
        return f, types
    if w.key == 5:
        sig = 0.15
        names = ["attention", "mamba", "moe", "dense"]
        idx = rng.choice(4, size=L, p=[0.2, 0.3, 0.3, 0.2])
        f = np.array([_lognormal_ns(rng, MEAN_NS[names[k]], sig) for k in idx], dtype=np.int64)
        return f, [names[k] for k in idx]
    raise KeyError(w.key)


# Memory per layer type, as multiples of one micro-batch's inter-stage activation (activation
# bytes a layer keeps for its backward) and static GiB (weights, gradients and optimizer state).
MEM_ACT = {"attention": 3.0, "mamba": 2.0, "moe": 2.5, "dense": 2.0}
MEM_STATIC_GIB = {"attention": 1.0, "mamba": 0.8, "moe": 6.0, "dense": 1.5}


def layer_mem(w: Workload):
    """int64 [L, 2] = {activation bytes per micro-batch, static bytes} per layer for workload w:
    per-type means (a combined "mixer+ffn" layer sums both parts), lognormal sigma 0.1, drawn
    from their own seed so that the cost tables stay as they are."""
    _, types = layer_costs(w, with_types=True)
    rng = np.random.default_rng(w.seed + 3000)
    act = np.empty(w.L, dtype=np.int64)
    st = np.empty(w.L, dtype=np.int64)
    for i, t in enumerate(types):
        parts = t.split("+")
        a = sum(MEM_ACT[p] for p in parts) * w.act_bytes
        g = sum(MEM_STATIC_GIB[p] for p in parts) * (1 << 30)
        act[i] = int(np.rint(a * np.exp(0.1 * rng.standard_normal())))
        st[i] = int(np.rint(g * np.exp(0.1 * rng.standard_normal())))
    # embedding and LM head of the DeepSeek-V3-like model carry large tables
    if w.key == 4:
        st[0] += 2 << 30
        st[w.L - 1] += 2 << 30
    return np.stack([act, st], axis=1)


# ---------------------------------------------------------------------------------------------
# Placements (input patterns; stage -> device maps)
# ---------------------------------------------------------------------------------------------

PLACEMENTS = ("blocked", "looped", "vshape", "random")


def placement(kind, P, v, rng=None):
    S = P * v
    s = np.arange(S)
    if kind == "blocked":
        return s // v
    if kind == "looped":
        return s % P
    if kind == "vshape":
        k, i = s // P, s % P
        return np.where(k % 2 == 0, i, P - 1 - i)
    if kind == "random":
        return rng.permutation(S) % P
    raise KeyError(kind)


def random_cuts(rng, L, S, n):
    """n uniform random (S-1)-subsets of {1..L-1}, sorted: uniform contiguous partitions."""
    if S <= 1:
        return np.zeros((n, 0), dtype=np.int64)
    keys = rng.random((n, L - 1))
    cuts = np.argsort(keys, axis=1)[:, :S - 1] + 1
    return np.sort(cuts, axis=1)


def _pad_bounds(cuts, s_max):
    n = cuts.shape[0]
    out = np.zeros((n, max(s_max - 1, 0)), dtype=np.int64)
    out[:, :cuts.shape[1]] = cuts
    return out


def _pad_dev(dev, s_max):
    n = dev.shape[0]
    out = np.zeros((n, s_max), dtype=np.int64)
    out[:, :dev.shape[1]] = dev
    return out


def candidates(w: Workload, n=None):
    """Candidate records for workload w (uint8 [n, stride]). Deterministic in w.seed."""
    rng = np.random.default_rng(w.seed + 1000)
    P, L, s_max = w.P, w.L, w.s_max
    if w.key == 1:
        rows = []
        for cuts in itertools.combinations(range(1, L), P - 1):
            for pol in (POLICY["AFAB"], POLICY["1F1B"]):
                rows.append((pol, cuts))
        if n is not None:
            rows = rows[:n]
        pol = np.array([r[0] for r in rows])
        bnd = np.array([r[1] for r in rows])
        dev = np.tile(np.arange(P), (len(rows), 1))
        return pack_records(P, w.v_max, w.max_pert, pol, np.ones(len(rows)), bnd, dev)
    n = w.n if n is None else n
    if w.key == 2:
        cuts = random_cuts(rng, L, P, n)
        dev = rng.permuted(np.tile(np.arange(P), (n, 1)), axis=1)
        pol = rng.integers(0, 2, size=n)
        return pack_records(P, 1, w.max_pert, pol, np.ones(n), cuts, dev)
    if w.key == 3:
        # 32 strata = v {1,2} x placement {blocked, looped, vshape, random} x policy {4},
        # equally filled, in a seeded random order.
        strata = np.arange(n) % 32
        rng.shuffle(strata)
        v = 1 + (strata // 16)
        plc = (strata // 4) % 4
        pol = strata % 4
        bnd = np.zeros((n, s_max - 1), dtype=np.int64)
        dev = np.zeros((n, s_max), dtype=np.int64)
        for vv in (1, 2):
            S = P * vv
            sel = np.nonzero(v == vv)[0]
            bnd[sel] = _pad_bounds(random_cuts(rng, L, S, len(sel)), s_max)
            for pi, pk in enumerate(PLACEMENTS):
                ss = sel[plc[sel] == pi]
                if pk == "random":
                    d = np.stack([placement("random", P, vv, rng) for _ in range(len(ss))]) \
                        if len(ss) else np.zeros((0, S), dtype=np.int64)
                else:
                    d = np.tile(placement(pk, P, vv), (len(ss), 1))
                dev[ss] = _pad_dev(d, s_max)
        return pack_records(P, w.v_max, w.max_pert, pol, v, bnd, dev)
    if w.key == 4:
        v = 2
        S = P * v
        cuts = random_cuts(rng, L, S, n)
        relabel = rng.integers(0, 2, size=n).astype(bool)
        pi = rng.permuted(np.tile(np.arange(P), (n, 1)), axis=1)
        pi[~relabel] = np.arange(P)
        dev = pi[:, np.arange(S) % P]
        pol = np.where(rng.integers(0, 2, size=n) == 0, POLICY["I1F1B"], POLICY["ZB"])
        # 1% deliberately cyclic orders: move a device's last op to the front, which puts a
        # backward (or weight-gradient) op ahead of the forward it needs (§3.3).
        n_cyc = n // 100
        cyc = rng.choice(n, size=n_cyc, replace=False)
        n_pert = np.zeros(n, dtype=np.int64)
        perts = np.zeros((n, w.max_pert, 3), dtype=np.int64)
        qlen = np.where(pol == POLICY["ZB"], 3, 2) * v * w.M
        n_pert[cyc] = 1
        perts[cyc, 0, 0] = rng.integers(0, P, size=n_cyc)
        perts[cyc, 0, 1] = qlen[cyc] - 1
        perts[cyc, 0, 2] = 0
        return pack_records(P, w.v_max, w.max_pert, pol, np.full(n, v), cuts, dev, perts,
                            n_pert)
    if w.key == 5:
        return tuner_chains(w, n)
    raise KeyError(w.key)


def cyclic_indices(w: Workload):
    """Indices of the deliberately cyclic candidates of workload 4."""
    recs = candidates(w)
    return np.nonzero(recs[:, 2] > 0)[0]


def tuner_chains(w: Workload, n=None):
    """Initial chain candidates: uniform partition, looped v=2 with a random device relabel,
    policy in {I1F1B, ZB}."""
    rng = np.random.default_rng(w.seed + 2000)
    n = w.n if n is None else n
    P, v = w.P, w.v_max
    S = P * v
    cuts = random_cuts(rng, w.L, S, n)
    pi = rng.permuted(np.tile(np.arange(P), (n, 1)), axis=1)
    dev = pi[:, np.arange(S) % P]
    pol = np.where(rng.integers(0, 2, size=n) == 0, POLICY["I1F1B"], POLICY["ZB"])
    return pack_records(P, v, w.max_pert, pol, np.full(n, v), cuts, dev)


# ---------------------------------------------------------------------------------------------
# Generic random candidates (parity fuzzing on small structures)
# ---------------------------------------------------------------------------------------------

def random_candidates(rng, L, P, v_max, M, n, max_pert=0, pert_rate=0.0, invalid_rate=0.0,
                      policies=(0, 1, 2, 3)):
    """Random candidates of every policy/v/placement kind, optional random moves, and a share of
    deliberately invalid records (empty stage, unbalanced placement, bad policy/flags/v, moves
    out of range)."""
    s_max = P * v_max
    vs = rng.integers(1, v_max + 1, size=n)
    if L < P * vs.max():
        vs = np.minimum(vs, max(1, L // P))
    pol = rng.choice(np.array(policies), size=n)
    bnd = np.zeros((n, max(s_max - 1, 0)), dtype=np.int64)
    dev = np.zeros((n, s_max), dtype=np.int64)
    for i in range(n):
        S = P * int(vs[i])
        c = random_cuts(rng, L, S, 1)[0]
        bnd[i, :S - 1] = c
        kind = PLACEMENTS[int(rng.integers(0, 4))]
        d = placement(kind, P, int(vs[i]), rng)
        if kind != "random" and rng.random() < 0.5:
            d = rng.permutation(P)[d]  # device relabel
        dev[i, :S] = d
    n_pert = np.zeros(n, dtype=np.int64)
    perts = np.zeros((n, max(max_pert, 1), 3), dtype=np.int64)
    if max_pert > 0:
        qlen = np.where(pol == POLICY["ZB"], 3, 2) * vs * M
        for i in range(n):
            if rng.random() < pert_rate:
                k = int(rng.integers(1, max_pert + 1))
                n_pert[i] = k
                for j in range(k):
                    perts[i, j] = (int(rng.integers(0, P)), int(rng.integers(0, qlen[i])),
                                   int(rng.integers(0, qlen[i])))
    flags = np.zeros(n, dtype=np.int64)
    v_field = vs.copy()
    for i in range(n):
        if rng.random() >= invalid_rate:
            continue
        S = P * int(vs[i])
        kind = int(rng.integers(0, 6))
        if kind == 0 and S >= 2:      # empty stage
            j = int(rng.integers(0, S - 1))
            bnd[i, j] = bnd[i, j - 1] if j > 0 else 0
        elif kind == 1 and P >= 2:    # unbalanced placement
            dev[i, 0] = (dev[i, 0] + 1) % P
        elif kind == 2:               # unknown policy
            pol[i] = 4 + int(rng.integers(0, 3))
        elif kind == 3:               # reserved flags
            flags[i] = 1
        elif kind == 4:               # v out of range
            v_field[i] = v_max + 1 if rng.random() < 0.5 else 0
        elif kind == 5 and max_pert > 0:  # move out of range
            qlen = (3 if pol[i] == POLICY["ZB"] else 2) * vs[i] * M
            n_pert[i] = 1
            perts[i, 0] = (int(rng.integers(0, P)), int(qlen), 0)
        else:
            pol[i] = 9
    return pack_records(P, v_max, max_pert, pol, v_field, bnd, dev,
                        perts[:, :max_pert] if max_pert else None, n_pert, flags)
