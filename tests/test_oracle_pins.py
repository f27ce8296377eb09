"""Pins of the CPU oracle against values the paper prints, closed forms from the schedules it
cites, and the paper's own counting arguments. None of these re-type the oracle's formulas."""
import itertools
import math

import numpy as np
import pytest

from conftest import read_golden
from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

F, B, W = 0, 1, 2


def homogeneous(P, v, M, policy, f, placement="looped", link=0):
    """One layer per stage, every layer costs {f, f, f}; returns (makespan, bubbles)."""
    S = P * v
    costs = np.array([[f, f, f]] * S, dtype=np.int64)
    prob = R.problem(L=S, P=P, v_max=v, M=M, cand_stride=I.record_stride(P, v, 0), max_pert=0)
    dev = I.placement(placement, P, v)
    rec = I.pack_records(P, v, 0, [policy], [v], [list(range(1, S))], [dev])
    ms, bub = R.sim_batch(prob, costs, I.link_matrix(P, link), rec)
    return int(ms[0]), bub[0]


def test_fig3_worked_example():
    """§3.2, Fig. 3: 1F1B on two stages costing 2T / 4T per workload, two micro-batches.
    The paper's 10T (≈33%) saving implies a 30T baseline."""
    kv, _ = read_golden("fig3_worked_example.txt")
    T = 1000
    c0, c1 = int(kv["stage0_cost_per_workload_T"]) * T, int(kv["stage1_cost_per_workload_T"]) * T
    costs = np.array([[c0, c0, c0], [c1, c1, c1]], dtype=np.int64)
    prob = R.problem(L=2, P=2, v_max=1, M=int(kv["micro_batches"]),
                     cand_stride=I.record_stride(2, 1, 0), max_pert=0)
    rec = I.pack_records(2, 1, 0, [I.POLICY[kv["policy"]]], [1], [[1]], [[0, 1]])
    ms, bub = R.sim_batch(prob, costs, I.link_matrix(2, 0), rec)
    assert ms[0] == int(kv["baseline_makespan_T"]) * T
    saving = int(kv["saving_T"]) * T
    assert abs(saving / ms[0] - float(kv["saving_fraction_approx"])) < 0.005
    # bubble = makespan - busy: S0 is busy 2 x (2T + 4T), S1 2 x (4T + 8T)
    assert list(bub[0]) == [30 * T - 12 * T, 30 * T - 24 * T]


@pytest.mark.parametrize("P,M", [(1, 1), (1, 5), (2, 1), (2, 2), (3, 7), (4, 2), (4, 8), (5, 3),
                                 (8, 1), (8, 7), (8, 64), (16, 5), (16, 33)])
def test_gpipe_and_1f1b_closed_form(P, M):
    """Homogeneous stages, no transfer cost: AFAB and 1F1B both take (M + P - 1)(f + b), the
    classic pipeline fill/drain bound (GPipe, 1F1B, cited in §1-§2)."""
    f = 7
    want = (M + P - 1) * (f + 2 * f)
    for pol in ("AFAB", "1F1B", "I1F1B"):
        ms, bub = homogeneous(P, 1, M, I.POLICY[pol], f)
        assert ms == want, pol
        assert all(b == (P - 1) * 3 * f for b in bub)


@pytest.mark.parametrize("P,v,M", [(2, 2, 2), (2, 2, 4), (4, 2, 4), (4, 2, 8), (8, 2, 8),
                                   (8, 2, 64), (3, 3, 5), (4, 3, 4), (4, 2, 3), (5, 3, 2),
                                   (16, 2, 8)])
def test_gpipe_looped_closed_form(P, v, M):
    """GPipe (AFAB) with v chunks per device on the looped placement, homogeneous stages, no
    transfer cost. Every forward wave of chunk k + 1 follows chunk k's: with M >= P a device
    is the bottleneck, F(kP + d, m) starts at (kM + d + m) f, so the forwards end at
    (vM + P - 1) f and the backwards mirror them; with M <= P the data are, F(s, m) starts at
    (s + m) f and the forwards end at (vP + M - 1) f. Makespan
    (v max(M, P) + min(M, P) - 1)(f + b). A micro-batch-major forward order (every chunk of
    micro-batch 0 before micro-batch 1), also deadlock-free, gives more, so this pins the
    order, not only the absence of cycles."""
    f = 5
    want = (v * max(M, P) + min(M, P) - 1) * 3 * f
    ms, bub = homogeneous(P, v, M, I.POLICY["AFAB"], f)
    assert ms == want
    S = P * v
    dev = I.placement("looped", P, v)
    qs = []
    for d in range(P):
        A = [s for s in range(S) if dev[s] == d]
        qs.append([(F, s, m) for m in range(M) for s in A] +
                  [(B, s, m) for m in range(M) for s in reversed(A)])
    rc, ms_mb, *_ = R.sim_queues(P, S, M, False, dev, [f] * S, [2 * f] * S, [0] * S,
                                 I.link_matrix(P, 0), qs)
    assert rc == 0 and ms_mb > want


@pytest.mark.parametrize("P,v,M", [(2, 2, 2), (2, 2, 6), (4, 2, 8), (8, 2, 64), (8, 2, 16),
                                   (4, 3, 8), (2, 4, 4), (16, 2, 32)])
def test_interleaved_closed_form(P, v, M):
    """Interleaved 1F1B (cited in §2.2 Placement) divides the fill/drain bubble by the number of
    chunks: with per-chunk costs f, b the step takes (M v + P - 1)(f + b)."""
    f = 5
    ms, _ = homogeneous(P, v, M, I.POLICY["I1F1B"], f)
    assert ms == (M * v + P - 1) * 3 * f


@pytest.mark.parametrize("P,v,M", [(2, 1, 2), (3, 1, 3), (4, 1, 9), (8, 1, 8), (8, 1, 64),
                                   (2, 2, 4), (4, 2, 8), (8, 2, 64)])
def test_zero_bubble_closed_form(P, v, M):
    """Deferred-W schedule (§6 Scheduling Tuning; ZeroBubble cited in §2.2): with F = B = W = t
    the bubble is (P - 1) t, the ZB-H1 value (p - 1)(T_F + T_B - T_W), once M >= P."""
    t = 5
    ms, _ = homogeneous(P, v, M, I.POLICY["ZB"], t)
    assert ms == (3 * M * v + P - 1) * t
    # eager W (lag 0 on every device) is worse: the lag matters
    ms_fused, _ = homogeneous(P, v, M, I.POLICY["I1F1B"], t)
    assert ms <= ms_fused


def test_comm_count_table():
    """§8 comm table: #Comm = send + recv nodes = 2 x cross-device edges = 4 (S-1) M."""
    kv, rows = read_golden("comm_table.txt")
    P, M = int(kv["devices"]), int(kv["micro_batches"])
    for S_str, comm_str in rows:
        S = int(S_str)
        v = S // P
        dev = I.placement("looped", P, v)
        ones = np.ones(S, dtype=np.int64)
        queues = [[(k, s, m) for s in range(S) if dev[s] == d for k in (F, B) for m in range(M)]
                  for d in range(P)]
        _, _, _, _, n_cross = R.sim_queues(P, S, M, False, dev, ones, ones, ones,
                                           I.link_matrix(P, 1), queues)
        assert 2 * n_cross == int(comm_str)


def test_order_count_matches_search_space():
    """§3.3: (2M)!/2^M valid orders of one stage. Enumerate every permutation of the 2M ops on a
    single device; the oracle must find exactly that many free of deadlock."""
    _, rows = read_golden("search_space.txt")
    orders = {int(r[0]): int(r[1]) for r in rows if len(r) == 2}
    one = np.ones(1, dtype=np.int64)
    for M, want in orders.items():
        ops = [(F, 0, m) for m in range(M)] + [(B, 0, m) for m in range(M)]
        ok = 0
        for perm in itertools.permutations(ops):
            rc, ms, _, _, _ = R.sim_queues(1, 1, M, False, [0], one, one, one,
                                           np.zeros((1, 1), np.int64), [list(perm)])
            assert rc in (0, 1)
            ok += rc == 0
            if rc == 0:
                assert ms == 3 * M
        assert ok == want == math.factorial(2 * M) // 2 ** M
    part = [r for r in rows if len(r) == 3][0]
    L, S, n = map(int, part)
    w = I.WORKLOADS[1]
    assert (w.L, w.P) == (L, S)
    assert len(I.candidates(w)) == 2 * n == 2 * math.comb(L - 1, S - 1)


def test_philox_matches_numpy():
    """Philox4x64-10 (Salmon et al., SC'11) against numpy's independent implementation.
    numpy generates the block of counter c+1 first, so it is seeded with c-1."""
    rng = np.random.default_rng(7)
    for _ in range(50):
        key = [int(x) for x in rng.integers(0, 2**63, size=2, dtype=np.uint64)]
        ctr = [int(x) for x in rng.integers(0, 2**63, size=4, dtype=np.uint64)]
        ctr[0] = max(ctr[0], 1)
        bg = np.random.Philox(key=np.array(key, dtype=np.uint64),
                              counter=np.array([ctr[0] - 1] + ctr[1:], dtype=np.uint64))
        assert R.philox4x64_10(ctr, key) == [int(x) for x in bg.random_raw(4)]
    # the tuner's counter shape (chain, step, 0, 0) with key (seed, 0)
    for chain, step in [(0, 1), (4095, 64), (17, 3)]:
        bg = np.random.Philox(key=np.array([12345, 0], dtype=np.uint64),
                              counter=np.array([chain - 1 if chain else 2**64 - 1,
                                                step if chain else step - 1, 0, 0],
                                               dtype=np.uint64))
        assert R.philox4x64_10([chain, step, 0, 0], [12345, 0]) == \
            [int(x) for x in bg.random_raw(4)]
