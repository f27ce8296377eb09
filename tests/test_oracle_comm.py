"""Pins of the oracle's communication accounting (§5: send and receive nodes of every
cross-device dependency; a node that can run beside subsequent computation is overlappable and
records the smaller of the computation's and the communication's durations; the #Comm column of
§8's communication table).

Reading: a send node can run beside the op that follows its producer on the producer's device,
a receive node beside the op that precedes its consumer on the consumer's device (the consumer
itself waits for the data); the node is overlappable when that op runs during the transfer
[end of producer, + c], and its overlap time is min(duration of that op, c)."""
import numpy as np
import pytest

from conftest import read_golden
from oracle import octoref as R
from paper_2509_23722_amd import inputs as I

NTHREADS = 4


def chain(P, M, pol, f, b, c, split_w=None):
    """One stage per device, uniform stage costs (fused backward b), link cost c."""
    recs = I.pack_records(P, 1, 0, [pol], [1], [np.arange(1, P)], [np.arange(P)])
    prob = R.problem(P, P, 1, M, recs.shape[1], 0)
    costs = np.tile(np.array([[f, b - (split_w or 0), split_w or 0]], np.int64), (P, 1))
    return R.sim_batch_comm(prob, costs, I.link_matrix(P, c), recs)


def test_worked_example():
    kv, _ = read_golden("comm_worked_example.txt")
    T = int(kv["T_ns"])
    recs = I.pack_records(2, 1, 0, [I.POLICY["1F1B"]], [1], [[1]], [[0, 1]])
    prob = R.problem(2, 2, 1, 2, recs.shape[1], 0)
    costs = np.array([[2, 2, 2], [4, 4, 4]], np.int64) * T
    ms, _, comm = R.sim_batch_comm(prob, costs, I.link_matrix(2, int(kv["transfer_T"]) * T), recs)
    assert ms[0] == int(kv["makespan_T"]) * T
    assert comm[0].tolist() == [int(kv["comm_nodes"]), int(kv["overlapped_nodes"]),
                                int(kv["comm_time_T"]) * T, int(kv["overlap_time_T"]) * T]


def test_min_rule_example():
    """A GPipe case worked by hand where a receive's transfer only partly meets the op it runs
    beside: §5's min(computation, communication) gives 6T, the intersection would give 5T."""
    kv, _ = read_golden("comm_min_rule_example.txt")
    T = int(kv["T_ns"])
    recs = I.pack_records(2, 1, 0, [I.POLICY["AFAB"]], [1], [[1]], [[0, 1]])
    prob = R.problem(2, 2, 1, 2, recs.shape[1], 0)
    f0, b0 = int(kv["stage0_F_T"]) * T, int(kv["stage0_bwd_T"]) * T
    f1, b1 = int(kv["stage1_F_T"]) * T, int(kv["stage1_bwd_T"]) * T
    costs = np.array([[f0, b0 // 2, b0 - b0 // 2], [f1, b1 // 2, b1 - b1 // 2]], np.int64)
    ms, _, comm = R.sim_batch_comm(prob, costs, I.link_matrix(2, int(kv["transfer_T"]) * T), recs)
    assert ms[0] == int(kv["makespan_T"]) * T
    assert comm[0].tolist() == [int(kv["comm_nodes"]), int(kv["overlapped_nodes"]),
                                int(kv["comm_time_T"]) * T, int(kv["overlap_time_T"]) * T]


def test_overlap_time_is_min_of_durations():
    """Overlap time per overlappable node is at most min(c, longest op) and, on uniform stages
    with every op at least as long as c, exactly c: the sum is then c x overlappable nodes."""
    for pol in ("1F1B", "AFAB"):
        ms, _, comm = chain(6, 12, I.POLICY[pol], 1000, 2000, 700)
        assert comm[0, 1] > 0 and comm[0, 3] == 700 * comm[0, 1]
    ms, _, comm = chain(6, 12, I.POLICY["1F1B"], 1000, 2000, 1500)
    assert 0 < comm[0, 3] <= 1500 * comm[0, 1]
    assert comm[0, 3] >= 1000 * comm[0, 1]


@pytest.mark.parametrize("P,M,f,b,c", [(2, 2, 1000, 2000, 300), (4, 8, 1000, 1000, 1000),
                                       (8, 16, 700, 1500, 50), (3, 5, 900, 1900, 899)])
def test_afab_closed_form(P, M, f, b, c):
    """GPipe on uniform stages with 0 < c <= min(f, b): F(d, m) runs [(m+d) f + d c, +f], so
    each forward's transfer runs beside the next forward of its device and arrives during the
    previous forward of the receiver — except the last forward's send and the first forward's
    receive; the backward sweep mirrors it. Overlapped nodes 4 (P-1)(M-1), each for
    min(op, c) = c."""
    ms, _, comm = chain(P, M, I.POLICY["AFAB"], f, b, c)
    n = 4 * (P - 1)
    assert comm[0].tolist() == [n * M, n * (M - 1), n * M * c, n * (M - 1) * c]


def test_comm_count_table():
    """§8 communication table: #Comm = 4 (S-1) M when every stage boundary crosses devices."""
    kv, rows = read_golden("comm_table.txt")
    P, M = int(kv["devices"]), int(kv["micro_batches"])
    for S_str, comm_str in rows:
        S = int(S_str)
        v = S // P
        recs = I.pack_records(P, v, 0, [I.POLICY["I1F1B"]], [v], [np.arange(1, S)],
                              [I.placement("looped", P, v)])
        prob = R.problem(S, P, v, M, recs.shape[1], 0)
        ms, _, comm = R.sim_batch_comm(prob, np.full((S, 3), 1000, np.int64),
                                       I.link_matrix(P, 200), recs)
        assert ms[0] > 0 and comm[0, 0] == int(comm_str)


def test_free_links_and_one_device():
    """Zero-cost transfers still are nodes but overlap nothing; one device has no nodes."""
    ms, _, comm = chain(4, 6, I.POLICY["1F1B"], 1000, 2000, 0)
    assert comm[0].tolist() == [4 * 3 * 6, 0, 0, 0]
    ms, _, comm = chain(1, 6, I.POLICY["1F1B"], 1000, 2000, 500)
    assert comm[0].tolist() == [0, 0, 0, 0]


def test_counts_and_bounds_on_random_candidates():
    """Nodes = 4 M per cross-device stage boundary and their time 2 M (c_fwd + c_bwd) per
    boundary — the schedule cannot change them; overlap counts and times are bounded by them;
    the times are those of the plain evaluation; sentinels for deadlock / invalid."""
    rng = np.random.default_rng(17)
    L, P, v, M = 20, 4, 2, 8
    recs = I.random_candidates(rng, L, P, v, M, 300, max_pert=2, pert_rate=0.3,
                               invalid_rate=0.1)
    prob = R.problem(L, P, v, M, recs.shape[1], 2)
    costs = rng.integers(1, 3_000_000, size=(L, 3)).astype(np.int64)
    link = rng.integers(0, 900_000, size=(P, P)).astype(np.int64)
    ms, bub, comm = R.sim_batch_comm(prob, costs, link, recs, NTHREADS)
    ms2, bub2 = R.sim_batch(prob, costs, link, recs, NTHREADS)
    assert (ms == ms2).all() and (bub == bub2).all()
    bad = ms < 0
    assert (comm[bad] == ms[bad, None]).all() and bad.sum() > 10
    for i in np.nonzero(~bad)[0]:
        c = I.unpack_record(recs[i], P, v, 2)
        dev = c["dev"]
        cross = [s for s in range(len(dev) - 1) if dev[s] != dev[s + 1]]
        assert comm[i, 0] == 4 * M * len(cross)
        assert comm[i, 2] == 2 * M * sum(int(link[dev[s], dev[s + 1]] + link[dev[s + 1], dev[s]])
                                         for s in cross)
    ok = ~bad
    assert (comm[ok, 1] <= comm[ok, 0]).all() and (comm[ok, 3] <= comm[ok, 2]).all()
    assert ((comm[ok, 1] > 0) == (comm[ok, 3] > 0)).all() and (comm[ok, 1] > 0).sum() > 100


def test_table_schedules_under_the_adopted_rule():
    """§8's communication table prints #Overlap 112 of 224 for 1F1B at 8 stages and 1,330 of
    1,760 for Interleaved at 56 stages (PP 8, M 8). Under the adopted reading of §5 the
    textbook schedules on uniform costs (a 1F1B stage of 7 chunk costs, transfers a tenth of a
    1F1B stage's forward) give 98 and 1,074 overlappable nodes, each overlapping for c (every op
    is longer): the table's overlap counts are not reproduced (its #Comm is). This records the
    figures the reading gives; it pins nothing of the paper."""
    P, M, f, c = 8, 8, 1000, 700
    ms, _, comm = chain(P, M, I.POLICY["1F1B"], 7 * f, 14 * f, c)
    assert comm[0].tolist() == [224, 98, 224 * c, 98 * c]
    v = 7
    S = P * v
    recs = I.pack_records(P, v, 0, [I.POLICY["I1F1B"]], [v], [np.arange(1, S)],
                          [I.placement("looped", P, v)])
    prob = R.problem(S, P, v, M, recs.shape[1], 0)
    costs = np.tile(np.array([[f, f, f]], np.int64), (S, 1))
    ms, _, comm = R.sim_batch_comm(prob, costs, I.link_matrix(P, c), recs)
    assert comm[0].tolist() == [1760, 1074, 1760 * c, 1074 * c]
