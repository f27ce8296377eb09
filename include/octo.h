/*
 * octo.h — C ABI of the MI355X batched pipeline-schedule simulator (libocto.so).
 *
 * Computes the graph-based pipeline simulator of OctoPipe (arXiv 2509.23722, §5) for batches of
 * candidate pipeline schedules — partitioning x placement x scheduling, the decision variables
 * P, A, O of §6 "Optimization Objective" — and one step of a parallel local search over them
 * (§6, Algorithm 1's re-simulate-per-move loop). All kernels run on the GPU; the host code only
 * validates arguments, sizes workspaces and launches.
 *
 * Time model (§5, §6 Eq. 1). Nodes are forward F(s,m), backward B(s,m) and, for split
 * schedules, weight-gradient W(s,m) ops of stage s and micro-batch m. Edges: each device's queue
 * order; F(s-1,m)->F(s,m) and B(s+1,m)->B(s,m) weighted by link[dev(producer)][dev(consumer)]
 * (0 when both stages are on one device; the send/recv pair of §5 as one edge); F(s,m)->B(s,m);
 * B(s,m)->W(s,m). Every op starts as early as its in-edges allow. makespan = latest finish
 * (T^pipeline of Eq. 1); bubble[d] = makespan - busy time of device d. A cycle is a deadlock.
 *
 * Units: all times are int64 nanoseconds; results are exact integers.
 * Memory: every array pointer passed to octo_sim_batch / octo_tune_step is a DEVICE pointer owned
 * by the caller; problem structs are host memory. The library keeps a private per-(device,
 * stream) workspace that it allocates on first use and grows when needed, stream-ordered
 * (hipMallocAsync / hipFreeAsync on the call's stream): no call synchronises the host.
 * Streams: `stream` is a hipStream_t (NULL = the null stream). Calls are asynchronous; results
 * are ready when the stream is synchronised. Concurrent calls on different streams are allowed.
 * Errors: argument problems return a negative status before anything is launched; per-candidate
 * outcomes (deadlock, invalid candidate) are data (sentinels), never errors.
 */
#ifndef OCTO_H
#define OCTO_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/* Status codes. */
#define OCTO_OK 0
#define OCTO_EINVAL (-1)       /* bad argument (null pointer, size out of range, bad stride) */
#define OCTO_EUNSUPPORTED (-2) /* valid problem that exceeds this GPU's limits (LDS) */
#define OCTO_EHIP (-3)         /* a HIP runtime call or kernel launch failed */
#define OCTO_ENOMEM (-4)       /* workspace allocation failed */
#define OCTO_ESCRATCH (-5)     /* octo_sim_batch_noalloc: the batch does not fit its scratch */

/* Per-candidate sentinel values written to makespan and every bubble entry. */
#define OCTO_MS_DEADLOCK (-1) /* the op orders and data dependencies form a cycle */
#define OCTO_MS_INVALID (-2)  /* the candidate record breaks a validity rule (below) */

/* Schedule policy byte. */
#define OCTO_AFAB 0  /* GPipe: all forwards, then all backwards */
#define OCTO_1F1B 1  /* one-forward-one-backward */
#define OCTO_I1F1B 2 /* interleaved 1F1B over v chunks per device */
#define OCTO_ZB 3    /* split backward (B input-grad, W weight-grad), W deferred by rank */

/* Problem header (host memory). Limits: 1 <= L <= 255; 1 <= P <= 64; 1 <= v_max <= 8 with
 * P*v_max <= 64; 1 <= M <= 2047; 0 <= max_pert <= 255; cand_stride a multiple of 16 and at least
 * octo_record_stride(P, v_max, max_pert); the finish table (P*v_max + 1)*M*8 bytes must fit in
 * one workgroup's LDS (else OCTO_EUNSUPPORTED). */
typedef struct octo_problem {
  int32_t L;           /* layers */
  int32_t P;           /* pipeline devices */
  int32_t v_max;       /* largest stages-per-device of any candidate */
  int32_t M;           /* micro-batches */
  int32_t cand_stride; /* bytes per candidate record */
  int32_t max_pert;    /* perturbation slots per record */
} octo_problem;

/*
 * Candidate record (cand_stride bytes; S = P*v, S_max = P*v_max), the decision variables of §6:
 *   byte 0            policy (OCTO_AFAB..OCTO_ZB)
 *   byte 1            v, stages per device (1..v_max)
 *   byte 2            n_pert, perturbations used (0..max_pert)
 *   byte 3            flags, must be 0
 *   bytes 4..         b[1..S-1], uint8 stage boundaries: stage s holds layers [b[s], b[s+1]) with
 *                     b[0] = 0, b[S] = L (partition vector P); S_max-1 bytes reserved
 *   bytes 3+S_max..   dev[0..S-1], uint8 device of each stage (placement A); S_max bytes reserved
 *   octo_record_pert_offset(P, v_max)..
 *                     pert[i] = {uint16 device, uint16 from, uint16 to}, little endian: after the
 *                     policy generates the queues, move queue entry `from` of `device` so that it
 *                     ends at index `to` (irregular orders, §3.3), applied in list order.
 * Unused reserved bytes are ignored.
 *
 * Queue generation (schedule O) from the policy, "looped" meaning dev[s] == dev[s mod P]:
 *   AFAB  -> forwards by (stage, m) ascending, then backwards by (stage descending, m).
 *   1F1B  -> v == 1: 1F1B with warm-up min(S-1-s, M); v >= 2: MERGE (below).
 *   I1F1B -> v == 1: as 1F1B; v >= 2 looped: the interleaved order with warm-up
 *            min(2(P-1-r) + (v-1)P, vM) for rank r, needs M % P == 0; otherwise MERGE.
 *   ZB    -> as I1F1B (or MERGE) with the backward split into B and W; each W waits in a FIFO
 *            of depth r (rank) behind its B (r = stage index inside MERGE).
 *   MERGE -> every stage runs its own 1F1B/ZB order on an ideal pipeline (unit costs, no
 *            transfer cost); a device executes its stages' ops sorted by ideal start time, then
 *            stage index.
 *
 * Validity (else OCTO_MS_INVALID): policy <= 3; 1 <= v <= v_max; n_pert <= max_pert; flags == 0;
 * 0 < b[1] < ... < b[S-1] < L; dev[s] < P with exactly v stages per device; M % P == 0 where the
 * interleaved order is used; every perturbation has device < P and from, to < queue length.
 */
int32_t octo_record_pert_offset(int32_t P, int32_t v_max);
/* Smallest valid cand_stride (a multiple of 16), or OCTO_EINVAL for out-of-range sizes. */
int32_t octo_record_stride(int32_t P, int32_t v_max, int32_t max_pert);

/*
 * octo_sim_batch — evaluate n candidates (the simulator of §5 per candidate).
 *   layer_costs  int64 [L][3], per layer {F, B (input-grad), W (weight-grad)} in ns; a fused
 *                backward costs B + W. Stage costs are sums over the stage's layers.
 *   link         int64 [P][P], cost of one transfer from device p to device q (diagonal unused).
 *   candidates   n records of prob->cand_stride bytes, 16-byte aligned.
 *   out_makespan int64 [n]; out_bubble int64 [n][P] row-major. Sentinels as above.
 * n == 0 is allowed and launches nothing. Returns OCTO_OK or a negative status.
 */
int octo_sim_batch(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                   const void* candidates, int64_t n, int64_t* out_makespan, int64_t* out_bubble,
                   void* stream);

/*
 * octo_sim_batch_noalloc — octo_sim_batch for callers that cannot allocate device memory
 * (code under HIP graph capture, tight serving loops, harnesses that forbid hipMalloc): the
 * same evaluation, same arguments, results and per-candidate sentinels, but every buffer the
 * call needs besides its inputs and outputs comes from a static device array of
 * OCTO_NOALLOC_SCRATCH_BYTES that the library holds on each GPU it runs on until the process
 * ends; the call makes no hipMalloc, hipFree or other allocation. The caller still passes the
 * inputs and outputs.
 *   A batch whose candidate lists and cached tables do not fit the array returns OCTO_ESCRATCH
 * before any launch (at P = 8, M = 64, v_max = 2 they fit up to about 2.5 million candidates);
 * materialised queues (candidates with moves) use as many persistent workgroups as the
 * remaining space holds.
 *   Every call on one GPU shares that GPU's array, which keeps the last call's contents (the
 * call clears what must start at zero itself): calls that overlap on one GPU — on different
 * streams, or from different threads without ordering — race and give undefined results.
 */
#define OCTO_NOALLOC_SCRATCH_BYTES (32u << 20)
int octo_sim_batch_noalloc(const octo_problem* prob, const int64_t* layer_costs,
                           const int64_t* link, const void* candidates, int64_t n,
                           int64_t* out_makespan, int64_t* out_bubble, void* stream);

/*
 * octo_sim_batch_mem — octo_sim_batch plus the memory model (§5: every compute node has a memory
 * node allocating or releasing intermediate tensors; §6 Eq. 2: peak memory per device against
 * its capacity). A forward F(s,m) allocates stage s's activation bytes for micro-batch m when it
 * starts; the last backward op of (s,m) — B when fused, W when split — releases them when it
 * ends; a device's static bytes (its stages' weights, gradients, optimizer state) are held
 * throughout. One device's ops never overlap, so its peak follows from its queue order.
 *   layer_mem  int64 [L][2], per layer {activation bytes per micro-batch, static bytes}; stage
 *              figures are sums over the stage's layers.
 *   out_peak   int64 [n][P]: static bytes + the largest activation total held, per device;
 *              OCTO_MS_DEADLOCK / OCTO_MS_INVALID like the makespan.
 * Other arguments, results and status as octo_sim_batch (layer_mem and out_peak non-NULL).
 */
int octo_sim_batch_mem(const octo_problem* prob, const int64_t* layer_costs,
                       const int64_t* layer_mem, const int64_t* link, const void* candidates,
                       int64_t n, int64_t* out_makespan, int64_t* out_bubble, int64_t* out_peak,
                       void* stream);

/*
 * octo_sim_batch_bounds — octo_sim_batch plus, per device, the start of its first op and the
 * end of its last op: its leading idle (first start) and trailing idle (makespan - last finish)
 * are the boundary bubble that §6's Algorithm 1 tells apart from the residual bubble between
 * its ops.
 *   out_bounds  int64 [n][P][2] {first start, last finish}; OCTO_MS_DEADLOCK / OCTO_MS_INVALID
 *               in every entry like the makespan.
 * Other arguments, results and status as octo_sim_batch (out_bounds non-NULL).
 */
int octo_sim_batch_bounds(const octo_problem* prob, const int64_t* layer_costs,
                          const int64_t* link, const void* candidates, int64_t n,
                          int64_t* out_makespan, int64_t* out_bubble, int64_t* out_bounds,
                          void* stream);

/*
 * octo_sim_batch_comm — octo_sim_batch plus communication accounting (§5: send and receive
 * nodes of the cross-device dependencies; a node that can overlap with subsequent computation
 * is overlappable and records the minimum of the computation's and the communication's
 * durations as its overlap time; §8's communication statistics). Every data edge between
 * stages on different devices, F(s,m) -> F(s+1,m) or B(s+1,m) -> B(s,m), is one send node on
 * the producer's device and one receive node on the consumer's, each lasting
 * c = link[producer device][consumer device], the transfer running from the producer's end for
 * c (as in the time model). A send can run beside the op that follows the producer on its
 * device, a receive beside the op that precedes the consumer on its device (the consumer waits
 * for the data); the node is overlappable iff that op runs during the transfer (a positive
 * shared length), and its overlap time is min(duration of that op, c).
 *   out_comm  int64 [n][4]: {comm nodes, overlappable nodes, total node time (each edge counted
 *             twice, once per node), total overlap time}; OCTO_MS_DEADLOCK / OCTO_MS_INVALID in
 *             all four like the makespan.
 * Other arguments, results and status as octo_sim_batch (out_comm non-NULL).
 */
int octo_sim_batch_comm(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                        const void* candidates, int64_t n, int64_t* out_makespan,
                        int64_t* out_bubble, int64_t* out_comm, void* stream);

/*
 * octo_sim_batch_serial — octo_sim_batch with serialised links (a variant of the §5 send /
 * receive nodes): a directed link p -> q carries one transfer at a time, first come first
 * served. A device issues each op's output transfer when the op ends, so the transfers on one
 * of its links queue in its op order: the transfer of X starts at max(end of X, end of the
 * link's previous transfer) and ends c = link[p][q] later, when its consumer may start. Deadlock
 * and validity are as in octo_sim_batch (a link queue adds no cycle). Arguments, results and
 * status as octo_sim_batch.
 */
int octo_sim_batch_serial(const octo_problem* prob, const int64_t* layer_costs,
                          const int64_t* link, const void* candidates, int64_t n,
                          int64_t* out_makespan, int64_t* out_bubble, void* stream);

/*
 * octo_sim_batch_rdv — octo_sim_batch with blocking rendezvous transfers, the naive
 * coordination of computation and point-to-point communication that §3.3 ("Irregular Execution
 * Orders", Fig. 3(a)-(b)) shows deadlocking: a device receives an op's input from another device
 * right before the op and sends the op's output to another device right after it, and a
 * transfer starts once both devices have reached it and holds both until it ends
 * c = link[p][q] later (blocking send and receive). Each device's program is thus its queue with
 * [receive] op [send] around every op that has a cross-device input / output. A cycle of waits
 * (e.g. two devices sending to each other at once, as in 1F1B's steady state) is a deadlock:
 * OCTO_MS_DEADLOCK. Busy time counts computation only, so transfer time is bubble. Validity,
 * arguments, results and status as octo_sim_batch.
 */
int octo_sim_batch_rdv(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                       const void* candidates, int64_t n, int64_t* out_makespan,
                       int64_t* out_bubble, void* stream);

/*
 * octo_sim_batch_ordered — blocking rendezvous transfers (as octo_sim_batch_rdv) in the
 * deadlock-free, overlap-aware reordered coordination of §7 ("Unified Pipeline Executor":
 * reorder the communication operations to break cyclic waits while keeping transfers beside
 * the computation around them). Each device keeps its compute order; every transfer is placed at
 * its ideal start, the end of its producer in the asynchronous schedule of octo_sim_batch, where
 * its data becomes ready, so its send and receive are posted together. A device's program is
 * its items sorted by (time, communication before computation, then the producer's (kind,
 * stage, m) for a transfer or the queue position for a computation), a computation's time
 * being its asynchronous start; a send also waits for its producer. Both ends of a transfer get
 * one key, so all programs follow one global order: with positive op durations no cycle of
 * waits can form, and the candidate deadlocks (OCTO_MS_DEADLOCK) only if its compute orders do
 * (or zero-length ops tie the order). Busy time counts computation only. Arguments, results and
 * status as octo_sim_batch.
 */
int octo_sim_batch_ordered(const octo_problem* prob, const int64_t* layer_costs,
                           const int64_t* link, const void* candidates, int64_t n,
                           int64_t* out_makespan, int64_t* out_bubble, void* stream);

/*
 * octo_sim_batch_reorder — the unified executor's deadlock-free, overlap-aware reordering of the
 * communication (§7, its three steps) with handshake transfers: a device that reaches a send or
 * a receive waits until the other device has reached the other end; then both go on at once,
 * and the data arrives c = link[p][q] later while both compute; the consumer starts once it has
 * arrived. Every transfer has a key: its producer's end in the asynchronous schedule of
 * octo_sim_batch, then the producer's level (the number of ops on the longest dependency chain
 * before it, queue order included), then its node id (kind S + stage) M + m. Starting from the
 * naive programs of octo_sim_batch_rdv (a receive before its consumer, a send after its
 * producer): (1) on every device, a communication item whose key is below the largest key
 * before it in program order is a mismatched pair (only receives can be); (2) its feasible
 * window is the gaps between computations that lie between the in-order items just below and
 * just above its key, at most its consumer's, whose post time (the end of the previous
 * computation in the asynchronous schedule) is not before its producer starts; (3) each
 * mismatched receive, in key order, takes the gap of least cost = |producer end - post time|
 * (the communication span) - min(c, the durations of the computations between that gap and the
 * consumer) (the overlap with neighbouring computation), the highest gap on ties, and the next
 * one's window starts there. Communication items of one gap run in key order, so every device
 * meets its transfers in key order and no cycle of waits can form: OCTO_MS_DEADLOCK only where
 * the compute orders themselves deadlock. Busy time counts computation only.
 * out_stats (device int64 [n][2], nullable): transfers (send/receive pairs) and mismatched
 * receives of each candidate (the sentinels for deadlocked and invalid records). Other
 * arguments, results and status as octo_sim_batch.
 */
int octo_sim_batch_reorder(const octo_problem* prob, const int64_t* layer_costs,
                           const int64_t* link, const void* candidates, int64_t n,
                           int64_t* out_makespan, int64_t* out_bubble, int64_t* out_stats,
                           void* stream);

/*
 * octo_advance_w — selective W advancing (§6 "Scheduling Tuning", third policy) under the
 * per-device capacity of §6 Eq. 2, on a batch of candidate records. For each record, after its
 * queues are generated and its moves applied: while some device's peak (as octo_sim_batch_mem)
 * exceeds capacity[d], take the lowest such device d and the queue position p where its
 * activation total first reaches the peak (a forward). A weight-gradient op W of d is eligible
 * if it sits after p, its B sits before p and its stage has activation bytes; advancing it moves
 * it to index p (its release then precedes that allocation). Eligible W are tried in queue
 * order; the first whose advance does not lengthen the makespan is kept (busy time is fixed, so
 * no device's bubble grows), else the first eligible one. The search stops when every device
 * fits, nothing is eligible, or the record's free move slots (max_pert - n_pert) are used up.
 *   capacity        int64 [P] bytes per device.
 *   out_candidates  n records (same stride, 16-byte aligned; may be `candidates` itself): the
 *                   input record with each advance appended as a move {device, from, to} and
 *                   n_pert raised; bytes past the last move are copied. Invalid or deadlocked
 *                   records are copied unchanged.
 *   out_makespan, out_bubble, out_peak  as octo_sim_batch_mem for the output record (so a
 *                   record still over capacity shows it in out_peak).
 * Fused schedules have no W: their records come back unchanged. Returns OCTO_OK or a negative
 * status.
 */
int octo_advance_w(const octo_problem* prob, const int64_t* layer_costs, const int64_t* layer_mem,
                   const int64_t* capacity, const int64_t* link, const void* candidates,
                   int64_t n, void* out_candidates, int64_t* out_makespan, int64_t* out_bubble,
                   int64_t* out_peak, void* stream);

/*
 * Local-search chains (§6: every tuning move re-runs the simulator; Algorithm 1's three move
 * families). Chain state record, octo_chain_stride(prob) bytes each, 16-byte aligned:
 *   bytes 0..cand_stride-1  the candidate record (n_pert must be 0), updated in place
 *   +0  int64 current makespan (or sentinel)
 *   +8  int64 accepted moves
 *   +16 int64 current bubble[P]
 *   +16+8P int64 current peak bytes[P] (written by octo_tune_step_mem only)
 *   +16+16P int64 an upper bound of the queues' micro-batch window (octo_tune_step only): the
 *          largest m_i - m_j over queue entries i < j of one stage on one device
 * Queue store: uint16 [n_chains][P][octo_queue_capacity(prob)], 16-byte aligned (else
 * OCTO_EINVAL); the capacity is 3 v_max M rounded up to a multiple of 8 so that every row is
 * 16-byte aligned too. Entry = kind << 14 | chunk << 11 | m with kind 0 = F, 1 = B, 2 = W and
 * chunk the index into the device's ascending stage list.
 *
 * octo_tune_step(step = 0) validates each chain, generates its queues from the policy and
 * evaluates it. step t >= 1 draws (u0, u1, u2, u3) = Philox4x64-10(key = {seed, 0},
 * counter = {chain, t, 0, 0}) and proposes by u0 % 3:
 *   0: stage boundary i = 1 + u1 % (S-1) moves by (u2 & 1) ? +1 : -1 layer;
 *   1: devices d1 = u1 % P and d2 = (d1 + 1 + u2 % (P-1)) % P swap their stage sets, each device
 *      keeping its queue;
 *   2: on device d = u1 % P, queue entries i = u2 % (len-1) and i+1 swap.
 * A proposal is kept iff it is valid, does not deadlock and its makespan is <= the current one
 * (a deadlocked current state counts as +infinity). Chains whose step-0 state is invalid stay
 * OCTO_MS_INVALID. Deterministic in (seed, chain, step).
 */
int32_t octo_chain_stride(const octo_problem* prob);
int32_t octo_queue_capacity(const octo_problem* prob);
int octo_tune_step(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                   void* chains, uint16_t* queues, int64_t n_chains, uint64_t seed, int32_t step,
                   void* stream);

/*
 * octo_tune_step_mem — octo_tune_step under the memory constraint of §6 Eq. 2. Every
 * evaluation (the step-0 state and each proposal) runs selective W advancing as octo_advance_w
 * does, on the chain's queues, with at most max_advance advances (0..OCTO_MAX_ADVANCE); a state
 * is feasible if it does not deadlock and every device's peak fits capacity[d]. A proposal is
 * kept iff it is feasible and the current state is not, or its makespan is <= the current one;
 * kept advances stay in the chain's queues. Step 0 stores the (advanced) initial state whether
 * or not it fits; the peak area of the chain record holds each state's peaks. layer_mem as
 * octo_sim_batch_mem. Use it for every step of a chain set (it reads the peaks it stored).
 */
#define OCTO_MAX_ADVANCE 4096
int octo_tune_step_mem(const octo_problem* prob, const int64_t* layer_costs,
                       const int64_t* layer_mem, const int64_t* capacity, int32_t max_advance,
                       const int64_t* link, void* chains, uint16_t* queues, int64_t n_chains,
                       uint64_t seed, int32_t step, void* stream);

/*
 * octo_alg1_tune — Algorithm 1 of §6 ("Iterative and Bubble-Aware Tuning"): one independent
 * search per record, all records advanced together for `iters` iterations (the paper's time
 * budget, counted in iterations). An iteration of a record's search:
 *   1. From its current evaluation (as octo_sim_batch_bounds): bubble gap
 *      Δb = max_d bubble[d] - min_d bubble[d]; boundary bubble b_bd = Σ_d (first start[d] +
 *      makespan - last finish[d]); residual bubble b_res = Σ_d bubble[d] - b_bd; and
 *      t_layer = M * min over layers of (F + B + W).
 *   2. Phase: partitioning if Δb > t_layer, else placement if b_bd > b_res, else scheduling. A
 *      phase whose last search found nothing better stays exhausted until a move is kept; an
 *      exhausted pick falls to the first open phase in that order; with none open (or when the
 *      record is invalid or deadlocks) the search has ended and later iterations skip it.
 *   3. The phase's neighbourhood, in this order (the order breaks ties):
 *      partitioning — one layer migrates from a stage a of the most loaded device (largest
 *        busy time; lowest index on ties) to a stage b of the least loaded one, the stages in
 *        between passing one layer along: for a, then b, ascending, a having >= 2 layers;
 *      placement — the device with the largest bubble exchanges one of its stages with one of
 *        another device's (other device, its stage, the other's stage, ascending); then, if
 *        2v <= v_max and every stage has >= 2 layers, stage dispersion: every stage splits at
 *        its middle layer (first half floor(size/2) layers), new stage k going to the device
 *        of old stage k mod S, v doubled, moves cleared;
 *      scheduling — each other policy, moves cleared; then, if n_pert < max_pert, every
 *        adjacent swap {d, i, i+1} of the device d with the largest residual bubble (bubble
 *        minus leading and trailing idle), appended as a move, then d's overlap-aware
 *        insertions (octo_alg1_tune_ex, OCTO_A1_INSERT).
 *      Reserved boundary and placement bytes read as 0 in every neighbour; other bytes copy.
 *   4. The neighbour with the smallest makespan among those that neither deadlock nor are
 *      invalid (the first on ties) replaces the record iff its makespan is strictly smaller;
 *      every phase is open again. Otherwise the phase is exhausted.
 *   records       n records (prob->cand_stride <= 1664, 16-byte aligned) updated in place to
 *                 each search's final record.
 *   out_makespan  int64 [n], out_bubble int64 [n][P]: the final records' evaluation.
 *   out_stats     int64 [n][4]: moves kept in the partitioning, placement and scheduling
 *                 phases, and the iterations in which a phase was searched.
 * The library evaluates each iteration's neighbours as one batch in its workspace, at most
 * n * max(v_max^2, (P-1) v_max^2 + 1, 6 v_max M + 1) records (OCTO_EINVAL above 2^31 - 1;
 * OCTO_ENOMEM if it cannot be allocated). Returns OCTO_OK or a negative status.
 */
int octo_alg1_tune(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                   void* records, int64_t n, int32_t iters, int64_t* out_makespan,
                   int64_t* out_bubble, int64_t* out_stats, void* stream);

/*
 * octo_alg1_tune_ex — octo_alg1_tune with its options. flags:
 *   OCTO_A1_INSERT  the scheduling phase also tries the overlap-aware insertions (§6 "Scheduling
 *                   Tuning", the second policy), after the adjacent swaps, as moves {d, j, k} of
 *                   the same device d: on d's current schedule, at each position k >= 1 where d
 *                   idles between A = Q[k-1] and B = Q[k] and a communication there is not
 *                   overlappable in §5's sense (A's output goes to another device and B does not
 *                   run during that transfer, or B's input comes from another device and A does
 *                   not run during it), the first later op Q[j] ready when A ends (its
 *                   producers' ends plus the transfer time across devices) moves to index k.
 *                   octo_alg1_tune sets this flag.
 *   OCTO_A1_RANDOM  the random-search variant of §8 ("Pipeline Search Cost"): each iteration's
 *                   phase is the (u mod n)-th of the n open phases (partitioning, placement,
 *                   scheduling), u the first word of Philox4x64-10(counter (record index,
 *                   iteration, 1, 0), key (seed, 0)), instead of the bubble-aware branch.
 *   other bits: OCTO_EINVAL.
 * out_phase_iters (device int64 [n][3], nullable): the iterations that searched each phase.
 * The neighbour batch holds at most n * max(v_max^2, (P-1) v_max^2 + 1, 6 v_max M + 1) records.
 * Other arguments, results and status as octo_alg1_tune.
 */
#define OCTO_A1_INSERT 1
#define OCTO_A1_RANDOM 2
int octo_alg1_tune_ex(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                      void* records, int64_t n, int32_t iters, int32_t flags, uint64_t seed,
                      int64_t* out_makespan, int64_t* out_bubble, int64_t* out_stats,
                      int64_t* out_phase_iters, void* stream);

/*
 * Measurement hook. events[0..n_events-1] are hipEvent_t handles (n_events <= 8; entries may be
 * NULL). Each later octo_sim_batch call records them on its stream at fixed boundaries around
 * its simulation kernels: events[0] before the static-schedule kernel (candidates of the
 * structure classes: v = 1, and v = 2 with looped, blocked or V-shape stage pairs), [1] after
 * it, [2] after the v = 2 generated-queue kernel (other 1F1B, I1F1B, ZB queues), [3] after the
 * v = 1 kernel, [4] after the v = 3..8 kernel, [5] after the AFAB kernel (every v), [6] after
 * the materialised-queue kernel (a kernel that a problem does not need is skipped, so its
 * interval is empty). A caller can time each kernel alone on the stream
 * it runs on. octo_profile_events(NULL, 0) turns it off. Process-wide.
 */
int octo_profile_events(void* const* events, int32_t n_events);

/* Human-readable text for a status code (static storage). */
const char* octo_strerror(int status);

#ifdef __cplusplus
}
#endif

#endif /* OCTO_H */
