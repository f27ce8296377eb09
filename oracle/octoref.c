/*
 * octoref.c — the CPU oracle for batched pipeline-schedule simulation.
 *
 * TEST INFRASTRUCTURE ONLY. This file is the plain, slow, obviously-correct reference that the
 * HIP path is checked against. Only tests, the smoke check and the benchmark's CPU-baseline leg
 * may load it. It shares no code, header or table with the HIP library; the two read the same
 * candidate-record byte format, each with its own decoder.
 *
 * What it computes (arXiv 2509.23722, "OctoPipe"):
 *   - §5 "Simulating Pipeline Execution": a candidate pipeline schedule becomes a DAG whose nodes
 *     are per-(stage, micro-batch) forward/backward ops and whose edges are data dependencies;
 *     the send/recv pair of a cross-device dependency is one weighted edge here.
 *   - §5 "Estimating Pipeline Performance": traverse the DAG recording start/end of each node;
 *     idle time on a device is bubble.
 *   - §6 "Optimization Objective", Eq. (1): T^pipeline = max over devices of T_d^execution.
 *   - §3.3: the backward of a micro-batch must follow its forward; orders can deadlock.
 *   - §6 "Scheduling Tuning": F of stage i depends on stage i-1, B of stage i on stage i+1, W only
 *     on B of the same device.
 * The traversal is Kahn's topological order with longest-path relaxation: the plain definition
 * of earliest start times. A cycle (ops left unvisited) is a deadlock.
 *
 * Parity pins (tests/test_oracle_*.py): closed forms for AFAB/1F1B/interleaved/ZB, the §3.2
 * Fig. 3 worked example, the §3.3 order count, the §8 comm-count table, invariants, a pure-Python
 * tick simulator and DFS cycle check on tiny instances, and numpy's Philox.
 */
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define REF_OK 0
#define REF_EINVAL (-1)
#define REF_DEADLOCK (-1) /* per-candidate sentinel */
#define REF_INVALID (-2)  /* per-candidate sentinel */
/* internal status of one DAG evaluation */
#define SIM_OK 0
#define SIM_CYCLE 1
#define SIM_BADQ 2

enum { KF = 0, KB = 1, KW = 2 };
enum { POL_AFAB = 0, POL_1F1B = 1, POL_I1F1B = 2, POL_ZB = 3 };
enum { GEN_AFAB = 0, GEN_INTER = 1, GEN_MERGE = 2 };

/* Problem description (scalars only; mirrors the ABI's problem header, decoded independently). */
typedef struct {
  int32_t L, P, v_max, M, cand_stride, max_pert;
} ref_problem;

/* One op in device-local terms: kind, local chunk (index into A_d), micro-batch. */
typedef struct {
  int kind, chunk, m;
} ref_op;

/* A decoded candidate. */
typedef struct {
  int policy, v, n_pert, flags, S;
  int b[66];   /* b[0..S] */
  int dev[64]; /* dev[0..S-1] */
  int pert[256][3];
} ref_cand;

static int imin(int a, int b) { return a < b ? a : b; }
static int imax(int a, int b) { return a > b ? a : b; }

/* ------------------------------------------------------------------------------------------ */
/* Candidate record decoding (byte layout of the ABI, read independently).                    */
/* ------------------------------------------------------------------------------------------ */

static int pert_offset(int S_max) { return (3 + 2 * S_max + 1) & ~1; }

static int rd16(const uint8_t* p) { return (int)p[0] | ((int)p[1] << 8); }

/* Decode without judging validity beyond what decoding itself needs. */
static void decode(const ref_problem* pr, const uint8_t* rec, ref_cand* c) {
  int S_max = pr->P * pr->v_max;
  c->policy = rec[0];
  c->v = rec[1];
  c->n_pert = rec[2];
  c->flags = rec[3];
  c->S = pr->P * c->v;
  if (c->v < 1 || c->v > pr->v_max) c->S = 0;
  c->b[0] = 0;
  for (int s = 1; s < c->S; ++s) c->b[s] = rec[4 + s - 1];
  if (c->S > 0) c->b[c->S] = pr->L;
  for (int s = 0; s < c->S; ++s) c->dev[s] = rec[3 + S_max + s];
  int po = pert_offset(S_max);
  int np = imin(c->n_pert, pr->max_pert);
  for (int i = 0; i < np && i < 256; ++i)
    for (int f = 0; f < 3; ++f) c->pert[i][f] = rd16(rec + po + 6 * i + 2 * f);
}

/* A_d: the stages of device d in ascending order. Returns |A_d|. */
static int stages_of(const ref_cand* c, int d, int* out) {
  int n = 0;
  for (int s = 0; s < c->S; ++s)
    if (c->dev[s] == d) out[n++] = s;
  return n;
}

/* Looped placement: dev[s] == dev[s mod P] for every stage. */
static int is_looped(const ref_cand* c, int P) {
  for (int s = 0; s < c->S; ++s)
    if (c->dev[s] != c->dev[s % P]) return 0;
  return 1;
}

/* Policy resolution (policy x v x placement). Returns -1 if the candidate cannot be resolved. */
static int resolve(const ref_problem* pr, const ref_cand* c, int* split) {
  *split = (c->policy == POL_ZB);
  if (c->policy == POL_AFAB) return GEN_AFAB;
  if (c->v == 1) return GEN_INTER;
  if (c->policy == POL_1F1B) return GEN_MERGE;
  if (!is_looped(c, pr->P)) return GEN_MERGE;
  if (pr->M % pr->P != 0) return -1;
  return GEN_INTER;
}

/* Structural validity, excluding perturbation ranges (checked once queues exist). */
static int valid_structure(const ref_problem* pr, const ref_cand* c) {
  if (c->policy > 3) return 0;
  if (c->v < 1 || c->v > pr->v_max) return 0;
  if (c->n_pert > pr->max_pert) return 0;
  if (c->flags != 0) return 0;
  for (int s = 0; s < c->S; ++s)
    if (c->b[s + 1] <= c->b[s]) return 0; /* covers 0 < b[1] < ... < b[S-1] < L */
  int cnt[64] = {0};
  for (int s = 0; s < c->S; ++s) {
    if (c->dev[s] >= pr->P) return 0;
    cnt[c->dev[s]]++;
  }
  for (int d = 0; d < pr->P; ++d)
    if (cnt[d] != c->v) return 0;
  int split;
  if (resolve(pr, c, &split) < 0) return 0;
  return 1;
}

/* ------------------------------------------------------------------------------------------ */
/* Queue generators.                                                                          */
/* ------------------------------------------------------------------------------------------ */

/* GPipe / all-forward-all-backward order. */
static int gen_afab(int v, int M, ref_op* q) {
  int n = 0;
  for (int k = 0; k < v; ++k)
    for (int m = 0; m < M; ++m) q[n++] = (ref_op){KF, k, m};
  for (int k = v - 1; k >= 0; --k)
    for (int m = 0; m < M; ++m) q[n++] = (ref_op){KB, k, m};
  return n;
}

/* Interleaved 1F1B virtual index j -> (chunk, micro-batch) (Narayanan et al., restated). */
static ref_op inter_fwd(int P, int v, int j) {
  ref_op o;
  o.kind = KF;
  o.chunk = (j % (P * v)) / P;
  o.m = (j / (P * v)) * P + (j % P);
  return o;
}
static ref_op inter_bwd(int P, int v, int i, int kind) {
  ref_op o = inter_fwd(P, v, i);
  o.kind = kind;
  o.chunk = v - 1 - o.chunk;
  return o;
}

/* INTER(P, v, M, r, split, lag). */
static int gen_inter(int P, int v, int M, int r, int split, int lag, ref_op* q) {
  int N = v * M;
  int w = (v == 1) ? imin(P - 1 - r, M) : imin(2 * (P - 1 - r) + (v - 1) * P, N);
  int n = 0;
  for (int j = 0; j < w; ++j) q[n++] = inter_fwd(P, v, j);
  for (int i = 0; i < N - w; ++i) {
    q[n++] = inter_fwd(P, v, w + i);
    q[n++] = inter_bwd(P, v, i, KB);
    if (split && i >= lag) q[n++] = inter_bwd(P, v, i - lag, KW);
  }
  for (int i = N - w; i < N; ++i) {
    q[n++] = inter_bwd(P, v, i, KB);
    if (split && i >= lag) q[n++] = inter_bwd(P, v, i - lag, KW);
  }
  if (split)
    for (int i = imax(0, N - lag); i < N; ++i) q[n++] = inter_bwd(P, v, i, KW);
  return n;
}

/* ------------------------------------------------------------------------------------------ */
/* The DAG and its traversal (the plain definition of the time model).                        */
/* ------------------------------------------------------------------------------------------ */

/* Ops in stage terms for the DAG: kind, stage, micro-batch. */
typedef struct {
  int kind, s, m;
} ref_sop;

typedef struct {
  int S, M, split, P;
  const int* dev;   /* [S] */
  const int64_t* F; /* [S] stage forward */
  const int64_t* B; /* [S] stage input-grad backward */
  const int64_t* W; /* [S] stage weight-grad backward */
  const int64_t* link; /* [P*P] */
  int serial;          /* transfers on one directed link run one at a time, in issue order */
} ref_dag_in;

static int node_id(int S, int M, int kind, int s, int m) { return (kind * S + s) * M + m; }

static int64_t op_dur(const ref_dag_in* g, int kind, int s) {
  if (kind == KF) return g->F[s];
  if (kind == KB) return g->split ? g->B[s] : g->B[s] + g->W[s];
  return g->W[s];
}

static int64_t edge_w(const ref_dag_in* g, int sp, int sc) {
  int dp = g->dev[sp], dc = g->dev[sc];
  return dp == dc ? 0 : g->link[dp * g->P + dc];
}

/*
 * Link serialisation (a variant of the §5 communication nodes): a directed link p -> q carries
 * one transfer at a time, first come first served. A device issues its sends as its ops end, so
 * its transfers on a link queue in its op order: the transfer of X starts at max(end of X, end of
 * the link's previous transfer) and arrives c = link[p][q] later; its consumer may start then.
 * Kahn's order below finishes a device's ops in queue order, so the link's FIFO is kept by
 * updating its free time as each producer is finished.
 *
 * Evaluate explicit device queues. qlen[d] ops of device d start at queue + qoff[d].
 * Outputs makespan, bubble[P]; start_out (optional) receives start times indexed by node id;
 * n_cross (optional) receives the number of cross-device data edges.
 * Returns SIM_OK, SIM_CYCLE on a cycle (deadlock), or SIM_BADQ if the queues are not exactly the
 * op set (each op once, on the device hosting its stage).
 */
static int simulate(const ref_dag_in* g, const ref_sop* queue, const int* qoff, const int* qlen,
                    int64_t* makespan, int64_t* bubble, int64_t* start_out, int64_t* n_cross) {
  int S = g->S, M = g->M, nk = g->split ? 3 : 2;
  int nn = nk * S * M;
  int* owner = (int*)malloc(sizeof(int) * nn);
  int* next = (int*)malloc(sizeof(int) * nn); /* queue successor or -1 */
  int* indeg = (int*)calloc(nn, sizeof(int));
  int64_t* est = (int64_t*)calloc(nn, sizeof(int64_t));
  int64_t* fin = (int64_t*)malloc(sizeof(int64_t) * nn);
  int* ready = (int*)malloc(sizeof(int) * nn);
  int64_t* lfree = g->serial ? (int64_t*)calloc((size_t)g->P * g->P, sizeof(int64_t)) : NULL;
  int rc = 0;
  for (int i = 0; i < nn; ++i) owner[i] = -1, next[i] = -1;
  /* queue edges */
  for (int d = 0; d < g->P; ++d) {
    for (int i = 0; i < qlen[d]; ++i) {
      ref_sop o = queue[qoff[d] + i];
      if (o.kind < 0 || o.kind >= nk || o.s < 0 || o.s >= S || o.m < 0 || o.m >= M ||
          g->dev[o.s] != d) {
        rc = SIM_BADQ;
        goto done;
      }
      int id = node_id(S, M, o.kind, o.s, o.m);
      if (owner[id] >= 0) {
        rc = SIM_BADQ;
        goto done;
      }
      owner[id] = d;
      if (i + 1 < qlen[d]) {
        ref_sop n2 = queue[qoff[d] + i + 1];
        if (n2.kind < 0 || n2.kind >= nk || n2.s < 0 || n2.s >= S || n2.m < 0 || n2.m >= M) {
          rc = SIM_BADQ;
          goto done;
        }
        next[id] = node_id(S, M, n2.kind, n2.s, n2.m);
      }
    }
  }
  for (int i = 0; i < nn; ++i)
    if (owner[i] < 0) {
      rc = SIM_BADQ;
      goto done;
    }
  /* in-degrees: queue edges + data edges */
  int64_t cross = 0;
  for (int i = 0; i < nn; ++i)
    if (next[i] >= 0) indeg[next[i]]++;
  for (int s = 0; s < S; ++s)
    for (int m = 0; m < M; ++m) {
      if (s > 0) {
        indeg[node_id(S, M, KF, s, m)]++; /* F(s-1,m) -> F(s,m) */
        if (g->dev[s - 1] != g->dev[s]) cross++;
      }
      if (s < S - 1) {
        indeg[node_id(S, M, KB, s, m)]++; /* B(s+1,m) -> B(s,m) */
        if (g->dev[s + 1] != g->dev[s]) cross++;
      }
      indeg[node_id(S, M, KB, s, m)]++; /* F(s,m) -> B(s,m) */
      if (g->split) indeg[node_id(S, M, KW, s, m)]++; /* B(s,m) -> W(s,m) */
    }
  if (n_cross) *n_cross = cross;
  /* Kahn traversal with longest-path relaxation */
  int nr = 0, head = 0, done_n = 0;
  for (int i = 0; i < nn; ++i)
    if (indeg[i] == 0) ready[nr++] = i;
  while (head < nr) {
    int u = ready[head++];
    int kind = u / (S * M), s = (u / M) % S, m = u % M;
    fin[u] = est[u] + op_dur(g, kind, s);
    done_n++;
    /* out-edges of u */
    int outs[4];
    int64_t ws[4];
    int no = 0;
    if (next[u] >= 0) outs[no] = next[u], ws[no++] = 0;
    if (kind == KF) {
      if (s + 1 < S) outs[no] = node_id(S, M, KF, s + 1, m), ws[no++] = edge_w(g, s, s + 1);
      outs[no] = node_id(S, M, KB, s, m), ws[no++] = 0;
    } else if (kind == KB) {
      if (s > 0) outs[no] = node_id(S, M, KB, s - 1, m), ws[no++] = edge_w(g, s, s - 1);
      if (g->split) outs[no] = node_id(S, M, KW, s, m), ws[no++] = 0;
    }
    for (int e = 0; e < no; ++e) {
      int x = outs[e];
      int64_t t = fin[u] + ws[e];
      const int sx = (x / M) % S;
      if (lfree && sx != s && g->dev[sx] != g->dev[s]) {
        /* the transfer waits for the link to be free */
        int64_t* lf = &lfree[g->dev[s] * g->P + g->dev[sx]];
        const int64_t go = fin[u] > *lf ? fin[u] : *lf;
        t = go + ws[e];
        *lf = t;
      }
      if (t > est[x]) est[x] = t;
      if (--indeg[x] == 0) ready[nr++] = x;
    }
  }
  if (done_n < nn) {
    rc = SIM_CYCLE;
    goto done;
  }
  int64_t ms = 0;
  for (int i = 0; i < nn; ++i)
    if (fin[i] > ms) ms = fin[i];
  *makespan = ms;
  for (int d = 0; d < g->P; ++d) {
    int64_t busy = 0;
    for (int i = 0; i < qlen[d]; ++i) {
      ref_sop o = queue[qoff[d] + i];
      busy += op_dur(g, o.kind, o.s);
    }
    bubble[d] = ms - busy;
  }
  if (start_out)
    for (int i = 0; i < nn; ++i) start_out[i] = est[i];
done:
  free(owner);
  free(next);
  free(indeg);
  free(est);
  free(fin);
  free(ready);
  free(lfree);
  return rc;
}

/*
 * Device programs with blocking rendezvous transfers. A program is a device's sequence of
 * items: computing an op, sending an op's output to another device, or receiving an op's input
 * from another device. A transfer (producer X on device p -> consumer Y on device q) is ONE node
 * of duration c = link[p][q] that sits in both p's program (as the send) and q's (as the
 * receive): it starts once both devices have reached it and holds both until it ends (blocking
 * point-to-point send and receive). Item codes: (kind << 28) | node, kind 0 compute (node = the
 * op's node id), 1 send, 2 receive (node = the PRODUCER's node id).
 */
#define PI_COMP 0
#define PI_SEND 1
#define PI_RECV 2

/* The consumer of X's output on another device, or -1. */
static int cross_consumer(const ref_dag_in* g, int kind, int s, int m) {
  const int S = g->S, M = g->M;
  if (kind == KF && s + 1 < S && g->dev[s + 1] != g->dev[s]) return node_id(S, M, KF, s + 1, m);
  if (kind == KB && s > 0 && g->dev[s - 1] != g->dev[s]) return node_id(S, M, KB, s - 1, m);
  return -1;
}

/* The producer of Y's input on another device, or -1. */
static int cross_producer(const ref_dag_in* g, int kind, int s, int m) {
  const int S = g->S, M = g->M;
  if (kind == KF && s > 0 && g->dev[s - 1] != g->dev[s]) return node_id(S, M, KF, s - 1, m);
  if (kind == KB && s + 1 < S && g->dev[s + 1] != g->dev[s]) return node_id(S, M, KB, s + 1, m);
  return -1;
}

/* The naive coordination of §3.3 ("Irregular Execution Orders"): receive an op's cross-device
 * input right before it, send its cross-device output right after it. prog gets at most 3 qlen[d]
 * items per device at poff[d] = 3 qoff[d]; plen[d] their number. */
static void naive_programs(const ref_dag_in* g, const ref_sop* queue, const int* qoff,
                           const int* qlen, int* prog, int* plen) {
  for (int d = 0; d < g->P; ++d) {
    int n = 0, *out = prog + 3 * qoff[d];
    for (int i = 0; i < qlen[d]; ++i) {
      const ref_sop o = queue[qoff[d] + i];
      const int x = cross_producer(g, o.kind, o.s, o.m);
      if (x >= 0) out[n++] = (PI_RECV << 28) | x;
      const int y = node_id(g->S, g->M, o.kind, o.s, o.m);
      out[n++] = (PI_COMP << 28) | y;
      if (cross_consumer(g, o.kind, o.s, o.m) >= 0) out[n++] = (PI_SEND << 28) | y;
    }
    plen[d] = n;
  }
}

/*
 * Deadlock-free, overlap-aware reordering of the communication (§7, "Unified Pipeline Executor"):
 * each device keeps its compute order, and every transfer is placed at its ideal start — the end
 * of its producer in the asynchronous schedule (start[] of the plain model), the moment its data
 * is ready. A device's items are sorted by one global key: (time, communication before
 * computation, node id), the time of a compute item being its start and of a transfer its
 * producer's end. The two ends of a transfer get the same key on both devices, so they are
 * posted together (the smallest communication span the schedule allows) and every program
 * follows one global order: with positive durations every dependency strictly increases the
 * key, so no cycle of waits can form.
 */
typedef struct {
  int64_t t;
  int cls, node, code;
} prog_key;

static int cmp_prog_key(const void* a, const void* b) {
  const prog_key *x = (const prog_key*)a, *y = (const prog_key*)b;
  if (x->t != y->t) return x->t < y->t ? -1 : 1;
  if (x->cls != y->cls) return x->cls < y->cls ? -1 : 1;
  return x->node < y->node ? -1 : x->node > y->node;
}

static void ordered_programs(const ref_dag_in* g, const ref_sop* queue, const int* qoff,
                             const int* qlen, const int64_t* start, int* prog, int* plen) {
  const int S = g->S, M = g->M;
  int total = 0;
  for (int d = 0; d < g->P; ++d) total += qlen[d];
  prog_key* keys = (prog_key*)malloc(sizeof(prog_key) * (size_t)(3 * total + 1));
  for (int d = 0; d < g->P; ++d) {
    int n = 0;
    for (int i = 0; i < qlen[d]; ++i) {
      const ref_sop o = queue[qoff[d] + i];
      const int y = node_id(S, M, o.kind, o.s, o.m);
      keys[n++] = (prog_key){start[y], 1, i, (PI_COMP << 28) | y}; /* ties: queue order */
      const int x = cross_producer(g, o.kind, o.s, o.m);
      if (x >= 0) {
        const int xk = x / (S * M), xs = (x / M) % S;
        keys[n++] = (prog_key){start[x] + op_dur(g, xk, xs), 0, x, (PI_RECV << 28) | x};
      }
      if (cross_consumer(g, o.kind, o.s, o.m) >= 0)
        keys[n++] = (prog_key){start[y] + op_dur(g, o.kind, o.s), 0, y, (PI_SEND << 28) | y};
    }
    qsort(keys, (size_t)n, sizeof(prog_key), cmp_prog_key);
    for (int i = 0; i < n; ++i) prog[3 * qoff[d] + i] = keys[i].code;
    plen[d] = n;
  }
  free(keys);
}

/*
 * Evaluate device programs (3 qoff[d] + i, i < plen[d]). Edges: program order on every device;
 * data edges between stages on one device (weight 0); F(s,m) -> B(s,m); B(s,m) -> W(s,m); a
 * producer before its transfer and a transfer before its consumer (both also implied by any
 * program a builder above makes). Longest path by Kahn's algorithm; a cycle is a deadlock.
 * Busy time counts computation only, so time spent in transfers is bubble.
 */
static int simulate_programs(const ref_dag_in* g, const ref_sop* queue, const int* qoff,
                             const int* qlen, const int* prog, const int* plen,
                             int64_t* makespan, int64_t* bubble) {
  int S = g->S, M = g->M, nk = g->split ? 3 : 2;
  int nc = nk * S * M;         /* compute nodes: node_id */
  int nn = nc + 2 * S * M;     /* transfer nodes: nc + (dir * S + producer stage) * M + m */
  /* successors: at most two program successors (a transfer sits in two programs) + 4 data */
  int* succ = (int*)malloc(sizeof(int) * (size_t)nn * 6);
  int* nsucc = (int*)calloc(nn, sizeof(int));
  int* indeg = (int*)calloc(nn, sizeof(int));
  int64_t* dur = (int64_t*)calloc(nn, sizeof(int64_t));
  int64_t* est = (int64_t*)calloc(nn, sizeof(int64_t));
  int64_t* fin = (int64_t*)malloc(sizeof(int64_t) * nn);
  int* ready = (int*)malloc(sizeof(int) * nn);
#define PG_EDGE(a, b) (succ[(size_t)(a) * 6 + nsucc[a]++] = (b), indeg[b]++)
  for (int s = 0; s < S; ++s)
    for (int m = 0; m < M; ++m) {
      for (int k = 0; k < nk; ++k) dur[node_id(S, M, k, s, m)] = op_dur(g, k, s);
      if (s + 1 < S && g->dev[s] != g->dev[s + 1])
        dur[nc + (0 * S + s) * M + m] = g->link[g->dev[s] * g->P + g->dev[s + 1]];
      if (s > 0 && g->dev[s] != g->dev[s - 1])
        dur[nc + (1 * S + s) * M + m] = g->link[g->dev[s] * g->P + g->dev[s - 1]];
    }
  for (int d = 0; d < g->P; ++d) {
    int prev = -1;
    for (int i = 0; i < plen[d]; ++i) {
      const int code = prog[3 * qoff[d] + i], node = code & 0x0FFFFFFF;
      int item = node;
      if ((code >> 28) != PI_COMP) {
        const int xk = node / (S * M), xs = (node / M) % S, xm = node % M;
        item = nc + ((xk == KF ? 0 : 1) * S + xs) * M + xm;
      }
      if (prev >= 0) PG_EDGE(prev, item);
      prev = item;
    }
  }
  for (int s = 0; s < S; ++s)
    for (int m = 0; m < M; ++m) {
      if (s + 1 < S) {
        if (g->dev[s] == g->dev[s + 1]) {
          PG_EDGE(node_id(S, M, KF, s, m), node_id(S, M, KF, s + 1, m));
        } else {
          PG_EDGE(node_id(S, M, KF, s, m), nc + (0 * S + s) * M + m);
          PG_EDGE(nc + (0 * S + s) * M + m, node_id(S, M, KF, s + 1, m));
        }
      }
      if (s > 0) {
        if (g->dev[s] == g->dev[s - 1]) {
          PG_EDGE(node_id(S, M, KB, s, m), node_id(S, M, KB, s - 1, m));
        } else {
          PG_EDGE(node_id(S, M, KB, s, m), nc + (1 * S + s) * M + m);
          PG_EDGE(nc + (1 * S + s) * M + m, node_id(S, M, KB, s - 1, m));
        }
      }
      PG_EDGE(node_id(S, M, KF, s, m), node_id(S, M, KB, s, m));
      if (g->split) PG_EDGE(node_id(S, M, KB, s, m), node_id(S, M, KW, s, m));
    }
#undef PG_EDGE
  int nr = 0, head = 0, rc = SIM_OK;
  for (int i = 0; i < nn; ++i)
    if (indeg[i] == 0) ready[nr++] = i;
  while (head < nr) {
    const int u = ready[head++];
    fin[u] = est[u] + dur[u];
    for (int e = 0; e < nsucc[u]; ++e) {
      const int x = succ[(size_t)u * 6 + e];
      if (fin[u] > est[x]) est[x] = fin[u];
      if (--indeg[x] == 0) ready[nr++] = x;
    }
  }
  if (nr < nn) { /* some node never became ready: a cycle (unused transfer slots have no edges) */
    rc = SIM_CYCLE;
  } else {
    int64_t ms = 0;
    for (int i = 0; i < nn; ++i)
      if (fin[i] > ms) ms = fin[i];
    *makespan = ms;
    for (int d = 0; d < g->P; ++d) {
      int64_t busy = 0;
      for (int i = 0; i < qlen[d]; ++i)
        busy += op_dur(g, queue[qoff[d] + i].kind, queue[qoff[d] + i].s);
      bubble[d] = ms - busy;
    }
  }
  free(succ);
  free(nsucc);
  free(indeg);
  free(dur);
  free(est);
  free(fin);
  free(ready);
  return rc;
}

/*
 * The executor's deadlock-free, overlap-aware reordering (§7, "Unified Pipeline Executor": its
 * three steps), evaluated with handshake transfers.
 *
 * Transfers: a device that reaches a send or a receive in its program waits there until the
 * other end has been reached too (a blocking point-to-point handshake); then both go on at
 * once, and the data arrives c = link[p][q] after the handshake, while both devices compute
 * (the transfer runs beside computation). The consumer may start once the data has arrived.
 *
 * Every transfer t (producer X on device p -> consumer Y on device q) has a key: the end of X in
 * the asynchronous schedule (§1.3), then X's level (the number of ops on the longest dependency
 * chain before X, queue order included), then X's node id. The key order is a total order in
 * which every dependency strictly increases (positive durations not needed: the level breaks
 * ties). The program starts as the naive coordination of §3.3: the receive of t in the gap
 * before Y, the send after X; a gap g of a device is the point before its computation g (gap
 * n: after the last of its n computations).
 *  1. Mismatched pairs: walk each device's communication items in program order; an item whose
 *     key is below the largest key before it is out of the order the other devices follow for
 *     their ends of the same transfers (a pair that can close a cycle of waits). Only receives
 *     can be out of order: whatever precedes a send ends before its producer does.
 *  2. Feasible window of a mismatched receive: its dependent computations are X (on p) and Y
 *     (on q). The receive must stay before Y and, to restore the order, after every in-order
 *     item of a smaller key and before the first one of a larger key; within that range, only
 *     gaps whose post time (the end of q's previous computation in the asynchronous schedule,
 *     0 for gap 0) is not before X starts (earlier, q would only wait): the window
 *     [max(lo, gX), hi] (just hi if that is empty).
 *  3. Cost of a gap: the communication span, |X's end - the gap's post time| (the time one end
 *     waits for the other), minus the overlap with neighbouring computation, min(c, the
 *     durations of q's computations from that gap up to Y) (what q computes while the data is
 *     in flight). Mismatched receives are placed greedily in key order, each at its cheapest
 *     gap (ties: the latest), and the next one's range starts at that gap.
 * Within a gap, communication items run in key order. Every device then meets its transfers in
 * key order, so no cycle of waits can form.
 */
typedef struct {
  int64_t t, lvl;
  int node, gap, code;
} comm_item;

static int cmp_comm_item(const void* a, const void* b) {
  const comm_item *x = (const comm_item*)a, *y = (const comm_item*)b;
  if (x->t != y->t) return x->t < y->t ? -1 : 1;
  if (x->lvl != y->lvl) return x->lvl < y->lvl ? -1 : 1;
  return x->node < y->node ? -1 : x->node > y->node;
}

/* Returns 0, or -1 if the programs' communication is not in key order (cannot happen). stats
 * (nullable): [0] += transfers (receives), [1] += mismatched receives. */
static int reorder_programs(const ref_dag_in* g, const ref_sop* queue, const int* qoff,
                            const int* qlen, const int64_t* start, const int64_t* lvl, int* prog,
                            int* plen, int64_t* stats) {
  const int S = g->S, M = g->M;
  int rc = 0;
  for (int d = 0; d < g->P && rc == 0; ++d) {
    const int n = qlen[d];
    const ref_sop* q = queue + qoff[d];
    comm_item* it = (comm_item*)malloc(sizeof(comm_item) * (size_t)(2 * n + 1));
    int* flagged = (int*)malloc(sizeof(int) * (size_t)(2 * n + 1));
    int64_t* post = (int64_t*)malloc(sizeof(int64_t) * (size_t)(n + 1)); /* post time of gap */
    post[0] = 0;
    for (int i = 0; i < n; ++i)
      post[i + 1] = start[node_id(S, M, q[i].kind, q[i].s, q[i].m)] + op_dur(g, q[i].kind, q[i].s);
    int ni = 0;
    for (int i = 0; i < n; ++i) {
      const int y = node_id(S, M, q[i].kind, q[i].s, q[i].m);
      const int x = cross_producer(g, q[i].kind, q[i].s, q[i].m);
      if (x >= 0) {
        const int xk = x / (S * M), xs = (x / M) % S;
        it[ni++] = (comm_item){start[x] + op_dur(g, xk, xs), lvl[x], x, i, (PI_RECV << 28) | x};
      }
      if (cross_consumer(g, q[i].kind, q[i].s, q[i].m) >= 0)
        it[ni++] = (comm_item){post[i + 1], lvl[y], y, i + 1, (PI_SEND << 28) | y};
    }
    /* step 1 */
    int nf = 0, top = -1, nrecv = 0;
    int* rec_ok = (int*)calloc((size_t)(ni + 1), sizeof(int)); /* 1: in order (a record) */
    for (int j = 0; j < ni; ++j) {
      nrecv += (it[j].code >> 28) == PI_RECV;
      if (top < 0 || cmp_comm_item(&it[j], &it[top]) > 0) {
        top = j;
        rec_ok[j] = 1;
      } else {
        flagged[nf++] = j;
      }
    }
    if (stats) stats[0] += nrecv, stats[1] += nf;
    /* steps 2 and 3, in key order */
    for (int a = 1; a < nf; ++a) { /* insertion sort of the flagged items by key */
      const int v = flagged[a];
      int b = a;
      while (b > 0 && cmp_comm_item(&it[v], &it[flagged[b - 1]]) < 0) {
        flagged[b] = flagged[b - 1];
        --b;
      }
      flagged[b] = v;
    }
    /* the in-order items are sorted by key and by gap; as the mismatched ones come in key
     * order, the in-order items below each one only grow: one cursor (j) serves them all */
    int lastg = 0, lo_rec = 0, j = 0;
    for (int a = 0; a < nf; ++a) {
      comm_item* f = &it[flagged[a]];
      for (; j < ni; ++j) {
        if (!rec_ok[j]) continue;
        if (cmp_comm_item(&it[j], f) > 0) break;
        lo_rec = it[j].gap; /* an in-order item of a smaller key */
      }
      if ((f->code >> 28) != PI_RECV || j == ni) { /* cannot happen (see above) */
        rc = -1;
        break;
      }
      const int lo = lastg > lo_rec ? lastg : lo_rec, hi = it[j].gap;
      const int X = f->node, iY = f->gap;
      const int xk = X / (S * M), xs = (X / M) % S;
      const int64_t c = g->link[g->dev[xs] * g->P + d];
      const int64_t xend = start[X] + op_dur(g, xk, xs);
      /* gx: the first gap whose post time is not before X starts (post[] never decreases) */
      int gx = 0, gend = n + 1;
      while (gx < gend) {
        const int mid = (gx + gend) / 2;
        if (post[mid] < start[X]) gx = mid + 1;
        else gend = mid;
      }
      int first = lo > gx ? lo : gx;
      if (first > hi) first = hi;
      int64_t D = 0; /* durations of the computations in gaps [gap, iY) */
      for (int i = hi; i < iY; ++i) D += op_dur(g, q[i].kind, q[i].s);
      int best = -1;
      int64_t bestc = 0;
      for (int gp = hi; gp >= first; --gp) {
        if (gp < hi) D += op_dur(g, q[gp].kind, q[gp].s);
        const int64_t span = xend > post[gp] ? xend - post[gp] : post[gp] - xend;
        const int64_t cost = span - (D < c ? D : c);
        if (best < 0 || cost < bestc) best = gp, bestc = cost;
      }
      f->gap = best;
      lastg = best;
    }
    if (rc == 0) {
      qsort(it, (size_t)ni, sizeof(comm_item), cmp_comm_item);
      for (int j = 1; j < ni; ++j)
        if (it[j].gap < it[j - 1].gap) rc = -1;
      int np = 0, j = 0;
      int* out = prog + 3 * qoff[d];
      for (int i = 0; i < n; ++i) {
        while (j < ni && it[j].gap <= i) out[np++] = it[j++].code;
        out[np++] = (PI_COMP << 28) | node_id(S, M, q[i].kind, q[i].s, q[i].m);
      }
      while (j < ni) out[np++] = it[j++].code;
      plen[d] = np;
    }
    free(it);
    free(flagged);
    free(post);
    free(rec_ok);
  }
  return rc;
}

/*
 * Evaluate device programs with handshake transfers. Nodes: the computations; per transfer a
 * handshake node (duration 0) in both its devices' programs and an arrival node (duration c)
 * between the handshake and the consumer. Edges: program order; the producer before its
 * handshake; same-device data edges; F(s,m) -> B(s,m); B(s,m) -> W(s,m). Longest path by Kahn's
 * algorithm; a cycle is a deadlock. Busy time counts computation only.
 */
static int simulate_handshake(const ref_dag_in* g, const ref_sop* queue, const int* qoff,
                              const int* qlen, const int* prog, const int* plen,
                              int64_t* makespan, int64_t* bubble) {
  const int S = g->S, M = g->M, nk = g->split ? 3 : 2;
  const int nc = nk * S * M, nt = 2 * S * M, nn = nc + 2 * nt;
  int* succ = (int*)malloc(sizeof(int) * (size_t)nn * 6);
  int* nsucc = (int*)calloc(nn, sizeof(int));
  int* indeg = (int*)calloc(nn, sizeof(int));
  int64_t* dur = (int64_t*)calloc(nn, sizeof(int64_t));
  int64_t* est = (int64_t*)calloc(nn, sizeof(int64_t));
  int64_t* fin = (int64_t*)malloc(sizeof(int64_t) * nn);
  int* ready = (int*)malloc(sizeof(int) * nn);
  char* used = (char*)calloc(nn, 1);
#define HS_EDGE(a, b) (succ[(size_t)(a) * 6 + nsucc[a]++] = (b), indeg[b]++)
  /* transfer index of producer (kind, s, m): (dir * S + s) * M + m, dir 0 forward, 1 backward */
  for (int s = 0; s < S; ++s)
    for (int m = 0; m < M; ++m) {
      for (int k = 0; k < nk; ++k) dur[node_id(S, M, k, s, m)] = op_dur(g, k, s), used[node_id(S, M, k, s, m)] = 1;
      if (s + 1 < S && g->dev[s] != g->dev[s + 1])
        dur[nc + nt + (0 * S + s) * M + m] = g->link[g->dev[s] * g->P + g->dev[s + 1]];
      if (s > 0 && g->dev[s] != g->dev[s - 1])
        dur[nc + nt + (1 * S + s) * M + m] = g->link[g->dev[s] * g->P + g->dev[s - 1]];
    }
  for (int d = 0; d < g->P; ++d) {
    int prev = -1;
    for (int i = 0; i < plen[d]; ++i) {
      const int code = prog[3 * qoff[d] + i], node = code & 0x0FFFFFFF;
      int item = node;
      if ((code >> 28) != PI_COMP) {
        const int xk = node / (S * M), xs = (node / M) % S, xm = node % M;
        item = nc + ((xk == KF ? 0 : 1) * S + xs) * M + xm;
      }
      used[item] = 1;
      if (prev >= 0) HS_EDGE(prev, item);
      prev = item;
    }
  }
  for (int s = 0; s < S; ++s)
    for (int m = 0; m < M; ++m) {
      if (s + 1 < S) {
        const int x = node_id(S, M, KF, s, m), y = node_id(S, M, KF, s + 1, m);
        if (g->dev[s] == g->dev[s + 1]) {
          HS_EDGE(x, y);
        } else {
          const int h = nc + (0 * S + s) * M + m;
          HS_EDGE(x, h);
          HS_EDGE(h, h + nt);
          HS_EDGE(h + nt, y);
          used[h] = used[h + nt] = 1;
        }
      }
      if (s > 0) {
        const int x = node_id(S, M, KB, s, m), y = node_id(S, M, KB, s - 1, m);
        if (g->dev[s] == g->dev[s - 1]) {
          HS_EDGE(x, y);
        } else {
          const int h = nc + (1 * S + s) * M + m;
          HS_EDGE(x, h);
          HS_EDGE(h, h + nt);
          HS_EDGE(h + nt, y);
          used[h] = used[h + nt] = 1;
        }
      }
      HS_EDGE(node_id(S, M, KF, s, m), node_id(S, M, KB, s, m));
      if (g->split) HS_EDGE(node_id(S, M, KB, s, m), node_id(S, M, KW, s, m));
    }
#undef HS_EDGE
  int nr = 0, head = 0, nused = 0, rc = SIM_OK;
  for (int i = 0; i < nn; ++i) {
    nused += used[i];
    if (used[i] && indeg[i] == 0) ready[nr++] = i;
  }
  while (head < nr) {
    const int u = ready[head++];
    fin[u] = est[u] + dur[u];
    for (int e = 0; e < nsucc[u]; ++e) {
      const int x = succ[(size_t)u * 6 + e];
      if (fin[u] > est[x]) est[x] = fin[u];
      if (--indeg[x] == 0) ready[nr++] = x;
    }
  }
  if (nr < nused) {
    rc = SIM_CYCLE;
  } else {
    int64_t ms = 0;
    for (int i = 0; i < nr; ++i)
      if (fin[ready[i]] > ms) ms = fin[ready[i]];
    *makespan = ms;
    for (int d = 0; d < g->P; ++d) {
      int64_t busy = 0;
      for (int i = 0; i < qlen[d]; ++i)
        busy += op_dur(g, queue[qoff[d] + i].kind, queue[qoff[d] + i].s);
      bubble[d] = ms - busy;
    }
  }
  free(succ);
  free(nsucc);
  free(indeg);
  free(dur);
  free(est);
  free(fin);
  free(ready);
  free(used);
  return rc;
}

/* The reordering above on the asynchronous schedule of the queues, then its evaluation. */
static int simulate_reordered(const ref_dag_in* g, const ref_sop* queue, const int* qoff,
                              const int* qlen, int64_t* makespan, int64_t* bubble,
                              int64_t* stats) {
  const int S = g->S, M = g->M, P = g->P, nk = g->split ? 3 : 2;
  int total = 0;
  for (int d = 0; d < P; ++d) total += qlen[d];
  int* prog = (int*)malloc(sizeof(int) * (size_t)(3 * total + 1));
  int plen[64];
  int64_t* start = (int64_t*)malloc(sizeof(int64_t) * (size_t)nk * S * M);
  int64_t* lvl = (int64_t*)malloc(sizeof(int64_t) * (size_t)nk * S * M);
  int64_t ms0, bub0[64];
  ref_dag_in plain = *g;
  plain.serial = 0;
  int rc = simulate(&plain, queue, qoff, qlen, &ms0, bub0, start, NULL);
  if (rc == SIM_OK) {
    /* levels: the same queues with every op taking 1 and every transfer nothing */
    int64_t one[64], zero_w[64];
    int64_t* nolink = (int64_t*)calloc((size_t)P * P, sizeof(int64_t));
    for (int s = 0; s < S; ++s) one[s] = 1, zero_w[s] = g->split ? 1 : 0;
    ref_dag_in unit = {S, M, g->split, P, g->dev, one, one, zero_w, nolink, 0};
    rc = simulate(&unit, queue, qoff, qlen, &ms0, bub0, lvl, NULL);
    free(nolink);
  }
  if (stats) stats[0] = stats[1] = 0;
  if (rc == SIM_OK &&
      reorder_programs(g, queue, qoff, qlen, start, lvl, prog, plen, stats) != 0)
    rc = SIM_BADQ;
  if (rc == SIM_OK) rc = simulate_handshake(g, queue, qoff, qlen, prog, plen, makespan, bubble);
  free(start);
  free(lvl);
  free(prog);
  return rc;
}

/* xfer 2: the naive coordination; xfer 3: the reordered one (needs the asynchronous schedule). */
static int simulate_coordinated(const ref_dag_in* g, const ref_sop* queue, const int* qoff,
                                const int* qlen, int ordered, int64_t* makespan,
                                int64_t* bubble) {
  int total = 0;
  for (int d = 0; d < g->P; ++d) total += qlen[d];
  int* prog = (int*)malloc(sizeof(int) * (size_t)(3 * total + 1));
  int plen[64];
  int rc = SIM_OK;
  if (ordered) {
    const int nk = g->split ? 3 : 2;
    int64_t* start = (int64_t*)malloc(sizeof(int64_t) * (size_t)nk * g->S * g->M);
    int64_t ms0, bub0[64];
    ref_dag_in plain = *g;
    plain.serial = 0;
    rc = simulate(&plain, queue, qoff, qlen, &ms0, bub0, start, NULL);
    if (rc == SIM_OK) ordered_programs(g, queue, qoff, qlen, start, prog, plen);
    free(start);
  } else {
    naive_programs(g, queue, qoff, qlen, prog, plen);
  }
  if (rc == SIM_OK) rc = simulate_programs(g, queue, qoff, qlen, prog, plen, makespan, bubble);
  free(prog);
  return rc;
}

/* ------------------------------------------------------------------------------------------ */
/* MERGE: the ideal stage-level order.                                                         */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
  int64_t tau;
  int s;     /* stage (tie-break) */
  ref_op op; /* the op in device-local terms */
} merge_key;

static int cmp_merge(const void* a, const void* b) {
  const merge_key* x = (const merge_key*)a;
  const merge_key* y = (const merge_key*)b;
  if (x->tau != y->tau) return x->tau < y->tau ? -1 : 1;
  if (x->s != y->s) return x->s < y->s ? -1 : 1;
  return 0;
}

/* Ideal start time of every op of the stage-level pipeline (node-id indexed).
 * Each stage s is its own virtual device running INTER(S, 1, M, s, split, s); unit costs
 * (F = 1; fused B = 2; split B = W = 1); zero transfer cost. */
static int merge_tau(int S, int M, int split, int64_t* tau) {
  int per = (split ? 3 : 2) * M;
  ref_sop* q = (ref_sop*)malloc(sizeof(ref_sop) * (size_t)per * S);
  ref_op* tmp = (ref_op*)malloc(sizeof(ref_op) * per);
  int* qoff = (int*)malloc(sizeof(int) * S);
  int* qlen = (int*)malloc(sizeof(int) * S);
  int* dev = (int*)malloc(sizeof(int) * S);
  int64_t* F = (int64_t*)malloc(sizeof(int64_t) * S);
  int64_t* B = (int64_t*)malloc(sizeof(int64_t) * S);
  int64_t* W = (int64_t*)malloc(sizeof(int64_t) * S);
  int64_t* link = (int64_t*)calloc((size_t)S * S, sizeof(int64_t));
  int64_t* bub = (int64_t*)malloc(sizeof(int64_t) * S);
  for (int s = 0; s < S; ++s) {
    dev[s] = s;
    F[s] = 1;
    B[s] = 1; /* split: B = 1, W = 1; fused op B + W = 2 */
    W[s] = 1;
    int n = gen_inter(S, 1, M, s, split, s, tmp);
    qoff[s] = s * per;
    qlen[s] = n;
    for (int i = 0; i < n; ++i) q[s * per + i] = (ref_sop){tmp[i].kind, s, tmp[i].m};
  }
  ref_dag_in g = {S, M, split, S, dev, F, B, W, link, 0};
  int64_t ms;
  int rc = simulate(&g, q, qoff, qlen, &ms, bub, tau, NULL);
  free(q);
  free(tmp);
  free(qoff);
  free(qlen);
  free(dev);
  free(F);
  free(B);
  free(W);
  free(link);
  free(bub);
  return rc;
}

/* ------------------------------------------------------------------------------------------ */
/* Building the queues of a candidate.                                                         */
/* ------------------------------------------------------------------------------------------ */

/* Local-op queues for every device of a structurally valid candidate, before perturbations.
 * q holds P rows of capacity qcap. Returns 0 or an error. */
static int build_local_queues(const ref_problem* pr, const ref_cand* c, ref_op* q, int qcap,
                              int* qlen) {
  int split;
  int gen = resolve(pr, c, &split);
  int P = pr->P, M = pr->M, v = c->v, S = c->S;
  if (gen == GEN_AFAB) {
    for (int d = 0; d < P; ++d) qlen[d] = gen_afab(v, M, q + (size_t)d * qcap);
    return 0;
  }
  if (gen == GEN_INTER) {
    for (int d = 0; d < P; ++d) {
      int A[64];
      stages_of(c, d, A);
      int r = A[0];
      qlen[d] = gen_inter(P, v, M, r, split, r, q + (size_t)d * qcap);
    }
    return 0;
  }
  /* MERGE */
  int nk = split ? 3 : 2;
  int64_t* tau = (int64_t*)malloc(sizeof(int64_t) * (size_t)nk * S * M);
  if (merge_tau(S, M, split, tau) != SIM_OK) {
    free(tau);
    return REF_EINVAL;
  }
  merge_key* keys = (merge_key*)malloc(sizeof(merge_key) * (size_t)nk * v * M);
  for (int d = 0; d < P; ++d) {
    int A[64];
    int nA = stages_of(c, d, A);
    int n = 0;
    for (int k = 0; k < nA; ++k)
      for (int kind = 0; kind < nk; ++kind)
        for (int m = 0; m < M; ++m) {
          keys[n].tau = tau[node_id(S, M, kind, A[k], m)];
          keys[n].s = A[k];
          keys[n].op = (ref_op){kind, k, m};
          n++;
        }
    qsort(keys, n, sizeof(merge_key), cmp_merge);
    for (int i = 0; i < n; ++i) q[(size_t)d * qcap + i] = keys[i].op;
    qlen[d] = n;
  }
  free(keys);
  free(tau);
  return 0;
}

/* Apply the perturbation moves in order. Returns 0, or REF_EINVAL if one is out of range. */
/* Move entry `from` of a queue row so that it ends at index `to`; the entries between shift by
 * one place. */
static void move_op(ref_op* row, int from, int to) {
  ref_op moved = row[from];
  if (from < to)
    memmove(row + from, row + from + 1, sizeof(ref_op) * (size_t)(to - from));
  else if (from > to)
    memmove(row + to + 1, row + to, sizeof(ref_op) * (size_t)(from - to));
  row[to] = moved;
}

static int apply_perturbations(const ref_problem* pr, const ref_cand* c, ref_op* q, int qcap,
                               const int* qlen) {
  for (int i = 0; i < c->n_pert; ++i) {
    int d = c->pert[i][0], from = c->pert[i][1], to = c->pert[i][2];
    if (d >= pr->P || from >= qlen[d] || to >= qlen[d]) return REF_EINVAL;
    move_op(q + (size_t)d * qcap, from, to);
  }
  return 0;
}

static void stage_costs(const ref_cand* c, const int64_t* costs, int64_t* F,
                        int64_t* B, int64_t* W) {
  for (int s = 0; s < c->S; ++s) {
    F[s] = B[s] = W[s] = 0;
    for (int l = c->b[s]; l < c->b[s + 1]; ++l) {
      F[s] += costs[3 * l + 0];
      B[s] += costs[3 * l + 1];
      W[s] += costs[3 * l + 2];
    }
  }
}

/* Memory model (§5 memory nodes; §6 Eq. 2's peak per device). Every op of a device holds its
 * memory node's tensors: a forward F(s,m) allocates the activations of stage s for micro-batch m
 * when it starts; the last backward op of (s,m) — B when fused, W when split — releases them
 * when it ends. Static bytes (weights, gradients, optimizer state) of the device's stages are
 * held throughout. Events are replayed in time order (an op's release before a later op's
 * allocation at the same instant; ties between ops of one device in their queue order), and
 * peak_d = static_d + the largest running activation total. act[s], stat[s]: per-stage bytes. */
typedef struct {
  int64_t t;
  int key; /* 2 * queue position, + 1 for a release */
  int64_t delta;
} mem_event;

static int cmp_event(const void* a, const void* b) {
  const mem_event* x = (const mem_event*)a;
  const mem_event* y = (const mem_event*)b;
  if (x->t != y->t) return x->t < y->t ? -1 : 1;
  return x->key < y->key ? -1 : x->key > y->key ? 1 : 0;
}

static void peak_memory(const ref_dag_in* g, const ref_sop* sq, const int* qoff, const int* qlen,
                        const int64_t* start, const int64_t* act, const int64_t* stat,
                        int64_t* peak, int* ppos) {
  for (int d = 0; d < g->P; ++d) {
    int64_t base = 0;
    for (int s = 0; s < g->S; ++s)
      if (g->dev[s] == d) base += stat[s];
    mem_event* ev = (mem_event*)malloc(sizeof(mem_event) * (size_t)(qlen[d] > 0 ? qlen[d] : 1));
    int ne = 0;
    for (int i = 0; i < qlen[d]; ++i) {
      ref_sop o = sq[qoff[d] + i];
      int64_t st = start[node_id(g->S, g->M, o.kind, o.s, o.m)];
      if (o.kind == KF)
        ev[ne++] = (mem_event){st, 2 * i, act[o.s]};
      else if ((o.kind == KB && !g->split) || o.kind == KW)
        ev[ne++] = (mem_event){st + op_dur(g, o.kind, o.s), 2 * i + 1, -act[o.s]};
    }
    qsort(ev, ne, sizeof(mem_event), cmp_event);
    int64_t cur = 0, hi = 0;
    int at = -1;
    for (int i = 0; i < ne; ++i) {
      cur += ev[i].delta;
      if (cur > hi) hi = cur, at = ev[i].key / 2;
    }
    peak[d] = base + hi;
    if (ppos) ppos[d] = at; /* queue position of the allocation that first reaches the peak */
    free(ev);
  }
}

/* Communication nodes and their overlap (§5 "Estimating Pipeline Performance"; the comm counts
 * of §8's communication table). Every cross-device data edge X -> Y is a send node on X's device
 * and a receive node on Y's, each lasting c = link[dev X][dev Y]; the transfer runs from X's
 * end for c. §5 marks a node overlappable when it can run beside subsequent computation and
 * then records the smaller of the computation's and the communication's durations. The
 * computation a node can run beside is the one adjacent to it in its device's order that does
 * not wait for it: for a send, the op that follows X; for a receive, the op that precedes Y
 * (Y itself needs the data). The node is overlappable when that op runs during the transfer
 * (their intervals share a positive length); overlap = min(duration of that op, c).
 * comm[4] += {nodes, overlappable nodes, node time (2c per edge), overlap time}. */
static void comm_overlap(const ref_dag_in* g, const ref_sop* sq, const int* qoff, const int* qlen,
                         const int64_t* start, int64_t* comm) {
  const int S = g->S, M = g->M;
  for (int d = 0; d < g->P; ++d) {
    for (int i = 0; i < qlen[d]; ++i) {
      const ref_sop o = sq[qoff[d] + i];
      const int64_t st = start[node_id(S, M, o.kind, o.s, o.m)];
      const int64_t fin = st + op_dur(g, o.kind, o.s);
      /* the op's input from another device, and the op it is received during */
      int sp = -1;
      if (o.kind == KF && o.s > 0) sp = o.s - 1;
      if (o.kind == KB && o.s < S - 1) sp = o.s + 1;
      if (sp >= 0 && g->dev[sp] != d) {
        const int64_t c = g->link[g->dev[sp] * g->P + d];
        const int64_t xs = start[node_id(S, M, o.kind, sp, o.m)];
        const int64_t xf = xs + op_dur(g, o.kind, sp);
        comm[0] += 1, comm[2] += c;
        if (i > 0) {
          const ref_sop z = sq[qoff[d] + i - 1];
          const int64_t zs = start[node_id(S, M, z.kind, z.s, z.m)];
          const int64_t zf = zs + op_dur(g, z.kind, z.s);
          const int64_t lo = zs > xf ? zs : xf, hi = zf < xf + c ? zf : xf + c;
          if (hi > lo) comm[1] += 1, comm[3] += zf - zs < c ? zf - zs : c;
        }
      }
      /* the op's output to another device, and the op it is sent during */
      int sc = -1;
      if (o.kind == KF && o.s < S - 1) sc = o.s + 1;
      if (o.kind == KB && o.s > 0) sc = o.s - 1;
      if (sc >= 0 && g->dev[sc] != d) {
        const int64_t c = g->link[d * g->P + g->dev[sc]];
        comm[0] += 1, comm[2] += c;
        if (i + 1 < qlen[d]) {
          const ref_sop nx = sq[qoff[d] + i + 1];
          const int64_t ns = start[node_id(S, M, nx.kind, nx.s, nx.m)];
          const int64_t nf = ns + op_dur(g, nx.kind, nx.s);
          const int64_t lo = ns > fin ? ns : fin, hi = nf < fin + c ? nf : fin + c;
          if (hi > lo) comm[1] += 1, comm[3] += nf - ns < c ? nf - ns : c;
        }
      }
    }
  }
}

/* Evaluate a candidate given its local queues (after perturbations). mem (nullable): layer
 * memory [L][2] = {activation bytes per micro-batch, static bytes}; then peak[P] is filled, and
 * ppos[P] (nullable) with the queue position at which each device first reaches its peak (-1
 * when it holds no activations). */
/* xfer: 0 asynchronous transfers (the plain model), 1 serialised links, 2 blocking rendezvous in
 * the naive coordination, 3 blocking rendezvous in the reordered coordination (transfers at
 * their ideal start), 4 the executor's three-step reordering with handshake transfers (comm then
 * receives its two statistics). */
static int eval_local_c(const ref_problem* pr, const ref_cand* c, const int64_t* costs,
                        const int64_t* link, const ref_op* q, int qcap, const int* qlen,
                        const int64_t* mem, int64_t* ms, int64_t* bub, int64_t* peak, int* ppos,
                        int64_t* comm, int xfer, int64_t* bounds) {
  int P = pr->P, S = c->S, split;
  resolve(pr, c, &split);
  int64_t F[64], B[64], W[64];
  stage_costs(c, costs, F, B, W);
  int total = 0;
  int qoff[64];
  for (int d = 0; d < P; ++d) qoff[d] = total, total += qlen[d];
  ref_sop* sq = (ref_sop*)malloc(sizeof(ref_sop) * (size_t)(total > 0 ? total : 1));
  for (int d = 0; d < P; ++d) {
    int A[64];
    int nA = stages_of(c, d, A);
    for (int i = 0; i < qlen[d]; ++i) {
      ref_op o = q[(size_t)d * qcap + i];
      int s = (o.chunk >= 0 && o.chunk < nA) ? A[o.chunk] : -1;
      sq[qoff[d] + i] = (ref_sop){o.kind, s, o.m};
    }
  }
  ref_dag_in g = {S, pr->M, split, P, c->dev, F, B, W, link, xfer == 1};
  int64_t* start = (mem || comm || bounds)
                       ? (int64_t*)malloc(sizeof(int64_t) * (size_t)3 * S * pr->M)
                       : NULL;
  int rc = xfer == 4   ? simulate_reordered(&g, sq, qoff, qlen, ms, bub, comm)
           : xfer >= 2 ? simulate_coordinated(&g, sq, qoff, qlen, xfer == 3, ms, bub)
                       : simulate(&g, sq, qoff, qlen, ms, bub, start, NULL);
  if (bounds && rc == SIM_OK) {
    /* per device: start of its first op, end of its last op (0, 0 for an empty queue) */
    for (int d = 0; d < P; ++d) {
      bounds[2 * d] = bounds[2 * d + 1] = 0;
      if (qlen[d] > 0) {
        const ref_sop a = sq[qoff[d]], z = sq[qoff[d] + qlen[d] - 1];
        bounds[2 * d] = start[node_id(S, pr->M, a.kind, a.s, a.m)];
        bounds[2 * d + 1] = start[node_id(S, pr->M, z.kind, z.s, z.m)] + op_dur(&g, z.kind, z.s);
      }
    }
  }
  if (comm && rc == SIM_OK && xfer != 4) {
    for (int k = 0; k < 4; ++k) comm[k] = 0;
    comm_overlap(&g, sq, qoff, qlen, start, comm);
  }
  if (mem && rc == SIM_OK) {
    int64_t act[64], stat[64];
    for (int s = 0; s < S; ++s) {
      act[s] = stat[s] = 0;
      for (int l = c->b[s]; l < c->b[s + 1]; ++l) act[s] += mem[2 * l], stat[s] += mem[2 * l + 1];
    }
    peak_memory(&g, sq, qoff, qlen, start, act, stat, peak, ppos);
  }
  free(start);
  free(sq);
  return rc;
}

static int eval_local(const ref_problem* pr, const ref_cand* c, const int64_t* costs,
                      const int64_t* link, const ref_op* q, int qcap, const int* qlen,
                      const int64_t* mem, int64_t* ms, int64_t* bub, int64_t* peak, int* ppos) {
  return eval_local_c(pr, c, costs, link, q, qcap, qlen, mem, ms, bub, peak, ppos, NULL, 0, NULL);
}

/* Full evaluation of one candidate record: makespan + bubbles, or sentinels. */
static void eval_record(const ref_problem* pr, const int64_t* costs, const int64_t* mem,
                        const int64_t* link, const uint8_t* rec, int64_t* ms, int64_t* bub,
                        int64_t* peak, int64_t* comm, int xfer, int64_t* bounds) {
  ref_cand* c = (ref_cand*)malloc(sizeof(ref_cand));
  decode(pr, rec, c);
  int P = pr->P;
  int64_t sentinel = 0;
  if (!valid_structure(pr, c)) {
    sentinel = REF_INVALID;
  } else {
    int qcap = 3 * c->v * pr->M;
    ref_op* q = (ref_op*)malloc(sizeof(ref_op) * (size_t)qcap * P);
    int qlen[64];
    if (build_local_queues(pr, c, q, qcap, qlen) != 0 ||
        apply_perturbations(pr, c, q, qcap, qlen) != 0) {
      sentinel = REF_INVALID;
    } else {
      int rc =
          eval_local_c(pr, c, costs, link, q, qcap, qlen, mem, ms, bub, peak, NULL, comm, xfer,
                       bounds);
      if (rc == SIM_CYCLE) sentinel = REF_DEADLOCK;
      else if (rc != SIM_OK) sentinel = REF_INVALID;
    }
    free(q);
  }
  if (sentinel != 0) {
    *ms = sentinel;
    for (int d = 0; d < P; ++d) bub[d] = sentinel;
    if (peak)
      for (int d = 0; d < P; ++d) peak[d] = sentinel;
    if (comm)
      for (int k = 0; k < (xfer == 4 ? 2 : 4); ++k) comm[k] = sentinel;
    if (bounds)
      for (int k = 0; k < 2 * P; ++k) bounds[k] = sentinel;
  }
  free(c);
}

/* ------------------------------------------------------------------------------------------ */
/* Selective W advancing (§6 "Scheduling Tuning", the third policy; §6 Eq. 2's capacity bound). */
/* While some device's peak exceeds its capacity, take the lowest-numbered such device and the */
/* queue position p at which its running activation total first reaches the peak (an F). A W   */
/* of that device is eligible when it sits after p, its B sits before p (so its stage's         */
/* activations are held at p) and the stage holds activations; advancing it moves it to index  */
/* p, so its release comes before that allocation. Eligible W are tried in queue order: the     */
/* first whose advance does not lengthen the makespan is taken (a device's busy time is fixed,  */
/* so then no bubble grows); if every one lengthens it, the first (earliest) is taken. Repeat   */
/* until all devices fit, nothing is eligible, or max_adv advances have been made.              */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
  int d, from, to;
} ref_move;

/* Runs the policy on queues q (changed in place). Returns the evaluation status (SIM_OK,
 * SIM_CYCLE, SIM_BADQ) of the given queues; on SIM_OK, ms/bub/peak describe the final queues,
 * *fits tells whether every device is within cap, and moves (nullable) receives the advances,
 * *n_moves of them, as perturbation triples (device, from, to). */
static int advance_w(const ref_problem* pr, const ref_cand* c, const int64_t* costs,
                     const int64_t* mem, const int64_t* cap, const int64_t* link, ref_op* q,
                     int qcap, const int* qlen, int max_adv, int64_t* ms, int64_t* bub,
                     int64_t* peak, int* fits, ref_move* moves, int* n_moves) {
  const int P = pr->P, M = pr->M;
  int ppos[64];
  *n_moves = 0;
  *fits = 0;
  int rc = eval_local(pr, c, costs, link, q, qcap, qlen, mem, ms, bub, peak, ppos);
  if (rc != SIM_OK) return rc;
  int64_t act[64];
  for (int s = 0; s < c->S; ++s) {
    act[s] = 0;
    for (int l = c->b[s]; l < c->b[s + 1]; ++l) act[s] += mem[2 * l];
  }
  int* posB = (int*)malloc(sizeof(int) * (size_t)c->v * M);
  int64_t tms, tbub[64], tpeak[64];
  int tpos[64];
  for (;;) {
    int d = -1;
    for (int e = 0; e < P; ++e)
      if (peak[e] > cap[e]) {
        d = e;
        break;
      }
    if (d < 0) {
      *fits = 1;
      break;
    }
    if (*n_moves >= max_adv || ppos[d] < 0) break;
    const int p = ppos[d];
    ref_op* row = q + (size_t)d * qcap;
    int A[64];
    stages_of(c, d, A);
    for (int i = 0; i < c->v * M; ++i) posB[i] = qlen[d];
    for (int i = 0; i < qlen[d]; ++i)
      if (row[i].kind == KB) posB[row[i].chunk * M + row[i].m] = i;
    int first = -1, chosen = -1;
    for (int j = p + 1; j < qlen[d]; ++j) {
      const ref_op o = row[j];
      if (o.kind != KW || act[A[o.chunk]] <= 0 || posB[o.chunk * M + o.m] > p) continue;
      if (first < 0) first = j;
      move_op(row, j, p);
      rc = eval_local(pr, c, costs, link, q, qcap, qlen, mem, &tms, tbub, tpeak, tpos);
      if (rc == SIM_OK && tms <= *ms) {
        chosen = j;
        break;
      }
      move_op(row, p, j);
    }
    if (first < 0) break;
    if (chosen < 0) {
      chosen = first;
      move_op(row, first, p);
      rc = eval_local(pr, c, costs, link, q, qcap, qlen, mem, &tms, tbub, tpeak, tpos);
    }
    /* a W has no consumers, so advancing it past other ops of its device creates no cycle */
    if (rc != SIM_OK) break;
    *ms = tms;
    for (int e = 0; e < P; ++e) bub[e] = tbub[e], peak[e] = tpeak[e], ppos[e] = tpos[e];
    if (moves) moves[*n_moves] = (ref_move){d, chosen, p};
    ++*n_moves;
  }
  free(posB);
  return rc;
}

static int check_problem(const ref_problem* pr) {
  if (!pr) return 0;
  if (pr->L < 1 || pr->L > 255 || pr->P < 1 || pr->P > 64 || pr->v_max < 1 || pr->v_max > 8 ||
      pr->P * pr->v_max > 64 || pr->M < 1 || pr->M > 2047 || pr->max_pert < 0 ||
      pr->max_pert > 255)
    return 0;
  int S_max = pr->P * pr->v_max;
  if (pr->cand_stride < pert_offset(S_max) + 6 * pr->max_pert) return 0;
  return 1;
}

/* ------------------------------------------------------------------------------------------ */
/* Exported: batch evaluation.                                                                 */
/* ------------------------------------------------------------------------------------------ */

typedef struct {
  const ref_problem* pr;
  const int64_t* costs;
  const int64_t* mem;
  const int64_t* link;
  const uint8_t* cands;
  int64_t lo, hi;
  int64_t* out_ms;
  int64_t* out_bub;
  int64_t* out_peak;
  int64_t* out_comm;
  int xfer;
  int64_t* out_bounds;
} batch_job;

static void* batch_worker(void* arg) {
  batch_job* j = (batch_job*)arg;
  for (int64_t i = j->lo; i < j->hi; ++i)
    eval_record(j->pr, j->costs, j->mem, j->link, j->cands + (size_t)i * j->pr->cand_stride,
                j->out_ms + i, j->out_bub + (size_t)i * j->pr->P,
                j->out_peak ? j->out_peak + (size_t)i * j->pr->P : NULL,
                j->out_comm ? j->out_comm + (size_t)i * (j->xfer == 4 ? 2 : 4) : NULL, j->xfer,
                j->out_bounds ? j->out_bounds + (size_t)i * 2 * j->pr->P : NULL);
  return NULL;
}

/* Evaluate n candidate records (host memory). nthreads >= 1 worker threads split the batch.
 * mem (nullable, with out_peak): layer memory [L][2]; out_peak[n][P] = peak bytes per device. */
static int run_batch(const ref_problem* pr, const int64_t* costs, const int64_t* mem,
                     const int64_t* link, const uint8_t* cands, int64_t n, int64_t* out_ms,
                     int64_t* out_bub, int64_t* out_peak, int64_t* out_comm, int xfer,
                     int64_t* out_bounds, int nthreads) {
  if (!check_problem(pr) || n < 0 || (n > 0 && (!costs || !link || !cands || !out_ms || !out_bub)))
    return REF_EINVAL;
  if ((mem == NULL) != (out_peak == NULL)) return REF_EINVAL;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (n < nthreads) nthreads = n > 0 ? (int)n : 1;
  pthread_t th[256];
  batch_job jobs[256];
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = (batch_job){pr,     costs,  mem,     link,    cands, n * t / nthreads,
                          n * (t + 1) / nthreads, out_ms, out_bub, out_peak, out_comm, xfer,
                          out_bounds};
    if (nthreads == 1) batch_worker(&jobs[t]);
    else pthread_create(&th[t], NULL, batch_worker, &jobs[t]);
  }
  if (nthreads > 1)
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  return REF_OK;
}

int oracle_sim_batch_mem(const ref_problem* pr, const int64_t* costs, const int64_t* mem,
                         const int64_t* link, const uint8_t* cands, int64_t n, int64_t* out_ms,
                         int64_t* out_bub, int64_t* out_peak, int nthreads) {
  return run_batch(pr, costs, mem, link, cands, n, out_ms, out_bub, out_peak, NULL, 0, NULL,
                   nthreads);
}

int oracle_sim_batch(const ref_problem* pr, const int64_t* costs, const int64_t* link,
                     const uint8_t* cands, int64_t n, int64_t* out_ms, int64_t* out_bub,
                     int nthreads) {
  return run_batch(pr, costs, NULL, link, cands, n, out_ms, out_bub, NULL, NULL, 0, NULL,
                   nthreads);
}

/* Evaluation with serialised links (see simulate). */
int oracle_sim_batch_serial(const ref_problem* pr, const int64_t* costs, const int64_t* link,
                            const uint8_t* cands, int64_t n, int64_t* out_ms, int64_t* out_bub,
                            int nthreads) {
  return run_batch(pr, costs, NULL, link, cands, n, out_ms, out_bub, NULL, NULL, 1, NULL,
                   nthreads);
}

/* Evaluation with blocking rendezvous transfers in the naive coordination (naive_programs). */
int oracle_sim_batch_rdv(const ref_problem* pr, const int64_t* costs, const int64_t* link,
                         const uint8_t* cands, int64_t n, int64_t* out_ms, int64_t* out_bub,
                         int nthreads) {
  return run_batch(pr, costs, NULL, link, cands, n, out_ms, out_bub, NULL, NULL, 2, NULL,
                   nthreads);
}

/* Evaluation with blocking rendezvous transfers in the reordered coordination (ordered_programs):
 * deadlocks only where the asynchronous schedule itself deadlocks (-1), or with zero-length
 * ops that tie the order. */
int oracle_sim_batch_ordered(const ref_problem* pr, const int64_t* costs, const int64_t* link,
                             const uint8_t* cands, int64_t n, int64_t* out_ms, int64_t* out_bub,
                             int nthreads) {
  return run_batch(pr, costs, NULL, link, cands, n, out_ms, out_bub, NULL, NULL, 3, NULL,
                   nthreads);
}

/* The executor's reordering of the communication (§7's three steps, reorder_programs) evaluated
 * with handshake transfers (simulate_handshake). out_stats (nullable) [n][2] = {transfers,
 * mismatched receives the reordering moved} (sentinels for deadlocked / invalid candidates).
 * Deadlocks (-1) only where the asynchronous schedule itself deadlocks. */
int oracle_sim_batch_reorder(const ref_problem* pr, const int64_t* costs, const int64_t* link,
                             const uint8_t* cands, int64_t n, int64_t* out_ms, int64_t* out_bub,
                             int64_t* out_stats, int nthreads) {
  return run_batch(pr, costs, NULL, link, cands, n, out_ms, out_bub, NULL, out_stats, 4, NULL,
                   nthreads);
}

/* Evaluation plus communication accounting: out_comm[n][4] = {comm nodes, overlappable nodes,
 * comm node time, overlap time} (sentinels for deadlocked / invalid candidates). */
int oracle_sim_batch_comm(const ref_problem* pr, const int64_t* costs, const int64_t* link,
                          const uint8_t* cands, int64_t n, int64_t* out_ms, int64_t* out_bub,
                          int64_t* out_comm, int nthreads) {
  if (n > 0 && !out_comm) return REF_EINVAL;
  return run_batch(pr, costs, NULL, link, cands, n, out_ms, out_bub, NULL, out_comm, 0, NULL,
                   nthreads);
}

/* Evaluation plus each device's first start and last finish: out_bounds[n][P][2] (sentinels for
 * deadlocked / invalid candidates). Leading idle fs_d and trailing idle makespan - lf_d are the
 * device's boundary bubble; the rest of its bubble lies between its ops. */
int oracle_sim_batch_bounds(const ref_problem* pr, const int64_t* costs, const int64_t* link,
                            const uint8_t* cands, int64_t n, int64_t* out_ms, int64_t* out_bub,
                            int64_t* out_bounds, int nthreads) {
  if (n > 0 && !out_bounds) return REF_EINVAL;
  return run_batch(pr, costs, NULL, link, cands, n, out_ms, out_bub, NULL, NULL, 0, out_bounds,
                   nthreads);
}

/* Selective W advancing on a batch of candidate records. Each record's queues (policy, then its
 * perturbations) are repaired with at most max_pert - n_pert advances, which are appended to the
 * record as perturbations (out_cands, same stride; the bytes after the last used perturbation
 * are copied unchanged). out_ms/out_bub/out_peak describe the output record; deadlocked or
 * invalid records are copied unchanged with the sentinels. cap: int64 [P] bytes per device. */
typedef struct {
  const ref_problem* pr;
  const int64_t *costs, *mem, *cap, *link;
  const uint8_t* cands;
  uint8_t* out_cands;
  int64_t lo, hi;
  int64_t *out_ms, *out_bub, *out_peak;
} advance_job;

static void advance_record(const advance_job* j, int64_t i) {
  const ref_problem* pr = j->pr;
  const int P = pr->P;
  const uint8_t* rec = j->cands + (size_t)i * pr->cand_stride;
  uint8_t* out = j->out_cands + (size_t)i * pr->cand_stride;
  int64_t* ms = j->out_ms + i;
  int64_t* bub = j->out_bub + (size_t)i * P;
  int64_t* peak = j->out_peak + (size_t)i * P;
  memmove(out, rec, (size_t)pr->cand_stride);
  ref_cand* c = (ref_cand*)malloc(sizeof(ref_cand));
  decode(pr, out, c);
  int64_t sentinel = 0;
  if (!valid_structure(pr, c)) {
    sentinel = REF_INVALID;
  } else {
    int qcap = 3 * c->v * pr->M;
    ref_op* q = (ref_op*)malloc(sizeof(ref_op) * (size_t)qcap * P);
    int qlen[64];
    if (build_local_queues(pr, c, q, qcap, qlen) != 0 ||
        apply_perturbations(pr, c, q, qcap, qlen) != 0) {
      sentinel = REF_INVALID;
    } else {
      const int room = pr->max_pert - c->n_pert;
      ref_move* mv = (ref_move*)malloc(sizeof(ref_move) * (size_t)(room > 0 ? room : 1));
      int fits, nm;
      int rc = advance_w(pr, c, j->costs, j->mem, j->cap, j->link, q, qcap, qlen, room, ms, bub,
                         peak, &fits, mv, &nm);
      if (rc == SIM_CYCLE) sentinel = REF_DEADLOCK;
      else if (rc != SIM_OK) sentinel = REF_INVALID;
      else {
        uint8_t* pp = out + pert_offset(P * pr->v_max) + 6 * c->n_pert;
        for (int k = 0; k < nm; ++k) {
          const int f[3] = {mv[k].d, mv[k].from, mv[k].to};
          for (int t = 0; t < 3; ++t) pp[6 * k + 2 * t] = (uint8_t)f[t],
                                      pp[6 * k + 2 * t + 1] = (uint8_t)(f[t] >> 8);
        }
        out[2] = (uint8_t)(c->n_pert + nm);
      }
      free(mv);
    }
    free(q);
  }
  if (sentinel != 0) {
    *ms = sentinel;
    for (int d = 0; d < P; ++d) bub[d] = peak[d] = sentinel;
  }
  free(c);
}

static void* advance_worker(void* arg) {
  advance_job* j = (advance_job*)arg;
  for (int64_t i = j->lo; i < j->hi; ++i) advance_record(j, i);
  return NULL;
}

int oracle_advance_w(const ref_problem* pr, const int64_t* costs, const int64_t* mem,
                     const int64_t* cap, const int64_t* link, const uint8_t* cands, int64_t n,
                     uint8_t* out_cands, int64_t* out_ms, int64_t* out_bub, int64_t* out_peak,
                     int nthreads) {
  if (!check_problem(pr) || n < 0 ||
      (n > 0 && (!costs || !mem || !cap || !link || !cands || !out_cands || !out_ms ||
                 !out_bub || !out_peak)))
    return REF_EINVAL;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (n < nthreads) nthreads = n > 0 ? (int)n : 1;
  pthread_t th[256];
  advance_job jobs[256];
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = (advance_job){pr, costs, mem, cap, link, cands, out_cands,
                            n * t / nthreads, n * (t + 1) / nthreads, out_ms, out_bub, out_peak};
    if (nthreads == 1) advance_worker(&jobs[t]);
    else pthread_create(&th[t], NULL, advance_worker, &jobs[t]);
  }
  if (nthreads > 1)
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  return REF_OK;
}

/* Dump the final (perturbed) queues of one candidate in stage terms: ops[d*qcap + i] =
 * (kind, stage, m) packed as kind*2^24 + stage*2^16 + m. Returns the sentinel-style status:
 * 0 ok, REF_INVALID if the candidate is invalid. */
int oracle_dump_queues(const ref_problem* pr, const uint8_t* rec, int32_t* ops, int32_t qcap,
                       int32_t* qlen_out) {
  if (!check_problem(pr)) return REF_EINVAL;
  ref_cand* c = (ref_cand*)malloc(sizeof(ref_cand));
  decode(pr, rec, c);
  int rc = 0;
  if (!valid_structure(pr, c)) {
    rc = REF_INVALID;
  } else {
    int cap = 3 * c->v * pr->M;
    ref_op* q = (ref_op*)malloc(sizeof(ref_op) * (size_t)cap * pr->P);
    int qlen[64];
    if (build_local_queues(pr, c, q, cap, qlen) != 0 || apply_perturbations(pr, c, q, cap, qlen) != 0) {
      rc = REF_INVALID;
    } else {
      for (int d = 0; d < pr->P; ++d) {
        int A[64];
        stages_of(c, d, A);
        qlen_out[d] = qlen[d];
        for (int i = 0; i < qlen[d] && i < qcap; ++i) {
          ref_op o = q[(size_t)d * cap + i];
          ops[d * qcap + i] = (o.kind << 24) | (A[o.chunk] << 16) | o.m;
        }
      }
    }
    free(q);
  }
  free(c);
  return rc;
}

/* Evaluate explicit queues given in stage terms (kind, stage, m) — for pins that build orders
 * by hand. Stage durations are given directly. Returns 0 (ok), 1 (cycle: deadlock) or 2 (the
 * queues are not exactly the op set), or REF_EINVAL for bad arguments. start_out (nullable) gets node-indexed start times
 * (node = (kind*S + s)*M + m); n_cross (nullable) the cross-device data-edge count. */
int oracle_sim_queues(int32_t P, int32_t S, int32_t M, int32_t split, const int32_t* dev,
                      const int64_t* F, const int64_t* B, const int64_t* W, const int64_t* link,
                      const int32_t* ops, const int32_t* qlen, int64_t* makespan, int64_t* bubble,
                      int64_t* start_out, int64_t* n_cross) {
  if (P < 1 || P > 64 || S < 1 || M < 1 || !dev || !F || !B || !W || !link || !ops || !qlen)
    return REF_EINVAL;
  int total = 0;
  int qoff[64];
  for (int d = 0; d < P; ++d) qoff[d] = total, total += qlen[d];
  ref_sop* sq = (ref_sop*)malloc(sizeof(ref_sop) * (size_t)(total > 0 ? total : 1));
  for (int i = 0; i < total; ++i)
    sq[i] = (ref_sop){(ops[i] >> 24) & 0xff, (ops[i] >> 16) & 0xff, ops[i] & 0xffff};
  int dv[64];
  for (int s = 0; s < S && s < 64; ++s) dv[s] = dev[s];
  ref_dag_in g = {S, M, split ? 1 : 0, P, dv, F, B, W, link, 0};
  int rc = simulate(&g, sq, qoff, qlen, makespan, bubble, start_out, n_cross);
  free(sq);
  return rc;
}

/* Ideal start times of the MERGE stage-level pipeline, node-indexed ((kind*S + s)*M + m). */
int oracle_merge_tau(int32_t S, int32_t M, int32_t split, int64_t* tau) {
  if (S < 1 || S > 64 || M < 1 || !tau) return REF_EINVAL;
  return merge_tau(S, M, split ? 1 : 0, tau);
}

/* ------------------------------------------------------------------------------------------ */
/* Philox4x64-10 (Salmon, Moraes, Dror, Shaw, "Parallel random numbers: as easy as 1, 2, 3",    */
/* SC'11): 10 rounds of the 4x64 S-box with the published multipliers and Weyl key constants.   */
/* ------------------------------------------------------------------------------------------ */

static void mulhilo64(uint64_t a, uint64_t b, uint64_t* hi, uint64_t* lo) {
  unsigned __int128 p = (unsigned __int128)a * b;
  *hi = (uint64_t)(p >> 64);
  *lo = (uint64_t)p;
}

void oracle_philox4x64_10(const uint64_t ctr_in[4], const uint64_t key_in[2], uint64_t out[4]) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ULL, M1 = 0xCA5A826395121157ULL;
  const uint64_t W0 = 0x9E3779B97F4A7C15ULL, W1 = 0xBB67AE8584CAA73BULL;
  uint64_t x0 = ctr_in[0], x1 = ctr_in[1], x2 = ctr_in[2], x3 = ctr_in[3];
  uint64_t k0 = key_in[0], k1 = key_in[1];
  for (int round = 0; round < 10; ++round) {
    if (round > 0) k0 += W0, k1 += W1;
    uint64_t hi0, lo0, hi1, lo1;
    mulhilo64(M0, x0, &hi0, &lo0);
    mulhilo64(M1, x2, &hi1, &lo1);
    uint64_t n0 = hi1 ^ x1 ^ k0, n1 = lo1, n2 = hi0 ^ x3 ^ k1, n3 = lo0;
    x0 = n0, x1 = n1, x2 = n2, x3 = n3;
  }
  out[0] = x0, out[1] = x1, out[2] = x2, out[3] = x3;
}

/* ------------------------------------------------------------------------------------------ */
/* Tuner: sequential local search per chain (§6, Algorithm 1's re-simulate-per-move loop, with   */
/* the three move kinds of partitioning, placement and scheduling tuning).                      */
/* ------------------------------------------------------------------------------------------ */

static void write_record(const ref_problem* pr, const ref_cand* c, uint8_t* rec) {
  int S_max = pr->P * pr->v_max;
  for (int s = 1; s < c->S; ++s) rec[4 + s - 1] = (uint8_t)c->b[s];
  for (int s = 0; s < c->S; ++s) rec[3 + S_max + s] = (uint8_t)c->dev[s];
}

typedef struct {
  const ref_problem* pr;
  const int64_t* costs;
  const int64_t* link;
  uint8_t* recs;
  int64_t lo, hi;
  uint64_t seed;
  int n_steps;
  int64_t* out_ms;
  int64_t* out_bub;
  int64_t* out_acc;
  int32_t* out_queues; /* nullable: [chain][P][qcap] packed kind<<14 | chunk<<11 | m */
  const int64_t* ids;  /* nullable: chain index of each record (Philox counter); default i */
  /* memory constraint (all NULL for the plain search) */
  const int64_t* mem; /* layer memory [L][2] */
  const int64_t* cap; /* capacity per device [P] */
  int max_adv;        /* W advances per evaluation */
  int64_t* out_peak;  /* [chain][P] */
} tune_job;

/* Evaluate a chain state. Plain: the simulator. With memory: selective W advancing on the
 * queues (changed in place); *fits tells whether every device ends within its capacity. */
static int tune_eval(const tune_job* j, const ref_cand* c, ref_op* q, int qcap, const int* qlen,
                     int64_t* ms, int64_t* bub, int64_t* peak, int* fits) {
  if (!j->mem) {
    *fits = 1;
    return eval_local(j->pr, c, j->costs, j->link, q, qcap, qlen, NULL, ms, bub, NULL, NULL);
  }
  int nm;
  return advance_w(j->pr, c, j->costs, j->mem, j->cap, j->link, q, qcap, qlen, j->max_adv, ms,
                   bub, peak, fits, NULL, &nm);
}

static void tune_chain(tune_job* j, int64_t ci) {
  const ref_problem* pr = j->pr;
  int P = pr->P;
  uint8_t* rec = j->recs + (size_t)ci * pr->cand_stride;
  int64_t* bub = j->out_bub + (size_t)ci * P;
  int64_t* opk = j->out_peak ? j->out_peak + (size_t)ci * P : NULL;
  ref_cand* c = (ref_cand*)malloc(sizeof(ref_cand));
  decode(pr, rec, c);
  j->out_acc[ci] = 0;
  if (!valid_structure(pr, c) || c->n_pert != 0) {
    j->out_ms[ci] = REF_INVALID;
    for (int d = 0; d < P; ++d) {
      bub[d] = REF_INVALID;
      if (opk) opk[d] = REF_INVALID;
    }
    free(c);
    return;
  }
  int qcap = 3 * c->v * pr->M;
  size_t qbytes = sizeof(ref_op) * (size_t)qcap * P;
  ref_op* q = (ref_op*)malloc(qbytes);
  ref_op* q2 = (ref_op*)malloc(qbytes); /* the proposal's queues */
  int qlen[64];
  build_local_queues(pr, c, q, qcap, qlen);
  /* the current state: its makespan, bubbles, peaks and whether it fits (a deadlocked state
   * counts as +infinity, an over-capacity one as infeasible) */
  int64_t cur_ms, cur_bub[64], cur_peak[64], ms, tb[64], tp[64];
  int cur_fits, fits;
  int rc = tune_eval(j, c, q, qcap, qlen, &cur_ms, cur_bub, cur_peak, &cur_fits);
  if (rc != SIM_OK) {
    cur_ms = rc == SIM_CYCLE ? REF_DEADLOCK : REF_INVALID;
    for (int d = 0; d < P; ++d) cur_bub[d] = cur_peak[d] = cur_ms;
    cur_fits = 0;
  }
  int S = c->S;
  for (int t = 1; t <= j->n_steps; ++t) {
    const uint64_t chain_id = j->ids ? (uint64_t)j->ids[ci] : (uint64_t)ci;
    uint64_t ctr[4] = {chain_id, (uint64_t)t, 0, 0}, key[2] = {j->seed, 0}, u[4];
    oracle_philox4x64_10(ctr, key, u);
    int kind = (int)(u[0] % 3);
    memcpy(q2, q, qbytes);
    /* apply the proposal to the record c (kinds 0, 1) or the queue copy q2 (kind 2) */
    int proposed = 0, saved_b = 0, saved_i = 0, saved_dev[64];
    if (kind == 0) {
      if (S >= 2) {
        int i = 1 + (int)(u[1] % (uint64_t)(S - 1));
        int nb = c->b[i] + ((u[2] & 1) ? 1 : -1);
        if (nb > c->b[i - 1] && nb < c->b[i + 1]) {
          saved_i = i, saved_b = c->b[i];
          c->b[i] = nb;
          proposed = 1;
        }
      }
    } else if (kind == 1) {
      if (P >= 2) {
        int d1 = (int)(u[1] % (uint64_t)P);
        int d2 = (int)((d1 + 1 + (int)(u[2] % (uint64_t)(P - 1))) % P);
        for (int s = 0; s < S; ++s) {
          saved_dev[s] = c->dev[s];
          if (c->dev[s] == d1) c->dev[s] = d2;
          else if (c->dev[s] == d2) c->dev[s] = d1;
        }
        proposed = 1;
      }
    } else {
      int d = (int)(u[1] % (uint64_t)P);
      if (qlen[d] >= 2) {
        int i = (int)(u[2] % (uint64_t)(qlen[d] - 1));
        ref_op* row = q2 + (size_t)d * qcap;
        ref_op tmp = row[i];
        row[i] = row[i + 1];
        row[i + 1] = tmp;
        proposed = 1;
      }
    }
    if (!proposed) continue;
    rc = tune_eval(j, c, q2, qcap, qlen, &ms, tb, tp, &fits);
    const int cur_ok = cur_ms >= 0 && cur_fits;
    if (rc == SIM_OK && fits && (!cur_ok || ms <= cur_ms)) {
      memcpy(q, q2, qbytes);
      cur_ms = ms;
      cur_fits = 1;
      for (int d = 0; d < P; ++d) cur_bub[d] = tb[d], cur_peak[d] = tp[d];
      j->out_acc[ci]++;
    } else if (kind == 0) {
      c->b[saved_i] = saved_b;
    } else if (kind == 1) {
      for (int s = 0; s < S; ++s) c->dev[s] = saved_dev[s];
    }
  }
  j->out_ms[ci] = cur_ms;
  for (int d = 0; d < P; ++d) {
    bub[d] = cur_bub[d];
    if (opk) opk[d] = cur_peak[d];
  }
  write_record(pr, c, rec);
  if (j->out_queues) {
    /* output rows have the queue store's capacity 3 * v_max * M, whatever this chain's v */
    const int ocap = 3 * pr->v_max * pr->M;
    int32_t* oq = j->out_queues + (size_t)ci * P * ocap;
    for (int d = 0; d < P; ++d)
      for (int i = 0; i < ocap; ++i) {
        ref_op o = i < qlen[d] ? q[(size_t)d * qcap + i] : (ref_op){0, 0, 0};
        oq[d * ocap + i] = i < qlen[d] ? ((o.kind << 14) | (o.chunk << 11) | o.m) : 0;
      }
  }
  free(q2);
  free(q);
  free(c);
}

static void* tune_worker(void* arg) {
  tune_job* j = (tune_job*)arg;
  for (int64_t i = j->lo; i < j->hi; ++i) tune_chain(j, i);
  return NULL;
}

/* Run steps 0..n_steps of the local search for n chains. recs (in/out) holds the chain
 * candidate records (updated to the final state); chain_ids (nullable) gives each record's chain
 * index for the Philox counter (default: its position). Outputs per chain: final makespan,
 * bubbles, accepted-move count, and optionally the final queues (qcap = 3*v_max*M entries per
 * device). With mem (layer memory [L][2]) and cap (bytes per device [P]), every evaluation
 * runs selective W advancing (at most max_adv advances) and a state counts as feasible only if
 * every device's peak fits; a proposal is kept iff feasible and (the current state is not, or
 * its makespan is not larger); out_peak[n][P] receives the final peaks. */
int oracle_tune_mem(const ref_problem* pr, const int64_t* costs, const int64_t* mem,
                    const int64_t* cap, int32_t max_adv, const int64_t* link, uint8_t* recs,
                    int64_t n, uint64_t seed, int32_t n_steps, int64_t* out_ms, int64_t* out_bub,
                    int64_t* out_peak, int64_t* out_acc, int32_t* out_queues,
                    const int64_t* chain_ids, int nthreads) {
  if (!check_problem(pr) || n < 0 || n_steps < 0) return REF_EINVAL;
  if (mem && (!cap || !out_peak || max_adv < 0)) return REF_EINVAL;
  if (nthreads < 1) nthreads = 1;
  if (nthreads > 256) nthreads = 256;
  if (n < nthreads) nthreads = n > 0 ? (int)n : 1;
  pthread_t th[256];
  tune_job jobs[256];
  for (int t = 0; t < nthreads; ++t) {
    jobs[t] = (tune_job){pr,       costs,      link,      recs,     n * t / nthreads,
                         n * (t + 1) / nthreads, seed, n_steps,   out_ms,   out_bub,
                         out_acc,  out_queues, chain_ids, mem,      mem ? cap : NULL,
                         max_adv,  mem ? out_peak : NULL};
    if (nthreads == 1) tune_worker(&jobs[t]);
    else pthread_create(&th[t], NULL, tune_worker, &jobs[t]);
  }
  if (nthreads > 1)
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
  return REF_OK;
}

int oracle_tune(const ref_problem* pr, const int64_t* costs, const int64_t* link, uint8_t* recs,
                int64_t n, uint64_t seed, int32_t n_steps, int64_t* out_ms, int64_t* out_bub,
                int64_t* out_acc, int32_t* out_queues, const int64_t* chain_ids, int nthreads) {
  return oracle_tune_mem(pr, costs, NULL, NULL, 0, link, recs, n, seed, n_steps, out_ms, out_bub,
                         NULL, out_acc, out_queues, chain_ids, nthreads);
}
