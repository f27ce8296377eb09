// octo_sim.hpp — the max-plus relaxation core: one wave simulates CPW candidates at once, G
// lanes per candidate, lane d = pipeline device d. Each candidate owns a finish table in LDS
// with one slot per (stage, micro-batch ring position).
//
// Slot value = fin << 3 | state, state bits: 1 = B(s,m) finished, 2 = F(s,m) finished (kept
// after B), 4 = parity of the occupant's micro-batch round m / R; empty = 0. One slot per (s,m)
// suffices because B(s,m) can only finish after F(s+1,m) (which consumed F(s,m)) has finished:
// B(s,m) needs B(s+1,m), which needs F(s+1,m).
//
// Every op reads exactly one slot and needs one state bit there (and the parity of its own m):
//   F(0,m): its own slot, always ready, weight 0: the slot is empty, or (ring rows) holds the
//   backward of m - R, which the same device ran earlier, so in <= the device clock;
//   F(s,m), s > 0: row s-1, bit 2; in = fin + link weight.
//   B(s,m), s < S-1: row s+1, bit 1; in = fin + link weight.
//   B(S-1,m): its own slot, bit 2 (the loss turns the forward around).
//   W(s,m): its own slot, bit 1; W writes nothing.
// Other dependencies are implied: F(s,m) -> B(s,m) for s < S-1 follows from F(s,m) ->
// F(s+1,m) -> B(s+1,m) -> B(s,m). start = max(device clock, in); fin = start + duration
// (§5: record start/end per node; §6 Eq. 1: makespan = latest finish).
//
// Ring rows: micro-batch m of stage s lives in slot s R + (m mod R). This is exact whenever no
// stage ever has more than R micro-batches in flight on its device (forwards issued minus
// backwards, and minus weight-gradient ops when split): then B(s,m) and W(s,m) precede
// F(s,m+R) in the device's queue, every reader of (s,m) — F(s+1,m), B(s-1,m), B(S-1,m) and
// W(s,m) — precedes F(s,m+R) in the graph, so it has read the slot in an earlier round than the
// overwrite; and a reader that finds the previous occupant m-R (never an older one) tells it
// apart by the parity bit. R = M (no wrap) is the plain table.
//
// Rounds: every live lane tries its head op once per round; readiness is structural, so when
// no lane of the wave advances in a round, every candidate that still has work is deadlocked.
// The round body is straight-line code: generators and descriptors advance under a predicate.
#pragma once

#include <type_traits>

#include "octo_device.hpp"

namespace octo {

constexpr uint32_t ST_B = 1, ST_F = 2, ST_PAR = 4;

// What an evaluation computes besides the plain times: the memory model (activation bytes held
// per device, §5 memory nodes), communication nodes and their overlap (§5), or times with
// serialised links (a directed link carries one transfer at a time, in issue order), or each
// device's first start and last finish (its leading and trailing idle).
// XR: blocking rendezvous transfers (a device receives an op's cross-device input right before
// the op and sends its cross-device output right after it; a transfer holds both devices).
// XT: the plain times, each op's finish recorded by node id (L.tb) for building programs.
constexpr int XP = 0, XM = 1, XC = 2, XS = 3, XB = 4, XR = 5, XT = 6;
// Weight of a weight-gradient op's read under serialised links: its B is on its own device and
// earlier in its queue, so only the readiness bit matters, not the (possibly delayed) slot time.
constexpr int64_t W_NO_TIME = -((int64_t)1 << 50);
// Communication flags of an op: its input comes from another device / its output goes to one.
constexpr int CX_IN = 1, CX_OUT = 2;

// Ring geometry of one finish table: R slots per stage row, slot of m = m & mask, parity
// (m >> lg) & 1. Without wrap (R = M): mask = all ones, lg = 30.
struct Ring {
  int R, mask, lg;
};
__host__ __device__ __forceinline__ Ring make_ring(int M, int R) {
  Ring r;
  if (R >= M) {
    r.R = M, r.mask = 0x7FFFFFFF, r.lg = 30;
  } else {
    int lg = 0;
    while ((1 << lg) < R) ++lg;
    r.R = 1 << lg, r.mask = r.R - 1, r.lg = lg;
  }
  return r;
}

// 64-bit slots: one int64 per (stage, micro-batch).
struct Table64 {
  int64_t* T;
  __device__ __forceinline__ void issue(int i, uint32_t& l, uint32_t& h) const {
    const uint64_t x = (uint64_t)T[i];
    l = (uint32_t)x;
    h = (uint32_t)(x >> 32);
  }
  __device__ __forceinline__ uint64_t load(int i) const { return (uint64_t)T[i]; }
  __device__ __forceinline__ void store(int i, uint64_t v) const { T[i] = (int64_t)v; }
  __device__ __forceinline__ void clear(int n, int d, int G) const {
    for (int i = d; i < n; i += G) T[i] = 0;
  }
  __host__ __device__ static size_t bytes(int slots) { return (size_t)slots * 8; }
};

// 40-bit slots: a 32-bit low array and an 8-bit high array (fin < 2^37 ns; larger times are
// detected and the candidate is recomputed with 64-bit slots). The CPW candidates of a wave
// (a power of two, 2^lg) share the arrays interleaved — slot i of group g lives at
// i * CPW + g — so that groups running the same op pattern in lockstep touch consecutive banks.
struct Table40 {
  uint32_t* lo;
  uint8_t* hi;
  int lg, g;
  __device__ __forceinline__ void issue(int i, uint32_t& l, uint32_t& h) const {
    const int j = (i << lg) | g;
    l = lo[j];
    h = hi[j];
  }
  __device__ __forceinline__ uint64_t load(int i) const {
    uint32_t l, h;
    issue(i, l, h);
    return (uint64_t)l | ((uint64_t)h << 32);
  }
  __device__ __forceinline__ void store(int i, uint64_t v) const {
    const int j = (i << lg) | g;
    lo[j] = (uint32_t)v;
    hi[j] = (uint8_t)(v >> 32);
  }
  // Clear n slots of this group (its G lanes together).
  __device__ __forceinline__ void clear(int n, int d, int G) const {
    for (int i = d; i < n; i += G) {
      const int j = (i << lg) | g;
      lo[j] = 0;
      hi[j] = 0;
    }
  }
  // Clear n slots of every group (all lanes of the wave together), 16 bytes per store; the
  // arrays start 16-byte aligned and a plan rounds both up to 16 bytes.
  __device__ __forceinline__ void clear_all(int n, int lane, int nlanes) const {
    const int tot = n << lg;
    uint4* l4 = reinterpret_cast<uint4*>(lo);
    for (int j = lane; j < (tot + 3) / 4; j += nlanes) l4[j] = make_uint4(0, 0, 0, 0);
    uint4* h4 = reinterpret_cast<uint4*>(hi);
    for (int j = lane; j < (tot + 15) / 16; j += nlanes) h4[j] = make_uint4(0, 0, 0, 0);
  }
  static constexpr int64_t LIMIT = (int64_t)1 << 37;
};

template <int VMAX>
struct Chunks {
  int st[VMAX];                      // stage of chunk k
  int base[VMAX];                    // first slot of the stage's own row: s R
  int frow[VMAX];                    // forward read row offset (-R; stage 0: its own row)
  int fmask[VMAX];                   // state bits a forward needs (0: always ready)
  int brow[VMAX], bmask[VMAX];       // backward read row offset / needed state bits
  int64_t dF[VMAX], dB[VMAX], dW[VMAX], wF[VMAX], wB[VMAX];
  int64_t mA[VMAX];                  // activation bytes of the stage per micro-batch
  int64_t cF[VMAX], cB[VMAX];        // transfer time of the forward's / backward's output
  int xF[VMAX], xB[VMAX];            // CX_IN | CX_OUT of the forward / backward
  int dnF[VMAX], dnB[VMAX];          // device the forward's / backward's output goes to
  int64_t wW;                        // weight of a weight-gradient op's read
  int split;                         // backward split into B and W
};

// Descriptor of one op: slot read, slot written, readiness test (slot & mask) == want, edge
// weight, duration.
struct Desc {
  int rd, wr, mask, want, store;
  uint32_t state;  // state bits written on finish
  int64_t w, dur;
  int64_t dm;      // activation bytes the op allocates (> 0) or releases (< 0)
  int64_t cout;    // transfer time of the op's output to another device
  int cx;          // CX_IN | CX_OUT
  int dst;         // device the op's output goes to (XR: the device its input comes from)
  __device__ __forceinline__ void take_if(bool t, const Desc& o) {
    dm = t ? o.dm : dm;
    cout = t ? o.cout : cout;
    cx = t ? o.cx : cx;
    dst = t ? o.dst : dst;
    rd = t ? o.rd : rd;
    wr = t ? o.wr : wr;
    mask = t ? o.mask : mask;
    want = t ? o.want : want;
    store = t ? o.store : store;
    state = t ? o.state : state;
    w = t ? o.w : w;
    dur = t ? o.dur : dur;
  }
};

// Communication tally of one device (XC): nodes and overlappable nodes, their time and the
// overlap time; the last op's start and the end of its outgoing transfer (-1: none).
// §5: a send or receive node is overlappable when the computation that can run beside it —
// for a send the op after its producer, for a receive the op before its consumer (the
// consumer itself waits for the data) — runs during the transfer; its overlap time is then the
// smaller of that computation's and the transfer's durations.
struct CommTally {
  int n, nov;
  int64_t t, tov, pst, pend;
  __device__ __forceinline__ void reset() { n = nov = 0, t = tov = 0, pst = 0, pend = -1; }
  // An op ran over [st, fin] after a device clock `clock` (the previous op's end, which ran
  // from pst); its input arrived at tin after a transfer of w (cx & CX_IN); its output leaves
  // for cout (cx & CX_OUT); the previous op's output transfer ends at pend, having left at
  // `clock`.
  __device__ __forceinline__ void op(bool ok, int cx, int64_t tin, int64_t w, int64_t clock,
                                     int64_t st, int64_t fin, int64_t cout) {
    const bool rin = ok && (cx & CX_IN);
    const int64_t rlo = pst > tin - w ? pst : tin - w, rhi = clock < tin ? clock : tin;
    const bool rov = rin && rhi > rlo;
    const int64_t shi = fin < pend ? fin : pend;
    const bool sov = ok && shi > st;
    const bool sout = ok && (cx & CX_OUT);
    const int64_t rcomp = clock - pst, scomp = fin - st, scomm = pend - clock;
    n += (rin ? 1 : 0) + (sout ? 1 : 0);
    t += (rin ? w : 0) + (sout ? cout : 0);
    nov += (rov ? 1 : 0) + (sov ? 1 : 0);
    tov += (rov ? (rcomp < w ? rcomp : w) : 0) + (sov ? (scomp < scomm ? scomp : scomm) : 0);
    pend = ok ? (sout ? fin + cout : -1) : pend;
    pst = ok ? st : pst;
  }
};

struct Lane : Desc {
  int64_t clock;
  int pos, nops;
  int64_t mem, peak;  // activation bytes held now / at most (memory-model variants)
  CommTally cm;       // communication variants
  int64_t lf[16];     // serialised links: when the link to device dst is free, per stream
                      // (forward outputs of chunk k at k, backward outputs at VMAX + k)
  int64_t fs;         // start of the device's first op (-1 before it), bounds variants
  int64_t* tb;        // XT: finish time of every op, at (kind * tS + stage) * tM + m
  int64_t* ts;        // XT (nullable): start time of every op, same index
  int32_t* tl;        // XT (nullable): the round each op ran in — its level, the number of ops on the
                      // longest dependency chain before it (queue order included)
  int tS, tM, rnd;
};

// Entry k of a per-chunk array: a select chain while the arrays stay in registers (v <= 2);
// the eight-chunk arrays live in private memory, where one indexed load beats reading all eight.
template <int VMAX, typename T>
__device__ __forceinline__ T pick(const T (&a)[VMAX], int k) {
  if constexpr (VMAX > 2) {
    return a[k];
  } else {
    T x = a[0];
#pragma unroll
    for (int i = 1; i < VMAX; ++i) x = k == i ? a[i] : x;
    return x;
  }
}

// Describe op (kind, chunk k, micro-batch m).
template <int VMAX>
__device__ __forceinline__ void describe(Desc& L, const Chunks<VMAX>& c, const Ring& ring,
                                         int kind, int k, int m) {
  const bool isF = kind == KF, isB = kind == KB;
  const int own = pick<VMAX>(c.base, k) + (m & ring.mask);
  const uint32_t par = ((uint32_t)m >> ring.lg) & 1u;
  const int fm = pick<VMAX>(c.fmask, k), bm = pick<VMAX>(c.bmask, k);
  const int fr = pick<VMAX>(c.frow, k), br = pick<VMAX>(c.brow, k);
  L.rd = own + (isF ? fr : isB ? br : 0);
  L.wr = own;
  L.store = isF || isB;
  L.mask = isF ? fm : isB ? bm : (int)(ST_B | ST_PAR);
  L.want = L.mask & (int)(par ? (ST_B | ST_F | ST_PAR) : (ST_B | ST_F));
  L.state = (isF ? ST_F : (ST_F | ST_B)) | (par << 2);
  const int64_t wf = pick<VMAX>(c.wF, k), wb = pick<VMAX>(c.wB, k);
  const int64_t df = pick<VMAX>(c.dF, k), db = pick<VMAX>(c.dB, k), dw = pick<VMAX>(c.dW, k);
  L.w = isF ? wf : isB ? wb : c.wW;
  L.dur = isF ? df : isB ? db : dw;
  // memory nodes: a forward allocates its stage's activations, the last backward op of the
  // micro-batch (B fused, W split) releases them
  const int64_t a = pick<VMAX>(c.mA, k);
  L.dm = isF ? a : (isB && c.split) ? 0 : -a;
  L.cout = isF ? pick<VMAX>(c.cF, k) : isB ? pick<VMAX>(c.cB, k) : 0;
  L.cx = isF ? pick<VMAX>(c.xF, k) : isB ? pick<VMAX>(c.xB, k) : 0;
  L.dst = isF ? pick<VMAX>(c.dnF, k) : isB ? pick<VMAX>(c.dnB, k) : -1;
}

// Fold every G-lane group of a 64-bit lane mask into the group's lowest bit.
__device__ __forceinline__ uint64_t fold_groups(uint64_t x, int G, uint64_t lsb) {
  for (int sh = 1; sh < G; sh <<= 1) x |= x >> sh;
  return x & lsb;
}

// Run the rounds until every candidate of the wave is done or deadlocked.
// gbit: this lane's group bit in folded masks; lsb: all group bits. rec (nullable): ideal-start
// recording for the MERGE table, rec[pos] = start << 16 | kind << 12 | m.
// SPEC: compute the next op and its descriptor while the slot read is in flight and keep them
// only if this op completes (pays when one wave per SIMD must hide the LDS latency itself);
// otherwise advance and describe after the readiness test (fewer instructions per round, the
// latency hidden by other waves).
// X: XM also tracks the activation bytes each device holds (L.mem) and their maximum
// (L.peak); XC tallies communication nodes and their overlap (L.cm).
// Queue-generator steps of one round. Generators ignore the round's slot U; GenMatK reads and
// refills its buffer U.
template <int U, class Gen>
__device__ __forceinline__ void gen_advance(Gen& g, bool ok) { g.advance(ok); }
template <int U, class Gen>
__device__ __forceinline__ void gen_take(Gen& g, bool t, const Gen& o) { g.take_if(t, o); }
template <int U, int K>
__device__ __forceinline__ void gen_advance(GenMatK<K>& g, bool ok) { g.template advance<U>(ok); }
template <int U, int K>
__device__ __forceinline__ void gen_take(GenMatK<K>& g, bool t, const GenMatK<K>& o) {
  g.template take_if<U>(t, o);
}

// One round of relax (U: the round's slot for generators that keep per-round buffers). Returns
// false once the wave has settled.
template <int VMAX, bool SPEC, int X, int U, class Tab, class Gen>
__device__ __forceinline__ bool relax_round(Gen& gen, const Chunks<VMAX>& c, const Ring& ring,
                                            Lane& L, const Tab& T, int G, uint64_t gbit,
                                            uint64_t lsb, bool& dead, uint32_t* rec, bool& live) {
  {
    uint32_t plo, phi;
    T.issue(live ? L.rd : 0, plo, phi);
    Gen g2 = gen;
    Desc d2;
    if constexpr (SPEC) {
      // the next op, computed while the read is in flight; kept only if this op completes
      gen_advance<U>(g2, true);
      describe<VMAX>(d2, c, ring, g2.kind, g2.k, g2.m);
      // the slot is consumed only after the next op's descriptor exists
      __asm__ volatile("" : "+v"(plo), "+v"(phi), "+v"(d2.rd), "+v"(d2.want), "+v"(d2.dur));
    }
    const uint64_t p = (uint64_t)plo | ((uint64_t)phi << 32);
    const bool ok = live && (plo & (uint32_t)L.mask) == (uint32_t)L.want;
    const int64_t tin = (int64_t)(p >> 3) + L.w;
    const int64_t st = tin > L.clock ? tin : L.clock;
    const int64_t fin = st + L.dur;
    int64_t put = fin;  // the time its readers see
    if constexpr (X == XS) {
      // the output's transfer queues on the link to its consumer's device: it leaves when both
      // the op and the link's previous transfer are done; the slot holds its arrival. Every
      // stream to the same device shares the link's free time.
      const bool out = ok && (L.cx & CX_OUT);
      const bool isF = gen.kind == KF;
      int64_t fr = 0;
#pragma unroll
      for (int k = 0; k < VMAX; ++k) fr = gen.k == k ? (isF ? L.lf[k] : L.lf[VMAX + k]) : fr;
      const int64_t arr = (fin > fr ? fin : fr) + L.cout;
#pragma unroll
      for (int k = 0; k < VMAX; ++k) {
        L.lf[k] = (out && c.dnF[k] == L.dst) ? arr : L.lf[k];
        L.lf[VMAX + k] = (out && c.dnB[k] == L.dst) ? arr : L.lf[VMAX + k];
      }
      put = (L.cx & CX_OUT) ? arr : fin;
    }
    if (ok && L.store) T.store(L.wr, ((uint64_t)put << 3) | L.state);
    if (rec && ok)
      rec[L.pos] = ((uint32_t)st << 16) | ((uint32_t)gen.kind << 12) | (uint32_t)gen.m;
    if constexpr (X == XC) L.cm.op(ok, L.cx, tin, L.w, L.clock, st, fin, L.cout);
    if constexpr (X == XB) L.fs = (ok && L.fs < 0) ? st : L.fs;
    if constexpr (X == XT) {
      const int nd = (gen.kind * L.tS + pick<VMAX>(c.st, gen.k)) * L.tM + gen.m;
      if (ok) {
        L.tb[nd] = fin;
        if (L.ts) L.ts[nd] = st;
        if (L.tl) L.tl[nd] = L.rnd;
      }
      L.rnd += 1;
    }
    L.clock = ok ? fin : L.clock;
    if constexpr (X == XM) {
      L.mem = ok ? L.mem + L.dm : L.mem;
      L.peak = L.mem > L.peak ? L.mem : L.peak;
    }
    L.pos += ok ? 1 : 0;
    live = L.pos < L.nops;
    if constexpr (SPEC) {
      gen_take<U>(gen, ok, g2);
      L.take_if(ok, d2);
    } else {
      gen_advance<U>(gen, ok);
      describe<VMAX>(L, c, ring, gen.kind, gen.k, gen.m);
    }
    __asm__ volatile("" ::: "memory");
    if (__ballot(ok) == 0) {
      const uint64_t actm = __ballot(live);
      if (actm != 0 && (fold_groups(actm, G, lsb) & gbit)) dead = true;
      return false;
    }
  }
  return true;
}

template <int VMAX, bool SPEC, int X, class Tab, class Gen>
__device__ __forceinline__ void relax(Gen& gen, const Chunks<VMAX>& c, const Ring& ring, Lane& L,
                                      const Tab& T, int G, uint64_t gbit, uint64_t lsb,
                                      bool& dead, uint32_t* rec) {
  bool live = L.pos < L.nops;
  while (relax_round<VMAX, SPEC, X, 0>(gen, c, ring, L, T, G, gbit, lsb, dead, rec, live)) {
  }
}

// relax over a queue read K rounds ahead (GenMatK): the loop is unrolled K times so that each
// round's buffer is fixed registers, and it leaves only after a whole group of K rounds (a round
// after the wave has settled changes nothing: no lane is ready, and the deadlock test gives the
// same answer), so the loop has one exit and the load of each buffer is awaited only K rounds
// after it was issued.
template <int VMAX, int X, int K, int U, class Tab>
__device__ __forceinline__ bool rounds_k(GenMatK<K>& gen, const Chunks<VMAX>& c, const Ring& ring,
                                         Lane& L, const Tab& T, int G, uint64_t gbit,
                                         uint64_t lsb, bool& dead, bool& live) {
  const bool go =
      relax_round<VMAX, true, X, U>(gen, c, ring, L, T, G, gbit, lsb, dead, nullptr, live);
  if constexpr (U + 1 < K) {
    const bool more = rounds_k<VMAX, X, K, U + 1>(gen, c, ring, L, T, G, gbit, lsb, dead, live);
    return go && more;
  } else {
    return go;
  }
}

template <int VMAX, int X, int K, class Tab>
__device__ __forceinline__ void relax_k(GenMatK<K>& gen, const Chunks<VMAX>& c, const Ring& ring,
                                        Lane& L, const Tab& T, int G, uint64_t gbit, uint64_t lsb,
                                        bool& dead) {
  bool live = L.pos < L.nops;
  while (rounds_k<VMAX, X, K, 0>(gen, c, ring, L, T, G, gbit, lsb, dead, live)) {
  }
}

// Blocking rendezvous transfers (XR). Per op a lane takes up to three steps: receive, when the
// op's input comes from another device — ready once the producer's slot shows it finished; the
// transfer runs from max(producer's finish, this device's clock) for the link time, this
// device's clock moves to its end, and the end goes to the producer's mailbox; compute, as in
// relax (in the same round as the receive); send, when the op's output goes to another device —
// the lane waits until its mailbox holds the transfer's end (posted by the receiver), takes it as
// its clock and clears the box. A producer reaches its send in the round it finishes the op, so
// the receiver (which reads the slot in a later round) always posts to a waiting sender, and
// each box has one writer at a time. mbox: one int64 per lane of the wave (RDV_EMPTY = nothing posted), set to RDV_EMPTY by
// the caller. A round in which no lane of the wave takes a step changes nothing, so every group
// with work left is deadlocked.
// GPipe queues (GenAfab) skip the readiness test of an input from the own device: such a
// producer always comes earlier in the queue (forwards by ascending stage, backwards by
// descending stage, all forwards first), so it has finished and the device clock covers it.
// Every other input crosses devices and is received while its producer waits at the send, so
// the producer writes its stage row again only after the value was taken, and a consumer wants
// micro-batch m only after taking m - 1 from the same row: one slot per stage, with the parity
// of m, is exact for any M.
constexpr int64_t RDV_EMPTY = -1;
template <int VMAX, class Tab, class Gen>
__device__ __forceinline__ void relax_rdv(Gen& gen, const Chunks<VMAX>& c, const Ring& ring,
                                          Lane& L, const Tab& T, int G, uint64_t gbit,
                                          uint64_t lsb, bool& dead, int64_t* mbox) {
  constexpr bool LOCAL = std::is_same<Gen, GenAfab>::value;
  const int me = (int)(threadIdx.x & 63);
  const int g0 = me - me % G;  // the group's first lane
  bool live = L.pos < L.nops;
  int step = (live && (L.cx & CX_IN)) ? 0 : 1;  // 0 receive, 1 compute, 2 send
  for (;;) {
    uint32_t plo, phi;
    T.issue(live ? L.rd : 0, plo, phi);
    const uint64_t p = (uint64_t)plo | ((uint64_t)phi << 32);
    const bool rdy = live && (plo & (uint32_t)L.mask) == (uint32_t)L.want;
    const int64_t tx = (int64_t)(p >> 3);
    const bool okR = step == 0 && rdy;
    const int64_t xend = (tx > L.clock ? tx : L.clock) + L.w;
    // a receive takes its op's compute in the same round: the input slot stays ready (it is
    // rewritten only after this consumer's own backward), and the op starts at the transfer's
    // end, which is at least tin
    const bool okC = (step == 1 && (LOCAL ? live : rdy)) || okR;
    const int64_t c0 = okR ? xend : L.clock;
    const int64_t tin = tx + L.w;
    const int64_t st = tin > c0 ? tin : c0;
    const int64_t fin = st + L.dur;
    if (okR) mbox[g0 + L.dst] = xend;
    __asm__ volatile("" ::: "memory");
    // the mailbox is read after this round's posts, so a send completes in the round its
    // receiver posts (a lane that computes this round cannot be posted to before the next one:
    // its receiver sees the slot only then)
    const int64_t box = mbox[me];
    const bool okS = step == 2 && box != RDV_EMPTY;
    if (okC && L.store) T.store(L.wr, ((uint64_t)fin << 3) | L.state);
    if (okS) mbox[me] = RDV_EMPTY;
    L.clock = okC ? fin : okS ? box : L.clock;
    const bool sends = (L.cx & CX_OUT) != 0;
    const bool done = (okC && !sends) || okS;
    step = (okC && sends) ? 2 : step;
    L.pos += done ? 1 : 0;
    live = L.pos < L.nops;
    gen.advance(done);
    describe<VMAX>(L, c, ring, gen.kind, gen.k, gen.m);
    step = done ? ((live && (L.cx & CX_IN)) ? 0 : 1) : step;
    __asm__ volatile("" ::: "memory");
    if (__ballot(okR || okC || okS) == 0) {
      const uint64_t actm = __ballot(live);
      if (actm != 0 && (fold_groups(actm, G, lsb) & gbit)) dead = true;
      break;
    }
  }
}

// The rounds of one evaluation: relax, or relax_rdv for rendezvous transfers (mbox: its
// mailboxes, unused otherwise).
template <int VMAX, bool SPEC, int X, class Tab, class Gen>
__device__ __forceinline__ void rounds(Gen& gen, const Chunks<VMAX>& c, const Ring& ring, Lane& L,
                                       const Tab& T, int G, uint64_t gbit, uint64_t lsb,
                                       bool& dead, int64_t* mbox) {
  if constexpr (X == XR)
    relax_rdv<VMAX>(gen, c, ring, L, T, G, gbit, lsb, dead, mbox);
  else
    relax<VMAX, SPEC, X>(gen, c, ring, L, T, G, gbit, lsb, dead, nullptr);
}

// ------------------------------------------------------------------------------------------
// Table-driven rounds. A queue-table row is a device queue for one stage set (its stages in
// ascending order), each op pre-encoded in 32 bits, for one launch geometry (ring R,
// CPW = 2^lg candidates per wave), with everything that does not depend on the candidate:
//   bits 0-14 read slot << lg | 15-16 write row relative to the read row, + 1 (the write slot
//   is read slot + (code - 1) RS << lg) | 17-19 state bits needed (B, F, parity) | 20-22 their
//   wanted values | 23-25 state bits written, parity included (0 = writes nothing) |
//   26-28 stream e = kind * v + chunk.
// The candidate's per-stream input weight and duration (32-bit) sit in LDS, 64 lanes
// interleaved: the pair of lane l for stream e at byte e * 512 + l * 8 (memory-model variants:
// 16-byte records {w, dur, activation delta} at e * 1024 + l * 16).
// ------------------------------------------------------------------------------------------
// Rows are RS = R + 5 slots apart: with rows of R slots (R and the interleave are powers of
// two) the same micro-batch of every stage falls in one LDS bank, and the lanes of a group
// often touch one micro-batch in several stages in the same round. Measured on the P = 8,
// M = 64 batch's generated v = 2 queues (ms per call of that kernel): R 0.452, R + 1 0.407,
// R + 3 0.394, R + 5 0.390, R + 7 0.390, R + 9 0.400.
__host__ __device__ __forceinline__ int qt_row_stride(const Ring& ring) { return ring.R + 5; }
__host__ __device__ __forceinline__ uint32_t qt_entry(int kind, int k, int m, int v, int s,
                                                      int S, const Ring& ring, int lg) {
  int rdrow, need, wst;
  if (kind == KF) {
    rdrow = s > 0 ? s - 1 : s;  // stage 0 reads its own slot, always ready (see relax_tab)
    need = s > 0 ? (int)(ST_F | ST_PAR) : 0;
    wst = ST_F;
  } else if (kind == KB) {
    rdrow = s < S - 1 ? s + 1 : s;
    need = (int)((s < S - 1 ? ST_B : ST_F) | ST_PAR);
    wst = ST_F | ST_B;
  } else {
    rdrow = s;
    need = (int)(ST_B | ST_PAR);
    wst = 0;
  }
  const int mr = m & ring.mask;
  const int par = (m >> ring.lg) & 1;
  const uint32_t rd = (uint32_t)(rdrow * qt_row_stride(ring) + mr) << lg;
  const uint32_t code = (uint32_t)(s - rdrow + 1);
  const int want = need & (par ? (int)(ST_B | ST_F | ST_PAR) : (int)(ST_B | ST_F));
  const int state = wst ? (wst | (par << 2)) : 0;
  return rd | code << 15 | (uint32_t)need << 17 | (uint32_t)want << 20 | (uint32_t)state << 23 |
         (uint32_t)(kind * v + k) << 26;
}

// Row terminator: needs nothing but wants a bit that is never there, so it is never ready.
constexpr uint32_t QT_END = 1u << 20;

// Rounds over one queue-table row starting at entry `row`; every row is followed by two
// QT_END entries (and the table by two more), so a lane that has run its last op stays on a
// terminator, and an idle lane starts on one. A stage-0 forward reads its own slot and needs
// nothing: the slot is empty or holds the backward of micro-batch m - R, which this device has
// already run, so its time never exceeds the device clock. Each round decodes its op first, so
// the stream read and the slot read are in flight together, and loads the entry after next at
// its start, to be taken at the end of the next round. Rl = RS << lg. XM: streams are 16-byte records
// {w, dur, activation delta}; mem / peak track the activation bytes held. XC: 16-byte records
// {w, dur, output transfer time, CX flags}; cm tallies the communication nodes.
template <int X>
__device__ __forceinline__ void relax_tab(const uint32_t* __restrict__ qt, uint32_t row, int Rl,
                                          const uint8_t* strm, int64_t& clock, const Table40& T,
                                          int G, uint64_t gbit, uint64_t lsb, bool& dead,
                                          int64_t& mem, int64_t& peak, CommTally& cm,
                                          int64_t& fs) {
  uint32_t cur = qt[row], nxt = qt[row + 1u];
  // byte offset of the entry after next (32 bits: the load takes the table's address as its
  // scalar base and this offset as its only per-lane address)
  uint32_t qb = (row + 2u) * 4u;
  const char* qtb = reinterpret_cast<const char*>(qt);
  bool okp = false;  // whether the previous round completed its op
  // One round: `prev` is the previous round's load of the entry after next, which becomes the
  // next entry if that round completed its op; `ahead` receives this round's load. Returns
  // whether any lane of the wave completed an op.
  auto round = [&](uint32_t prev, uint32_t& ahead) -> bool {
    ahead = *reinterpret_cast<const uint32_t*>(qtb + qb);
    const int rdj = (int)(cur & 0x7FFFu) | T.g;
    const int wrj = rdj + __mul24((int)((cur >> 15) & 3u), Rl) - Rl;
    const uint32_t mask = (cur >> 17) & 7u, want = (cur >> 20) & 7u, state = (cur >> 23) & 7u;
    const uint32_t soff = X != XP ? ((cur >> 16) & 0x1C00u) : ((cur >> 17) & 0xE00u);
    const uint2 wd = *reinterpret_cast<const uint2*>(strm + soff);
    const uint32_t plo = T.lo[rdj], phi = T.hi[rdj];
    const uint64_t p = (uint64_t)plo | ((uint64_t)phi << 32);
    const bool ok = (plo & mask) == want;
    const int64_t tin = (int64_t)(p >> 3) + (int64_t)wd.x;
    const int64_t st = tin > clock ? tin : clock;
    const int64_t fin = st + (int64_t)wd.y;
    if (ok && state != 0) {
      T.lo[wrj] = (uint32_t)(((uint64_t)fin << 3) | state);
      T.hi[wrj] = (uint8_t)((uint64_t)fin >> 29);
    }
    if constexpr (X == XC) {
      const uint2 cc = *reinterpret_cast<const uint2*>(strm + soff + 8);
      cm.op(ok, (int)cc.y, tin, (int64_t)wd.x, clock, st, fin, (int64_t)cc.x);
    }
    if constexpr (X == XB) fs = (ok && fs < 0) ? st : fs;
    clock = ok ? fin : clock;
    if constexpr (X == XM) {
      const int64_t dm = *reinterpret_cast<const int64_t*>(strm + soff + 8);
      mem = ok ? mem + dm : mem;
      peak = mem > peak ? mem : peak;
    }
    __asm__ volatile("" : "+v"(prev));  // the previous load is used here, after this one issued
    const uint32_t n1 = okp ? prev : nxt;
    qb += ok ? 4u : 0u;
    cur = ok ? n1 : cur;
    nxt = n1;
    okp = ok;
    return __ballot(ok) != 0;
  };
  // two rounds per iteration, the loads alternating between a0 and a1, and one exit: a round
  // after one in which no lane moved changes nothing either, so the wave has settled
  uint32_t a0 = 0, a1 = 0;
  for (;;) {
    const bool g0 = round(a1, a0);
    const bool g1 = round(a0, a1);
    if (!(g0 && g1)) break;
  }
  const uint64_t actm = __ballot(cur != QT_END);
  if (actm != 0 && (fold_groups(actm, G, lsb) & gbit)) dead = true;
}

__device__ __forceinline__ int64_t group_sum(int64_t x, int G) {
  for (int off = G >> 1; off > 0; off >>= 1) x += __shfl_xor(x, off, G);
  return x;
}

__device__ __forceinline__ int64_t group_max(int64_t x, int G) {
  for (int off = G >> 1; off > 0; off >>= 1) {
    const int64_t y = __shfl_xor(x, off, G);
    x = y > x ? y : x;
  }
  return x;
}

}  // namespace octo
