// octo_device.hpp — device-side building blocks of the batched pipeline-schedule simulator:
// candidate-record decoding and validation, the per-device queue generators (one lane = one
// pipeline device) and Philox4x64-10.
//
// The time model is that of OctoPipe's graph-based simulator (arXiv 2509.23722, §5, §6 Eq. 1):
// ops F(s,m), B(s,m), W(s,m); queue-order edges; F(s-1,m)->F(s,m) and B(s+1,m)->B(s,m) with the
// link cost between the hosting devices (the send/recv pair of §5 as one edge weight);
// F(s,m)->B(s,m); B(s,m)->W(s,m). Earliest starts; makespan = latest finish; bubble = makespan -
// busy time; a cycle is a deadlock.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace octo {

constexpr int KF = 0, KB = 1, KW = 2;                 // op kinds
constexpr int POL_AFAB = 0, POL_1F1B = 1, POL_I1F1B = 2, POL_ZB = 3;
constexpr int GEN_AFAB = 0, GEN_INTER = 1, GEN_MERGE = 2, GEN_MAT = 3;

// Work bins. Generated queues are binned by (v, generator) so that the lanes of a wave run one
// code path; bins are numbered heaviest first (large v first; within one v: AFAB, then split
// backward, then fused).
constexpr int NBIN_GEN = 40;          // (8 - v) * 5 + rank, v = 1..8
// candidates of a structure class with a static round schedule: bins BIN_STATIC + class
constexpr int NSC = 9;
constexpr int BIN_STATIC = 40;
// candidates with perturbations (queues materialised): bins BIN_MAT + mat_sub(v, split), the
// last ones, by queue length like the generated bins (large v first, split first)
constexpr int BIN_MAT = BIN_STATIC + NSC;
constexpr int NBINS = BIN_MAT + 16;
__host__ __device__ __forceinline__ int mat_sub(int v, int split) { return (8 - v) * 2 + (split ? 0 : 1); }
constexpr int BIN_NONE = 0xFF;        // invalid: sentinel already written
// rank of a generator within one v: 0 AFAB, 1 MERGE split, 2 INTER split, 3 MERGE fused,
// 4 INTER fused
__host__ __device__ __forceinline__ int bin_of(int v, int gen, int split) {
  int r = gen == GEN_AFAB ? 0 : gen == GEN_INTER ? (split ? 2 : 4) : (split ? 1 : 3);
  return (8 - v) * 5 + r;
}
__host__ __device__ __forceinline__ int first_bin(int v) { return (8 - v) * 5; }
__host__ __device__ __forceinline__ void bin_decode(int bin, int* v, int* gen, int* split) {
  *v = 8 - bin / 5;
  int r = bin % 5;
  *gen = r == 0 ? GEN_AFAB : (r == 2 || r == 4) ? GEN_INTER : GEN_MERGE;
  *split = (r == 1 || r == 2);
}

__host__ __device__ __forceinline__ int pert_off(int s_max) { return (3 + 2 * s_max + 1) & ~1; }

// MERGE table entry: ideal start << 16 | kind << 12 | m; END sorts after every real entry.
constexpr uint32_t MERGE_END = 0xFFFFFFFFu;

// Entry offset of the MERGE table for (v, split), v >= 2: tables are stored for v = 2, 3, ...,
// each a fused table (S rows of 2M) followed by a split one (S rows of 3M), S = P v.
__host__ __device__ inline int64_t merge_offset(int P, int M, int v, int split) {
  const int64_t before = (int64_t)P * 5 * M * ((int64_t)(v - 1) * v / 2 - 1);
  return before + (split ? (int64_t)P * v * 2 * M : 0);
}

// Queue-store entry (materialised queues): kind << 14 | chunk << 11 | m.
__host__ __device__ __forceinline__ uint16_t qpack(int kind, int chunk, int m) {
  return (uint16_t)((kind << 14) | (chunk << 11) | m);
}

struct Problem {
  int L, P, v_max, M, stride, max_pert;
  int s_max;  // P * v_max
};

// ------------------------------------------------------------------------------------------
// Candidate header decoding and validation (one thread per candidate; plain byte reads).
// ------------------------------------------------------------------------------------------

struct Resolved {
  int valid;  // 1 if every validity rule holds
  int v, S, gen, split, n_pert;
};

// Validity, looped-placement and balanced-placement tests of one record.
// head: the record's first pert_off(s_max) bytes (may be a staged copy); pert: its perturbation
// list (in the record itself). The stage loops run to the end and fold their tests into one
// flag (no early exit per lane: the lanes of a wave would otherwise leave at different stages).
__device__ __forceinline__ Resolved resolve_record(const Problem& pr, const uint8_t* head,
                                                  const uint8_t* pert) {
  const uint8_t* rec = head;
  Resolved r;
  int policy = rec[0], v = rec[1], n_pert = rec[2], flags = rec[3];
  r.v = v;
  r.S = pr.P * v;
  r.n_pert = n_pert;
  r.split = policy == POL_ZB;
  r.gen = GEN_AFAB;
  r.valid = 0;
  if (policy > 3 || v < 1 || v > pr.v_max || n_pert > pr.max_pert || flags != 0) return r;
  const int S = r.S;
  const uint8_t* bnd = rec + 4;
  const uint8_t* dev = rec + 3 + pr.s_max;
  bool ok = true;
  int prev = 0;
#pragma unroll 8
  for (int s = 1; s < S; ++s) {
    const int b = bnd[s - 1];
    ok &= b > prev;
    prev = b;
  }
  ok &= prev < pr.L;
  // balanced placement: every device at most (so exactly) v stages, counted in 4-bit fields
  // (one 64-bit word up to P = 16, four beyond); looped: stage s on the device of s mod P
  bool looped = true;
  int j = 0;
  if (pr.P <= 16) {
    uint64_t c = 0;
#pragma unroll 8
    for (int s = 0; s < S; ++s) {
      const int d = dev[s];
      ok &= d < pr.P;
      const int sh = (d & 15) * 4;
      const bool room = (int)((c >> sh) & 15) < v;
      ok &= room;
      c += room ? (uint64_t)1 << sh : 0;
      looped &= s < pr.P || d == dev[j];
      j = j + 1 == pr.P ? 0 : j + 1;
    }
  } else {
    uint64_t c0 = 0, c1 = 0, c2 = 0, c3 = 0;
    for (int s = 0; s < S; ++s) {
      const int d = dev[s];
      ok &= d < pr.P;
      const int w = (d >> 4) & 3, sh = (d & 15) * 4;
      const uint64_t cw = w == 0 ? c0 : w == 1 ? c1 : w == 2 ? c2 : c3;
      const bool room = (int)((cw >> sh) & 15) < v;
      ok &= room;
      const uint64_t inc = room ? (uint64_t)1 << sh : 0;
      c0 += w == 0 ? inc : 0;
      c1 += w == 1 ? inc : 0;
      c2 += w == 2 ? inc : 0;
      c3 += w == 3 ? inc : 0;
      looped &= s < pr.P || d == dev[j];
      j = j + 1 == pr.P ? 0 : j + 1;
    }
  }
  if (!ok) return r;
  // every device got v stages: total S = P v stages and no device exceeds v
  if (policy == POL_AFAB) {
    r.gen = GEN_AFAB;
  } else if (v == 1) {
    r.gen = GEN_INTER;
  } else if (policy == POL_1F1B || !looped) {
    r.gen = GEN_MERGE;
  } else {
    if (pr.M % pr.P != 0) return r;
    r.gen = GEN_INTER;
  }
  // perturbations in range (queue length = (split ? 3 : 2) v M)
  const int qlen = (r.split ? 3 : 2) * v * pr.M;
  const uint8_t* pp = pert;
  for (int i = 0; i < n_pert; ++i) {
    int d = pp[6 * i] | (pp[6 * i + 1] << 8);
    int from = pp[6 * i + 2] | (pp[6 * i + 3] << 8);
    int to = pp[6 * i + 4] | (pp[6 * i + 5] << 8);
    if (d >= pr.P || from >= qlen || to >= qlen) return r;
  }
  r.valid = 1;
  return r;
}

// ------------------------------------------------------------------------------------------
// Structure classes with static round schedules. In the lockstep rounds an op is ready when its
// producers finished in earlier rounds, which depends on the structure — which stages share a
// device, the generator, a split backward — and never on the costs. These classes recur among
// candidates, so each has one precomputed schedule: v = 1 (any placement: relabelling devices
// does not change the structure), and v = 2 with the looped {c, c+P}, blocked {2c, 2c+1} or
// V-shape {c, 2P-1-c} stage pairs. A device's row is picked by its role, the canonical device
// that hosts the same stages.
//   class: 0 v1 INTER fused, 1 v1 INTER split, 2 looped INTER fused, 3 looped INTER split,
//          4 looped MERGE fused, 5 blocked MERGE fused, 6 blocked MERGE split,
//          7 V-shape MERGE fused, 8 V-shape MERGE split
// pattern: 0 one stage per device, 1 looped, 2 blocked, 3 V-shape.
// ------------------------------------------------------------------------------------------
__host__ __device__ __forceinline__ void sc_decode(int c, int* v, int* gen, int* split, int* pat) {
  *v = c < 2 ? 1 : 2;
  *gen = (c < 4) ? GEN_INTER : GEN_MERGE;
  *split = (c == 1 || c == 3 || c == 6 || c == 8) ? 1 : 0;
  *pat = c < 2 ? 0 : c < 5 ? 1 : c < 7 ? 2 : 3;
}

// Class of a valid record (resolved as r), or -1: its queues are generated per candidate.
__device__ __forceinline__ int static_class(const Problem& pr, const uint8_t* dev,
                                            const Resolved& r) {
  if (r.n_pert > 0 || r.gen == GEN_AFAB || r.v > 2) return -1;
  if (r.v == 1) return r.split ? 1 : 0;
  const int P = pr.P;
  bool lp = true, bl = true, vs = true;
#pragma unroll 4
  for (int i = 0; i < P; ++i) {
    lp = lp && dev[i] == dev[i + P];
    bl = bl && dev[2 * i] == dev[2 * i + 1];
    vs = vs && dev[i] == dev[2 * P - 1 - i];
  }
  if (lp) return r.gen == GEN_INTER ? (r.split ? 3 : 2) : (r.split ? -1 : 4);
  if (r.gen != GEN_MERGE) return -1;
  if (bl) return r.split ? 6 : 5;
  if (vs) return r.split ? 8 : 7;
  return -1;
}

// Canonical device of stage s under a pattern, and the role of a device whose lowest stage
// is s0.
__host__ __device__ __forceinline__ int sc_device(int pat, int P, int s) {
  return pat == 0 ? s : pat == 1 ? s % P : pat == 2 ? s / 2 : (s < P ? s : 2 * P - 1 - s);
}
__host__ __device__ __forceinline__ int sc_role(int pat, int s0) { return pat == 2 ? s0 / 2 : s0; }
// Stages of canonical device c (the second is unused at v = 1).
__host__ __device__ __forceinline__ void sc_stages(int pat, int P, int c, int* s0, int* s1) {
  *s0 = pat == 2 ? 2 * c : c;
  *s1 = pat == 1 ? c + P : pat == 2 ? 2 * c + 1 : pat == 3 ? 2 * P - 1 - c : c;
}

// Schedule entry of one device in one round: the slot its op reads (a cross-device producer's
// finish time, else the sentinel slot sc_neg, which holds a time far below zero), the stream of
// its duration and input weight (kind * v + chunk; SC_NOP_STREAM: zero duration), and the slot
// it writes (its finish time if another device reads it, else the sink slot sc_dummy). Bits:
// read slot << 3, stream << 9, write slot << 12, so that address = (entry & mask) | base needs
// one instruction. A round in which the device runs nothing is sc_nop.
// Slots per candidate: 32 up to P = 8 (the classes there keep at most 16 values live at M = 64,
// and the smaller LDS block lets more waves run), else 64; the last two are the sentinel and the
// sink. A class that needs more is left to the generated-queue kernels.
constexpr int SC_NOP_STREAM = 7;
__host__ __device__ __forceinline__ int sc_slots(int P) { return P <= 8 ? 32 : 64; }
__host__ __device__ __forceinline__ int sc_neg(int ns) { return ns - 2; }
__host__ __device__ __forceinline__ int sc_dummy(int ns) { return ns - 1; }
__host__ __device__ __forceinline__ uint32_t sc_entry(int rd, int stream, int wr) {
  return (uint32_t)rd << 3 | (uint32_t)stream << 9 | (uint32_t)wr << 12;
}
__host__ __device__ __forceinline__ uint32_t sc_nop(int ns) {
  return sc_entry(sc_neg(ns), SC_NOP_STREAM, sc_dummy(ns));
}

// ------------------------------------------------------------------------------------------
// Queue generators. Each lane owns one device queue and walks it front to back. A generator
// holds the current op in (kind, k, m) — kind, local chunk, micro-batch — and advance(ok) steps
// to the next op when ok is true. The step is straight-line code (selects), so lanes that do
// not advance cost no divergent branches.
// ------------------------------------------------------------------------------------------

// GPipe order: forwards by (chunk asc, m), then backwards by (chunk desc, m).
struct GenAfab {
  int v, M;
  int kind, k, m;
  __device__ __forceinline__ void init(int v_, int M_) { v = v_, M = M_, kind = KF, k = 0, m = 0; }
  __device__ __forceinline__ void advance(bool ok) {
    const int m1 = m + 1;
    const bool wrap = m1 == M;
    const bool isF = kind == KF;
    const int kf = k + (wrap ? 1 : 0);
    const bool flip = isF && kf == v;
    const int kn = isF ? (flip ? v - 1 : kf) : k - (wrap ? 1 : 0);
    m = ok ? (wrap ? 0 : m1) : m;
    k = ok ? kn : k;
    kind = ok ? ((isF && !flip) ? KF : KB) : kind;
  }
  __device__ __forceinline__ void take_if(bool t, const GenAfab& o) {
    kind = t ? o.kind : kind, k = t ? o.k : k, m = t ? o.m : m;
  }
};

// Interleaved 1F1B (Narayanan et al.): virtual index j = c*P*v + b*P + a maps to chunk b and
// micro-batch c*P + a for forwards; backwards take chunk v-1-b. Warm-up w forwards, then
// (F, B) pairs, then the remaining B; with a split backward each B's W follows `lag` B's later
// (a FIFO of depth lag), flushed at the end. At v = 1 this is 1F1B.
__host__ __device__ __forceinline__ int imin(int a, int b) { return a < b ? a : b; }
__host__ __device__ __forceinline__ int inter_warmup(int P, int v, int M, int r) {
  return v == 1 ? imin(P - 1 - r, M) : imin(2 * (P - 1 - r) + (v - 1) * P, v * M);
}
__host__ __device__ __forceinline__ int inter_kind(int nF, int nB, int nW, int w, int N,
                                                   int split, int lag) {
  const int fcap = imin(N, w + nB + 1);
  const int body = nF < fcap ? KF : KB;
  const int k1 = nB < N ? body : KW;
  const int k2 = (split && nW < nB - lag) ? KW : k1;
  return nF < w ? KF : k2;
}

// Power-of-two P and v: the virtual index decomposes with shifts and masks.
struct GenInterP2 {
  int lgP, lgPv, Pm1, vm1, N, w, lag, split;
  int nF, nB, nW;
  int kind, k, m;
  __device__ __forceinline__ void init(int P, int v, int M, int r, int split_, int lag_) {
    lgP = __ffs(P) - 1;
    lgPv = lgP + __ffs(v) - 1;
    Pm1 = P - 1, vm1 = v - 1, N = v * M, split = split_, lag = lag_;
    w = inter_warmup(P, v, M, r);
    nF = nB = nW = 0;
    update();
  }
  __device__ __forceinline__ void update() {
    kind = inter_kind(nF, nB, nW, w, N, split, lag);
    const int j = kind == KF ? nF : kind == KB ? nB : nW;
    const int kx = (j >> lgP) & vm1;
    m = ((j >> lgPv) << lgP) | (j & Pm1);
    k = kind == KF ? kx : vm1 - kx;
  }
  __device__ __forceinline__ void advance(bool ok) {
    nF += (ok && kind == KF) ? 1 : 0;
    nB += (ok && kind == KB) ? 1 : 0;
    nW += (ok && kind == KW) ? 1 : 0;
    update();
  }
  __device__ __forceinline__ void take_if(bool t, const GenInterP2& o) {
    nF = t ? o.nF : nF, nB = t ? o.nB : nB, nW = t ? o.nW : nW;
    kind = t ? o.kind : kind, k = t ? o.k : k, m = t ? o.m : m;
  }
};

// Any P and v: each stream keeps its virtual index decomposed as (a, b, c).
struct GenInter {
  int P, v, N, w, lag, split;
  int nF, nB, nW;
  int fa, fb, fc, ba, bb, bc, wa, wb, wc;
  int kind, k, m;
  __host__ __device__ __forceinline__ void init(int P_, int v_, int M, int r, int split_,
                                                int lag_) {
    P = P_, v = v_, N = v_ * M, split = split_, lag = lag_;
    w = inter_warmup(P, v, M, r);
    nF = nB = nW = 0;
    fa = fb = fc = ba = bb = bc = wa = wb = wc = 0;
    update();
  }
  __host__ __device__ __forceinline__ void update() {
    kind = inter_kind(nF, nB, nW, w, N, split, lag);
    k = kind == KF ? fb : kind == KB ? v - 1 - bb : v - 1 - wb;
    m = kind == KF ? fc * P + fa : kind == KB ? bc * P + ba : wc * P + wa;
  }
  __host__ __device__ __forceinline__ static void inc(int& a, int& b, int& c, int P, int v) {
    if (++a == P) {
      a = 0;
      if (++b == v) b = 0, ++c;
    }
  }
  __host__ __device__ __forceinline__ void advance(bool ok) {
    if (ok) {
      if (kind == KF) ++nF, inc(fa, fb, fc, P, v);
      else if (kind == KB) ++nB, inc(ba, bb, bc, P, v);
      else ++nW, inc(wa, wb, wc, P, v);
    }
    update();
  }
  __host__ __device__ __forceinline__ void take_if(bool t, const GenInter& o) {
    if (t) *this = o;
  }
};

// MERGE: a device's stages each follow the ideal stage-level order of a shared table (rows of
// `rowlen` entries, one row per stage); the device takes the entry with the smallest ideal
// start, the lower stage on ties. Each chunk keeps its head entry and the next one in
// registers. The load for a chunk's following entry is issued when the chunk advances and
// committed at the next advance, so its latency overlaps a whole round.
template <int VMAX>
struct GenMerge {
  const uint32_t* tab;
  int rowlen;
  int row[VMAX], pos[VMAX];
  uint32_t ent[VMAX], nxt[VMAX];
  uint32_t px;  // raw word of the load in flight for chunk pk (pk < 0: none)
  bool pv;      // that load is inside the row (else the row has ended)
  int pk;
  int kind, k, m;
  __device__ __forceinline__ uint32_t fetch(int r, int p) const {
    const uint32_t x = tab[r + min(p, rowlen - 1)];
    return p < rowlen ? x : MERGE_END;
  }
  template <class StageOf>
  __device__ __forceinline__ void init(const uint32_t* tab_, int rowlen_, int v, StageOf stage_of) {
    tab = tab_, rowlen = rowlen_;
#pragma unroll
    for (int c = 0; c < VMAX; ++c) {
      row[c] = c < v ? stage_of(c) * rowlen : 0;
      pos[c] = 0;
      ent[c] = c < v ? fetch(row[c], 0) : MERGE_END;
      nxt[c] = c < v ? fetch(row[c], 1) : MERGE_END;
    }
    px = MERGE_END, pv = false, pk = -1;
    update();
  }
  __device__ __forceinline__ void update() {
    uint32_t best = ent[0];
    int b = 0;
#pragma unroll
    for (int c = 1; c < VMAX; ++c) {
      const bool lt = (ent[c] >> 16) < (best >> 16);
      best = lt ? ent[c] : best;
      b = lt ? c : b;
    }
    k = b;
    kind = (best >> 12) & 3;
    m = best == MERGE_END ? 0 : best & 0x7FF;
  }
  __device__ __forceinline__ void advance(bool ok) {
    // commit the load issued at the previous advance (its latency covered a whole round)
    const uint32_t got = pv ? px : MERGE_END;
#pragma unroll
    for (int c = 0; c < VMAX; ++c) nxt[c] = pk == c ? got : nxt[c];
    int r = row[0], p = pos[0];
#pragma unroll
    for (int c = 1; c < VMAX; ++c) r = k == c ? row[c] : r, p = k == c ? pos[c] : p;
    px = tab[r + min(p + 2, rowlen - 1)];
    pv = p + 2 < rowlen;
    pk = ok ? k : -1;
#pragma unroll
    for (int c = 0; c < VMAX; ++c) {
      const bool t = ok && k == c;
      pos[c] += t ? 1 : 0;
      ent[c] = t ? nxt[c] : ent[c];
    }
    update();
  }
  __device__ __forceinline__ void take_if(bool t, const GenMerge& o) {
#pragma unroll
    for (int c = 0; c < VMAX; ++c) {
      pos[c] = t ? o.pos[c] : pos[c];
      ent[c] = t ? o.ent[c] : ent[c];
      nxt[c] = t ? o.nxt[c] : nxt[c];
    }
    px = t ? o.px : px, pv = t ? o.pv : pv, pk = t ? o.pk : pk;
    kind = t ? o.kind : kind, k = t ? o.k : k, m = t ? o.m : m;
  }
};

// Materialised queue row in global memory (perturbed candidates, tuner chains). The entry after
// next is loaded at each step and committed at the following step.
struct GenMat {
  const uint16_t* rowp;
  int len, pos;
  uint32_t cur, nxt, px;
  bool pv;
  int kind, k, m;
  __device__ __forceinline__ uint32_t fetch(int p) const { return rowp[min(p, max(len - 1, 0))]; }
  __device__ __forceinline__ void init(const uint16_t* r, int len_) {
    rowp = r, len = len_, pos = 0;
    cur = fetch(0);
    nxt = fetch(1);
    px = 0, pv = false;
    update();
  }
  __device__ __forceinline__ void update() {
    kind = (cur >> 14) & 3;
    k = (cur >> 11) & 7;
    m = cur & 0x7FF;
  }
  __device__ __forceinline__ void advance(bool ok) {
    nxt = pv ? px : nxt;
    px = fetch(pos + 2);
    pv = ok;
    pos += ok ? 1 : 0;
    cur = ok ? nxt : cur;
    update();
  }
  __device__ __forceinline__ void take_if(bool t, const GenMat& o) {
    pos = t ? o.pos : pos, cur = t ? o.cur : cur, nxt = t ? o.nxt : nxt;
    px = t ? o.px : px, pv = t ? o.pv : pv;
    kind = t ? o.kind : kind, k = t ? o.k : k, m = t ? o.m : m;
  }
};

// Materialised queue row read K rounds ahead, for the unrolled speculative relaxation
// (relax_k): in round t every lane loads a 16-byte span of eight entries starting at its
// position (rounded down to a dword) into buffer t mod K, which round t + K consumes. A lane
// advances at most one entry a round, so the entry after its position K rounds later is still
// in that span (K <= 6); the loads are unconditional, so each buffer keeps its registers and a
// round waits only for the load issued K rounds before. Spans are clamped to the row's capacity
// (cap entries, rounded up to a dword), so every dword read holds a byte of the row: no read
// leaves the pages the row lies in. Needs cap >= 8.
template <int K>
struct GenMatK {
  static_assert(K >= 1 && K <= 6, "the span of eight entries covers K + 1 advances");
  const uint32_t* base;  // the row's first entry, rounded down to a dword
  int off, e0max;        // the row's first entry within that dword; the last span's start
  int pos;               // position in the row
  int kind, k, m;
  uint4 buf[K];
  int e0[K];             // first entry (from base, even) of each buffer's span
  struct __attribute__((aligned(4))) Span {
    uint32_t x, y, z, w;
  };
  __device__ __forceinline__ uint4 load(int e) const {
    const Span v = *reinterpret_cast<const Span*>(base + (e >> 1));
    return make_uint4(v.x, v.y, v.z, v.w);
  }
  __device__ __forceinline__ int span_of(int p) const {
    const int e = (p + off) & ~1;
    return e < e0max ? e : e0max;
  }
  // entry j of a span: a select of one 64-bit half and a shift (a select chain over the four
  // words would be turned into an indexed copy in private memory)
  __device__ __forceinline__ void set(const uint4& b, int j) {
    const uint64_t lo = (uint64_t)b.x | ((uint64_t)b.y << 32);
    const uint64_t hi = (uint64_t)b.z | ((uint64_t)b.w << 32);
    const uint64_t q = (j & 4) ? hi : lo;
    const uint32_t e = (uint32_t)(q >> ((j & 3) * 16)) & 0xFFFFu;
    kind = (int)((e >> 14) & 3);
    k = (int)((e >> 11) & 7);
    m = (int)(e & 0x7FF);
  }
  __device__ __forceinline__ void init(const uint16_t* r, int cap) {
    off = (int)((reinterpret_cast<uintptr_t>(r) & 3) >> 1);
    base = reinterpret_cast<const uint32_t*>(r - off);
    e0max = ((off + cap + 1) & ~1) - 8;
    pos = 0;
    const uint4 b = load(0);
#pragma unroll
    for (int u = 0; u < K; ++u) buf[u] = b, e0[u] = 0;
    set(b, off);
  }
  // speculative: the entry after the current one, from buffer U
  template <int U>
  __device__ __forceinline__ void advance(bool ok) {
    pos += ok ? 1 : 0;
    set(buf[U], pos + off - e0[U]);
  }
  // once per round, after the outcome: keep o's position if t, then refill buffer U
  template <int U>
  __device__ __forceinline__ void take_if(bool t, const GenMatK& o) {
    pos = t ? o.pos : pos;
    kind = t ? o.kind : kind, k = t ? o.k : k, m = t ? o.m : m;
    e0[U] = span_of(pos);
    buf[U] = load(e0[U]);
  }
};

// ------------------------------------------------------------------------------------------
// Philox4x64-10 (Salmon, Moraes, Dror, Shaw, SC'11): published multipliers and Weyl constants.
// ------------------------------------------------------------------------------------------
struct U4 {
  uint64_t x[4];
};
__device__ __forceinline__ U4 philox4x64_10(uint64_t c0, uint64_t c1, uint64_t c2, uint64_t c3, uint64_t k0,
                                   uint64_t k1) {
  const uint64_t M0 = 0xD2E7470EE14C6C93ull, M1 = 0xCA5A826395121157ull;
  const uint64_t W0 = 0x9E3779B97F4A7C15ull, W1 = 0xBB67AE8584CAA73Bull;
#pragma unroll
  for (int i = 0; i < 10; ++i) {
    if (i) k0 += W0, k1 += W1;
    uint64_t hi0 = __umul64hi(M0, c0), lo0 = M0 * c0;
    uint64_t hi1 = __umul64hi(M1, c2), lo1 = M1 * c2;
    uint64_t n0 = hi1 ^ c1 ^ k0, n2 = hi0 ^ c3 ^ k1;
    c0 = n0, c1 = lo1, c2 = n2, c3 = lo0;
  }
  U4 r;
  r.x[0] = c0, r.x[1] = c1, r.x[2] = c2, r.x[3] = c3;
  return r;
}

}  // namespace octo

namespace octo {
__device__ __forceinline__ Resolved resolve_record(const Problem& pr, const uint8_t* rec) {
  return resolve_record(pr, rec, rec + pert_off(pr.s_max));
}
}  // namespace octo
