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
// code path; bins are numbered heaviest first (large v, split backward first).
constexpr int NBIN_GEN = 40;          // (8 - v) * 5 + rank, v = 1..8
constexpr int BIN_MAT = 40;           // candidates with perturbations: queues materialised
constexpr int NBINS = 41;
constexpr int BIN_NONE = 0xFF;        // invalid: sentinel already written

// rank of a generator within one v: 0 MERGE split, 1 INTER split, 2 MERGE fused,
// 3 INTER fused, 4 AFAB
__host__ __device__ __forceinline__ int bin_of(int v, int gen, int split) {
  int r = gen == GEN_AFAB ? 4 : gen == GEN_INTER ? (split ? 1 : 3) : (split ? 0 : 2);
  return (8 - v) * 5 + r;
}
__host__ __device__ __forceinline__ void bin_decode(int bin, int* v, int* gen, int* split) {
  *v = 8 - bin / 5;
  int r = bin % 5;
  *gen = r == 4 ? GEN_AFAB : (r == 1 || r == 3) ? GEN_INTER : GEN_MERGE;
  *split = (r == 0 || r == 1);
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

// Looped placement test and balanced-placement test for a record in memory `rec`.
__device__ __forceinline__ Resolved resolve_record(const Problem& pr, const uint8_t* rec) {
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
  int prev = 0;
  for (int s = 1; s < S; ++s) {
    int b = bnd[s - 1];
    if (b <= prev) return r;
    prev = b;
  }
  if (pr.L <= prev) return r;
  // balanced placement: every device exactly v stages (counts kept as 4-bit fields)
  uint64_t cnt[4] = {0, 0, 0, 0};
  bool looped = true;
  for (int s = 0; s < S; ++s) {
    int d = dev[s];
    if (d >= pr.P) return r;
    int w = d >> 4, sh = (d & 15) * 4;
    uint64_t c = (cnt[w] >> sh) & 15;
    if ((int)c >= v) return r;
    cnt[w] += (uint64_t)1 << sh;
    if (s >= pr.P && dev[s] != dev[s % pr.P]) looped = false;
  }
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
  const uint8_t* pp = rec + pert_off(pr.s_max);
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
// Queue generators. Each lane owns one device queue and walks it front to back; a generator
// exposes the current op (kind, chunk, m) and steps to the next one.
// ------------------------------------------------------------------------------------------

// GPipe order: forwards by (chunk asc, m), then backwards by (chunk desc, m).
struct GenAfab {
  int v, M, ph, k, m;
  __device__ __forceinline__ void init(int v_, int M_) { v = v_, M = M_, ph = 0, k = 0, m = 0; }
  __device__ __forceinline__ int kind() const { return ph; }
  __device__ __forceinline__ int chunk() const { return k; }
  __device__ __forceinline__ int mb() const { return m; }
  __device__ __forceinline__ void step() {
    if (++m == M) {
      m = 0;
      if (ph == 0) {
        if (++k == v) ph = 1, k = v - 1;
      } else {
        --k;
      }
    }
  }
};

// Interleaved 1F1B (Narayanan et al.): virtual index j = c*P*v + b*P + a maps to chunk b and
// micro-batch c*P + a for forwards; backwards take chunk v-1-b. Warm-up w forwards, then
// (F, B) pairs, then the remaining B; with a split backward each B's W follows `lag` B's later
// (a FIFO of depth lag), flushed at the end. At v = 1 this is 1F1B.
struct GenInter {
  int P, v, N, w, lag, split;
  int nF, nB, nW;
  int fa, fb, fc, ba, bb, bc, wa, wb, wc;
  int cur;  // kind of the current op

  __device__ __forceinline__ void init(int P_, int v_, int M, int r, int split_, int lag_) {
    P = P_, v = v_, N = v_ * M, split = split_, lag = lag_;
    w = v == 1 ? min(P - 1 - r, M) : min(2 * (P - 1 - r) + (v - 1) * P, N);
    nF = nB = nW = 0;
    fa = fb = fc = ba = bb = bc = wa = wb = wc = 0;
    cur = next_kind();
  }
  __device__ __forceinline__ int next_kind() const {
    if (nF < w) return KF;
    if (split && nW < nB - lag) return KW;
    if (nB < N) return nF < min(N, w + nB + 1) ? KF : KB;
    return KW;
  }
  __device__ __forceinline__ int kind() const { return cur; }
  __device__ __forceinline__ int chunk() const {
    return cur == KF ? fb : cur == KB ? v - 1 - bb : v - 1 - wb;
  }
  __device__ __forceinline__ int mb() const {
    return cur == KF ? fc * P + fa : cur == KB ? bc * P + ba : wc * P + wa;
  }
  __device__ __forceinline__ static void inc(int& a, int& b, int& c, int P, int v) {
    if (++a == P) {
      a = 0;
      if (++b == v) b = 0, ++c;
    }
  }
  __device__ __forceinline__ void step() {
    if (cur == KF) ++nF, inc(fa, fb, fc, P, v);
    else if (cur == KB) ++nB, inc(ba, bb, bc, P, v);
    else ++nW, inc(wa, wb, wc, P, v);
    cur = next_kind();
  }
};

// MERGE: a device's stages each follow the ideal stage-level order of a shared table (rows of
// `rowlen` entries, one row per stage); the device takes the entry with the smallest ideal
// start, the lower stage on ties. Two entries per chunk are kept in registers so the table
// load for a chunk is issued one step before it is needed.
template <int VMAX>
struct GenMerge {
  const uint32_t* tab;
  int rowlen, v;
  int row[VMAX], pos[VMAX];
  uint32_t ent[VMAX], nxt[VMAX];
  int sel;

  __device__ __forceinline__ uint32_t fetch(int k, int p) const {
    return p < rowlen ? tab[row[k] + p] : MERGE_END;
  }
  template <class StageOf>
  __device__ __forceinline__ void init(const uint32_t* tab_, int rowlen_, int v_, StageOf stage_of) {
    tab = tab_, rowlen = rowlen_, v = v_;
#pragma unroll
    for (int k = 0; k < VMAX; ++k) {
      row[k] = k < v ? stage_of(k) * rowlen : 0;
      pos[k] = 0;
      ent[k] = k < v ? fetch(k, 0) : MERGE_END;
      nxt[k] = k < v ? fetch(k, 1) : MERGE_END;
    }
    pick();
  }
  __device__ __forceinline__ void pick() {
    uint32_t best = ent[0];
    int b = 0;
#pragma unroll
    for (int k = 1; k < VMAX; ++k)
      if ((ent[k] >> 16) < (best >> 16)) best = ent[k], b = k;
    sel = b;
  }
  __device__ __forceinline__ uint32_t cur_entry() const {
    uint32_t e = ent[0];
#pragma unroll
    for (int k = 1; k < VMAX; ++k)
      if (sel == k) e = ent[k];
    return e;
  }
  __device__ __forceinline__ int kind() const { return (cur_entry() >> 12) & 3; }
  __device__ __forceinline__ int chunk() const { return sel; }
  __device__ __forceinline__ int mb() const { return cur_entry() & 0x7FF; }
  __device__ __forceinline__ void step() {
#pragma unroll
    for (int k = 0; k < VMAX; ++k)
      if (sel == k) {
        pos[k] += 1;
        ent[k] = nxt[k];
        nxt[k] = fetch(k, pos[k] + 1);
      }
    pick();
  }
};

// Materialised queue row in global memory (perturbed candidates, tuner chains). The next entry
// is loaded one step ahead.
struct GenMat {
  const uint16_t* rowp;
  int len, pos;
  uint32_t cur, nxt;
  __device__ __forceinline__ void init(const uint16_t* r, int len_) {
    rowp = r, len = len_, pos = 0;
    cur = len > 0 ? rowp[0] : 0;
    nxt = len > 1 ? rowp[1] : 0;
  }
  __device__ __forceinline__ int kind() const { return (cur >> 14) & 3; }
  __device__ __forceinline__ int chunk() const { return (cur >> 11) & 7; }
  __device__ __forceinline__ int mb() const { return cur & 0x7FF; }
  __device__ __forceinline__ void step() {
    ++pos;
    cur = nxt;
    nxt = pos + 1 < len ? rowp[pos + 1] : 0;
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
