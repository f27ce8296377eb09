// octo_sim.hpp — the max-plus relaxation core: one wave simulates CPW candidates at once, G
// lanes per candidate, lane d = pipeline device d. Each candidate owns a finish table in LDS
// with one slot per (stage, micro-batch).
//
// Slot encoding: empty = -2; after F(s,m) finishes the slot holds fin << 1; after B(s,m) it
// holds fin << 1 | 1. A single slot suffices because B(s,m) can only finish after F(s+1,m)
// (which consumed F(s,m)) has finished: B(s,m) needs B(s+1,m), which needs F(s+1,m). Row -1 is
// all zeros (F of stage 0 is always ready at time 0).
//
// Every op reads exactly one slot:
//   F(s,m): row s-1, ready when finished (>= 0); in = fin + link weight of the stage boundary.
//   B(s,m), s < S-1: row s+1, ready when it holds a B finish; in = fin + link weight.
//   B(S-1,m): its own row, ready when F(S-1,m) finished (the loss turns the forward around).
//   W(s,m): its own row, ready when B(s,m) finished.
// Other dependencies are implied: F(s,m) -> B(s,m) for s < S-1 follows from F(s,m) ->
// F(s+1,m) -> B(s+1,m) -> B(s,m). start = max(device clock, in); fin = start + duration
// (§5: record start/end per node; §6 Eq. 1: makespan = latest finish).
//
// Rounds: every live lane tries its head op once per round; a round in which no lane of a
// candidate advances while some still have ops is a deadlock (nothing can ever change again).
#pragma once

#include "octo_device.hpp"

namespace octo {

template <int VMAX>
struct Chunks {
  int st[VMAX];                                        // stage of chunk k
  int64_t dF[VMAX], dB[VMAX], dW[VMAX], wF[VMAX], wB[VMAX];
};

struct Lane {
  int64_t clock;
  int pos, nops;
  bool live;
  // current op
  int rd, wr, tag, needB;
  int64_t w, dur;
  int s, kind, m;  // for recording ideal starts
};

template <int VMAX, typename T>
__device__ __forceinline__ T pick(const T (&a)[VMAX], int k) {
  T x = a[0];
#pragma unroll
  for (int i = 1; i < VMAX; ++i)
    if (k == i) x = a[i];
  return x;
}

// Describe op (kind, chunk k, micro-batch m) for the slot layout index(row r, m) = (r+1)*M + m.
template <int VMAX>
__device__ __forceinline__ void describe(Lane& L, const Chunks<VMAX>& c, int kind, int k, int m, int M,
                                int S, int sink) {
  const int s = pick<VMAX>(c.st, k);
  const int own = (s + 1) * M + m;
  L.s = s, L.kind = kind, L.m = m;
  if (kind == KF) {
    L.rd = own - M;
    L.wr = own;
    L.needB = 0;
    L.tag = 0;
    L.w = pick<VMAX>(c.wF, k);
    L.dur = pick<VMAX>(c.dF, k);
  } else if (kind == KB) {
    const bool last = s == S - 1;
    L.rd = last ? own : own + M;
    L.wr = own;
    L.needB = last ? 0 : 1;
    L.tag = 1;
    L.w = last ? 0 : pick<VMAX>(c.wB, k);
    L.dur = pick<VMAX>(c.dB, k);
  } else {
    L.rd = own;
    L.wr = sink;
    L.needB = 1;
    L.tag = 0;
    L.w = 0;
    L.dur = pick<VMAX>(c.dW, k);
  }
}

// Run the rounds until every candidate of the wave is done or deadlocked.
// gmask: the lanes of this lane's candidate. rec (nullable): ideal-start recording for the
// MERGE table, rec[pos] = start << 16 | kind << 12 | m.
template <int VMAX, class Gen>
__device__ __forceinline__ void relax(Gen& gen, const Chunks<VMAX>& c, Lane& L, int64_t* T, int M, int S,
                             int sink, uint64_t gmask, bool& dead, uint32_t* rec) {
  for (;;) {
    int adv = 0;
    if (L.live) {
      const int64_t p = T[L.rd];
      const bool ok = L.needB ? ((p & 1) != 0) : (p >= 0);
      if (ok) {
        const int64_t tin = (p >> 1) + L.w;
        const int64_t st = tin > L.clock ? tin : L.clock;
        L.clock = st + L.dur;
        T[L.wr] = (L.clock << 1) | L.tag;
        if (rec) rec[L.pos] = ((uint32_t)st << 16) | ((uint32_t)L.kind << 12) | (uint32_t)L.m;
        adv = 1;
        if (++L.pos < L.nops) {
          gen.step();
          describe<VMAX>(L, c, gen.kind(), gen.chunk(), gen.mb(), M, S, sink);
        } else {
          L.live = false;
        }
      }
    }
    __asm__ volatile("" ::: "memory");
    const uint64_t advm = __ballot(adv);
    const uint64_t actm = __ballot(L.live);
    if ((actm & gmask) != 0 && (advm & gmask) == 0) {
      dead = true;
      L.live = false;
    }
    if (__ballot(L.live) == 0) break;
  }
}

__device__ __forceinline__ int64_t group_max(int64_t x, int G) {
  for (int off = G >> 1; off > 0; off >>= 1) {
    const int64_t y = __shfl_xor(x, off, G);
    x = y > x ? y : x;
  }
  return x;
}

}  // namespace octo
