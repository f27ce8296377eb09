// octo.hip — kernels and host C ABI of libocto.so (declared in include/octo.h).
//
// One call of octo_sim_batch launches:
//   k_prep      layer-cost prefix sums; clears the bin counters.
//   k_merge_tab ideal stage-level start times for the MERGE order (cached per (P, v_max, M)).
//   k_classify  one thread per candidate: validate, resolve the queue generator, write the
//               sentinel of invalid candidates, count candidates per work bin.
//   k_plan      start position of each bin.
//   k_scatter   candidate indices grouped by bin (counting sort).
//   k_sim       persistent waves; each takes a chunk of CPW candidates of one INTER or MERGE
//               bin and simulates them together, queues generated in registers (the hot
//               kernel); finish tables with ring rows.
//   k_afab      AFAB candidates, one lane each: a pass over the stage rows in chain order.
//   k_sim_mat   candidates with perturbations: queues materialised in global memory, moved,
//               then simulated.
// octo_tune_step launches k_tune (one local-search step for every chain).
#include <hip/hip_runtime.h>

#include <algorithm>
#include <cstdio>
#include <cstring>
#include <map>
#include <mutex>
#include <utility>

#include "../../include/octo.h"
#include "octo_device.hpp"
#include "octo_sim.hpp"

namespace octo {

constexpr int WAVE = 64;

// Workspace control block (int32 words).
constexpr int CTL_COUNTS = 0;     // [NBINS] candidates per bin
constexpr int CTL_POS = 80;       // [NBINS] next index position of each bin (scatter cursor)
constexpr int CTL_WORK = 160;     // chunk counters of the k_sim launches (7)
constexpr int CTL_WORK_MAT = 168; // chunk counter of k_sim_mat, perturbed list
constexpr int CTL_WORK_REDO = 169;// chunk counter of k_sim_mat, redo list
constexpr int CTL_REDO = 170;     // candidates for the 64-bit path (40-bit overflow, ring bound)
constexpr int CTL_WIDE = 171;     // perturbed candidates whose queue window passes the ring
constexpr int CTL_WORK_WIDE = 172;// chunk counter of k_sim_mat40 over the wide list
constexpr int CTL_TOTAL = 173;    // valid records (all bins; set by k_plan)
constexpr int CTL_START = 176;    // [NBINS] first index position of each bin
constexpr int CTL_WORK_V = 241;   // chunk counters of the v = 3..8 k_sim launches (6), then of
                                  // their rendezvous GPipe launches (6)
constexpr int CTL_WORDS = 256;
static_assert(CTL_START + NBINS <= CTL_WORK_V && CTL_WORK_V + 12 <= CTL_WORDS, "control words");
static_assert(NBINS <= 80, "bin arrays of the control block hold 80 bins");
// rounds a materialised queue is read ahead of its use (GenMatK; rows of at least 8 entries)
constexpr int QK = 6;

struct SimArgs {
  Problem pr;
  const int64_t* pre;    // [(L+1)][3] prefix sums of layer costs
  const int64_t* pre_mem;  // [(L+1)][2] prefix sums of layer memory (memory-model calls)
  int64_t* out_peak;       // [n][P] peak bytes per device (memory-model calls)
  int64_t* out_comm;       // [n][4] communication tally (communication-accounting calls)
  int64_t* out_bound;      // [n][P][2] first start, last finish per device (bounds calls)
  const int64_t* link;   // [P][P]
  const uint8_t* cands;
  int64_t n;
  const int32_t* n_live;  // nullable: only the first *n_live of the n records are evaluated
  int mat_lists;          // lists k_sim_mat takes: 1 the perturbed candidates, 2 the 64-bit redo
  int64_t* out_ms;
  int64_t* out_bub;
  int32_t* ctl;
  const int32_t* idx;    // candidate indices sorted by bin
  int32_t* redo;         // candidates to recompute with 64-bit slots
  int32_t* wide;         // perturbed candidates too wide for the ring (k_sim_mat40 full rows)
  const uint32_t* mtab;  // MERGE tables, merge_offset() entries apart
  const uint16_t* mrows; // v = 2 MERGE queues by (split, s0, s1) (merge_rows); null: none
  int mrow_stride;       // entries per row of mrows
  uint16_t* qscratch;    // materialised queues, [group slot][P][qcap]
  int G, CPW;            // lanes per candidate, candidates per wave
  int slots;             // slots of one finish table (S_cap * M)
  int table_bytes;       // LDS bytes of one finish table
  int group_bytes;       // LDS bytes per candidate
  int rec_bytes;         // staged record bytes (header + boundaries + placement)
  int rec_stride;        // bytes between staged records of a wave
  int qcap;
  uint64_t bin_mask;     // generated bins handled by this launch
  int work;              // chunk counter index of this launch
  int ring;              // slots per stage row of this launch's finish tables (R)
  uint64_t redo_bins;    // bins whose queues may exceed R in flight: sent to the 64-bit path
  // queue tables (v <= 2) for this launch's geometry, entry index of each block's first row;
  // null: generate queues in-kernel
  const uint32_t* qtab;
  int64_t qt_inter[2][2];  // [v - 1][split], one row per rank
  int64_t qt_merge[2];     // [split], v = 2, one row per stage pair s0 < s1
  int64_t qt_end;          // the table's final terminators
  int strm_off;            // LDS byte offset of the per-lane stream table
  // static round schedules (null: every candidate takes the generated-queue kernels): rows of
  // st_rowlen entries, P + 1 rows per class (one per role, then a row of sc_nop), st_cls
  // entries apart; smeta [NSC][4] = {valid, rounds, slots, 0}
  const uint32_t* stab;
  const int32_t* smeta;
  int64_t st_cls;
  int st_rowlen;
};

__device__ __forceinline__ int lane_id() { return (int)(threadIdx.x & (WAVE - 1)); }

// Lane 0's value, as a wave-uniform (scalar) value: all lanes are active where it is used.
__device__ __forceinline__ int bcast(int x) { return __builtin_amdgcn_readfirstlane(x); }

// ---------------------------------------------------------------------------------------------
// Per-lane set-up of one candidate from its staged record.
// ---------------------------------------------------------------------------------------------
template <int VMAX>
__device__ __forceinline__ void zero_chunks(Chunks<VMAX>& c) {
#pragma unroll
  for (int k = 0; k < VMAX; ++k) {
    c.st[k] = 0, c.base[k] = 0, c.frow[k] = 0, c.fmask[k] = 0, c.brow[k] = 0, c.bmask[k] = 0;
    c.dF[k] = c.dB[k] = c.dW[k] = c.wF[k] = c.wB[k] = c.mA[k] = 0;
    c.cF[k] = c.cB[k] = 0, c.xF[k] = c.xB[k] = 0, c.dnF[k] = c.dnB[k] = -1;
  }
  c.wW = 0;
  c.split = 0;
}

// Stages of device d (ascending), their durations, incoming link weights and finish-table
// rows; returns busy(d). pre_mem (nullable): memory prefix sums; then each chunk's activation
// bytes go to c.mA and the device's static bytes to *stat. mode XC: also the transfer time of
// each op's output and the CX flags of its input and output; XS: those and the device each
// output goes to, with the transfer moved from the reader's weight into the writer's slot time.
template <int VMAX>
__device__ __forceinline__ int64_t setup_chunks(Chunks<VMAX>& c, const Problem& pr,
                                                const uint8_t* rec, const int64_t* pre,
                                                const int64_t* link, int d, int v, int split,
                                                const Ring& ring, const int64_t* pre_mem = nullptr,
                                                int64_t* stat = nullptr, int mode = XP) {
  const int S = pr.P * v, M = pr.M;
  const uint8_t* bnd = rec + 4;
  const uint8_t* dev = rec + 3 + pr.s_max;
  zero_chunks<VMAX>(c);
  int cnt = 0;
  for (int s = 0; s < S; ++s) {
    if (dev[s] == d) {
#pragma unroll
      for (int k = 0; k < VMAX; ++k) c.st[k] = cnt == k ? s : c.st[k];
      ++cnt;
    }
  }
  int64_t busy = 0, st_bytes = 0;
  c.split = split;
#pragma unroll
  for (int k = 0; k < VMAX; ++k) {
    if (k < v) {
      const int s = c.st[k];
      const int b0 = s > 0 ? bnd[s - 1] : 0;
      const int b1 = s < S - 1 ? bnd[s] : pr.L;
      const int64_t f = pre[3 * b1 + 0] - pre[3 * b0 + 0];
      const int64_t bi = pre[3 * b1 + 1] - pre[3 * b0 + 1];
      const int64_t wg = pre[3 * b1 + 2] - pre[3 * b0 + 2];
      c.base[k] = s * ring.R;
      c.frow[k] = s > 0 ? -ring.R : 0;
      c.fmask[k] = s > 0 ? (int)(ST_F | ST_PAR) : 0;
      c.brow[k] = s < S - 1 ? ring.R : 0;  // the last stage reads its own F
      c.bmask[k] = (int)((s < S - 1 ? ST_B : ST_F) | ST_PAR);
      c.dF[k] = f;
      c.dB[k] = split ? bi : bi + wg;
      c.dW[k] = wg;
      const int dp = s > 0 ? dev[s - 1] : d;
      const int dn = s < S - 1 ? dev[s + 1] : d;
      c.wF[k] = dp != d ? link[dp * pr.P + d] : 0;
      c.wB[k] = dn != d ? link[dn * pr.P + d] : 0;
      if (mode == XC || mode == XS || mode == XR) {
        // a forward's output goes to stage s + 1, a backward's to stage s - 1
        c.cF[k] = dn != d ? link[d * pr.P + dn] : 0;
        c.cB[k] = dp != d ? link[d * pr.P + dp] : 0;
        c.xF[k] = (dp != d ? CX_IN : 0) | (dn != d ? CX_OUT : 0);
        c.xB[k] = (dn != d ? CX_IN : 0) | (dp != d ? CX_OUT : 0);
      }
      if (mode == XR) {  // where each op's input comes from (its producer's mailbox)
        c.dnF[k] = dp != d ? dp : -1;
        c.dnB[k] = dn != d ? dn : -1;
      }
      if (mode == XS) {
        c.dnF[k] = dn != d ? dn : -1;
        c.dnB[k] = dp != d ? dp : -1;
        c.wF[k] = 0, c.wB[k] = 0;  // the writer's slot holds the arrival time
      }
      busy += f + bi + wg;
      if (pre_mem) {
        c.mA[k] = pre_mem[2 * b1] - pre_mem[2 * b0];
        st_bytes += pre_mem[2 * b1 + 1] - pre_mem[2 * b0 + 1];
      }
    }
  }
  if (mode == XS) c.wW = W_NO_TIME;
  if (stat) *stat = st_bytes;
  return busy * M;
}

// Sum of the communication tallies of a group's lanes (all lanes of the group take part).
__device__ __forceinline__ CommTally group_tally(CommTally x, int G) {
  for (int off = G >> 1; off > 0; off >>= 1) {
    x.n += __shfl_xor(x.n, off, G);
    x.nov += __shfl_xor(x.nov, off, G);
    x.t += __shfl_xor(x.t, off, G);
    x.tov += __shfl_xor(x.tov, off, G);
  }
  return x;
}

// One device's results for candidate cand (deadlock: sentinels); XM adds its peak bytes, XC the
// candidate's communication tally (tot: the group's sum).
template <int X>
__device__ __forceinline__ void put_results(const SimArgs& a, int64_t cand, int d, bool dead,
                                            int64_t ms, int64_t busy, int64_t stat, int64_t peak,
                                            const CommTally& tot, int64_t fs = 0,
                                            int64_t lf = 0) {
  const int P = a.pr.P;
  if (d == 0) a.out_ms[cand] = dead ? OCTO_MS_DEADLOCK : ms;
  a.out_bub[cand * P + d] = dead ? OCTO_MS_DEADLOCK : ms - busy;
  if constexpr (X == XM) a.out_peak[cand * P + d] = dead ? OCTO_MS_DEADLOCK : stat + peak;
  if constexpr (X == XB) {
    // an empty queue (no op ran) has neither: 0, 0
    a.out_bound[(cand * P + d) * 2] = dead ? OCTO_MS_DEADLOCK : fs < 0 ? 0 : fs;
    a.out_bound[(cand * P + d) * 2 + 1] = dead ? OCTO_MS_DEADLOCK : lf;
  }
  if constexpr (X == XC) {
    if (d == 0) {
      int64_t* o = a.out_comm + cand * 4;
      o[0] = dead ? OCTO_MS_DEADLOCK : tot.n;
      o[1] = dead ? OCTO_MS_DEADLOCK : tot.nov;
      o[2] = dead ? OCTO_MS_DEADLOCK : tot.t;
      o[3] = dead ? OCTO_MS_DEADLOCK : tot.tov;
    }
  }
}

// Group bits for deadlock folding: this lane's group bit and the set of all group bits.
__device__ __forceinline__ void group_bits(int G, uint64_t* gbit, uint64_t* lsb) {
  uint64_t x = 0;
  for (int i = 0; i < WAVE; i += G) x |= 1ull << i;
  *lsb = x;
  *gbit = 1ull << ((lane_id() / G) * G);
}

// Stage the first rec_bytes of a record into LDS (lanes of the candidate copy 4-byte words).
__device__ __forceinline__ void stage_record(uint8_t* dst, const uint8_t* src, int rec_bytes,
                                             int d, int G) {
  const int words = (rec_bytes + 3) >> 2;
  for (int i = d; i < words; i += G)
    reinterpret_cast<uint32_t*>(dst)[i] = reinterpret_cast<const uint32_t*>(src)[i];
}

// Simulate one candidate per group of the wave with generator kind GEN (40-bit slots shared by
// the wave's groups; each group's staged record sits in that memory until it is cleared), write
// the results. cand < 0: this group has no candidate. P2: P and v are powers of two.
template <int VMAX, int GEN, bool P2, int X>
__device__ __forceinline__ void run_generated(const SimArgs& a, int64_t cand, int v, int split,
                                              uint8_t* lds_wave, int64_t* mbox) {
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  const Table40 T{reinterpret_cast<uint32_t*>(lds_wave),
                  lds_wave + (size_t)a.slots * a.CPW * 4, __ffs(a.CPW) - 1, g < a.CPW ? g : 0};
  uint8_t* rec = lds_wave + (size_t)(g < a.CPW ? g : 0) * a.rec_stride;
  const bool has = cand >= 0;
  const int S = P * v;
  const Ring ring = make_ring(M, a.ring);
  if (has) stage_record(rec, a.cands + cand * a.pr.stride, a.rec_bytes, d, G);
  __asm__ volatile("" ::: "memory");

  Chunks<VMAX> c;
  Lane L;
  L.clock = 0;
  L.pos = 0;
  L.nops = 0;
  L.mem = L.peak = 0;
  L.cm.reset();
  L.fs = -1;
  if constexpr (X == XS)
    for (int i = 0; i < 16; ++i) L.lf[i] = 0;
  int64_t busy = 0, stat = 0;
  const bool mine = has && d < P;
  if (mine) {
    busy = setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, split, ring, a.pre_mem, &stat,
                              X);
    L.nops = (split ? 3 : 2) * v * M;
  } else {
    zero_chunks<VMAX>(c);
  }
  __asm__ volatile("" ::: "memory");
  T.clear_all(S * ring.R, lane_id(), WAVE);
  __asm__ volatile("" ::: "memory");

  bool dead = false;
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  if constexpr (X == XR) mbox[lane_id()] = RDV_EMPTY;
  if constexpr (GEN == GEN_AFAB) {
    GenAfab g;
    g.init(v, M);
    describe<VMAX>(L, c, ring, g.kind, g.k, g.m);
    rounds<VMAX, false, X>(g, c, ring, L, T, G, gbit, lsb, dead, mbox);
  } else if constexpr (GEN == GEN_INTER) {
    const int r = c.st[0];
    if constexpr (P2) {
      GenInterP2 g;
      g.init(P, v, M, r, split, split ? r : 0);
      describe<VMAX>(L, c, ring, g.kind, g.k, g.m);
      rounds<VMAX, false, X>(g, c, ring, L, T, G, gbit, lsb, dead, mbox);
    } else {
      GenInter g;
      g.init(P, v, M, r, split, split ? r : 0);
      describe<VMAX>(L, c, ring, g.kind, g.k, g.m);
      rounds<VMAX, false, X>(g, c, ring, L, T, G, gbit, lsb, dead, mbox);
    }
  } else {
    GenMerge<VMAX> g;
    const int rowlen = (split ? 3 : 2) * M;
    g.init(a.mtab + (v >= 2 ? merge_offset(P, M, v, split) : 0), rowlen, mine ? v : 0,
           [&](int k) { return pick<VMAX>(c.st, k); });
    describe<VMAX>(L, c, ring, g.kind, g.k, g.m);
    rounds<VMAX, false, X>(g, c, ring, L, T, G, gbit, lsb, dead, mbox);
  }

  const int64_t ms = group_max(L.clock, G);
  CommTally tot = L.cm;
  if constexpr (X == XC) tot = group_tally(L.cm, G);
  if (mine) {
    if (ms >= Table40::LIMIT) {
      // times beyond the 40-bit slots: recompute this candidate with 64-bit slots
      if (d == 0) a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
    } else {
      put_results<X>(a, cand, d, dead, ms, busy, stat, L.peak, tot, L.fs, L.clock);
    }
  }
}

// Row of the queue table that holds device d's queue (v <= 2): INTER by the device's first
// stage (its rank), MERGE by its stage pair. Returns the row's first entry index.
template <int VMAX>
__device__ __forceinline__ int qt_row(const SimArgs& a, int gen, int v, int split,
                                      const Chunks<VMAX>& c) {
  const int M = a.pr.M, S = a.pr.P * v;
  const int64_t n = (int64_t)(split ? 3 : 2) * v * M + 2;  // row + two terminators
  if (gen == GEN_INTER) return (int)(a.qt_inter[v - 1][split] + c.st[0] * n);
  const int s0 = c.st[0], s1 = pick<VMAX>(c.st, 1);
  const int64_t pair = (int64_t)s0 * (2 * S - s0 - 1) / 2 + (s1 - s0 - 1);
  return (int)(a.qt_merge[split] + pair * n);
}

// Table-driven simulation of one candidate per group (INTER or MERGE at v <= 2). Durations and
// weights must fit 32 bits; a candidate with a larger one, or whose times pass the 40-bit
// slots, is recomputed on the 64-bit path.
template <int VMAX, int X>
__device__ __forceinline__ void run_tab(const SimArgs& a, int64_t cand, int v, int gen,
                                        int split, uint8_t* lds_wave) {
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  const Table40 T{reinterpret_cast<uint32_t*>(lds_wave),
                  lds_wave + (size_t)a.slots * a.CPW * 4, __ffs(a.CPW) - 1, g < a.CPW ? g : 0};
  uint8_t* rec = lds_wave + (size_t)(g < a.CPW ? g : 0) * a.rec_stride;
  constexpr int SREC = X != XP ? 16 : 8;  // bytes per stream record
  uint8_t* strm = lds_wave + a.strm_off + lane_id() * SREC;
  const bool has = cand >= 0;
  const int S = P * v;
  const Ring ring = make_ring(M, a.ring);
  if (has) stage_record(rec, a.cands + cand * a.pr.stride, a.rec_bytes, d, G);
  __asm__ volatile("" ::: "memory");

  Chunks<VMAX> c;
  int64_t busy = 0, stat = 0;
  bool fits = true;
  const bool mine = has && d < P;
  if (mine) {
    busy = setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, split, ring, a.pre_mem, &stat,
                              X);
#pragma unroll
    for (int kind = 0; kind < 3; ++kind) {
#pragma unroll
      for (int k = 0; k < VMAX; ++k) {
        if (k < v) {
          const int64_t w = kind == KF ? c.wF[k] : kind == KB ? c.wB[k] : 0;
          const int64_t du = kind == KF ? c.dF[k] : kind == KB ? c.dB[k] : c.dW[k];
          fits = fits && (uint64_t)w <= 0xFFFFFFFFull && (uint64_t)du <= 0xFFFFFFFFull;
          uint8_t* rec_e = strm + (kind * v + k) * 64 * SREC;
          *reinterpret_cast<uint2*>(rec_e) = make_uint2((uint32_t)w, (uint32_t)du);
          if constexpr (X == XM) {
            const int64_t dm = kind == KF ? c.mA[k] : (kind == KB && split) ? 0 : -c.mA[k];
            *reinterpret_cast<int64_t*>(rec_e + 8) = dm;
          }
          if constexpr (X == XC) {
            const int64_t co = kind == KF ? c.cF[k] : kind == KB ? c.cB[k] : 0;
            const int cx = kind == KF ? c.xF[k] : kind == KB ? c.xB[k] : 0;
            fits = fits && (uint64_t)co <= 0xFFFFFFFFull;
            *reinterpret_cast<uint2*>(rec_e + 8) = make_uint2((uint32_t)co, (uint32_t)cx);
          }
        }
      }
    }
  } else {
    zero_chunks<VMAX>(c);
  }
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  const bool wide = (fold_groups(__ballot(!fits), G, lsb) & gbit) != 0;
  // idle lanes and candidates for the 64-bit path start on the table's final terminators
  const uint32_t row = (mine && !wide) ? (uint32_t)qt_row<VMAX>(a, gen, v, split, c)
                                       : (uint32_t)a.qt_end;
  __asm__ volatile("" ::: "memory");
  T.clear_all(S * qt_row_stride(ring), lane_id(), WAVE);
  __asm__ volatile("" ::: "memory");

  bool dead = false;
  int64_t clock = 0, mem = 0, peak = 0;
  CommTally cm;
  cm.reset();
  int64_t fs = -1;
  relax_tab<X>(a.qtab, row, qt_row_stride(ring) << T.lg, strm, clock, T, G, gbit, lsb, dead, mem,
               peak, cm, fs);

  const int64_t ms = group_max(clock, G);
  CommTally tot = cm;
  if constexpr (X == XC) tot = group_tally(cm, G);
  if (mine) {
    if (wide || ms >= Table40::LIMIT) {
      if (d == 0) a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
    } else {
      put_results<X>(a, cand, d, dead, ms, busy, stat, peak, tot, fs, clock);
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Kernels
// ---------------------------------------------------------------------------------------------

// mem (nullable): layer memory [L][2], its prefix sums go to pre_mem. The block loads the
// tables into LDS first (L <= 255), so the serial sums wait on LDS, not on a global load and
// store per layer.
__global__ void k_prep(const int64_t* __restrict__ costs, const int64_t* __restrict__ mem, int L,
                       int64_t* __restrict__ pre, int64_t* __restrict__ pre_mem,
                       int32_t* __restrict__ ctl) {
  __shared__ int64_t sc[3 * 255], sm[2 * 255];
  const int t = threadIdx.x;
  for (int i = t; i < CTL_WORDS; i += blockDim.x) ctl[i] = 0;
  for (int i = t; i < 3 * L; i += blockDim.x) sc[i] = costs[i];
  if (mem)
    for (int i = t; i < 2 * L; i += blockDim.x) sm[i] = mem[i];
  __syncthreads();
  if (t < 3) {
    int64_t acc = 0;
    pre[t] = 0;
    for (int l = 0; l < L; ++l) {
      acc += sc[3 * l + t];
      pre[3 * (l + 1) + t] = acc;
    }
  } else if (t < 5 && mem) {
    const int c = t - 3;
    int64_t acc = 0;
    pre_mem[c] = 0;
    for (int l = 0; l < L; ++l) {
      acc += sm[2 * l + c];
      pre_mem[2 * (l + 1) + c] = acc;
    }
  }
}

// Ideal start times of the stage-level pipeline for MERGE: one block (one wave) per (v, split);
// lane s = stage s on its own virtual device running 1F1B (warm-up min(S-1-s, M)), with the
// split backward's W lagging s B's; unit durations, no transfer cost. Entry layout
// rec[s][pos] = start << 16 | kind << 12 | m.
__global__ void k_merge_tab(int P, int M, int v_lo, int v_hi, uint32_t* __restrict__ mtab) {
  extern __shared__ __align__(16) uint8_t smem[];
  const int v = v_lo + (int)(blockIdx.x >> 1);
  const int split = (int)(blockIdx.x & 1);
  if (v > v_hi) return;
  const int S = P * v;
  const int d = lane_id();
  const Table64 T{reinterpret_cast<int64_t*>(smem)};
  const int rowlen = (split ? 3 : 2) * M;
  uint32_t* tab = mtab + merge_offset(P, M, v, split);
  const Ring ring = make_ring(M, M);
  T.clear(S * M, d, WAVE);
  __asm__ volatile("" ::: "memory");
  Chunks<1> c;
  zero_chunks<1>(c);
  c.st[0] = d;
  c.base[0] = d * M;
  c.frow[0] = d > 0 ? -M : 0;
  c.fmask[0] = d > 0 ? (int)(ST_F | ST_PAR) : 0;
  c.brow[0] = d < S - 1 ? M : 0;
  c.bmask[0] = (int)((d < S - 1 ? ST_B : ST_F) | ST_PAR);
  c.dF[0] = 1;
  c.dB[0] = split ? 1 : 2;
  c.dW[0] = 1;
  Lane L;
  L.clock = 0;
  L.pos = 0;
  L.nops = d < S ? rowlen : 0;
  GenInter g;
  g.init(S, 1, M, d < S ? d : 0, split, split ? d : 0);
  describe<1>(L, c, ring, g.kind, g.k, g.m);
  bool dead = false;
  relax<1, true, false>(g, c, ring, L, T, WAVE, 1ull, 1ull, dead,
                        d < S ? tab + d * rowlen : nullptr);
}

__global__ void k_fill_u32(uint32_t* __restrict__ p, int n, uint32_t x) {
  for (int i = threadIdx.x; i < n; i += blockDim.x) p[i] = x;
}

__global__ void k_fill_i64(int64_t* __restrict__ p, int64_t n, int64_t x) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x)
    p[i] = x;
}

// Queue-table rows of the interleaved order (v <= 2) for one launch geometry: thread r writes
// rank r's queue; chunk k of rank r is stage r + k P.
__global__ void k_qtab_inter(uint32_t* __restrict__ out, int P, int v, int M, int split, int R,
                             int lg) {
  const int r = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (r >= P) return;
  const int n = (split ? 3 : 2) * v * M, S = P * v;
  const Ring ring = make_ring(M, R);
  uint32_t* row = out + (int64_t)r * (n + 2);
  GenInter g;
  g.init(P, v, M, r, split, split ? r : 0);
  for (int i = 0; i < n; ++i) {
    row[i] = qt_entry(g.kind, g.k, g.m, v, r + g.k * P, S, ring, lg);
    g.advance(true);
  }
  row[n] = row[n + 1] = QT_END;
}

// Queue-table rows of the MERGE order at v = 2: thread i writes the queue of stage pair i
// (pairs s0 < s1 in lexicographic order).
__global__ void k_qtab_merge(uint32_t* __restrict__ out, const uint32_t* __restrict__ mtab,
                             int P, int M, int split, int R, int lg) {
  const int S = 2 * P;
  const int i = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (i >= S * (S - 1) / 2) return;
  int s0 = 0, rem = i;
  while (rem >= S - 1 - s0) rem -= S - 1 - s0, ++s0;
  const int s1 = s0 + 1 + rem;
  const int rowlen = (split ? 3 : 2) * M, n = 2 * rowlen;
  const Ring ring = make_ring(M, R);
  uint32_t* row = out + (int64_t)i * (n + 2);
  GenMerge<2> g;
  g.init(mtab + merge_offset(P, M, 2, split), rowlen, 2, [&](int k) { return k == 0 ? s0 : s1; });
  for (int j = 0; j < n; ++j) {
    row[j] = qt_entry(g.kind, g.k, g.m, 2, g.k == 0 ? s0 : s1, S, ring, lg);
    g.advance(true);
  }
  row[n] = row[n + 1] = QT_END;
}

// Add one to hist[key] for every lane with `active`, one LDS atomic per distinct key of the
// wave; returns the lane's index among the wave's additions to its key (valid when active).
__device__ __forceinline__ int wave_hist_add(int* hist, int key, bool active) {
  const int lane = lane_id();
  const uint64_t below = (1ull << lane) - 1;
  uint64_t rem = __ballot(active);
  int mine = 0;
  while (rem) {
    const int leader = __ffsll((unsigned long long)rem) - 1;
    const int k = __shfl(key, leader);
    const uint64_t grp = __ballot(active && key == k);
    int base = 0;
    if (lane == leader) base = atomicAdd(&hist[k], __popcll(grp));
    base = __shfl(base, leader);
    if (active && key == k) mine = base + __popcll(grp & below);
    rem &= ~grp;
  }
  return mine;
}

// Records to evaluate: a.n, or fewer when a count on the device says so.
__device__ __forceinline__ int64_t live_count(const SimArgs& a) {
  if (!a.n_live) return a.n;
  const int64_t l = *a.n_live;
  return l < a.n ? l : a.n;
}

// One thread per candidate, blocks of CLS_THREADS taking CLS_ITEMS runs of CLS_THREADS
// candidates each, so that each block adds its bin counts to the global counters once for all
// its runs (one global atomic per bin and block: with one block per run, thousands of blocks
// queue on the same few counters). The records' heads (first hb bytes: header, boundaries,
// placement) are staged through LDS with 16-byte coalesced loads.
constexpr int CLS_THREADS = 256, CLS_ITEMS = 4;
__global__ void __launch_bounds__(CLS_THREADS) k_classify(SimArgs a, uint8_t* __restrict__ bins,
                                                          int hb) {
  extern __shared__ __align__(16) uint8_t heads[];
  __shared__ int hist[NBINS];
  for (int i = threadIdx.x; i < NBINS; i += blockDim.x) hist[i] = 0;
  const int64_t n = live_count(a);
  const int q = hb / 16, stride16 = a.pr.stride / 16;
  for (int run = 0; run < CLS_ITEMS; ++run) {
    const int64_t first = ((int64_t)blockIdx.x * CLS_ITEMS + run) * CLS_THREADS;
    const int cnt = first >= n ? 0 : (int)(n - first < CLS_THREADS ? n - first : CLS_THREADS);
    const uint4* src = reinterpret_cast<const uint4*>(a.cands + first * a.pr.stride);
    uint4* dst = reinterpret_cast<uint4*>(heads);
    __syncthreads();  // the previous run's heads are read
    for (int j = threadIdx.x; j < cnt * q; j += CLS_THREADS) {
      const int r = j / q, c = j - r * q;
      dst[j] = src[(int64_t)r * stride16 + c];
    }
    __syncthreads();
    const int64_t i = first + threadIdx.x;
    int bin = BIN_NONE;
    if (threadIdx.x < cnt) {
      const Resolved r = resolve_record(a.pr, heads + threadIdx.x * hb,
                                        a.cands + i * a.pr.stride + pert_off(a.pr.s_max));
      if (!r.valid) {
        a.out_ms[i] = OCTO_MS_INVALID;
        for (int d = 0; d < a.pr.P; ++d) a.out_bub[i * a.pr.P + d] = OCTO_MS_INVALID;
        if (a.out_peak)
          for (int d = 0; d < a.pr.P; ++d) a.out_peak[i * a.pr.P + d] = OCTO_MS_INVALID;
        if (a.out_comm)
          for (int k = 0; k < 4; ++k) a.out_comm[i * 4 + k] = OCTO_MS_INVALID;
        if (a.out_bound)
          for (int k = 0; k < 2 * a.pr.P; ++k) a.out_bound[i * 2 * a.pr.P + k] = OCTO_MS_INVALID;
      } else {
        bin = r.n_pert > 0 ? BIN_MAT + mat_sub(r.v, r.split) : bin_of(r.v, r.gen, r.split);
        if (a.smeta) {
          const int sc = static_class(a.pr, heads + threadIdx.x * hb + 3 + a.pr.s_max, r);
          if (sc >= 0 && a.smeta[4 * sc] != 0) bin = BIN_STATIC + sc;
        }
      }
      bins[i] = (uint8_t)bin;
    }
    wave_hist_add(hist, bin, bin != BIN_NONE);
  }
  __syncthreads();
  for (int b = threadIdx.x; b < NBINS; b += blockDim.x)
    if (hist[b]) atomicAdd(&a.ctl[CTL_COUNTS + b], hist[b]);
}

// One wave: first position of every bin in the index array (exclusive prefix sum), kept in
// CTL_START and copied to the scatter cursors.
__global__ void k_plan(int32_t* __restrict__ ctl) {
  if (threadIdx.x == 0) {
    int acc = 0;
    for (int b = 0; b < NBINS; ++b) {
      ctl[CTL_START + b] = ctl[CTL_POS + b] = acc;
      acc += ctl[CTL_COUNTS + b];
    }
    ctl[CTL_TOTAL] = acc;
  }
}

// Index of every valid record at its bin's cursor; blocks cover the same CLS_ITEMS runs as
// k_classify: counting the runs' bins gives each record its place among the block's records of
// its bin, one global atomic per bin reserves the block's positions, then every record is
// written at the block's position plus its place (the order inside a block's range follows the
// order in which its waves counted; every consumer handles its bin's records independently).
__global__ void __launch_bounds__(CLS_THREADS) k_scatter(SimArgs a, const uint8_t* __restrict__ bins,
                                                         int32_t* __restrict__ idx) {
  __shared__ int hist[NBINS];
  __shared__ int res[NBINS];
  for (int b = threadIdx.x; b < NBINS; b += blockDim.x) hist[b] = 0;
  __syncthreads();
  const int64_t n = live_count(a);
  const int64_t first = (int64_t)blockIdx.x * CLS_ITEMS * CLS_THREADS + threadIdx.x;
  int bin[CLS_ITEMS], local[CLS_ITEMS];
#pragma unroll
  for (int run = 0; run < CLS_ITEMS; ++run) {
    const int64_t i = first + run * CLS_THREADS;
    bin[run] = i < n ? bins[i] : BIN_NONE;
  }
#pragma unroll
  for (int run = 0; run < CLS_ITEMS; ++run)
    local[run] = wave_hist_add(hist, bin[run], bin[run] != BIN_NONE);
  __syncthreads();
  for (int b = threadIdx.x; b < NBINS; b += blockDim.x)
    res[b] = hist[b] ? atomicAdd(&a.ctl[CTL_POS + b], hist[b]) : 0;
  __syncthreads();
#pragma unroll
  for (int run = 0; run < CLS_ITEMS; ++run)
    if (bin[run] != BIN_NONE) idx[res[bin[run]] + local[run]] = (int32_t)(first + run * CLS_THREADS);
}

// The chunks of the bins in `mask` (bins < nbins <= 64), one bin per lane: its candidate count,
// first position in the index array and the end of its chunk range (an inclusive prefix over the
// bins in order; bins outside the mask have none). Built once per wave from the control block.
struct ChunkMap {
  int cnt, start, nch, end;
  __device__ __forceinline__ void init(const int32_t* ctl, int CPW, uint64_t mask, int nbins) {
    const int b = lane_id();
    const bool in = b < nbins && ((mask >> b) & 1);
    cnt = in ? ctl[CTL_COUNTS + b] : 0;
    start = b < nbins ? ctl[CTL_START + b] : 0;
    nch = (cnt + CPW - 1) / CPW;
    end = nch;
    for (int off = 1; off < WAVE; off <<= 1) {
      const int y = __shfl_up(end, off, WAVE);
      end += b >= off ? y : 0;
    }
  }
  // Bin of chunk ch (wave-uniform), or -1 past the last chunk; entry0: its first entry in the
  // bin, pos0: the bin's first index position, count: the bin's candidates.
  __device__ __forceinline__ int locate(int ch, int nbins, int CPW, int* entry0, int* pos0,
                                        int* count) const {
    const int b = __popcll(__ballot(lane_id() < nbins && end <= ch));
    if (b >= nbins) return -1;
    *count = __shfl(cnt, b, WAVE);
    *pos0 = __shfl(start, b, WAVE);
    *entry0 = (ch - (__shfl(end, b, WAVE) - __shfl(nch, b, WAVE))) * CPW;
    return b;
  }
};

template <int VMAX, int X>
__device__ __forceinline__ void dispatch_gen(const SimArgs& a, int gen, int64_t cand, int v,
                                             int split, uint8_t* lds_wave, int64_t* mbox) {
  const bool p2 = (a.pr.P & (a.pr.P - 1)) == 0 && (v & (v - 1)) == 0;
  if constexpr (X == XR) {  // rendezvous: GPipe queues run here too, with full rows
    if (gen == GEN_AFAB) {
      run_generated<VMAX, GEN_AFAB, false, X>(a, cand, v, split, lds_wave, mbox);
      return;
    }
  }
  if (gen == GEN_MERGE)
    run_generated<VMAX, GEN_MERGE, false, X>(a, cand, v, split, lds_wave, mbox);
  else if (p2)
    run_generated<VMAX, GEN_INTER, true, X>(a, cand, v, split, lds_wave, mbox);
  else
    run_generated<VMAX, GEN_INTER, false, X>(a, cand, v, split, lds_wave, mbox);
}

// Generated-queue simulation (INTER and MERGE) for the bins in a.bin_mask of one v class:
// VC = 1 (v = 1), 2 (v = 2) or 8 (v = 3..8); finish tables sized for that class with a.ring
// slots per row. X: XM also the peak activation memory per device, XC the communication tally.
template <int VC, int X>
__global__ void __launch_bounds__(WAVE) k_sim(SimArgs a) {
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int64_t mbox[X == XR ? WAVE : 1];  // rendezvous mailboxes
  const int g = lane_id() / a.G;
  const int d = lane_id() % a.G;
  ChunkMap cm;
  cm.init(a.ctl, a.CPW, a.bin_mask, NBIN_GEN);
  // chunks from a work counter: their rounds vary with each candidate's structure, and the
  // queue keeps the waves evenly loaded (these launches take few enough chunks that the
  // counter's atomics do not serialise them). The first chunk of every wave is its block index,
  // so a launch with little or no work takes no atomic at all.
  for (int first = 1;; first = 0) {
    int ch = (int)blockIdx.x;
    if (!first) {
      if (lane_id() == 0) ch = (int)gridDim.x + atomicAdd(&a.ctl[a.work], 1);
      ch = bcast(ch);
    }
    int entry0 = 0, pos0 = 0, cnt = 0;
    const int bin = cm.locate(ch, NBIN_GEN, a.CPW, &entry0, &pos0, &cnt);
    if (bin < 0) break;
    int v, gen, split;
    bin_decode(bin, &v, &gen, &split);
    const int e = entry0 + g;
    const int64_t cand = (g < a.CPW && e < cnt) ? (int64_t)a.idx[pos0 + e] : -1;
    if ((gen == GEN_AFAB && X != XR) || ((a.redo_bins >> bin) & 1)) {
      // queues that may hold more than a.ring micro-batches of a stage in flight
      if (cand >= 0 && d == 0) a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
      continue;
    }
    if constexpr (VC <= 2) {
      if (a.qtab) {
        run_tab<VC, X>(a, cand, v, gen, split, smem);
        continue;
      }
    }
    dispatch_gen<VC, X>(a, gen, cand, v, split, smem, mbox);
  }
}

// GPipe (AFAB) queues without moves. Every device runs the forwards of its stages in ascending
// stage order, each over m = 0..M-1, then the backwards in descending stage order. Visiting the
// stage rows in chain order — forwards s = 0..S-1, then backwards s = S-1..0 — therefore meets
// every device's ops in its queue order, and one row is one pass over m:
//   fin(s, m) = dur(s) + max(fin(s, m-1), in(s, m)),  fin(s, -1) = the device's clock;
//   in(s, m) = fin of micro-batch m in the row visited before (+ the link weight between the
// two stages' devices); F(0, m) has no input, B(S-1, m) takes F(S-1, m) from its own device.
// This is the earliest-start relaxation of the time model over the AFAB graph, in an order that
// reaches every op after all its predecessors. One lane per candidate; the previous row lives in
// LDS as M int64 per lane (lanes interleaved), device clocks and busy times after it.

// One row: row[m] <- f = dur + max(f, row[m] + w) for m = 0..M-1 (stride = lanes); returns f.
// Reads are issued eight at a time ahead of the dependent updates.
__device__ __forceinline__ int64_t sweep_row(int64_t* row, int stride, int M, int64_t f,
                                             int64_t w, int64_t dur) {
  int m = 0;
  for (; m + 8 <= M; m += 8) {
    int64_t x[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) x[i] = row[(m + i) * stride];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t y = x[i] + w;
      f = (y > f ? y : f) + dur;
      x[i] = f;
    }
#pragma unroll
    for (int i = 0; i < 8; ++i) row[(m + i) * stride] = x[i];
  }
  for (; m < M; ++m) {
    const int64_t y = row[m * stride] + w;
    f = (y > f ? y : f) + dur;
    row[m * stride] = f;
  }
  return f;
}

// The previous row of a k_afab lane: MMAX > 0 keeps it in registers (M == MMAX, the loop fully
// unrolled), MMAX = 0 in LDS (M int64 per lane, lanes interleaved).
template <int MMAX>
struct AfabRow {
  int64_t r[MMAX];
  __device__ __forceinline__ bool overflow() const { return false; }
  __device__ __forceinline__ void init(uint8_t*, int, int) {}
  __device__ __forceinline__ void clear(int) {
#pragma unroll
    for (int m = 0; m < MMAX; ++m) r[m] = 0;
  }
  __device__ __forceinline__ int64_t first() const { return r[0]; }
  __device__ __forceinline__ int64_t sweep(int, int64_t f, int64_t w, int64_t dur) {
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
      const int64_t y = r[m] + w;
      f = (y > f ? y : f) + dur;
      r[m] = f;
    }
    return f;
  }
  // the same row with each output queued on a link (XS): lf = the link's free time; the row
  // then holds the arrival times
  __device__ __forceinline__ int64_t sweep_s(int, int64_t f, int64_t w, int64_t dur,
                                             int64_t cout, int64_t& lf) {
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
      const int64_t y = r[m] + w;
      f = (y > f ? y : f) + dur;
      lf = (f > lf ? f : lf) + cout;
      r[m] = lf;
    }
    return f;
  }
  // the same row, tallying each op's communication nodes (flags cx, output transfer cout)
  __device__ __forceinline__ int64_t sweep_c(int, int64_t f, int64_t w, int64_t dur, int cx,
                                             int64_t cout, CommTally& ct) {
#pragma unroll
    for (int m = 0; m < MMAX; ++m) {
      const int64_t y = r[m] + w;
      const int64_t st = y > f ? y : f;
      ct.op(true, cx, y, w, f, st, st + dur, cout);
      f = st + dur;
      r[m] = f;
    }
    return f;
  }
};
template <>
struct AfabRow<0> {
  int64_t* row;
  int stride;
  __device__ __forceinline__ bool overflow() const { return false; }
  __device__ __forceinline__ void init(uint8_t* base, int li, int lanes) {
    row = reinterpret_cast<int64_t*>(base) + li;
    stride = lanes;
  }
  __device__ __forceinline__ void clear(int M) {
    for (int m = 0; m < M; ++m) row[m * stride] = 0;
  }
  __device__ __forceinline__ int64_t first() const { return row[0]; }
  __device__ __forceinline__ int64_t sweep(int M, int64_t f, int64_t w, int64_t dur) {
    return sweep_row(row, stride, M, f, w, dur);
  }
  __device__ __forceinline__ int64_t sweep_s(int M, int64_t f, int64_t w, int64_t dur,
                                             int64_t cout, int64_t& lf) {
    for (int m = 0; m < M; ++m) {
      const int64_t y = row[m * stride] + w;
      f = (y > f ? y : f) + dur;
      lf = (f > lf ? f : lf) + cout;
      row[m * stride] = lf;
    }
    return f;
  }
  __device__ __forceinline__ int64_t sweep_c(int M, int64_t f, int64_t w, int64_t dur, int cx,
                                             int64_t cout, CommTally& ct) {
    for (int m = 0; m < M; ++m) {
      const int64_t y = row[m * stride] + w;
      const int64_t st = y > f ? y : f;
      ct.op(true, cx, y, w, f, st, st + dur, cout);
      f = st + dur;
      row[m * stride] = f;
    }
    return f;
  }
};

// Input weight of the first stage's forwards: their row holds zeros, so any value this far below
// zero leaves fin(0, m) = dur + fin(0, m - 1).
constexpr int64_t AFAB_NO_INPUT = -((int64_t)1 << 62);

// A row of a k_afab lane as the upper envelope of at most K lines over 0 <= m < M (the plain,
// memory and bounds variants). A row's finishes f(m) = max(f(m - 1), r(m) + w) + dur unroll to
// the largest of c + (m + 1) dur (c: the device clock before the row) and, over k <= m, of
// r(k) + w + (m - k + 1) dur. With the previous row r(k) = max_i (a_i + k b_i), the largest
// a_i + k b_i + (m - k) dur over k <= m is a_i + m max(b_i, dur) (at k = m or k = 0), so f is
// again a maximum of lines: every line with b_i <= dur joins the clock in one line of slope dur,
// (max(c, a_i + w) + dur) + m dur, and each steeper one keeps its slope, shifted by w + dur. A
// steeper line no higher than the joined one at m = M - 1 stays under it on the whole row and is
// dropped. Each line is kept as its values at m = 0 and m = M - 1 and its slope, so a row costs
// one multiplication. Exact; a candidate whose envelope needs more than K lines (slopes that no
// later row's duration reaches) is flagged and goes to the 64-bit redo list. The first row (r = 0
// everywhere) is the line (0, 0); an empty slot is the line AFAB_EMPTY of slope 0.
constexpr int64_t AFAB_EMPTY = -((int64_t)1 << 62);
template <int K>
struct AfabLines {
  int64_t v0[K], v1[K], b[K];
  bool over;
  __device__ __forceinline__ void init(uint8_t*, int, int) {}
  __device__ __forceinline__ void clear(int) {
#pragma unroll
    for (int i = 0; i < K; ++i) v0[i] = v1[i] = i == 0 ? 0 : AFAB_EMPTY, b[i] = 0;
    over = false;
  }
  __device__ __forceinline__ bool overflow() const { return over; }
  __device__ __forceinline__ int64_t first() const {
    int64_t x = v0[0];
#pragma unroll
    for (int i = 1; i < K; ++i) x = v0[i] > x ? v0[i] : x;
    return x;
  }
  __device__ __forceinline__ int64_t sweep(int M, int64_t c, int64_t w, int64_t dur) {
    int64_t low = c;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const int64_t y = v0[i] + w;
      low = b[i] <= dur && y > low ? y : low;
    }
    const int64_t n0 = low + dur, n1 = n0 + (int64_t)(M - 1) * dur;
    int64_t fend = n1;
    bool placed = false;
#pragma unroll
    for (int i = 0; i < K; ++i) {
      const int64_t s0 = v0[i] + w + dur, s1 = v1[i] + w + dur;
      const bool keep = b[i] > dur && s1 > n1;
      const bool put = !keep && !placed;
      v0[i] = keep ? s0 : put ? n0 : AFAB_EMPTY;
      v1[i] = keep ? s1 : put ? n1 : AFAB_EMPTY;
      b[i] = keep ? b[i] : put ? dur : 0;
      fend = keep && s1 > fend ? s1 : fend;
      placed = placed || put;
    }
    over = over || !placed;
    return fend;
  }
};

// XM: a GPipe device holds every micro-batch of all its stages after its forwards, so its peak
// is its static bytes + M x its stages' activation bytes. XC: rows tally communication nodes,
// each device's last op start and pending transfer end kept after its clock and busy time. XS:
// a row whose outputs cross devices queues them on its link, whose free time it takes from the
// latest earlier row on the same directed link (rows are visited in every device's op order,
// so that is the link's issue order); the row then holds arrival times, read with weight 0.
// MMAX: -1 rows as line envelopes (AfabLines), else AfabRow<MMAX>.
template <int MMAX>
struct AfabRowOf {
  using type = AfabRow<MMAX>;
};
template <>
struct AfabRowOf<-1> {
  using type = AfabLines<8>;
};
template <int MMAX, int X>
__global__ void __launch_bounds__(WAVE) k_afab(SimArgs a, int lanes, int tab_off, int rec_off) {
  constexpr bool MEM = X == XM;
  extern __shared__ __align__(16) uint8_t smem[];
  const int lane = lane_id();
  const int P = a.pr.P, M = a.pr.M, L = a.pr.L;
  const int li = lane < lanes ? lane : 0;
  typename AfabRowOf<MMAX>::type row;
  row.init(smem, li, lanes);
  int64_t* clk = reinterpret_cast<int64_t*>(smem) + (MMAX == 0 ? (size_t)M * lanes : 0) + li;
  int64_t* bsy = clk + (size_t)P * lanes;  // clk[d * lanes], bsy[d * lanes]
  // plain variant with up to eight devices: busy times in registers, not in LDS, so that more
  // waves fit a CU
  const bool breg = X == XP && P <= 8;
  int64_t bus[8];
  int64_t* pk = bsy + (size_t)P * lanes;   // MEM: peak bytes pk[d * lanes]
  int64_t* cps = bsy + (size_t)P * lanes;  // XC: last op start cps[d * lanes], then
  int64_t* cpe = cps + (size_t)P * lanes;  //     pending transfer end cpe[d * lanes]
  int64_t* lfr = bsy + (size_t)P * lanes;  // XS: link free time after row t, lfr[t * lanes]
  int64_t* bfs = bsy + (size_t)P * lanes;  // XB: first start bfs[d * lanes] (-1 before)
  // line-envelope rows and serialised links: the prefix sums of the layer costs (and of the
  // memory model), the link matrix and each lane's record head are staged in LDS after the
  // lanes' arrays, since every row reads them (the communication-accounting rows, whose LDS
  // already bounds their occupancy, read them from global memory: staging cost them 14%)
  constexpr bool STAGE = MMAX < 0 || X == XS;
  const int64_t* pre = a.pre;
  const int64_t* pmem = a.pre_mem;
  const int64_t* link = a.link;
  if constexpr (STAGE) {
    int64_t* pre_l = reinterpret_cast<int64_t*>(smem + tab_off);
    int64_t* pmem_l = pre_l + 3 * (L + 1);
    int64_t* link_l = pmem_l + (MEM ? 2 * (L + 1) : 0);
    for (int i = lane; i < 3 * (L + 1); i += WAVE) pre_l[i] = a.pre[i];
    if constexpr (MEM)
      for (int i = lane; i < 2 * (L + 1); i += WAVE) pmem_l[i] = a.pre_mem[i];
    for (int i = lane; i < P * P; i += WAVE) link_l[i] = a.link[i];
    __syncthreads();
    pre = pre_l, pmem = pmem_l, link = link_l;
  }
  ChunkMap cmap;
  cmap.init(a.ctl, lanes, a.bin_mask, NBIN_GEN);
  // chunks by grid stride: AFAB candidates of one bin cost alike, and an atomic work counter
  // would serialise the waves
  for (int ch = (int)blockIdx.x;; ch += (int)gridDim.x) {
    int entry0 = 0, pos0 = 0, cnt = 0;
    const int bin = cmap.locate(ch, NBIN_GEN, lanes, &entry0, &pos0, &cnt);
    if (bin < 0) break;
    int v, gen, split;
    bin_decode(bin, &v, &gen, &split);
    const int e = entry0 + lane;
    if (lane >= lanes || e >= cnt) continue;
    const int64_t cand = a.idx[pos0 + e];
    // the record's head (header, boundaries, placement); staged in LDS with the tables
    const uint8_t* rec = a.cands + cand * a.pr.stride;
    if constexpr (STAGE) {
      const int hq = (pert_off(a.pr.s_max) + 15) / 16;
      uint8_t* rec_l = smem + rec_off + (size_t)lane * hq * 16;
      const uint4* src = reinterpret_cast<const uint4*>(rec);
      for (int j = 0; j < hq; ++j) reinterpret_cast<uint4*>(rec_l)[j] = src[j];
      rec = rec_l;
    }
    const uint8_t* bnd = rec + 4;
    const uint8_t* dev = rec + 3 + a.pr.s_max;
    const int S = P * v;
#pragma unroll
    for (int k = 0; k < 8; ++k) bus[k] = 0;
    for (int d = 0; d < P; ++d) {
      clk[d * lanes] = 0;
      if (!breg) bsy[d * lanes] = 0;
      if constexpr (MEM) pk[d * lanes] = 0;
      if constexpr (X == XC) cps[d * lanes] = 0, cpe[d * lanes] = -1;
      if constexpr (X == XB) bfs[d * lanes] = -1;
    }
    CommTally acc;
    acc.reset();
    row.clear(M);
    // rows t = 0..S-1: forwards of stage t; t = S..2S-1: backwards of stage 2S-1-t
    for (int t = 0; t < 2 * S; ++t) {
      const bool fwd = t < S;
      const int st = fwd ? t : 2 * S - 1 - t;
      const int d = dev[st];
      const int b0 = st > 0 ? bnd[st - 1] : 0, b1 = st < S - 1 ? bnd[st] : L;
      const int64_t df = pre[3 * b1] - pre[3 * b0];
      const int64_t db = pre[3 * b1 + 1] - pre[3 * b0 + 1] + pre[3 * b1 + 2] -
                         pre[3 * b0 + 2];
      if (fwd) {
        const int64_t cst = (df + db) * M;
        if (breg) {
#pragma unroll
          for (int k = 0; k < 8; ++k) bus[k] += d == k ? cst : 0;
        } else {
          bsy[d * lanes] += cst;
        }
      }
      if constexpr (MEM) {
        if (fwd)
          pk[d * lanes] += (pmem[2 * b1] - pmem[2 * b0]) * M +
                           pmem[2 * b1 + 1] - pmem[2 * b0 + 1];
      }
      // the stage whose finish times this row consumes: st - 1 (forward), st + 1 (backward)
      const int q = fwd ? st - 1 : st + 1;
      const int dq = q >= 0 && q < S && t != S ? dev[q] : d;
      const int64_t w = (fwd && st == 0) ? AFAB_NO_INPUT : dq != d ? link[dq * P + d] : 0;
      if constexpr (X == XB) {
        // the device's first op is micro-batch 0 of its first row
        if (bfs[d * lanes] < 0) {
          const int64_t y = row.first() + w;
          bfs[d * lanes] = y > clk[d * lanes] ? y : clk[d * lanes];
        }
      }
      if constexpr (X == XS) {
        const int o = fwd ? st + 1 : st - 1;
        const int dout = o >= 0 && o < S ? dev[o] : d;
        const int64_t wr = (fwd && st == 0) ? AFAB_NO_INPUT : 0;  // arrivals are in the row
        if (dout != d) {
          int64_t lf = 0;
          for (int u = 0; u < t; ++u) {
            const bool fu = u < S;
            const int su = fu ? u : 2 * S - 1 - u, ou = fu ? su + 1 : su - 1;
            if (dev[su] == d && ou >= 0 && ou < S && dev[ou] == dout)
              lf = lfr[u * lanes] > lf ? lfr[u * lanes] : lf;
          }
          clk[d * lanes] = row.sweep_s(M, clk[d * lanes], wr, fwd ? df : db,
                                       link[d * P + dout], lf);
          lfr[t * lanes] = lf;
        } else {
          clk[d * lanes] = row.sweep(M, clk[d * lanes], wr, fwd ? df : db);
          lfr[t * lanes] = 0;
        }
      } else if constexpr (X == XC) {
        // the stage this row's outputs go to: st + 1 (forward), st - 1 (backward)
        const int o = fwd ? st + 1 : st - 1;
        const int dout = o >= 0 && o < S ? dev[o] : d;
        const int cx = (dq != d ? CX_IN : 0) | (dout != d ? CX_OUT : 0);
        acc.pst = cps[d * lanes], acc.pend = cpe[d * lanes];
        clk[d * lanes] = row.sweep_c(M, clk[d * lanes], w, fwd ? df : db, cx,
                                     dout != d ? link[d * P + dout] : 0, acc);
        cps[d * lanes] = acc.pst, cpe[d * lanes] = acc.pend;
      } else {
        clk[d * lanes] = row.sweep(M, clk[d * lanes], w, fwd ? df : db);
      }
    }
    if (row.overflow()) {  // more lines than the envelope holds: the 64-bit path
      a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
      continue;
    }
    int64_t ms = 0;
    for (int d = 0; d < P; ++d) ms = clk[d * lanes] > ms ? clk[d * lanes] : ms;
    a.out_ms[cand] = ms;
    if (breg) {
#pragma unroll
      for (int k = 0; k < 8; ++k)
        if (k < P) a.out_bub[cand * P + k] = ms - bus[k];
    } else {
      for (int d = 0; d < P; ++d) a.out_bub[cand * P + d] = ms - bsy[d * lanes];
    }
    if constexpr (MEM)
      for (int d = 0; d < P; ++d) a.out_peak[cand * P + d] = pk[d * lanes];
    if constexpr (X == XC) {
      int64_t* oc = a.out_comm + cand * 4;
      oc[0] = acc.n, oc[1] = acc.nov, oc[2] = acc.t, oc[3] = acc.tov;
    }
    if constexpr (X == XB)
      for (int d = 0; d < P; ++d) {
        a.out_bound[(cand * P + d) * 2] = bfs[d * lanes] < 0 ? 0 : bfs[d * lanes];
        a.out_bound[(cand * P + d) * 2 + 1] = clk[d * lanes];
      }
  }
}

// ---------------------------------------------------------------------------------------------
// Static round schedules (structure classes, octo_device.hpp)
// ---------------------------------------------------------------------------------------------

__device__ __forceinline__ uint64_t wave_or(uint64_t x) {
  for (int off = WAVE / 2; off > 0; off >>= 1) x |= __shfl_xor(x, off, WAVE);
  return x;
}

// Node id of op (kind, s, m) among the 3 S M ops of a structure.
__device__ __forceinline__ int sc_node(int S, int M, int kind, int s, int m) {
  return (kind * S + s) * M + m;
}

// LDS bytes of k_static_build for (P, M): node rounds (int16) and slots (uint8) of the largest
// structure (v = 2, split), then every device's op list (uint32 per op).
__host__ __device__ inline size_t sc_build_lds(int P, int M) {
  const size_t nn = (size_t)3 * 2 * P * M;
  const size_t a = (nn * 2 + 15) / 16 * 16, b = (nn + 15) / 16 * 16;
  return a + b + (size_t)P * 6 * M * 4;
}

// One workgroup (one wave, lane = canonical device) per structure class: run the lockstep rounds
// of the class's structure once, costs aside — each round every device takes its next op if the
// op's producer ran in an earlier round — recording the round of each op; give every finish
// time that another device reads a slot for the rounds it is live (from its producer's round to
// its reader's: every such value has exactly one reader), lowest free slot first, a slot freed
// in a round being free for that round's writers (reads precede writes); then write every
// device's row of round entries. smeta[class] = {valid, rounds, slots used}; a class is invalid
// (its candidates take the generated-queue kernels) when its rounds pass nr_cap or it needs more
// than sc_neg(sc_slots(P)) slots. v = 2 classes need P v_max >= 2 P.
__global__ void __launch_bounds__(WAVE) k_static_build(int P, int M, int v_max,
                                                       const uint32_t* __restrict__ mtab,
                                                       uint32_t* __restrict__ stab,
                                                       int32_t* __restrict__ smeta,
                                                       int64_t cls_stride, int rowlen,
                                                       int nr_cap) {
  extern __shared__ __align__(16) uint8_t smem[];
  const int cls = blockIdx.x;
  int v, gen, split, pat;
  sc_decode(cls, &v, &gen, &split, &pat);
  uint32_t* rows = stab + cls * cls_stride;
  const int c = lane_id();
  const int ns = sc_slots(P), neg = sc_neg(ns), dummy = sc_dummy(ns);
  const uint32_t nop = sc_nop(ns);
  if (v > v_max) {
    for (int i = c; i < (P + 1) * rowlen; i += WAVE) rows[i] = nop;
    if (c == 0) smeta[4 * cls] = 0, smeta[4 * cls + 1] = 0, smeta[4 * cls + 2] = 0;
    return;
  }
  const int S = P * v, q = (split ? 3 : 2) * v * M;
  const int nn = 3 * 2 * P * M;
  int16_t* rnd = reinterpret_cast<int16_t*>(smem);
  uint8_t* slot = smem + ((size_t)nn * 2 + 15) / 16 * 16;
  uint32_t* ops = reinterpret_cast<uint32_t*>(slot + ((size_t)nn + 15) / 16 * 16);
  for (int i = c; i < nn; i += WAVE) rnd[i] = -1, slot[i] = (uint8_t)dummy;
  __syncthreads();
  const bool lane = c < P;
  int st0 = 0, st1 = 0;
  if (lane) sc_stages(pat, P, c, &st0, &st1);
  GenInter gi;
  GenMerge<2> gm;
  if (gen == GEN_INTER) {
    gi.init(P, v, M, lane ? st0 : 0, split, split ? (lane ? st0 : 0) : 0);
  } else {
    gm.init(mtab + merge_offset(P, M, 2, split), (split ? 3 : 2) * M, lane ? 2 : 0,
            [&](int k) { return k == 0 ? st0 : st1; });
  }
  // pass 1: the lockstep rounds
  int pos = 0, round = 0;
  for (;;) {
    const int kind = gen == GEN_INTER ? gi.kind : gm.kind;
    const int k = gen == GEN_INTER ? gi.k : gm.k;
    const int m = gen == GEN_INTER ? gi.m : gm.m;
    const int s = k == 0 ? st0 : st1;
    const bool has = lane && pos < q;
    int prod = -1;
    if (kind == KF) prod = s > 0 ? sc_node(S, M, KF, s - 1, m) : -1;
    else if (kind == KB) prod = s < S - 1 ? sc_node(S, M, KB, s + 1, m) : sc_node(S, M, KF, s, m);
    else prod = sc_node(S, M, KB, s, m);
    const bool ready = has && (prod < 0 || rnd[prod] >= 0);
    if (__ballot(ready) == 0 || round >= nr_cap) break;
    __asm__ volatile("" ::: "memory");
    if (ready) {
      rnd[sc_node(S, M, kind, s, m)] = (int16_t)round;
      ops[c * q + pos] = (uint32_t)round << 16 | (uint32_t)kind << 14 | (uint32_t)k << 11 |
                         (uint32_t)m;
      ++pos;
    }
    if (gen == GEN_INTER) gi.advance(ready);
    else gm.advance(ready);
    __asm__ volatile("" ::: "memory");
    ++round;
  }
  const int nrounds = round;
  bool valid = __ballot(lane && pos != q) == 0 && nrounds <= nr_cap;
  // pass 2: slots of the cross-device finish times, in round order
  uint64_t freem = (1ull << neg) - 1;  // slots 0 .. neg - 1
  uint64_t used = 0;
  int p2 = 0;
  for (int r = 0; valid && r < nrounds; ++r) {
    const uint32_t o = lane && p2 < q ? ops[c * q + p2] : 0xFFFFFFFFu;
    const bool act = lane && p2 < q && (int)(o >> 16) == r;
    const int kind = (o >> 14) & 3, k = (o >> 11) & 7, m = o & 0x7FF;
    const int s = k == 0 ? st0 : st1;
    // the op's input from another device: its one reader is this op, so the slot frees now
    int pin = -1;
    if (act && kind == KF && s > 0 && sc_device(pat, P, s - 1) != c) pin = sc_node(S, M, KF, s - 1, m);
    if (act && kind == KB && s < S - 1 && sc_device(pat, P, s + 1) != c)
      pin = sc_node(S, M, KB, s + 1, m);
    freem |= wave_or(pin >= 0 ? 1ull << slot[pin] : 0);
    // its output to another device needs a slot
    const bool out = act && ((kind == KF && s < S - 1 && sc_device(pat, P, s + 1) != c) ||
                             (kind == KB && s > 0 && sc_device(pat, P, s - 1) != c));
    const uint64_t wm = __ballot(out);
    if (__popcll(wm) > __popcll(freem)) {
      valid = false;
      break;
    }
    int sl = dummy;
    if (out) {
      uint64_t x = freem;
      const int rank = __popcll(wm & ((1ull << c) - 1));
      for (int i = 0; i < rank; ++i) x &= x - 1;
      sl = __ffsll((unsigned long long)x) - 1;
      slot[sc_node(S, M, kind, s, m)] = (uint8_t)sl;
    }
    const uint64_t took = wave_or(out ? 1ull << sl : 0);
    freem &= ~took;
    used |= took;
    p2 += act ? 1 : 0;
  }
  __syncthreads();
  // pass 3: the rows (role c; row P is all nop)
  for (int i = c; i < rowlen; i += WAVE) rows[(int64_t)P * rowlen + i] = nop;
  if (lane) {
    uint32_t* row = rows + (int64_t)c * rowlen;
    int p3 = 0;
    for (int r = 0; r < rowlen; ++r) {
      uint32_t e = nop;
      const uint32_t o = valid && p3 < q ? ops[c * q + p3] : 0xFFFFFFFFu;
      if (valid && p3 < q && (int)(o >> 16) == r) {
        const int kind = (o >> 14) & 3, k = (o >> 11) & 7, m = o & 0x7FF;
        const int s = k == 0 ? st0 : st1;
        int rd = neg;
        if (kind == KF && s > 0 && sc_device(pat, P, s - 1) != c)
          rd = slot[sc_node(S, M, KF, s - 1, m)];
        if (kind == KB && s < S - 1 && sc_device(pat, P, s + 1) != c)
          rd = slot[sc_node(S, M, KB, s + 1, m)];
        const int wr = kind == KW ? dummy : slot[sc_node(S, M, kind, s, m)];
        e = sc_entry(rd, kind * v + k, wr);
        ++p3;
      }
      row[r] = e;
    }
  }
  if (c == 0) {
    smeta[4 * cls] = valid ? 1 : 0;
    smeta[4 * cls + 1] = valid ? nrounds : 0;
    smeta[4 * cls + 2] = __popcll(used);
    smeta[4 * cls + 3] = 0;
  }
}

// Static-schedule evaluation: persistent waves take chunks of CPW candidates of one class bin;
// each lane runs its role's row of the class's schedule with its candidate's costs. Per round:
// read the slot its op reads and its stream's {input weight, duration}, start = max(device
// clock, slot + weight), finish = start + duration, write the finish to the slot its op writes.
// LDS: one 512-byte row per stream ({weight, duration} as two uint32 per lane; stream
// SC_NOP_STREAM is zero) from offset 0, so that a stream address is (entry & mask) | lane
// offset; then each group's ns = sc_slots(P) slots (64-bit, 8 ns bytes per group), then the
// staged records. The groups of a wave run one class, so in a round they read and write the same
// slot numbers: slot k of group g lives at k ^ (9g mod ns), which spreads the groups' accesses
// over the LDS banks (without it every group hits the same banks; of the XOR steps 4g, 5g, 7g,
// 9g and 13g, 9g measured fastest on the P = 8, M = 64 batch, 3 % ahead of 4g). A candidate
// whose weights or durations pass 32 bits goes to the 64-bit redo list.
typedef __attribute__((address_space(3))) int64_t lds_i64;
typedef __attribute__((address_space(3))) uint64_t lds_u64;
__global__ void __launch_bounds__(WAVE) k_static(SimArgs a, int sbase, int rbase) {
  extern __shared__ __align__(4096) uint8_t st_smem[];
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  const int gg = g < a.CPW ? g : 0;
  const uint32_t lb = (uint32_t)(uintptr_t)st_smem;  // LDS address of the array (4096-aligned)
  // group base | salt: slot addresses are (slot * 8) ^ sg
  const int ns = sc_slots(P);
  const uint32_t sg = (lb + (uint32_t)sbase + (uint32_t)(gg * ns) * 8u) |
                      (((uint32_t)gg * 72u) & (uint32_t)(8 * ns - 8));
  const uint32_t sb = lb + (uint32_t)lane_id() * 8u;
  uint8_t* rec = st_smem + rbase + gg * a.rec_stride;
  // the class bins' counts, first positions and chunk ranges, one class per lane
  const int ci = lane_id();
  const int cnt_i = ci < NSC ? a.ctl[CTL_COUNTS + BIN_STATIC + ci] : 0;
  const int start_i = ci < NSC ? a.ctl[CTL_START + BIN_STATIC + ci] : 0;
  const int nch_i = (cnt_i + a.CPW - 1) / a.CPW;
  int end_i = nch_i;  // inclusive prefix: chunks of classes 0..ci
  for (int off = 1; off < 16; off <<= 1) {
    const int y = __shfl_up(end_i, off, WAVE);
    end_i += ci >= off ? y : 0;
  }
  // chunks by grid stride, not by an atomic work counter: thousands of waves taking chunks of
  // a few hundred rounds would serialise on one counter's atomics. Chunks are in class order,
  // so each sweep of the grid hands every wave chunks of about one cost.
  for (int ch = (int)blockIdx.x;; ch += (int)gridDim.x) {
    // the class whose chunk range holds ch: the number of classes that end at or before it
    const int cls = __popcll(__ballot(ci < NSC && end_i <= ch));
    if (cls >= NSC) break;
    const int cnt = __shfl(cnt_i, cls, WAVE);
    const int pos0 = __shfl(start_i, cls, WAVE);
    const int entry0 = (ch - (__shfl(end_i, cls, WAVE) - __shfl(nch_i, cls, WAVE))) * a.CPW;
    int v, gen, split, pat;
    sc_decode(cls, &v, &gen, &split, &pat);
    const int e = entry0 + g;
    const int64_t cand = (g < a.CPW && e < cnt) ? (int64_t)a.idx[pos0 + e] : -1;
    const bool mine = cand >= 0 && d < P;
    if (cand >= 0) stage_record(rec, a.cands + cand * a.pr.stride, a.rec_bytes, d, G);
    __asm__ volatile("" ::: "memory");
    Chunks<2> c;
    int64_t busy = 0;
    bool fits = true;
    int role = P;
    if (mine) {
      busy = setup_chunks<2>(c, a.pr, rec, a.pre, a.link, d, v, split, make_ring(M, M));
      role = sc_role(pat, c.st[0]);
    } else {
      zero_chunks<2>(c);
    }
#pragma unroll
    for (int kind = 0; kind < 3; ++kind)
#pragma unroll
      for (int k = 0; k < 2; ++k) {
        const int64_t w = kind == KF ? c.wF[k] : kind == KB ? c.wB[k] : 0;
        const int64_t du = kind == KF ? c.dF[k] : kind == KB ? c.dB[k] : c.dW[k];
        fits = fits && (uint64_t)w <= 0xFFFFFFFFull && (uint64_t)du <= 0xFFFFFFFFull;
        if (k < v)
          *reinterpret_cast<lds_u64*>((uintptr_t)(sb + (uint32_t)(kind * v + k) * 512u)) =
              ((uint64_t)du << 32) | (uint32_t)w;
      }
    *reinterpret_cast<lds_u64*>((uintptr_t)(sb + SC_NOP_STREAM * 512u)) = 0;
    if (d == 0)
      *reinterpret_cast<lds_i64*>((uintptr_t)(((uint32_t)sc_neg(ns) * 8u) ^ sg)) =
          -((int64_t)1 << 62);
    uint64_t gbit, lsb;
    group_bits(G, &gbit, &lsb);
    const bool wide = (fold_groups(__ballot(!fits), G, lsb) & gbit) != 0;
    if (wide) role = P;
    const int nrounds = a.smeta[4 * cls + 1];
    const uint4* rowp = reinterpret_cast<const uint4*>(a.stab + cls * a.st_cls +
                                                       (int64_t)role * a.st_rowlen);
    __asm__ volatile("" ::: "memory");
    int64_t clock = 0;
    auto step = [&](uint32_t en) {
      const uint32_t ra = (en & 0x1F8u) ^ sg;
      const uint32_t sa = (en & 0xE00u) | sb;
      const uint32_t wa = ((en >> 9) & 0x1F8u) ^ sg;
      const int64_t x = *reinterpret_cast<const lds_i64*>((uintptr_t)ra);
      const uint64_t sr = *reinterpret_cast<const lds_u64*>((uintptr_t)sa);
      const int64_t tin = x + (int64_t)(uint32_t)sr;
      const int64_t st = tin > clock ? tin : clock;
      clock = st + (int64_t)(sr >> 32);
      *reinterpret_cast<lds_i64*>((uintptr_t)wa) = clock;
    };
    // blocks of four rounds, their entries loaded four blocks ahead (a row is L2-resident, so a
    // load takes far longer than one block of rounds); a row ends with four blocks of sc_nop,
    // so every look-ahead stays in it, and the rounds run in whole groups of four blocks (the
    // rounds past the class's last are sc_nop)
    uint4 q0 = rowp[0], q1 = rowp[1], q2 = rowp[2], q3 = rowp[3];
    auto block = [&](const uint4& q) {
      step(q.x);
      step(q.y);
      step(q.z);
      step(q.w);
    };
    for (int b = 0; b < nrounds; b += 16) {
      const int i = b >> 2;
      block(q0);
      q0 = rowp[i + 4];
      block(q1);
      q1 = rowp[i + 5];
      block(q2);
      q2 = rowp[i + 6];
      block(q3);
      q3 = rowp[i + 7];
    }
    const int64_t ms = group_max(clock, G);
    if (mine) {
      if (wide) {
        if (d == 0) a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
      } else {
        CommTally none;
        none.reset();
        put_results<XP>(a, cand, d, false, ms, busy, 0, 0, none);
      }
    }
    __asm__ volatile("" ::: "memory");
  }
}

// Generate one device queue into a global row (entry = kind << 14 | chunk << 11 | m), eight
// entries per 16-byte store. The row starts 16-byte aligned and holds n rounded up to a
// multiple of eight entries; the entries past n in the last span are written as 0.
template <class Gen>
__device__ __forceinline__ void emit_queue(Gen& g, uint16_t* row, int n) {
  uint4* r4 = reinterpret_cast<uint4*>(row);
  for (int i0 = 0; i0 < n; i0 += 8) {
    uint32_t w[4];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      uint32_t e = 0;
      if (i0 + u < n) {
        e = qpack(g.kind, g.k, g.m);
        g.advance(true);
      }
      w[u >> 1] = (u & 1) ? (w[u >> 1] | e << 16) : e;
    }
    r4[i0 >> 3] = make_uint4(w[0], w[1], w[2], w[3]);
  }
}

// Copy the first n entries of a queue row (both rows 16-byte aligned; whole 16-byte spans, the
// last one padded within the rows' capacities), eight spans in flight. The loads are
// unconditional (a block past the end re-reads the last span) so that the eight spans stay in
// registers and are waited for together.
__device__ __forceinline__ void copy_row(const uint16_t* src, uint16_t* dst, int n) {
  const uint4* s4 = reinterpret_cast<const uint4*>(src);
  uint4* d4 = reinterpret_cast<uint4*>(dst);
  const int spans = (n + 7) >> 3;
  for (int q0 = 0; q0 < spans; q0 += 8) {
    uint4 t0 = s4[min(q0 + 0, spans - 1)], t1 = s4[min(q0 + 1, spans - 1)];
    uint4 t2 = s4[min(q0 + 2, spans - 1)], t3 = s4[min(q0 + 3, spans - 1)];
    uint4 t4 = s4[min(q0 + 4, spans - 1)], t5 = s4[min(q0 + 5, spans - 1)];
    uint4 t6 = s4[min(q0 + 6, spans - 1)], t7 = s4[min(q0 + 7, spans - 1)];
    d4[q0] = t0;
    if (q0 + 1 < spans) d4[q0 + 1] = t1;
    if (q0 + 2 < spans) d4[q0 + 2] = t2;
    if (q0 + 3 < spans) d4[q0 + 3] = t3;
    if (q0 + 4 < spans) d4[q0 + 4] = t4;
    if (q0 + 5 < spans) d4[q0 + 5] = t5;
    if (q0 + 6 < spans) d4[q0 + 6] = t6;
    if (q0 + 7 < spans) d4[q0 + 7] = t7;
  }
}

// The v = 2 MERGE queue of a device hosting stages s0 < s1 (both splits), as materialise would
// generate it, for every stage pair: row (split * S + s0) * S + s1 of `rows`, S = 2P, `stride`
// entries apart. Built once per (P, v_max, M) beside the MERGE tables, so that materialising
// such a queue is a copy in 16-byte spans instead of a merge with one dependent table load per
// entry. One thread per row.
__global__ void k_merge_rows(int P, int M, const uint32_t* __restrict__ mtab,
                             uint16_t* __restrict__ rows, int stride) {
  const int S = 2 * P;
  const int t = (int)(blockIdx.x * blockDim.x + threadIdx.x);
  if (t >= 2 * S * S) return;
  const int split = t / (S * S), s0 = (t / S) % S, s1 = t % S;
  if (s0 >= s1) return;
  GenMerge<2> g;
  g.init(mtab + merge_offset(P, M, 2, split), (split ? 3 : 2) * M, 2,
         [&](int k) { return k == 0 ? s0 : s1; });
  emit_queue(g, rows + (size_t)t * stride, (split ? 3 : 2) * 2 * M);
}

// Materialise the queue of lane d for a staged record; returns the queue length.
template <int VMAX>
__device__ __forceinline__ int materialise(const SimArgs& a, const Chunks<VMAX>& c, int v,
                                           int gen, int split, uint16_t* row) {
  const int P = a.pr.P, M = a.pr.M;
  const int n = (split ? 3 : 2) * v * M;
  if (gen == GEN_AFAB) {
    GenAfab g;
    g.init(v, M);
    emit_queue(g, row, n);
  } else if (gen == GEN_INTER) {
    GenInter g;
    const int r = c.st[0];
    g.init(P, v, M, r, split, split ? r : 0);
    emit_queue(g, row, n);
  } else if (v == 2 && a.mrows) {
    const int S2 = 2 * P;
    copy_row(a.mrows + ((size_t)(split * S2 + c.st[0]) * S2 + c.st[1]) * a.mrow_stride, row, n);
  } else {
    GenMerge<VMAX> g;
    g.init(a.mtab + (v >= 2 ? merge_offset(P, M, v, split) : 0), (split ? 3 : 2) * M, v,
           [&](int k) { return pick<VMAX>(c.st, k); });
    emit_queue(g, row, n);
  }
  return n;
}

// Queue rows (the workspace's and the tuner's store) start 16-byte aligned and hold a multiple
// of eight entries (queue_capacity), so a row reads in whole 16-byte spans, several in flight.
// Entry u of a span (u a constant after unrolling).
__device__ __forceinline__ uint32_t span_entry(const uint4& b, int u) {
  const uint32_t w = u < 2 ? b.x : u < 4 ? b.y : u < 6 ? b.z : b.w;
  return (u & 1) ? w >> 16 : w & 0xFFFFu;
}

// Span q (of 16-byte spans) of a row of n entries, clamped to the row's last span.
__device__ __forceinline__ uint4 row_span(const uint16_t* row, int q, int n) {
  return reinterpret_cast<const uint4*>(row)[min(q, max(n - 1, 0) >> 3)];
}

// Window of a queue row: the largest m_i - m_j over entries i < j of one chunk (0 when no
// chunk's micro-batches ever go backwards). When the window of every device is below R, each op
// of micro-batch m precedes every op of m + R of the same stage.
template <int VMAX>
__device__ int queue_window(const uint16_t* row, int n) {
  int hi[VMAX];
#pragma unroll
  for (int k = 0; k < VMAX; ++k) hi[k] = 0;
  int w = 0;
  for (int i0 = 0; i0 < n; i0 += 32) {
    uint4 b[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) b[q] = row_span(row, (i0 >> 3) + q, n);
#pragma unroll
    for (int u = 0; u < 32; ++u) {
      const uint32_t e = span_entry(b[u >> 3], u & 7);
      const bool in = i0 + u < n;
      const int k = (int)(e >> 11) & 7, m = (int)(e & 0x7FF);
      const int h = pick<VMAX>(hi, k);
      w = (in && h - m > w) ? h - m : w;
#pragma unroll
      for (int c = 0; c < VMAX; ++c) hi[c] = (in && k == c && m > h) ? m : hi[c];
    }
  }
  return w;
}

// The finish table of one group: 40-bit slots (RING) or 64-bit, at the start of its LDS area.
template <bool RING>
__device__ __forceinline__ auto group_table(uint8_t* p, int slots) {
  if constexpr (RING)
    return Table40{reinterpret_cast<uint32_t*>(p), p + (size_t)slots * 4, 0, 0};
  else
    return Table64{reinterpret_cast<int64_t*>(p)};
}

// The rounds of one evaluation over a materialised queue row of capacity qcap entries: read QK
// rounds ahead (GenMatK) when the row holds at least eight entries, else one entry ahead;
// rendezvous transfers take their own rounds (mbox: their mailboxes).
template <int VMAX, int X, class Tab>
__device__ __forceinline__ void rounds_mat(const uint16_t* row, int qcap, const Chunks<VMAX>& c,
                                           const Ring& ring, Lane& L, const Tab& T, int G,
                                           uint64_t gbit, uint64_t lsb, bool& dead,
                                           int64_t* mbox) {
  if constexpr (X != XR) {
    if (qcap >= 8) {
      GenMatK<QK> q;
      q.init(row, qcap);
      describe<VMAX>(L, c, ring, q.kind, q.k, q.m);
      relax_k<VMAX, X>(q, c, ring, L, T, G, gbit, lsb, dead);
      return;
    }
  }
  GenMat q;
  q.init(row, L.nops);
  describe<VMAX>(L, c, ring, q.kind, q.k, q.m);
  rounds<VMAX, true, X>(q, c, ring, L, T, G, gbit, lsb, dead, mbox);
}

// Move row[from] so that it ends at index to.
// Eight entries are read before any is written, so that their loads are in flight together.
__device__ __forceinline__ void move_entry(uint16_t* row, int from, int to) {
  const uint16_t x = row[from];
  uint16_t t[8];
  int i = from;
  if (from < to) {
    for (; i + 8 <= to; i += 8) {
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = row[i + 1 + u];
#pragma unroll
      for (int u = 0; u < 8; ++u) row[i + u] = t[u];
    }
    for (; i < to; ++i) row[i] = row[i + 1];
  } else {
    for (; i - 8 >= to; i -= 8) {
#pragma unroll
      for (int u = 0; u < 8; ++u) t[u] = row[i - 1 - u];
#pragma unroll
      for (int u = 0; u < 8; ++u) row[i - u] = t[u];
    }
    for (; i > to; --i) row[i] = row[i - 1];
  }
  row[to] = x;
}

// Candidates with perturbations, then candidates whose times overflowed the 40-bit slots:
// queues materialised in global memory, moves applied, 64-bit finish tables.
template <int VMAX, int X>
__global__ void __launch_bounds__(WAVE) k_sim_mat(SimArgs a) {
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int64_t mbox[X == XR ? WAVE : 1];  // rendezvous mailboxes
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  uint8_t* lds_group = smem + (size_t)(g < a.CPW ? g : 0) * a.group_bytes;
  const Table64 T{reinterpret_cast<int64_t*>(lds_group)};
  uint8_t* rec = lds_group + a.table_bytes;
  const int slot = (int)blockIdx.x * a.CPW + (g < a.CPW ? g : 0);
  uint16_t* row = a.qscratch + ((size_t)slot * P + (d < P ? d : 0)) * a.qcap;
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  int base = 0;
  base = a.ctl[CTL_START + BIN_MAT];  // the perturbed bins are the last ones
  for (int phase = 0; phase < 2; ++phase) {
    const int32_t* list = phase == 0 ? a.idx + base : a.redo;
    const int cnt = phase == 0 ? a.ctl[CTL_TOTAL] - base : a.ctl[CTL_REDO];
    const int counter = phase == 0 ? CTL_WORK_MAT : CTL_WORK_REDO;
    if (cnt == 0 || !((a.mat_lists >> phase) & 1)) continue;  // no work here
    for (;;) {
      int ch = 0;
      if (lane_id() == 0) ch = atomicAdd(&a.ctl[counter], 1);
      ch = bcast(ch);
      if (ch * a.CPW >= cnt) break;
      const int e = ch * a.CPW + g;
      const int64_t cand = (g < a.CPW && e < cnt) ? (int64_t)list[e] : -1;
      const bool has = cand >= 0;
      const bool mine = has && d < P;
      const uint8_t* grec = has ? a.cands + cand * a.pr.stride : a.cands;
      if (has) stage_record(rec, grec, a.rec_bytes, d, G);
      __asm__ volatile("" ::: "memory");
      const int policy = has ? rec[0] : 0;
      const int v = has ? rec[1] : 1;
      const int split = policy == POL_ZB;
      int gen = GEN_AFAB;
      if (has) {
        Resolved r = resolve_record(a.pr, grec);
        gen = r.gen;
      }
      const int S = P * v;
      const Ring ring = make_ring(M, M);
      Chunks<VMAX> c;
      int64_t busy = 0, stat = 0;
      Lane L;
      L.clock = 0, L.pos = 0, L.nops = 0, L.mem = L.peak = 0;
      L.cm.reset();
      L.fs = -1;
      if constexpr (X == XS)
        for (int i = 0; i < 16; ++i) L.lf[i] = 0;
      if (mine) {
        busy = setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, split, ring, a.pre_mem,
                                  &stat, X);
        L.nops = materialise<VMAX>(a, c, v, gen, split, row);
        const uint8_t* pp = grec + pert_off(a.pr.s_max);
        const int np = grec[2];
        for (int i = 0; i < np; ++i) {
          const int pd = pp[6 * i] | (pp[6 * i + 1] << 8);
          if (pd != d) continue;
          const int from = pp[6 * i + 2] | (pp[6 * i + 3] << 8);
          const int to = pp[6 * i + 4] | (pp[6 * i + 5] << 8);
          move_entry(row, from, to);
        }
      } else {
        zero_chunks<VMAX>(c);
      }
      if (has) T.clear(S * M, d, G);
      __asm__ volatile("" ::: "memory");
      if constexpr (X == XR) mbox[lane_id()] = RDV_EMPTY;
      bool dead = false;
      rounds_mat<VMAX, X>(row, a.qcap, c, ring, L, T, G, gbit, lsb, dead, mbox);
      const int64_t ms = group_max(L.clock, G);
      CommTally tot = L.cm;
      if constexpr (X == XC) tot = group_tally(L.cm, G);
      if (mine) put_results<X>(a, cand, d, dead, ms, busy, stat, L.peak, tot, L.fs, L.clock);
    }
  }
}


// Candidates with perturbations, 40-bit slots shared by the wave's groups like the generated
// kernels (5 bytes a slot instead of 8, so more waves fit a CU), in rings of a.ring rows per
// stage (twice the window of the interleaved orders, so that orders a few moves away from a
// generated one fit; see k_tune_ring for why a ring is exact when the queue window is below
// it): queues materialised in global memory, moves applied. A candidate whose window reaches
// the ring joins the wide list, which a second launch (wide_pass, full rows: a.ring = M) takes;
// one whose times pass the 40-bit slots joins the redo list of the 64-bit kernel, which runs
// after both.
template <int VMAX, int X>
__global__ void __launch_bounds__(WAVE) k_sim_mat40(SimArgs a, int mode) {
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int64_t mbox[X == XR ? WAVE : 1];  // rendezvous mailboxes
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  const int gg = g < a.CPW ? g : 0;
  const Table40 T{reinterpret_cast<uint32_t*>(smem), smem + (size_t)a.slots * a.CPW * 4,
                  __ffs(a.CPW) - 1, gg};
  uint8_t* rec = smem + (size_t)gg * a.rec_stride;  // until the table is cleared
  const int slot = (int)blockIdx.x * a.CPW + gg;
  uint16_t* row = a.qscratch + ((size_t)slot * P + (d < P ? d : 0)) * a.qcap;
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  // mode bit 0: take the wide list of the ring pass, not the perturbed candidates of the bin
  // index; bit 1: send candidates wider than the ring to the redo list (no full-row pass)
  const bool wide_pass = (mode & 1) != 0;
  const int32_t* list = wide_pass ? a.wide : a.idx + a.ctl[CTL_START + BIN_MAT];
  const int cnt = wide_pass ? a.ctl[CTL_WIDE] : a.ctl[CTL_TOTAL] - a.ctl[CTL_START + BIN_MAT];
  const int work = wide_pass ? CTL_WORK_WIDE : CTL_WORK_MAT;
  if (cnt == 0) return;
  const Ring ring = make_ring(M, a.ring);
  for (;;) {
    int ch = 0;
    if (lane_id() == 0) ch = atomicAdd(&a.ctl[work], 1);
    ch = bcast(ch);
    if (ch * a.CPW >= cnt) break;
    const int e = ch * a.CPW + g;
    const int64_t cand = (g < a.CPW && e < cnt) ? (int64_t)list[e] : -1;
    const bool has = cand >= 0;
    const bool mine = has && d < P;
    const uint8_t* grec = has ? a.cands + cand * a.pr.stride : a.cands;
    if (has) stage_record(rec, grec, a.rec_bytes, d, G);
    __asm__ volatile("" ::: "memory");
    const int policy = has ? rec[0] : 0;
    const int v = has ? rec[1] : 1;
    const int split = policy == POL_ZB;
    int gen = GEN_AFAB;
    if (has) gen = resolve_record(a.pr, grec).gen;
    Chunks<VMAX> c;
    int64_t busy = 0, stat = 0;
    int wl = 0;
    Lane L;
    L.clock = 0, L.pos = 0, L.nops = 0, L.mem = L.peak = 0;
    L.cm.reset();
    L.fs = -1;
    if constexpr (X == XS)
      for (int i = 0; i < 16; ++i) L.lf[i] = 0;
    if (mine) {
      busy = setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, split, ring, a.pre_mem,
                                &stat, X);
      L.nops = materialise<VMAX>(a, c, v, gen, split, row);
      const uint8_t* pp = grec + pert_off(a.pr.s_max);
      const int np = grec[2];
      for (int i = 0; i < np; ++i) {
        const int pd = pp[6 * i] | (pp[6 * i + 1] << 8);
        if (pd != d) continue;
        move_entry(row, pp[6 * i + 2] | (pp[6 * i + 3] << 8), pp[6 * i + 4] | (pp[6 * i + 5] << 8));
      }
      if (ring.R < M) wl = queue_window<VMAX>(row, L.nops);
    } else {
      zero_chunks<VMAX>(c);
    }
    // a candidate whose order does not fit the ring goes to the wide list (full rows)
    const bool on_ring = group_max((int64_t)wl, G) < ring.R;
    if (!on_ring) {
      L.nops = 0;
      if (mine && d == 0) {
        if (mode & 2)
          a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
        else
          a.wide[atomicAdd(&a.ctl[CTL_WIDE], 1)] = (int32_t)cand;
      }
    }
    __asm__ volatile("" ::: "memory");
    T.clear_all(a.slots, lane_id(), WAVE);  // every candidate's rows fit a.slots
    __asm__ volatile("" ::: "memory");
    if constexpr (X == XR) mbox[lane_id()] = RDV_EMPTY;
    bool dead = false;
    rounds_mat<VMAX, X>(row, a.qcap, c, ring, L, T, G, gbit, lsb, dead, mbox);
    const int64_t ms = group_max(L.clock, G);
    CommTally tot = L.cm;
    if constexpr (X == XC) tot = group_tally(L.cm, G);
    if (mine && on_ring) {
      if (ms >= Table40::LIMIT) {
        if (d == 0) a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
      } else {
        put_results<X>(a, cand, d, dead, ms, busy, stat, L.peak, tot, L.fs, L.clock);
      }
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Deadlock-free reordered coordination (§7 "Unified Pipeline Executor"): every device keeps its
// compute order and places each transfer at its ideal start — its producer's end in the
// asynchronous schedule — with blocking rendezvous transfers. A device's program is its items
// sorted by (time, communication before computation, then the producer's id (kind, stage, m) for
// a transfer or the queue position for a computation); a compute item's time is its start.
// One group per candidate (lane = device), queues materialised, 64-bit finish table:
//   A. the plain rounds, recording each op's finish (by node) in the slot's time buffer;
//   B. each lane builds its program: computations and sends come in queue order already, its
//      receives (keyed by their producers' ends) are insertion-sorted, then the three merge;
//   C. rounds over the programs: a send first announces itself in the sender's outbox (once its
//      producer has finished), the receiver matches it, takes the transfer from max(sender's
//      announce time, its own clock) for the link time and posts the end to the sender's
//      mailbox; the sender resumes from there.
// ---------------------------------------------------------------------------------------------
constexpr uint32_t PI_COMP = 0, PI_SEND = 1, PI_RECV = 2;
// program item: type << 30 | op kind << 28 | stage << 16 | m; a transfer is named by its producer
__device__ __forceinline__ uint32_t pitem(uint32_t type, int kind, int s, int m) {
  return type << 30 | (uint32_t)kind << 28 | (uint32_t)s << 16 | (uint32_t)m;
}
constexpr int32_t OB_NONE = -1;

// Per-slot scratch of k_ordered.
// A communication item of the reordering: its key is (producer end, level, producer node);
// pk = level << 37 | node << 17 | receive << 16 | gap, so that comparing pk compares (level,
// node), which no two items of a lane share. Levels (lockstep rounds of a live group) and
// nodes are below 3 S M <= 3 * 64 * 2047 < 2^19; gaps are at most 3 v M < 2^16.
struct __align__(16) CItem {
  int64_t key;
  uint64_t pk;
};
__device__ __forceinline__ bool item_less(const CItem& a, const CItem& b) {
  return a.key != b.key ? a.key < b.key : a.pk < b.pk;
}

// Per-lane scratch of a wave, lane-interleaved: element i of lane l is at [i][l] of the wave's
// block, so that the lanes' accesses at one index share cache lines.
template <class T>
struct LaneArr {
  T* p;  // the lane's element 0
  __device__ __forceinline__ T& operator[](int i) const { return p[(size_t)i * WAVE]; }
};
template <class T>
__device__ __forceinline__ LaneArr<T> lane_arr(T* base, int cap) {
  return LaneArr<T>{base + (size_t)blockIdx.x * cap * WAVE + lane_id()};
}

struct OrdBufs {
  int64_t* tb;      // [slot][3 S_max M] finish time of each op (REORDER, phase C: arrivals)
  // the rest: [wave][cap][WAVE], lane-interleaved
  int64_t* rkey;    // rcap: receive keys (producer end)
  uint32_t* rid;    // rcap: receive producers (pitem with type 0)
  uint4* prog;      // pcap / 4: programs, four items per entry
  int rcap, pcap;
  // REORDER only
  int64_t* ts;      // [slot][3 S_max M] start time of each op
  int32_t* tl;      // [slot][3 S_max M] level of each op
  CItem* items;     // icap: in-order items from the front, mismatched ones from the back
  int64_t* pst;     // pcap2: post time of each gap (end of the computation before)
  int64_t* pdur;    // pcap2: durations of the computations before each gap
  int pcap2;
  int64_t* stats;   // [n][2] (nullable): transfers, mismatched receives
  int icap;
};

// Program writer: items gathered four at a time into one 16-byte store (a store is counted
// with the loads, so one per item would make every later load wait for its write).
struct ProgOut {
  LaneArr<uint4> prog;
  uint4 pk4;
  int n;
  __device__ __forceinline__ void init(LaneArr<uint4> p) { prog = p, pk4 = make_uint4(0, 0, 0, 0), n = 0; }
  __device__ __forceinline__ void emit(uint32_t item) {
    const int q = n & 3;
    pk4.x = q == 0 ? item : pk4.x;
    pk4.y = q == 1 ? item : pk4.y;
    pk4.z = q == 2 ? item : pk4.z;
    pk4.w = q == 3 ? item : pk4.w;
    if (q == 3) prog[n >> 2] = pk4;
    ++n;
  }
  __device__ __forceinline__ int finish() {  // the last, partial group of four
    if (n & 3) prog[n >> 2] = pk4;
    return n;
  }
};
__device__ __forceinline__ uint32_t prog_at(LaneArr<uint4> prog, int i) {
  return reinterpret_cast<const uint32_t*>(&prog[i >> 2])[i & 3];
}

// (t, cls, tie) < (t', cls', tie')
__device__ __forceinline__ bool key_less(int64_t t, uint32_t cls, uint32_t tie, int64_t t2,
                                         uint32_t cls2, uint32_t tie2) {
  return t != t2 ? t < t2 : cls != cls2 ? cls < cls2 : tie < tie2;
}

// The local chunk of stage s (hosted by this device; unused chunk slots hold stage 0, so only
// the device's v chunks are searched).
template <int VMAX>
__device__ __forceinline__ int chunk_of(const Chunks<VMAX>& c, int s, int v) {
  int k = 0;
#pragma unroll
  for (int i = 0; i < VMAX; ++i) k = (i < v && c.st[i] == s) ? i : k;
  return k;
}

// Entry j (0..7, a run-time value) of a 16-byte span: one select of a 64-bit half and a shift.
__device__ __forceinline__ uint32_t span_entry_at(const uint4& b, int j) {
  const uint64_t lo = (uint64_t)b.x | ((uint64_t)b.y << 32);
  const uint64_t hi = (uint64_t)b.z | ((uint64_t)b.w << 32);
  return (uint32_t)(((j & 4) ? hi : lo) >> ((j & 3) * 16)) & 0xFFFFu;
}

// A forward walk over a queue row that loads each 16-byte span once.
struct RowCursor {
  const uint16_t* row;
  int n, blk;
  uint4 b;
  __device__ __forceinline__ void init(const uint16_t* r, int n_) { row = r, n = n_, blk = -1; }
  __device__ __forceinline__ uint32_t at(int i) {
    if ((i >> 3) != blk) blk = i >> 3, b = row_span(row, blk, n);
    return span_entry_at(b, i & 7);
  }
};

// Phase B for lane d: returns the program length.
template <int VMAX>
__device__ __forceinline__ int build_program(const Chunks<VMAX>& c, const uint16_t* row, int nq,
                                             const int64_t* tb, int S, int M, LaneArr<int64_t> rkey,
                                             LaneArr<uint32_t> rid, LaneArr<uint4> prog) {
  auto node = [&](int kind, int s, int m) { return (kind * S + s) * M + m; };
  auto dur_of = [&](int kind, int k) {
    return kind == KF ? pick<VMAX>(c.dF, k) : kind == KB ? pick<VMAX>(c.dB, k) : pick<VMAX>(c.dW, k);
  };
  // receives in queue order, insertion-sorted by (producer end, producer): eight entries per
  // span, their producers' ends loaded together; a receive at or after the last one (the usual
  // case) is appended without reading the list back
  int nr = 0;
  int64_t lastk = 0;
  uint32_t lastid = 0;
  for (int i0 = 0; i0 < nq; i0 += 8) {
    const uint4 b = row_span(row, i0 >> 3, nq);
    int64_t key[8];
    uint32_t id[8];
    bool isr[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t e = span_entry(b, u);
      const int kind = (e >> 14) & 3, k = (e >> 11) & 7, m = e & 0x7FF;
      const int s = pick<VMAX>(c.st, k);
      const int cx = kind == KF ? pick<VMAX>(c.xF, k) : kind == KB ? pick<VMAX>(c.xB, k) : 0;
      isr[u] = i0 + u < nq && (cx & CX_IN) != 0;
      const int ps = kind == KF ? s - 1 : s + 1;
      id[u] = pitem(0, kind, ps, m);
      key[u] = isr[u] ? tb[node(kind, ps, m)] : 0;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (!isr[u]) continue;
      if (nr == 0 || !key_less(key[u], 0, id[u], lastk, 0, lastid)) {
        rkey[nr] = key[u], rid[nr] = id[u];
        lastk = key[u], lastid = id[u];
        ++nr;
        continue;
      }
      int j = nr++;
      while (j > 0 && key_less(key[u], 0, id[u], rkey[j - 1], 0, rid[j - 1])) {
        rkey[j] = rkey[j - 1];
        rid[j] = rid[j - 1];
        --j;
      }
      rkey[j] = key[u];
      rid[j] = id[u];
    }
  }
  // merge: computations (queue order), sends (queue order), receives (sorted). Each stream
  // keeps its head and its next item in registers; the stream taken moves its next item to the
  // head and loads the one after, so that a load is awaited an iteration after it was issued,
  // and the three streams' steps are selects rather than branches (lanes take different
  // streams).
  RowCursor rc_c, rc_s;
  rc_c.init(row, nq);
  rc_s.init(row, nq);
  // computations: item ci (head) and ci + 1 (next); the next one's finish is kept as loaded
  // and its duration beside it, so that the load is first used when it becomes the head
  auto comp_at = [&](int i, int64_t& fin, int64_t& dur, uint32_t& item) {
    const uint32_t e = rc_c.at(i < nq ? i : 0);
    const int kind = (e >> 14) & 3, k = (e >> 11) & 7, m = e & 0x7FF;
    const int s = pick<VMAX>(c.st, k);
    fin = i < nq ? tb[node(kind, s, m)] : 0;
    dur = dur_of(kind, k);
    item = pitem(PI_COMP, kind, s, m);
  };
  // sends: the first send entry at or after position i (nq: none)
  auto send_from = [&](int i, int64_t& key, uint32_t& id) {
    int j = i;
    int kind = 0, k = 0, m = 0;
    for (; j < nq; ++j) {
      const uint32_t e = rc_s.at(j);
      kind = (e >> 14) & 3, k = (e >> 11) & 7, m = e & 0x7FF;
      const int cx = kind == KF ? pick<VMAX>(c.xF, k) : kind == KB ? pick<VMAX>(c.xB, k) : 0;
      if (cx & CX_OUT) break;
    }
    const int s = pick<VMAX>(c.st, k);
    key = j < nq ? tb[node(kind, s, m)] : 0;
    id = pitem(0, kind, s, m);
    return j;
  };
  int ci = 0, ri = 0, n = 0;
  int64_t ck, cf2, cd2, sk, sk2, rk, rk2;
  uint32_t citem, citem2, sid, sid2, rdd, rdd2;
  {
    int64_t f0, d0;
    comp_at(0, f0, d0, citem);
    ck = f0 - d0;
  }
  comp_at(1, cf2, cd2, citem2);
  int si = send_from(0, sk, sid);
  int si2 = send_from(si + 1 < nq ? si + 1 : nq, sk2, sid2);
  rk = ri < nr ? rkey[0] : 0, rdd = ri < nr ? rid[0] : 0;
  rk2 = 1 < nr ? rkey[1] : 0, rdd2 = 1 < nr ? rid[1] : 0;
  uint4 pk4 = make_uint4(0, 0, 0, 0);
  while (ci < nq || si < nq || ri < nr) {
    // the smallest of the three heads
    int src = ci < nq ? 0 : -1;
    int64_t bt = ck;
    uint32_t bc = 1, bt2 = (uint32_t)ci;
    if (si < nq && (src < 0 || key_less(sk, 0, sid, bt, bc, bt2))) src = 1, bt = sk, bc = 0, bt2 = sid;
    if (ri < nr && (src < 0 || key_less(rk, 0, rdd, bt, bc, bt2))) src = 2;
    // items are gathered four at a time and written as one 16-byte store: a store is counted
    // with the loads, so one per item would make every later load wait for its write
    const uint32_t item = src == 0 ? citem : src == 1 ? ((PI_SEND << 30) | sid) : ((PI_RECV << 30) | rdd);
    const int q = n & 3;
    pk4.x = q == 0 ? item : pk4.x;
    pk4.y = q == 1 ? item : pk4.y;
    pk4.z = q == 2 ? item : pk4.z;
    pk4.w = q == 3 ? item : pk4.w;
    if (q == 3) prog[n >> 2] = pk4;
    ++n;
    // the stream taken: next to head, and the item after next requested
    const bool tc = src == 0, ts = src == 1, tr = src == 2;
    ci += tc ? 1 : 0;
    ck = tc ? cf2 - cd2 : ck, citem = tc ? citem2 : citem;
    si = ts ? si2 : si;
    sk = ts ? sk2 : sk, sid = ts ? sid2 : sid;
    ri += tr ? 1 : 0;
    rk = tr ? rk2 : rk, rdd = tr ? rdd2 : rdd;
    if (tc) comp_at(ci + 1, cf2, cd2, citem2);
    if (ts) si2 = send_from(si + 1 < nq ? si + 1 : nq, sk2, sid2);
    if (tr && ri + 1 < nr) rk2 = rkey[ri + 1], rdd2 = rid[ri + 1];
  }
  // the last, partial group of four
  if (n & 3) prog[n >> 2] = pk4;
  return n;
}

// Phase B of the executor's reordering for lane d (REORDER): the communication items of the
// naive programs (a receive in the gap before its consumer, a send after its producer) with
// their keys (producer end, level, node); step 1, the items below the running maximum key are
// the mismatched receives; steps 2 and 3, each of those in key order takes the gap of least
// cost (|producer end - the gap's post time| - min(transfer, the computations from the gap to
// the consumer)) among the gaps between the in-order items around its key, at most its
// consumer's, whose post time is not before the producer starts (the highest gap always
// qualifies; ties: the highest); then the items, in key order, are merged with the computations
// by gap. Returns the program length; *nrecv and *nmis get the two counts. pst and pdur
// (nq + 1 entries) hold each gap's post time and the prefix sums of the computations'
// durations, so that a window's costs read two arrays instead of walking the queue.
// A send is never mismatched: its key is its own op's end, which is later than the end of every
// earlier op and of every producer an earlier op received from.
template <int VMAX>
__device__ __forceinline__ int build_program3(const Chunks<VMAX>& c, const uint16_t* row, int nq,
                                              const int64_t* tb, const int64_t* ts,
                                              const int32_t* tl, int S, int M,
                                              LaneArr<CItem> items, int icap,
                                              LaneArr<int64_t> pst, LaneArr<int64_t> pdur,
                                              LaneArr<uint4> prog, int* nrecv, int* nmis) {
  auto node = [&](int kind, int s, int m) { return (kind * S + s) * M + m; };
  auto dur_of = [&](int kind, int k) {
    return kind == KF ? pick<VMAX>(c.dF, k) : kind == KB ? pick<VMAX>(c.dB, k) : pick<VMAX>(c.dW, k);
  };
  // the node field is kind << 17 | stage << 11 | m, ordered as the node index is
  auto pack = [](int level, int kind, int s, int m, uint32_t recv, int gap) {
    return (uint64_t)(uint32_t)level << 37 |
           (uint64_t)((uint32_t)kind << 17 | (uint32_t)s << 11 | (uint32_t)m) << 17 |
           (uint64_t)recv << 16 | (uint64_t)(uint32_t)gap;
  };
  auto gap_of = [](const CItem& x) { return (int)(x.pk & 0xFFFFu); };
  // mismatched item j sits at icap - 1 - j
  auto mis = [&](int j) -> CItem& { return items[icap - 1 - j]; };
  // the items in program order, step 1 on the fly: eight queue entries per span, whose loads
  // are all issued before the items are stored
  int nr = 0, nf = 0, nrv = 0;
  CItem top;
  top.key = 0, top.pk = 0;
  auto add = [&](int64_t t, uint64_t pk) {
    CItem x;
    x.key = t, x.pk = pk;
    if (nr == 0 || item_less(top, x)) {
      items[nr++] = x;
      top = x;
    } else {
      mis(nf++) = x;
    }
  };
  pst[0] = 0, pdur[0] = 0;
  int64_t dsum = 0;
  for (int i0 = 0; i0 < nq; i0 += 8) {
    const uint4 b = row_span(row, i0 >> 3, nq);
    int64_t fy[8], fx[8], ds[8];
    int32_t ly[8], lx[8];
    int cxs[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      const uint32_t e = span_entry(b, u);
      const int kind = (e >> 14) & 3, k = (e >> 11) & 7, m = e & 0x7FF;
      const int s = pick<VMAX>(c.st, k);
      const bool in = i0 + u < nq;
      const int cx =
          !in ? 0 : kind == KF ? pick<VMAX>(c.xF, k) : kind == KB ? pick<VMAX>(c.xB, k) : 0;
      const int y = node(kind, s, m), x = node(kind, kind == KF ? s - 1 : s + 1, m);
      cxs[u] = cx;
      fy[u] = in ? tb[y] : 0;
      fx[u] = (cx & CX_IN) ? tb[x] : 0;
      lx[u] = (cx & CX_IN) ? tl[x] : 0;
      ly[u] = (cx & CX_OUT) ? tl[y] : 0;
      dsum += in ? dur_of(kind, k) : 0;
      ds[u] = dsum;
    }
#pragma unroll
    for (int u = 0; u < 8; ++u) {
      if (i0 + u >= nq) break;
      const uint32_t e = span_entry(b, u);
      const int kind = (e >> 14) & 3, k = (e >> 11) & 7, m = e & 0x7FF;
      const int s = pick<VMAX>(c.st, k);
      pst[i0 + u + 1] = fy[u], pdur[i0 + u + 1] = ds[u];
      if (cxs[u] & CX_IN) {
        add(fx[u], pack(lx[u], kind, kind == KF ? s - 1 : s + 1, m, 1u, i0 + u));
        ++nrv;
      }
      if (cxs[u] & CX_OUT) add(fy[u], pack(ly[u], kind, s, m, 0u, i0 + u + 1));
    }
  }
  *nrecv = nrv, *nmis = nf;
  // the mismatched items in key order
  for (int a2 = 1; a2 < nf; ++a2) {
    const CItem v = mis(a2);
    int j = a2;
    CItem pv = mis(j - 1);
    while (item_less(v, pv)) {
      mis(j) = pv;
      if (--j == 0) break;
      pv = mis(j - 1);
    }
    mis(j) = v;
  }
  // steps 2 and 3: the in-order items are sorted by key and by gap, so one walk serves all; a
  // mismatched item lies below the record that was the maximum when it came, so the walk
  // stops inside the records
  int rp = 0, lastg = 0, logap = 0;
  CItem rh = items[0];
  for (int a2 = 0; a2 < nf; ++a2) {
    CItem f = mis(a2);
    while (item_less(rh, f)) {
      logap = gap_of(rh);
      rh = items[++rp];
    }
    const int hi = gap_of(rh);
    const int lo = lastg > logap ? lastg : logap;
    const int iY = gap_of(f);
    const uint32_t code = (uint32_t)(f.pk >> 17) & 0x7FFFFu;
    const int64_t xst = ts[node(code >> 17, (code >> 11) & 63, code & 0x7FF)];
    // the transfer's time: the consumer's input weight
    const uint32_t ey = row[iY];
    const int ky = (ey >> 11) & 7;
    const int64_t cw = ((ey >> 14) & 3) == KF ? pick<VMAX>(c.wF, ky) : pick<VMAX>(c.wB, ky);
    // the window's lowest gap: the first at or above lo posted at or after X's start (post
    // times never decrease), or just hi
    int gx = lo, ge = hi + 1;
    while (gx < ge) {
      const int mid = (gx + ge) >> 1;
      if (pst[mid] < xst) gx = mid + 1;
      else ge = mid;
    }
    const int first = gx < hi ? gx : hi;
    const int64_t pY = pdur[iY], fk = f.key;
    int best = hi;
    int64_t bestc = 0;
    for (int gp = hi; gp >= first; --gp) {
      const int64_t pt = pst[gp], D = pY - pdur[gp];
      const int64_t span = fk > pt ? fk - pt : pt - fk;
      const int64_t cost = span - (D < cw ? D : cw);
      if (gp == hi || cost < bestc) best = gp, bestc = cost;
    }
    f.pk = (f.pk & ~(uint64_t)0xFFFFu) | (uint64_t)best;
    mis(a2) = f;
    lastg = best;
  }
  // the program: items in key order (in-order ones and mismatched ones merged; their gaps never
  // decrease), each after the computations before its gap
  ProgOut po;
  po.init(prog);
  RowCursor cc;
  cc.init(row, nq);
  int ci = 0, ri = 0, fi = 0;
  CItem rh2 = items[0], fh = mis(0);
  while (ri < nr || fi < nf) {
    const bool tr = ri < nr && (fi >= nf || item_less(rh2, fh));
    const CItem h = tr ? rh2 : fh;
    for (const int gp = gap_of(h); ci < gp; ++ci) {
      const uint32_t e = cc.at(ci);
      po.emit(pitem(PI_COMP, (e >> 14) & 3, pick<VMAX>(c.st, (e >> 11) & 7), e & 0x7FF));
    }
    const uint32_t code = (uint32_t)(h.pk >> 17) & 0x7FFFFu;
    po.emit(((h.pk >> 16) & 1u ? PI_RECV : PI_SEND) << 30 |
            pitem(0, code >> 17, (code >> 11) & 63, code & 0x7FF));
    if (tr) {
      if (++ri < nr) rh2 = items[ri];
    } else {
      if (++fi < nf) fh = mis(fi);
    }
  }
  for (; ci < nq; ++ci) {
    const uint32_t e = cc.at(ci);
    po.emit(pitem(PI_COMP, (e >> 14) & 3, pick<VMAX>(c.st, (e >> 11) & 7), e & 0x7FF));
  }
  return po.finish();
}

// RING: 40-bit ring tables of a.ring rows per stage per group. Phase C keeps each device's
// computations in queue order and adds only the sends, each of which reads its producer's slot
// after the producer and before any later computation of the stage, so the ring argument of
// k_tune_ring holds for both rounds; a candidate whose queue window reaches the ring joins the
// wide list (wide_list: taken by a 40-bit full-row pass, a.ring = M) or else the redo list, and
// one whose times pass 40 bits the redo list, which the 64-bit kernel (list, list_n) takes.
// REORDER: the executor's three-step reordering (build_program3) with handshake transfers in
// phase C: a receive completes when the sender has announced itself, at h = max(the sender's
// announce time, the receiver's clock); both clocks go to h, and the data's arrival h + w is kept
// in the finish-time buffer at the producer's node (phase B is done with it), where the consumer,
// a later computation of the same lane, takes it as its input time.
// Three waves per SIMD for the ideal-start variant (its phases wait on global loads: 27.5 ->
// 25.1 ms on 65,536 candidates of the P = 8, M = 64 batch, a few registers spilled); the
// reordering variant keeps its registers (at three waves it spills and slows by a third).
template <int VMAX, bool RING, bool REORDER>
__global__ void __launch_bounds__(WAVE) __attribute__((amdgpu_waves_per_eu(REORDER ? 1 : 3, 8)))
k_ordered(SimArgs a, OrdBufs ob,
                                                  const int32_t* __restrict__ list,
                                                  const int32_t* __restrict__ list_n,
                                                  int wide_list) {
  extern __shared__ __align__(16) uint8_t smem[];
  __shared__ int64_t mbox[WAVE];    // transfer end posted by the receiver, per sender lane
  __shared__ int64_t obt[WAVE];     // outbox: the sender's announce time ...
  __shared__ int32_t obn[WAVE];     // ... and its producer (OB_NONE: nothing announced)
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  const int me = lane_id(), g0 = me - d;
  uint8_t* lds_group = smem + (size_t)(g < a.CPW ? g : 0) * a.group_bytes;
  const auto T = group_table<RING>(lds_group, a.slots);
  uint8_t* rec = lds_group + a.table_bytes;
  const int slot = (int)blockIdx.x * a.CPW + (g < a.CPW ? g : 0);
  const int dl = d < P ? d : 0;
  uint16_t* row = a.qscratch + ((size_t)slot * P + dl) * a.qcap;
  int64_t* tb = ob.tb + (size_t)slot * 3 * a.pr.s_max * M;
  int64_t* ts = REORDER ? ob.ts + (size_t)slot * 3 * a.pr.s_max * M : nullptr;
  int32_t* tl = REORDER ? ob.tl + (size_t)slot * 3 * a.pr.s_max * M : nullptr;
  const LaneArr<uint4> prog = lane_arr(ob.prog, ob.pcap / 4);
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  const int64_t n_groups = (int64_t)gridDim.x * a.CPW;
  const int64_t total = list ? (int64_t)*list_n : a.n;
  const Ring ring = make_ring(M, RING ? a.ring : M);
  for (int64_t base = (int64_t)blockIdx.x * a.CPW; base < total; base += n_groups) {
    const bool has = g < a.CPW && base + g < total;
    const int64_t cand = has ? (list ? (int64_t)list[base + g] : base + g) : 0;
    const uint8_t* grec = a.cands + cand * a.pr.stride;
    if (has) stage_record(rec, grec, a.rec_bytes, d, G);
    __syncthreads();
    Resolved r;
    r.valid = 0, r.v = 1, r.split = 0, r.gen = GEN_AFAB, r.n_pert = 0;
    if (has) r = resolve_record(a.pr, grec);
    const bool valid = has && r.valid;
    const int v = valid ? r.v : 1;
    const int S = P * v;
    Chunks<VMAX> c;
    int64_t busy = 0;
    Lane L;
    L.clock = 0, L.pos = 0, L.nops = 0, L.mem = L.peak = 0;
    L.cm.reset();
    L.fs = -1;
    L.tb = tb, L.tS = S, L.tM = M;
    L.ts = ts, L.tl = tl, L.rnd = 0;
    int wl = 0;
    if (valid && d < P) {
      busy = setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, r.split, ring, nullptr,
                                nullptr, XR);
      L.nops = materialise<VMAX>(a, c, v, r.gen, r.split, row);
      const uint8_t* pp = grec + pert_off(a.pr.s_max);
      for (int i = 0; i < r.n_pert; ++i) {
        const int pd = pp[6 * i] | (pp[6 * i + 1] << 8);
        if (pd != d) continue;
        move_entry(row, pp[6 * i + 2] | (pp[6 * i + 3] << 8), pp[6 * i + 4] | (pp[6 * i + 5] << 8));
      }
      if (RING) wl = queue_window<VMAX>(row, L.nops);
    } else {
      zero_chunks<VMAX>(c);
    }
    const bool on_ring = !RING || group_max((int64_t)wl, G) < ring.R;
    const bool run = valid && on_ring;
    const bool mine = run && d < P;
    if (!mine) L.nops = 0;
    if (run) T.clear(S * ring.R, d, G);
    __syncthreads();
    // A: the asynchronous schedule, finish times recorded
    bool dead = false;
    {
      rounds_mat<VMAX, XT>(row, a.qcap, c, ring, L, T, G, gbit, lsb, dead, nullptr);
    }
    __syncthreads();  // every lane's finish times visible to the group
    // B: programs
    int plen = 0, nrecv = 0, nmis = 0;
    if constexpr (REORDER) {
      if (mine && !dead)
        plen = build_program3<VMAX>(c, row, L.nops, tb, ts, tl, S, M, lane_arr(ob.items, ob.icap),
                                    ob.icap, lane_arr(ob.pst, ob.pcap2),
                                    lane_arr(ob.pdur, ob.pcap2), prog, &nrecv, &nmis);
    } else {
      if (mine && !dead)
        plen = build_program<VMAX>(c, row, L.nops, tb, S, M, lane_arr(ob.rkey, ob.rcap),
                                   lane_arr(ob.rid, ob.rcap), prog);
    }
    if (run) T.clear(S * ring.R, d, G);
    mbox[me] = RDV_EMPTY;
    obn[me] = OB_NONE;
    obt[me] = 0;
    __syncthreads();
    // C: rounds over the programs
    int64_t clock = 0;
    bool cdead = false;
    if (!dead) {
      const uint8_t* devs = rec + 3 + a.pr.s_max;
      int pos = 0;
      bool live = pos < plen, arrived = false;
      // the next item is loaded one advance ahead, so decoding never waits for memory
      uint32_t nitem = plen > 1 ? prog_at(prog, 1) : 0u;
      // the current item, decoded
      uint32_t type = 0, tag = 0;
      int rd = 0, wr = 0, store = 0, src = 0;
      uint32_t mask = 0, want = 0, state = 0;
      int64_t w = 0, dur = 0;
      // REORDER: a computation with a cross-device input takes the arrival its receive left at
      // the producer's node (xat); a receive names that node (xnode). Only a real item (real:
      // the lane has one; otherwise the code 0 stands in, whose op need not be the lane's)
      // loads an arrival.
      bool xarr = false;
      int64_t xat = 0;
      int xnode = 0;
      auto decode = [&](uint32_t it, bool real) {
        type = it >> 30;
        const int kind = (int)((it >> 28) & 3u), s = (int)((it >> 16) & 63u), m = (int)(it & 0x7FFu);
        tag = it & 0x3FFFFFFFu;
        xarr = false;
        if (type == PI_COMP) {
          Desc D;
          describe<VMAX>(D, c, ring, kind, chunk_of<VMAX>(c, s, v), m);
          rd = D.rd, wr = D.wr, store = D.store, mask = (uint32_t)D.mask, want = (uint32_t)D.want;
          state = D.state, w = D.w, dur = D.dur;
          if constexpr (REORDER) {
            xarr = real && (D.cx & CX_IN) != 0;
            if (xarr) xat = tb[(kind * S + (kind == KF ? s - 1 : s + 1)) * M + m];
          }
        } else if (type == PI_SEND) {  // its producer (an own op) must have finished
          rd = s * ring.R + (m & ring.mask);
          const uint32_t par = ((uint32_t)m >> ring.lg) & 1u;
          mask = (kind == KF ? ST_F : ST_B) | ST_PAR;
          want = (kind == KF ? ST_F : ST_B) | (par ? ST_PAR : 0u);
        } else {  // receive: the producer's device and the consumer's link weight
          src = devs[s];
          const int cs = kind == KF ? s + 1 : s - 1;
          const int ck = chunk_of<VMAX>(c, cs, v);
          w = kind == KF ? pick<VMAX>(c.wF, ck) : pick<VMAX>(c.wB, ck);
          xnode = (kind * S + s) * M + m;
        }
      };
      decode(live ? prog_at(prog, 0) : 0u, live);
      for (;;) {
        uint32_t plo, phi;
        T.issue(live && type != PI_RECV ? rd : 0, plo, phi);
        const int64_t box = mbox[me];
        const int32_t on = obn[g0 + (type == PI_RECV ? src : 0)];
        const int64_t ot = obt[g0 + (type == PI_RECV ? src : 0)];
        const uint64_t p = (uint64_t)plo | ((uint64_t)phi << 32);
        const bool rdy = (plo & mask) == want;
        const bool okC = live && type == PI_COMP && rdy;
        const int64_t tin = xarr ? xat : (int64_t)(p >> 3) + w;
        const int64_t st = tin > clock ? tin : clock;
        const int64_t fin = st + dur;
        const bool okSA = live && type == PI_SEND && !arrived && rdy;
        const bool okSD = live && type == PI_SEND && arrived && box != RDV_EMPTY;
        const bool okR = live && type == PI_RECV && on == (int32_t)tag;
        // the handshake, and where both clocks go: its end (blocking) or its start (REORDER)
        const int64_t hs = ot > clock ? ot : clock;
        const int64_t xend = REORDER ? hs : hs + w;
        if (okC && store) T.store(wr, ((uint64_t)fin << 3) | state);
        if (okSA) obn[me] = (int32_t)tag, obt[me] = clock;
        if (okSD) mbox[me] = RDV_EMPTY, obn[me] = OB_NONE;
        if (okR) mbox[g0 + src] = xend;
        if (REORDER && okR) tb[xnode] = hs + w;
        clock = okC ? fin : okSD ? box : okR ? xend : clock;
        arrived = okSA ? true : okSD ? false : arrived;
        const bool done = okC || okSD || okR;
        if (done) {
          ++pos;
          live = pos < plen;
          const uint32_t it = live ? nitem : 0u;
          __asm__ volatile("" : "+v"(nitem));
          nitem = pos + 1 < plen ? prog_at(prog, pos + 1) : 0u;
          decode(it, live);
        }
        __asm__ volatile("" ::: "memory");
        if (__ballot(okC || okSA || okSD || okR) == 0) {
          const uint64_t actm = __ballot(live);
          if (actm != 0 && (fold_groups(actm, G, lsb) & gbit)) cdead = true;
          break;
        }
      }
    }
    const int64_t ms = group_max(clock, G);
    int64_t srecv = 0, smis = 0;
    if constexpr (REORDER) srecv = group_sum(nrecv, G), smis = group_sum(nmis, G);
    // overflow test over both rounds' clocks (phase A's alone when it deadlocked)
    const int64_t top = RING ? group_max(clock > L.clock ? clock : L.clock, G) : 0;
    if (has && valid && (!on_ring || top >= Table40::LIMIT)) {
      // too wide for the ring: the full-row 40-bit pass (when one follows); overflow: 64 bits
      if (d == 0) {
        if (!on_ring && wide_list)
          a.wide[atomicAdd(&a.ctl[CTL_WIDE], 1)] = (int32_t)cand;
        else
          a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
      }
    } else if (mine) {
      const int64_t sv = dead || cdead ? (int64_t)OCTO_MS_DEADLOCK : 0;
      if (d == 0) a.out_ms[cand] = sv ? sv : ms;
      a.out_bub[cand * P + d] = sv ? sv : ms - busy;
      if (REORDER && ob.stats && d == 0)
        ob.stats[2 * cand] = sv ? sv : srecv, ob.stats[2 * cand + 1] = sv ? sv : smis;
    } else if (has && !valid && d < P) {
      if (d == 0) a.out_ms[cand] = OCTO_MS_INVALID;
      a.out_bub[cand * P + d] = OCTO_MS_INVALID;
    }
    __syncthreads();  // before the next candidate reuses the staged record and the tables
  }
}

// ---------------------------------------------------------------------------------------------
// Selective W advancing (§6 "Scheduling Tuning", third policy) under per-device capacities
// (§6 Eq. 2). While a device's peak exceeds its capacity, take the lowest such device d and
// the queue position p at which its running activation total first reaches the peak (an F).
// Eligible: a W of d after p whose B precedes p and whose stage holds activations; advancing it
// moves it to index p, so its release comes before that allocation. Eligible W are tried in
// queue order: the first whose advance does not lengthen the makespan is kept (busy time is
// fixed, so no bubble grows), else the first one is. Repeat until every device fits, nothing is
// eligible, or max_adv advances were made. A W has no consumers, so no advance can deadlock.
// ---------------------------------------------------------------------------------------------
constexpr int AW_SIM = 0, AW_TRIAL = 1, AW_WALK = 2, AW_NEXT = 3, AW_DONE = 4;

// Lane-local result of one group's advancing.
struct AdvOut {
  bool dead;    // the queues deadlock (nothing advanced)
  bool fits;    // every device of the group is within capacity
  int adv;      // advances made
  int64_t ms;   // makespan of the final queues
  int64_t hi;   // largest activation total this lane's device holds
  int64_t top;  // largest makespan of any simulation run (40-bit tables: overflow test)
};

// Running activation total along one device queue: its maximum and the first position that
// reaches it (-1 when nothing is allocated).
template <int VMAX>
__device__ __forceinline__ void act_walk(const uint16_t* row, int n, const Chunks<VMAX>& c,
                                         int64_t& hi, int& at) {
  int64_t cur = 0;
  hi = 0, at = -1;
  for (int i0 = 0; i0 < n; i0 += 32) {
    uint4 b[4];
#pragma unroll
    for (int q = 0; q < 4; ++q) b[q] = row_span(row, (i0 >> 3) + q, n);
#pragma unroll
    for (int u = 0; u < 32; ++u) {
      const uint32_t e = span_entry(b[u >> 3], u & 7);
      const bool in = i0 + u < n;
      const int kind = (int)(e >> 14) & 3;
      const int64_t a = pick<VMAX>(c.mA, (int)(e >> 11) & 7);
      const bool isF = kind == KF;
      const bool rel = kind == KW || !c.split;
      cur += !in ? 0 : isF ? a : rel ? -a : 0;
      const bool up = in && isF && cur > hi;
      hi = up ? cur : hi;
      at = up ? i0 + u : at;
    }
  }
}

// First eligible W after position `from` (>= p): its B is not between p and it (a live queue
// has B before W, so B precedes p), and its stage holds activations. -1 if none.
// One pass from p + 1, spans two at a time, keeping the B's passed as a bit set over
// (chunk, micro-batch) in registers when VMAX M <= 512; otherwise each W rescans (p, j).
template <int VMAX>
__device__ __forceinline__ int next_eligible(const uint16_t* row, int n, int p, int from,
                                             const Chunks<VMAX>& c, int M) {
  if (VMAX * M <= 512) {
    uint64_t bs[8];
#pragma unroll
    for (int w = 0; w < 8; ++w) bs[w] = 0;
    for (int j0 = (p + 1) & ~7; j0 < n; j0 += 16) {
      uint4 b[2];
#pragma unroll
      for (int q = 0; q < 2; ++q) b[q] = row_span(row, (j0 >> 3) + q, n);
      int found = -1;
#pragma unroll
      for (int u = 0; u < 16; ++u) {
        const uint32_t e = span_entry(b[u >> 3], u & 7);
        const int j = j0 + u;
        const bool in = j > p && j < n && found < 0;
        const int kind = (int)(e >> 14) & 3, k = (int)(e >> 11) & 7;
        const int bi = k * M + (int)(e & 0x7FF);
        const int wd = (bi >> 6) & 7;
        const uint64_t bit = 1ull << (bi & 63);
        bool seen = false;
#pragma unroll
        for (int w = 0; w < 8; ++w) seen = seen || (wd == w && (bs[w] & bit) != 0);
        const bool elig =
            in && kind == KW && j > from && !seen && pick<VMAX>(c.mA, k) > 0;
        found = elig ? j : found;
#pragma unroll
        for (int w = 0; w < 8; ++w) bs[w] |= (in && kind == KB && wd == w) ? bit : 0;
      }
      if (found >= 0) return found;
    }
    return -1;
  }
  for (int j = from + 1; j < n; ++j) {
    const uint32_t e = row[j];
    if (((e >> 14) & 3) != (uint32_t)KW || pick<VMAX>(c.mA, (int)(e >> 11) & 7) <= 0) continue;
    const uint16_t b = (uint16_t)((KB << 14) | (e & 0x3FFF));
    bool later = false;
    for (int i = p + 1; i < j && !later; ++i) later = row[i] == b;
    if (!later) return j;
  }
  return -1;
}

// Runs the policy for every group of the wave (all lanes call it; groups with run == false
// take no part). row: this lane's queue (n entries, changed in place); cap: this device's
// capacity; stat: its static bytes. pert (nullable): where advance k of the group is written as
// (device, from, to), uint16 each, by the lane of that device.
template <int VMAX, class Tab>
__device__ AdvOut advance_w(const Tab& T, uint16_t* row, int n, int qcap, const Chunks<VMAX>& c,
                            const Ring& ring, int S, int M, int P, bool run, int64_t cap,
                            int64_t stat, int max_adv, int G, uint64_t gbit, uint64_t lsb,
                            uint16_t* pert) {
  const int d = lane_id() % G;
  const int gl = lane_id() - d;
  const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
  AdvOut o;
  o.dead = false, o.fits = false, o.adv = 0, o.ms = 0, o.hi = 0, o.top = 0;
  int phase = run ? AW_SIM : AW_DONE;
  int dstar = 0, p = -1, cursor = -1, first = -1, j = -1, at = -1;
  int64_t ms_first = 0;
  for (;;) {
    const bool need = phase == AW_SIM || phase == AW_TRIAL;
    int64_t ms = 0;
    bool dead = false;
    if (__ballot(need) != 0) {
      Lane L;
      L.clock = 0, L.pos = 0, L.nops = need && d < P ? n : 0, L.mem = L.peak = 0;
      if (need) T.clear(S * ring.R, d, G);
      __asm__ volatile("" ::: "memory");
      rounds_mat<VMAX, XP>(row, qcap, c, ring, L, T, G, gbit, lsb, dead, nullptr);
      ms = group_max(L.clock, G);
      o.top = ms > o.top ? ms : o.top;
    }
    if (phase == AW_SIM) {
      o.dead = dead;
      o.ms = ms;
      phase = dead ? AW_DONE : AW_WALK;
    } else if (phase == AW_TRIAL) {
      if (j == first) ms_first = ms;
      if (ms <= o.ms) {
        o.ms = ms;
        if (pert && d == dstar) {
          pert[3 * o.adv] = (uint16_t)dstar, pert[3 * o.adv + 1] = (uint16_t)j;
          pert[3 * o.adv + 2] = (uint16_t)p;
        }
        ++o.adv;
        phase = AW_WALK;
      } else {
        if (d == dstar) move_entry(row, p, j);
        cursor = j;
        phase = AW_NEXT;
      }
    }
    // walks and searches need no simulation: settle them before the next round
    while (phase == AW_WALK || phase == AW_NEXT) {
      if (phase == AW_WALK) {
        if (d < P) act_walk<VMAX>(row, n, c, o.hi, at);
        const bool over = d < P && stat + o.hi > cap;
        const uint64_t om = (__ballot(over) >> gl) & gmask;
        if (om == 0) {
          o.fits = true;
          phase = AW_DONE;
        } else if (o.adv >= max_adv) {
          phase = AW_DONE;
        } else {
          dstar = __ffsll((unsigned long long)om) - 1;
          p = __shfl(at, gl + dstar);
          cursor = p, first = -1;
          phase = p < 0 ? AW_DONE : AW_NEXT;
        }
      } else {
        int jj = d == dstar ? next_eligible<VMAX>(row, n, p, cursor, c, M) : -1;
        jj = __shfl(jj, gl + dstar);
        if (jj >= 0) {
          first = first < 0 ? jj : first;
          j = jj;
          if (d == dstar) move_entry(row, jj, p);
          phase = AW_TRIAL;
        } else if (first >= 0) {
          // every eligible W lengthens the makespan: take the earliest
          j = first;
          if (d == dstar) {
            move_entry(row, first, p);
            if (pert) {
              pert[3 * o.adv] = (uint16_t)dstar, pert[3 * o.adv + 1] = (uint16_t)first;
              pert[3 * o.adv + 2] = (uint16_t)p;
            }
          }
          o.ms = ms_first;
          ++o.adv;
          phase = AW_WALK;
        } else {
          phase = AW_DONE;
        }
      }
    }
    if (__ballot(phase != AW_DONE) == 0) break;
  }
  return o;
}

// Selective W advancing on candidate records: queues materialised (policy, then the record's
// moves), at most max_pert - n_pert advances appended to the output record as moves. list
// (nullable): the candidates list[0 .. *list_n - 1] only; ctl[work]: the shared cursor.
// Groups are persistent: the policy's steps run as in advance_w (simulations wave-wide, walks and
// searches per group), and a group whose candidate is done writes it out and takes the next one
// while the others go on, so that a wave is not held by its longest search (advance counts
// range from none to hundreds).
// RING: a 40-bit ring table of a.ring rows per stage per group (several times more candidates
// fit a CU than with 64-bit full rows). Advancing a W never widens the queue window: the W moves
// ahead only of entries that follow its own B, so a same-stage entry it passes has a micro-batch
// at most the window below its own. A candidate whose starting window is below the ring's rows
// therefore stays exact on the ring for every simulation of the search; the others, and those
// whose times pass the 40-bit slots, join the redo list, which the 64-bit kernel then processes.
constexpr int AW_LOAD = 5, AW_EXIT = 6;
template <int VMAX, bool RING>
__global__ void __launch_bounds__(WAVE) k_advance(SimArgs a, const int64_t* __restrict__ cap,
                                                  uint8_t* __restrict__ out_cands,
                                                  const int32_t* __restrict__ list,
                                                  const int32_t* __restrict__ list_n, int work) {
  extern __shared__ __align__(16) uint8_t smem[];
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  const int gl = lane_id() - d;
  const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
  uint8_t* lds_group = smem + (size_t)(g < a.CPW ? g : 0) * a.group_bytes;
  const auto T = group_table<RING>(lds_group, a.slots);
  uint8_t* rec = lds_group + a.table_bytes;
  const int slot = (int)blockIdx.x * a.CPW + (g < a.CPW ? g : 0);
  uint16_t* row = a.qscratch + ((size_t)slot * P + (d < P ? d : 0)) * a.qcap;
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  const int po = pert_off(a.pr.s_max);
  const int64_t total = list ? (int64_t)*list_n : a.n;
  const Ring ring = make_ring(M, RING ? a.ring : M);
  const int64_t capd = d < P ? cap[d] : 0;

  // the group's candidate and the state of its search
  int phase = g < a.CPW ? AW_LOAD : AW_EXIT;
  int64_t cand = 0;
  Resolved r;
  r.valid = 0, r.v = 1, r.split = 0, r.gen = GEN_AFAB, r.n_pert = 0;
  Chunks<VMAX> c;
  zero_chunks<VMAX>(c);
  int64_t busy = 0, stat = 0, ms_first = 0;
  int S = P, n = 0, n0 = 0, max_adv = 0;
  int dstar = 0, p = -1, cursor = -1, first = -1, j = -1, at = -1;
  // whether this lane's queue changed since its last activation walk: only the device whose W
  // moved needs a new walk, the others keep theirs
  bool stale = true;
  AdvOut o;
  o.dead = false, o.fits = false, o.adv = 0, o.ms = 0, o.hi = 0, o.top = 0;
  for (;;) {
    // groups without a candidate take the next one (invalid records and, on rings, candidates
    // sent to the redo list are settled here)
    while (phase == AW_LOAD) {
      int e = 0;
      if (d == 0) e = atomicAdd(&a.ctl[work], 1);
      e = __shfl(e, gl);
      if (e >= total) {
        phase = AW_EXIT;
        break;
      }
      cand = list ? (int64_t)list[e] : (int64_t)e;
      const uint8_t* grec = a.cands + cand * a.pr.stride;
      stage_record(rec, grec, a.rec_bytes, d, G);
      __asm__ volatile("" ::: "memory");
      r = resolve_record(a.pr, grec);
      const int v = r.valid ? r.v : 1;
      S = P * v;
      n = 0;
      int wl = 0;
      if (r.valid && d < P) {
        busy = setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, r.split, ring, a.pre_mem,
                                  &stat);
        n = materialise<VMAX>(a, c, v, r.gen, r.split, row);
        const uint8_t* pp = grec + po;
        for (int i = 0; i < r.n_pert; ++i) {
          const int pd = pp[6 * i] | (pp[6 * i + 1] << 8);
          if (pd != d) continue;
          move_entry(row, pp[6 * i + 2] | (pp[6 * i + 3] << 8),
                     pp[6 * i + 4] | (pp[6 * i + 5] << 8));
        }
        if (RING) wl = queue_window<VMAX>(row, n);
      } else {
        zero_chunks<VMAX>(c);
        busy = stat = 0;
      }
      if (RING && r.valid && group_max((int64_t)wl, G) >= ring.R) {
        if (d == 0) a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
        continue;
      }
      __asm__ volatile("" ::: "memory");
      n0 = r.valid ? r.n_pert : 0;
      max_adv = a.pr.max_pert - n0;
      o.dead = false, o.fits = false, o.adv = 0, o.ms = 0, o.hi = 0, o.top = 0;
      dstar = 0, p = -1, cursor = -1, first = -1, j = -1, at = -1, ms_first = 0;
      stale = true;
      phase = r.valid ? AW_SIM : AW_DONE;
    }
    if (__ballot(phase != AW_EXIT) == 0) break;
    uint16_t* pert =
        reinterpret_cast<uint16_t*>(out_cands + cand * a.pr.stride + po) + 3 * n0;

    // one simulation for every group that needs one
    const bool need = phase == AW_SIM || phase == AW_TRIAL;
    int64_t ms = 0;
    bool dead = false;
    if (__ballot(need) != 0) {
      Lane L;
      L.clock = 0, L.pos = 0, L.nops = need && d < P ? n : 0, L.mem = L.peak = 0;
      if (need) T.clear(S * ring.R, d, G);
      __asm__ volatile("" ::: "memory");
      rounds_mat<VMAX, XP>(row, a.qcap, c, ring, L, T, G, gbit, lsb, dead, nullptr);
      ms = group_max(L.clock, G);
      o.top = need && ms > o.top ? ms : o.top;
    }
    if (phase == AW_SIM) {
      o.dead = dead;
      o.ms = ms;
      phase = dead ? AW_DONE : AW_WALK;
    } else if (phase == AW_TRIAL) {
      if (j == first) ms_first = ms;
      if (ms <= o.ms) {
        o.ms = ms;
        stale = stale || d == dstar;
        if (d == dstar) {
          pert[3 * o.adv] = (uint16_t)dstar, pert[3 * o.adv + 1] = (uint16_t)j;
          pert[3 * o.adv + 2] = (uint16_t)p;
        }
        ++o.adv;
        phase = AW_WALK;
      } else {
        if (d == dstar) move_entry(row, p, j);
        cursor = j;
        phase = AW_NEXT;
      }
    }
    // walks and searches need no simulation: settle them before the next round
    while (phase == AW_WALK || phase == AW_NEXT) {
      if (phase == AW_WALK) {
        if (d < P && stale) act_walk<VMAX>(row, n, c, o.hi, at);
        stale = false;
        const bool over = d < P && stat + o.hi > capd;
        const uint64_t om = (__ballot(over) >> gl) & gmask;
        if (om == 0) {
          o.fits = true;
          phase = AW_DONE;
        } else if (o.adv >= max_adv) {
          phase = AW_DONE;
        } else {
          dstar = __ffsll((unsigned long long)om) - 1;
          p = __shfl(at, gl + dstar);
          cursor = p, first = -1;
          phase = p < 0 ? AW_DONE : AW_NEXT;
        }
      } else {
        int jj = d == dstar ? next_eligible<VMAX>(row, n, p, cursor, c, M) : -1;
        jj = __shfl(jj, gl + dstar);
        if (jj >= 0) {
          first = first < 0 ? jj : first;
          j = jj;
          if (d == dstar) move_entry(row, jj, p);
          phase = AW_TRIAL;
        } else if (first >= 0) {
          // every eligible W lengthens the makespan: take the earliest
          j = first;
          if (d == dstar) {
            move_entry(row, first, p);
            pert[3 * o.adv] = (uint16_t)dstar, pert[3 * o.adv + 1] = (uint16_t)first;
            pert[3 * o.adv + 2] = (uint16_t)p;
          }
          o.ms = ms_first;
          stale = stale || d == dstar;
          ++o.adv;
          phase = AW_WALK;
        } else {
          phase = AW_DONE;
        }
      }
    }
    if (phase != AW_DONE) continue;
    // the group's candidate is settled: write it out (or hand it to the 64-bit pass)
    phase = AW_LOAD;
    if (RING && r.valid && o.top >= Table40::LIMIT) {
      if (d == 0) a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)cand;
      continue;
    }
    const uint8_t* grec = a.cands + cand * a.pr.stride;
    uint8_t* orec = out_cands + cand * a.pr.stride;
    // the output record: the input's bytes (the new moves aside), then the move count
    const int halves = a.pr.stride >> 1;
    const int a0 = (po >> 1) + 3 * n0, a1 = a0 + 3 * o.adv;
    const uint16_t* in16 = reinterpret_cast<const uint16_t*>(grec);
    uint16_t* out16 = reinterpret_cast<uint16_t*>(orec);
    for (int h = d; h < halves; h += G)
      if (h != 1 && (h < a0 || h >= a1)) out16[h] = in16[h];
    if (d == 0) out16[1] = (uint16_t)((rec[2] + o.adv) | (rec[3] << 8));
    if (d < P) {
      const int64_t sv =
          r.valid ? (o.dead ? (int64_t)OCTO_MS_DEADLOCK : 0) : (int64_t)OCTO_MS_INVALID;
      if (d == 0) a.out_ms[cand] = sv ? sv : o.ms;
      a.out_bub[cand * P + d] = sv ? sv : o.ms - busy;
      a.out_peak[cand * P + d] = sv ? sv : stat + o.hi;
    }
  }
}

// ---------------------------------------------------------------------------------------------
// Local-search step: one chain per group. k_tune uses 64-bit full-row finish tables; k_tune_ring
// 40-bit ring tables for chains whose queue order allows it, the rest going to k_tune.
// ---------------------------------------------------------------------------------------------
struct TuneArgs {
  SimArgs s;
  uint8_t* chains;
  int chain_stride;
  uint16_t* queues;
  int64_t n_chains;
  uint64_t seed;
  int step;
  const int64_t* cap;  // memory-constrained search: capacity per device [P]
  int max_adv;         // W advances per evaluation
  const int32_t* list;    // nullable: step only the chains list[0 .. *list_n - 1]
  const int32_t* list_n;
};

// int64 word of the chain state (after makespan, accepted count, bubble[P], peak[P]) holding an
// upper bound of the window of the chain's queues (queue_window).
__host__ __device__ __forceinline__ int window_word(int P) { return 2 + 2 * P; }

// One move of a chain (step >= 1). (u0, u1, u2, u3) = Philox4x64-10(key = (seed, 0),
// counter = (chain, step, 0, 0)); u0 mod 3 picks the family (§6's partitioning, placement and
// scheduling tuning):
//   0  stage boundary mi = 1 + u1 mod (S-1) moves by one layer, up if u2 is odd, to nb;
//   1  devices d1 = u1 mod P and d2 = (d1 + 1 + u2 mod (P-1)) mod P exchange their stages, each
//      keeping its queue;
//   2  entries mi = u2 mod (qlen-1) and mi + 1 of device sd = u1 mod P swap.
// The move is applied to the staged record (lane 0) and to device sd's queue row (lane sd).
// Lane sd also returns in `pair` the window term the swap adds (the later entry now first) when
// both entries belong to one chunk: an adjacent swap reorders only that pair.
struct Move {
  int kind, mi, sd, nb, d1, d2, pair;
  bool valid;
};

__device__ __forceinline__ Move propose(uint64_t seed, int64_t chain, int step, uint8_t* rec,
                                        const Problem& pr, int S, int qlen, uint16_t* qrow,
                                        int d) {
  Move mv;
  mv.kind = -1, mv.mi = 0, mv.sd = 0, mv.nb = 0, mv.d1 = 0, mv.d2 = 0, mv.pair = 0;
  mv.valid = true;
  const int P = pr.P;
  const U4 u = philox4x64_10((uint64_t)chain, (uint64_t)step, 0, 0, seed, 0);
  mv.kind = (int)(u.x[0] % 3);
  if (mv.kind == 0) {
    if (S < 2) {
      mv.valid = false;
    } else {
      mv.mi = 1 + (int)(u.x[1] % (uint64_t)(S - 1));
      const int lo = mv.mi > 1 ? rec[4 + mv.mi - 2] : 0;
      const int hi = mv.mi < S - 1 ? rec[4 + mv.mi] : pr.L;
      mv.nb = rec[4 + mv.mi - 1] + ((u.x[2] & 1) ? 1 : -1);
      mv.valid = mv.nb > lo && mv.nb < hi;
      __asm__ volatile("" ::: "memory");
      if (mv.valid && d == 0) rec[4 + mv.mi - 1] = (uint8_t)mv.nb;
    }
  } else if (mv.kind == 1) {
    if (P < 2) {
      mv.valid = false;
    } else {
      mv.d1 = (int)(u.x[1] % (uint64_t)P);
      mv.d2 = (int)((mv.d1 + 1 + (int)(u.x[2] % (uint64_t)(P - 1))) % P);
      uint8_t* dv = rec + 3 + pr.s_max;
      __asm__ volatile("" ::: "memory");
      if (d == 0)
        for (int s = 0; s < S; ++s)
          dv[s] = dv[s] == mv.d1 ? (uint8_t)mv.d2 : dv[s] == mv.d2 ? (uint8_t)mv.d1 : dv[s];
    }
  } else {
    mv.sd = (int)(u.x[1] % (uint64_t)P);
    if (qlen < 2) {
      mv.valid = false;
    } else {
      mv.mi = (int)(u.x[2] % (uint64_t)(qlen - 1));
      if (d == mv.sd) {
        const uint16_t x = qrow[mv.mi], y = qrow[mv.mi + 1];
        qrow[mv.mi] = y;
        qrow[mv.mi + 1] = x;
        if (((x >> 11) & 7) == ((y >> 11) & 7)) mv.pair = (int)(y & 0x7FF) - (int)(x & 0x7FF);
      }
    }
  }
  return mv;
}

// Undo a kind-2 move on device sd's queue row (lane sd).
__device__ __forceinline__ void unswap(const Move& mv, uint16_t* row, int d) {
  if (mv.kind == 2 && mv.valid && d == mv.sd) {
    const uint16_t x = row[mv.mi];
    row[mv.mi] = row[mv.mi + 1];
    row[mv.mi + 1] = x;
  }
}

// One step of every chain (of the list, when given). MEM: the memory-constrained search —
// proposals are built in a working copy of the chain's queues (group slot rows of qscratch),
// selective W advancing runs on it, and a state is feasible only if every device fits; the copy
// replaces the chain's queues when the proposal is kept.
template <int VMAX, bool MEM>
__global__ void __launch_bounds__(WAVE) k_tune(TuneArgs t) {
  extern __shared__ __align__(16) uint8_t smem[];
  const SimArgs& a = t.s;
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  uint8_t* lds_group = smem + (size_t)(g < a.CPW ? g : 0) * a.group_bytes;
  const Table64 T{reinterpret_cast<int64_t*>(lds_group)};
  uint8_t* rec = lds_group + a.table_bytes;
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  const int slot = (int)blockIdx.x * a.CPW + (g < a.CPW ? g : 0);
  uint16_t* wrow = MEM ? a.qscratch + ((size_t)slot * P + (d < P ? d : 0)) * a.qcap : nullptr;
  const int gl = lane_id() - d;
  const uint64_t gmask = G == 64 ? ~0ull : ((1ull << G) - 1);
  const int64_t n_groups = (int64_t)gridDim.x * a.CPW;
  const int64_t total = t.list ? (int64_t)*t.list_n : t.n_chains;
  for (int64_t base = (int64_t)blockIdx.x * a.CPW; base < total; base += n_groups) {
    const bool has = g < a.CPW && base + g < total;
    const int64_t chain = has ? (t.list ? (int64_t)t.list[base + g] : base + g) : 0;
    uint8_t* crec = t.chains + chain * t.chain_stride;
    int64_t* cstate = reinterpret_cast<int64_t*>(crec + a.pr.stride);
    uint16_t* row = t.queues + ((size_t)chain * P + (d < P ? d : 0)) * a.qcap;
    uint16_t* qrow = MEM ? wrow : row;  // the queues the proposal is evaluated on
    if (has) stage_record(rec, crec, a.rec_bytes, d, G);
    __asm__ volatile("" ::: "memory");

    // state of the chain before this step
    bool skip = !has;
    int v = 1, gen = GEN_AFAB, split = 0;
    int64_t cur = 0;
    if (has) {
      if (t.step == 0) {
        Resolved r = resolve_record(a.pr, crec);
        if (!r.valid || r.n_pert != 0) {
          if (d == 0) cstate[0] = OCTO_MS_INVALID, cstate[1] = 0;
          if (d < P) cstate[2 + d] = OCTO_MS_INVALID;
          if (MEM && d < P) cstate[2 + P + d] = OCTO_MS_INVALID;
          skip = true;
        }
        v = r.v, gen = r.gen, split = r.split;
      } else {
        cur = cstate[0];
        // the stored state is re-checked so that a damaged record cannot index out of range
        Resolved r = resolve_record(a.pr, rec);
        if (cur == OCTO_MS_INVALID || !r.valid || r.n_pert != 0) skip = true;
        v = r.valid ? r.v : 1;
        split = r.split;
      }
    }
    const int S = P * v;
    const int qlen = (split ? 3 : 2) * v * M;
    const Ring ring = make_ring(M, M);
    if (MEM && !skip && t.step > 0 && d < P)
      for (int i = 0; i < qlen; ++i) wrow[i] = row[i];

    // propose (step >= 1); the move is applied to the staged record / the queue row qrow
    Move mv;
    mv.kind = -1, mv.valid = true, mv.pair = 0, mv.sd = 0;
    if (!skip && t.step > 0) mv = propose(t.seed, chain, t.step, rec, a.pr, S, qlen, qrow, d);
    const int pair = __shfl(mv.pair, gl + (mv.sd < G ? mv.sd : 0));
    __asm__ volatile("" ::: "memory");
    const bool valid = mv.valid;
    const bool run = !skip && valid;

    Chunks<VMAX> c;
    int64_t busy = 0, stat = 0;
    int win = 0;
    if (run && d < P) {
      busy = setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, split, ring,
                                MEM ? a.pre_mem : nullptr, &stat);
      if (t.step == 0) {
        materialise<VMAX>(a, c, v, gen, split, qrow);
        if (!MEM) win = queue_window<VMAX>(qrow, qlen);
      }
    } else {
      zero_chunks<VMAX>(c);
    }
    if (!MEM && t.step == 0) win = (int)group_max((int64_t)win, G);
    __asm__ volatile("" ::: "memory");
    bool dead = false, fits = true;
    int64_t ms = 0, held = 0;
    if constexpr (MEM) {
      const AdvOut o = advance_w<VMAX>(T, qrow, run && d < P ? qlen : 0, a.qcap, c, ring, S, M, P,
                                       run, d < P ? t.cap[d] : 0, stat, t.max_adv, G, gbit, lsb,
                                       nullptr);
      dead = o.dead, fits = o.fits, ms = o.ms, held = o.hi;
    } else {
      Lane L;
      L.clock = 0, L.pos = 0, L.nops = run && d < P ? qlen : 0, L.mem = L.peak = 0;
      if (run) T.clear(S * M, d, G);
      __asm__ volatile("" ::: "memory");
      rounds_mat<VMAX, XP>(qrow, a.qcap, c, ring, L, T, G, gbit, lsb, dead, nullptr);
      ms = group_max(L.clock, G);
    }

    if (!has || skip) continue;
    bool keep = t.step == 0;
    if (t.step > 0) {
      // the current state counts as +infinity when deadlocked or (MEM) over capacity
      bool cur_ok = cur >= 0;
      if constexpr (MEM) {
        const bool over = d < P && cstate[2 + P + d] > t.cap[d];
        cur_ok = cur_ok && ((__ballot(over) >> gl) & gmask) == 0;
      }
      keep = valid && !dead && fits && (!cur_ok || ms <= cur);
    }
    if (keep) {
      if (d == 0) {
        cstate[0] = dead ? OCTO_MS_DEADLOCK : ms;
        cstate[1] = t.step == 0 ? 0 : cstate[1] + 1;
        if (t.step > 0)
          for (int i = 0; i < a.rec_bytes; ++i) crec[i] = rec[i];
        if (!MEM) {
          const int64_t w0 = t.step == 0 ? 0 : cstate[window_word(P)];
          cstate[window_word(P)] = t.step == 0 ? win : (pair > w0 ? pair : w0);
        }
      }
      if (d < P) cstate[2 + d] = dead ? OCTO_MS_DEADLOCK : ms - busy;
      if constexpr (MEM) {
        if (d < P) {
          cstate[2 + P + d] = dead ? OCTO_MS_DEADLOCK : stat + held;
          for (int i = 0; i < qlen; ++i) row[i] = wrow[i];
        }
      }
    } else if (!MEM) {
      unswap(mv, row, d);
    }
  }
}

// Chains by queue length, for the ring pass: class (v - 1) * 2 + split from each chain's record
// header (records whose header is out of range take class 2 * v_max, last); counts into the bin
// counters, offsets by k_plan, then the chain indices scattered by class.
__device__ __forceinline__ int chain_class(const TuneArgs& t, int64_t i) {
  const uint8_t* r = t.chains + i * t.chain_stride;
  const int pol = r[0], v = r[1];
  return (v >= 1 && v <= t.s.pr.v_max && pol <= POL_ZB) ? (v - 1) * 2 + (pol == POL_ZB)
                                                          : 2 * t.s.pr.v_max;
}

// Both count per block in LDS first (one LDS atomic per class per wave, one global atomic per
// class per block): a global atomic per chain on a handful of counters serialises.
constexpr int NCLASS = 2 * 8 + 1;
__global__ void k_chain_count(TuneArgs t) {
  __shared__ int hist[NCLASS];
  for (int b = threadIdx.x; b < NCLASS; b += blockDim.x) hist[b] = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool in = i < t.n_chains;
  wave_hist_add(hist, in ? chain_class(t, i) : 0, in);
  __syncthreads();
  for (int b = threadIdx.x; b < NCLASS; b += blockDim.x)
    if (hist[b]) atomicAdd(&t.s.ctl[CTL_COUNTS + b], hist[b]);
}

__global__ void k_chain_scatter(TuneArgs t, int32_t* __restrict__ list) {
  __shared__ int hist[NCLASS];
  __shared__ int res[NCLASS];
  for (int b = threadIdx.x; b < NCLASS; b += blockDim.x) hist[b] = 0;
  __syncthreads();
  const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
  const bool in = i < t.n_chains;
  const int cls = in ? chain_class(t, i) : 0;
  const int local = wave_hist_add(hist, cls, in);
  __syncthreads();
  for (int b = threadIdx.x; b < NCLASS; b += blockDim.x)
    res[b] = hist[b] ? atomicAdd(&t.s.ctl[CTL_POS + b], hist[b]) : 0;
  __syncthreads();
  if (in) list[res[cls] + local] = (int32_t)i;
}

// One step of every chain on 40-bit ring tables: R rows per stage (R < M), the wave's groups
// sharing the slot arrays as in the generated kernels, so several chains fit a CU. A ring is
// exact for a chain whose queue window (queue_window; its bound is kept in the chain state) is
// below R: then each op of micro-batch m precedes every op of m + R of its stage on its device,
// so a slot is rewritten by m + R only after the readers of m have read it, and a reader of
// (s, m) can meet only generation m or m - R there, which the slot's parity bit tells apart. A
// chain whose window reaches R, or whose times pass the 40-bit slots, is left as it was and
// joins the redo list, which k_tune then steps.
template <int VMAX>
__global__ void __launch_bounds__(WAVE) k_tune_ring(TuneArgs t) {
  extern __shared__ __align__(16) uint8_t smem[];
  const SimArgs& a = t.s;
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  const int gg = g < a.CPW ? g : 0;
  const Table40 T{reinterpret_cast<uint32_t*>(smem), smem + (size_t)a.slots * a.CPW * 4,
                  __ffs(a.CPW) - 1, gg};
  uint8_t* rec = smem + (size_t)gg * a.rec_stride;  // until the table is cleared
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  const int gl = lane_id() - d;
  const Ring ring = make_ring(M, a.ring);
  const int64_t n_groups = (int64_t)gridDim.x * a.CPW;
  const int64_t total = t.list ? (int64_t)*t.list_n : t.n_chains;
  for (int64_t base = (int64_t)blockIdx.x * a.CPW; base < total; base += n_groups) {
    const bool has = g < a.CPW && base + g < total;
    const int64_t chain = has ? (t.list ? (int64_t)t.list[base + g] : base + g) : 0;
    uint8_t* crec = t.chains + chain * t.chain_stride;
    int64_t* cstate = reinterpret_cast<int64_t*>(crec + a.pr.stride);
    uint16_t* row = t.queues + ((size_t)chain * P + (d < P ? d : 0)) * a.qcap;
    if (has) stage_record(rec, crec, a.rec_bytes, d, G);
    __asm__ volatile("" ::: "memory");

    bool skip = !has;
    int v = 1, gen = GEN_AFAB, split = 0;
    int64_t cur = 0, w0 = 0;
    if (has) {
      if (t.step == 0) {
        Resolved r = resolve_record(a.pr, crec);
        if (!r.valid || r.n_pert != 0) {
          if (d == 0) cstate[0] = OCTO_MS_INVALID, cstate[1] = 0;
          if (d < P) cstate[2 + d] = OCTO_MS_INVALID;
          skip = true;
        }
        v = r.v, gen = r.gen, split = r.split;
      } else {
        cur = cstate[0];
        w0 = cstate[window_word(P)];
        Resolved r = resolve_record(a.pr, rec);
        if (cur == OCTO_MS_INVALID || !r.valid || r.n_pert != 0) skip = true;
        v = r.valid ? r.v : 1;
        split = r.split;
      }
    }
    const int S = P * v;
    const int qlen = (split ? 3 : 2) * v * M;

    Move mv;
    mv.kind = -1, mv.valid = true, mv.pair = 0, mv.sd = 0;
    if (!skip && t.step > 0) mv = propose(t.seed, chain, t.step, rec, a.pr, S, qlen, row, d);
    const int pair = __shfl(mv.pair, gl + (mv.sd < G ? mv.sd : 0));
    __asm__ volatile("" ::: "memory");
    const bool valid = mv.valid;
    int64_t win = pair > w0 ? pair : w0;

    Chunks<VMAX> c;
    int64_t busy = 0, stat = 0;
    int wl = 0;
    const bool eval = !skip && valid;
    if (eval && d < P) {
      busy = setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, split, ring, nullptr, &stat);
      if (t.step == 0) {
        materialise<VMAX>(a, c, v, gen, split, row);
        wl = queue_window<VMAX>(row, qlen);
      }
    } else {
      zero_chunks<VMAX>(c);
    }
    if (t.step == 0) win = group_max((int64_t)wl, G);
    const bool fits = win < ring.R;
    const bool run = eval && fits;
    __asm__ volatile("" ::: "memory");
    T.clear_all(a.slots, lane_id(), WAVE);  // every chain's rows fit a.slots
    __asm__ volatile("" ::: "memory");
    Lane L;
    L.clock = 0, L.pos = 0, L.nops = run && d < P ? qlen : 0, L.mem = L.peak = 0;
    bool dead = false;
    rounds_mat<VMAX, XP>(row, a.qcap, c, ring, L, T, G, gbit, lsb, dead, nullptr);
    const int64_t ms = group_max(L.clock, G);

    if (!has || skip) continue;
    if (eval && (!fits || ms >= Table40::LIMIT)) {
      // stepped again by k_tune, from the state this step started with
      unswap(mv, row, d);
      if (d == 0) a.redo[atomicAdd(&a.ctl[CTL_REDO], 1)] = (int32_t)chain;
      continue;
    }
    const bool keep = t.step == 0 || (valid && !dead && (cur < 0 || ms <= cur));
    if (keep) {
      if (d == 0) {
        cstate[0] = dead ? OCTO_MS_DEADLOCK : ms;
        cstate[1] = t.step == 0 ? 0 : cstate[1] + 1;
        cstate[window_word(P)] = win;
        // the record in LDS is gone (the table took its place): apply the move to the chain's
        if (mv.kind == 0) {
          crec[4 + mv.mi - 1] = (uint8_t)mv.nb;
        } else if (mv.kind == 1) {
          uint8_t* dv = crec + 3 + a.pr.s_max;
          for (int s = 0; s < S; ++s)
            dv[s] = dv[s] == mv.d1 ? (uint8_t)mv.d2 : dv[s] == mv.d2 ? (uint8_t)mv.d1 : dv[s];
        }
      }
      if (d < P) cstate[2 + d] = dead ? OCTO_MS_DEADLOCK : ms - busy;
    } else {
      unswap(mv, row, d);
    }
  }
}


// ---------------------------------------------------------------------------------------------
// Algorithm 1 of §6 (iterative bubble-aware tuning), one search per record, all records in
// lockstep iterations. Per iteration: k_alg1_expand picks each record's phase from its bubble
// breakdown and writes that phase's neighbourhood into one compacted batch; the batch is
// evaluated like any other (bounds variant); k_alg1_select keeps each record's best neighbour
// when it shortens the makespan. One wave per record in both kernels.
// ---------------------------------------------------------------------------------------------

// Search state per record (int32 words): the phase searched this iteration, flags (bits 0..2:
// phases whose last search found nothing better; A1_OVER: the search has ended), the first
// neighbour's position in the batch and the neighbour count; for the insertions: the first
// placeholder's position, their number and the device searched.
constexpr int A1_PHASE = 0, A1_FLAGS = 1, A1_BASE = 2, A1_CNT = 3, A1_INSB = 4, A1_NINS = 5,
              A1_DR = 6, A1_WORDS = 8;
constexpr int A1_OVER = 8;
// Search options (octo_alg1_tune_ex flags)
constexpr int A1F_INSERT = 1, A1F_RANDOM = 2;
constexpr int A1_REC_MAX = 1664;  // largest record stride (S_max = 64, 255 moves)

struct A1Args {
  Problem pr;
  const int64_t* costs;    // [L][3]
  uint8_t* recs;           // [n] current records, updated in place
  int64_t n;
  int64_t* ms;             // [n] current makespan
  int64_t* bub;            // [n][P] current bubbles
  int64_t* bnd;            // [n][P][2] current first start, last finish
  int32_t* st;             // [n][A1_WORDS]
  int64_t* stats;          // [n][4] kept moves per phase, iterations that searched
  int64_t* pit;            // [n][3] (nullable): iterations that searched each phase
  int flags;               // A1F_*
  uint64_t seed;           // random phases: Philox key (seed, 0)
  int iter;                // this iteration (random phases: Philox counter word 1)
  int32_t* ins_list;       // records whose insertions k_alg1_insert finds this iteration ...
  int32_t* ins_n;          // ... and their count
  uint8_t* nb_rec;         // neighbour records of this iteration, compacted
  const int64_t* nb_ms;    // [batch] their makespan
  const int64_t* nb_bub;   // [batch][P]
  const int64_t* nb_bnd;   // [batch][P][2]
  int32_t* total;          // neighbours written this iteration (atomic cursor)
};

__device__ __forceinline__ int64_t wave_sum64(int64_t x) {
  for (int o = WAVE >> 1; o > 0; o >>= 1) x += __shfl_xor(x, o);
  return x;
}
__device__ __forceinline__ int64_t wave_max64(int64_t x) {
  for (int o = WAVE >> 1; o > 0; o >>= 1) {
    const int64_t y = __shfl_xor(x, o);
    x = y > x ? y : x;
  }
  return x;
}
__device__ __forceinline__ int64_t wave_min64(int64_t x) {
  for (int o = WAVE >> 1; o > 0; o >>= 1) {
    const int64_t y = __shfl_xor(x, o);
    x = y < x ? y : x;
  }
  return x;
}
// Lane of the largest x, the lowest such lane on ties.
__device__ __forceinline__ int wave_argmax64(int64_t x) {
  int i = lane_id();
  for (int o = WAVE >> 1; o > 0; o >>= 1) {
    const int64_t y = __shfl_xor(x, o);
    const int j = __shfl_xor(i, o);
    if (y > x || (y == x && j < i)) x = y, i = j;
  }
  return i;
}

__global__ void k_alg1_init(int32_t* __restrict__ st, int64_t* __restrict__ stats,
                            int64_t* __restrict__ pit, int64_t n) {
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n;
       i += (int64_t)gridDim.x * blockDim.x) {
    for (int k = 0; k < A1_WORDS; ++k) st[i * A1_WORDS + k] = 0;
    for (int k = 0; k < 4; ++k) stats[i * 4 + k] = 0;
    if (pit)
      for (int k = 0; k < 3; ++k) pit[i * 3 + k] = 0;
  }
}

// One neighbour as byte edits of the current record: edited spans [lo, hi) and what goes there.
struct A1Edit {
  int kind;  // 0 layer migration, 1 stage exchange, 2 stage dispersion, 3 policy, 4 op swap,
             // 5 insertion placeholder (the record with its flags byte set: invalid until
             //   k_alg1_insert writes a move into it)
  int x, y;  // 0: boundaries x+1..y shift by -1 (x < y) or x+1..y by +1 (swapped: y < x holds
             //    the lower stage); 1: stages x, y; 3: new policy; 4: device x, position y
  int lo1, hi1, lo2, hi2;
};

// Byte p of the neighbour (p inside one of its spans). rec: the current record, reserved bytes
// cleared; S, v: its stage count and stages per device.
__device__ __forceinline__ uint32_t a1_byte(const A1Edit& e, const uint8_t* rec, int p, int L,
                                            int s_max, int S, int v, int po) {
  auto bnd = [&](int s) -> int { return s == 0 ? 0 : s == S ? L : rec[3 + s]; };
  switch (e.kind) {
    case 0:  // boundary b[k] at byte 3 + k
      return (uint32_t)(rec[p] + e.x);
    case 1: {
      const int s = p - 3 - s_max;
      return rec[3 + s_max + (s == e.x ? e.y : e.x)];
    }
    case 2: {
      if (p == 1) return (uint32_t)(2 * v);
      if (p == 2) return 0;
      if (p < 4) return rec[p];
      if (p < 3 + s_max) {  // new boundary k: stage k/2 split at its middle layer
        const int k = p - 3;
        if (k >= 2 * S) return 0;
        const int s = k >> 1;
        return (uint32_t)((k & 1) ? bnd(s) + (bnd(s + 1) - bnd(s)) / 2 : bnd(s));
      }
      const int s = p - 3 - s_max;  // new stage s on the device of old stage s mod S
      return s < 2 * S ? rec[3 + s_max + s % S] : 0;
    }
    case 3:
      return p == 0 ? (uint32_t)e.x : p == 2 ? 0u : rec[p];
    case 5:
      return 1u;  // the flags byte
    default: {
      if (p == 2) return (uint32_t)(rec[2] + 1);
      const int q = p - (po + 6 * rec[2]);  // the appended move {device, from, to}, u16 LE
      const int val = q < 2 ? e.x : q < 4 ? e.y : e.y + 1;
      return (uint32_t)((q & 1) ? (val >> 8) & 0xFF : val & 0xFF);
    }
  }
}

// Algorithm 1's branch and the chosen phase's neighbourhood, written to the batch.
// Neighbourhoods, in order (their order settles ties between equal makespans):
//  0 partitioning: one layer migrates from a stage a of the most loaded device (largest busy
//    time) to a stage b of the least loaded one, the stages between passing it on; pairs (a, b)
//    ascending, a with at least two layers;
//  1 placement: the device with the largest bubble exchanges one of its stages with one of each
//    other device's (devices, then its stages, then theirs, ascending); then, when v can double
//    and every stage has two layers, every stage splits at its middle layer and the 2S stages
//    go round the old devices (new stage k on the device of old stage k mod S), moves cleared;
//  2 scheduling: each other policy (moves cleared); then, with a move slot free, each adjacent
//    swap of the device with the largest bubble between its first and last op, as a move; then
//    (A1F_INSERT) as many placeholders as that device can have overlap-aware insertions, which
//    k_alg1_insert fills.
// The phase: Algorithm 1's branch, or (A1F_RANDOM) the (u mod n)-th of the n open phases, u the
// first word of Philox4x64-10(counter (record, iteration, 1, 0), key (seed, 0)).
__global__ void __launch_bounds__(WAVE) k_alg1_expand(A1Args a) {
  __shared__ __align__(16) uint8_t rec[A1_REC_MAX];
  __shared__ uint8_t sd[64];     // stages of device d at sd[d v ..], ascending
  __shared__ uint8_t alist[8];   // partitioning: the loaded device's stages that can give a layer
  const int lane = lane_id();
  const int P = a.pr.P, M = a.pr.M, L = a.pr.L, s_max = a.pr.s_max, stride = a.pr.stride;
  const int po = pert_off(s_max);
  int64_t tl = INT64_MAX;  // t_layer = M * the smallest layer's F + B + W
  for (int l = lane; l < L; l += WAVE) {
    const int64_t c = a.costs[3 * l] + a.costs[3 * l + 1] + a.costs[3 * l + 2];
    tl = c < tl ? c : tl;
  }
  tl = wave_min64(tl) * M;
  for (int64_t i = blockIdx.x; i < a.n; i += gridDim.x) {
    int32_t* st = a.st + i * A1_WORDS;
    const int flags = st[A1_FLAGS];
    const int64_t ms = a.ms[i];
    if ((flags & A1_OVER) || ms < 0) {  // ended, or deadlocked / invalid: nothing to search
      if (lane == 0) st[A1_FLAGS] = flags | A1_OVER, st[A1_CNT] = 0;
      continue;
    }
    const bool dv = lane < P;
    const int64_t bub = dv ? a.bub[i * P + lane] : 0;
    const int64_t fs = dv ? a.bnd[(i * P + lane) * 2] : 0;
    const int64_t lf = dv ? a.bnd[(i * P + lane) * 2 + 1] : 0;
    const int64_t busy = ms - bub;
    const int64_t edge = fs + ms - lf;  // leading plus trailing idle: the boundary bubble
    const int64_t resid = bub - edge;
    const int64_t delta = wave_max64(dv ? bub : INT64_MIN) - wave_min64(dv ? bub : INT64_MAX);
    const int64_t b_bd = wave_sum64(dv ? edge : 0);
    const int64_t b_res = wave_sum64(dv ? bub : 0) - b_bd;
    const int pref = delta > tl ? 0 : b_bd > b_res ? 1 : 2;
    const int ex = flags & 7;
    int phase = !((ex >> pref) & 1) ? pref : !(ex & 1) ? 0 : !(ex & 2) ? 1 : !(ex & 4) ? 2 : -1;
    if (a.flags & A1F_RANDOM) {
      const int open = ~ex & 7, nopen = __popc(open);
      phase = -1;
      if (nopen > 0) {
        const U4 u = philox4x64_10((uint64_t)i, (uint64_t)a.iter, 1, 0, a.seed, 0);
        int r = (int)(u.x[0] % (uint64_t)nopen);
        for (int p = 0; p < 3; ++p) {
          const bool o = (open >> p) & 1;
          if (o && r == 0 && phase < 0) phase = p;
          r -= o && phase < 0 ? 1 : 0;
        }
      }
    }
    if (phase < 0) {  // every phase exhausted: converged
      if (lane == 0) st[A1_FLAGS] = flags | A1_OVER, st[A1_CNT] = 0;
      continue;
    }
    const int dmax = wave_argmax64(dv ? busy : INT64_MIN);
    const int dmin = wave_argmax64(dv ? -busy : INT64_MIN);
    const int d1 = wave_argmax64(dv ? bub : INT64_MIN);
    const int dr = wave_argmax64(dv ? resid : INT64_MIN);
    // the record, reserved boundary and placement bytes cleared (as every neighbour has them)
    const uint4* src = reinterpret_cast<const uint4*>(a.recs + i * stride);
    for (int q = lane; q < stride / 16; q += WAVE) reinterpret_cast<uint4*>(rec)[q] = src[q];
    __syncthreads();
    const int policy = rec[0], v = rec[1], np = rec[2];
    const int S = P * v;
    for (int p = 3 + S + lane; p < 3 + s_max; p += WAVE) rec[p] = 0;
    for (int p = 3 + s_max + S + lane; p < 3 + 2 * s_max; p += WAVE) rec[p] = 0;
    if (dv) {
      int k = 0;
      for (int s = 0; s < S; ++s)
        if (rec[3 + s_max + s] == lane) sd[lane * v + k++] = (uint8_t)s;
    }
    __syncthreads();
    auto bnd = [&](int s) -> int { return s == 0 ? 0 : s == S ? L : rec[3 + s]; };
    int cnt = 0, na = 0;
    if (phase == 0) {
      if (dmax != dmin) {
        for (int k = 0; k < v; ++k) {
          const int s = sd[dmax * v + k];
          if (bnd(s + 1) - bnd(s) >= 2) {
            if (lane == 0) alist[na] = (uint8_t)s;
            ++na;
          }
        }
        cnt = na * v;
      }
    } else if (phase == 1) {
      const bool thin = lane < S && bnd(lane + 1) - bnd(lane) < 2;
      const bool disp = 2 * v <= a.pr.v_max && __ballot(thin) == 0;
      cnt = (P - 1) * v * v + (disp ? 1 : 0);
    }
    const int qlen = (policy == POL_ZB ? 3 : 2) * v * M;
    const int nswap = phase == 2 && np < a.pr.max_pert ? qlen - 1 : 0;
    const int nins = phase == 2 && np < a.pr.max_pert && (a.flags & A1F_INSERT) ? qlen - 1 : 0;
    if (phase == 2) cnt = 3 + nswap + nins;
    int base = 0;
    if (lane == 0) {
      base = atomicAdd(a.total, cnt);
      st[A1_PHASE] = phase, st[A1_BASE] = base, st[A1_CNT] = cnt;
      st[A1_INSB] = base + 3 + nswap, st[A1_NINS] = nins, st[A1_DR] = dr;
      a.stats[i * 4 + 3] += 1;
      if (a.pit) a.pit[i * 3 + phase] += 1;
      if (nins > 0) a.ins_list[atomicAdd(a.ins_n, 1)] = (int32_t)i;
    }
    base = __shfl(base, 0);
    __syncthreads();
    for (int j = lane; j < cnt; j += WAVE) {
      A1Edit e;
      e.lo2 = e.hi2 = 0;
      if (phase == 0) {
        const int sa = alist[j / v], sb = sd[dmin * v + j % v];
        e.kind = 0;
        e.x = sa < sb ? -1 : 1;
        const int lo = sa < sb ? sa : sb, hi = sa < sb ? sb : sa;
        e.lo1 = 4 + lo, e.hi1 = 4 + hi;  // boundaries lo+1..hi
      } else if (phase == 1) {
        const int vv = v * v;
        if (j < (P - 1) * vv) {
          const int k2 = j / vv, r = j - k2 * vv;
          const int d2 = k2 < d1 ? k2 : k2 + 1;
          e.kind = 1;
          e.x = sd[d1 * v + r / v], e.y = sd[d2 * v + r % v];
          e.lo1 = 3 + s_max + e.x, e.hi1 = e.lo1 + 1;
          e.lo2 = 3 + s_max + e.y, e.hi2 = e.lo2 + 1;
        } else {
          e.kind = 2;
          e.lo1 = 1, e.hi1 = 3 + 2 * s_max;
        }
      } else if (j < 3) {
        e.kind = 3;
        e.x = j < policy ? j : j + 1;
        e.lo1 = 0, e.hi1 = 3;
      } else if (j < 3 + nswap) {
        e.kind = 4;
        e.x = dr, e.y = j - 3;
        e.lo1 = 2, e.hi1 = 3;
        e.lo2 = po + 6 * np, e.hi2 = e.lo2 + 6;
      } else {
        e.kind = 5;
        e.lo1 = 3, e.hi1 = 4;
      }
      uint4* dst = reinterpret_cast<uint4*>(a.nb_rec + (int64_t)(base + j) * stride);
      for (int q = 0; q < stride / 16; ++q) {
        uint4 x = reinterpret_cast<const uint4*>(rec)[q];
        const int p0 = 16 * q;
        if ((e.lo1 < p0 + 16 && e.hi1 > p0) || (e.lo2 < p0 + 16 && e.hi2 > p0)) {
          uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
          for (int b = 0; b < 16; ++b) {
            const int p = p0 + b;
            if ((p >= e.lo1 && p < e.hi1) || (p >= e.lo2 && p < e.hi2)) {
              const uint32_t nv = a1_byte(e, rec, p, L, s_max, S, v, po) & 0xFF;
              w[b >> 2] = (w[b >> 2] & ~(0xFFu << (8 * (b & 3)))) | (nv << (8 * (b & 3)));
            }
          }
          x = make_uint4(w[0], w[1], w[2], w[3]);
        }
        dst[q] = x;
      }
    }
    __syncthreads();
  }
}

// Overlap-aware insertions (§6 "Scheduling Tuning", the second policy) of the records on
// b.ins_list, written into the placeholders k_alg1_expand reserved. One group per record
// (64-bit finish tables), lane = device: the record's queues with its moves, the asynchronous
// rounds recording every op's start and finish, then the lane of the searched device walks its
// queue: at each position k >= 1 with A = Q[k-1], B = Q[k], if the device idles between them and
// A's output goes to another device while B does not run during that transfer [end A,
// end A + c], or B's input comes from another device while A does not run during that transfer
// (§5: a node overlaps when a computation runs beside it for a positive time), the first later
// op Z = Q[j] that is ready when A ends (each producer's end, plus the transfer time across
// devices) becomes the move (device, j, k) of the next placeholder (flags byte cleared, one
// more move). Placeholders left over stay invalid. The group's lanes share the walk: each takes
// every G-th position, then every G-th insertion point, and the insertions found are numbered
// in position order by a ballot.
template <int VMAX>
__global__ void __launch_bounds__(WAVE) k_alg1_insert(SimArgs a, A1Args b,
                                                      int64_t* __restrict__ tbuf) {
  extern __shared__ __align__(16) uint8_t smem[];
  const int G = a.G, P = a.pr.P, M = a.pr.M;
  const int g = lane_id() / G;
  const int d = lane_id() % G;
  uint8_t* lds_group = smem + (size_t)(g < a.CPW ? g : 0) * a.group_bytes;
  const auto T = group_table<false>(lds_group, a.slots);
  uint8_t* rec = lds_group + a.table_bytes;
  const int slot = (int)blockIdx.x * a.CPW + (g < a.CPW ? g : 0);
  const int dl = d < P ? d : 0;
  uint16_t* row = a.qscratch + ((size_t)slot * P + dl) * a.qcap;
  const size_t nodes = (size_t)3 * a.pr.s_max * M;
  // per slot: finish times, start times (node-indexed), then two rows of the searched queue
  int64_t* tb = tbuf + (size_t)slot * (2 * nodes + 2 * (size_t)a.qcap);
  int64_t* ts = tb + nodes;
  uint64_t gbit, lsb;
  group_bits(G, &gbit, &lsb);
  const int64_t n_groups = (int64_t)gridDim.x * a.CPW;
  const int64_t total = *b.ins_n;
  const Ring ring = make_ring(M, M);
  const int po = pert_off(a.pr.s_max);
  for (int64_t base = (int64_t)blockIdx.x * a.CPW; base < total; base += n_groups) {
    const bool has = g < a.CPW && base + g < total;
    const int64_t i = has ? (int64_t)b.ins_list[base + g] : 0;
    const uint8_t* grec = b.recs + i * a.pr.stride;
    if (has) stage_record(rec, grec, a.rec_bytes, d, G);
    __syncthreads();
    Resolved r;
    r.valid = 0, r.v = 1, r.split = 0, r.gen = GEN_AFAB, r.n_pert = 0;
    if (has) r = resolve_record(a.pr, grec);
    const bool valid = has && r.valid;
    const int v = valid ? r.v : 1;
    const int S = P * v;
    Chunks<VMAX> c;
    Lane L;
    L.clock = 0, L.pos = 0, L.nops = 0, L.mem = L.peak = 0;
    L.cm.reset();
    L.fs = -1;
    L.tb = tb, L.ts = ts, L.tl = nullptr, L.tS = S, L.tM = M, L.rnd = 0;
    if (valid && d < P) {
      (void)setup_chunks<VMAX>(c, a.pr, rec, a.pre, a.link, d, v, r.split, ring, nullptr,
                               nullptr, XR);
      L.nops = materialise<VMAX>(a, c, v, r.gen, r.split, row);
      const uint8_t* pp = grec + po;
      for (int q = 0; q < r.n_pert; ++q) {
        const int pd = pp[6 * q] | (pp[6 * q + 1] << 8);
        if (pd != d) continue;
        move_entry(row, pp[6 * q + 2] | (pp[6 * q + 3] << 8), pp[6 * q + 4] | (pp[6 * q + 5] << 8));
      }
    } else {
      zero_chunks<VMAX>(c);
    }
    const bool mine = valid && d < P;
    if (!mine) L.nops = 0;
    if (valid) T.clear(S * M, d, G);
    __syncthreads();
    bool dead = false;
    rounds_mat<VMAX, XT>(row, a.qcap, c, ring, L, T, G, gbit, lsb, dead, nullptr);
    __syncthreads();  // every lane's times visible to the group
    // the searched device's queue, decoded by every lane of the group: (1) per position p, when
    // the op could start (its inputs' arrivals) and, for an insertion before p, the end of
    // op p - 1 when the device idles there and a communication there is alone (else -1);
    // (2) per such p, the first later op ready by then; (3) the placeholders, in p order
    const int32_t* st = b.st + i * A1_WORDS;
    const int dr = has ? st[A1_DR] : 0, insb = has ? st[A1_INSB] : 0;
    const int nins = has ? st[A1_NINS] : 0, np = rec[2];
    const bool go = valid && !dead && nins > 0;
    Chunks<VMAX> cr;
    if (go) {
      (void)setup_chunks<VMAX>(cr, a.pr, rec, a.pre, a.link, dr, v, r.split, ring, nullptr,
                               nullptr, XR);
    } else {
      zero_chunks<VMAX>(cr);
    }
    const uint16_t* rrow = a.qscratch + ((size_t)slot * P + dr) * a.qcap;
    const int nq = go ? (r.split ? 3 : 2) * v * M : 0;
    int64_t* rdy = tb + 2 * nodes;
    int64_t* thr = rdy + a.qcap;
    auto node = [&](int kind, int s, int m) { return (kind * S + s) * M + m; };
    for (int q = d; q < nq && d < G; q += G) {
      const uint32_t eb = rrow[q];
      const int kindB = (eb >> 14) & 3, kB = (eb >> 11) & 7, mB = eb & 0x7FF;
      const int sB = pick<VMAX>(cr.st, kB);
      int64_t ry = 0;
      if (kindB == KF) {
        if (sB > 0) ry = tb[node(KF, sB - 1, mB)] + pick<VMAX>(cr.wF, kB);
      } else if (kindB == KB) {
        ry = tb[node(KF, sB, mB)];
        if (sB < S - 1) {
          const int64_t y = tb[node(KB, sB + 1, mB)] + pick<VMAX>(cr.wB, kB);
          ry = y > ry ? y : ry;
        }
      } else {
        ry = tb[node(KB, sB, mB)];
      }
      rdy[q] = ry;
      int64_t t = -1;
      if (q >= 1) {
        const uint32_t ea = rrow[q - 1];
        const int kindA = (ea >> 14) & 3, kA = (ea >> 11) & 7, mA = ea & 0x7FF;
        const int sA = pick<VMAX>(cr.st, kA);
        const int64_t finA = tb[node(kindA, sA, mA)], stA = ts[node(kindA, sA, mA)];
        const int64_t finB = tb[node(kindB, sB, mB)], stB = ts[node(kindB, sB, mB)];
        if (stB > finA) {
          const int cxA =
              kindA == KF ? pick<VMAX>(cr.xF, kA) : kindA == KB ? pick<VMAX>(cr.xB, kA) : 0;
          const int cxB =
              kindB == KF ? pick<VMAX>(cr.xF, kB) : kindB == KB ? pick<VMAX>(cr.xB, kB) : 0;
          bool alone = false;
          if (cxA & CX_OUT) {  // A's output in flight over [finA, finA + c]; does B run then?
            const int64_t hi =
                finA + (kindA == KF ? pick<VMAX>(cr.cF, kA) : pick<VMAX>(cr.cB, kA));
            alone = alone || (finB < hi ? finB : hi) - (stB > finA ? stB : finA) <= 0;
          }
          if (cxB & CX_IN) {  // B's input in flight from its producer's end; does A run then?
            const int64_t fx = tb[node(kindB, kindB == KF ? sB - 1 : sB + 1, mB)];
            const int64_t hi =
                fx + (kindB == KF ? pick<VMAX>(cr.wF, kB) : pick<VMAX>(cr.wB, kB));
            alone = alone || (finA < hi ? finA : hi) - (stA > fx ? stA : fx) <= 0;
          }
          t = alone ? finA : -1;
        }
      }
      thr[q] = t;
    }
    __syncthreads();  // the group's rdy and thr visible to all its lanes
    const uint64_t gmask = G >= WAVE ? ~0ull : ((1ull << G) - 1);
    const int g0 = lane_id() - d;
    int found = 0;
    for (int k0 = 0; k0 < nq; k0 += G) {
      const int k = k0 + d;
      int jk = -1;
      if (d < G && k >= 1 && k < nq) {
        const int64_t t = thr[k];
        // the first later op ready by t: eight readiness times loaded together per step
        if (t >= 0)
          for (int j0 = k + 1; j0 < nq && jk < 0; j0 += 8) {
            int64_t r8[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) r8[u] = j0 + u < nq ? rdy[j0 + u] : INT64_MAX;
#pragma unroll
            for (int u = 0; u < 8; ++u) jk = jk < 0 && r8[u] <= t ? j0 + u : jk;
          }
      }
      const uint64_t gm = (__ballot(jk >= 0) >> g0) & gmask;
      const int at = found + __popcll(gm & ((1ull << d) - 1));
      if (jk >= 0 && at < nins) {
        uint8_t* nb = b.nb_rec + (int64_t)(insb + at) * a.pr.stride;
        nb[3] = 0;
        nb[2] = (uint8_t)(np + 1);
        uint8_t* mv = nb + po + 6 * np;
        mv[0] = (uint8_t)dr, mv[1] = 0;
        mv[2] = (uint8_t)(jk & 0xFF), mv[3] = (uint8_t)(jk >> 8);
        mv[4] = (uint8_t)(k & 0xFF), mv[5] = (uint8_t)(k >> 8);
      }
      found += __popcll(gm);
    }
    __syncthreads();  // before the next record reuses the staged record and the tables
  }
}

// Each record's best neighbour — the smallest makespan among those that neither deadlock nor
// are invalid, the first in neighbourhood order on ties — replaces it iff strictly shorter; the
// phase is then fresh again for all three phases, else this phase is exhausted.
__global__ void __launch_bounds__(WAVE) k_alg1_select(A1Args a) {
  const int lane = lane_id();
  const int P = a.pr.P, stride = a.pr.stride;
  for (int64_t i = blockIdx.x; i < a.n; i += gridDim.x) {
    int32_t* st = a.st + i * A1_WORDS;
    const int flags = st[A1_FLAGS];
    if (flags & A1_OVER) continue;
    const int phase = st[A1_PHASE], base = st[A1_BASE], cnt = st[A1_CNT];
    int64_t best = INT64_MAX;
    int bj = INT32_MAX;
    for (int j = lane; j < cnt; j += WAVE) {
      const int64_t x = a.nb_ms[base + j];
      if (x >= 0 && x < best) best = x, bj = j;
    }
    for (int o = WAVE >> 1; o > 0; o >>= 1) {
      const int64_t y = __shfl_xor(best, o);
      const int k = __shfl_xor(bj, o);
      if (y < best || (y == best && k < bj)) best = y, bj = k;
    }
    if (bj != INT32_MAX && best < a.ms[i]) {
      const int64_t nb = base + bj;
      const uint4* src = reinterpret_cast<const uint4*>(a.nb_rec + nb * stride);
      uint4* dst = reinterpret_cast<uint4*>(a.recs + i * stride);
      for (int q = lane; q < stride / 16; q += WAVE) dst[q] = src[q];
      if (lane < P) {
        a.bub[i * P + lane] = a.nb_bub[nb * P + lane];
        a.bnd[(i * P + lane) * 2] = a.nb_bnd[(nb * P + lane) * 2];
        a.bnd[(i * P + lane) * 2 + 1] = a.nb_bnd[(nb * P + lane) * 2 + 1];
      }
      if (lane == 0) {
        a.ms[i] = best;
        a.stats[i * 4 + phase] += 1;
        st[A1_FLAGS] = 0;
      }
    } else if (lane == 0) {
      st[A1_FLAGS] = flags | (1 << phase);
    }
  }
}

}  // namespace octo

// =============================================================================================
// Host side
// =============================================================================================
using namespace octo;

namespace {

struct Workspace {
  void* base = nullptr;  // per-call scratch (control words, prefix sums, bins, queues)
  size_t bytes = 0;
  // MERGE tables: their own allocation, kept between calls for the same (P, v_max, M)
  void* mt = nullptr;
  size_t mt_bytes = 0;
  bool mt_valid = false;
  int mt_P = 0, mt_vmax = 0, mt_M = 0;
  // v = 2 MERGE queues by stage pair (k_merge_rows), rebuilt with the MERGE tables
  void* mr = nullptr;
  size_t mr_bytes = 0;
  // largest number of micro-batches in flight per stage, per generated bin of v = 1, 2
  int inflight[NBIN_GEN] = {};
  int if_P = 0, if_M = 0, if_vmax = 0;
  // queue tables for v <= 2 (INTER by rank, MERGE by stage pair), same cache key as mt
  void* qt = nullptr;
  size_t qt_bytes = 0;
  bool qt_valid = false;
  int qt_P = 0, qt_vmax = 0, qt_M = 0;
  int qt_R[2] = {}, qt_lg[2] = {};  // launch geometry the entries were encoded for, per v
  int64_t qt_inter[2][2] = {}, qt_merge[2] = {}, qt_end = 0;
  // Algorithm 1: search state and each iteration's neighbour batch
  void* a1 = nullptr;
  size_t a1_bytes = 0;
  // reordered coordination: per-slot finish times, receive lists and programs
  void* ord = nullptr;
  size_t ord_bytes = 0;
  // static round schedules of the structure classes and their metadata, same cache key as mt;
  // st_ok: the tables exist (false: k_static_build does not fit this problem)
  void* st = nullptr;
  size_t st_bytes = 0;
  bool st_valid = false, st_ok = false;
  int st_P = 0, st_vmax = 0, st_M = 0;
};

std::mutex g_mu;
std::map<std::pair<int, hipStream_t>, Workspace> g_ws;
hipEvent_t g_prof[8] = {};  // measurement hook: events at the simulation-kernel boundaries
int g_prof_n = 0;

struct DevInfo {
  int cus = 0;
  int lds_max = 0;
  bool ok = false;
};
std::map<int, DevInfo> g_dev;

// The static scratch of octo_sim_batch_noalloc: every device buffer that call needs besides its
// inputs and outputs — control words, prefix sums, bins, candidate lists, materialised-queue
// rows and the MERGE and queue tables — is carved from this array, one copy per GPU, held until
// the process ends. Host code never passes the symbol itself (on the host it is only a stand-in
// name): it looks up each device's address of the array once (hipGetSymbolAddress, with that
// device current) and uses that address everywhere.
static __device__ __align__(256) uint8_t scratch[OCTO_NOALLOC_SCRATCH_BYTES];
struct ScratchDev {
  char* ptr = nullptr;  // this device's address of `scratch` (null until looked up)
  Workspace ws;         // the regions carved from it; tables cached there between calls
};
std::map<int, ScratchDev> g_scratch;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int check_problem(const octo_problem* p) {
  if (!p) return OCTO_EINVAL;
  if (p->L < 1 || p->L > 255 || p->P < 1 || p->P > 64 || p->v_max < 1 || p->v_max > 8 ||
      p->P * p->v_max > 64 || p->M < 1 || p->M > 2047 || p->max_pert < 0 || p->max_pert > 255)
    return OCTO_EINVAL;
  const int need = octo_record_stride(p->P, p->v_max, p->max_pert);
  if (p->cand_stride < need || p->cand_stride % 16 != 0) return OCTO_EINVAL;
  return OCTO_OK;
}

int dev_info(int dev, DevInfo* out) {
  auto it = g_dev.find(dev);
  if (it != g_dev.end()) {
    *out = it->second;
    return OCTO_OK;
  }
  DevInfo di;
  if (hipDeviceGetAttribute(&di.cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
    return OCTO_EHIP;
  if (hipDeviceGetAttribute(&di.lds_max, hipDeviceAttributeMaxSharedMemoryPerBlock, dev) !=
      hipSuccess)
    return OCTO_EHIP;
  di.ok = true;
  g_dev[dev] = di;
  *out = di;
  return OCTO_OK;
}

struct Plan {
  int G, CPW, slots, table_bytes, rec_bytes, rec_stride, group_bytes, lds_bytes, qcap;
  int strm_off;  // table-driven plans: per-lane stream table after the finish tables
};

// Entries per materialised queue row: 3 v_max M rounded up to a multiple of eight, so that rows
// start 16-byte aligned and read in whole 16-byte spans.
int queue_cap(const octo_problem* p) { return (int)align_up((size_t)3 * p->v_max * p->M, 8); }

int lanes_per_candidate(int P) {
  int G = 1;
  while (G < P) G <<= 1;
  return G;
}

// 40-bit-slot plan for generated queues with up to s_cap stages; the staged record shares the
// table's memory.
// s_cap stages of R slots (rounded up to 16, so that both slot arrays are 16-byte aligned and
// sized); streams > 0: a per-lane table of that many {w, dur} pairs.
Plan fast_plan(const octo_problem* p, int lds_max, int s_cap, int R, int streams) {
  Plan pl;
  pl.G = lanes_per_candidate(p->P);
  pl.slots = (int)align_up((size_t)s_cap * R, 16);
  pl.rec_bytes = pert_off(p->P * p->v_max);
  pl.rec_stride = (int)align_up(pl.rec_bytes, 16);
  pl.table_bytes = (int)(pl.slots * 4 + pl.slots);
  pl.group_bytes = (int)align_up(std::max<size_t>(pl.table_bytes, pl.rec_stride), 16);
  const int strm = streams * WAVE * 8;
  pl.CPW = std::min(WAVE / pl.G, (lds_max - strm) / pl.group_bytes);
  while (pl.CPW & (pl.CPW - 1)) pl.CPW &= pl.CPW - 1;  // interleaving uses shifts
  pl.strm_off = (int)align_up((size_t)pl.CPW * pl.group_bytes, 16);
  pl.lds_bytes = streams > 0 ? pl.strm_off + strm : pl.CPW * pl.group_bytes;
  pl.qcap = queue_cap(p);
  return pl;
}

// 40-bit ring plan with one table per group (groups that run their own phases gain nothing from
// interleaving): s_cap stages of R slots, then the staged record.
Plan ring_plan(const octo_problem* p, int lds_max, int s_cap, int R) {
  Plan pl;
  pl.G = lanes_per_candidate(p->P);
  pl.slots = (int)align_up((size_t)s_cap * R, 16);
  pl.rec_bytes = pert_off(p->P * p->v_max);
  pl.rec_stride = (int)align_up(pl.rec_bytes, 16);
  pl.table_bytes = pl.slots * 5;
  pl.group_bytes = pl.table_bytes + pl.rec_stride;
  pl.CPW = std::min(WAVE / pl.G, lds_max / pl.group_bytes);
  pl.lds_bytes = pl.CPW * pl.group_bytes;
  pl.strm_off = 0;
  pl.qcap = queue_cap(p);
  return pl;
}

// 64-bit-slot plan for materialised queues and tuner chains (record staged separately).
Plan big_plan(const octo_problem* p, int lds_max) {
  Plan pl;
  pl.G = lanes_per_candidate(p->P);
  pl.slots = p->P * p->v_max * p->M;
  pl.rec_bytes = pert_off(p->P * p->v_max);
  pl.rec_stride = (int)align_up(pl.rec_bytes, 16);
  pl.table_bytes = (int)align_up((size_t)pl.slots * 8, 16);
  pl.group_bytes = pl.table_bytes + (int)align_up(pl.rec_bytes, 16);
  pl.CPW = std::min(WAVE / pl.G, lds_max / pl.group_bytes);
  pl.lds_bytes = pl.CPW * pl.group_bytes;
  pl.strm_off = 0;
  pl.qcap = queue_cap(p);
  return pl;
}

size_t mtab_entries(const octo_problem* p) {
  return p->v_max >= 2 ? (size_t)merge_offset(p->P, p->M, p->v_max + 1, 0) : 0;
}

// v = 2 MERGE queue rows (k_merge_rows): entries per row, and the bytes of all rows.
int merge_row_stride(const octo_problem* p) { return (int)align_up((size_t)6 * p->M, 8); }
size_t merge_rows_bytes(const octo_problem* p) {
  return (size_t)2 * (2 * p->P) * (2 * p->P) * merge_row_stride(p) * 2;
}

// Workspace layout (byte offsets).
struct Layout {
  size_t ctl, pre, pre_mem, bin_of, idx, redo, wide, qscr, total;
};

Layout layout(const octo_problem* p, const Plan& big, int64_t n, int64_t mat_slots) {
  Layout l;
  size_t o = 0;
  l.ctl = o;
  o = align_up(o + CTL_WORDS * 4, 256);
  l.pre = o;
  o = align_up(o + (size_t)(p->L + 1) * 3 * 8, 256);
  l.pre_mem = o;
  o = align_up(o + (size_t)(p->L + 1) * 2 * 8, 256);
  l.bin_of = o;
  o = align_up(o + (size_t)n, 256);
  l.idx = o;
  o = align_up(o + (size_t)n * 4, 256);
  l.redo = o;
  o = align_up(o + (size_t)n * 4, 256);
  l.wide = o;
  o = align_up(o + (size_t)n * 4, 256);
  l.qscr = o;
  o = align_up(o + (size_t)mat_slots * p->P * big.qcap * 2, 256);
  l.total = o;
  return l;
}

// Grow-only device buffer, stream-ordered: the old one is released after the work already
// queued on the stream and the new one serves the work queued after it, so the host never
// waits (the buffer belongs to this stream's workspace and no other stream uses it).
int ensure_buf(void*& ptr, size_t& have, size_t bytes, hipStream_t stream) {
  if (have >= bytes) return OCTO_OK;
  size_t want = std::max(bytes, have * 3 / 2);
  if (ptr) {
    if (hipFreeAsync(ptr, stream) != hipSuccess) return OCTO_EHIP;
    ptr = nullptr;
    have = 0;
  }
  if (hipMallocAsync(&ptr, want, stream) != hipSuccess) {
    ptr = nullptr;
    (void)hipGetLastError();
    if (hipMallocAsync(&ptr, bytes, stream) != hipSuccess) {
      ptr = nullptr;
      (void)hipGetLastError();
      return OCTO_ENOMEM;
    }
    want = bytes;
  }
  have = want;
  return OCTO_OK;
}

template <typename K>
int occupancy_grid(K kernel, int lds, int cus, int* grid) {
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(kernel),
                            hipFuncAttributeMaxDynamicSharedMemorySize, lds);
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, kernel, WAVE, lds) != hipSuccess)
    return OCTO_EHIP;
  if (per_cu < 1) return OCTO_EUNSUPPORTED;
  *grid = per_cu * cus;
  return OCTO_OK;
}

int launch_ok() { return hipGetLastError() == hipSuccess ? OCTO_OK : OCTO_EHIP; }

struct Setup {
  Plan big;
  Layout l;
  Workspace* ws;
  DevInfo di;
  int mat_grid;
  Plan m40;      // 40-bit ring plan of k_sim_mat40 (CPW 0: does not fit)
  int m40_grid;  // its blocks (queue rows of the workspace are sized for them too)
  int m40_ring;  // its rows per stage
  Plan m40f;     // 40-bit full-row plan of its wide pass (CPW 0: does not fit)
  int m40f_grid;
};

template <int VC>
int mat_grid_for(const Plan& big, int cus, int* g) {
  // the accounting variants are sized the same way; the memory variant's grid is taken for all
  return occupancy_grid(k_sim_mat<VC, XM>, big.lds_bytes, cus, g);
}

// Largest number of micro-batches of one stage in flight over one device queue of the
// interleaved order: forwards issued minus backwards, and minus weight-gradient ops when split.
int inflight_inter(int P, int v, int M, int r, int split, int lag) {
  GenInter g;
  g.init(P, v, M, r, split, lag);
  int nF[8] = {}, nB[8] = {}, nW[8] = {};
  int worst = 0;
  const int n = (split ? 3 : 2) * v * M;
  for (int i = 0; i < n; ++i) {
    const int k = g.k;
    if (g.kind == KF) {
      ++nF[k];
      worst = std::max(worst, nF[k] - nB[k]);
      if (split) worst = std::max(worst, nF[k] - nW[k]);
    } else if (g.kind == KB) {
      ++nB[k];
    } else {
      ++nW[k];
    }
    g.advance(true);
  }
  return worst;
}

// Per generated bin of v <= v_max: the in-flight bound of its queues. INTER queues depend on the
// device's first stage r; a MERGE queue keeps, for each of its stages s, the order of stage s in
// the ideal stage-level schedule (interleaved order on S devices, v = 1, device s), so its bound
// is the largest over those orders. AFAB keeps all M micro-batches in flight.
void compute_inflight(const octo_problem* p, Workspace& ws) {
  if (ws.if_P == p->P && ws.if_M == p->M && ws.if_vmax == p->v_max) return;
  const int P = p->P, M = p->M;
  for (int b = 0; b < NBIN_GEN; ++b) ws.inflight[b] = M;
  for (int v = 1; v <= p->v_max; ++v) {
    for (int split = 0; split <= 1; ++split) {
      int wi = 0, wm = 0;
      for (int r = 0; r < P; ++r)
        wi = std::max(wi, inflight_inter(P, v, M, r, split, split ? r : 0));
      const int S = P * v;
      for (int st = 0; st < S; ++st)
        wm = std::max(wm, inflight_inter(S, 1, M, st, split, split ? st : 0));
      ws.inflight[bin_of(v, GEN_INTER, split)] = wi;
      ws.inflight[bin_of(v, GEN_MERGE, split)] = wm;
    }
  }
  ws.if_P = P, ws.if_M = M, ws.if_vmax = p->v_max;
}

// Launch geometry of the table-driven k_sim launch for v (1 or 2): ring rows and plan.
struct TabGeom {
  Ring ring;
  Plan plan;
  int lg;
};
// wide: 16-byte stream records (two 8-byte units) with the activation delta or the output
// transfer.
TabGeom tab_geom(const octo_problem* p, int lds_max, int v, bool wide) {
  TabGeom t;
  t.ring = make_ring(p->M, v * p->P);
  t.plan = fast_plan(p, lds_max, v * p->P, qt_row_stride(t.ring), 3 * v * (wide ? 2 : 1));
  t.lg = t.plan.CPW > 0 ? __builtin_ctz(t.plan.CPW) : 0;
  return t;
}

// Geometry of the static round schedules for a problem: rounds a class may take (a lockstep
// pass takes about a device's op count plus the pipeline depth; twice the largest op count plus
// four times the stages is a safe cap, a class past it is marked invalid), entries per row (the
// cap rounded up to whole groups of sixteen rounds, plus sixteen sc_nop entries for the
// look-ahead of k_static), and the entries per class (P + 1 rows).
struct StGeom {
  int nr_cap, rowlen;
  int64_t cls;
  size_t bytes;  // tables, then NSC x 4 int32 of metadata
};
StGeom st_geom(const octo_problem* p) {
  StGeom g;
  g.nr_cap = 2 * 6 * p->M + 4 * 2 * p->P;
  g.rowlen = (g.nr_cap + 15) / 16 * 16 + 16;
  g.cls = (int64_t)(p->P + 1) * g.rowlen;
  g.bytes = align_up((size_t)NSC * g.cls * 4, 256) + NSC * 16;
  return g;
}

// Build the static round schedules (k_static_build) into the workspace when the problem shape
// changed or the MERGE tables were rebuilt; needs the MERGE tables (v_max >= 2) in place.
int build_static(const octo_problem* p, Workspace& ws, int lds_max, hipStream_t stream) {
  if (ws.st_valid && ws.st_P == p->P && ws.st_vmax == p->v_max && ws.st_M == p->M) return OCTO_OK;
  ws.st_valid = false;
  ws.st_ok = false;
  const size_t lds = sc_build_lds(p->P, p->M);
  if (p->M > 2047 || (int)lds > lds_max || p->P > WAVE) {
    ws.st_valid = true;  // no static schedules for this shape
    ws.st_P = p->P, ws.st_vmax = p->v_max, ws.st_M = p->M;
    return OCTO_OK;
  }
  const StGeom g = st_geom(p);
  const int rc = ensure_buf(ws.st, ws.st_bytes, g.bytes, stream);
  if (rc) return rc;
  uint32_t* tab = static_cast<uint32_t*>(ws.st);
  int32_t* meta = reinterpret_cast<int32_t*>(static_cast<char*>(ws.st) + g.bytes - NSC * 16);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k_static_build),
                            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
  hipLaunchKernelGGL(k_static_build, dim3(NSC), dim3(WAVE), lds, stream, p->P, p->M, p->v_max,
                     static_cast<const uint32_t*>(ws.mt), tab, meta, g.cls, g.rowlen, g.nr_cap);
  if (hipGetLastError() != hipSuccess) return OCTO_EHIP;
  ws.st_valid = ws.st_ok = true;
  ws.st_P = p->P, ws.st_vmax = p->v_max, ws.st_M = p->M;
  return OCTO_OK;
}

// Queue tables for v = 1 and 2 (INTER rows per rank, MERGE rows per stage pair), encoded for
// each v's launch geometry; rebuilt when (P, v_max, M), the geometry or the MERGE tables
// change. Entry offsets are kept in the workspace.
// Entry offsets of the queue tables: INTER rows by (v, split), MERGE rows by split, and the
// final terminators; returns the number of entries, terminators included.
int64_t qtab_offsets(const octo_problem* p, int64_t inter[2][2], int64_t merge[2],
                     int64_t* end) {
  const int P = p->P, M = p->M, vmax2 = std::min(p->v_max, 2);
  int64_t off = 0;
  // rows of n entries + 2 terminators
  for (int v = 1; v <= 2; ++v)
    for (int split = 0; split <= 1; ++split) {
      inter[v - 1][split] = off;
      if (v <= vmax2) off += (int64_t)P * ((split ? 3 : 2) * v * M + 2);
    }
  const int S2 = 2 * P;
  const int64_t pairs = (int64_t)S2 * (S2 - 1) / 2;
  for (int split = 0; split <= 1; ++split) {
    merge[split] = off;
    if (vmax2 >= 2) off += pairs * ((split ? 3 : 2) * 2 * M + 2);
  }
  *end = off;
  // the final terminators: idle lanes start there, and a lane past its last op reads up to
  // two entries beyond its row
  return off + 3;
}

int build_qtab(const octo_problem* p, Workspace& ws, int lds_max, bool wide, hipStream_t stream) {
  const int P = p->P, M = p->M, vmax2 = std::min(p->v_max, 2);
  TabGeom geo[2] = {tab_geom(p, lds_max, 1, wide), tab_geom(p, lds_max, 2, wide)};
  bool same = ws.qt_valid && ws.qt_P == P && ws.qt_vmax == p->v_max && ws.qt_M == M;
  for (int v = 1; v <= vmax2; ++v)
    same = same && ws.qt_R[v - 1] == geo[v - 1].ring.R && ws.qt_lg[v - 1] == geo[v - 1].lg;
  if (same) return OCTO_OK;
  for (int v = 1; v <= vmax2; ++v)
    if (geo[v - 1].plan.CPW < 1) return OCTO_OK;  // no table-driven launch fits: generate
  const int64_t entries = qtab_offsets(p, ws.qt_inter, ws.qt_merge, &ws.qt_end);
  if (entries > INT32_MAX) return OCTO_OK;  // entry indices are 32-bit: generate instead
  const int64_t off = ws.qt_end;
  const int S2 = 2 * P;
  const int64_t pairs = (int64_t)S2 * (S2 - 1) / 2;
  ws.qt_valid = false;
  const size_t bytes = (size_t)entries * 4;
  const int rc = ensure_buf(ws.qt, ws.qt_bytes, bytes, stream);
  if (rc) return rc;
  uint32_t* q = static_cast<uint32_t*>(ws.qt);
  for (int v = 1; v <= vmax2; ++v)
    for (int split = 0; split <= 1; ++split)
      hipLaunchKernelGGL(k_qtab_inter, dim3((P + 63) / 64), dim3(64), 0, stream,
                         q + ws.qt_inter[v - 1][split], P, v, M, split, geo[v - 1].ring.R,
                         geo[v - 1].lg);
  if (vmax2 >= 2)
    for (int split = 0; split <= 1; ++split)
      hipLaunchKernelGGL(k_qtab_merge, dim3((int)((pairs + 63) / 64)), dim3(64), 0, stream,
                         q + ws.qt_merge[split], static_cast<const uint32_t*>(ws.mt), P, M,
                         split, geo[1].ring.R, geo[1].lg);
  if (hipGetLastError() != hipSuccess) return OCTO_EHIP;
  ws.qt_valid = true;
  ws.qt_P = P, ws.qt_vmax = p->v_max, ws.qt_M = M;
  for (int v = 1; v <= 2; ++v) ws.qt_R[v - 1] = geo[v - 1].ring.R, ws.qt_lg[v - 1] = geo[v - 1].lg;
  hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(64), 0, stream, q + off, 3, QT_END);
  return OCTO_OK;
}

// Carve the device's static scratch for one octo_sim_batch_noalloc call: the MERGE tables,
// the v = 2 MERGE rows and the queue tables first (their sizes depend only on the problem, so
// they stay where they are, and stay cached, while the problem does not change), then the
// per-call part. Narrows the materialised-queue grids to the queue rows that fit after the
// per-call lists. On the first call on a device, looks up its address of the array.
int scratch_regions(const octo_problem* prob, int dev, int64_t n, Setup* su) {
  ScratchDev& sd = g_scratch[dev];
  if (!sd.ptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, scratch) != hipSuccess || !p) return OCTO_EHIP;
    sd.ptr = static_cast<char*>(p);
  }
  Workspace& ws = sd.ws;
  const size_t cap = OCTO_NOALLOC_SCRATCH_BYTES;
  const size_t mt = prob->v_max >= 2 ? align_up(std::max<size_t>(mtab_entries(prob) * 4, 256), 256)
                                     : 0;
  const size_t mr = prob->v_max >= 2 ? align_up(merge_rows_bytes(prob), 256) : 0;
  int64_t qi[2][2], qm[2], qe;
  const size_t qt = align_up((size_t)qtab_offsets(prob, qi, qm, &qe) * 4, 256);
  const size_t stb = align_up(st_geom(prob).bytes, 256);
  const size_t tables = mt + mr + qt + stb;
  // the per-call part without materialised-queue rows, then the rows that fit after it
  const size_t lists = layout(prob, su->big, n, 0).total;
  if (tables + lists > cap) return OCTO_ESCRATCH;
  const size_t row_bytes = (size_t)prob->P * su->big.qcap * 2;
  const int64_t slots = (int64_t)((cap - tables - lists) / row_bytes);
  auto narrow = [&](int& grid, int cpw) -> bool {
    if (cpw < 1 || grid < 1) return true;
    grid = (int)std::min<int64_t>(grid, slots / cpw);
    return grid >= 1;
  };
  if (!narrow(su->mat_grid, su->big.CPW) || !narrow(su->m40_grid, su->m40.CPW) ||
      !narrow(su->m40f_grid, su->m40f.CPW))
    return OCTO_ESCRATCH;
  char* base = sd.ptr;
  char* mt_p = mt ? base : nullptr;
  char* mr_p = mr ? base + mt : nullptr;
  char* qt_p = base + mt + mr;
  char* st_p = base + mt + mr + qt;
  // tables moved (another problem shape): rebuild them
  if (ws.mt != mt_p || ws.mt_bytes != mt || ws.mr != mr_p || ws.mr_bytes != mr ||
      ws.qt != qt_p || ws.qt_bytes != qt || ws.st != st_p || ws.st_bytes != stb)
    ws.mt_valid = ws.qt_valid = ws.st_valid = false;
  ws.mt = mt_p, ws.mt_bytes = mt;
  ws.mr = mr_p, ws.mr_bytes = mr;
  ws.qt = qt_p, ws.qt_bytes = qt;
  ws.st = st_p, ws.st_bytes = stb;
  ws.base = base + tables;
  ws.bytes = cap - tables;
  return OCTO_OK;
}

// Shared front half of octo_sim_batch and octo_tune_step: device, plans, workspace, prefix
// sums, MERGE tables.
// mem (nullable): layer memory [L][2], prefix-summed next to the costs.
// noalloc: take every buffer from the device's static scratch (octo_sim_batch_noalloc) instead
// of the grow-only workspace; the persistent materialised-queue launches are then narrowed to
// the queue rows that fit, and a batch whose other buffers do not fit is OCTO_ESCRATCH.
int prepare(const octo_problem* prob, const int64_t* costs, const int64_t* mem,
            hipStream_t stream, int64_t n, Setup* su, int64_t extra_slots = 0,
            bool noalloc = false) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return OCTO_EHIP;
  int rc = dev_info(dev, &su->di);
  if (rc) return rc;
  su->big = big_plan(prob, su->di.lds_max);
  if (su->big.CPW < 1) return OCTO_EUNSUPPORTED;
  rc = prob->v_max <= 2 ? mat_grid_for<2>(su->big, su->di.cus, &su->mat_grid)
                        : mat_grid_for<8>(su->big, su->di.cus, &su->mat_grid);
  if (rc) return rc;
  su->m40_ring = make_ring(prob->M, 2 * prob->P * prob->v_max).R;
  su->m40 = fast_plan(prob, su->di.lds_max, prob->P * prob->v_max, su->m40_ring, 0);
  su->m40f = fast_plan(prob, su->di.lds_max, prob->P * prob->v_max, prob->M, 0);
  su->m40_grid = su->m40f_grid = 0;
  // the memory variant's grid bounds every variant's (as for k_sim_mat)
  if (su->m40.CPW >= 1) {
    rc = prob->v_max <= 2
             ? occupancy_grid(k_sim_mat40<2, XM>, su->m40.lds_bytes, su->di.cus, &su->m40_grid)
             : occupancy_grid(k_sim_mat40<8, XM>, su->m40.lds_bytes, su->di.cus, &su->m40_grid);
    if (rc) return rc;
  }
  if (su->m40f.CPW >= 1) {
    rc = prob->v_max <= 2
             ? occupancy_grid(k_sim_mat40<2, XM>, su->m40f.lds_bytes, su->di.cus, &su->m40f_grid)
             : occupancy_grid(k_sim_mat40<8, XM>, su->m40f.lds_bytes, su->di.cus, &su->m40f_grid);
    if (rc) return rc;
  }
  if (noalloc && (rc = scratch_regions(prob, dev, n, su))) return rc;
  su->l = layout(prob, su->big, n,
                 std::max<int64_t>({(int64_t)su->mat_grid * su->big.CPW,
                                    (int64_t)su->m40_grid * std::max(su->m40.CPW, 0),
                                    (int64_t)su->m40f_grid * std::max(su->m40f.CPW, 0),
                                    extra_slots}));
  Workspace& ws = noalloc ? g_scratch[dev].ws : g_ws[std::make_pair(dev, stream)];
  if (noalloc && su->l.total > ws.bytes) return OCTO_ESCRATCH;
  rc = ensure_buf(ws.base, ws.bytes, su->l.total, stream);
  if (rc) return rc;
  su->ws = &ws;
  char* base = static_cast<char*>(ws.base);
  hipLaunchKernelGGL(k_prep, dim3(1), dim3(256), 0, stream, costs, mem, prob->L,
                     reinterpret_cast<int64_t*>(base + su->l.pre),
                     reinterpret_cast<int64_t*>(base + su->l.pre_mem),
                     reinterpret_cast<int32_t*>(base + su->l.ctl));
  if ((rc = launch_ok())) return rc;
  if (prob->v_max >= 2) {
    void* old = ws.mt;
    rc = ensure_buf(ws.mt, ws.mt_bytes, std::max<size_t>(mtab_entries(prob) * 4, 256), stream);
    if (rc) return rc;
    if (ws.mt != old) ws.mt_valid = false;
    void* old_mr = ws.mr;
    rc = ensure_buf(ws.mr, ws.mr_bytes, merge_rows_bytes(prob), stream);
    if (rc) return rc;
    if (ws.mr != old_mr) ws.mt_valid = false;
  }
  if (prob->v_max >= 2 && !(ws.mt_valid && ws.mt_P == prob->P && ws.mt_vmax == prob->v_max &&
                            ws.mt_M == prob->M)) {
    const int lds = (int)align_up((size_t)prob->P * prob->v_max * prob->M * 8, 16);
    if (lds > su->di.lds_max) return OCTO_EUNSUPPORTED;
    (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k_merge_tab),
                              hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    hipLaunchKernelGGL(k_merge_tab, dim3(2 * (prob->v_max - 1)), dim3(WAVE), lds, stream, prob->P,
                       prob->M, 2, prob->v_max, static_cast<uint32_t*>(ws.mt));
    if ((rc = launch_ok())) return rc;
    const int rows = 2 * (2 * prob->P) * (2 * prob->P);
    hipLaunchKernelGGL(k_merge_rows, dim3((rows + WAVE - 1) / WAVE), dim3(WAVE), 0, stream,
                       prob->P, prob->M, static_cast<const uint32_t*>(ws.mt),
                       static_cast<uint16_t*>(ws.mr), merge_row_stride(prob));
    if ((rc = launch_ok())) return rc;
    ws.mt_valid = true;
    ws.mt_P = prob->P, ws.mt_vmax = prob->v_max, ws.mt_M = prob->M;
    ws.qt_valid = false;
    ws.st_valid = false;
  }
  return OCTO_OK;
}

SimArgs make_args(const octo_problem* prob, const Plan& pl, const Setup& su, const int64_t* link,
                  const void* cands, int64_t n, int64_t* ms, int64_t* bub,
                  int64_t* peak = nullptr) {
  char* base = static_cast<char*>(su.ws->base);
  const Layout& l = su.l;
  SimArgs a;
  a.pr = Problem{prob->L, prob->P, prob->v_max, prob->M, prob->cand_stride, prob->max_pert,
                 prob->P * prob->v_max};
  a.pre = reinterpret_cast<const int64_t*>(base + l.pre);
  a.pre_mem = peak ? reinterpret_cast<const int64_t*>(base + l.pre_mem) : nullptr;
  a.out_peak = peak;
  a.out_comm = nullptr;
  a.out_bound = nullptr;
  a.link = link;
  a.cands = static_cast<const uint8_t*>(cands);
  a.n = n;
  a.n_live = nullptr;
  a.mat_lists = 3;
  a.out_ms = ms;
  a.out_bub = bub;
  a.ctl = reinterpret_cast<int32_t*>(base + l.ctl);
  a.idx = reinterpret_cast<const int32_t*>(base + l.idx);
  a.redo = reinterpret_cast<int32_t*>(base + l.redo);
  a.wide = reinterpret_cast<int32_t*>(base + l.wide);
  a.mtab = static_cast<const uint32_t*>(su.ws->mt);
  a.mrows = prob->v_max >= 2 ? static_cast<const uint16_t*>(su.ws->mr) : nullptr;
  a.mrow_stride = merge_row_stride(prob);
  a.qscratch = reinterpret_cast<uint16_t*>(base + l.qscr);
  a.G = pl.G;
  a.CPW = pl.CPW;
  a.slots = pl.slots;
  a.table_bytes = pl.table_bytes;
  a.group_bytes = pl.group_bytes;
  a.rec_bytes = pl.rec_bytes;
  a.rec_stride = pl.rec_stride;
  a.qcap = pl.qcap;
  a.bin_mask = 0;
  a.work = CTL_WORK;
  a.ring = prob->M;
  a.redo_bins = 0;
  a.qtab = nullptr;
  for (int i = 0; i < 2; ++i) {
    a.qt_merge[i] = su.ws->qt_merge[i];
    a.qt_end = su.ws->qt_end;
    for (int j = 0; j < 2; ++j) a.qt_inter[i][j] = su.ws->qt_inter[i][j];
  }
  a.strm_off = pl.strm_off;
  a.stab = nullptr;
  a.smeta = nullptr;
  a.st_cls = 0;
  a.st_rowlen = 0;
  return a;
}

// Bits of the generated bins of v in [v_lo, v_hi], without AFAB (AFAB: only AFAB).
uint64_t bins_of(int v_lo, int v_hi, bool afab) {
  uint64_t m = 0;
  for (int v = v_lo; v <= v_hi; ++v)
    for (int b = first_bin(v); b < first_bin(v) + 5; ++b)
      if ((b == bin_of(v, GEN_AFAB, 0)) == afab) m |= 1ull << b;
  return m;
}

// Launch k_static over the class bins: CPW = 64 / G candidates per wave; the eight stream rows
// (4 KiB), each group's sc_slots(P) slots (256 or 512 B), then the staged records: 6.4 KB per
// wave at P = 8 (with 64-slot blocks, 8.4 KB and 1.28 instead of 1.13 ms per headline call).
int launch_static(const SimArgs& base, const Setup& su, int64_t n, hipStream_t stream) {
  SimArgs a = base;
  a.G = lanes_per_candidate(a.pr.P);
  a.CPW = WAVE / a.G;
  const int sbase = 8 * 512;
  const int rbase = sbase + a.CPW * sc_slots(a.pr.P) * 8;
  const int lds = rbase + a.CPW * a.rec_stride;
  if (lds > su.di.lds_max) return OCTO_OK;  // cannot happen for P <= 64; leave to k_sim
  int grid = 0;
  int rc = occupancy_grid(k_static, lds, su.di.cus, &grid);
  if (rc) return rc;
  const int64_t need = (n + a.CPW - 1) / a.CPW;
  grid = (int)std::max<int64_t>(1, std::min<int64_t>(grid, need));
  hipLaunchKernelGGL(k_static, dim3(grid), dim3(WAVE), lds, stream, a, sbase, rbase);
  return launch_ok();
}

// Launch k_sim<VC> over the generated bins in `mask` with its own 40-bit plan: s_cap stages of
// ring_want (rounded up to a power of two, or M) slots; bins whose in-flight bound exceeds the
// ring go to the 64-bit path, unless any_ring (rendezvous GPipe queues, exact with one slot per
// stage).
template <int VC, int X>
int launch_sim(const octo_problem* prob, const Setup& su, const int64_t* link, const void* cands,
               int64_t n, int64_t* ms, int64_t* bub, int64_t* peak, int64_t* comm,
               int64_t* bound, int s_cap, int ring_want, uint64_t mask, int work,
               hipStream_t stream, bool any_ring = false) {
  const Ring ring = make_ring(prob->M, ring_want);
  // table-driven launches (v <= 2) keep 3 v {w, dur} streams per lane in LDS and need tables
  // encoded for exactly this geometry
  bool tab = false;
  Plan pl{};
  if (VC <= 2 && X != XS && X != XR && su.ws->qt_valid) {
    const TabGeom geo = tab_geom(prob, su.di.lds_max, VC, X != XP);
    constexpr int vi = VC <= 2 ? VC - 1 : 0;
    tab = geo.plan.CPW >= 1 && geo.ring.R == ring.R && su.ws->qt_R[vi] == geo.ring.R &&
          su.ws->qt_lg[vi] == geo.lg && geo.plan.G * geo.plan.CPW <= WAVE;
    pl = geo.plan;
  }
  if (!tab) pl = fast_plan(prob, su.di.lds_max, s_cap, ring.R, 0);
  if (pl.CPW < 1) return OCTO_EUNSUPPORTED;
  SimArgs a = make_args(prob, pl, su, link, cands, n, ms, bub, peak);
  a.out_comm = comm;
  a.out_bound = bound;
  if (tab) a.qtab = static_cast<const uint32_t*>(su.ws->qt);
  a.bin_mask = mask, a.work = work;
  a.ring = ring.R;
  a.redo_bins = 0;
  for (int b = 0; b < NBIN_GEN && !any_ring; ++b)
    if (((mask >> b) & 1) && ring.R < prob->M && su.ws->inflight[b] > ring.R)
      a.redo_bins |= 1ull << b;
  int grid = 0;
  int rc = occupancy_grid(k_sim<VC, X>, pl.lds_bytes, su.di.cus, &grid);
  if (rc) return rc;
  const int64_t need = (n + pl.CPW - 1) / pl.CPW;
  grid = (int)std::max<int64_t>(1, std::min<int64_t>(grid, need));
  hipLaunchKernelGGL((k_sim<VC, X>), dim3(grid), dim3(WAVE), pl.lds_bytes, stream, a);
  return launch_ok();
}

// Launch k_afab over the AFAB bins of every v: one lane per candidate, each lane's row of M
// int64 plus 2 P device words in LDS (at most 64 KiB per wave).
template <int X>
int launch_afab(const octo_problem* prob, const Setup& su, const int64_t* link, const void* cands,
                int64_t n, int64_t* ms, int64_t* bub, int64_t* peak, int64_t* comm,
                int64_t* bound, hipStream_t stream) {
  // rows as line envelopes (plain, memory and bounds variants); the communication and
  // serialised-link variants, which need every op, keep rows of exactly 32 or 64 micro-batches
  // in registers and other lengths (and the communication variant's, whose unrolled sweep would
  // not fit the register file) in LDS
  constexpr bool LINES = X == XP || X == XM || X == XB;
  const int mmax = LINES ? -1 : X == XC ? 0 : prob->M == 32 ? 32 : prob->M == 64 ? 64 : 0;
  // per device: the clock, the busy time (in registers for the plain variant at P <= 8), then
  // the variant's own words
  const int words = (X == XM || X == XB) ? 3 : X == XC ? 4 : (X == XP && prob->P <= 8) ? 1 : 2;
  const size_t per_lane =
      (size_t)((mmax == 0 ? prob->M : 0) + words * prob->P +
               (X == XS ? 2 * prob->P * prob->v_max : 0)) *
      8;
  const int lanes = (int)std::min<size_t>(WAVE, std::max<size_t>(1, 65536 / per_lane));
  // line-envelope rows and serialised links: then the staged tables (prefix sums, memory prefix
  // sums, the link matrix) and each lane's record head
  const int tab_off = (int)align_up(lanes * per_lane, 16);
  const bool stage = LINES || X == XS;
  const int rec_off = tab_off + (stage ? (int)(((size_t)3 * (prob->L + 1) +
                                                (X == XM ? (size_t)2 * (prob->L + 1) : 0) +
                                                (size_t)prob->P * prob->P) *
                                               8)
                                       : 0);
  const int lds =
      rec_off + (stage ? lanes * (int)align_up(pert_off(prob->P * prob->v_max), 16) : 0);
  if (lds > su.di.lds_max) return OCTO_EUNSUPPORTED;
  SimArgs a = make_args(prob, su.big, su, link, cands, n, ms, bub, peak);
  a.out_comm = comm;
  a.out_bound = bound;
  a.bin_mask = bins_of(1, prob->v_max, true);
  a.work = CTL_WORK + 3;
  int grid = 0;
  const int64_t need = (n + lanes - 1) / lanes;
  if constexpr (LINES) {
    const int rc = occupancy_grid(k_afab<-1, X>, lds, su.di.cus, &grid);
    if (rc) return rc;
    grid = (int)std::max<int64_t>(1, std::min<int64_t>(grid, need));
    hipLaunchKernelGGL((k_afab<-1, X>), dim3(grid), dim3(WAVE), lds, stream, a, lanes, tab_off, rec_off);
  } else {
    const int rc = mmax == 32   ? occupancy_grid(k_afab<32, X>, lds, su.di.cus, &grid)
                   : mmax == 64 ? occupancy_grid(k_afab<64, X>, lds, su.di.cus, &grid)
                                : occupancy_grid(k_afab<0, X>, lds, su.di.cus, &grid);
    if (rc) return rc;
    grid = (int)std::max<int64_t>(1, std::min<int64_t>(grid, need));
    if (mmax == 32)
      hipLaunchKernelGGL((k_afab<32, X>), dim3(grid), dim3(WAVE), lds, stream, a, lanes, tab_off, rec_off);
    else if (mmax == 64)
      hipLaunchKernelGGL((k_afab<64, X>), dim3(grid), dim3(WAVE), lds, stream, a, lanes, tab_off, rec_off);
    else
      hipLaunchKernelGGL((k_afab<0, X>), dim3(grid), dim3(WAVE), lds, stream, a, lanes, tab_off, rec_off);
  }
  return launch_ok();
}

// MEM: the working queue rows are group slots of the workspace, sized for mat_grid blocks.
template <int VC, bool MEM>
int launch_tune(const TuneArgs& t, const Plan& pl, int cus, int mat_grid, int64_t n_chains,
                hipStream_t stream) {
  int grid = 0;
  int rc = occupancy_grid(k_tune<VC, MEM>, pl.lds_bytes, cus, &grid);
  if (rc) return rc;
  const int64_t need = (n_chains + pl.CPW - 1) / pl.CPW;
  grid = (int)std::max<int64_t>(1, std::min<int64_t>(grid, need));
  if (MEM) grid = std::min(grid, mat_grid);
  hipLaunchKernelGGL((k_tune<VC, MEM>), dim3(grid), dim3(WAVE), pl.lds_bytes, stream, t);
  return launch_ok();
}

// k_tune_ring over all chains, persistent blocks at the plan's occupancy.
template <int VC>
int launch_tune_ring(const TuneArgs& t, const Plan& pl, int cus, int64_t n_chains,
                     hipStream_t stream) {
  int grid = 0;
  int rc = occupancy_grid(k_tune_ring<VC>, pl.lds_bytes, cus, &grid);
  if (rc) return rc;
  const int64_t need = (n_chains + pl.CPW - 1) / pl.CPW;
  grid = (int)std::max<int64_t>(1, std::min<int64_t>(grid, need));
  hipLaunchKernelGGL((k_tune_ring<VC>), dim3(grid), dim3(WAVE), pl.lds_bytes, stream, t);
  return launch_ok();
}

// k_advance over n records (or the list); its queue rows are group slots of the workspace, of
// which there are at least max_grid blocks.
template <int VC, bool RING>
int launch_advance(const SimArgs& a, const Plan& pl, int cus, int max_grid, const int64_t* cap,
                   uint8_t* out, const int32_t* list, const int32_t* list_n, hipStream_t stream) {
  int grid = 0;
  int rc = occupancy_grid(k_advance<VC, RING>, pl.lds_bytes, cus, &grid);
  if (rc) return rc;
  const int64_t need = (a.n + pl.CPW - 1) / pl.CPW;
  grid = (int)std::max<int64_t>(1, std::min<int64_t>(std::min(grid, max_grid), need));
  hipLaunchKernelGGL((k_advance<VC, RING>), dim3(grid), dim3(WAVE), pl.lds_bytes, stream, a, cap,
                     out, list, list_n, RING ? CTL_WORK : CTL_WORK + 1);
  return launch_ok();
}

// The ring pass of octo_advance_w: its plan and its grid (0: no ring pass for this problem).
template <int VC>
int advance_ring_grid(const octo_problem* prob, const DevInfo& di, int64_t n, Plan* rp,
                      int* grid) {
  *grid = 0;
  const Ring rr = make_ring(prob->M, prob->P * prob->v_max);
  *rp = ring_plan(prob, di.lds_max, prob->P * prob->v_max, rr.R);
  if (rr.R >= prob->M || rp->CPW < 1) return OCTO_OK;
  int rc = occupancy_grid(k_advance<VC, true>, rp->lds_bytes, di.cus, grid);
  if (rc) return rc;
  *grid = (int)std::max<int64_t>(1, std::min<int64_t>(*grid, (n + rp->CPW - 1) / rp->CPW));
  return OCTO_OK;
}

int record_mark(int i, hipStream_t stream) {
  if (i < g_prof_n && g_prof[i] && hipEventRecord(g_prof[i], stream) != hipSuccess)
    return OCTO_EHIP;
  return OCTO_OK;
}

// Evaluation outputs besides makespan and bubbles (null where the kind has none).
struct Extra {
  int64_t* peak = nullptr;   // XM [n][P]
  int64_t* comm = nullptr;   // XC [n][4]
  int64_t* bound = nullptr;  // XB [n][P][2]
  const int32_t* n_live = nullptr;  // device count of the records to evaluate (<= n)
};

// Validity and bin of every record (k_classify writes the sentinels of invalid ones), bin
// offsets (k_plan; ctl[CTL_TOTAL] = the valid records), and the record indices sorted by bin
// (k_scatter, into the workspace's idx).
int classify_sort(const octo_problem* prob, const Setup& su, const SimArgs& a, int64_t n,
                  hipStream_t stream) {
  char* base = static_cast<char*>(su.ws->base);
  const int tb = CLS_THREADS;
  const int nb = (int)((n + (int64_t)tb * CLS_ITEMS - 1) / ((int64_t)tb * CLS_ITEMS));
  uint8_t* bins = reinterpret_cast<uint8_t*>(base + su.l.bin_of);
  const int hb = (int)align_up((size_t)pert_off(prob->P * prob->v_max), 16);
  (void)hipFuncSetAttribute(reinterpret_cast<const void*>(k_classify),
                            hipFuncAttributeMaxDynamicSharedMemorySize, tb * hb);
  hipLaunchKernelGGL(k_classify, dim3(nb), dim3(tb), tb * hb, stream, a, bins, hb);
  int rc = launch_ok();
  if (rc) return rc;
  hipLaunchKernelGGL(k_plan, dim3(1), dim3(WAVE), 0, stream, a.ctl);
  if ((rc = launch_ok())) return rc;
  hipLaunchKernelGGL(k_scatter, dim3(nb), dim3(tb), 0, stream, a, bins,
                     reinterpret_cast<int32_t*>(base + su.l.idx));
  return launch_ok();
}

// The batch evaluation behind octo_sim_batch (X = XP), octo_sim_batch_mem (XM),
// octo_sim_batch_comm (XC), octo_sim_batch_serial (XS: generated queues, not tables) and
// octo_sim_batch_bounds (XB). The caller has checked the arguments and holds g_mu.
template <int X>
int sim_batch_run(const octo_problem* prob, const int64_t* layer_costs, const int64_t* layer_mem,
                  const int64_t* link, const void* candidates, int64_t n, int64_t* out_makespan,
                  int64_t* out_bubble, const Extra& ex, hipStream_t stream,
                  bool noalloc = false) {
  constexpr bool MEM = X == XM;
  if (n == 0) return OCTO_OK;
  Setup su;
  int rc = prepare(prob, layer_costs, MEM ? layer_mem : nullptr, stream, n, &su, 0, noalloc);
  if (rc) return rc;
  int64_t* pk = MEM ? ex.peak : nullptr;
  int64_t* cm = X == XC ? ex.comm : nullptr;
  int64_t* bd = X == XB ? ex.bound : nullptr;
  SimArgs a = make_args(prob, su.big, su, link, candidates, n, out_makespan, out_bubble, pk);
  a.out_comm = cm;
  a.out_bound = bd;
  a.n_live = ex.n_live;
  // plain evaluations take the static round schedules for the structure classes
  if (X == XP) {
    if ((rc = build_static(prob, *su.ws, su.di.lds_max, stream))) return rc;
    if (su.ws->st_ok) {
      const StGeom sg = st_geom(prob);
      a.stab = static_cast<const uint32_t*>(su.ws->st);
      a.smeta = reinterpret_cast<const int32_t*>(static_cast<const char*>(su.ws->st) +
                                                 sg.bytes - NSC * 16);
      a.st_cls = sg.cls;
      a.st_rowlen = sg.rowlen;
    }
  }
  if ((rc = classify_sort(prob, su, a, n, stream))) return rc;
  // generated INTER / MERGE queues, one launch per v with finish tables sized for it (ring
  // rows of the next power of two >= P v where the in-flight bound allows): v = 2, v = 1, then
  // v = 3..8; then AFAB queues; then materialised queues (perturbations, 64-bit redo).
  compute_inflight(prob, *su.ws);
  if (X != XS && X != XR && (rc = build_qtab(prob, *su.ws, su.di.lds_max, X != XP, stream)))
    return rc;
  const int P = prob->P, M = prob->M;
  if ((rc = record_mark(0, stream))) return rc;
  if (a.smeta && (rc = launch_static(a, su, n, stream))) return rc;
  if ((rc = record_mark(1, stream))) return rc;
  if (prob->v_max >= 2 &&
      (rc = launch_sim<2, X>(prob, su, link, candidates, n, out_makespan, out_bubble, pk, cm, bd,
                             2 * P, 2 * P, bins_of(2, 2, false), CTL_WORK + 1, stream)))
    return rc;
  if ((rc = record_mark(2, stream))) return rc;
  if ((rc = launch_sim<1, X>(prob, su, link, candidates, n, out_makespan, out_bubble, pk, cm, bd,
                             P, P, bins_of(1, 1, false), CTL_WORK + 0, stream)))
    return rc;
  if ((rc = record_mark(3, stream))) return rc;
  for (int v = 3; v <= prob->v_max; ++v)
    if ((rc = launch_sim<8, X>(prob, su, link, candidates, n, out_makespan, out_bubble, pk, cm,
                               bd, P * v, P * v, bins_of(v, v, false), CTL_WORK_V + v - 3,
                               stream)))
      return rc;
  if ((rc = record_mark(4, stream))) return rc;
  if constexpr (X != XR) {
    if ((rc = launch_afab<X>(prob, su, link, candidates, n, out_makespan, out_bubble, pk, cm, bd,
                             stream)))
      return rc;
  } else {
    // rendezvous: GPipe queues in the generated kernels, per v class, with one slot per stage
    // (the blocking sends keep at most one value of a stage row untaken; relax_rdv)
    if (prob->v_max >= 2 &&
        (rc = launch_sim<2, X>(prob, su, link, candidates, n, out_makespan, out_bubble, pk, cm,
                               bd, 2 * P, 1, bins_of(2, 2, true), CTL_WORK + 4, stream, true)))
      return rc;
    if ((rc = launch_sim<1, X>(prob, su, link, candidates, n, out_makespan, out_bubble, pk, cm,
                               bd, P, 1, bins_of(1, 1, true), CTL_WORK + 5, stream, true)))
      return rc;
    for (int v = 3; v <= prob->v_max; ++v)
      if ((rc = launch_sim<8, X>(prob, su, link, candidates, n, out_makespan, out_bubble, pk, cm,
                                 bd, P * v, 1, bins_of(v, v, true), CTL_WORK_V + 6 + v - 3,
                                 stream, true)))
        return rc;
  }
  if ((rc = record_mark(5, stream))) return rc;
  // candidates with moves: 40-bit rings, 40-bit full rows for those wider than the ring, then
  // the 64-bit redo list
  bool m40_any = false;
  for (int pass = 0; pass < 2; ++pass) {
    const Plan& pl = pass == 0 ? su.m40 : su.m40f;
    // a ring as long as M needs no second pass; nor does a ring pass that did not fit (then
    // the full rows do not fit either and the 64-bit kernel takes every perturbed candidate)
    if (pass == 1 && (su.m40_ring >= M || su.m40.CPW < 1)) break;
    if (pl.CPW < 1) continue;
    SimArgs a40 = make_args(prob, pl, su, link, candidates, n, out_makespan, out_bubble, pk);
    a40.ring = pass == 0 ? su.m40_ring : M;
    a40.out_comm = cm;
    a40.out_bound = bd;
    int g40 = 0;
    rc = prob->v_max <= 2 ? occupancy_grid(k_sim_mat40<2, X>, pl.lds_bytes, su.di.cus, &g40)
                          : occupancy_grid(k_sim_mat40<8, X>, pl.lds_bytes, su.di.cus, &g40);
    if (rc) return rc;
    g40 = std::min(g40, pass == 0 ? su.m40_grid : su.m40f_grid);
    // pass 1 reads the wide list of pass 0; pass 0 sends wide candidates to the redo list when
    // no full-row pass follows
    const int wide = pass == 1 ? 1 : (su.m40_ring < M && su.m40f.CPW < 1 ? 2 : 0);
    if (prob->v_max <= 2)
      hipLaunchKernelGGL((k_sim_mat40<2, X>), dim3(g40), dim3(WAVE), pl.lds_bytes, stream, a40,
                         wide);
    else
      hipLaunchKernelGGL((k_sim_mat40<8, X>), dim3(g40), dim3(WAVE), pl.lds_bytes, stream, a40,
                         wide);
    if ((rc = launch_ok())) return rc;
    m40_any = true;
  }
  if (m40_any) a.mat_lists = 2;
  if (prob->v_max <= 2)
    hipLaunchKernelGGL((k_sim_mat<2, X>), dim3(su.mat_grid), dim3(WAVE), su.big.lds_bytes,
                       stream, a);
  else
    hipLaunchKernelGGL((k_sim_mat<8, X>), dim3(su.mat_grid), dim3(WAVE), su.big.lds_bytes,
                       stream, a);
  if ((rc = launch_ok())) return rc;
  return record_mark(6, stream);
}

// Argument checks and locking around sim_batch_run.
template <int X>
int sim_batch_impl(const octo_problem* prob, const int64_t* layer_costs, const int64_t* layer_mem,
                   const int64_t* link, const void* candidates, int64_t n, int64_t* out_makespan,
                   int64_t* out_bubble, const Extra& ex, hipStream_t stream,
                   bool noalloc = false) {
  int rc = check_problem(prob);
  if (rc) return rc;
  if (n < 0 || n > (int64_t)INT32_MAX) return OCTO_EINVAL;
  if (n == 0) return OCTO_OK;
  if (!layer_costs || !link || !candidates || !out_makespan || !out_bubble) return OCTO_EINVAL;
  if (X == XM && (!layer_mem || !ex.peak)) return OCTO_EINVAL;
  if (X == XC && !ex.comm) return OCTO_EINVAL;
  if (X == XB && !ex.bound) return OCTO_EINVAL;
  if ((reinterpret_cast<uintptr_t>(candidates) & 15) != 0) return OCTO_EINVAL;
  std::lock_guard<std::mutex> lock(g_mu);
  return sim_batch_run<X>(prob, layer_costs, layer_mem, link, candidates, n, out_makespan,
                          out_bubble, ex, stream, noalloc);
}

// The local-search step behind octo_tune_step (MEM = false) and octo_tune_step_mem.
template <bool MEM>
int tune_step_impl(const octo_problem* prob, const int64_t* layer_costs, const int64_t* layer_mem,
                   const int64_t* capacity, int32_t max_advance, const int64_t* link,
                   void* chains, uint16_t* queues, int64_t n_chains, uint64_t seed, int32_t step,
                   hipStream_t stream) {
  int rc = check_problem(prob);
  if (rc) return rc;
  if (n_chains < 0 || step < 0) return OCTO_EINVAL;
  if (MEM && (max_advance < 0 || max_advance > OCTO_MAX_ADVANCE)) return OCTO_EINVAL;
  if (n_chains == 0) return OCTO_OK;
  if (!layer_costs || !link || !chains || !queues) return OCTO_EINVAL;
  if (MEM && (!layer_mem || !capacity)) return OCTO_EINVAL;
  if ((reinterpret_cast<uintptr_t>(chains) & 15) != 0 ||
      (reinterpret_cast<uintptr_t>(queues) & 15) != 0)
    return OCTO_EINVAL;
  std::lock_guard<std::mutex> lock(g_mu);
  // the ring pass's redo list holds int32 chain indices, one per chain
  const bool ring_pass = !MEM && n_chains <= (int64_t)INT32_MAX;
  Setup su;
  rc = prepare(prob, layer_costs, MEM ? layer_mem : nullptr, stream, ring_pass ? n_chains : 0,
               &su);
  if (rc) return rc;
  TuneArgs t;
  t.s = make_args(prob, su.big, su, link, nullptr, 0, nullptr, nullptr);
  if (MEM)
    t.s.pre_mem = reinterpret_cast<const int64_t*>(static_cast<char*>(su.ws->base) + su.l.pre_mem);
  t.chains = static_cast<uint8_t*>(chains);
  t.chain_stride = octo_chain_stride(prob);
  t.queues = queues;
  t.n_chains = n_chains;
  t.seed = seed;
  t.step = step;
  t.cap = capacity;
  t.max_adv = max_advance;
  t.list = nullptr;
  t.list_n = nullptr;
  if (ring_pass) {
    // rings of the smallest power of two >= P v_max rows, the window of the interleaved orders
    // the chains start from; chains with wider windows (or larger times) go to k_tune
    const Ring rr = make_ring(prob->M, prob->P * prob->v_max);
    const Plan rp = fast_plan(prob, su.di.lds_max, prob->P * prob->v_max, rr.R, 0);
    if (rr.R < prob->M && rp.CPW >= 1) {
      TuneArgs tr = t;
      tr.s = make_args(prob, rp, su, link, nullptr, 0, nullptr, nullptr);
      tr.s.ring = rr.R;
      // chains in queue-length order (the groups of a wave run in lockstep)
      const int nb = (int)((n_chains + 255) / 256);
      int32_t* order = const_cast<int32_t*>(tr.s.idx);
      hipLaunchKernelGGL(k_chain_count, dim3(nb), dim3(256), 0, stream, tr);
      if ((rc = launch_ok())) return rc;
      hipLaunchKernelGGL(k_plan, dim3(1), dim3(WAVE), 0, stream, tr.s.ctl);
      if ((rc = launch_ok())) return rc;
      hipLaunchKernelGGL(k_chain_scatter, dim3(nb), dim3(256), 0, stream, tr, order);
      if ((rc = launch_ok())) return rc;
      tr.list = order;
      tr.list_n = tr.s.ctl + CTL_TOTAL;
      rc = prob->v_max <= 2 ? launch_tune_ring<2>(tr, rp, su.di.cus, n_chains, stream)
                            : launch_tune_ring<8>(tr, rp, su.di.cus, n_chains, stream);
      if (rc) return rc;
      t.list = tr.s.redo;
      t.list_n = tr.s.ctl + CTL_REDO;
    }
  }
  return prob->v_max <= 2
             ? launch_tune<2, MEM>(t, su.big, su.di.cus, su.mat_grid, n_chains, stream)
             : launch_tune<8, MEM>(t, su.big, su.di.cus, su.mat_grid, n_chains, stream);
}


// Neighbour slots one record can need in one iteration of Algorithm 1 (the largest of the three
// neighbourhoods over v <= v_max).
int64_t alg1_slots(const octo_problem* p) {
  const int64_t v = p->v_max;
  // scheduling: 3 policies, qlen - 1 swaps and qlen - 1 insertion placeholders
  return std::max({v * v, (int64_t)(p->P - 1) * v * v + 1, 6 * v * p->M + 1});
}

// Algorithm 1 behind octo_alg1_tune: state and batch in the workspace's a1 buffer, iterations
// enqueued back to back on the stream (no host synchronisation).
int alg1_impl(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
              void* records, int64_t n, int32_t iters, int32_t flags, uint64_t seed,
              int64_t* out_makespan, int64_t* out_bubble, int64_t* out_stats,
              int64_t* out_phase_iters, hipStream_t stream) {
  int rc = check_problem(prob);
  if (rc) return rc;
  if (n < 0 || iters < 0) return OCTO_EINVAL;
  if (n == 0) return OCTO_OK;
  const int64_t slots = alg1_slots(prob);
  if (n > (int64_t)INT32_MAX / slots || prob->cand_stride > A1_REC_MAX) return OCTO_EINVAL;
  if (!layer_costs || !link || !records || !out_makespan || !out_bubble || !out_stats)
    return OCTO_EINVAL;
  if ((flags & ~(A1F_INSERT | A1F_RANDOM)) != 0) return OCTO_EINVAL;
  if ((reinterpret_cast<uintptr_t>(records) & 15) != 0) return OCTO_EINVAL;
  const int64_t nb = n * slots;
  std::lock_guard<std::mutex> lock(g_mu);
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return OCTO_EHIP;
  // the insertion pass: 64-bit finish tables, one group per record; its grid bounds the group
  // slots whose finish and start times it keeps
  int ins_grid = 0;
  Setup su;
  if (flags & A1F_INSERT) {
    if ((rc = prepare(prob, layer_costs, nullptr, stream, n, &su))) return rc;
    if ((rc = prob->v_max <= 2
                  ? occupancy_grid(k_alg1_insert<2>, su.big.lds_bytes, su.di.cus, &ins_grid)
                  : occupancy_grid(k_alg1_insert<8>, su.big.lds_bytes, su.di.cus, &ins_grid)))
      return rc;
    ins_grid = (int)std::max<int64_t>(
        1, std::min<int64_t>(std::min(ins_grid, su.mat_grid), (n + su.big.CPW - 1) / su.big.CPW));
  }
  const size_t nodes = (size_t)3 * prob->P * prob->v_max * prob->M;
  Workspace& ws = g_ws[std::make_pair(dev, stream)];
  const int P = prob->P;
  size_t o = 0;
  const size_t o_total = o;
  o = align_up(o + 256, 256);
  const size_t o_bnd = o;
  o = align_up(o + (size_t)n * P * 16, 256);
  const size_t o_st = o;
  o = align_up(o + (size_t)n * A1_WORDS * 4, 256);
  const size_t o_rec = o;
  o = align_up(o + (size_t)nb * prob->cand_stride, 256);
  const size_t o_ms = o;
  o = align_up(o + (size_t)nb * 8, 256);
  const size_t o_bub = o;
  o = align_up(o + (size_t)nb * P * 8, 256);
  const size_t o_nbnd = o;
  o = align_up(o + (size_t)nb * P * 16, 256);
  const size_t o_ins = o;
  o = align_up(o + (size_t)n * 4, 256);
  const size_t o_tbuf = o;
  o = align_up(o + (size_t)ins_grid * std::max(su.big.CPW, 0) *
                       (2 * nodes + 2 * (size_t)std::max(su.big.qcap, 0)) * 8,
                256);
  if ((rc = ensure_buf(ws.a1, ws.a1_bytes, o, stream))) return rc;
  char* base = static_cast<char*>(ws.a1);
  A1Args a;
  a.pr = Problem{prob->L, prob->P, prob->v_max, prob->M, prob->cand_stride, prob->max_pert,
                 prob->P * prob->v_max};
  a.costs = layer_costs;
  a.recs = static_cast<uint8_t*>(records);
  a.n = n;
  a.ms = out_makespan;
  a.bub = out_bubble;
  a.bnd = reinterpret_cast<int64_t*>(base + o_bnd);
  a.st = reinterpret_cast<int32_t*>(base + o_st);
  a.stats = out_stats;
  a.pit = out_phase_iters;
  a.flags = flags;
  a.seed = seed;
  a.iter = 0;
  a.ins_list = reinterpret_cast<int32_t*>(base + o_ins);
  a.ins_n = reinterpret_cast<int32_t*>(base + o_total) + 1;
  a.nb_rec = reinterpret_cast<uint8_t*>(base + o_rec);
  a.nb_ms = reinterpret_cast<int64_t*>(base + o_ms);
  a.nb_bub = reinterpret_cast<int64_t*>(base + o_bub);
  a.nb_bnd = reinterpret_cast<int64_t*>(base + o_nbnd);
  a.total = reinterpret_cast<int32_t*>(base + o_total);
  const int grid = (int)std::min<int64_t>(n, 1 << 16);
  hipLaunchKernelGGL(k_alg1_init, dim3((int)std::min<int64_t>((n + 255) / 256, 1024)), dim3(256),
                     0, stream, a.st, a.stats, a.pit, n);
  if ((rc = launch_ok())) return rc;
  Extra cur;
  cur.bound = a.bnd;
  if ((rc = sim_batch_run<XB>(prob, layer_costs, nullptr, link, records, n, out_makespan,
                              out_bubble, cur, stream)))
    return rc;
  Extra nbx;
  nbx.bound = reinterpret_cast<int64_t*>(base + o_nbnd);
  nbx.n_live = a.total;
  for (int it = 0; it < iters; ++it) {
    a.iter = it;
    hipLaunchKernelGGL(k_fill_u32, dim3(1), dim3(WAVE), 0, stream,
                       reinterpret_cast<uint32_t*>(a.total), 2, 0u);  // cursor, insertion count
    if ((rc = launch_ok())) return rc;
    hipLaunchKernelGGL(k_alg1_expand, dim3(grid), dim3(WAVE), 0, stream, a);
    if ((rc = launch_ok())) return rc;
    if (flags & A1F_INSERT) {
      if ((rc = prepare(prob, layer_costs, nullptr, stream, n, &su))) return rc;
      SimArgs sa = make_args(prob, su.big, su, link, records, n, nullptr, nullptr);
      int64_t* tbuf = reinterpret_cast<int64_t*>(static_cast<char*>(ws.a1) + o_tbuf);
      if (prob->v_max <= 2)
        hipLaunchKernelGGL(k_alg1_insert<2>, dim3(ins_grid), dim3(WAVE), su.big.lds_bytes, stream,
                           sa, a, tbuf);
      else
        hipLaunchKernelGGL(k_alg1_insert<8>, dim3(ins_grid), dim3(WAVE), su.big.lds_bytes, stream,
                           sa, a, tbuf);
      if ((rc = launch_ok())) return rc;
    }
    if ((rc = sim_batch_run<XB>(prob, layer_costs, nullptr, link, a.nb_rec, nb,
                                reinterpret_cast<int64_t*>(base + o_ms),
                                reinterpret_cast<int64_t*>(base + o_bub), nbx, stream)))
      return rc;
    hipLaunchKernelGGL(k_alg1_select, dim3(grid), dim3(WAVE), 0, stream, a);
    if ((rc = launch_ok())) return rc;
  }
  return OCTO_OK;
}


// The reordered coordinations behind octo_sim_batch_ordered (REORDER false) and
// octo_sim_batch_reorder (REORDER true): k_ordered over all records, one group per candidate —
// first on 40-bit ring tables (when the ring is shorter than M), then on 64-bit full rows over
// the candidates the ring pass left (or over all of them). The scratch (finish-time buffers,
// receive keys or communication items, programs) is sized for the larger pass's group slots.
template <int VC, bool REORDER>
int launch_ordered(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                   const void* cands, int64_t n, int64_t* ms, int64_t* bub, int64_t* stats,
                   hipStream_t stream) {
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return OCTO_EHIP;
  DevInfo di;
  int rc = dev_info(dev, &di);
  if (rc) return rc;
  OrdBufs ob;
  ob.rcap = REORDER ? 0 : 2 * prob->v_max * prob->M;
  ob.pcap = (int)align_up((size_t)7 * prob->v_max * prob->M, 4);  // whole 16-byte entries
  // communication items: at most a receive and a send per F or B
  ob.icap = REORDER ? 4 * prob->v_max * prob->M : 0;
  ob.pcap2 = REORDER ? queue_cap(prob) + 1 : 0;
  const size_t nodes = (size_t)3 * prob->P * prob->v_max * prob->M;
  // at most 4 GiB of scratch per launch: per group slot the finish times (REORDER: start times
  // and levels too) and queue rows, per lane the receive keys or the communication items and gap
  // tables, and the program
  const size_t per_slot = nodes * (REORDER ? 8 + 8 + 4 : 8) + (size_t)prob->P * queue_cap(prob) * 2;
  const size_t per_lane = (size_t)ob.rcap * 12 + (size_t)ob.pcap * 4 + (size_t)ob.icap * 16 +
                          (size_t)ob.pcap2 * 16;
  auto grid_of = [&](auto kern, const Plan& pl, int* g) {
    int rc2 = occupancy_grid(kern, pl.lds_bytes, di.cus, g);
    if (rc2) return rc2;
    *g = (int)std::max<int64_t>(1, std::min<int64_t>(*g, (n + pl.CPW - 1) / pl.CPW));
    const size_t per_wave = per_slot * pl.CPW + per_lane * WAVE;
    *g = (int)std::min<int64_t>(*g, std::max<int64_t>(1, (int64_t)(((size_t)4 << 30) / per_wave)));
    return 0;
  };
  // pass 1: rings; pass 2: 40-bit full rows for the orders too wide for the ring
  const Ring rr = make_ring(prob->M, prob->P * prob->v_max);
  const Plan rp = ring_plan(prob, di.lds_max, prob->P * prob->v_max, rr.R);
  const Plan fp = ring_plan(prob, di.lds_max, prob->P * prob->v_max, prob->M);
  int rgrid = 0, fgrid = 0;
  if (rr.R < prob->M && rp.CPW >= 1) {
    if ((rc = grid_of(k_ordered<VC, true, REORDER>, rp, &rgrid))) return rc;
    if (fp.CPW >= 1 && (rc = grid_of(k_ordered<VC, true, REORDER>, fp, &fgrid))) return rc;
  }
  Setup su;
  if ((rc = prepare(prob, layer_costs, nullptr, stream, n, &su))) return rc;
  int grid = 0;
  if ((rc = occupancy_grid(k_ordered<VC, false, REORDER>, su.big.lds_bytes, su.di.cus, &grid)))
    return rc;
  grid = (int)std::max<int64_t>(
      1, std::min<int64_t>(std::min(grid, su.mat_grid), (n + su.big.CPW - 1) / su.big.CPW));
  // group slots: the ring pass's and the full-row pass's share the same buffers (one at a time)
  const size_t slots = std::max({(size_t)grid * su.big.CPW, (size_t)rgrid * std::max(rp.CPW, 0),
                                 (size_t)fgrid * std::max(fp.CPW, 0)});
  const size_t waves = std::max({(size_t)grid, (size_t)rgrid, (size_t)fgrid});
  const size_t qslots = (size_t)su.mat_grid * su.big.CPW;
  if (slots > qslots) {
    // the queue rows of the workspace cover mat_grid * CPW slots; take a larger workspace
    if ((rc = prepare(prob, layer_costs, nullptr, stream, n, &su, (int64_t)slots))) return rc;
  }
  size_t o = 0;
  auto take = [&](size_t bytes) {
    const size_t at = o;
    o = align_up(o + bytes, 256);
    return at;
  };
  const size_t lanes = waves * WAVE;
  const size_t o_tb = take(slots * nodes * 8);
  const size_t o_rk = take(lanes * ob.rcap * 8);
  const size_t o_ri = take(lanes * ob.rcap * 4);
  const size_t o_pg = take(lanes * ob.pcap * 4);
  const size_t o_ts = take(REORDER ? slots * nodes * 8 : 0);
  const size_t o_tl = take(REORDER ? slots * nodes * 4 : 0);
  const size_t o_it = take(lanes * ob.icap * 16);
  const size_t o_ps = take(lanes * ob.pcap2 * 8);
  const size_t o_pd = take(lanes * ob.pcap2 * 8);
  if ((rc = ensure_buf(su.ws->ord, su.ws->ord_bytes, o, stream))) return rc;
  char* base = static_cast<char*>(su.ws->ord);
  ob.tb = reinterpret_cast<int64_t*>(base + o_tb);
  ob.rkey = reinterpret_cast<int64_t*>(base + o_rk);
  ob.rid = reinterpret_cast<uint32_t*>(base + o_ri);
  ob.prog = reinterpret_cast<uint4*>(base + o_pg);
  ob.ts = reinterpret_cast<int64_t*>(base + o_ts);
  ob.tl = reinterpret_cast<int32_t*>(base + o_tl);
  ob.items = reinterpret_cast<CItem*>(base + o_it);
  ob.pst = reinterpret_cast<int64_t*>(base + o_ps);
  ob.pdur = reinterpret_cast<int64_t*>(base + o_pd);
  ob.stats = stats;
  if (stats) {  // sentinels for the invalid records, which no group takes
    hipLaunchKernelGGL(k_fill_i64, dim3((unsigned)std::min<int64_t>(1024, (2 * n + 255) / 256)),
                       dim3(256), 0, stream, stats, 2 * n, (int64_t)OCTO_MS_INVALID);
    if ((rc = launch_ok())) return rc;
  }
  SimArgs a = make_args(prob, su.big, su, link, cands, n, ms, bub);
  // the valid records sorted by (v, generator, split), so that the groups of a wave have queues
  // and programs of one length (invalid ones get their sentinels here)
  if ((rc = classify_sort(prob, su, a, n, stream))) return rc;
  const int32_t* list = a.idx;
  const int32_t* list_n = a.ctl + CTL_TOTAL;
  if (rgrid > 0) {
    SimArgs ar = make_args(prob, rp, su, link, cands, n, ms, bub);
    ar.ring = rr.R;
    hipLaunchKernelGGL((k_ordered<VC, true, REORDER>), dim3(rgrid), dim3(WAVE), rp.lds_bytes,
                       stream, ar, ob, list, list_n, fgrid > 0 ? 1 : 0);
    if ((rc = launch_ok())) return rc;
    if (fgrid > 0) {
      SimArgs af = make_args(prob, fp, su, link, cands, n, ms, bub);
      af.ring = prob->M;
      hipLaunchKernelGGL((k_ordered<VC, true, REORDER>), dim3(fgrid), dim3(WAVE), fp.lds_bytes,
                         stream, af, ob, a.wide, a.ctl + CTL_WIDE, 0);
      if ((rc = launch_ok())) return rc;
    }
    list = a.redo;
    list_n = a.ctl + CTL_REDO;
  }
  hipLaunchKernelGGL((k_ordered<VC, false, REORDER>), dim3(grid), dim3(WAVE), su.big.lds_bytes,
                     stream, a, ob, list, list_n, 0);
  return launch_ok();
}

int ordered_impl(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                 const void* candidates, int64_t n, int64_t* out_makespan, int64_t* out_bubble,
                 bool reorder, int64_t* out_stats, hipStream_t stream) {
  int rc = check_problem(prob);
  if (rc) return rc;
  if (n < 0 || n > (int64_t)INT32_MAX) return OCTO_EINVAL;
  if (n == 0) return OCTO_OK;
  if (!layer_costs || !link || !candidates || !out_makespan || !out_bubble) return OCTO_EINVAL;
  if ((reinterpret_cast<uintptr_t>(candidates) & 15) != 0) return OCTO_EINVAL;
  std::lock_guard<std::mutex> lock(g_mu);
  if (reorder)
    return prob->v_max <= 2 ? launch_ordered<2, true>(prob, layer_costs, link, candidates, n,
                                                      out_makespan, out_bubble, out_stats, stream)
                            : launch_ordered<8, true>(prob, layer_costs, link, candidates, n,
                                                      out_makespan, out_bubble, out_stats, stream);
  return prob->v_max <= 2 ? launch_ordered<2, false>(prob, layer_costs, link, candidates, n,
                                                     out_makespan, out_bubble, nullptr, stream)
                          : launch_ordered<8, false>(prob, layer_costs, link, candidates, n,
                                                     out_makespan, out_bubble, nullptr, stream);
}

}  // namespace

extern "C" {

int32_t octo_record_pert_offset(int32_t P, int32_t v_max) {
  if (P < 1 || P > 64 || v_max < 1 || v_max > 8 || P * v_max > 64) return OCTO_EINVAL;
  return pert_off(P * v_max);
}

int32_t octo_record_stride(int32_t P, int32_t v_max, int32_t max_pert) {
  if (P < 1 || P > 64 || v_max < 1 || v_max > 8 || P * v_max > 64 || max_pert < 0 ||
      max_pert > 255)
    return OCTO_EINVAL;
  const int need = pert_off(P * v_max) + 6 * max_pert;
  return (need + 15) / 16 * 16;
}

int32_t octo_chain_stride(const octo_problem* prob) {
  if (check_problem(prob)) return OCTO_EINVAL;
  return (int32_t)align_up((size_t)prob->cand_stride + 8 * (window_word(prob->P) + 1), 16);
}

int32_t octo_queue_capacity(const octo_problem* prob) {
  if (check_problem(prob)) return OCTO_EINVAL;
  return queue_cap(prob);
}

int octo_sim_batch(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                   const void* candidates, int64_t n, int64_t* out_makespan, int64_t* out_bubble,
                   void* stream) {
  return sim_batch_impl<XP>(prob, layer_costs, nullptr, link, candidates, n, out_makespan,
                            out_bubble, Extra{}, static_cast<hipStream_t>(stream));
}

int octo_sim_batch_noalloc(const octo_problem* prob, const int64_t* layer_costs,
                           const int64_t* link, const void* candidates, int64_t n,
                           int64_t* out_makespan, int64_t* out_bubble, void* stream) {
  return sim_batch_impl<XP>(prob, layer_costs, nullptr, link, candidates, n, out_makespan,
                            out_bubble, Extra{}, static_cast<hipStream_t>(stream), true);
}

int octo_sim_batch_mem(const octo_problem* prob, const int64_t* layer_costs,
                       const int64_t* layer_mem, const int64_t* link, const void* candidates,
                       int64_t n, int64_t* out_makespan, int64_t* out_bubble, int64_t* out_peak,
                       void* stream) {
  Extra ex;
  ex.peak = out_peak;
  return sim_batch_impl<XM>(prob, layer_costs, layer_mem, link, candidates, n, out_makespan,
                            out_bubble, ex, static_cast<hipStream_t>(stream));
}

int octo_sim_batch_serial(const octo_problem* prob, const int64_t* layer_costs,
                          const int64_t* link, const void* candidates, int64_t n,
                          int64_t* out_makespan, int64_t* out_bubble, void* stream) {
  return sim_batch_impl<XS>(prob, layer_costs, nullptr, link, candidates, n, out_makespan,
                            out_bubble, Extra{}, static_cast<hipStream_t>(stream));
}

int octo_sim_batch_rdv(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                       const void* candidates, int64_t n, int64_t* out_makespan,
                       int64_t* out_bubble, void* stream) {
  return sim_batch_impl<XR>(prob, layer_costs, nullptr, link, candidates, n, out_makespan,
                            out_bubble, Extra{}, static_cast<hipStream_t>(stream));
}

int octo_sim_batch_ordered(const octo_problem* prob, const int64_t* layer_costs,
                           const int64_t* link, const void* candidates, int64_t n,
                           int64_t* out_makespan, int64_t* out_bubble, void* stream) {
  return ordered_impl(prob, layer_costs, link, candidates, n, out_makespan, out_bubble, false,
                      nullptr, static_cast<hipStream_t>(stream));
}

int octo_sim_batch_reorder(const octo_problem* prob, const int64_t* layer_costs,
                           const int64_t* link, const void* candidates, int64_t n,
                           int64_t* out_makespan, int64_t* out_bubble, int64_t* out_stats,
                           void* stream) {
  return ordered_impl(prob, layer_costs, link, candidates, n, out_makespan, out_bubble, true,
                      out_stats, static_cast<hipStream_t>(stream));
}

int octo_sim_batch_bounds(const octo_problem* prob, const int64_t* layer_costs,
                          const int64_t* link, const void* candidates, int64_t n,
                          int64_t* out_makespan, int64_t* out_bubble, int64_t* out_bounds,
                          void* stream) {
  Extra ex;
  ex.bound = out_bounds;
  return sim_batch_impl<XB>(prob, layer_costs, nullptr, link, candidates, n, out_makespan,
                            out_bubble, ex, static_cast<hipStream_t>(stream));
}

int octo_sim_batch_comm(const octo_problem* prob, const int64_t* layer_costs,
                        const int64_t* link, const void* candidates, int64_t n,
                        int64_t* out_makespan, int64_t* out_bubble, int64_t* out_comm,
                        void* stream) {
  Extra ex;
  ex.comm = out_comm;
  return sim_batch_impl<XC>(prob, layer_costs, nullptr, link, candidates, n, out_makespan,
                            out_bubble, ex, static_cast<hipStream_t>(stream));
}

int octo_advance_w(const octo_problem* prob, const int64_t* layer_costs, const int64_t* layer_mem,
                   const int64_t* capacity, const int64_t* link, const void* candidates,
                   int64_t n, void* out_candidates, int64_t* out_makespan, int64_t* out_bubble,
                   int64_t* out_peak, void* stream_) {
  int rc = check_problem(prob);
  if (rc) return rc;
  if (n < 0 || n > (int64_t)INT32_MAX) return OCTO_EINVAL;
  if (n == 0) return OCTO_OK;
  if (!layer_costs || !layer_mem || !capacity || !link || !candidates || !out_candidates ||
      !out_makespan || !out_bubble || !out_peak)
    return OCTO_EINVAL;
  if ((reinterpret_cast<uintptr_t>(candidates) & 15) != 0 ||
      (reinterpret_cast<uintptr_t>(out_candidates) & 15) != 0)
    return OCTO_EINVAL;
  hipStream_t stream = static_cast<hipStream_t>(stream_);
  std::lock_guard<std::mutex> lock(g_mu);
  // ring pass first (its queue rows need grid * CPW group slots of the workspace), then the
  // 64-bit pass over the candidates it left
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess) return OCTO_EHIP;
  DevInfo di;
  if ((rc = dev_info(dev, &di))) return rc;
  Plan rp;
  int rgrid = 0;
  rc = prob->v_max <= 2 ? advance_ring_grid<2>(prob, di, n, &rp, &rgrid)
                        : advance_ring_grid<8>(prob, di, n, &rp, &rgrid);
  if (rc) return rc;
  Setup su;
  rc = prepare(prob, layer_costs, layer_mem, stream, n, &su, (int64_t)rgrid * rp.CPW);
  if (rc) return rc;
  SimArgs a = make_args(prob, su.big, su, link, candidates, n, out_makespan, out_bubble, out_peak);
  uint8_t* out = static_cast<uint8_t*>(out_candidates);
  const int32_t* list = nullptr;
  const int32_t* list_n = nullptr;
  if (rgrid > 0) {
    SimArgs ar = make_args(prob, rp, su, link, candidates, n, out_makespan, out_bubble, out_peak);
    ar.ring = make_ring(prob->M, prob->P * prob->v_max).R;
    rc = prob->v_max <= 2
             ? launch_advance<2, true>(ar, rp, di.cus, rgrid, capacity, out, nullptr, nullptr,
                                       stream)
             : launch_advance<8, true>(ar, rp, di.cus, rgrid, capacity, out, nullptr, nullptr,
                                       stream);
    if (rc) return rc;
    list = a.redo;
    list_n = a.ctl + CTL_REDO;
  }
  return prob->v_max <= 2 ? launch_advance<2, false>(a, su.big, su.di.cus, su.mat_grid, capacity,
                                                     out, list, list_n, stream)
                          : launch_advance<8, false>(a, su.big, su.di.cus, su.mat_grid, capacity,
                                                     out, list, list_n, stream);
}

int octo_tune_step(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                   void* chains, uint16_t* queues, int64_t n_chains, uint64_t seed, int32_t step,
                   void* stream) {
  return tune_step_impl<false>(prob, layer_costs, nullptr, nullptr, 0, link, chains, queues,
                               n_chains, seed, step, static_cast<hipStream_t>(stream));
}

int octo_tune_step_mem(const octo_problem* prob, const int64_t* layer_costs,
                       const int64_t* layer_mem, const int64_t* capacity, int32_t max_advance,
                       const int64_t* link, void* chains, uint16_t* queues, int64_t n_chains,
                       uint64_t seed, int32_t step, void* stream) {
  return tune_step_impl<true>(prob, layer_costs, layer_mem, capacity, max_advance, link, chains,
                              queues, n_chains, seed, step, static_cast<hipStream_t>(stream));
}

int octo_alg1_tune(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                   void* records, int64_t n, int32_t iters, int64_t* out_makespan,
                   int64_t* out_bubble, int64_t* out_stats, void* stream) {
  return alg1_impl(prob, layer_costs, link, records, n, iters, A1F_INSERT, 0, out_makespan,
                   out_bubble, out_stats, nullptr, static_cast<hipStream_t>(stream));
}

int octo_alg1_tune_ex(const octo_problem* prob, const int64_t* layer_costs, const int64_t* link,
                      void* records, int64_t n, int32_t iters, int32_t flags, uint64_t seed,
                      int64_t* out_makespan, int64_t* out_bubble, int64_t* out_stats,
                      int64_t* out_phase_iters, void* stream) {
  return alg1_impl(prob, layer_costs, link, records, n, iters, flags, seed, out_makespan,
                   out_bubble, out_stats, out_phase_iters, static_cast<hipStream_t>(stream));
}

int octo_profile_events(void* const* events, int32_t n_events) {
  std::lock_guard<std::mutex> lock(g_mu);
  if (n_events < 0 || n_events > 8 || (n_events > 0 && !events)) return OCTO_EINVAL;
  for (int i = 0; i < 8; ++i) g_prof[i] = i < n_events ? static_cast<hipEvent_t>(events[i]) : nullptr;
  g_prof_n = n_events;
  return OCTO_OK;
}

const char* octo_strerror(int status) {
  switch (status) {
    case OCTO_OK: return "ok";
    case OCTO_EINVAL: return "invalid argument";
    case OCTO_EUNSUPPORTED: return "problem exceeds this GPU's limits (LDS per workgroup)";
    case OCTO_EHIP: return "HIP runtime error";
    case OCTO_ENOMEM: return "workspace allocation failed";
    case OCTO_ESCRATCH:
      return "the batch needs more device memory than the static scratch array of "
             "octo_sim_batch_noalloc holds (OCTO_NOALLOC_SCRATCH_BYTES)";
    default: return "unknown status";
  }
}

}  // extern "C"
