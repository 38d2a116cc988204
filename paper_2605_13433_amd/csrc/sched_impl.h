// Device body of the seq_offsets tile scheduler, shared by the standalone
// scheduler launch and by the LayerNorm-backward launch, whose extra
// work-group builds the backward's lists while the other work-groups
// normalise (one launch fewer per backward call).
//
// The paper balances jagged work by sorting samples by cost and assigning
// them greedily (Sec. 3.1.3, "Global Token Reallocation"), and balances
// work across the compute elements of one device (Sec. 3.1.1, step 3).  On
// one GPU the same idea becomes a longest-processing-time-first work list
// consumed by persistent work-groups through an atomic pop counter:
//
//   * q-list: entries (b, qt) for every 64-row query tile of every sequence,
//     cost qt+1 k-tiles (causal: only kt <= qt is visited), sorted by cost
//     descending.  Consumed by the forward kernels and the dQ kernels.
//   * k-list: entries (b, kt), cost ntiles_b - kt q-tiles, same order rule.
//     Consumed by the dK/dV kernels.
//   * combined backward list: both kinds merged bin by bin (dQ entries
//     flagged), consumed by the combined bf16 backward kernel.
//
// Built on the device from seq_offsets (no host round trip) by one
// work-group: a histogram of tile counts, a descending exclusive scan of the
// cost bins, then a scatter in which each entry takes the next slot of its
// bin.  Order inside a bin is arbitrary; no result depends on it except the
// summation order of the table gradients.
#pragma once

#include "internal.h"

namespace hstu {

constexpr int SCHED_MAX_BINS = 65536 / TILE + 2;   // max_len <= 65536

struct SchedSmem {
  int32_t count_ge[SCHED_MAX_BINS];   // # sequences with ntiles == c
  int32_t start[SCHED_MAX_BINS];      // first slot of cost bin c
  int32_t fill_q[SCHED_MAX_BINS];
  int32_t fill_k[SCHED_MAX_BINS];
  int32_t ge[SCHED_MAX_BINS];         // # sequences with ntiles >= c
  int32_t total;
};

struct SchedArgs {
  const int64_t *off;
  int32_t B, N;
  int64_t T;
  int32_t *ctrl;
  SeqInfo *info;
  WorkEntry *list_q, *list_k, *list_b;
  int32_t nbins, cap;
  float *zero_out;
  int32_t n_zero;
};

// Runs in one work-group of NT threads.
template <int NT>
__device__ __forceinline__ void build_schedule(const SchedArgs &a, SchedSmem &sm, int tid) {
  for (int x = tid; x < a.n_zero; x += NT) a.zero_out[x] = 0.0f;
  for (int c = tid; c < a.nbins; c += NT) {
    sm.count_ge[c] = 0;
    sm.fill_q[c] = 0;
    sm.fill_k[c] = 0;
  }
  if (tid == 0) sm.total = 0;
  __syncthreads();

  // Clamp every sequence into [0, N] rows and into [0, T): a violating
  // offsets array must never make a kernel read outside its buffers.
  for (int b = tid; b < a.B; b += NT) {
    int64_t s = a.off[b], e = a.off[b + 1];
    s = s < 0 ? 0 : (s > a.T ? a.T : s);
    e = e < s ? s : (e > a.T ? a.T : e);
    int64_t L = e - s;
    if (L > a.N) L = a.N;
    const int nt = (int)((L + TILE - 1) / TILE);
    a.info[b].start = s;
    a.info[b].len = (int32_t)L;
    a.info[b].ntiles = nt;
    if (nt > 0) {
      atomicAdd(&sm.count_ge[nt], 1);
      atomicAdd(&sm.total, nt);
    }
  }
  __syncthreads();

  // Bin c (cost c) holds one entry per sequence with ntiles >= c; bins are
  // laid out from the most expensive down.  Serial over at most 1026 bins.
  if (tid == 0) {
    int32_t run = 0, ge = 0;
    for (int c = a.nbins - 1; c >= 1; --c) {
      ge += sm.count_ge[c];        // sequences with ntiles >= c
      sm.start[c] = run;
      sm.ge[c] = ge;
      run += ge;
    }
    // Valid offsets never exceed the list capacity; overlapping (invalid)
    // ones can, and then only the first `cap` slots are kept -- every slot
    // below the total is filled exactly once, so the kept prefix is dense.
    a.ctrl[CTRL_N_ENTRIES] = sm.total < a.cap ? sm.total : a.cap;
    a.ctrl[CTRL_POP_FWD] = 0;
    a.ctrl[CTRL_POP_DQ] = 0;
    a.ctrl[CTRL_POP_DKV] = 0;
    a.ctrl[CTRL_POP_BWD] = 0;
  }
  __syncthreads();

  for (int b = tid; b < a.B; b += NT) {
    const SeqInfo si = a.info[b];
    const int nt = si.ntiles;
    for (int t = 0; t < nt; ++t) {
      const WorkEntry we{b, t, si.len, 0, si.start};
      WorkEntry wq = we;
      wq.tile |= BWD_DQ_FLAG;
      const int cq = t + 1;          // q-tile t visits k-tiles 0..t
      const int ck = nt - t;         // k-tile t is visited by q-tiles t..nt-1
      const int sq = sm.start[cq] + atomicAdd(&sm.fill_q[cq], 1);
      const int sk = sm.start[ck] + atomicAdd(&sm.fill_k[ck], 1);
      if (sq < a.cap) a.list_q[sq] = we;
      if (a.list_k && sk < a.cap) a.list_k[sk] = we;
      if (a.list_b) {
        // combined backward list: bin c spans 2 ge[c] slots from 2 start[c],
        // dK/dV entries first (the heavier item of equal cost), then dQ ones
        const int bk = sk + sm.start[ck];
        const int bq = sq + sm.start[cq] + sm.ge[cq];
        if (bk < 2 * a.cap) a.list_b[bk] = we;
        if (bq < 2 * a.cap) a.list_b[bq] = wq;
      }
    }
  }
}

inline SchedArgs sched_args(const int64_t *seq_offsets, const Problem &p, void *ws,
                            const Layout &L) {
  char *base = (char *)ws;
  SchedArgs a;
  a.off = seq_offsets;
  a.B = p.B;
  a.N = p.N;
  a.T = p.T;
  a.ctrl = (int32_t *)(base + L.ctrl);
  a.info = (SeqInfo *)(base + L.seqinfo);
  a.list_q = (WorkEntry *)(base + L.list_q);
  a.list_k = L.list_k ? (WorkEntry *)(base + L.list_k) : nullptr;
  a.list_b = L.list_b ? (WorkEntry *)(base + L.list_b) : nullptr;
  a.nbins = (int)((p.N + TILE - 1) / TILE) + 2;
  a.cap = (int32_t)p.max_entries;
  a.zero_out = L.dtime_part ? (float *)(base + L.dtime_part) : nullptr;
  a.n_zero = L.dtime_part ? DTIME_BINS * p.H * p.nb : 0;
  return a;
}

}  // namespace hstu
