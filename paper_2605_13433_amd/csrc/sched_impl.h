// Device body of the seq_offsets tile scheduler, shared by the standalone
// scheduler launch and by the LayerNorm-backward launch, whose extra
// work-group builds the backward's lists while the other work-groups
// normalise (one launch fewer per backward call).
//
// The paper balances jagged work by sorting samples by cost and assigning
// them greedily (Sec. 4.1.3, "Global Token Reallocation"), and balances
// work across the compute elements of one device (Sec. 4.1.1, "Load
// balancing across device computing elements").  On
// one GPU the same idea becomes a longest-first work list consumed by
// persistent work-groups through an atomic pop counter (every entry expands
// to H adjacent items, one per head):
//
//   * q-list: entries (b, qt) for every 64-row query tile, cost qt+1 k-tiles
//     (causal: only kt <= qt is visited).  Consumed by the forward kernels
//     and the dQ kernels.
//   * k-list: entries (b, kt), cost ntiles_b - kt q-tiles.  Consumed by the
//     dK/dV kernels.
//   * pair list (forward calls on deep batches): entries (b, p) for every
//     pair of query tiles 2p, 2p+1 (the second past the sequence when
//     ntiles_b is odd), cost ~ p+1; consumed by the bf16 forward's two-tile
//     items.
//   * combined backward list: both kinds, dK/dV entries before dQ entries of
//     equal cost (dQ entries flagged), consumed by the combined bf16
//     backward kernel.  With `fuse_dq0` set, no sequence gets a dQ entry for
//     its first q-tile (the dK/dV item of its first k-tile computes it); in
//     cost-major order those entries would be the list's last ones, in
//     sequence-major order the last one of each sequence's run, so the
//     list is one entry per sequence shorter.
//
// Two orders, chosen on the device per call:
//   * cost-major: entries sorted by cost, longest first -- the makespan
//     bound of longest-processing-time-first when the work per work-group
//     is not far above the longest item;
//   * sequence-major: sequence by sequence, longest sequence first, each
//     sequence's entries longest first -- when the work per work-group is
//     many times the longest item, so that balance is easy, the items that
//     run at the same time stay on a few sequences, whose K/V (or Q/dO)
//     rows they share through the caches.
//
// Built on the device from seq_offsets (no host round trip) by one
// work-group: a histogram of tile counts, a rank per sequence (tile count
// descending, ties in arbitrary order), then a scatter in which every entry's
// slot follows from its sequence's rank.  No result depends on the order of
// ties except the summation order of the table gradients.
#pragma once

#include "internal.h"

namespace hstu {

constexpr int SCHED_MAX_BINS = 65536 / TILE + 2;   // max_len <= 65536

// The sequence-major order needs this many times the longest item's cost of
// work per work-group (in 64 x 64 tile pairs).
constexpr int SCHED_SEQ_MAJOR_SLACK = 4;

struct SchedSmem {
  int32_t count[SCHED_MAX_BINS];      // # sequences with ntiles == n
  int32_t rank0[SCHED_MAX_BINS];      // first rank of tile-count bin n (# with ntiles > n)
  int32_t fill[SCHED_MAX_BINS];       // sequences ranked in bin n so far
  int32_t cstart[SCHED_MAX_BINS];     // cost-major: first entry of cost bin c
  int32_t sstart[SCHED_MAX_BINS];     // sequence-major: first entry of bin n's sequences
  int32_t cstart_p[SCHED_MAX_BINS / 2 + 1];   // pair list, cost-major: first entry of bin c
  int32_t sstart_p[SCHED_MAX_BINS];           // pair list, sequence-major: bin n's first
  int32_t total;
  int32_t seq_major;
  int32_t status;                     // HSTU_SEQ_* bits found by the contract check
};

struct SchedArgs {
  const int64_t *off;
  int32_t B, N;
  int64_t T;
  int32_t *ctrl;
  SeqInfo *info;
  WorkEntry *list_q, *list_k, *list_b, *list_p;
  int32_t nbins, cap, cap_p;
  int32_t H;
  int32_t grid_hint;                  // nominal persistent work-groups
  int32_t fuse_dq0;                   // no dQ entries for first q-tiles
  int32_t check;                      // check the seq_offsets contract
  float *zero_out;
  int32_t n_zero;
};

// Runs in one work-group of NT threads.
template <int NT>
__device__ __forceinline__ void build_schedule(const SchedArgs &a, SchedSmem &sm, int tid) {
  for (int x = tid; x < a.n_zero; x += NT) a.zero_out[x] = 0.0f;
  for (int c = tid; c < a.nbins; c += NT) {
    sm.count[c] = 0;
    sm.fill[c] = 0;
  }
  if (tid == 0) {
    sm.total = 0;
    sm.status = 0;
  }
  __syncthreads();

  // Clamp every sequence into [0, N] rows and into [0, T): a violating
  // offsets array must never make a kernel read outside its buffers.  With
  // the contract check on, each violation sets its bit of the status word.
  for (int b = tid; b < a.B; b += NT) {
    int64_t s = a.off[b], e = a.off[b + 1];
    if (a.check) {
      int bad = 0;
      if (b == 0 && s != 0) bad |= HSTU_SEQ_FIRST_NOT_ZERO;
      if (e < s) bad |= HSTU_SEQ_DECREASING;
      else if (e - s > a.N) bad |= HSTU_SEQ_TOO_LONG;
      if (b == a.B - 1 && e != a.T) bad |= HSTU_SEQ_LAST_NOT_T;
      if (bad) atomicOr(&sm.status, bad);
    }
    s = s < 0 ? 0 : (s > a.T ? a.T : s);
    e = e < s ? s : (e > a.T ? a.T : e);
    int64_t L = e - s;
    if (L > a.N) L = a.N;
    const int nt = (int)((L + TILE - 1) / TILE);
    a.info[b].start = s;
    a.info[b].len = (int32_t)L;
    a.info[b].ntiles = nt;
    if (nt > 0) {
      atomicAdd(&sm.count[nt], 1);
      atomicAdd(&sm.total, nt);
    }
  }
  __syncthreads();

  // Ranks, bin starts of both orders, and the choice of order.  Serial over
  // at most 1026 bins.
  if (tid == 0) {
    int32_t ranks = 0, seq_run = 0, ge = 0, cost_run = 0, nt_max = 0;
    int64_t work = 0;                              // causal tile pairs per head
    for (int n = a.nbins - 1; n >= 1; --n) {
      const int32_t c = sm.count[n];
      if (c > 0 && nt_max == 0) nt_max = n;
      sm.rank0[n] = ranks;
      ranks += c;
      sm.sstart[n] = seq_run;                      // sequences of n tiles, n entries each
      seq_run += n * c;
      ge += c;                                     // sequences with ntiles >= n
      sm.cstart[n] = cost_run;                     // cost bin n: one entry per such sequence
      cost_run += ge;
      work += (int64_t)c * n * (n + 1) / 2;
    }
    sm.seq_major = work * a.H >= (int64_t)SCHED_SEQ_MAJOR_SLACK * nt_max * a.grid_hint;
    // pair list: a sequence of n tiles has (n+1)/2 pair entries; cost bin c
    // (pair index c-1) holds one entry per sequence with n >= 2c-1, i.e. the
    // ranks below rank0[2c-1] + count[2c-1]
    int32_t run_p = 0, ge_p = 0, cost_p = 0;
    for (int n = a.nbins - 1; n >= 1; --n) {
      sm.sstart_p[n] = run_p;
      run_p += sm.count[n] * ((n + 1) / 2);
    }
    for (int c = a.nbins / 2; c >= 1; --c) {
      ge_p += sm.count[2 * c - 1] + (2 * c < a.nbins ? sm.count[2 * c] : 0);
      sm.cstart_p[c] = cost_p;
      cost_p += ge_p;
    }
    a.ctrl[CTRL_N_PAIRS] = a.list_p ? (run_p < a.cap_p ? run_p : a.cap_p) : 0;
    // Valid offsets never exceed the list capacity; overlapping (invalid)
    // ones can, and then only the first `cap` slots are kept -- every slot
    // below the total is filled exactly once, so the kept prefix is dense.
    a.ctrl[CTRL_N_ENTRIES] = sm.total < a.cap ? sm.total : a.cap;
    a.ctrl[CTRL_STATUS] = a.check ? sm.status : HSTU_SEQ_UNCHECKED;
    a.ctrl[CTRL_POP_FWD] = 0;
    a.ctrl[CTRL_POP_DQ] = 0;
    a.ctrl[CTRL_POP_DKV] = 0;
    a.ctrl[CTRL_POP_BWD] = 0;
    // every non-empty sequence (sm.rank0[1] + sm.count[1] of them) has one
    // first q-tile
    const int32_t n_bwd = 2 * sm.total - (a.fuse_dq0 ? sm.rank0[1] + sm.count[1] : 0);
    a.ctrl[CTRL_N_BWD] = n_bwd < 2 * a.cap ? n_bwd : 2 * a.cap;
    // a violated contract: the attention kernels find empty lists and skip
    if (sm.status != 0) {
      a.ctrl[CTRL_N_ENTRIES] = 0;
      a.ctrl[CTRL_N_BWD] = 0;
      a.ctrl[CTRL_N_PAIRS] = 0;
    }
  }
  __syncthreads();

  const bool seq_major = sm.seq_major != 0;
  for (int b = tid; b < a.B; b += NT) {
    const SeqInfo si = a.info[b];
    const int nt = si.ntiles;
    if (nt == 0) continue;
    const int r = sm.rank0[nt] + atomicAdd(&sm.fill[nt], 1);   // rank, by tile count
    // sequence-major: this sequence's first entry
    const int base = sm.sstart[nt] + (r - sm.rank0[nt]) * nt;
    if (a.list_p) {
      const int np = (nt + 1) / 2;
      const int base_p = sm.sstart_p[nt] + (r - sm.rank0[nt]) * np;
      for (int t = 0; t < np; ++t) {
        const int sp = seq_major ? base_p + (np - 1 - t) : sm.cstart_p[t + 1] + r;
        if (sp < a.cap_p) a.list_p[sp] = WorkEntry{b, t, si.len, 0, si.start};
      }
    }
    for (int t = 0; t < nt; ++t) {
      const WorkEntry we{b, t, si.len, 0, si.start};
      const int cq = t + 1;          // q-tile t visits k-tiles 0..t
      const int ck = nt - t;         // k-tile t is visited by q-tiles t..nt-1
      // cost-major: cost bin c holds one entry per sequence with ntiles >= c,
      // i.e. per rank below rank0[c] + count[c], in rank order
      const int sq = seq_major ? base + (nt - 1 - t) : sm.cstart[cq] + r;
      const int sk = seq_major ? base + t : sm.cstart[ck] + r;
      if (sq < a.cap) a.list_q[sq] = we;
      if (a.list_k && sk < a.cap) a.list_k[sk] = we;
      if (a.list_b) {
        // combined list: cost-major, bin c spans 2 ge(c) slots, its dK/dV
        // entries then its dQ entries; sequence-major, per sequence the
        // dK/dV then the dQ entry of each cost, from nt down to 1
        WorkEntry wq = we;
        wq.tile |= BWD_DQ_FLAG;
        // sequence-major with fuse_dq0: each earlier sequence's run is one
        // entry shorter (its first q-tile's dQ entry, the run's last, is gone)
        const int run0 = 2 * base - (a.fuse_dq0 ? r : 0);
        const int bk = seq_major ? run0 + 2 * t : 2 * sm.cstart[ck] + r;
        const int bq = seq_major ? run0 + 2 * (nt - 1 - t) + 1
                                 : 2 * sm.cstart[cq] + sm.rank0[cq] + sm.count[cq] + r;
        if (bk < 2 * a.cap) a.list_b[bk] = we;
        if (!(a.fuse_dq0 && t == 0) && bq < 2 * a.cap) a.list_b[bq] = wq;
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
  a.list_p = L.list_p ? (WorkEntry *)(base + L.list_p) : nullptr;
  a.nbins = (int)((p.N + TILE - 1) / TILE) + 2;
  a.cap = (int32_t)p.max_entries;
  a.cap_p = (int32_t)pair_entries(p);
  a.H = p.H;
  a.grid_hint = 4 * L.num_cu;
  a.fuse_dq0 = L.list_b && L.bwd_combined && p.d == 64 ? 1 : 0;
  a.check = p.check_offsets ? 1 : 0;
  a.zero_out = L.dtime_part ? (float *)(base + L.dtime_part) : nullptr;
  // 8 bytes per partial entry (see make_layout): DTIME_BINS histograms for
  // the bf16 backward, one table for the fp32 one
  a.n_zero = L.dtime_part ? 2 * (p.dtype == HSTU_BF16 ? DTIME_BINS : 1) * p.H * p.nb : 0;
  return a;
}

}  // namespace hstu
