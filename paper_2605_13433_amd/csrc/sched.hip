// seq_offsets-driven tile scheduler.
//
// The paper balances jagged work by sorting samples by cost and assigning
// them greedily (Sec. 3.1.3, "Global Token Reallocation"), and balances
// work across the compute elements of one device (Sec. 3.1.1, step 3).  On
// one GPU the same idea becomes a longest-processing-time-first work list
// consumed by persistent work-groups through an atomic pop counter:
//
//   * q-list: entries (b, qt) for every 64-row query tile of every sequence,
//     cost qt+1 k-tiles (causal: only kt <= qt is visited), sorted by cost
//     descending.  Consumed by the forward and the dQ kernels.
//   * k-list: entries (b, kt), cost ntiles_b - kt q-tiles, same order rule.
//     Consumed by the dK/dV kernel.
//
// Built on the device from seq_offsets (no host round trip) by one
// work-group: a histogram of tile counts, a descending exclusive scan of the
// cost bins, then a scatter in which each entry takes the next slot of its
// bin.  Order inside a bin is arbitrary; no result depends on it except the
// summation order of the table gradients.
#include "internal.h"
#include "device.h"

namespace hstu {

namespace {

constexpr int SCHED_THREADS = 1024;
constexpr int MAX_BINS = 65536 / TILE + 2;   // max_len <= 65536

__global__ void __launch_bounds__(SCHED_THREADS)
schedule_kernel(const int64_t *__restrict__ off, int32_t B, int32_t N,
                int64_t T, int32_t *__restrict__ ctrl,
                SeqInfo *__restrict__ info, WorkEntry *__restrict__ list_q,
                WorkEntry *__restrict__ list_k, int32_t nbins, int32_t cap,
                float *__restrict__ zero_out, int32_t n_zero) {
  __shared__ int32_t count_ge[MAX_BINS];   // # sequences with ntiles == c
  __shared__ int32_t start[MAX_BINS];      // first slot of cost bin c
  __shared__ int32_t fill_q[MAX_BINS];
  __shared__ int32_t fill_k[MAX_BINS];
  __shared__ int32_t total;
  const int tid = threadIdx.x;

  for (int x = tid; x < n_zero; x += SCHED_THREADS) zero_out[x] = 0.0f;
  for (int c = tid; c < nbins; c += SCHED_THREADS) {
    count_ge[c] = 0;
    fill_q[c] = 0;
    fill_k[c] = 0;
  }
  if (tid == 0) total = 0;
  __syncthreads();

  // Clamp every sequence into [0, N] rows and into [0, T): a violating
  // offsets array must never make a kernel read outside its buffers.
  for (int b = tid; b < B; b += SCHED_THREADS) {
    int64_t s = off[b], e = off[b + 1];
    s = s < 0 ? 0 : (s > T ? T : s);
    e = e < s ? s : (e > T ? T : e);
    int64_t L = e - s;
    if (L > N) L = N;
    const int nt = (int)((L + TILE - 1) / TILE);
    info[b].start = s;
    info[b].len = (int32_t)L;
    info[b].ntiles = nt;
    if (nt > 0) {
      atomicAdd(&count_ge[nt], 1);
      atomicAdd(&total, nt);
    }
  }
  __syncthreads();

  // Bin c (cost c) holds one entry per sequence with ntiles >= c; bins are
  // laid out from the most expensive down.  Serial over at most 1026 bins.
  if (tid == 0) {
    int32_t run = 0, ge = 0;
    for (int c = nbins - 1; c >= 1; --c) {
      ge += count_ge[c];        // sequences with ntiles >= c
      start[c] = run;
      run += ge;
    }
    // Valid offsets never exceed the list capacity; overlapping (invalid)
    // ones can, and then only the first `cap` slots are kept -- every slot
    // below the total is filled exactly once, so the kept prefix is dense.
    ctrl[CTRL_N_ENTRIES] = total < cap ? total : cap;
    ctrl[CTRL_POP_FWD] = 0;
    ctrl[CTRL_POP_DQ] = 0;
    ctrl[CTRL_POP_DKV] = 0;
  }
  __syncthreads();

  for (int b = tid; b < B; b += SCHED_THREADS) {
    const int nt = info[b].ntiles;
    for (int t = 0; t < nt; ++t) {
      const int cq = t + 1;          // q-tile t visits k-tiles 0..t
      const int ck = nt - t;         // k-tile t is visited by q-tiles t..nt-1
      const int sq = start[cq] + atomicAdd(&fill_q[cq], 1);
      const int sk = start[ck] + atomicAdd(&fill_k[ck], 1);
      if (sq < cap) list_q[sq] = WorkEntry{b, t};
      if (list_k && sk < cap) list_k[sk] = WorkEntry{b, t};
    }
  }
}

}  // namespace

hipError_t launch_schedule(const int64_t *seq_offsets, const Problem &p,
                           void *ws, const Layout &L, hipStream_t s) {
  char *base = (char *)ws;
  const int nbins = (int)((p.N + TILE - 1) / TILE) + 2;
  hipLaunchKernelGGL(schedule_kernel, dim3(1), dim3(SCHED_THREADS), 0, s,
                     seq_offsets, p.B, p.N, p.T, (int32_t *)(base + L.ctrl),
                     (SeqInfo *)(base + L.seqinfo),
                     (WorkEntry *)(base + L.list_q),
                     L.list_k ? (WorkEntry *)(base + L.list_k) : nullptr, nbins,
                     (int32_t)p.max_entries,
                     L.dtime_part ? (float *)(base + L.dtime_part) : nullptr,
                     L.dtime_part ? DTIME_BINS * p.H * p.nb : 0);
  return hipGetLastError();
}

}  // namespace hstu
