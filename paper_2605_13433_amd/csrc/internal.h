// Host-side internals of the jagged HSTU attention library: the workspace
// layout and the kernel launchers each .hip file provides.
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

#include "../../include/hstu_jagged.h"

namespace hstu {

// Tile edge (queries per q-tile and keys per k-tile) of every kernel and of
// the work lists the scheduler builds.
constexpr int TILE = 64;

// The dK/dV work-groups fold their d_time histograms into this many partial
// tables (work-group index mod DTIME_BINS) with float atomics; the finalize
// kernel sums the bins in a fixed order.
constexpr int DTIME_BINS = 16;

// Control block at the head of every workspace (int32 words).
enum CtrlSlot {
  CTRL_N_ENTRIES = 0,   // (sequence, tile) entries in each work list
  CTRL_POP_FWD = 1,     // pop counter of the attention forward kernel
  CTRL_POP_DQ = 2,      // pop counter of the dQ kernel
  CTRL_POP_DKV = 3,     // pop counter of the dK/dV kernel
  CTRL_WORDS = 64
};

// Per-sequence record the scheduler writes: clamped start row and length.
struct SeqInfo {
  int64_t start;
  int32_t len;
  int32_t ntiles;
};

// One work-list entry: a sequence and a 64-row tile index inside it.  The
// heads of an entry are expanded by the consumer (item = entry * H + h).
struct WorkEntry {
  int32_t seq;
  int32_t tile;
};

struct Problem {
  int32_t B, N, H, d;
  int64_t T;
  hstu_dtype dtype;
  bool has_pos, has_time;
  int32_t nb;
  int64_t max_entries;   // upper bound on sum_b ceil(L_b / 64)
};

// Workspace carve-up; offsets in bytes from the workspace base, each region
// 256-byte aligned.  Regions with size 0 are absent.
struct Layout {
  size_t ctrl, seqinfo, list_q, list_k, dO, dpos_part, dtime_part, total;
  int dkv_grid;          // persistent grid of the dK/dV kernel (WG count)
};

// Device properties the launch shapes depend on (cached per device).
struct DeviceInfo {
  int num_cu;
};
const DeviceInfo &device_info(int dev);

Layout make_layout(const Problem &p, bool for_bwd, int dev);

// ---- launchers (each returns hipSuccess or the launch error) ----
// Builds the work lists (and zeroes the d_time bins when the layout has
// them, so the backward's later kernels can accumulate into them).
hipError_t launch_schedule(const int64_t *seq_offsets, const Problem &p,
                           void *ws, const Layout &L, hipStream_t s);

struct AttnArgs {
  const void *q, *k, *v, *u;
  const float *pos_w, *time_w;
  const int64_t *ts;
  void *ws;
  Layout L;
  Problem p;
};

hipError_t launch_attn_fwd_bf16(const AttnArgs &a, void *o, hipStream_t s);
hipError_t launch_attn_dq_bf16(const AttnArgs &a, const void *dO, void *dq,
                               hipStream_t s);
hipError_t launch_attn_dkv_bf16(const AttnArgs &a, const void *dO, void *dk,
                                void *dv, hipStream_t s);

hipError_t launch_attn_fwd_f32(const AttnArgs &a, void *o, hipStream_t s);
hipError_t launch_attn_bwd_f32(const AttnArgs &a, const void *dO, void *dq,
                               void *dk, void *dv, float *d_pos,
                               float *d_time, hipStream_t s);

hipError_t launch_ln_fwd(const Problem &p, const void *o, const void *u,
                         void *y, float *mean, float *rstd, hipStream_t s);
hipError_t launch_ln_bwd(const Problem &p, const void *dy, const void *u,
                         const void *o, const float *mean, const float *rstd,
                         void *du, void *dO, float *dpos_part, hipStream_t s);
hipError_t launch_finalize_tables(const AttnArgs &a, float *d_pos,
                                  float *d_time, hipStream_t s);

// Persistent-grid sizes (work-groups) of the bf16 attention kernels.
int attn_fwd_grid(const Problem &p, int dev);
int attn_dq_grid(const Problem &p, int dev);
int attn_dkv_grid(const Problem &p, int dev);

}  // namespace hstu
