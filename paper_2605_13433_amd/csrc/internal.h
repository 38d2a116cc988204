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

// Fixed-point unit of the deterministic backward's table-gradient partials:
// a partial sum x of N log2(e) dS is kept as the 64-bit integer
// round(x * FIX_ONE) (resolution 2^-32, |x| < 2^31).
constexpr double FIX_ONE = 4294967296.0;

// The bf16 backward's table-gradient partials hold N log2(e) dS (the dK/dV
// items carry A and dS in base-2 units); the finalize pass multiplies by
// TABLE_UNIT / N.
constexpr double TABLE_UNIT = 0.693147180559945309;   // ln 2 = 1 / log2(e)

// The bf16 d=64 forward takes items of two query tiles (sharing every
// streamed K/V tile) when the batch's mean sequence length is at least this
// (at d=128 the two-tile items, one eight-wave work-group per CU, measured
// slower).
constexpr int64_t FWD_PAIR_MIN_AVG_LEN = 256;

// The backward runs as one combined launch while the work list holds fewer
// than this many (entry, head) items per persistent work-group.
constexpr int BWD_COMBINED_ITEMS_PER_WG = 4;

// Control block at the head of every workspace (int32 words).
enum CtrlSlot {
  CTRL_N_ENTRIES = 0,   // (sequence, tile) entries in each work list
  CTRL_POP_FWD = 1,     // pop counter of the attention forward kernel
  CTRL_POP_DQ = 2,      // pop counter of the dQ kernel
  CTRL_POP_DKV = 3,     // pop counter of the dK/dV kernel (and fp32 pass)
  CTRL_POP_BWD = 4,     // pop counter of the combined bf16 backward kernel
  CTRL_N_BWD = 5,       // entries in the combined backward list
  CTRL_STATUS = 6,      // seq_offsets contract status (HSTU_SEQ_* word)
  CTRL_N_PAIRS = 7,     // (sequence, query-tile pair) entries in the pair list
  CTRL_WORDS = 64
};

// Per-sequence record the scheduler writes: clamped start row and length.
struct SeqInfo {
  int64_t start;
  int32_t len;
  int32_t ntiles;
};

// One work-list entry: a sequence and a 64-row tile index inside it, with
// the sequence's clamped start row and length copied in, so that a consumer
// needs one load per entry.  The heads of an entry are expanded by the
// consumer (item = entry * H + h).
struct WorkEntry {
  int32_t seq;
  int32_t tile;
  int32_t len;
  int32_t reserved;
  int64_t start;
};

// In the combined backward list, dQ entries carry this bit in `tile`
// (dK/dV entries do not).
constexpr int32_t BWD_DQ_FLAG = 1 << 30;

struct Problem {
  int32_t B, N, H, d;
  int64_t T;
  hstu_dtype dtype;
  bool has_pos, has_time;
  int32_t nb;
  int64_t max_entries;   // upper bound on sum_b ceil(L_b / 64)
  bool check_offsets;    // HSTU_VALIDATE=1: the scheduler checks the contract
  float alpha;           // scale of <q, k> (1 = plain operator)
  bool deterministic;    // backward: fixed-point table accumulation
};

// Workspace carve-up; offsets in bytes from the workspace base, each region
// 256-byte aligned.  Regions with size 0 are absent.
struct Layout {
  size_t ctrl, seqinfo, list_q, list_k, list_b, list_p, dO, dpos_part, dtime_part, total;
  // persistent grids of the bf16 backward kernels (combined, dQ, dK/dV) and
  // whether the combined one runs (small problems) or the other two
  int bwd_grid_both, bwd_grid_dq, bwd_grid_dkv;
  bool bwd_combined;
  int num_cu;                         // compute units of the device
};

// ---- host helpers shared by the C-ABI translation units ----
// Records a formatted message as the thread's last error; returns `code`.
int fail(int code, const char *fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_last_error();
int hip_fail(hipError_t e, const char *what);
int current_device(int *dev);
// Validates every host-visible argument of an attention call; fills `p`.
int validate(const void *q, const void *k, const void *v, const void *u,
             const int64_t *off, int32_t B, int32_t N, int32_t H, int32_t d,
             const hstu_rab *rab, hstu_dtype dtype, int64_t T, Problem *p);
// Workspace pointer non-null, 256-byte aligned and at least `need` bytes.
int check_workspace_bytes(size_t need, void *ws, size_t bytes);

constexpr size_t kAlign = 256;
inline size_t align_up(size_t x) { return (x + kAlign - 1) / kAlign * kAlign; }

// Optional per-kernel timing (hstu_profile_enable): a Scope brackets one
// launch with two HIP events recorded on the launch stream.
namespace prof {
struct Scope {
  const char *name;
  hipStream_t s;
  hipEvent_t a = nullptr;
  Scope(const char *n, hipStream_t st);
  ~Scope();
};
}  // namespace prof

// Device properties the launch shapes depend on (cached per device).
struct DeviceInfo {
  int num_cu;
};
const DeviceInfo &device_info(int dev);

Layout make_layout(const Problem &p, bool for_bwd, int dev);

// A fixed device buffer that stands in for the caller's workspace: addr(dev)
// returns its address on device `dev` (or nullptr after recording the
// error), `bytes` its size.
struct FixedScratch {
  void *(*addr)(int dev);
  size_t bytes;
};

// The attention forward (schedule, attention, LayerNorm x U) on the
// caller's workspace (out->workspace), or, with `fixed`, on that buffer.
int attn_fwd_call(const void *q, const void *k, const void *v, const void *u,
                  const int64_t *seq_offsets, int32_t B, int32_t max_len, int32_t H,
                  int32_t d, const hstu_rab *rab, hstu_fwd_out *out, void *stream,
                  const FixedScratch *fixed);


// Form of the bf16 backward's dq, dk, dv, du outputs: rows of `stride`
// elements, and with h_* set, each gradient multiplied by silu' of the h_*
// element at the same index before its store (the HSTU layer writes
// dh = dz silu'(h) straight into its [T][4C] gradient this way).  Without a
// GradOut the outputs are plain [T][H*d].
struct GradOut {
  int32_t stride;
  const void *h_dq, *h_dk, *h_dv, *h_du;
};

// The attention backward (LayerNorm backward with the schedule, attention
// backward, table finalize); `go` (bf16 only) sets the outputs' form.
int attn_bwd_call(const void *q, const void *k, const void *v, const void *u,
                  const int64_t *seq_offsets, int32_t B, int32_t max_len, int32_t H,
                  int32_t d, const hstu_rab *rab, hstu_bwd_io *io, void *stream,
                  const GradOut *go);

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
// dQ, dK, dV and the table-gradient partials: one combined launch, or a
// dK/dV launch then a dQ launch (see Layout::bwd_combined).
hipError_t launch_attn_bwd_bf16(const AttnArgs &a, const void *dO, void *dq, void *dk,
                                void *dv, const GradOut *go, hipStream_t s);

hipError_t launch_attn_fwd_f32(const AttnArgs &a, void *o, hipStream_t s);
hipError_t launch_attn_bwd_f32(const AttnArgs &a, const void *dO, void *dq,
                               void *dk, void *dv, float *d_pos,
                               float *d_time, hipStream_t s);

hipError_t launch_ln_fwd(const Problem &p, const void *o, const void *u,
                         void *y, float *mean, float *rstd, hipStream_t s);
// LayerNorm backward with the scheduler's work-group appended: builds the
// backward's lists (as launch_schedule) in the same launch.
hipError_t launch_ln_bwd_sched(const Problem &p, const void *dy, const void *u,
                               const void *o, const float *mean, const float *rstd,
                               void *du, void *dO, void *dpos_part,
                               const int64_t *seq_offsets, void *ws, const Layout &L,
                               const GradOut *go, hipStream_t s);
hipError_t launch_finalize_tables(const AttnArgs &a, float *d_pos,
                                  float *d_time, hipStream_t s);

// HSTU layer shell pointwise passes; C = H*d (a multiple of 64).
// z planes [4][T][C] = silu(h [T][4C]) split by column blocks.
hipError_t launch_silu_split(const void *h, void *z, int64_t T, int32_t C,
                             int dev, hipStream_t s);
// Fused f1 of the layer (csrc/gemm.hip): h [M][N] = x [M][K] . w1 [K][N]
// (bf16, float32 accumulation) and z = silu(h) split into four [M][N/4]
// planes, in one hand-written MFMA kernel.  Supported when N is a multiple
// of 128, N/4 of 8 and K of 64.
bool gemm_f1_silu_supported(int64_t N, int64_t K);
hipError_t launch_gemm_f1_silu(const void *x, const void *w1, void *h, void *z, int64_t M,
                               int32_t N, int32_t K, hipStream_t s);
// Zero `bytes` (a multiple of 4) of device memory with a kernel.
// out (bf16, n elements, n % 4 == 0) = sum of `parts` float32 arrays of n
// elements stored back to back at `part`.
hipError_t launch_sum_parts(const float *part, void *out, int64_t n, int32_t parts, int dev,
                            hipStream_t s);
hipError_t launch_zero(void *p, size_t bytes, int dev, hipStream_t s);

// Whether the bf16 forward runs on the pair list (two query tiles per item),
// and that list's capacity: every pair but one per sequence covers two of
// the sum_b ceil(L_b / 64) <= max_entries tiles.
bool fwd_pairs(const Problem &p);
inline int64_t pair_entries(const Problem &p) { return (p.max_entries + p.B) / 2 + 1; }
// Persistent-grid sizes (work-groups) of the bf16 attention kernels.
int attn_fwd_grid(const Problem &p, int dev);
int attn_bwd_grid(const Problem &p, int dev);
int attn_bwd_dq_grid(const Problem &p, int dev);
int attn_bwd_dkv_grid(const Problem &p, int dev);

}  // namespace hstu
