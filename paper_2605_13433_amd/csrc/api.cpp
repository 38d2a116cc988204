// C ABI of the jagged HSTU attention library: argument validation, workspace
// carving and the launch sequence of each call.  No call allocates device
// memory or synchronises; every kernel goes onto the caller's stream.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <cmath>
#include <cstdarg>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <mutex>
#include <string>
#include <vector>

#include "internal.h"

namespace hstu {

thread_local std::string g_last_error;

int fail(int code, const char *fmt, ...) {
  char buf[512];
  va_list ap;
  va_start(ap, fmt);
  vsnprintf(buf, sizeof buf, fmt, ap);
  va_end(ap);
  g_last_error = buf;
  return code;
}

void clear_last_error() { g_last_error.clear(); }

int hip_fail(hipError_t e, const char *what) {
  return fail(HSTU_EHIP, "%s: %s", what, hipGetErrorString(e));
}

namespace {
int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
}  // namespace

// Validates everything the host can see; on success fills `p`.
int validate(const void *q, const void *k, const void *v, const void *u,
             const int64_t *off, int32_t B, int32_t N, int32_t H, int32_t d,
             const hstu_rab *rab, hstu_dtype dtype, int64_t T, Problem *p) {
  if (dtype != HSTU_BF16 && dtype != HSTU_F32)
    return fail(HSTU_EINVAL, "dtype %d is not HSTU_BF16 or HSTU_F32", (int)dtype);
  if (B < 0) return fail(HSTU_EINVAL, "B = %d < 0", B);
  if (T < 0) return fail(HSTU_EINVAL, "total_tokens = %lld < 0", (long long)T);
  if (B == 0 && T != 0)
    return fail(HSTU_EINVAL, "B = 0 but total_tokens = %lld", (long long)T);
  if (N < 1) return fail(HSTU_EINVAL, "max_len = %d < 1", N);
  if (H < 1) return fail(HSTU_EINVAL, "H = %d < 1", H);
  if (d != 32 && d != 64 && d != 128)
    return fail(HSTU_EINVAL, "d = %d is not 32, 64 or 128", d);
  if (dtype == HSTU_BF16 && d == 32)
    return fail(HSTU_ENOTSUP, "bf16 path supports d = 64 or 128, got 32");
  if (N > 65536) return fail(HSTU_ENOTSUP, "max_len = %d > 65536", N);
  if (H > 64) return fail(HSTU_ENOTSUP, "H = %d > 64", H);
  if (!off) return fail(HSTU_EINVAL, "seq_offsets must be non-null");
  if (T > 0 && (!q || !k || !v || !u))
    return fail(HSTU_EINVAL, "q, k, v, u must be non-null when total_tokens > 0");
  const bool has_pos = rab && rab->pos_w;
  const bool has_time = rab && rab->time_w;
  int32_t nb = 0;
  if (has_time) {
    if (!rab->timestamps && T > 0)
      return fail(HSTU_EINVAL, "rab->time_w given without rab->timestamps");
    if (rab->num_buckets < 1)
      return fail(HSTU_EINVAL, "rab->num_buckets = %d < 1", rab->num_buckets);
    nb = rab->num_buckets;
    if (dtype == HSTU_BF16 && (int64_t)H * nb > 4096)
      return fail(HSTU_ENOTSUP, "H * num_buckets = %lld > 4096",
                  (long long)H * nb);
  }
  p->B = B; p->N = N; p->H = H; p->d = d; p->T = T; p->dtype = dtype;
  const char *chk = getenv("HSTU_VALIDATE");
  p->check_offsets = chk && chk[0] == '1';
  p->has_pos = has_pos; p->has_time = has_time; p->nb = nb;
  float alpha = rab ? rab->alpha : 0.0f;
  if (!std::isfinite(alpha)) return fail(HSTU_EINVAL, "rab->alpha is not finite");
  p->alpha = alpha == 0.0f ? 1.0f : alpha;
  p->deterministic = false;
  // sum_b ceil(L_b/64) <= min(B * ceil(N/64), floor((T + 63 B) / 64))
  p->max_entries = std::min<int64_t>((int64_t)B * ceil_div(N, TILE),
                                     (T + (int64_t)(TILE - 1) * B) / TILE);
  return HSTU_OK;
}

int check_workspace_bytes(size_t need, void *ws, size_t bytes) {
  if (!ws) return fail(HSTU_EWORKSPACE, "workspace is NULL (%zu bytes needed)", need);
  if ((uintptr_t)ws % kAlign)
    return fail(HSTU_EINVAL, "workspace is not %zu-byte aligned", kAlign);
  if (bytes < need)
    return fail(HSTU_EWORKSPACE, "workspace has %zu bytes, %zu needed", bytes, need);
  return HSTU_OK;
}

namespace {
int check_workspace(const Layout &L, void *ws, size_t bytes) {
  return check_workspace_bytes(L.total, ws, bytes);
}
}  // namespace

int current_device(int *dev) {
  hipError_t e = hipGetDevice(dev);
  if (e != hipSuccess) return hip_fail(e, "hipGetDevice");
  return HSTU_OK;
}

namespace prof {
namespace {
struct Rec {
  const char *name;
  hipEvent_t a, b;
};
std::atomic<bool> on{false};
std::mutex mu;
std::vector<Rec> recs;
std::vector<hipEvent_t> pool;

hipEvent_t take_event() {
  if (!pool.empty()) {
    hipEvent_t e = pool.back();
    pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  return hipEventCreate(&e) == hipSuccess ? e : nullptr;
}

}  // namespace

Scope::Scope(const char *n, hipStream_t st) : name(n), s(st) {
  if (!n || !on.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lock(mu);
  a = take_event();
  if (a && hipEventRecord(a, s) != hipSuccess) {
    pool.push_back(a);
    a = nullptr;
  }
}

Scope::~Scope() {
  if (!a) return;
  std::lock_guard<std::mutex> lock(mu);
  hipEvent_t b = take_event();
  if (b && hipEventRecord(b, s) == hipSuccess) {
    recs.push_back(Rec{name, a, b});
  } else {
    pool.push_back(a);
    if (b) pool.push_back(b);
  }
}
}  // namespace prof

const DeviceInfo &device_info(int dev) {
  static std::mutex mu;
  static std::vector<DeviceInfo> cache;
  static std::vector<bool> have;
  std::lock_guard<std::mutex> lock(mu);
  if ((int)cache.size() <= dev) {
    cache.resize(dev + 1);
    have.resize(dev + 1, false);
  }
  if (!have[dev]) {
    int cu = 0;
    if (hipDeviceGetAttribute(&cu, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess ||
        cu <= 0)
      cu = 256;
    cache[dev].num_cu = cu;
    have[dev] = true;
  }
  return cache[dev];
}

Layout make_layout(const Problem &p, bool for_bwd, int dev) {
  Layout L{};
  size_t at = 0;
  auto take = [&](size_t bytes) {
    size_t off = at;
    at += align_up(bytes);
    return off;
  };
  const size_t elem = p.dtype == HSTU_BF16 ? 2 : 4;
  L.ctrl = take(sizeof(int32_t) * CTRL_WORDS);
  L.seqinfo = take(sizeof(SeqInfo) * (size_t)std::max(p.B, 1));
  L.list_q = take(sizeof(WorkEntry) * (size_t)std::max<int64_t>(p.max_entries, 1));
  L.list_k = for_bwd ? take(sizeof(WorkEntry) * (size_t)std::max<int64_t>(p.max_entries, 1)) : 0;
  L.list_b = for_bwd ? take(2 * sizeof(WorkEntry) * (size_t)std::max<int64_t>(p.max_entries, 1)) : 0;
  L.list_p = !for_bwd && fwd_pairs(p) ? take(sizeof(WorkEntry) * (size_t)pair_entries(p)) : 0;
  L.dO = for_bwd ? take(elem * (size_t)p.T * p.H * p.d) : 0;
  const bool bf16_bwd = for_bwd && p.dtype == HSTU_BF16;
  L.num_cu = device_info(dev).num_cu;
  L.bwd_grid_both = bf16_bwd ? attn_bwd_grid(p, dev) : 0;
  L.bwd_grid_dq = bf16_bwd ? attn_bwd_dq_grid(p, dev) : 0;
  L.bwd_grid_dkv = bf16_bwd ? attn_bwd_dkv_grid(p, dev) : 0;
  // Few items per work-group (short sequences): one launch over both item
  // kinds balances better than two launches with a tail each.  Otherwise
  // each kind runs at its own occupancy.
  L.bwd_combined = bf16_bwd && p.max_entries * p.H < (int64_t)BWD_COMBINED_ITEMS_PER_WG *
                                                      std::max(L.bwd_grid_both, 1);
  // Table-gradient partials: 8 bytes per entry, which the deterministic
  // backward uses as 64-bit fixed point and the default one as float (in
  // the first half).  bf16: per-sequence diagonal partials and DTIME_BINS
  // histograms; fp32: one table-shaped fixed-point staging buffer each
  // (used by the deterministic mode only).
  const bool f32_bwd = for_bwd && p.dtype == HSTU_F32;
  const size_t span = 2 * (size_t)p.N - 1;
  L.dpos_part = !p.has_pos ? 0
                : bf16_bwd ? take(sizeof(int64_t) * (size_t)p.T * p.H)
                : f32_bwd  ? take(sizeof(int64_t) * span * p.H)
                           : 0;
  L.dtime_part = !p.has_time ? 0
                 : bf16_bwd ? take(sizeof(int64_t) * (size_t)DTIME_BINS * p.H * p.nb)
                 : f32_bwd  ? take(sizeof(int64_t) * (size_t)p.H * p.nb)
                            : 0;
  L.total = at;
  return L;
}


int attn_fwd_call(const void *q, const void *k, const void *v, const void *u,
                  const int64_t *seq_offsets, int32_t B, int32_t max_len, int32_t H,
                  int32_t d, const hstu_rab *rab, hstu_fwd_out *out, void *stream,
                  const FixedScratch *fixed) {
  clear_last_error();
  if (!out) return fail(HSTU_EINVAL, "out is NULL");
  Problem p;
  int rc = validate(q, k, v, u, seq_offsets, B, max_len, H, d, rab, out->dtype,
                    out->total_tokens, &p);
  if (rc != HSTU_OK) return rc;
  if (p.T > 0 && (!out->y || !out->o || !out->ln_mean || !out->ln_rstd))
    return fail(HSTU_EINVAL, "out->y, o, ln_mean and ln_rstd must be non-null");
  if (p.T == 0) return HSTU_OK;
  int dev = 0;
  if ((rc = current_device(&dev)) != HSTU_OK) return rc;
  Layout L = make_layout(p, false, dev);
  void *ws = out->workspace;
  if (fixed) {
    if (L.total > fixed->bytes)
      return fail(HSTU_EWORKSPACE,
                  "this problem needs %zu bytes of workspace; the no-allocation entry "
                  "point's fixed scratch holds %zu",
                  L.total, fixed->bytes);
    if (!(ws = fixed->addr(dev))) return HSTU_EHIP;   // addr() recorded the error
  } else if ((rc = check_workspace(L, ws, out->workspace_bytes)) != HSTU_OK) {
    return rc;
  }
  hipStream_t s = (hipStream_t)stream;
  AttnArgs a{q, k, v, u,
             rab ? rab->pos_w : nullptr,
             p.has_time ? rab->time_w : nullptr,
             p.has_time ? rab->timestamps : nullptr,
             ws, L, p};
  // the no-allocation path never records profiler events (creating one may
  // allocate)
  const bool prof_on = !fixed;
  hipError_t e;
  {
    prof::Scope ps(prof_on ? "schedule" : nullptr, s);
    e = launch_schedule(seq_offsets, p, ws, L, s);
  }
  if (e != hipSuccess) return hip_fail(e, "schedule launch");
  {
    prof::Scope ps(!prof_on ? nullptr : p.dtype == HSTU_BF16 ? "attn_fwd" : "attn_fwd_f32", s);
    e = p.dtype == HSTU_BF16 ? launch_attn_fwd_bf16(a, out->o, s)
                             : launch_attn_fwd_f32(a, out->o, s);
  }
  if (e != hipSuccess) return hip_fail(e, "attention forward launch");
  {
    prof::Scope ps(prof_on ? "ln_fwd" : nullptr, s);
    e = launch_ln_fwd(p, out->o, u, out->y, out->ln_mean, out->ln_rstd, s);
  }
  if (e != hipSuccess) return hip_fail(e, "layernorm forward launch");
  return HSTU_OK;
}

int attn_bwd_call(const void *q, const void *k, const void *v, const void *u,
                  const int64_t *seq_offsets, int32_t B, int32_t max_len, int32_t H,
                  int32_t d, const hstu_rab *rab, hstu_bwd_io *io, void *stream,
                  const GradOut *go) {
  if (!io) return fail(HSTU_EINVAL, "io is NULL");
  Problem p;
  int rc = validate(q, k, v, u, seq_offsets, B, max_len, H, d, rab, io->dtype,
                    io->total_tokens, &p);
  if (rc != HSTU_OK) return rc;
  if (go && p.dtype != HSTU_BF16)
    return fail(HSTU_ENOTSUP, "fused gradient outputs need HSTU_BF16");
  if (p.T > 0 && (!io->dy || !io->o || !io->ln_mean || !io->ln_rstd || !io->dq ||
                  !io->dk || !io->dv || !io->du))
    return fail(HSTU_EINVAL, "io->dy, o, ln_mean, ln_rstd, dq, dk, dv, du must be non-null");
  if (p.has_pos && !io->d_pos_w)
    return fail(HSTU_EINVAL, "rab->pos_w given but io->d_pos_w is NULL");
  if (p.has_time && !io->d_time_w)
    return fail(HSTU_EINVAL, "rab->time_w given but io->d_time_w is NULL");
  if (p.T == 0 && !p.has_pos && !p.has_time) return HSTU_OK;
  p.deterministic = io->deterministic != 0;
  int dev = 0;
  if ((rc = current_device(&dev)) != HSTU_OK) return rc;
  Layout L = make_layout(p, true, dev);
  if ((rc = check_workspace(L, io->workspace, io->workspace_bytes)) != HSTU_OK)
    return rc;
  hipStream_t s = (hipStream_t)stream;
  AttnArgs a{q, k, v, u,
             rab ? rab->pos_w : nullptr,
             p.has_time ? rab->time_w : nullptr,
             p.has_time ? rab->timestamps : nullptr,
             io->workspace, L, p};
  char *ws = (char *)io->workspace;
  float *d_pos = p.has_pos ? io->d_pos_w : nullptr;
  float *d_time = p.has_time ? io->d_time_w : nullptr;
  hipError_t e;
  if (p.T > 0) {
    // the LayerNorm backward launch also builds the work lists
    prof::Scope ps("ln_bwd", s);
    e = launch_ln_bwd_sched(p, io->dy, u, io->o, io->ln_mean, io->ln_rstd, io->du,
                            ws + L.dO,
                            (L.dpos_part && p.dtype == HSTU_BF16) ? ws + L.dpos_part : nullptr,
                            seq_offsets, ws, L, go, s);
    if (e != hipSuccess) return hip_fail(e, "layernorm backward launch");
  } else {
    prof::Scope ps("schedule", s);
    e = launch_schedule(seq_offsets, p, ws, L, s);
    if (e != hipSuccess) return hip_fail(e, "schedule launch");
  }
  if (p.dtype == HSTU_BF16) {
    e = launch_attn_bwd_bf16(a, ws + L.dO, io->dq, io->dk, io->dv, go, s);
    if (e != hipSuccess) return hip_fail(e, "attention backward launch");
    {
      prof::Scope ps("finalize_tables", s);
      e = launch_finalize_tables(a, d_pos, d_time, s);
    }
    if (e != hipSuccess) return hip_fail(e, "table finalize launch");
  } else {
    prof::Scope ps("attn_bwd_f32", s);
    e = launch_attn_bwd_f32(a, ws + L.dO, io->dq, io->dk, io->dv, d_pos, d_time, s);
    if (e != hipSuccess) return hip_fail(e, "attention backward launch");
  }
  return HSTU_OK;
}

}  // namespace hstu

using namespace hstu;

extern "C" {

const char *hstu_last_error(void) { return g_last_error.c_str(); }

const char *hstu_version(void) { return "hstu_jagged 0.1 gfx950"; }

size_t hstu_jagged_attn_workspace_bytes(int32_t B, int32_t max_len, int32_t H,
                                        int32_t d, int64_t total_tokens,
                                        int32_t for_bwd, hstu_dtype dtype,
                                        const hstu_rab *rab) {
  Problem p;
  static const char dummy = 0;
  g_last_error.clear();
  if (validate(&dummy, &dummy, &dummy, &dummy, (const int64_t *)&dummy, B,
               max_len, H, d, rab, dtype, total_tokens, &p) != HSTU_OK)
    return 0;
  int dev = 0;
  if (current_device(&dev) != HSTU_OK) return 0;
  return make_layout(p, for_bwd != 0, dev).total;
}

int hstu_jagged_schedule(const int64_t *seq_offsets, int32_t B,
                         int32_t max_len, int64_t total_tokens,
                         int32_t *n_entries, int32_t *list_q, int32_t *list_k,
                         void *workspace, size_t workspace_bytes, void *stream) {
  g_last_error.clear();
  Problem p;
  static const char dummy = 0;
  int rc = validate(&dummy, &dummy, &dummy, &dummy, seq_offsets, B, max_len, 1,
                    64, nullptr, HSTU_F32, total_tokens, &p);
  if (rc != HSTU_OK) return rc;
  if (!n_entries || (p.max_entries > 0 && (!list_q || !list_k)))
    return fail(HSTU_EINVAL, "n_entries, list_q and list_k must be non-null");
  int dev = 0;
  if ((rc = current_device(&dev)) != HSTU_OK) return rc;
  Layout L = make_layout(p, true, dev);
  if ((rc = check_workspace(L, workspace, workspace_bytes)) != HSTU_OK) return rc;
  hipStream_t s = (hipStream_t)stream;
  hipError_t e = launch_schedule(seq_offsets, p, workspace, L, s);
  if (e != hipSuccess) return hip_fail(e, "schedule launch");
  const char *ws = (const char *)workspace;
  // the exported lists are the (sequence, tile) pairs of the entries
  const size_t rows = (size_t)p.max_entries;
  e = hipMemcpyAsync(n_entries, ws + L.ctrl + sizeof(int32_t) * CTRL_N_ENTRIES,
                     sizeof(int32_t), hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess && rows)
    e = hipMemcpy2DAsync(list_q, 2 * sizeof(int32_t), ws + L.list_q, sizeof(WorkEntry),
                         2 * sizeof(int32_t), rows, hipMemcpyDeviceToDevice, s);
  if (e == hipSuccess && rows)
    e = hipMemcpy2DAsync(list_k, 2 * sizeof(int32_t), ws + L.list_k, sizeof(WorkEntry),
                         2 * sizeof(int32_t), rows, hipMemcpyDeviceToDevice, s);
  if (e != hipSuccess) return hip_fail(e, "work-list copy");
  return HSTU_OK;
}

int hstu_jagged_attn_fwd(const void *q, const void *k, const void *v,
                         const void *u, const int64_t *seq_offsets, int32_t B,
                         int32_t max_len, int32_t H, int32_t d,
                         const hstu_rab *rab, hstu_fwd_out *out, void *stream) {
  return attn_fwd_call(q, k, v, u, seq_offsets, B, max_len, H, d, rab, out, stream, nullptr);
}

int hstu_jagged_attn_bwd(const void *q, const void *k, const void *v,
                         const void *u, const int64_t *seq_offsets, int32_t B,
                         int32_t max_len, int32_t H, int32_t d,
                         const hstu_rab *rab, hstu_bwd_io *io, void *stream) {
  g_last_error.clear();
  return attn_bwd_call(q, k, v, u, seq_offsets, B, max_len, H, d, rab, io, stream, nullptr);
}

int hstu_jagged_status(const void *workspace, int32_t *status, void *stream) {
  g_last_error.clear();
  if (!workspace || !status) return fail(HSTU_EINVAL, "workspace and status must be non-null");
  const char *ws = (const char *)workspace;
  const hipError_t e = hipMemcpyAsync(status, ws + sizeof(int32_t) * CTRL_STATUS,
                                      sizeof(int32_t), hipMemcpyDefault, (hipStream_t)stream);
  if (e != hipSuccess) return hip_fail(e, "status copy");
  return HSTU_OK;
}

int hstu_profile_enable(int on) {
  prof::on.store(on != 0);
  return HSTU_OK;
}

int hstu_profile_read(int max, const char **names, double *total_ms,
                      int *launches) {
  g_last_error.clear();
  if (max < 0 || (max > 0 && (!names || !total_ms || !launches)))
    return fail(HSTU_EINVAL, "bad profile_read arguments");
  std::lock_guard<std::mutex> lock(prof::mu);
  int rows = 0;
  int rc = 0;
  for (const prof::Rec &r : prof::recs) {
    float ms = 0.0f;
    hipError_t e = hipEventSynchronize(r.b);
    if (e == hipSuccess) e = hipEventElapsedTime(&ms, r.a, r.b);
    if (e != hipSuccess) rc = hip_fail(e, "profile event");
    int k = 0;
    while (k < rows && std::strcmp(names[k], r.name) != 0) ++k;
    if (k == rows) {
      if (rows == max) continue;
      names[k] = r.name;
      total_ms[k] = 0.0;
      launches[k] = 0;
      ++rows;
    }
    total_ms[k] += ms;
    launches[k] += 1;
  }
  for (const prof::Rec &r : prof::recs) {
    prof::pool.push_back(r.a);
    prof::pool.push_back(r.b);
  }
  prof::recs.clear();
  return rc < 0 ? rc : rows;
}

}  // extern "C"
