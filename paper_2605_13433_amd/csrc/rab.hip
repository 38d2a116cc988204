// Standalone relative attention bias (RAB) of Sec. 4.1.1's operator on
// gfx950: the jagged bias tensor (one L x L square per sequence, no
// padding) from the position table, the bucketed time table and a
// functional time encoding, and its backward into those parameters.
//
// Square tiling: work-group (b, it, h) owns the 64-row band it of sequence
// b's square for head h and walks its 64 x 64 tiles; the tile's position
// slice and the head's time table sit in LDS; lane c of a wave handles column c of
// a tile and the wave's rows, so every store (forward) and load (backward)
// of a wave is one contiguous 256-byte row segment, whatever the square's
// alignment.  Per element the forward adds the biases in registers; the
// backward sums the incoming gradient by diagonal (an LDS window of the
// tile's 127 diagonals), by time bucket (per-lane runs over the row order
// into an LDS histogram) and into the functional encoding's two parameter
// gradients (per-lane sums, reduced across the work-group in a fixed
// order).  All table sums are 64-bit fixed point added with integer
// atomics: the result does not depend on the order in which work-groups
// finish, so the backward is bitwise reproducible.
#include <algorithm>

#include "internal.h"
#include "device.h"

namespace hstu {
namespace {

constexpr int RT = 256;                 // threads: 4 waves x 64 columns
constexpr int ROWS_PER_THREAD = TILE / (RT / TILE);   // 16

struct RabArgs {
  const int64_t *off;
  int64_t *sq;                          // [B+1] square offsets (workspace)
  const float *pos_w, *time_w, *time_fn;
  const int64_t *ts;
  float *rab;
  const float *d_rab;
  unsigned long long *fix_pos, *fix_time, *fix_fn;
  int64_t T, total_square;
  int B, N, H, nb;
};

// Clamped start and length of sequence b (as the attention's scheduler
// clamps them: every row index stays inside [0, T)).
__device__ __forceinline__ void seq_of(const RabArgs &a, int b, int64_t &start, int &len) {
  int64_t s0 = a.off[b], s1 = a.off[b + 1];
  s0 = s0 < 0 ? 0 : (s0 > a.T ? a.T : s0);
  s1 = s1 < s0 ? s0 : (s1 > a.T ? a.T : s1);
  int64_t L = s1 - s0;
  start = s0;
  len = (int)(L > a.N ? a.N : L);
}

// sq[b] = sum of L_b'^2 over b' < b: each thread sums a contiguous run of
// sequences, the run totals are scanned in LDS, then every run is written.
__global__ void __launch_bounds__(1024) rab_sq_kernel(RabArgs a) {
  __shared__ int64_t part[1024];
  const int t = threadIdx.x;
  const int per = (a.B + 1023) / 1024;
  const int b0 = t * per, b1 = min(a.B, b0 + per);
  int64_t s = 0;
  for (int b = b0; b < b1; ++b) {
    int64_t st; int L;
    seq_of(a, b, st, L);
    s += (int64_t)L * L;
  }
  part[t] = s;
  __syncthreads();
  if (t == 0) {
    int64_t run = 0;
    for (int x = 0; x < 1024; ++x) { const int64_t v = part[x]; part[x] = run; run += v; }
    a.sq[a.B] = run;
  }
  __syncthreads();
  s = part[t];
  for (int b = b0; b < b1; ++b) {
    a.sq[b] = s;
    int64_t st; int L;
    seq_of(a, b, st, L);
    s += (int64_t)L * L;
  }
}

__global__ void rab_zero_kernel(unsigned long long *p, int64_t n) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n;
       x += (int64_t)gridDim.x * blockDim.x)
    p[x] = 0;
}

__global__ void rab_fix_to_float_kernel(const unsigned long long *fix, float *out, int64_t n) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n;
       x += (int64_t)gridDim.x * blockDim.x)
    out[x] = (float)((double)(long long)fix[x] * (1.0 / FIX_ONE));
}

// 64-bit fixed-point value of a double partial sum (as to_fix).
__device__ __forceinline__ unsigned long long fix_d(double v) {
  return (unsigned long long)(long long)__builtin_rint(v * FIX_ONE);
}

// log2(1 + |dt|) of the functional time term g = (1 + |dt|)^(-beta)
// (32-bit conversion while |dt| fits, the common case).
__device__ __forceinline__ float fn_lg2(int64_t dt) {
  const uint64_t x = dt < 0 ? (uint64_t)0 - (uint64_t)dt : (uint64_t)dt;
  const float xf = x < (1u << 31) ? (float)(uint32_t)x : (float)x;
  return __builtin_amdgcn_logf(1.0f + xf);
}

// The bucket rule on a time gap, with a 32-bit path while |dt| < 2^32.
__device__ __forceinline__ int bucket_fast(int64_t dt, int nb) {
  const uint64_t x = dt < 0 ? (uint64_t)0 - (uint64_t)dt : (uint64_t)dt;
  if (x >> 32) return time_bucket(dt, nb);
  const uint32_t y = (uint32_t)x;
  int b;
  if (y < 4) {
    b = (int)y;
  } else {
    const int e = 31 - __clz((int)y);
    b = 4 * (e - 1) + (int)((y >> (e - 2)) & 3u);
  }
  return b < nb - 1 ? b : nb - 1;
}

// Band setup shared by both passes: sequence, band rows of this thread and
// their timestamps.  Returns false when the band lies past the sequence (or
// the square would not fit the caller's tensor).
struct Band {
  int64_t start, base;                  // first row; sq[b]
  int L, it, nt, c, rg;
  int64_t ts_i[ROWS_PER_THREAD];
};

__device__ __forceinline__ bool band_of(const RabArgs &a, Band &bd) {
  const int b = blockIdx.x;
  bd.it = blockIdx.y;
  seq_of(a, b, bd.start, bd.L);
  if ((int64_t)bd.it * TILE >= bd.L) return false;
  bd.base = a.sq[b];
  if (bd.base < 0 || bd.base + (int64_t)bd.L * bd.L > a.total_square) return false;
  bd.nt = (bd.L + TILE - 1) / TILE;
  bd.c = threadIdx.x & 63;
  bd.rg = threadIdx.x >> 6;
  if (a.ts) {
#pragma unroll
    for (int k = 0; k < ROWS_PER_THREAD; ++k) {
      const int i = bd.it * TILE + bd.rg + 4 * k;
      bd.ts_i[k] = a.ts[bd.start + (i < bd.L ? i : bd.L - 1)];
    }
  }
  return true;
}

// Dynamic LDS: the head's time table (nb floats) when time_w is given.  The
// next tile's position-slice entry and column timestamp are loaded while
// the current tile is computed (double-buffered slice, one barrier a tile).
template <bool POS, bool TIME, bool FN>
__global__ void __launch_bounds__(RT) rab_fwd_kernel(RabArgs a) {
  __shared__ float pos[2][2 * TILE];
  extern __shared__ float ttab[];
  Band bd;
  if (!band_of(a, bd)) return;
  const int h = blockIdx.z, tid = threadIdx.x;
  const int span = 2 * a.N - 1;
  float fa = 0.0f, fb = 0.0f;
  if (FN) { fa = a.time_fn[2 * h]; fb = a.time_fn[2 * h + 1]; }
  if (TIME)
    for (int x = tid; x < a.nb; x += RT) ttab[x] = a.time_w[(int64_t)h * a.nb + x];
  // slice entry x of tile jt: offset j - i = (jt - it) 64 + x - 63
  auto pos_at = [&](int jt) {
    const int m = (jt - bd.it) * TILE + tid - (TILE - 1) + a.N - 1;
    return (tid < 2 * TILE - 1 && m >= 0 && m < span) ? a.pos_w[(int64_t)h * span + m] : 0.0f;
  };
  auto ts_at = [&](int jt) {
    const int j = jt * TILE + bd.c;
    return (TIME || FN) ? a.ts[bd.start + (j < bd.L ? j : bd.L - 1)] : (int64_t)0;
  };
  float pv = POS ? pos_at(0) : 0.0f;
  int64_t ts_j = ts_at(0);
  // rows of this thread past the sequence (band of the last tile) store
  // nothing; columns are checked per tile
  const int rows_ok = min(ROWS_PER_THREAD, (bd.L - bd.it * TILE - bd.rg + 3) / 4);
  float *plane = a.rab + (int64_t)h * a.total_square + bd.base +
                 (int64_t)(bd.it * TILE + bd.rg) * bd.L + bd.c;
  for (int jt = 0; jt < bd.nt; ++jt) {
    float *pb = pos[jt & 1];
    if (POS && tid < 2 * TILE - 1) pb[tid] = pv;
    __syncthreads();
    const int64_t ts_cur = ts_j;
    if (jt + 1 < bd.nt) {
      if (POS) pv = pos_at(jt + 1);
      ts_j = ts_at(jt + 1);
    }
    if (jt * TILE + bd.c >= bd.L) continue;
    float *col = plane + jt * TILE;
#pragma unroll
    for (int k = 0; k < ROWS_PER_THREAD; ++k) {
      if (k < rows_ok) {
        const int r = bd.rg + 4 * k;
        float v = 0.0f;
        if (POS) v += pb[bd.c - r + TILE - 1];
        if (TIME || FN) {
          const int64_t dt = bd.ts_i[k] - ts_cur;
          if (TIME) v += ttab[bucket_fast(dt, a.nb)];
          if (FN) v += fa * __builtin_amdgcn_exp2f(-fb * fn_lg2(dt));
        }
        col[(int64_t)(4 * k) * bd.L] = v;
      }
    }
  }
}

// Backward: dynamic LDS = the head's [nb] fixed-point time histogram (if
// time_w).
template <bool POS, bool TIME, bool FN>
__global__ void __launch_bounds__(RT) rab_bwd_kernel(RabArgs a) {
  __shared__ unsigned long long win[2 * TILE];
  __shared__ double red[2][RT];
  extern __shared__ unsigned long long hist[];
  Band bd;
  if (!band_of(a, bd)) return;
  const int tid = threadIdx.x;
  const int span = 2 * a.N - 1;
  for (int x = tid; x < 2 * TILE; x += RT) win[x] = 0;
  if (TIME)
    for (int x = tid; x < a.nb; x += RT) hist[x] = 0;
  __syncthreads();
  const int rows_ok = min(ROWS_PER_THREAD, (bd.L - bd.it * TILE - bd.rg + 3) / 4);
  constexpr float LN2 = 0.693147180559945309f;
  {
    const int h = blockIdx.z;
    // per-lane sums in double: the incoming gradient has both signs, and
    // its long sums cancel
    float fa = 0.0f, fb = 0.0f;
    double s_a = 0.0, s_b = 0.0;
    if (FN) { fa = a.time_fn[2 * h]; fb = a.time_fn[2 * h + 1]; }
    const float *plane = a.d_rab + (int64_t)h * a.total_square + bd.base +
                         (int64_t)(bd.it * TILE + bd.rg) * bd.L + bd.c;
    unsigned long long *hh = hist;
    for (int jt = 0; jt < bd.nt; ++jt) {
      const int j = jt * TILE + bd.c;
      if (j < bd.L) {
        const int64_t ts_j = (TIME || FN) ? a.ts[bd.start + j] : 0;
        const float *col = plane + jt * TILE;
        double run = 0.0;
        int cur = -1;
        float gv[ROWS_PER_THREAD];
#pragma unroll
        for (int k = 0; k < ROWS_PER_THREAD; ++k)
          gv[k] = k < rows_ok ? col[(int64_t)(4 * k) * bd.L] : 0.0f;
#pragma unroll
        for (int k = 0; k < ROWS_PER_THREAD; ++k) {
          if (k >= rows_ok) continue;
          const float g = gv[k];
          if (POS) atomicAdd(&win[bd.c - (bd.rg + 4 * k) + TILE - 1], to_fix(g));
          const int64_t dt = bd.ts_i[k] - ts_j;
          if (TIME) {
            const int bk = bucket_fast(dt, a.nb);
            if (bk != cur && cur >= 0) atomicAdd(&hh[cur], fix_d(run));
            run = bk != cur ? (double)g : run + g;
            cur = bk;
          }
          if (FN) {
            const float l2 = fn_lg2(dt);
            const float e = __builtin_amdgcn_exp2f(-fb * l2);
            s_a += (double)(g * e);
            s_b -= (double)(g * fa * e) * (double)(l2 * LN2);
          }
        }
        if (TIME && cur >= 0) atomicAdd(&hh[cur], fix_d(run));
      }
      if (POS) {
        // the tile's 127 diagonal sums go to the table, the window is cleared
        __syncthreads();
        if (tid < 2 * TILE - 1) {
          const unsigned long long v = win[tid];
          const int m = (jt - bd.it) * TILE + tid - (TILE - 1) + a.N - 1;
          if (v != 0 && m >= 0 && m < span) atomicAdd(&a.fix_pos[(int64_t)h * span + m], v);
          win[tid] = 0;
        }
        __syncthreads();
      }
    }
    if (FN) {
      // work-group sums of the two parameter gradients, fixed order
      red[0][tid] = s_a;
      red[1][tid] = s_b;
      __syncthreads();
      if (tid < 2) {
        double t = 0.0;
        for (int x = 0; x < RT; ++x) t += red[tid][x];
        atomicAdd(&a.fix_fn[2 * h + tid], fix_d(t));
      }
      __syncthreads();
    }
  }
  if (TIME) {
    __syncthreads();
    for (int x = tid; x < a.nb; x += RT)
      if (hist[x] != 0) atomicAdd(&a.fix_time[(int64_t)blockIdx.z * a.nb + x], hist[x]);
  }
}

// ------------------------------------------------------------------- host
int check_rab(const int64_t *off, int32_t B, int32_t N, int32_t H, int64_t T,
              int64_t total_square, const hstu_rab_params *rp) {
  if (B < 0) return fail(HSTU_EINVAL, "B = %d < 0", B);
  if (N < 1 || N > 65536) return fail(HSTU_EINVAL, "max_len = %d outside [1, 65536]", N);
  if (H < 1 || H > 64) return fail(HSTU_EINVAL, "H = %d outside [1, 64]", H);
  if (T < 0 || total_square < 0)
    return fail(HSTU_EINVAL, "total_tokens and total_square must be >= 0");
  if (!off && B > 0) return fail(HSTU_EINVAL, "seq_offsets must be non-null");
  if (!rp) return fail(HSTU_EINVAL, "rp is NULL");
  if ((rp->time_w || rp->time_fn) && !rp->timestamps && T > 0)
    return fail(HSTU_EINVAL, "time_w or time_fn given without timestamps");
  if (rp->time_w && (rp->num_buckets < 1 || (int64_t)H * rp->num_buckets > 4096))
    return fail(HSTU_EINVAL, "num_buckets = %d (need >= 1 and H * num_buckets <= 4096)",
                rp->num_buckets);
  return HSTU_OK;
}

struct RabLayout {
  size_t sq, fpos, ftime, ffn, total;
};

RabLayout rab_layout(int32_t B, int32_t N, int32_t H, const hstu_rab_params *rp) {
  RabLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = align_up(o + bytes); return at; };
  L.sq = take(sizeof(int64_t) * ((size_t)B + 1));
  L.fpos = rp->pos_w ? take(8 * (size_t)H * (2 * (size_t)N - 1)) : 0;
  L.ftime = rp->time_w ? take(8 * (size_t)H * rp->num_buckets) : 0;
  L.ffn = rp->time_fn ? take(8 * 2 * (size_t)H) : 0;
  L.total = o;
  return L;
}

RabArgs rab_args(const int64_t *off, int32_t B, int32_t N, int32_t H, int64_t T,
                 int64_t total_square, const hstu_rab_params *rp, char *ws,
                 const RabLayout &L) {
  RabArgs a{};
  a.off = off;
  a.sq = (int64_t *)(ws + L.sq);
  a.pos_w = rp->pos_w;
  a.time_w = rp->time_w;
  a.time_fn = rp->time_fn;
  a.ts = (rp->time_w || rp->time_fn) ? rp->timestamps : nullptr;
  a.fix_pos = rp->pos_w ? (unsigned long long *)(ws + L.fpos) : nullptr;
  a.fix_time = rp->time_w ? (unsigned long long *)(ws + L.ftime) : nullptr;
  a.fix_fn = rp->time_fn ? (unsigned long long *)(ws + L.ffn) : nullptr;
  a.T = T;
  a.total_square = total_square;
  a.B = B;
  a.N = N;
  a.H = H;
  a.nb = rp->time_w ? rp->num_buckets : 0;
  return a;
}

}  // namespace
}  // namespace hstu

using namespace hstu;

extern "C" size_t hstu_jagged_rab_workspace_bytes(int32_t B, int32_t max_len, int32_t H,
                                                  const hstu_rab_params *rp) {
  clear_last_error();
  static const int64_t dummy = 0;
  if (check_rab(&dummy, B, max_len, H, 0, 0, rp)) return 0;
  return rab_layout(B, max_len, H, rp).total;
}

extern "C" int hstu_jagged_rab_fwd(const int64_t *seq_offsets, int32_t B, int32_t max_len,
                                   int32_t H, int64_t total_tokens, int64_t total_square,
                                   const hstu_rab_params *rp, float *rab, void *workspace,
                                   size_t workspace_bytes, void *stream) {
  clear_last_error();
  int rc = check_rab(seq_offsets, B, max_len, H, total_tokens, total_square, rp);
  if (rc) return rc;
  if (B == 0 || total_square == 0) return HSTU_OK;
  if (!rab) return fail(HSTU_EINVAL, "rab must be non-null");
  const RabLayout L = rab_layout(B, max_len, H, rp);
  if ((rc = check_workspace_bytes(L.total, workspace, workspace_bytes))) return rc;
  const hipStream_t s = (hipStream_t)stream;
  RabArgs a = rab_args(seq_offsets, B, max_len, H, total_tokens, total_square, rp,
                       (char *)workspace, L);
  a.rab = rab;
  prof::Scope ps("rab_fwd", s);
  hipLaunchKernelGGL(rab_sq_kernel, dim3(1), dim3(1024), 0, s, a);
  const bool P = rp->pos_w, Tm = rp->time_w, F = rp->time_fn;
  auto kfn = P ? (Tm ? (F ? rab_fwd_kernel<true, true, true> : rab_fwd_kernel<true, true, false>)
                     : (F ? rab_fwd_kernel<true, false, true> : rab_fwd_kernel<true, false, false>))
               : (Tm ? (F ? rab_fwd_kernel<false, true, true> : rab_fwd_kernel<false, true, false>)
                     : (F ? rab_fwd_kernel<false, false, true>
                          : rab_fwd_kernel<false, false, false>));
  hipLaunchKernelGGL(kfn, dim3(B, (max_len + TILE - 1) / TILE, H), dim3(RT),
                     rp->time_w ? sizeof(float) * (size_t)rp->num_buckets : 0, s, a);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? HSTU_OK : hip_fail(e, "rab forward launch");
}

extern "C" int hstu_jagged_rab_bwd(const int64_t *seq_offsets, int32_t B, int32_t max_len,
                                   int32_t H, int64_t total_tokens, int64_t total_square,
                                   const hstu_rab_params *rp, const float *d_rab,
                                   float *d_pos_w, float *d_time_w, float *d_time_fn,
                                   void *workspace, size_t workspace_bytes, void *stream) {
  clear_last_error();
  int rc = check_rab(seq_offsets, B, max_len, H, total_tokens, total_square, rp);
  if (rc) return rc;
  if ((rp->pos_w && !d_pos_w) || (rp->time_w && !d_time_w) || (rp->time_fn && !d_time_fn))
    return fail(HSTU_EINVAL, "a gradient output is NULL for a given parameter");
  if (B > 0 && total_square > 0 && !d_rab) return fail(HSTU_EINVAL, "d_rab must be non-null");
  const RabLayout L = rab_layout(B, max_len, H, rp);
  if ((rc = check_workspace_bytes(L.total, workspace, workspace_bytes))) return rc;
  const hipStream_t s = (hipStream_t)stream;
  char *ws = (char *)workspace;
  RabArgs a = rab_args(seq_offsets, B, max_len, H, total_tokens, total_square, rp, ws, L);
  a.d_rab = d_rab;
  const int64_t n_pos = (int64_t)H * (2 * (int64_t)max_len - 1);
  const int64_t n_time = rp->time_w ? (int64_t)H * rp->num_buckets : 0;
  prof::Scope ps("rab_bwd", s);
  if (a.fix_pos) hipLaunchKernelGGL(rab_zero_kernel, dim3(64), dim3(256), 0, s, a.fix_pos, n_pos);
  if (a.fix_time) hipLaunchKernelGGL(rab_zero_kernel, dim3(8), dim3(256), 0, s, a.fix_time, n_time);
  if (a.fix_fn) hipLaunchKernelGGL(rab_zero_kernel, dim3(1), dim3(256), 0, s, a.fix_fn,
                                   (int64_t)2 * H);
  if (B > 0 && total_square > 0) {
    hipLaunchKernelGGL(rab_sq_kernel, dim3(1), dim3(1024), 0, s, a);
    const size_t dyn = rp->time_w ? 8 * (size_t)rp->num_buckets : 0;
    const bool P = rp->pos_w, Tm = rp->time_w, F = rp->time_fn;
    auto kfn =
        P ? (Tm ? (F ? rab_bwd_kernel<true, true, true> : rab_bwd_kernel<true, true, false>)
                : (F ? rab_bwd_kernel<true, false, true> : rab_bwd_kernel<true, false, false>))
          : (Tm ? (F ? rab_bwd_kernel<false, true, true> : rab_bwd_kernel<false, true, false>)
                : (F ? rab_bwd_kernel<false, false, true> : rab_bwd_kernel<false, false, false>));
    hipLaunchKernelGGL(kfn, dim3(B, (max_len + TILE - 1) / TILE, H), dim3(RT), dyn, s, a);
  }
  if (a.fix_pos)
    hipLaunchKernelGGL(rab_fix_to_float_kernel, dim3(64), dim3(256), 0, s, a.fix_pos, d_pos_w,
                       n_pos);
  if (a.fix_time)
    hipLaunchKernelGGL(rab_fix_to_float_kernel, dim3(8), dim3(256), 0, s, a.fix_time, d_time_w,
                       n_time);
  if (a.fix_fn)
    hipLaunchKernelGGL(rab_fix_to_float_kernel, dim3(1), dim3(256), 0, s, a.fix_fn, d_time_fn,
                       (int64_t)2 * H);
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? HSTU_OK : hip_fail(e, "rab backward launch");
}
