// LayerNorm + U-gating around the jagged attention, and the reduction of the
// bias-table gradient partials.
//
//   forward   y = (o - mean) * rstd * u, per token over all H*d features,
//             biased variance, rstd = 1/sqrt(var + eps); saves mean, rstd
//   backward  du = n * dy;  g = dy * u;
//             dO = rstd * (g - mean(g) - n * mean(g * n)),  n = (o - mean) * rstd
//
// When a token's F = H*d features are 8 x (a power of two <= 64) -- F <= 512,
// every configuration of the benchmarks -- a wave holds 64/(F/8) whole tokens,
// each lane 8 consecutive features of one token loaded once (16 bytes per
// bf16 tensor, every load of the token issued before the first use), and the
// statistics are shuffle sums over the token's lane group.  Otherwise one
// wave64 walks a token in 512-wide chunks.  These kernels are HBM-bound
// (each feature is read and written once or twice).
#include <algorithm>

#include "internal.h"
#include "device.h"
#include "sched_impl.h"

namespace hstu {

namespace {

constexpr int LN_THREADS = 256;   // 4 tokens per work-group
constexpr int LN_WAVES = LN_THREADS / 64;

__device__ __forceinline__ float wave_sum(float x) {
#pragma unroll
  for (int m = 32; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

template <typename T>
struct Vec8;

template <>
struct Vec8<u16> {
  __device__ static void load(const u16 *p, float (&f)[8]) {
    const uint4 x = *(const uint4 *)p;
    const uint32_t w[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
    for (int e = 0; e < 4; ++e) {
      f[2 * e] = bf2f((u16)(w[e] & 0xffffu));
      f[2 * e + 1] = bf2f((u16)(w[e] >> 16));
    }
  }
  __device__ static void store(u16 *p, const float (&f)[8]) {
    uint4 x;
    x.x = pack2(f[0], f[1]);
    x.y = pack2(f[2], f[3]);
    x.z = pack2(f[4], f[5]);
    x.w = pack2(f[6], f[7]);
    *(uint4 *)p = x;
  }
};

template <>
struct Vec8<float> {
  __device__ static void load(const float *p, float (&f)[8]) {
    const float4 a = *(const float4 *)p, b = *(const float4 *)(p + 4);
    f[0] = a.x; f[1] = a.y; f[2] = a.z; f[3] = a.w;
    f[4] = b.x; f[5] = b.y; f[6] = b.z; f[7] = b.w;
  }
  __device__ static void store(float *p, const float (&f)[8]) {
    *(float4 *)p = make_float4(f[0], f[1], f[2], f[3]);
    *(float4 *)(p + 4) = make_float4(f[4], f[5], f[6], f[7]);
  }
};

// Sum over the aligned group of L lanes (L a power of two) holding one token.
template <int L>
__device__ __forceinline__ float group_sum(float x) {
#pragma unroll
  for (int m = L / 2; m >= 1; m >>= 1) x += __shfl_xor(x, m, 64);
  return x;
}

// Fast path: F = 8 L, L = 64 / TPW lanes per token, TPW tokens per wave.
template <typename T, int L>
__global__ void __launch_bounds__(LN_THREADS)
ln_fwd_group_kernel(const T *__restrict__ o, const T *__restrict__ u,
                    T *__restrict__ y, float *__restrict__ mean_out,
                    float *__restrict__ rstd_out, int64_t T_tokens) {
  constexpr int F = 8 * L, TPW = 64 / L;
  const int lane = threadIdx.x & 63, sub = lane % L;
  const int64_t r = ((int64_t)blockIdx.x * LN_WAVES + (threadIdx.x >> 6)) * TPW + lane / L;
  if (r >= T_tokens) return;
  const int64_t at = r * F + 8 * sub;
  float z[8], uu[8];
  Vec8<T>::load(o + at, z);
  Vec8<T>::load(u + at, uu);
  float sum = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) sum += z[e];
  const float mu = group_sum<L>(sum) / (float)F;
  float sq = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) sq += (z[e] - mu) * (z[e] - mu);
  const float rstd = rsqrtf(group_sum<L>(sq) / (float)F + HSTU_LN_EPS);
  float out[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) out[e] = (z[e] - mu) * rstd * uu[e];
  Vec8<T>::store(y + at, out);
  if (sub == 0) {
    mean_out[r] = mu;
    rstd_out[r] = rstd;
  }
}

// g[e] *= silu'(h[e]) for eight consecutive elements.
template <typename T>
__device__ __forceinline__ void silu_back8(const T *__restrict__ h, float g[8]) {
  float hh[8];
  Vec8<T>::load(h, hh);
#pragma unroll
  for (int e = 0; e < 8; ++e) g[e] *= dsilu_f(hh[e]);
}

template <typename T, int L>
__device__ __forceinline__ void ln_bwd_group(const T *__restrict__ dy, const T *__restrict__ u,
                                             const T *__restrict__ o,
                                             const float *__restrict__ mean,
                                             const float *__restrict__ rstd,
                                             T *__restrict__ du, T *__restrict__ dO,
                                             uint64_t *__restrict__ dpos_part, int H,
                                             int64_t T_tokens, int block, int64_t du_stride,
                                             const T *__restrict__ du_h) {
  constexpr int F = 8 * L, TPW = 64 / L;
  const int lane = threadIdx.x & 63, sub = lane % L;
  const int64_t r = ((int64_t)block * LN_WAVES + (threadIdx.x >> 6)) * TPW + lane / L;
  if (r >= T_tokens) return;
  const int64_t at = r * F + 8 * sub;
  float z[8], g[8], uu[8];
  Vec8<T>::load(o + at, z);
  Vec8<T>::load(dy + at, g);
  Vec8<T>::load(u + at, uu);
  const float mu = mean[r], rs = rstd[r];
  float sg = 0.0f, sgn = 0.0f;
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float n = (z[e] - mu) * rs;
    const float gg = g[e] * uu[e];
    sg += gg;
    sgn += gg * n;
  }
  const float mg = group_sum<L>(sg) / (float)F;
  const float mgn = group_sum<L>(sgn) / (float)F;
  float o_du[8], o_do[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) {
    const float n = (z[e] - mu) * rs;
    o_du[e] = n * g[e];
    o_do[e] = rs * (g[e] * uu[e] - mg - n * mgn);
  }
  const int64_t du_at = r * du_stride + 8 * sub;
  if (du_h) silu_back8(du_h + du_at, o_du);
  Vec8<T>::store(du + du_at, o_du);
  Vec8<T>::store(dO + at, o_do);
  // the attention backward accumulates this token's d_pos partials (8
  // bytes each: a float, or 64-bit fixed point in the deterministic mode)
  if (dpos_part && sub < H) dpos_part[r * H + sub] = 0;
}

template <typename T>
__global__ void __launch_bounds__(LN_THREADS)
ln_fwd_kernel(const T *__restrict__ o, const T *__restrict__ u,
              T *__restrict__ y, float *__restrict__ mean_out,
              float *__restrict__ rstd_out, int64_t T_tokens, int F) {
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)blockIdx.x * LN_WAVES + (threadIdx.x >> 6);
  if (r >= T_tokens) return;
  const T *orow = o + r * F;
  float sum = 0.0f;
  for (int f0 = lane * 8; f0 < F; f0 += 512) {
    float z[8];
    Vec8<T>::load(orow + f0, z);
#pragma unroll
    for (int e = 0; e < 8; ++e) sum += z[e];
  }
  const float mu = wave_sum(sum) / (float)F;
  float sq = 0.0f;
  for (int f0 = lane * 8; f0 < F; f0 += 512) {
    float z[8];
    Vec8<T>::load(orow + f0, z);
#pragma unroll
    for (int e = 0; e < 8; ++e) sq += (z[e] - mu) * (z[e] - mu);
  }
  const float rstd = rsqrtf(wave_sum(sq) / (float)F + HSTU_LN_EPS);
  for (int f0 = lane * 8; f0 < F; f0 += 512) {
    float z[8], uu[8], out[8];
    Vec8<T>::load(orow + f0, z);
    Vec8<T>::load(u + r * F + f0, uu);
#pragma unroll
    for (int e = 0; e < 8; ++e) out[e] = (z[e] - mu) * rstd * uu[e];
    Vec8<T>::store(y + r * F + f0, out);
  }
  if (lane == 0) {
    mean_out[r] = mu;
    rstd_out[r] = rstd;
  }
}

// With `sched` set, the launch's first work-group (dispatched first, so its
// serial phases overlap the rest) builds the backward's work lists
// (sched_impl.h) while the others normalise.
template <typename T>
__global__ void __launch_bounds__(LN_THREADS)
ln_bwd_kernel(const T *__restrict__ dy, const T *__restrict__ u,
              const T *__restrict__ o, const float *__restrict__ mean,
              const float *__restrict__ rstd, T *__restrict__ du,
              T *__restrict__ dO, uint64_t *__restrict__ dpos_part, int H,
              int64_t T_tokens, int F, SchedArgs sa, int sched, int64_t du_stride,
              const T *__restrict__ du_h) {
  if (sched && blockIdx.x == 0) {
    __shared__ SchedSmem ssm;
    build_schedule<LN_THREADS>(sa, ssm, threadIdx.x);
    return;
  }
  // F = 8 x (power of two <= 64): whole tokens per lane group
  switch (F) {
#define HSTU_LN_GROUP(LL)                                                               \
  case 8 * LL:                                                                          \
    ln_bwd_group<T, LL>(dy, u, o, mean, rstd, du, dO, dpos_part, H, T_tokens,            \
                        (int)blockIdx.x - sched, du_stride, du_h);                      \
    return;
    HSTU_LN_GROUP(1) HSTU_LN_GROUP(2) HSTU_LN_GROUP(4) HSTU_LN_GROUP(8)
    HSTU_LN_GROUP(16) HSTU_LN_GROUP(32) HSTU_LN_GROUP(64)
#undef HSTU_LN_GROUP
    default:
      break;
  }
  const int lane = threadIdx.x & 63;
  const int64_t r = (int64_t)(blockIdx.x - sched) * LN_WAVES + (threadIdx.x >> 6);
  if (r >= T_tokens) return;
  const float mu = mean[r], rs = rstd[r];
  const int64_t base = r * F;
  float sg = 0.0f, sgn = 0.0f;
  for (int f0 = lane * 8; f0 < F; f0 += 512) {
    float z[8], g[8], uu[8];
    Vec8<T>::load(o + base + f0, z);
    Vec8<T>::load(dy + base + f0, g);
    Vec8<T>::load(u + base + f0, uu);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float n = (z[e] - mu) * rs;
      const float gg = g[e] * uu[e];
      sg += gg;
      sgn += gg * n;
    }
  }
  const float mg = wave_sum(sg) / (float)F;
  const float mgn = wave_sum(sgn) / (float)F;
  for (int f0 = lane * 8; f0 < F; f0 += 512) {
    float z[8], g[8], uu[8], o_du[8], o_do[8];
    Vec8<T>::load(o + base + f0, z);
    Vec8<T>::load(dy + base + f0, g);
    Vec8<T>::load(u + base + f0, uu);
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const float n = (z[e] - mu) * rs;
      o_du[e] = n * g[e];
      o_do[e] = rs * (g[e] * uu[e] - mg - n * mgn);
    }
    if (du_h) silu_back8(du_h + r * du_stride + f0, o_du);
    Vec8<T>::store(du + r * du_stride + f0, o_du);
    Vec8<T>::store(dO + base + f0, o_do);
  }
  // the attention backward accumulates this token's d_pos partials
  if (dpos_part && lane < H) dpos_part[r * H + lane] = 0;
}

// Table-gradient finalize, one launch with two block roles:
//   d_pos[h, x]: x >= N is unreachable (j > i) and written 0; otherwise the
//     offset m = N-1-x sums the per-sequence partials of every sequence
//     longer than m.  Block = (h, 64 consecutive m); lane = m, waves stride
//     over the sequences, then a cross-wave sum in LDS.
//   d_time[h, k]: sum of the DTIME_BINS partial histograms the dK/dV
//     work-groups folded theirs into.  Block = 64 consecutive (h, k)
//     columns; waves stride over the bins.
// Summation order is fixed, so the result is deterministic given the
// partials.  `scale` multiplies every entry (ln 2 / N: the backward kernel
// accumulates N log2(e) dS).
// The deterministic backward keeps the partials as 64-bit fixed point
// (FIX_ONE per unit); they are summed as integers, which no order changes,
// and converted once.
constexpr int FIN_THREADS = 1024;
constexpr int FIN_WAVES = FIN_THREADS / 64;

template <bool DET> struct FinAcc { typedef float T; };
template <> struct FinAcc<true> { typedef unsigned long long T; };
__device__ __forceinline__ float fin_value(float x) { return x; }
__device__ __forceinline__ float fin_value(unsigned long long x) {
  return (float)((double)(long long)x * (1.0 / FIX_ONE));
}

template <bool DET>
__global__ void __launch_bounds__(FIN_THREADS)
finalize_tables_kernel(const SeqInfo *__restrict__ info, int B,
                       const void *__restrict__ pos_part_v, int H, int N,
                       float *__restrict__ d_pos, int pos_blocks,
                       const void *__restrict__ time_part_v, int n_parts,
                       int width, float *__restrict__ d_time, float scale) {
  typedef typename FinAcc<DET>::T A;
  const A *pos_part = (const A *)pos_part_v;
  const A *time_part = (const A *)time_part_v;
  __shared__ A red[FIN_WAVES][64];
  const int lane = threadIdx.x & 63, wv = threadIdx.x >> 6;
  A acc = 0;
  if ((int)blockIdx.x < pos_blocks) {
    const int chunks = (N + 63) / 64;
    const int h = blockIdx.x / chunks;
    const int m = (blockIdx.x % chunks) * 64 + lane;
    if (m < N) {
      // eight sequences per step: their records, then their partials, each
      // group of loads issued together (two memory latencies per step)
      constexpr int G = 8;
      A part[G];
#pragma unroll
      for (int k = 0; k < G; ++k) part[k] = 0;
      int b = wv;
      for (; b + (G - 1) * FIN_WAVES < B; b += G * FIN_WAVES) {
        SeqInfo si[G];
#pragma unroll
        for (int k = 0; k < G; ++k) si[k] = info[b + k * FIN_WAVES];
#pragma unroll
        for (int k = 0; k < G; ++k)
          part[k] += si[k].len > m ? pos_part[(si[k].start + m) * H + h] : (A)0;
      }
      for (; b < B; b += FIN_WAVES) {
        const SeqInfo si = info[b];
        if (si.len > m) acc += pos_part[(si.start + m) * H + h];
      }
#pragma unroll
      for (int k = 0; k < G; ++k) acc += part[k];
    }
    red[wv][lane] = acc;
    __syncthreads();
    if (wv == 0 && m < N) {
      A s = 0;
      for (int x = 0; x < FIN_WAVES; ++x) s += red[x][lane];
      const int64_t span = 2 * (int64_t)N - 1;
      d_pos[h * span + (N - 1 - m)] = scale * fin_value(s);
      if (N + m < span) d_pos[h * span + N + m] = 0.0f;
    }
  } else {
    const int c = ((int)blockIdx.x - pos_blocks) * 64 + lane;
    if (c < width)
      for (int g = wv; g < n_parts; g += FIN_WAVES) acc += time_part[(int64_t)g * width + c];
    red[wv][lane] = acc;
    __syncthreads();
    if (wv == 0 && c < width) {
      A s = 0;
      for (int x = 0; x < FIN_WAVES; ++x) s += red[x][lane];
      d_time[c] = scale * fin_value(s);
    }
  }
}

}  // namespace

// Lanes per token of the fast path (F = 8 L, L a power of two <= 64), else 0.
static int ln_group_lanes(int F) {
  if (F % 8 != 0 || F > 512) return 0;
  const int L = F / 8;
  return (L & (L - 1)) == 0 ? L : 0;
}

// Work-groups covering T tokens, LN_WAVES waves of `tpw` tokens each.
static unsigned ln_blocks(int64_t T, int tpw) {
  const int64_t per = (int64_t)LN_WAVES * tpw;
  return (unsigned)((T + per - 1) / per);
}

template <typename T>
hipError_t launch_ln_fwd_t(const Problem &p, const T *o, const T *u, T *y, float *mean,
                           float *rstd, hipStream_t s) {
  const int F = p.H * p.d;
  const int L = ln_group_lanes(F);
  switch (L) {
#define HSTU_LN_GROUP(LL)                                                               \
  case LL:                                                                              \
    hipLaunchKernelGGL((ln_fwd_group_kernel<T, LL>), dim3(ln_blocks(p.T, 64 / LL)),      \
                       dim3(LN_THREADS), 0, s, o, u, y, mean, rstd, p.T);               \
    return hipGetLastError();
    HSTU_LN_GROUP(1) HSTU_LN_GROUP(2) HSTU_LN_GROUP(4) HSTU_LN_GROUP(8)
    HSTU_LN_GROUP(16) HSTU_LN_GROUP(32) HSTU_LN_GROUP(64)
#undef HSTU_LN_GROUP
    default:
      break;
  }
  hipLaunchKernelGGL(ln_fwd_kernel<T>, dim3(ln_blocks(p.T, 1)), dim3(LN_THREADS), 0, s, o, u,
                     y, mean, rstd, p.T, F);
  return hipGetLastError();
}

hipError_t launch_ln_fwd(const Problem &p, const void *o, const void *u,
                         void *y, float *mean, float *rstd, hipStream_t s) {
  if (p.dtype == HSTU_BF16)
    return launch_ln_fwd_t<u16>(p, (const u16 *)o, (const u16 *)u, (u16 *)y, mean, rstd, s);
  return launch_ln_fwd_t<float>(p, (const float *)o, (const float *)u, (float *)y, mean, rstd,
                                s);
}

hipError_t launch_ln_bwd_sched(const Problem &p, const void *dy, const void *u,
                               const void *o, const float *mean, const float *rstd,
                               void *du, void *dO, void *dpos_part_v,
                               const int64_t *seq_offsets, void *ws, const Layout &L,
                               const GradOut *go, hipStream_t s) {
  uint64_t *dpos_part = (uint64_t *)dpos_part_v;
  const int F = p.H * p.d;
  const SchedArgs sa = sched_args(seq_offsets, p, ws, L);
  const int GL = ln_group_lanes(F);
  const dim3 grid(ln_blocks(p.T, GL ? 64 / GL : 1) + 1);
  if (p.dtype == HSTU_BF16)
    hipLaunchKernelGGL(ln_bwd_kernel<u16>, grid, dim3(LN_THREADS), 0, s,
                       (const u16 *)dy, (const u16 *)u, (const u16 *)o, mean, rstd,
                       (u16 *)du, (u16 *)dO, dpos_part, p.H, p.T, F, sa, 1,
                       go ? go->stride : (int64_t)F, go ? (const u16 *)go->h_du : nullptr);
  else
    hipLaunchKernelGGL(ln_bwd_kernel<float>, grid, dim3(LN_THREADS), 0, s,
                       (const float *)dy, (const float *)u, (const float *)o, mean, rstd,
                       (float *)du, (float *)dO, dpos_part, p.H, p.T, F, sa, 1, (int64_t)F,
                       (const float *)nullptr);
  return hipGetLastError();
}

hipError_t launch_finalize_tables(const AttnArgs &a, float *d_pos,
                                  float *d_time, hipStream_t s) {
  const char *ws = (const char *)a.ws;
  const Problem &p = a.p;
  const int pos_blocks = d_pos ? p.H * ((p.N + 63) / 64) : 0;
  const int width = d_time ? p.H * p.nb : 0;
  const int time_blocks = (width + 63) / 64;
  if (pos_blocks + time_blocks == 0) return hipSuccess;
  auto kfn = p.deterministic ? finalize_tables_kernel<true> : finalize_tables_kernel<false>;
  hipLaunchKernelGGL(kfn, dim3(pos_blocks + time_blocks),
                     dim3(FIN_THREADS), 0, s, (const SeqInfo *)(ws + a.L.seqinfo), p.B,
                     d_pos ? (const void *)(ws + a.L.dpos_part) : nullptr, p.H, p.N,
                     d_pos, pos_blocks,
                     d_time ? (const void *)(ws + a.L.dtime_part) : nullptr,
                     DTIME_BINS, width, d_time, (float)(TABLE_UNIT / p.N));
  return hipGetLastError();
}

}  // namespace hstu
