// float32 jagged HSTU attention (forward and backward) on the vector ALUs.
//
// Same definition as the bf16 MFMA kernels, all arithmetic in fp32.  One
// work-group of 64 threads per (work-list entry, head); each thread owns one
// row of the 64-row tile (a query for the forward and dQ, a key for dK/dV)
// and walks its causal partners; every thread of a wave reads the same
// partner row at the same time, so those loads are broadcasts.  Table
// gradients are float atomics straight into the (zeroed) outputs, or, in the
// deterministic mode, 64-bit fixed-point atomics into workspace tables that a
// last pass converts (integer sums do not depend on order).  This path
// serves the fp32 workload and precision checks; it is not the throughput
// path.
#include "internal.h"
#include "device.h"

namespace hstu {

namespace {

constexpr int F32_THREADS = TILE;

struct F32Params {
  const float *q, *k, *v, *dO;
  const float *pos_w, *time_w;
  const int64_t *ts;
  const int32_t *ctrl;
  const SeqInfo *info;
  const WorkEntry *list;
  float *out0, *out1, *out2;
  // table-gradient sums in the workspace: double (default mode; many
  // thousands of terms land on one entry, more than float keeps to 1e-5 of
  // the table) or 64-bit fixed point (deterministic mode)
  double *acc_pos, *acc_time;
  unsigned long long *fix_pos, *fix_time;
  int32_t H, N, nb;
  float inv_n, alpha;
};

__device__ __forceinline__ float bias(const F32Params &P, int h, int64_t i,
                                      int64_t j, int64_t ri, int64_t rj) {
  float b = 0.0f;
  if (P.pos_w) b += P.pos_w[(int64_t)h * (2 * (int64_t)P.N - 1) + (j - i + P.N - 1)];
  if (P.time_w) b += P.time_w[(int64_t)h * P.nb + time_bucket(P.ts[ri] - P.ts[rj], P.nb)];
  return b;
}

template <int D>
__global__ void __launch_bounds__(F32_THREADS)
f32_fwd_kernel(F32Params P) {
  const int entry = blockIdx.x / P.H, h = blockIdx.x % P.H;
  if (entry >= P.ctrl[CTRL_N_ENTRIES]) return;
  const WorkEntry e = P.list[entry];
  const SeqInfo si = P.info[e.seq];
  const int64_t i = (int64_t)e.tile * TILE + threadIdx.x;
  if (i >= si.len) return;
  const int64_t ri = si.start + i;
  float qi[D], acc[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    qi[c] = P.q[(ri * P.H + h) * D + c];
    acc[c] = 0.0f;
  }
  for (int64_t j = 0; j <= i; ++j) {
    const int64_t rj = si.start + j;
    const float *kj = P.k + (rj * P.H + h) * D;
    const float *vj = P.v + (rj * P.H + h) * D;
    float s = 0.0f;
#pragma unroll
    for (int c = 0; c < D; ++c) s = fmaf(qi[c], kj[c], s);
    s = P.alpha * s + bias(P, h, i, j, ri, rj);
    const float a = s * sigmoid_f(s) * P.inv_n;
#pragma unroll
    for (int c = 0; c < D; ++c) acc[c] = fmaf(a, vj[c], acc[c]);
  }
#pragma unroll
  for (int c = 0; c < D; ++c) P.out0[(ri * P.H + h) * D + c] = acc[c];
}

template <int D>
__global__ void __launch_bounds__(F32_THREADS)
f32_dq_kernel(F32Params P) {
  const int entry = blockIdx.x / P.H, h = blockIdx.x % P.H;
  if (entry >= P.ctrl[CTRL_N_ENTRIES]) return;
  const WorkEntry e = P.list[entry];
  const SeqInfo si = P.info[e.seq];
  const int64_t i = (int64_t)e.tile * TILE + threadIdx.x;
  if (i >= si.len) return;
  const int64_t ri = si.start + i;
  float qi[D], doi[D], acc[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    qi[c] = P.q[(ri * P.H + h) * D + c];
    doi[c] = P.dO[(ri * P.H + h) * D + c];
    acc[c] = 0.0f;
  }
  for (int64_t j = 0; j <= i; ++j) {
    const int64_t rj = si.start + j;
    const float *kj = P.k + (rj * P.H + h) * D;
    const float *vj = P.v + (rj * P.H + h) * D;
    float s = 0.0f, da = 0.0f;
#pragma unroll
    for (int c = 0; c < D; ++c) {
      s = fmaf(qi[c], kj[c], s);
      da = fmaf(doi[c], vj[c], da);
    }
    s = P.alpha * s + bias(P, h, i, j, ri, rj);
    const float sg = sigmoid_f(s);
    const float ds = da * sg * (1.0f + s * (1.0f - sg)) * P.inv_n;
#pragma unroll
    for (int c = 0; c < D; ++c) acc[c] = fmaf(ds, kj[c], acc[c]);
  }
#pragma unroll
  for (int c = 0; c < D; ++c) P.out0[(ri * P.H + h) * D + c] = P.alpha * acc[c];
}

template <int D>
__global__ void __launch_bounds__(F32_THREADS)
f32_dkv_kernel(F32Params P) {
  const int entry = blockIdx.x / P.H, h = blockIdx.x % P.H;
  if (entry >= P.ctrl[CTRL_N_ENTRIES]) return;
  const WorkEntry e = P.list[entry];
  const SeqInfo si = P.info[e.seq];
  const int64_t j = (int64_t)e.tile * TILE + threadIdx.x;
  if (j >= si.len) return;
  const int64_t rj = si.start + j;
  float kj[D], vj[D], dk[D], dv[D];
#pragma unroll
  for (int c = 0; c < D; ++c) {
    kj[c] = P.k[(rj * P.H + h) * D + c];
    vj[c] = P.v[(rj * P.H + h) * D + c];
    dk[c] = 0.0f;
    dv[c] = 0.0f;
  }
  for (int64_t i = j; i < si.len; ++i) {
    const int64_t ri = si.start + i;
    const float *qi = P.q + (ri * P.H + h) * D;
    const float *doi = P.dO + (ri * P.H + h) * D;
    float s = 0.0f, da = 0.0f;
#pragma unroll
    for (int c = 0; c < D; ++c) {
      s = fmaf(qi[c], kj[c], s);
      da = fmaf(doi[c], vj[c], da);
    }
    s = P.alpha * s + bias(P, h, i, j, ri, rj);
    const float sg = sigmoid_f(s);
    const float a = s * sg * P.inv_n;
    const float ds = da * sg * (1.0f + s * (1.0f - sg)) * P.inv_n;
#pragma unroll
    for (int c = 0; c < D; ++c) {
      dv[c] = fmaf(a, doi[c], dv[c]);
      dk[c] = fmaf(ds, qi[c], dk[c]);
    }
    const int64_t xp = (int64_t)h * (2 * (int64_t)P.N - 1) + (j - i + P.N - 1);
    if (P.acc_pos) atomicAdd(&P.acc_pos[xp], (double)ds);
    if (P.fix_pos) atomicAdd(&P.fix_pos[xp], to_fix(ds));
    if (P.acc_time || P.fix_time) {
      const int64_t xt = (int64_t)h * P.nb + time_bucket(P.ts[ri] - P.ts[rj], P.nb);
      if (P.acc_time) atomicAdd(&P.acc_time[xt], (double)ds);
      if (P.fix_time) atomicAdd(&P.fix_time[xt], to_fix(ds));
    }
  }
#pragma unroll
  for (int c = 0; c < D; ++c) {
    P.out1[(rj * P.H + h) * D + c] = P.alpha * dk[c];
    P.out2[(rj * P.H + h) * D + c] = dv[c];
  }
}

__global__ void fill_zero_kernel(float *p, int64_t n) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n;
       x += (int64_t)gridDim.x * blockDim.x)
    p[x] = 0.0f;
}

// Double table sums -> float tables.
__global__ void double_to_float_kernel(const double *acc, float *out, int64_t n) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n;
       x += (int64_t)gridDim.x * blockDim.x)
    out[x] = (float)acc[x];
}

// Fixed-point table sums -> float tables.
__global__ void fix_to_float_kernel(const unsigned long long *fix, float *out, int64_t n) {
  for (int64_t x = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; x < n;
       x += (int64_t)gridDim.x * blockDim.x)
    out[x] = (float)((double)(long long)fix[x] * (1.0 / FIX_ONE));
}

F32Params make_params(const AttnArgs &a, const WorkEntry *list) {
  const char *ws = (const char *)a.ws;
  F32Params P{};
  P.q = (const float *)a.q;
  P.k = (const float *)a.k;
  P.v = (const float *)a.v;
  P.pos_w = a.pos_w;
  P.time_w = a.time_w;
  P.ts = a.ts;
  P.ctrl = (const int32_t *)(ws + a.L.ctrl);
  P.info = (const SeqInfo *)(ws + a.L.seqinfo);
  P.list = list;
  P.H = a.p.H;
  P.N = a.p.N;
  P.nb = a.p.has_time ? a.p.nb : 0;
  P.inv_n = 1.0f / (float)a.p.N;
  P.alpha = a.p.alpha;
  return P;
}

#define HSTU_F32_DISPATCH(NAME, D, GRID, S, P)                                       \
  do {                                                                              \
    if (D == 32) hipLaunchKernelGGL(NAME<32>, GRID, dim3(F32_THREADS), 0, S, P);     \
    else if (D == 64) hipLaunchKernelGGL(NAME<64>, GRID, dim3(F32_THREADS), 0, S, P); \
    else hipLaunchKernelGGL(NAME<128>, GRID, dim3(F32_THREADS), 0, S, P);            \
  } while (0)

}  // namespace

hipError_t launch_attn_fwd_f32(const AttnArgs &a, void *o, hipStream_t s) {
  const char *ws = (const char *)a.ws;
  F32Params P = make_params(a, (const WorkEntry *)(ws + a.L.list_q));
  P.out0 = (float *)o;
  const dim3 grid((unsigned)(a.p.max_entries * a.p.H));
  HSTU_F32_DISPATCH(f32_fwd_kernel, a.p.d, grid, s, P);
  return hipGetLastError();
}

hipError_t launch_attn_bwd_f32(const AttnArgs &a, const void *dO, void *dq,
                               void *dk, void *dv, float *d_pos, float *d_time,
                               hipStream_t s) {
  const char *ws = (const char *)a.ws;
  const Problem &p = a.p;
  const int64_t n_pos = (int64_t)p.H * (2 * (int64_t)p.N - 1), n_time = (int64_t)p.H * p.nb;
  // table-shaped staging sums in the workspace (8 bytes per entry): 64-bit
  // fixed point in the deterministic mode, double otherwise; converted to
  // the float tables after the dK/dV kernel (zeros when T = 0)
  void *st_pos = d_pos ? (void *)(ws + a.L.dpos_part) : nullptr;
  void *st_time = d_time ? (void *)(ws + a.L.dtime_part) : nullptr;
  if (st_pos)
    hipLaunchKernelGGL(fill_zero_kernel, dim3(64), dim3(256), 0, s, (float *)st_pos, 2 * n_pos);
  if (st_time)
    hipLaunchKernelGGL(fill_zero_kernel, dim3(8), dim3(256), 0, s, (float *)st_time, 2 * n_time);
  unsigned long long *fix_pos = p.deterministic ? (unsigned long long *)st_pos : nullptr;
  unsigned long long *fix_time = p.deterministic ? (unsigned long long *)st_time : nullptr;
  double *acc_pos = p.deterministic ? nullptr : (double *)st_pos;
  double *acc_time = p.deterministic ? nullptr : (double *)st_time;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return e;
  if (p.T > 0) {
  const dim3 grid((unsigned)(p.max_entries * p.H));
  F32Params P = make_params(a, (const WorkEntry *)(ws + a.L.list_q));
  P.dO = (const float *)dO;
  P.out0 = (float *)dq;
  HSTU_F32_DISPATCH(f32_dq_kernel, p.d, grid, s, P);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  F32Params K = make_params(a, (const WorkEntry *)(ws + a.L.list_k));
  K.dO = (const float *)dO;
  K.out1 = (float *)dk;
  K.out2 = (float *)dv;
  K.acc_pos = acc_pos;
  K.acc_time = acc_time;
  K.fix_pos = fix_pos;
  K.fix_time = fix_time;
  HSTU_F32_DISPATCH(f32_dkv_kernel, p.d, grid, s, K);
  if ((e = hipGetLastError()) != hipSuccess) return e;
  }
  if (fix_pos)
    hipLaunchKernelGGL(fix_to_float_kernel, dim3(64), dim3(256), 0, s, fix_pos, d_pos, n_pos);
  if (fix_time)
    hipLaunchKernelGGL(fix_to_float_kernel, dim3(8), dim3(256), 0, s, fix_time, d_time, n_time);
  if (acc_pos)
    hipLaunchKernelGGL(double_to_float_kernel, dim3(64), dim3(256), 0, s, acc_pos, d_pos, n_pos);
  if (acc_time)
    hipLaunchKernelGGL(double_to_float_kernel, dim3(8), dim3(256), 0, s, acc_time, d_time,
                       n_time);
  return hipGetLastError();
}

}  // namespace hstu
