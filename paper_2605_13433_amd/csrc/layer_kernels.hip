// Pointwise kernels of the HSTU layer shell: the SiLU + column split that
// turns f1's output into the attention's U, V, Q, K planes (for f1 shapes
// the fused GEMM does not tile), the sum of split-K partial products, and a
// zero fill.
//
// The split is a pure streaming pass (HBM-bound): each thread moves
// 16-byte chunks of eight bf16, a chunk never straddles two planes (the
// plane width H*d is a multiple of 64), and consecutive threads touch
// consecutive chunks of both the [T][4C] matrix and a plane row, so loads
// and stores are fully coalesced.
#include <algorithm>

#include "internal.h"
#include "device.h"

namespace hstu {

namespace {

constexpr int PW_THREADS = 256;

__device__ __forceinline__ void unpack8(uint4 v, float f[8]) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    f[2 * i] = __uint_as_float(w[i] << 16);
    f[2 * i + 1] = __uint_as_float(w[i] & 0xffff0000u);
  }
}

__device__ __forceinline__ uint4 pack8(const float f[8]) {
  uint4 r;
  r.x = pack2(f[0], f[1]);
  r.y = pack2(f[2], f[3]);
  r.z = pack2(f[4], f[5]);
  r.w = pack2(f[6], f[7]);
  return r;
}

// z[p][t][c] = silu(h[t][p*C + c]) for p in 0..3 (planes U, V, Q, K).
// `chunks` = T * 4C / 8; `row_chunks` = 4C / 8; `plane_chunks` = C / 8.
__global__ void __launch_bounds__(PW_THREADS)
silu_split_kernel(const uint4 *__restrict__ h, uint4 *__restrict__ z,
                  int64_t chunks, int32_t row_chunks, int32_t plane_chunks,
                  int64_t plane_stride_chunks) {
  const int64_t stride = (int64_t)gridDim.x * PW_THREADS;
  for (int64_t x = (int64_t)blockIdx.x * PW_THREADS + threadIdx.x; x < chunks;
       x += stride) {
    const int64_t t = x / row_chunks;
    const int32_t cc = (int32_t)(x - t * row_chunks);
    const int32_t p = cc / plane_chunks;
    const int32_t c = cc - p * plane_chunks;
    float f[8];
    unpack8(h[x], f);
#pragma unroll
    for (int i = 0; i < 8; ++i) f[i] = silu_f(f[i]);
    z[p * plane_stride_chunks + t * plane_chunks + c] = pack8(f);
  }
}

// out[x] = bf16(sum_{s < parts} part[s][x]) for x < n (n % 4 == 0), summed
// in the order s = 0, 1, ...
__global__ void __launch_bounds__(PW_THREADS)
sum_parts_kernel(const float4 *__restrict__ part, uint2 *__restrict__ out, int64_t n4,
                 int32_t parts) {
  const int64_t stride = (int64_t)gridDim.x * PW_THREADS;
  for (int64_t x = (int64_t)blockIdx.x * PW_THREADS + threadIdx.x; x < n4; x += stride) {
    float4 a = part[x];
    for (int32_t p = 1; p < parts; ++p) {
      const float4 b = part[(int64_t)p * n4 + x];
      a.x += b.x; a.y += b.y; a.z += b.z; a.w += b.w;
    }
    out[x] = make_uint2(pack2(a.x, a.y), pack2(a.z, a.w));
  }
}

__global__ void __launch_bounds__(PW_THREADS)
zero_kernel(uint32_t *__restrict__ p, int64_t words) {
  const int64_t stride = (int64_t)gridDim.x * PW_THREADS;
  for (int64_t x = (int64_t)blockIdx.x * PW_THREADS + threadIdx.x; x < words;
       x += stride)
    p[x] = 0u;
}

int pw_grid(int64_t chunks, int dev) {
  // Enough resident waves to cover HBM latency; the loops stride the rest.
  const int64_t want = (chunks + PW_THREADS - 1) / PW_THREADS;
  const int64_t cap = (int64_t)device_info(dev).num_cu * 8;
  return (int)std::max<int64_t>(1, std::min<int64_t>(want, cap));
}

}  // namespace

hipError_t launch_silu_split(const void *h, void *z, int64_t T, int32_t C,
                             int dev, hipStream_t s) {
  const int64_t chunks = T * 4 * (int64_t)C / 8;
  if (chunks == 0) return hipSuccess;
  hipLaunchKernelGGL(silu_split_kernel, dim3(pw_grid(chunks, dev)),
                     dim3(PW_THREADS), 0, s, (const uint4 *)h, (uint4 *)z,
                     chunks, 4 * C / 8, C / 8, T * (int64_t)C / 8);
  return hipGetLastError();
}

hipError_t launch_sum_parts(const float *part, void *out, int64_t n, int32_t parts, int dev,
                            hipStream_t s) {
  const int64_t n4 = n / 4;
  if (n4 == 0) return hipSuccess;
  hipLaunchKernelGGL(sum_parts_kernel, dim3(pw_grid(n4, dev)), dim3(PW_THREADS), 0, s,
                     (const float4 *)part, (uint2 *)out, n4, parts);
  return hipGetLastError();
}

hipError_t launch_zero(void *p, size_t bytes, int dev, hipStream_t s) {
  const int64_t words = (int64_t)(bytes / 4);
  if (words == 0) return hipSuccess;
  hipLaunchKernelGGL(zero_kernel, dim3(pw_grid(words, dev)), dim3(PW_THREADS),
                     0, s, (uint32_t *)p, words);
  return hipGetLastError();
}

}  // namespace hstu
