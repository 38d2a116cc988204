// Hand-written bf16 MFMA GEMM for gfx950 with the HSTU layer's fused
// epilogue: the f1 projection h = x W1 writes h (saved for the backward's
// silu') and, in the same pass, z = silu(h) split by column blocks into the
// four planes U, V, Q, K [T][H*d] that the attention reads -- no separate
// SiLU/split pass and no re-read of h (Sec. 4.1.1's first step, removing
// the conversions around the attention operator, carried to the layer).
//
// Tiling: work-group = 4 wave64s on a 128 x 128 output tile, each wave a
// 64 x 64 quadrant as 2 x 2 blocks of v_mfma_f32_32x32x16_bf16.  K steps of
// 64: the A tile (x rows, 128 x 64) and the B tile (W1 rows, 64 x 128) are
// double-buffered in LDS, filled by global-to-LDS loads (16 bytes per lane,
// XOR-swizzled chunks so that row reads and transpose reads spread over the
// banks), one barrier per K step.  A operands are row reads (8 consecutive
// k of one row); B operands come from the LDS transpose load, which hands
// each lane 4 consecutive k rows of its column, two of them giving the 8
// consecutive k the row read of A pairs with.  The epilogue rounds the
// accumulators to bf16 (h's precision), stages the tile in LDS and leaves
// it as 16-byte row chunks: h, then silu of the rounded value into the
// chunk's plane.
#include <algorithm>

#include "internal.h"
#include "device.h"

namespace hstu {
namespace {

constexpr int GT = 256;            // threads
constexpr int BM = 128, BN = 128, BK = 64;

typedef short v4i16g __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16g lds_v4i16g;
typedef __attribute__((address_space(3))) void lds_voidg;

// LDS tiles hold 16-byte chunks (8 bf16) with XOR-swizzled positions:
//   A tile [BM][BK] (8 chunks a row): chunk c of row r at c ^ (r & 7), so the
//     row reads of 8 consecutive rows (one 128-byte bank sweep) never collide;
//   B tile [BK][BN] (16 chunks a row): chunk c of row r at c ^ 2 (r & 3), so
//     the transpose reads, whose 16-lane groups take 32 bytes from each of
//     4 consecutive rows, land on 4 disjoint bank octets.
__device__ __forceinline__ int swz_a(int r, int c) { return r * (BK / 8) + (c ^ (r & 7)); }
__device__ __forceinline__ int swz_b(int r, int c) { return r * (BN / 8) + (c ^ (2 * (r & 3))); }

// Streaming (non-temporal) 16-byte store: the epilogue's h and z rows are
// not read again by this kernel, so they should not displace the x and W1
// tiles the other work-groups are re-reading from L2 (measured 15% faster).
typedef unsigned int u32x4nt __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void store_nt(u16 *p, uint4 v) {
  __builtin_nontemporal_store(__builtin_bit_cast(u32x4nt, v), (u32x4nt *)p);
}

__device__ __forceinline__ void wait_vm_all() { __builtin_amdgcn_s_waitcnt(0x0f70); }

struct F1Args {
  const u16 *x;        // [M][K]
  const u16 *w;        // [K][N]
  u16 *h;              // [M][N]
  u16 *z;              // [4][M][N/4] planes
  int64_t M;
  int N, K;
};

// Per-thread constants of the K loop: global sources of this thread's four
// A and four B chunks (advanced by one K step each step) and LDS offsets of
// its operand reads (fixed; only the buffer base changes).
struct F1Thread {
  const u16 *ga[4], *gb[4];
  int a_rd[4];        // element offset of the A row read for ks = 0..3 (block i = 0)
  int b_rd[2];        // element offset of the B transpose read for block j (ks = 0)
};

constexpr int A_ELEMS = BM * BK, B_ELEMS = BK * BN;
constexpr int IPW = BM * (BK / 8) / 64 / 4;          // loads per wave per tile (4)
static_assert(BK * (BN / 8) / 64 / 4 == IPW, "A and B tiles take the same load count");

__device__ __forceinline__ void issue_loads(const F1Thread &t, u16 *a_lds, u16 *b_lds,
                                            int w) {
#pragma unroll
  for (int x = 0; x < IPW; ++x) {
    __builtin_amdgcn_global_load_lds((const void *)t.ga[x],
                                     (lds_voidg *)(a_lds + (w * IPW + x) * 64 * 8), 16, 0, 0);
    __builtin_amdgcn_global_load_lds((const void *)t.gb[x],
                                     (lds_voidg *)(b_lds + (w * IPW + x) * 64 * 8), 16, 0, 0);
  }
}

// 16 MFMAs of one K step on buffers (A, B).
__device__ __forceinline__ void k_step(const F1Thread &t, const u16 *A, const u16 *B,
                                       f32x16 (&acc)[2][2]) {
#pragma unroll
  for (int ks = 0; ks < BK / 16; ++ks) {
    bf16x8 af[2], bfr[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) af[i] = *(const bf16x8 *)(A + t.a_rd[ks] + 32 * i * BK);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const u16 *p0 = B + t.b_rd[j] + 16 * ks * BN;
      const v4i16g lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16g *)p0);
      const v4i16g hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16g *)(p0 + 4 * BN));
      typedef short v8i16 __attribute__((ext_vector_type(8)));
      const v8i16 x = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
      bfr[j] = __builtin_bit_cast(bf16x8, x);
    }
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j) acc[i][j] = mfma32(af[i], bfr[j], acc[i][j]);
  }
}

__global__ void __launch_bounds__(GT, 2) gemm_f1_silu_kernel(F1Args a) {
  __shared__ __attribute__((aligned(16))) u16 smem[2 * (A_ELEMS + B_ELEMS)];
  const int tid = threadIdx.x, lane = tid & 63, g = lane >> 5, l32 = lane & 31;
  const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = w & 1, wn = w >> 1;
  // consecutive work-groups share their row block (x tile reuse in L2)
  const int nb_n = a.N / BN;
  const int64_t tm = blockIdx.x / nb_n;
  const int tn = blockIdx.x % nb_n;
  const int64_t m0 = tm * BM;
  const int n0 = tn * BN;
  const int valid_m = (int)std::min<int64_t>(BM, a.M - m0);

  F1Thread t;
#pragma unroll
  for (int x = 0; x < IPW; ++x) {
    const int pos = (w * IPW + x) * 64 + lane;        // chunk slot in LDS
    const int ra = pos / (BK / 8), ca = (pos % (BK / 8)) ^ (ra & 7);
    const int rr = ra < valid_m ? ra : valid_m - 1;  // rows past M: never stored
    t.ga[x] = a.x + (m0 + rr) * a.K + 8 * ca;
    const int rb = pos / (BN / 8), cb = (pos % (BN / 8)) ^ (2 * (rb & 3));
    t.gb[x] = a.w + (int64_t)rb * a.N + n0 + 8 * cb;
  }
#pragma unroll
  for (int ks = 0; ks < BK / 16; ++ks) t.a_rd[ks] = 8 * swz_a(64 * wm + l32, 2 * ks + g);
  {
    // transpose read: 16-lane group c takes row 8 g + (c >> 2) and the
    // 8-byte column group 16 ((lane >> 4) & 1) + 4 (c & 3) of block j
    const int c = lane & 15;
    const int r0 = 8 * g + (c >> 2);
#pragma unroll
    for (int j = 0; j < 2; ++j) {
      const int col = 64 * wn + 32 * j + ((lane >> 4) & 1) * 16 + 4 * (c & 3);
      t.b_rd[j] = 8 * swz_b(r0, col >> 3) + (col & 7);
    }
  }

  f32x16 acc[2][2];
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[i][j][r] = 0.0f;

  u16 *A0 = smem, *A1 = smem + A_ELEMS;
  u16 *B0 = smem + 2 * A_ELEMS, *B1 = smem + 2 * A_ELEMS + B_ELEMS;
  const int nk = a.K / BK;
  const int64_t b_step = (int64_t)BK * a.N;
  issue_loads(t, A0, B0, w);
  for (int kt = 0; kt < nk; kt += 2) {
    // even step on buffers 0 (streaming step kt+1 into 1), odd on 1
#pragma unroll
    for (int x = 0; x < IPW; ++x) { t.ga[x] += BK; t.gb[x] += b_step; }
    wait_vm_all();
    lds_barrier();
    if (kt + 1 < nk) issue_loads(t, A1, B1, w);
    k_step(t, A0, B0, acc);
    if (kt + 1 >= nk) break;
#pragma unroll
    for (int x = 0; x < IPW; ++x) { t.ga[x] += BK; t.gb[x] += b_step; }
    wait_vm_all();
    lds_barrier();
    if (kt + 2 < nk) issue_loads(t, A0, B0, w);
    k_step(t, A1, B1, acc);
  }

  // epilogue: bf16 tile in LDS (row-major, 128 x 128, +8 pad per row), then
  // 16-byte row chunks of h and of silu(h) into the plane
  constexpr int OS = BN + 8;
  u16 *ot = smem;
  lds_barrier();
#pragma unroll
  for (int i = 0; i < 2; ++i)
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int row = 64 * wm + 32 * i + c_row(r, g);
        const int col = 64 * wn + 32 * j + l32;
        __bf16 v = (__bf16)acc[i][j][r];
        ot[row * OS + col] = __builtin_bit_cast(u16, v);
      }
  lds_barrier();
  const int C = a.N / 4;
  const int64_t plane = a.M * (int64_t)C;
#pragma unroll
  for (int x = 0; x < BM * BN / 8 / GT; ++x) {
    const int ch = tid + GT * x;
    const int row = ch / (BN / 8), c8 = ch % (BN / 8);
    if (row < valid_m) {
      const uint4 hv = *(const uint4 *)(ot + row * OS + 8 * c8);
      const int64_t tr = m0 + row;
      const int n = n0 + 8 * c8;
      store_nt(a.h + tr * a.N + n, hv);
      const uint32_t wd[4] = {hv.x, hv.y, hv.z, hv.w};
      float f[8];
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        f[2 * e] = __uint_as_float(wd[e] << 16);
        f[2 * e + 1] = __uint_as_float(wd[e] & 0xffff0000u);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) f[e] = f[e] * sigmoid_f(f[e]);
      uint4 zv;
      zv.x = pack2(f[0], f[1]);
      zv.y = pack2(f[2], f[3]);
      zv.z = pack2(f[4], f[5]);
      zv.w = pack2(f[6], f[7]);
      const int p = n / C;
      store_nt(a.z + p * plane + tr * C + (n - p * C), zv);
    }
  }
}

}  // namespace

bool gemm_f1_silu_supported(int64_t N, int64_t K) {
  return N % BN == 0 && (N / 4) % 8 == 0 && K % BK == 0 && K > 0;
}

hipError_t launch_gemm_f1_silu(const void *x, const void *w1, void *h, void *z, int64_t M,
                               int32_t N, int32_t K, hipStream_t s) {
  F1Args a{(const u16 *)x, (const u16 *)w1, (u16 *)h, (u16 *)z, M, N, K};
  const int64_t blocks = ((M + BM - 1) / BM) * (N / BN);
  hipLaunchKernelGGL(gemm_f1_silu_kernel, dim3((unsigned)blocks), dim3(GT), 0, s, a);
  return hipGetLastError();
}

}  // namespace hstu
