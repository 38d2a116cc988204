// bf16 MFMA kernels of jagged HSTU attention for gfx950 (Sec. 3.1.1: jagged
// QKV with the relative position and relative time biases fused into the
// attention kernel, no padding and no dense<->jagged conversion).
//
// Three persistent kernels pop (sequence, 64-row tile, head) items from the
// scheduler's longest-first lists:
//
//   attn_fwd   q-stationary: O_i = sum_{j<=i} silu(s_ij)/N v_j
//   attn_dq    q-stationary: dQ_i = sum_{j<=i} dS_ij k_j
//   attn_dkv   k-stationary: dV_j = sum_{i>=j} a_ij dO_i,
//                            dK_j = sum_{i>=j} dS_ij q_i, plus the table
//                            gradients (per-sequence diagonal partials for
//                            d_pos, per-work-group histograms for d_time)
//
// with s_ij = <q_i,k_j> + pos_w[h, j-i+N-1] + time_w[h, bucket(ts_i-ts_j)],
// dS_ij = <dO_i, v_j> silu'(s_ij) / N, and the causal mask applied after the
// SiLU (a masked pair is exactly zero).
//
// Work-group = 4 wave64s on a 64x64 tile pair; each wave owns a 32x32
// quadrant (half of the stationary rows x half of the streamed rows) and all
// contractions use the 32x32x16 bf16 MFMA.  The stationary operand lives in
// registers.  The streamed tile is staged in LDS once, row-major: the
// score-side products read it along d with 16-byte loads, the accumulating
// products (contracted over tile rows) read it through the gfx950 LDS
// transpose load, which hands each lane one column of 4 consecutive rows.
// Score accumulators come out with one fixed stationary row per lane, which
// is exactly the operand layout of the accumulating product, so scores
// never leave registers.  The two halves of the streamed side are summed
// through LDS once per item.  The next streamed tile is fetched into
// registers while the current one is being computed.
#include <algorithm>

#include "internal.h"
#include "device.h"

namespace hstu {

namespace {

constexpr int THREADS = 256;     // 4 waves
constexpr int RM_PAD = 8;        // row-major LDS stride D+8 bf16
constexpr int POS_COPY = 2 * TILE + 4;

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

struct KParams {
  const u16 *q, *k, *v;
  const u16 *dO;
  const float *pos_w, *time_w;
  const int64_t *ts;
  const int32_t *ctrl;
  int32_t *pop;
  const SeqInfo *info;
  const WorkEntry *list;
  u16 *out0, *out1;
  float *dpos_part, *dtime_part;
  int32_t H, N, nb;
  float inv_n;
};

// ------------------------------------------------------------ tile staging
// A 64-row tile of one head, D bf16 per row, moved global -> registers ->
// LDS in 16-byte chunks; rows at or beyond `valid` are zeros, so padded
// keys/queries contribute exact zeros to every product.
template <int D>
struct TileRegs {
  static constexpr int CPT = TILE * D / 8 / THREADS;   // chunks per thread
  uint4 c[CPT];

  __device__ __forceinline__ void load(const u16 *__restrict__ tile_base,
                                       int valid, int row_stride, int tid) {
#pragma unroll
    for (int x = 0; x < CPT; ++x) {
      const int ch = tid + THREADS * x;
      const int r = ch / (D / 8), d0 = (ch % (D / 8)) * 8;
      c[x] = r < valid ? *(const uint4 *)(tile_base + r * row_stride + d0)
                       : make_uint4(0, 0, 0, 0);
    }
  }
  __device__ __forceinline__ void store(u16 *lds, int tid) const {
#pragma unroll
    for (int x = 0; x < CPT; ++x) {
      const int ch = tid + THREADS * x;
      const int r = ch / (D / 8), d0 = (ch % (D / 8)) * 8;
      *(uint4 *)(lds + r * (D + RM_PAD) + d0) = c[x];
    }
  }
};

// A operand (or B operand of a score product) from a row-major LDS tile:
// 8 consecutive d of row `row`, starting at column col.
__device__ __forceinline__ bf16x8 read_rm(const u16 *lds, int stride, int row, int col) {
  return *(const bf16x8 *)(lds + row * stride + col);
}

// Operand holding, for lane l, column ncol + (l & 31) of rows
// krow .. krow+3 and krow+8 .. krow+11 of a row-major LDS tile (krow
// already includes this lane's 4*(l/32)), via two LDS transpose loads.
// Within a 16-lane group, lane c addresses row (c>>2), columns 4*(c&3)..+3
// of its group's 16-column slab; the transpose hands lane i the column
// slab+i of the four rows.
__device__ __forceinline__ bf16x8 read_tr(const u16 *lds, int stride, int krow,
                                          int ncol, int lane) {
  const int c = lane & 15;
  const u16 *p = lds + (krow + (c >> 2)) * stride + ncol + ((lane >> 4) & 1) * 16 + 4 * (c & 3);
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)p);
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)(p + 8 * stride));
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  const v8i16 x = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, x);
}

// Stationary 32-row operand: lane holds row `row` of the tile (zero when
// row >= valid), dims 16*ks + 8*g .. +7, ks = 0 .. D/16-1.
template <int D>
__device__ __forceinline__ void load_stationary(const u16 *__restrict__ tile_base,
                                                int row, int valid, int row_stride,
                                                int g, bf16x8 (&reg)[D / 16]) {
  const bool ok = row < valid;
  const u16 *p = tile_base + row * row_stride + 8 * g;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks)
    reg[ks] = as_bf16x8(ok ? *(const uint4 *)(p + 16 * ks) : make_uint4(0, 0, 0, 0));
}

// Position-bias slice of tile pair (qt, kt), stored four times with shifts
// 0..3 so that any lane can read 4 consecutive entries with one aligned
// 16-byte load: copy s, entry x = bias of local offset j_loc - i_loc =
// x + s - 63.  Indices outside the table are only reached by masked pairs
// and read as 0.
__device__ __forceinline__ void stage_pos(const KParams &P, int h, int qt, int kt,
                                          float *pos, int tid) {
  const int64_t span = 2 * (int64_t)P.N - 1;
  const int64_t base = (int64_t)(kt - qt) * TILE + P.N - 1 - (TILE - 1);
  const float *tab = P.pos_w + (int64_t)h * span;
  for (int x = tid; x < 4 * POS_COPY; x += THREADS) {
    const int s = x / POS_COPY, e = x % POS_COPY;
    const int64_t idx = base + e + s;
    pos[x] = (idx >= 0 && idx < span) ? tab[idx] : 0.0f;
  }
}

// Bias lookups of one lane: 16 consecutive-in-register scores whose
// streamed-side local index is sbase + c_row(r, g) and whose stationary
// local index is `st`.  Returns a pointer p such that p[c_row(r,g)-4g]
// is the position bias of register r; aligned for 16-byte reads.
//   q-stationary (fwd, dq): offset = j - i = (sbase + 4g + c) - st
//   k-stationary (dkv):     offset = j - i = st - (sbase + 4g + c)
// handled by the callers through the sign of the register walk.
__device__ __forceinline__ const float *pos_lane_q(const float *pos, int st, int sbase, int g) {
  const int x0 = sbase + 4 * g - st + (TILE - 1);     // x for c_row offset 0, >= 0
  const int s = x0 & 3;
  return pos + s * POS_COPY + (x0 - s);
}

// 32-bit time bucket of |d| (exact for |d| < 2^31): branch-free.
__device__ __forceinline__ int bucket32(int32_t dlt, int nb) {
  const uint32_t x = (uint32_t)(dlt < 0 ? -dlt : dlt);
  const int e = 31 - __builtin_clz(x | 1u);
  const uint32_t m = __builtin_amdgcn_ubfe(x, (uint32_t)(e - 2) & 31u, 2u);
  int b = 4 * e - 4 + (int)m;
  b = x < 4u ? (int)x : b;
  return b < nb - 1 ? b : nb - 1;
}

// Relative-time bucket of a pair: the 32-bit path on timestamps relative to
// the sequence start (exact while both lie within +-2^30 of it), else the
// 64-bit rule on the raw timestamps.
template <bool SLOW>
__device__ __forceinline__ int pair_bucket(int32_t a32, int32_t b32, int64_t a64,
                                           int64_t b64, int nb) {
  return SLOW ? time_bucket(a64 - b64, nb) : bucket32(a32 - b32, nb);
}

// Biased scores of a q-stationary lane (query i fixed, 16 keys): x[r] =
// s[r] + pos bias + time bias.  pl: this lane's aligned position-bias
// pointer; tk / tk64: key timestamps of its first key (32-bit relative /
// raw); the lane's keys sit at offsets 8*q4 + c, c = 0..3.
template <bool POS, bool TIME, bool SLOW>
__device__ __forceinline__ void biased_scores_q(const f32x16 &s, float (&x)[16],
                                                const float *pl, const int32_t *tk,
                                                const int64_t *tk64, const float *tw,
                                                int32_t ts_i32, int64_t ts_i, int nb) {
#pragma unroll
  for (int q4 = 0; q4 < 4; ++q4) {
    const float4 pb = POS ? *(const float4 *)(pl + 8 * q4) : make_float4(0.f, 0.f, 0.f, 0.f);
    const int4 t4 = (TIME && !SLOW) ? *(const int4 *)(tk + 8 * q4) : make_int4(0, 0, 0, 0);
    const float pbv[4] = {pb.x, pb.y, pb.z, pb.w};
    const int32_t tv[4] = {t4.x, t4.y, t4.z, t4.w};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      float v = s[4 * q4 + c];
      if (POS) v += pbv[c];
      if (TIME) {
        const int64_t t64 = SLOW ? tk64[8 * q4 + c] : 0;
        v += tw[pair_bucket<SLOW>(ts_i32, tv[c], ts_i, t64, nb)];
      }
      x[4 * q4 + c] = v;
    }
  }
}

// Biased scores of a k-stationary lane (key j fixed, 16 queries at offsets
// i_rel = 8*q4 + c from its first query): position bias at pos[x0 - i_rel]
// (descending), time bias of ts_i - ts_j; bk[r] receives the bucket.
template <bool POS, bool TIME, bool SLOW>
__device__ __forceinline__ void biased_scores_k(const f32x16 &s, float (&x)[16], int (&bk)[16],
                                                const float *pos, int x0, const int32_t *tq,
                                                const int64_t *tq64, const float *tw,
                                                int32_t ts_j32, int64_t ts_j, int nb) {
#pragma unroll
  for (int q4 = 0; q4 < 4; ++q4) {
    const int4 t4 = (TIME && !SLOW) ? *(const int4 *)(tq + 8 * q4) : make_int4(0, 0, 0, 0);
    const int32_t tv[4] = {t4.x, t4.y, t4.z, t4.w};
#pragma unroll
    for (int c = 0; c < 4; ++c) {
      const int r = 4 * q4 + c, i_rel = 8 * q4 + c;
      float v = s[r];
      if (POS) v += pos[x0 - i_rel];
      bk[r] = 0;
      if (TIME) {
        const int64_t t64 = SLOW ? tq64[i_rel] : 0;
        bk[r] = pair_bucket<SLOW>(tv[c], ts_j32, t64, ts_j, nb);
        v += tw[bk[r]];
      }
      x[r] = v;
    }
  }
}

// silu(x) / N = x / (N (1 + e^-x)); hardware exp2 and reciprocal.
__device__ __forceinline__ float silu_over_n(float x, float n) {
  const float t = __builtin_amdgcn_exp2f(x * -1.44269504088896341f);
  return x * __builtin_amdgcn_rcpf(__builtin_fmaf(n, t, n));
}

constexpr int32_t REL_LIMIT = 1 << 30;   // |ts - ts_start| below this -> 32-bit deltas

template <int D>
struct StreamSmem {
  union {
    struct {
      u16 a[TILE * (D + RM_PAD)];
      u16 b[TILE * (D + RM_PAD)];
    } t;
    float red[2][32 * D];                // cross-wave sums at the end of an item
  };
  alignas(16) float pos[4 * POS_COPY];
  alignas(16) int32_t ts32[TILE];
  int64_t ts64[TILE];
  int item;
};

__device__ __forceinline__ int pop_item(const KParams &P, int &slot_item, int tid) {
  if (tid == 0) slot_item = atomicAdd(P.pop, 1);
  __syncthreads();
  return slot_item;
}

// ---------------------------------------------------------------- forward
template <int D, bool POS, bool TIME>
__global__ void __launch_bounds__(THREADS)
attn_fwd_kernel(KParams P) {
  __shared__ StreamSmem<D> sm;
  extern __shared__ float tw[];               // time_w row of the item's head
  constexpr int ST = D + RM_PAD;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int wi = w & 1, wj = w >> 1;          // query half, key half
  const int n_items = P.ctrl[CTRL_N_ENTRIES] * P.H;
  const int row_stride = P.H * D;

  for (;;) {
    const int item = pop_item(P, sm.item, tid);
    if (item >= n_items) break;
    const WorkEntry e = P.list[item / P.H];
    const int h = item % P.H;
    const SeqInfo si = P.info[e.seq];
    const int qt = e.tile;
    const int q_valid = si.len - qt * TILE;
    const int i_loc = 32 * wi + l32;
    const u16 *qbase = P.q + ((si.start + (int64_t)qt * TILE) * P.H + h) * D;

    bf16x8 qreg[D / 16];
    load_stationary<D>(qbase, i_loc, q_valid, row_stride, g, qreg);

    int64_t ts_start = 0, ts_i = 0;
    int32_t ts_i32 = 0;
    bool item_slow = false;
    if (TIME) {
      ts_start = P.ts[si.start];
      ts_i = i_loc < q_valid ? P.ts[si.start + (int64_t)qt * TILE + i_loc] : ts_start;
      const int64_t rel = ts_i - ts_start;
      ts_i32 = (int32_t)rel;
      for (int x = tid; x < P.nb; x += THREADS) tw[x] = P.time_w[(int64_t)h * P.nb + x];
      item_slow = __syncthreads_or(rel >= REL_LIMIT || rel <= -REL_LIMIT);
    }

    f32x16 oacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;

    TileRegs<D> kr, vr;
    int64_t ts_k = 0;
    {
      const u16 *kb = P.k + ((si.start) * P.H + h) * (int64_t)D;
      const u16 *vb = P.v + ((si.start) * P.H + h) * (int64_t)D;
      kr.load(kb, si.len, row_stride, tid);
      vr.load(vb, si.len, row_stride, tid);
      if (TIME && tid < TILE) ts_k = tid < si.len ? P.ts[si.start + tid] : ts_start;
    }

    for (int kt = 0; kt <= qt; ++kt) {
      __syncthreads();
      kr.store(sm.t.a, tid);
      vr.store(sm.t.b, tid);
      if (POS) stage_pos(P, h, qt, kt, sm.pos, tid);
      bool tile_slow = item_slow;
      if (TIME) {
        int far = 0;
        if (tid < TILE) {
          const int64_t rel = ts_k - ts_start;
          sm.ts32[tid] = (int32_t)rel;
          sm.ts64[tid] = ts_k;
          far = rel >= REL_LIMIT || rel <= -REL_LIMIT;
        }
        tile_slow |= __syncthreads_or(far) != 0;
      } else {
        __syncthreads();
      }
      if (kt < qt) {       // prefetch the next key tile while this one computes
        const int k_valid = si.len - (kt + 1) * TILE;
        const int64_t r0 = si.start + (int64_t)(kt + 1) * TILE;
        kr.load(P.k + (r0 * P.H + h) * D, k_valid, row_stride, tid);
        vr.load(P.v + (r0 * P.H + h) * D, k_valid, row_stride, tid);
        if (TIME && tid < TILE) ts_k = tid < k_valid ? P.ts[r0 + tid] : ts_start;
      }

      // S^T quadrant [32 keys x 32 queries] = K_wj Q_wi^T
      f32x16 s;
#pragma unroll
      for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks)
        s = mfma32(read_rm(sm.t.a, ST, 32 * wj + l32, 16 * ks + 8 * g), qreg[ks], s);

      // a_ij = silu(s_ij + bias) / N; causal mask (after the SiLU) only on
      // the diagonal tile
      const float *pl = POS ? pos_lane_q(sm.pos, i_loc, 32 * wj, g) : nullptr;
      const int32_t *tk = sm.ts32 + 32 * wj + 4 * g;
      const int64_t *tk64 = sm.ts64 + 32 * wj + 4 * g;
      const float fN = (float)P.N;
      float av[16];
      if (TIME && tile_slow)
        biased_scores_q<POS, TIME, true>(s, av, pl, tk, tk64, tw, ts_i32, ts_i, P.nb);
      else
        biased_scores_q<POS, TIME, false>(s, av, pl, tk, tk64, tw, ts_i32, ts_i, P.nb);
#pragma unroll
      for (int r = 0; r < 16; ++r) av[r] = silu_over_n(av[r], fN);
      if (kt == qt) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (32 * wj + c_row(r, g) > i_loc) av[r] = 0.0f;
      }

      // O_wi += P V over this wave's 32 keys (two 16-key k-steps)
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        uint4 pk;
        pk.x = pack2(av[8 * ks + 0], av[8 * ks + 1]);
        pk.y = pack2(av[8 * ks + 2], av[8 * ks + 3]);
        pk.z = pack2(av[8 * ks + 4], av[8 * ks + 5]);
        pk.w = pack2(av[8 * ks + 6], av[8 * ks + 7]);
        const bf16x8 pa = as_bf16x8(pk);
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
          oacc[db] = mfma32(pa, read_tr(sm.t.b, ST, 32 * wj + 16 * ks + 4 * g, 32 * db, lane),
                            oacc[db]);
      }
    }

    // sum the two key halves, store O (bf16)
    __syncthreads();
    if (wj == 1) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sm.red[wi][(c_row(r, g)) * D + 32 * db + l32] = oacc[db][r];
    }
    __syncthreads();
    if (wj == 0) {
      u16 *o = P.out0 + ((si.start + (int64_t)qt * TILE) * P.H + h) * D;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int il = 32 * wi + c_row(r, g);
          const float val = oacc[db][r] + sm.red[wi][c_row(r, g) * D + 32 * db + l32];
          if (il < q_valid) {
            __bf16 bv = (__bf16)val;
            o[il * row_stride + 32 * db + l32] = __builtin_bit_cast(u16, bv);
          }
        }
    }
  }
}

// --------------------------------------------------------------------- dQ
template <int D, bool POS, bool TIME>
__global__ void __launch_bounds__(THREADS)
attn_dq_kernel(KParams P) {
  __shared__ StreamSmem<D> sm;
  extern __shared__ float tw[];
  constexpr int ST = D + RM_PAD;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int wi = w & 1, wj = w >> 1;
  const int n_items = P.ctrl[CTRL_N_ENTRIES] * P.H;
  const int row_stride = P.H * D;

  for (;;) {
    const int item = pop_item(P, sm.item, tid);
    if (item >= n_items) break;
    const WorkEntry e = P.list[item / P.H];
    const int h = item % P.H;
    const SeqInfo si = P.info[e.seq];
    const int qt = e.tile;
    const int q_valid = si.len - qt * TILE;
    const int i_loc = 32 * wi + l32;
    const int64_t qoff = ((si.start + (int64_t)qt * TILE) * P.H + h) * D;

    bf16x8 qreg[D / 16], doreg[D / 16];
    load_stationary<D>(P.q + qoff, i_loc, q_valid, row_stride, g, qreg);
    load_stationary<D>(P.dO + qoff, i_loc, q_valid, row_stride, g, doreg);

    int64_t ts_start = 0, ts_i = 0;
    int32_t ts_i32 = 0;
    bool item_slow = false;
    if (TIME) {
      ts_start = P.ts[si.start];
      ts_i = i_loc < q_valid ? P.ts[si.start + (int64_t)qt * TILE + i_loc] : ts_start;
      const int64_t rel = ts_i - ts_start;
      ts_i32 = (int32_t)rel;
      for (int x = tid; x < P.nb; x += THREADS) tw[x] = P.time_w[(int64_t)h * P.nb + x];
      item_slow = __syncthreads_or(rel >= REL_LIMIT || rel <= -REL_LIMIT);
    }

    f32x16 acc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[db][r] = 0.0f;

    TileRegs<D> kr, vr;
    int64_t ts_k = 0;
    {
      const int64_t r0 = si.start;
      kr.load(P.k + (r0 * P.H + h) * D, si.len, row_stride, tid);
      vr.load(P.v + (r0 * P.H + h) * D, si.len, row_stride, tid);
      if (TIME && tid < TILE) ts_k = tid < si.len ? P.ts[r0 + tid] : ts_start;
    }

    for (int kt = 0; kt <= qt; ++kt) {
      __syncthreads();
      kr.store(sm.t.a, tid);
      vr.store(sm.t.b, tid);
      if (POS) stage_pos(P, h, qt, kt, sm.pos, tid);
      bool tile_slow = item_slow;
      if (TIME) {
        int far = 0;
        if (tid < TILE) {
          const int64_t rel = ts_k - ts_start;
          sm.ts32[tid] = (int32_t)rel;
          sm.ts64[tid] = ts_k;
          far = rel >= REL_LIMIT || rel <= -REL_LIMIT;
        }
        tile_slow |= __syncthreads_or(far) != 0;
      } else {
        __syncthreads();
      }
      if (kt < qt) {
        const int k_valid = si.len - (kt + 1) * TILE;
        const int64_t r0 = si.start + (int64_t)(kt + 1) * TILE;
        kr.load(P.k + (r0 * P.H + h) * D, k_valid, row_stride, tid);
        vr.load(P.v + (r0 * P.H + h) * D, k_valid, row_stride, tid);
        if (TIME && tid < TILE) ts_k = tid < k_valid ? P.ts[r0 + tid] : ts_start;
      }

      f32x16 s, da;
#pragma unroll
      for (int r = 0; r < 16; ++r) { s[r] = 0.0f; da[r] = 0.0f; }
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        s = mfma32(read_rm(sm.t.a, ST, 32 * wj + l32, 16 * ks + 8 * g), qreg[ks], s);
        da = mfma32(read_rm(sm.t.b, ST, 32 * wj + l32, 16 * ks + 8 * g), doreg[ks], da);
      }

      const float *pl = POS ? pos_lane_q(sm.pos, i_loc, 32 * wj, g) : nullptr;
      const int32_t *tk = sm.ts32 + 32 * wj + 4 * g;
      const int64_t *tk64 = sm.ts64 + 32 * wj + 4 * g;
      float dsv[16];
      if (TIME && tile_slow)
        biased_scores_q<POS, TIME, true>(s, dsv, pl, tk, tk64, tw, ts_i32, ts_i, P.nb);
      else
        biased_scores_q<POS, TIME, false>(s, dsv, pl, tk, tk64, tw, ts_i32, ts_i, P.nb);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const float x = dsv[r];
        const float sg = sigmoid_f(x);
        dsv[r] = da[r] * sg * __builtin_fmaf(x, 1.0f - sg, 1.0f) * P.inv_n;
      }
      if (kt == qt) {
#pragma unroll
        for (int r = 0; r < 16; ++r)
          if (32 * wj + c_row(r, g) > i_loc) dsv[r] = 0.0f;
      }

#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        uint4 pk;
        pk.x = pack2(dsv[8 * ks + 0], dsv[8 * ks + 1]);
        pk.y = pack2(dsv[8 * ks + 2], dsv[8 * ks + 3]);
        pk.z = pack2(dsv[8 * ks + 4], dsv[8 * ks + 5]);
        pk.w = pack2(dsv[8 * ks + 6], dsv[8 * ks + 7]);
        const bf16x8 pa = as_bf16x8(pk);
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
          acc[db] = mfma32(pa, read_tr(sm.t.a, ST, 32 * wj + 16 * ks + 4 * g, 32 * db, lane),
                           acc[db]);
      }
    }

    __syncthreads();
    if (wj == 1) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sm.red[wi][c_row(r, g) * D + 32 * db + l32] = acc[db][r];
    }
    __syncthreads();
    if (wj == 0) {
      u16 *dq = P.out0 + qoff;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int il = 32 * wi + c_row(r, g);
          const float val = acc[db][r] + sm.red[wi][c_row(r, g) * D + 32 * db + l32];
          if (il < q_valid) {
            __bf16 bv = (__bf16)val;
            dq[il * row_stride + 32 * db + l32] = __builtin_bit_cast(u16, bv);
          }
        }
    }
  }
}

// ------------------------------------------------------------------ dK/dV
template <int D>
struct DkvSmem {
  StreamSmem<D> s;
  float diag_acc[2 * TILE];     // d_pos of the current tile pair by local offset
};

template <int D, bool POS, bool TIME>
__global__ void __launch_bounds__(THREADS)
attn_dkv_kernel(KParams P) {
  __shared__ DkvSmem<D> smx;
  StreamSmem<D> &sm = smx.s;
  extern __shared__ float dyn[];             // [nb] time_w row, then [H][nb] d_time
  float *tw = dyn;
  float *tacc = dyn + P.nb;
  constexpr int ST = D + RM_PAD;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int wj = w & 1, wi = w >> 1;          // key half (stationary), query half
  const int n_items = P.ctrl[CTRL_N_ENTRIES] * P.H;
  const int row_stride = P.H * D;

  if (TIME)
    for (int x = tid; x < P.H * P.nb; x += THREADS) tacc[x] = 0.0f;
  for (int x = tid; x < 2 * TILE; x += THREADS) smx.diag_acc[x] = 0.0f;

  for (;;) {
    const int item = pop_item(P, sm.item, tid);
    if (item >= n_items) break;
    const WorkEntry e = P.list[item / P.H];
    const int h = item % P.H;
    const SeqInfo si = P.info[e.seq];
    const int kt = e.tile;
    const int k_valid = si.len - kt * TILE;
    const int j_loc = 32 * wj + l32;
    const int64_t koff = ((si.start + (int64_t)kt * TILE) * P.H + h) * D;

    bf16x8 kreg[D / 16], vreg[D / 16];
    load_stationary<D>(P.k + koff, j_loc, k_valid, row_stride, g, kreg);
    load_stationary<D>(P.v + koff, j_loc, k_valid, row_stride, g, vreg);

    int64_t ts_start = 0, ts_j = 0;
    int32_t ts_j32 = 0;
    bool item_slow = false;
    if (TIME) {
      ts_start = P.ts[si.start];
      ts_j = j_loc < k_valid ? P.ts[si.start + (int64_t)kt * TILE + j_loc] : ts_start;
      const int64_t rel = ts_j - ts_start;
      ts_j32 = (int32_t)rel;
      for (int x = tid; x < P.nb; x += THREADS) tw[x] = P.time_w[(int64_t)h * P.nb + x];
      item_slow = __syncthreads_or(rel >= REL_LIMIT || rel <= -REL_LIMIT);
    }
    float *my_t = TIME ? tacc + h * P.nb : nullptr;
    // run-length pre-combined d_time: this lane's pairs (its key against
    // increasing queries) visit non-decreasing buckets when timestamps are
    // ordered, so a run is flushed only when its bucket changes
    float tsum = 0.0f;
    int tcur = -1;

    f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) { dk[db][r] = 0.0f; dv[db][r] = 0.0f; }

    TileRegs<D> qr, dr;
    int64_t ts_q = 0;
    {
      const int q_valid = si.len - kt * TILE;
      const int64_t r0 = si.start + (int64_t)kt * TILE;
      qr.load(P.q + (r0 * P.H + h) * D, q_valid, row_stride, tid);
      dr.load(P.dO + (r0 * P.H + h) * D, q_valid, row_stride, tid);
      if (TIME && tid < TILE) ts_q = tid < q_valid ? P.ts[r0 + tid] : ts_start;
    }

    for (int qt = kt; qt < si.ntiles; ++qt) {
      const int q_valid = si.len - qt * TILE;
      __syncthreads();
      qr.store(sm.t.a, tid);
      dr.store(sm.t.b, tid);
      if (POS) stage_pos(P, h, qt, kt, sm.pos, tid);
      bool tile_slow = item_slow;
      if (TIME) {
        int far = 0;
        if (tid < TILE) {
          const int64_t rel = ts_q - ts_start;
          sm.ts32[tid] = (int32_t)rel;
          sm.ts64[tid] = ts_q;
          far = rel >= REL_LIMIT || rel <= -REL_LIMIT;
        }
        tile_slow |= __syncthreads_or(far) != 0;
      } else {
        __syncthreads();
      }
      if (qt + 1 < si.ntiles) {
        const int nv = si.len - (qt + 1) * TILE;
        const int64_t r0 = si.start + (int64_t)(qt + 1) * TILE;
        qr.load(P.q + (r0 * P.H + h) * D, nv, row_stride, tid);
        dr.load(P.dO + (r0 * P.H + h) * D, nv, row_stride, tid);
        if (TIME && tid < TILE) ts_q = tid < nv ? P.ts[r0 + tid] : ts_start;
      }

      // S and dA quadrants [32 queries x 32 keys]; lane holds key j_loc
      f32x16 s, da;
#pragma unroll
      for (int r = 0; r < 16; ++r) { s[r] = 0.0f; da[r] = 0.0f; }
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        s = mfma32(read_rm(sm.t.a, ST, 32 * wi + l32, 16 * ks + 8 * g), kreg[ks], s);
        da = mfma32(read_rm(sm.t.b, ST, 32 * wi + l32, 16 * ks + 8 * g), vreg[ks], da);
      }

      // offset j - i = j_loc - (32 wi + 4 g + c_row'): walk the position
      // slice downwards from x0 = j_loc - 32 wi - 4 g + 63
      const int x0 = j_loc - 32 * wi - 4 * g + (TILE - 1);
      const int32_t *tq = sm.ts32 + 32 * wi + 4 * g;
      const int64_t *tq64 = sm.ts64 + 32 * wi + 4 * g;
      const bool diag = (qt == kt);
      float av[16], dsv[16];
      int bk[16];
      if (TIME && tile_slow)
        biased_scores_k<POS, TIME, true>(s, av, bk, sm.pos, x0, tq, tq64, tw, ts_j32, ts_j, P.nb);
      else
        biased_scores_k<POS, TIME, false>(s, av, bk, sm.pos, x0, tq, tq64, tw, ts_j32, ts_j, P.nb);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int i_rel = 8 * (r >> 2) + (r & 3);          // c_row(r, g) - 4g
        const int i_loc = 32 * wi + 4 * g + i_rel;
        const bool valid = (i_loc < q_valid) && (!diag || i_loc >= j_loc);
        const float x = av[r];
        const float sg = sigmoid_f(x);
        const float a = x * sg * P.inv_n;
        const float ds = da[r] * sg * __builtin_fmaf(x, 1.0f - sg, 1.0f) * P.inv_n;
        av[r] = valid ? a : 0.0f;
        dsv[r] = valid ? ds : 0.0f;
        if (POS && valid) atomicAdd(&smx.diag_acc[x0 - i_rel], ds);
        if (TIME && valid) {
          if (bk[r] != tcur) {
            if (tcur >= 0) atomicAdd(&my_t[tcur], tsum);
            tcur = bk[r];
            tsum = 0.0f;
          }
          tsum += ds;
        }
      }

      // dV_wj += A^T dO, dK_wj += dS^T Q over this wave's 32 queries
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        uint4 pa, pd;
        pa.x = pack2(av[8 * ks + 0], av[8 * ks + 1]);
        pa.y = pack2(av[8 * ks + 2], av[8 * ks + 3]);
        pa.z = pack2(av[8 * ks + 4], av[8 * ks + 5]);
        pa.w = pack2(av[8 * ks + 6], av[8 * ks + 7]);
        pd.x = pack2(dsv[8 * ks + 0], dsv[8 * ks + 1]);
        pd.y = pack2(dsv[8 * ks + 2], dsv[8 * ks + 3]);
        pd.z = pack2(dsv[8 * ks + 4], dsv[8 * ks + 5]);
        pd.w = pack2(dsv[8 * ks + 6], dsv[8 * ks + 7]);
        const bf16x8 a8 = as_bf16x8(pa), d8 = as_bf16x8(pd);
        const int krow = 32 * wi + 16 * ks + 4 * g;
#pragma unroll
        for (int db = 0; db < D / 32; ++db) {
          dv[db] = mfma32(a8, read_tr(sm.t.b, ST, krow, 32 * db, lane), dv[db]);
          dk[db] = mfma32(d8, read_tr(sm.t.a, ST, krow, 32 * db, lane), dk[db]);
        }
      }
      if (POS) {
        // the diagonals of this tile pair are complete: fold them into the
        // sequence's d_pos partial (index m = i - j >= 0)
        __syncthreads();
        if (tid < 2 * TILE - 1) {
          const float val = smx.diag_acc[tid];
          smx.diag_acc[tid] = 0.0f;
          const int m = (qt - kt) * TILE - (tid - (TILE - 1));
          if (val != 0.0f && m >= 0 && m < si.len)
            atomicAdd(&P.dpos_part[(si.start + m) * P.H + h], val);
        }
      }
    }
    if (TIME && tcur >= 0) atomicAdd(&my_t[tcur], tsum);

    // sum the two query halves, store dK, dV (bf16)
    __syncthreads();
    if (wi == 1) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sm.red[wj][c_row(r, g) * D + 32 * db + l32] = dk[db][r];
    }
    __syncthreads();
    if (wi == 0) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) dk[db][r] += sm.red[wj][c_row(r, g) * D + 32 * db + l32];
    }
    __syncthreads();
    if (wi == 1) {
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r)
          sm.red[wj][c_row(r, g) * D + 32 * db + l32] = dv[db][r];
    }
    __syncthreads();
    if (wi == 0) {
      u16 *dko = P.out0 + koff;
      u16 *dvo = P.out1 + koff;
#pragma unroll
      for (int db = 0; db < D / 32; ++db)
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int jl = 32 * wj + c_row(r, g);
          const float vv = dv[db][r] + sm.red[wj][c_row(r, g) * D + 32 * db + l32];
          if (jl < k_valid) {
            __bf16 bk = (__bf16)dk[db][r], bv = (__bf16)vv;
            dko[jl * row_stride + 32 * db + l32] = __builtin_bit_cast(u16, bk);
            dvo[jl * row_stride + 32 * db + l32] = __builtin_bit_cast(u16, bv);
          }
        }
    }
  }
  if (TIME) {
    __syncthreads();
    float *part = P.dtime_part + (int64_t)blockIdx.x * P.H * P.nb;
    for (int x = tid; x < P.H * P.nb; x += THREADS) part[x] = tacc[x];
  }
}

// ------------------------------------------------------------- launchers
template <typename K>
int persistent_grid(K kernel, size_t dyn, int64_t items, int dev) {
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, THREADS, dyn) != hipSuccess ||
      occ < 1)
    occ = 1;
  const int64_t cap = (int64_t)device_info(dev).num_cu * occ;
  return (int)std::max<int64_t>(1, std::min<int64_t>(cap, items));
}

KParams make_params(const AttnArgs &a, int32_t *pop, const WorkEntry *list) {
  const char *ws = (const char *)a.ws;
  KParams P{};
  P.q = (const u16 *)a.q;
  P.k = (const u16 *)a.k;
  P.v = (const u16 *)a.v;
  P.pos_w = a.pos_w;
  P.time_w = a.time_w;
  P.ts = a.ts;
  P.ctrl = (const int32_t *)(ws + a.L.ctrl);
  P.pop = pop;
  P.info = (const SeqInfo *)(ws + a.L.seqinfo);
  P.list = list;
  P.H = a.p.H;
  P.N = a.p.N;
  P.nb = a.p.has_time ? a.p.nb : 0;
  P.inv_n = 1.0f / (float)a.p.N;
  return P;
}

#define HSTU_DISPATCH(KERNEL, D, POS, TIME, ...)                               \
  do {                                                                        \
    if (D == 64) {                                                            \
      if (POS && TIME) { auto kfn = KERNEL<64, true, true>; __VA_ARGS__; }    \
      else if (POS) { auto kfn = KERNEL<64, true, false>; __VA_ARGS__; }     \
      else if (TIME) { auto kfn = KERNEL<64, false, true>; __VA_ARGS__; }    \
      else { auto kfn = KERNEL<64, false, false>; __VA_ARGS__; }             \
    } else {                                                                  \
      if (POS && TIME) { auto kfn = KERNEL<128, true, true>; __VA_ARGS__; }   \
      else if (POS) { auto kfn = KERNEL<128, true, false>; __VA_ARGS__; }    \
      else if (TIME) { auto kfn = KERNEL<128, false, true>; __VA_ARGS__; }   \
      else { auto kfn = KERNEL<128, false, false>; __VA_ARGS__; }            \
    }                                                                         \
  } while (0)

int current_dev() {
  int dev = 0;
  (void)hipGetDevice(&dev);
  return dev;
}

}  // namespace

int attn_fwd_grid(const Problem &p, int dev) {
  int grid = 1;
  const size_t dyn = p.has_time ? sizeof(float) * p.nb : 0;
  HSTU_DISPATCH(attn_fwd_kernel, p.d, p.has_pos, p.has_time,
                grid = persistent_grid(kfn, dyn, p.max_entries * p.H, dev));
  return grid;
}

int attn_dq_grid(const Problem &p, int dev) {
  int grid = 1;
  const size_t dyn = p.has_time ? sizeof(float) * p.nb : 0;
  HSTU_DISPATCH(attn_dq_kernel, p.d, p.has_pos, p.has_time,
                grid = persistent_grid(kfn, dyn, p.max_entries * p.H, dev));
  return grid;
}

int attn_dkv_grid(const Problem &p, int dev) {
  int grid = 1;
  const size_t dyn = p.has_time ? sizeof(float) * (size_t)p.nb * (p.H + 1) : 0;
  HSTU_DISPATCH(attn_dkv_kernel, p.d, p.has_pos, p.has_time,
                grid = persistent_grid(kfn, dyn, p.max_entries * p.H, dev));
  return grid;
}

hipError_t launch_attn_fwd_bf16(const AttnArgs &a, void *o, hipStream_t s) {
  const char *ws = (const char *)a.ws;
  KParams P = make_params(a, (int32_t *)(ws + a.L.ctrl) + CTRL_POP_FWD,
                          (const WorkEntry *)(ws + a.L.list_q));
  P.out0 = (u16 *)o;
  const Problem &p = a.p;
  const int grid = attn_fwd_grid(p, current_dev());
  const size_t dyn = p.has_time ? sizeof(float) * p.nb : 0;
  HSTU_DISPATCH(attn_fwd_kernel, p.d, p.has_pos, p.has_time,
                hipLaunchKernelGGL(kfn, dim3(grid), dim3(THREADS), dyn, s, P));
  return hipGetLastError();
}

hipError_t launch_attn_dq_bf16(const AttnArgs &a, const void *dO, void *dq,
                               hipStream_t s) {
  const char *ws = (const char *)a.ws;
  KParams P = make_params(a, (int32_t *)(ws + a.L.ctrl) + CTRL_POP_DQ,
                          (const WorkEntry *)(ws + a.L.list_q));
  P.dO = (const u16 *)dO;
  P.out0 = (u16 *)dq;
  const Problem &p = a.p;
  const int grid = attn_dq_grid(p, current_dev());
  const size_t dyn = p.has_time ? sizeof(float) * p.nb : 0;
  HSTU_DISPATCH(attn_dq_kernel, p.d, p.has_pos, p.has_time,
                hipLaunchKernelGGL(kfn, dim3(grid), dim3(THREADS), dyn, s, P));
  return hipGetLastError();
}

hipError_t launch_attn_dkv_bf16(const AttnArgs &a, const void *dO, void *dk,
                                void *dv, hipStream_t s) {
  const char *ws = (const char *)a.ws;
  KParams P = make_params(a, (int32_t *)(ws + a.L.ctrl) + CTRL_POP_DKV,
                          (const WorkEntry *)(ws + a.L.list_k));
  P.dO = (const u16 *)dO;
  P.out0 = (u16 *)dk;
  P.out1 = (u16 *)dv;
  P.dpos_part = a.L.dpos_part ? (float *)(ws + a.L.dpos_part) : nullptr;
  P.dtime_part = a.L.dtime_part ? (float *)(ws + a.L.dtime_part) : nullptr;
  const Problem &p = a.p;
  const int grid = a.L.dkv_grid;   // the d_time partials are sized for it
  const size_t dyn = p.has_time ? sizeof(float) * (size_t)p.nb * (p.H + 1) : 0;
  HSTU_DISPATCH(attn_dkv_kernel, p.d, p.has_pos, p.has_time,
                hipLaunchKernelGGL(kfn, dim3(grid), dim3(THREADS), dyn, s, P));
  return hipGetLastError();
}

}  // namespace hstu
