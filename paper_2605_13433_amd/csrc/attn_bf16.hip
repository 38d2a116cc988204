// bf16 MFMA kernels of jagged HSTU attention for gfx950 (Sec. 3.1.1: jagged
// QKV, relative position + relative time bias fused into the attention
// kernel, no padding and no dense<->jagged conversion).
//
// Three persistent kernels pop (sequence, tile, head) items from the
// scheduler's longest-first lists:
//
//   attn_fwd   q-stationary: O_i = sum_{j<=i} silu(s_ij)/N v_j
//   attn_dq    q-stationary: dQ_i = sum_{j<=i} dS_ij k_j
//   attn_dkv   k-stationary: dV_j = sum_{i>=j} a_ij dO_i,
//                            dK_j = sum_{i>=j} dS_ij q_i, and the table
//                            gradients (per-sequence diagonal partials for
//                            d_pos, per-work-group histograms for d_time)
//
// with s_ij = <q_i,k_j> + pos_w[h, j-i+N-1] + time_w[h, bucket(ts_i-ts_j)],
// dS_ij = <dO_i, v_j> silu'(s_ij) / N and the causal mask applied after the
// SiLU (a masked pair is exactly zero).
//
// Work-group = 2 wave64s over a 64x64 tile pair; wave w owns 32 rows of the
// stationary side.  All contractions use the 32x32x16 bf16 MFMA.  The
// stationary operand lives in registers; the streamed tile is staged in LDS
// row-major (operand of the score-side products, contracted over d) and
// transposed (operand of the accumulating products, contracted over the
// tile rows), because an MFMA operand holds 8 consecutive contraction
// indices per lane.  Score accumulators come out with one fixed stationary
// row per lane, which is exactly the layout the accumulating product needs
// for its own operand, so scores never leave registers.
#include <algorithm>

#include "internal.h"
#include "device.h"

namespace hstu {

namespace {

constexpr int THREADS = 128;     // 2 waves
constexpr int RM_PAD = 8;        // row-major LDS stride D+8 bf16 (conflict-free b128 reads)
constexpr int TR_STRIDE = TILE + 4;  // transposed LDS stride (conflict-free b64 reads)

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

// Cooperative load of tile rows [0, 64) (local), global rows row0 + r for
// r < valid, of head h, into LDS row-major and/or transposed copies; rows at
// or beyond `valid` are zero so that padded keys/queries contribute exact
// zeros to every MFMA.
template <int D, bool RM, bool TR>
__device__ __forceinline__ void load_tile(const u16 *__restrict__ src,
                                          int64_t row0, int valid, int H,
                                          int h, u16 *rm, u16 *tr, int tid) {
  constexpr int CH = D / 8;
  constexpr int TOTAL = TILE * CH;
#pragma unroll
  for (int c = tid; c < TOTAL; c += THREADS) {
    const int r = c / CH, d0 = (c % CH) * 8;
    uint4 x = make_uint4(0, 0, 0, 0);
    if (r < valid)
      x = *(const uint4 *)(src + ((row0 + r) * H + h) * (int64_t)D + d0);
    if (RM) *(uint4 *)(rm + r * (D + RM_PAD) + d0) = x;
    if (TR) {
      const uint32_t w4[4] = {x.x, x.y, x.z, x.w};
#pragma unroll
      for (int e = 0; e < 4; ++e) {
        tr[(d0 + 2 * e) * TR_STRIDE + r] = (u16)(w4[e] & 0xffffu);
        tr[(d0 + 2 * e + 1) * TR_STRIDE + r] = (u16)(w4[e] >> 16);
      }
    }
  }
}

// Stationary 32-row operand in registers: lane holds row `row` (local
// index in the tile, or >= valid -> zero), dims 16*ks + 8*g .. +7.
template <int D>
__device__ __forceinline__ void load_rows_reg(const u16 *__restrict__ src,
                                              int64_t row0, int row, int valid,
                                              int H, int h, int g,
                                              bf16x8 (&reg)[D / 16]) {
  const bool ok = row < valid;
  const u16 *p = src + ((row0 + row) * H + h) * (int64_t)D + 8 * g;
#pragma unroll
  for (int ks = 0; ks < D / 16; ++ks) {
    uint4 x = make_uint4(0, 0, 0, 0);
    if (ok) x = *(const uint4 *)(p + 16 * ks);
    reg[ks] = as_bf16x8(x);
  }
}

// Bias slice for tile pair (query tile qt, key tile kt): entry x holds
// pos_w[h, (kt-qt)*64 + x - 63 + N - 1], i.e. the bias of local offset
// j_loc - i_loc = x - 63.  Indices outside the table (only reachable by
// masked pairs) read as 0.
__device__ __forceinline__ void load_pos_slice(const KParams &P, int h, int qt,
                                               int kt, float *pos, int tid) {
  const int64_t span = 2 * (int64_t)P.N - 1;
  const int64_t base = (int64_t)(kt - qt) * TILE + P.N - 1 - (TILE - 1);
  for (int x = tid; x < 2 * TILE; x += THREADS) {
    const int64_t idx = base + x;
    pos[x] = (x < 2 * TILE - 1 && idx >= 0 && idx < span)
                 ? P.pos_w[(int64_t)h * span + idx] : 0.0f;
  }
}

template <int D>
struct FwdSmem {
  u16 k[TILE * (D + RM_PAD)];
  u16 vt[D * TR_STRIDE];
  float pos[2 * TILE];
  int64_t tsk[TILE];
  int item;
};

// ---------------------------------------------------------------- forward
template <int D, bool POS, bool TIME>
__global__ void __launch_bounds__(THREADS)
attn_fwd_kernel(KParams P) {
  __shared__ FwdSmem<D> sm;
  extern __shared__ float tw[];              // time_w row of the item's head
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int n_items = P.ctrl[CTRL_N_ENTRIES] * P.H;

  for (;;) {
    if (tid == 0) sm.item = atomicAdd(P.pop, 1);
    __syncthreads();
    const int item = sm.item;
    if (item >= n_items) break;
    const WorkEntry e = P.list[item / P.H];
    const int h = item % P.H;
    const SeqInfo si = P.info[e.seq];
    const int64_t row0 = si.start;
    const int qt = e.tile;
    const int q_valid = si.len - qt * TILE;       // valid rows of this q-tile
    const int i_loc = 32 * w + l32;               // this lane's query row

    bf16x8 qreg[D / 16];
    load_rows_reg<D>(P.q, row0 + (int64_t)qt * TILE, i_loc, q_valid, P.H, h, g, qreg);
    int64_t ts_i = 0;
    if (TIME) {
      if (i_loc < q_valid) ts_i = P.ts[row0 + (int64_t)qt * TILE + i_loc];
      for (int x = tid; x < P.nb; x += THREADS) tw[x] = P.time_w[(int64_t)h * P.nb + x];
    }

    f32x16 oacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;

    for (int kt = 0; kt <= qt; ++kt) {
      __syncthreads();
      const int k_valid = si.len - kt * TILE;
      const int64_t krow0 = row0 + (int64_t)kt * TILE;
      load_tile<D, true, false>(P.k, krow0, k_valid, P.H, h, sm.k, nullptr, tid);
      load_tile<D, false, true>(P.v, krow0, k_valid, P.H, h, nullptr, sm.vt, tid);
      if (POS) load_pos_slice(P, h, qt, kt, sm.pos, tid);
      if (TIME)
        for (int x = tid; x < TILE; x += THREADS)
          sm.tsk[x] = x < k_valid ? P.ts[krow0 + x] : 0;
      __syncthreads();

      const bool diag = (kt == qt);
#pragma unroll
      for (int jb = 0; jb < 2; ++jb) {
        // S^T block [32 keys x 32 queries] = K_jb Q^T
        f32x16 s;
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.0f;
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          const bf16x8 a = *(const bf16x8 *)(sm.k + (32 * jb + l32) * (D + RM_PAD) + 16 * ks + 8 * g);
          s = mfma32(a, qreg[ks], s);
        }
        // a_ij = silu(s_ij) / N, causal mask after the SiLU
        float av[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j_loc = 32 * jb + c_row(r, g);
          float x = s[r];
          if (POS) x += sm.pos[j_loc - i_loc + TILE - 1];
          if (TIME) x += tw[time_bucket(ts_i - sm.tsk[j_loc], P.nb)];
          float a = x * sigmoid_f(x) * P.inv_n;
          if (diag && j_loc > i_loc) a = 0.0f;
          av[r] = a;
        }
        // O += P V over the two 16-key k-steps of this block
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int ks = 2 * jb + half;
          uint4 pk;
          pk.x = pack2(av[8 * half + 0], av[8 * half + 1]);
          pk.y = pack2(av[8 * half + 2], av[8 * half + 3]);
          pk.z = pack2(av[8 * half + 4], av[8 * half + 5]);
          pk.w = pack2(av[8 * half + 6], av[8 * half + 7]);
          const bf16x8 pa = as_bf16x8(pk);
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            const u16 *vrow = sm.vt + (32 * db + l32) * TR_STRIDE + 16 * ks + 4 * g;
            const bf16x8 vb = join8(*(const uint2 *)vrow, *(const uint2 *)(vrow + 8));
            oacc[db] = mfma32(pa, vb, oacc[db]);
          }
        }
      }
    }

    // O tile: lane holds dim 32*db + l32 of query rows 32*w + c_row(r, g)
    u16 *o = P.out0;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int il = 32 * w + c_row(r, g);
        if (il < q_valid) {
          const int64_t row = row0 + (int64_t)qt * TILE + il;
          __bf16 b = (__bf16)oacc[db][r];
          o[(row * P.H + h) * D + 32 * db + l32] = __builtin_bit_cast(u16, b);
        }
      }
    __syncthreads();
  }
}

// --------------------------------------------------------------------- dQ
template <int D>
struct DqSmem {
  u16 k[TILE * (D + RM_PAD)];
  u16 v[TILE * (D + RM_PAD)];
  u16 kt[D * TR_STRIDE];
  float pos[2 * TILE];
  int64_t tsk[TILE];
  int item;
};

template <int D, bool POS, bool TIME>
__global__ void __launch_bounds__(THREADS)
attn_dq_kernel(KParams P) {
  __shared__ DqSmem<D> sm;
  extern __shared__ float tw[];
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int n_items = P.ctrl[CTRL_N_ENTRIES] * P.H;

  for (;;) {
    if (tid == 0) sm.item = atomicAdd(P.pop, 1);
    __syncthreads();
    const int item = sm.item;
    if (item >= n_items) break;
    const WorkEntry e = P.list[item / P.H];
    const int h = item % P.H;
    const SeqInfo si = P.info[e.seq];
    const int64_t row0 = si.start;
    const int qt = e.tile;
    const int q_valid = si.len - qt * TILE;
    const int i_loc = 32 * w + l32;

    bf16x8 qreg[D / 16], doreg[D / 16];
    load_rows_reg<D>(P.q, row0 + (int64_t)qt * TILE, i_loc, q_valid, P.H, h, g, qreg);
    load_rows_reg<D>(P.dO, row0 + (int64_t)qt * TILE, i_loc, q_valid, P.H, h, g, doreg);
    int64_t ts_i = 0;
    if (TIME) {
      if (i_loc < q_valid) ts_i = P.ts[row0 + (int64_t)qt * TILE + i_loc];
      for (int x = tid; x < P.nb; x += THREADS) tw[x] = P.time_w[(int64_t)h * P.nb + x];
    }

    f32x16 acc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[db][r] = 0.0f;

    for (int kt = 0; kt <= qt; ++kt) {
      __syncthreads();
      const int k_valid = si.len - kt * TILE;
      const int64_t krow0 = row0 + (int64_t)kt * TILE;
      load_tile<D, true, true>(P.k, krow0, k_valid, P.H, h, sm.k, sm.kt, tid);
      load_tile<D, true, false>(P.v, krow0, k_valid, P.H, h, sm.v, nullptr, tid);
      if (POS) load_pos_slice(P, h, qt, kt, sm.pos, tid);
      if (TIME)
        for (int x = tid; x < TILE; x += THREADS)
          sm.tsk[x] = x < k_valid ? P.ts[krow0 + x] : 0;
      __syncthreads();

      const bool diag = (kt == qt);
#pragma unroll
      for (int jb = 0; jb < 2; ++jb) {
        f32x16 s, da;
#pragma unroll
        for (int r = 0; r < 16; ++r) { s[r] = 0.0f; da[r] = 0.0f; }
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          const int off = (32 * jb + l32) * (D + RM_PAD) + 16 * ks + 8 * g;
          s = mfma32(*(const bf16x8 *)(sm.k + off), qreg[ks], s);     // S^T
          da = mfma32(*(const bf16x8 *)(sm.v + off), doreg[ks], da);  // dA^T
        }
        float dsv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int j_loc = 32 * jb + c_row(r, g);
          float x = s[r];
          if (POS) x += sm.pos[j_loc - i_loc + TILE - 1];
          if (TIME) x += tw[time_bucket(ts_i - sm.tsk[j_loc], P.nb)];
          const float sg = sigmoid_f(x);
          float ds = da[r] * sg * (1.0f + x * (1.0f - sg)) * P.inv_n;
          if (diag && j_loc > i_loc) ds = 0.0f;
          dsv[r] = ds;
        }
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int ks = 2 * jb + half;
          uint4 pk;
          pk.x = pack2(dsv[8 * half + 0], dsv[8 * half + 1]);
          pk.y = pack2(dsv[8 * half + 2], dsv[8 * half + 3]);
          pk.z = pack2(dsv[8 * half + 4], dsv[8 * half + 5]);
          pk.w = pack2(dsv[8 * half + 6], dsv[8 * half + 7]);
          const bf16x8 pa = as_bf16x8(pk);
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            const u16 *krow = sm.kt + (32 * db + l32) * TR_STRIDE + 16 * ks + 4 * g;
            acc[db] = mfma32(pa, join8(*(const uint2 *)krow, *(const uint2 *)(krow + 8)), acc[db]);
          }
        }
      }
    }

    u16 *dq = P.out0;
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int il = 32 * w + c_row(r, g);
        if (il < q_valid) {
          const int64_t row = row0 + (int64_t)qt * TILE + il;
          __bf16 b = (__bf16)acc[db][r];
          dq[(row * P.H + h) * D + 32 * db + l32] = __builtin_bit_cast(u16, b);
        }
      }
    __syncthreads();
  }
}

// ------------------------------------------------------------------ dK/dV
template <int D>
struct DkvSmem {
  u16 q[TILE * (D + RM_PAD)];
  u16 dO[TILE * (D + RM_PAD)];
  u16 qt[D * TR_STRIDE];
  u16 dOt[D * TR_STRIDE];
  float pos[2 * TILE];
  float diag_acc[2 * TILE];     // d_pos of this tile pair by local offset
  int64_t tsq[TILE];
  int item;
};

template <int D, bool POS, bool TIME>
__global__ void __launch_bounds__(THREADS)
attn_dkv_kernel(KParams P) {
  __shared__ DkvSmem<D> sm;
  extern __shared__ float dyn[];             // [nb] time_w row, then [H][nb] d_time
  float *tw = dyn;
  float *tacc = dyn + P.nb;
  const int tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
  const int g = lane >> 5, l32 = lane & 31;
  const int n_items = P.ctrl[CTRL_N_ENTRIES] * P.H;

  if (TIME)
    for (int x = tid; x < P.H * P.nb; x += THREADS) tacc[x] = 0.0f;
  for (int x = tid; x < 2 * TILE; x += THREADS) sm.diag_acc[x] = 0.0f;

  for (;;) {
    if (tid == 0) sm.item = atomicAdd(P.pop, 1);
    __syncthreads();
    const int item = sm.item;
    if (item >= n_items) break;
    const WorkEntry e = P.list[item / P.H];
    const int h = item % P.H;
    const SeqInfo si = P.info[e.seq];
    const int64_t row0 = si.start;
    const int kt = e.tile;
    const int k_valid = si.len - kt * TILE;
    const int j_loc = 32 * w + l32;               // this lane's key row

    bf16x8 kreg[D / 16], vreg[D / 16];
    load_rows_reg<D>(P.k, row0 + (int64_t)kt * TILE, j_loc, k_valid, P.H, h, g, kreg);
    load_rows_reg<D>(P.v, row0 + (int64_t)kt * TILE, j_loc, k_valid, P.H, h, g, vreg);
    int64_t ts_j = 0;
    if (TIME) {
      if (j_loc < k_valid) ts_j = P.ts[row0 + (int64_t)kt * TILE + j_loc];
      for (int x = tid; x < P.nb; x += THREADS) tw[x] = P.time_w[(int64_t)h * P.nb + x];
    }
    // run-length pre-combined d_time: consecutive pairs of this lane (its
    // key against increasing queries) usually share a bucket
    float tsum = 0.0f;
    int tcur = -1;

    f32x16 dk[D / 32], dv[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) { dk[db][r] = 0.0f; dv[db][r] = 0.0f; }

    for (int qt = kt; qt < si.ntiles; ++qt) {
      __syncthreads();
      const int q_valid = si.len - qt * TILE;
      const int64_t qrow0 = row0 + (int64_t)qt * TILE;
      load_tile<D, true, true>(P.q, qrow0, q_valid, P.H, h, sm.q, sm.qt, tid);
      load_tile<D, true, true>(P.dO, qrow0, q_valid, P.H, h, sm.dO, sm.dOt, tid);
      if (POS) load_pos_slice(P, h, qt, kt, sm.pos, tid);
      if (TIME)
        for (int x = tid; x < TILE; x += THREADS)
          sm.tsq[x] = x < q_valid ? P.ts[qrow0 + x] : 0;
      __syncthreads();

      const bool diag = (kt == qt);
#pragma unroll
      for (int ib = 0; ib < 2; ++ib) {
        // S and dA blocks [32 queries x 32 keys]; lane holds key j_loc
        f32x16 s, da;
#pragma unroll
        for (int r = 0; r < 16; ++r) { s[r] = 0.0f; da[r] = 0.0f; }
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          const int off = (32 * ib + l32) * (D + RM_PAD) + 16 * ks + 8 * g;
          s = mfma32(*(const bf16x8 *)(sm.q + off), kreg[ks], s);
          da = mfma32(*(const bf16x8 *)(sm.dO + off), vreg[ks], da);
        }
        float av[16], dsv[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
          const int i_loc = 32 * ib + c_row(r, g);
          float x = s[r];
          if (POS) x += sm.pos[j_loc - i_loc + TILE - 1];
          int bk = 0;
          if (TIME) {
            bk = time_bucket(sm.tsq[i_loc] - ts_j, P.nb);
            x += tw[bk];
          }
          const bool valid = (i_loc < q_valid) && (!diag || i_loc >= j_loc);
          const float sg = sigmoid_f(x);
          const float a = valid ? x * sg * P.inv_n : 0.0f;
          const float ds = valid ? da[r] * sg * (1.0f + x * (1.0f - sg)) * P.inv_n : 0.0f;
          av[r] = a;
          dsv[r] = ds;
          if (POS && valid) atomicAdd(&sm.diag_acc[j_loc - i_loc + TILE - 1], ds);
          if (TIME && valid) {
            if (bk != tcur) {
              if (tcur >= 0) atomicAdd(&tacc[h * P.nb + tcur], tsum);
              tcur = bk;
              tsum = 0.0f;
            }
            tsum += ds;
          }
        }
        // dV += A^T dO, dK += dS^T Q over this block's two 16-query k-steps
#pragma unroll
        for (int half = 0; half < 2; ++half) {
          const int ks = 2 * ib + half;
          uint4 pa, pd;
          pa.x = pack2(av[8 * half + 0], av[8 * half + 1]);
          pa.y = pack2(av[8 * half + 2], av[8 * half + 3]);
          pa.z = pack2(av[8 * half + 4], av[8 * half + 5]);
          pa.w = pack2(av[8 * half + 6], av[8 * half + 7]);
          pd.x = pack2(dsv[8 * half + 0], dsv[8 * half + 1]);
          pd.y = pack2(dsv[8 * half + 2], dsv[8 * half + 3]);
          pd.z = pack2(dsv[8 * half + 4], dsv[8 * half + 5]);
          pd.w = pack2(dsv[8 * half + 6], dsv[8 * half + 7]);
          const bf16x8 a8 = as_bf16x8(pa), d8 = as_bf16x8(pd);
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            const int toff = (32 * db + l32) * TR_STRIDE + 16 * ks + 4 * g;
            const u16 *dor = sm.dOt + toff;
            const u16 *qr = sm.qt + toff;
            dv[db] = mfma32(a8, join8(*(const uint2 *)dor, *(const uint2 *)(dor + 8)), dv[db]);
            dk[db] = mfma32(d8, join8(*(const uint2 *)qr, *(const uint2 *)(qr + 8)), dk[db]);
          }
        }
      }
      if (POS) {
        // diagonals of this tile pair are complete: fold them into the
        // sequence's d_pos partial (index m = i - j >= 0)
        __syncthreads();
        for (int x = tid; x < 2 * TILE - 1; x += THREADS) {
          const float val = sm.diag_acc[x];
          sm.diag_acc[x] = 0.0f;
          const int m = (qt - kt) * TILE - (x - (TILE - 1));
          if (val != 0.0f && m >= 0 && m < si.len)
            atomicAdd(&P.dpos_part[(row0 + m) * P.H + h], val);
        }
      }
    }
    if (TIME && tcur >= 0) atomicAdd(&tacc[h * P.nb + tcur], tsum);

    // dK, dV tiles: lane holds dim 32*db + l32 of key rows 32*w + c_row(r, g)
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int jl = 32 * w + c_row(r, g);
        if (jl < k_valid) {
          const int64_t idx = ((row0 + (int64_t)kt * TILE + jl) * P.H + h) * D + 32 * db + l32;
          __bf16 bk = (__bf16)dk[db][r], bv = (__bf16)dv[db][r];
          P.out0[idx] = __builtin_bit_cast(u16, bk);
          P.out1[idx] = __builtin_bit_cast(u16, bv);
        }
      }
    __syncthreads();
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
