// bf16 MFMA kernels of jagged HSTU attention for gfx950 (Sec. 4.1.1: jagged
// QKV with the relative position and relative time biases fused into the
// attention kernel, no padding and no dense<->jagged conversion).
//
// Persistent kernels pop (sequence, 64-row tile, head) items from the
// scheduler's longest-first lists:
//
//   attn_fwd   q-stationary: O_i = sum_{j<=i} silu(s_ij)/N v_j
//   attn_bwd_dkv  k-stationary: dV_j = sum_{i>=j} a_ij dO_i,
//                 dK_j = sum_{i>=j} dS_ij q_i, plus the table gradients
//                 (per-sequence diagonal partials for d_pos, binned
//                 per-work-group histograms for d_time)
//   attn_bwd_dq   q-stationary: dQ_i = sum_{j<=i} dS_ij k_j
//   attn_bwd      both item kinds in one launch (small problems); at d=64
//                 the dK/dV item of k-tile 0 also produces the dQ of q-tile
//                 0, which depends on tile pair (0, 0) alone, so the merged
//                 list has no dQ item for any sequence's first q-tile
//
// With many items per work-group the two backward item kinds run as two
// launches, each at the occupancy its own register footprint allows (the dQ
// item holds two operands and one accumulator, the dK/dV item two and two);
// with few (short sequences), one launch over a merged list balances better.
//
// with s_ij = <q_i,k_j> + pos_w[h, j-i+N-1] + time_w[h, bucket(ts_i-ts_j)],
// dS_ij = <dO_i, v_j> silu'(s_ij) / N, and the causal mask applied after the
// SiLU (a masked pair is exactly zero).
//
// Work-group = 4 wave64s on a 64x64 tile pair; each wave owns a 32x32
// quadrant (half of the stationary rows x half of the streamed rows) and all
// contractions use the 32x32x16 bf16 MFMA.  The stationary operand lives in
// registers (the dK/dV items' K and V at d=64: in LDS).  The streamed tile is
// staged in LDS once: the score-side products read it along d with 16-byte
// loads, the accumulating products (contracted over tile rows) read it
// through the gfx950 LDS transpose load, which hands each lane one column of
// 4 consecutive rows.  Score accumulators come out with one fixed stationary
// row per lane, which is exactly the operand layout of the accumulating
// product, so scores never leave registers.  The two halves of the streamed
// side are summed through LDS once per item.  The next streamed tile (with
// its bias slice and timestamps) is fetched while the current one computes:
// straight into LDS by global-to-LDS loads in the forward, through registers
// in the backward.
//
// Relative-time bias fast path: while every timestamp of the tile pair lies
// within 2^23 of the sequence's first one, |ts_i - ts_j| < 2^24 converts to
// float exactly, and bits 21..30 of that float are 4*(e+127) + m with e =
// floor(log2|x|) and m the two bits under the leading one -- the bucket
// rule's own quantities.  A 604-entry LDS table per head maps that index
// straight to the bias.  Otherwise the exact 64-bit rule is used.
#include <algorithm>

#include "internal.h"
#include "device.h"

namespace hstu {

namespace {

constexpr int THREADS = 256;     // 4 waves
constexpr int RM_PAD = 8;        // backward: row-major LDS stride D+8 bf16
constexpr int DS_STRIDE = TILE + RM_PAD;   // backward: staged dS^T tile
// Stride (floats) of the four shifted copies of a position-bias slice: at
// least 2*TILE + 3 entries, and 16 (mod 64) so that the 16 lanes of a 16-byte
// read phase, whose 4-entry windows start at 16 consecutive entries, fall on
// 16 distinct 4-bank groups of the 64 banks.
constexpr int POS_COPY = 144;
constexpr int KTAB = 608;        // float-exponent time index 0..603 (+pad)
constexpr int32_t NEAR = 1 << 23;  // |ts - ts_start| < NEAR -> float-exponent path
constexpr float L2E = 1.44269504088896341f;      // log2(e)

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
  u16 *dq_out;
  // backward outputs: row stride (elements), and with h_* set, each stored
  // gradient multiplied by silu' of h_* at the same index
  const u16 *h_dq, *h_dk, *h_dv;
  int32_t out_stride;
  void *dpos_part, *dtime_part;        // float, or fixed point (deterministic)
  int32_t H, N, nb;
  float inv_n;
  // scale of <q, k>: the forward works on x' = s alpha log2e with the biases
  // staged pre-scaled, the backward on s/alpha-scaled biases (inv_alpha)
  float alpha, inv_alpha, neg_al2e;
  float dqk_scale;                     // alpha / N: dQ and dK stores
  // the dK/dV items carry A and dS multiplied by log2e: their dK, dQ and
  // dV stores take dqk_scale / log2e and 1 / (N log2e)
  float al2e, dk_scale_l2, dv_scale_l2;
  int32_t all_heads;      // time tables of every head staged once per work-group
  int32_t fuse_dq0;       // combined backward, d=64: the dK/dV items of first
                          // k-tiles compute their q-tile's dQ (no such dQ items)
};

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

// Position-bias slice of tile pair (qt, kt): entry x (0..126) is the bias of
// local offset j_loc - i_loc = x - 63, i.e. pos_w[h, (kt-qt)*64 + x - 63 +
// N - 1]; indices outside the table are only reached by masked pairs and
// read as 0.  Thread x fetches entry x one tile ahead (pos_fetch); the store
// writes it into four LDS copies shifted by 0..3 so that 4 consecutive
// entries are one aligned 16-byte load for any lane: forward order (copy s,
// entry x - s) for the q-stationary kernels, reversed order (copy s, entry
// 126 - x - s) for the k-stationary one, whose lanes walk the offsets
// downwards.  Threads past the slice store nothing; the shifted copies of
// the first entries land in never-read tail slots of the copy before.
// The entry is multiplied by `scale` when stored (1/alpha, or the forward's
// base-2 factor).  The fetch is an unconditional load through a buffer
// resource over the head's table (an index outside it reads 0, so no clamp)
// whose scale waits for the store: a use right after the load would make
// the wave wait for it there, and with it for every load it has in flight
// (the next tile's prefetches).
struct PosEntry {
  float raw;
  bool ok;
};

// A slice of `len` entries (2*TILE - 1 for one query tile; the forward's
// two-tile items take TILE*3 - 1, entry x of the upper tile's slice being
// entry x + TILE of the lower one's), copies `COPY` floats apart.
// The table of head h as a buffer source (entries outside it read as 0).
__device__ __forceinline__ __amdgpu_buffer_rsrc_t pos_source(const KParams &P, int h) {
  const int span = 2 * P.N - 1;
  return make_rsrc(P.pos_w + (int64_t)h * span, 4u * (uint32_t)span);
}

__device__ __forceinline__ PosEntry pos_fetch(__amdgpu_buffer_rsrc_t rs, int N, int qt, int kt,
                                              int tid, int len = 2 * TILE - 1) {
  const int idx = (kt - qt) * TILE + N - TILE + tid;    // < 0 or past the table: reads 0
  const uint32_t raw = __builtin_amdgcn_raw_buffer_load_b32(rs, (int)(4u * (uint32_t)idx), 0, 0);
  return PosEntry{__uint_as_float(raw), tid < len};
}

template <bool REVERSED, int COPY = POS_COPY, int LEN = 2 * TILE - 1>
__device__ __forceinline__ void pos_store(PosEntry e, float scale, float *pos, int tid) {
  const float v = e.ok ? scale * e.raw : 0.0f;
  if (tid < LEN) {
    // copy s, entry x - s: one address, the copies at immediate offsets; for
    // x < s that is one of the last three slots of copy s - 1, which no
    // read reaches (reads stay below slot LEN <= COPY - 3)
    static_assert(LEN <= COPY - 3, "copy stride");
    float *p = pos + (REVERSED ? LEN - 1 - tid : tid);
#pragma unroll
    for (int s = 0; s < 4; ++s) p[s * (COPY - 1)] = v;
  }
}

// Aligned pointer to 4 consecutive slice entries starting at entry x0 (any
// x0 >= 0): copy x0 & 3, entry x0 - (x0 & 3).
template <int COPY = POS_COPY>
__device__ __forceinline__ const float *pos_lane(const float *pos, int x0) {
  const int s = x0 & 3;
  return pos + s * COPY + (x0 - s);
}

// Float-exponent index of a time difference held exactly in a float
// (|delta| < 2^24; see file comment).  The sign bit is not in the field.
__device__ __forceinline__ int time_index(float delta) {
  return (int)__builtin_amdgcn_ubfe(__float_as_uint(delta), 21u, 10u);
}

// Bucket of float-exponent index k (k = 0 <-> 0; 508, 512, 514 <-> 1, 2, 3;
// k >= 516 <-> k - 512), clamped to nb-1.  Indices no integer reaches map
// to some valid bucket.
__device__ __forceinline__ int bucket_of_index(int k, int nb) {
  int b = k >= 516 ? k - 512 : (k >= 514 ? 3 : (k >= 512 ? 2 : (k >= 508 ? 1 : 0)));
  return b < nb - 1 ? b : nb - 1;
}

// Scores are handled in the base-2 domain x' = x log2(e): the MFMA result is
// scaled once and the bias tables are staged pre-scaled, so that e^-x is a
// single exp2 of -x'.
//   silu(x) / N = x' / (N log2e (1 + 2^-x'));  nl = N log2e
__device__ __forceinline__ float silu2_over_n(float xs, float nl) {
  const float t = __builtin_amdgcn_exp2f(-xs);
  return xs * __builtin_amdgcn_rcpf(__builtin_fmaf(nl, t, nl));
}

// d_time is accumulated in LDS in double precision: the gfx950 LDS f64 add
// atomic runs at a few cycles per wave instruction on distinct addresses,
// while the f32 one costs hundreds.



// Time tables in dynamic LDS, one slot per head (or a single slot restaged
// per item when all heads do not fit): KTAB entries by float-exponent index,
// then the nb raw buckets for the exact path.
__device__ __forceinline__ int time_slot_floats(const KParams &P) { return KTAB + P.nb; }

// Slots of heads h0 .. h0+nh-1, back to back from `dyn`.  Each thread
// issues the loads of BATCH entries before it stores any, so staging costs a
// few memory latencies rather than one per entry (a smaller batch where the
// caller's registers are scarce).
template <int BATCH, int NT = THREADS>
__device__ __forceinline__ void stage_time_heads(const KParams &P, float *dyn, int h0, int nh,
                                                 int tid, float scale) {
  const int per = time_slot_floats(P);
  if constexpr (BATCH == 1) {
    for (int hl = 0; hl < nh; ++hl) {
      const float *tab = P.time_w + (int64_t)(h0 + hl) * P.nb;
      float *slot = dyn + hl * per;
      for (int x = tid; x < KTAB; x += NT) slot[x] = scale * tab[bucket_of_index(x, P.nb)];
      for (int x = tid; x < P.nb; x += NT) slot[KTAB + x] = scale * tab[x];
    }
    return;
  }
  const int total = nh * per;
  for (int i0 = tid; i0 < total; i0 += BATCH * NT) {
    float v[BATCH];
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int i = min(i0 + k * NT, total - 1);         // in bounds, used if < total
      const int hl = i / per, x = i - hl * per;
      const int src = x < KTAB ? bucket_of_index(x, P.nb) : x - KTAB;
      v[k] = P.time_w[(int64_t)(h0 + hl) * P.nb + src];
    }
#pragma unroll
    for (int k = 0; k < BATCH; ++k) {
      const int i = i0 + k * NT;
      if (i < total) dyn[i] = scale * v[k];
    }
  }
}

// Kernel start: every head's tables when they fit (then no per-item staging).
template <int BATCH, int NT = THREADS>
__device__ __forceinline__ void stage_all_heads(const KParams &P, float *dyn, int tid,
                                                float scale) {
  if (P.all_heads) stage_time_heads<BATCH, NT>(P, dyn, 0, P.H, tid, scale);
}

// Item start: the slot of head h (staged now if tables are per item).
template <int NT = THREADS>
__device__ __forceinline__ float *item_time_slot(const KParams &P, float *dyn, int h, int tid,
                                                 float scale) {
  if (P.all_heads) return dyn + h * time_slot_floats(P);
  stage_time_heads<1, NT>(P, dyn, h, 1, tid, scale);
  return dyn;
}

// Chunks of a 64 x D bf16 tile per thread: chunk tid + THREADS x (x < this)
// is row ch / (D/8), columns 8 (ch % (D/8)) .. +7.
template <int D> constexpr int TILE_CHUNKS = TILE * D / 8 / THREADS;

// Coalesced bf16 store of a 64 x D fp32 tile in LDS: every thread converts 8
// consecutive floats of one row, scales them by `scale` and writes them as a
// single 16-byte chunk; rows at or beyond `valid` are not written.  With
// `silu` set, each value is also multiplied by silu'(h) for the bf16 h of
// the same chunk in `hv` (a SiLU's backward fused into the store; the
// caller loads hv early so that its latency is hidden).
template <int D>
__device__ __forceinline__ void store_rows(const float *red, int tid, u16 *__restrict__ out,
                                           int row_stride, int valid, float scale, bool silu,
                                           const uint4 (&hv)[TILE_CHUNKS<D>]) {
#pragma unroll
  for (int x = 0; x < TILE_CHUNKS<D>; ++x) {
    const int ch = tid + THREADS * x;
    const int row = ch / (D / 8), c8 = ch % (D / 8);
    if (row < valid) {
      const float4 a = *(const float4 *)(red + row * D + 8 * c8);
      const float4 b = *(const float4 *)(red + row * D + 8 * c8 + 4);
      float f[8] = {scale * a.x, scale * a.y, scale * a.z, scale * a.w,
                    scale * b.x, scale * b.y, scale * b.z, scale * b.w};
      if (silu) {
        const uint32_t hw[4] = {hv[x].x, hv[x].y, hv[x].z, hv[x].w};
#pragma unroll
        for (int e = 0; e < 4; ++e) {
          f[2 * e] *= dsilu_f(__uint_as_float(hw[e] << 16));
          f[2 * e + 1] *= dsilu_f(__uint_as_float(hw[e] & 0xffff0000u));
        }
      }
      uint4 pk;
      pk.x = pack2(f[0], f[1]);
      pk.y = pack2(f[2], f[3]);
      pk.z = pack2(f[4], f[5]);
      pk.w = pack2(f[6], f[7]);
      *(uint4 *)(out + (int64_t)row * row_stride + 8 * c8) = pk;
    }
  }
}

// Cross-wave sum of a 64 x D fp32 output tile and its coalesced bf16 store.
// The two waves of each stationary row half hold partial sums over the two
// halves of the streamed side, in accumulator layout (rows 32*half +
// c_row(r, g), columns 32*db + l32).  The writer wave stores its blocks to
// LDS, its partner adds its own in place, then store_rows writes the tile.
// (The partner reads, adds and writes back its own addresses: LDS float
// atomics are far slower here even without conflicts.)
// With SUM false the writer waves' blocks are the whole result (no partner
// adds).
template <int D, bool SUM = true>
__device__ __forceinline__ void sum_store_tile(float *red, const f32x16 (&acc)[D / 32],
                                               bool writer, int half, int g, int l32,
                                               int tid, u16 *__restrict__ out,
                                               int row_stride, int valid, float scale,
                                               bool silu, const uint4 (&hv)[TILE_CHUNKS<D>]) {
  lds_barrier();
  if (writer) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[(32 * half + c_row(r, g)) * D + 32 * db + l32] = acc[db][r];
  }
  lds_barrier();
  if (SUM && !writer) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[(32 * half + c_row(r, g)) * D + 32 * db + l32] += acc[db][r];
  }
  if (SUM) lds_barrier();
  store_rows<D>(red, tid, out, row_stride, valid, scale, silu, hv);
}

// Store of a 64 x D fp32 output tile whose 32 x 32 blocks are held by one
// wave each: wave (half, cb) holds rows 32*half + c_row(r, g), columns
// 32*cb + l32 (D = 64: the four waves cover the tile).
template <int D>
__device__ __forceinline__ void quad_store_tile(float *red, const f32x16 &acc, int half, int cb,
                                                int g, int l32, int tid, u16 *__restrict__ out,
                                                int row_stride, int valid, float scale,
                                                bool silu, const uint4 (&hv)[TILE_CHUNKS<D>]) {
  static_assert(D == 64, "four 32 x 32 blocks");
  lds_barrier();
#pragma unroll
  for (int r = 0; r < 16; ++r) red[(32 * half + c_row(r, g)) * D + 32 * cb + l32] = acc[r];
  lds_barrier();
  store_rows<D>(red, tid, out, row_stride, valid, scale, silu, hv);
}

// ------------------------------------------------- swizzled DMA-fed tiles
// A 64-row tile of one head in LDS without padding: 16-byte chunk c of row r
// sits at chunk position c ^ swz_key<D, K>(r) of that row.  The LDS has 64
// banks of 4 bytes (one 256-byte line) and serves a 16-byte read in phases of
// 16 lanes, an 8-byte (or transpose) read in phases of 32 lanes.  The reads:
//   row reads: 16 lanes on 16 consecutive rows (aligned), one chunk each;
//   transpose reads: 32 lanes on 4 consecutive rows (aligned) x 4 chunks
//     (an aligned group of four), and the same 8 rows further.
// SWZ_CF makes both conflict-free.  D = 64 (two rows per line, half r & 1):
// the key takes the 8 values over the 8 rows of each half of a 16-row group,
// and bit 2 of it (which picks the aligned chunk group) differs between rows
// r and r+2.  D = 128 (one row per line): the key takes 16 values over 16
// rows, and its chunk group (bits 2-3) differs between the 4 rows of a
// transpose read.  SWZ_ROWS8 (key r & 7) leaves 2-way conflicts at D = 64
// (rows r and r+8 of a row read share a bank group) but gives rows 8 and 16
// apart the same key, so their addresses differ by an immediate offset: the
// d=64 forward, bound by its vector ALU work, keeps it (the conflict-free key
// costs it 11 registers and a wave per SIMD, 9% on the Zipf batch).  Tiles
// are filled straight from global memory by the gfx950 global-to-LDS loads
// (each lane's 16 bytes land at the instruction's LDS base + 16 * lane, a
// contiguous write), so no registers or LDS-store instructions stage them.
typedef __attribute__((address_space(3))) void lds_void;

enum SwzKind { SWZ_ROWS8 = 0, SWZ_CF = 1 };

template <int D, int K>
__device__ __forceinline__ int swz_key(int r) {
  static_assert(D == 64 || D == 128, "head dim");
  if (K == SWZ_ROWS8) return r & 7;
  return D == 64 ? ((((r >> 1) & 1) << 2) | ((r >> 2) & 3))
                 : (((r & 3) << 2) | ((r >> 2) & 3));
}

template <int D, int K>
__device__ __forceinline__ int swz(int r, int c) {
  return r * D + 8 * (c ^ swz_key<D, K>(r));
}

// Key of the forward's K/V tiles.
template <int D> constexpr int FWD_SWZ = D == 64 ? SWZ_ROWS8 : SWZ_CF;

typedef int i32x4 __attribute__((ext_vector_type(4)));

// Raw buffer descriptor words over `bytes` bytes from `base` (read from the
// first active lane, so the descriptor sits in scalar registers).
__device__ __forceinline__ i32x4 rsrc_words(const void *base, uint32_t bytes) {
  const uint64_t a = (uint64_t)(uintptr_t)base;
  i32x4 r;
  r[0] = (int)__builtin_amdgcn_readfirstlane((uint32_t)a);
  r[1] = (int)(__builtin_amdgcn_readfirstlane((uint32_t)(a >> 32)) & 0xffffu);   // stride 0
  r[2] = (int)__builtin_amdgcn_readfirstlane(bytes);
  r[3] = 0x00020000;
  return r;
}

// LDS byte address of a pointer into the work-group's shared memory: the
// low 32 bits of its generic address (the shared aperture begins at a
// multiple of 2^32), without the null test an address-space cast emits.
__device__ __forceinline__ uint32_t lds_addr(const void *p) { return (uint32_t)(uintptr_t)p; }

// One 16-byte-per-lane buffer load into LDS (lane i's bytes land at LDS
// address lds + 16 i).  Issued from inline assembly on purpose: the compiler
// cannot tell which LDS bytes such a load writes, so after the builtin form
// it makes the wave wait for the load before its next LDS read -- also when
// that read is of the other buffer, which would turn every prefetch of the
// next tile into a synchronous load.  The callers wait for these loads
// themselves (wait_vm) before the barrier that publishes the tile.  The
// leading s_nop covers the wait states a vector-memory instruction needs
// after a vector instruction wrote the scalar registers it reads.
__device__ __forceinline__ void buf_load_lds16(const i32x4 &r, uint32_t lds_addr, uint32_t voff) {
  asm volatile("s_nop 4\n\ts_mov_b32 m0, %0\n\tbuffer_load_dwordx4 %1, %2, 0 offen lds"
               :
               : "s"(__builtin_amdgcn_readfirstlane(lds_addr)), "v"(voff), "s"(r)
               : "memory", "m0");
}

// Issue the loads of a 64 x D tile (rows of `row_stride` elements from
// `base`) into `lds`; wave w of NW covers 1/NW of it.  Rows at or beyond `valid`
// read as zeros (finite data that the caller always masks out): the loads go
// through a buffer resource that ends after row valid-1, so each lane's
// offsets are the same for every tile of a given row stride and stay in
// registers across a loop over tiles (no per-tile address arithmetic).
template <int D, int K, int NW = 4>
__device__ __forceinline__ void dma_tile(const u16 *__restrict__ base, int valid, int row_stride,
                                         u16 *lds, int w, int lane) {
  constexpr int CPR = D / 8;                       // 16-byte chunks per row
  constexpr int IPW = TILE * CPR / 64 / NW;        // load instructions per wave (NW waves)
  const int rows = valid < TILE ? (valid > 0 ? valid : 0) : TILE;
  const i32x4 rs = rsrc_words(base, 2u * (uint32_t)rows * (uint32_t)row_stride);
#pragma unroll
  for (int x = 0; x < IPW; ++x) {
    const int pos = (w * IPW + x) * 64 + lane;     // chunk position in LDS
    const int r = pos / CPR;
    const int c = (pos % CPR) ^ swz_key<D, K>(r);
    buf_load_lds16(rs,
                   lds_addr(lds + (w * IPW + x) * 64 * 8),
                   2u * (uint32_t)(r * row_stride + 8 * c));
  }
}

// As dma_tile, from a sequence-wide source `rs` (one head's rows of a whole
// sequence, built once per item; rows at or beyond the sequence's length
// read as zeros): the tile `row0_bytes` bytes in, its offset added to each
// lane's offset (no per-tile descriptor).
template <int D, int K, int NW = 4>
__device__ __forceinline__ void dma_tile_at(const i32x4 &rs, uint32_t row0_bytes, int row_stride,
                                            u16 *lds, int w, int lane) {
  constexpr int CPR = D / 8;
  constexpr int IPW = TILE * CPR / 64 / NW;
#pragma unroll
  for (int x = 0; x < IPW; ++x) {
    const int pos = (w * IPW + x) * 64 + lane;
    const int r = pos / CPR;
    const int c = (pos % CPR) ^ swz_key<D, K>(r);
    buf_load_lds16(rs,
                   lds_addr(lds + (w * IPW + x) * 64 * 8),
                   row0_bytes + 2u * (uint32_t)(r * row_stride + 8 * c));
  }
}

// Compiler-only barrier for memory operations: keeps the prefetch loads
// issued above it from being sunk toward their use in the next step (which
// would expose their latency there); emits no instruction and no wait.
__device__ __forceinline__ void issue_fence() { asm volatile("" ::: "memory"); }

// Wait for this wave's outstanding global loads, the LDS-filling ones
// included (they count as vector memory operations, not LDS operations).
__device__ __forceinline__ void wait_vm() { __builtin_amdgcn_s_waitcnt(0x0f70); }

template <int D, int K>
__device__ __forceinline__ bf16x8 sread_rm(const u16 *lds, int row, int col) {
  return *(const bf16x8 *)(lds + swz<D, K>(row, col >> 3));
}

// As read_tr, on a swizzled tile.
template <int D, int K>
__device__ __forceinline__ bf16x8 sread_tr(const u16 *lds, int krow, int ncol, int lane) {
  const int c = lane & 15;
  const int row = krow + (c >> 2);
  const int col = ncol + ((lane >> 4) & 1) * 16 + 4 * (c & 3);
  const u16 *p0 = lds + swz<D, K>(row, col >> 3) + (col & 7);
  const u16 *p1 = lds + swz<D, K>(row + 8, col >> 3) + (col & 7);
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)p0);
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)p1);
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  const v8i16 x = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, x);
}

// sread_tr from per-lane byte offsets (the two halves' p0 and p1 relative
// to the tile) instead of its coordinates.
__device__ __forceinline__ bf16x8 sread_tr_at(const u16 *lds, uint32_t off0, uint32_t off1) {
  const v4i16 lo = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)((const char *)lds + off0));
  const v4i16 hi = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16 *)((const char *)lds + off1));
  typedef short v8i16 __attribute__((ext_vector_type(8)));
  const v8i16 x = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
  return __builtin_bit_cast(bf16x8, x);
}

// Forward shared memory: two K/V buffers (tile kt computes from one while
// tile kt+1 streams into the other), per-parity bias slices, a three-slot
// "far timestamp" flag.  An item's output is summed across waves in the
// buffer of its last tile.
// Position-slice copy stride and slice length of the forward's items of QT
// query tiles (the stride again 16 mod 64 floats, see POS_COPY).
template <int QT> constexpr int FWD_POS_COPY = QT == 1 ? POS_COPY : 208;
template <int QT> constexpr int FWD_POS_LEN = TILE * (QT + 1) - 1;

template <int D, int QT>
struct FwdSmem {
  u16 tile[2][2][TILE * D];              // [buffer][K, V]
  alignas(16) float pos[2][4 * FWD_POS_COPY<QT>];
  alignas(16) float ts32[2][TILE];
  int64_t ts64[2][TILE];
  int flag[3];
  int next[2];                           // item index published by thread 0,
                                         // by parity of the publishing item
};

// A work-list item decoded: sequence start and length, tile, head.
struct Item {
  int64_t start;
  int32_t len, tile, h;
};

__device__ __forceinline__ Item load_item(const KParams &P, int idx) {
  const WorkEntry e = P.list[idx / P.H];
  Item it;
  it.start = e.start;
  it.len = e.len;
  it.tile = e.tile;
  it.h = idx % P.H;
  return it;
}

// Streams an item's first key tile into (kbuf, vbuf) and fetches its bias
// slice and timestamps into registers.  Timestamps of rows past the
// sequence repeat its last row (those rows are always masked).
// Streams an item's first key tile into (kbuf, vbuf) and fetches its bias
// slice and this lane's timestamps into registers (query tile QT*tile + sub
// for the lane's wave).  Timestamps of rows past the sequence repeat its last
// row (those rows are always masked).
template <int D, bool POS, bool TIME, int QT>
__device__ __forceinline__ void fwd_item_start(const KParams &P, const Item &it, u16 *kbuf,
                                               u16 *vbuf, int w, int lane, int tid, int i_loc,
                                               int sub, int row_stride, int64_t &ts_start,
                                               int64_t &ts_i, int64_t &ts_k, PosEntry &pos_v) {
  const int64_t hb = (it.start * P.H + it.h) * D;
  dma_tile<D, FWD_SWZ<D>, 4 * QT>(P.k + hb, it.len, row_stride, kbuf, w, lane);
  dma_tile<D, FWD_SWZ<D>, 4 * QT>(P.v + hb, it.len, row_stride, vbuf, w, lane);
  if (TIME) {
    const int qt = QT * it.tile + sub;
    const int q_valid = it.len - qt * TILE;
    ts_start = P.ts[it.start];
    ts_i = P.ts[it.start + (int64_t)qt * TILE + (i_loc < q_valid ? i_loc : q_valid - 1)];
    if (tid < TILE) ts_k = P.ts[it.start + (tid < it.len ? tid : it.len - 1)];
  }
  if (POS) pos_v = pos_fetch(pos_source(P, it.h), P.N, QT * it.tile + QT - 1, 0, tid,
                             FWD_POS_LEN<QT>);
}

// Cross-wave sum of the O tile of one query tile (waves with `mine` set, in
// two key halves: `writer` stores, its partner adds) and its coalesced bf16
// store by all NT threads; rows at or beyond `valid` are not written.
template <int D, int NT>
__device__ __forceinline__ void fwd_store_o(float *red, const f32x16 (&acc)[D / 32], bool mine,
                                            bool writer, int half, int g, int l32, int tid,
                                            u16 *__restrict__ out, int row_stride, int valid) {
  lds_barrier();
  if (mine && writer) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[(32 * half + c_row(r, g)) * D + 32 * db + l32] = acc[db][r];
  }
  lds_barrier();
  if (mine && !writer) {
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r)
        red[(32 * half + c_row(r, g)) * D + 32 * db + l32] += acc[db][r];
  }
  lds_barrier();
  constexpr int CH = TILE * D / 8 / NT;
#pragma unroll
  for (int x = 0; x < CH; ++x) {
    const int ch = tid + NT * x;
    const int row = ch / (D / 8), c8 = ch % (D / 8);
    if (row < valid) {
      const float4 a = *(const float4 *)(red + row * D + 8 * c8);
      const float4 b = *(const float4 *)(red + row * D + 8 * c8 + 4);
      uint4 pk;
      pk.x = pack2(a.x, a.y);
      pk.y = pack2(a.z, a.w);
      pk.z = pack2(b.x, b.y);
      pk.w = pack2(b.z, b.w);
      *(uint4 *)(out + (int64_t)row * row_stride + 8 * c8) = pk;
    }
  }
}

// ---------------------------------------------------------------- forward
// An item is QT consecutive query tiles of one head: QT = 1 (four waves, 64
// rows) or QT = 2 (eight waves, 128 rows) -- with two, every streamed K/V
// tile serves twice the query rows, which halves the K/V traffic of long
// sequences (the forward on deep batches is bound by it).  Wave w covers
// query tile QT*tile + sub (sub = w / 4), query half w & 1 and key half
// (w / 2) & 1; the item runs over the key tiles of its highest query tile,
// and a wave whose tile ends earlier (or is past the sequence) idles through
// the remaining steps' barriers.
//
// One work-group barrier per key tile: the barrier of tile kt publishes its
// DMA-filled buffers and bias slices, and proves every wave is done with
// tile kt-1, whose buffer then takes tile kt+1.  Items are pipelined: each
// work-group's first two items are static (the list's head, longest first,
// the second ones paired in reverse), the pop for the item after next is
// issued one step before an item's last, and an
// item's last tile streams the next item's first key tile, query rows, bias
// slice and timestamps, so no item starts with an exposed memory latency.
template <int D, bool POS, bool TIME, int QT>
__global__ void __launch_bounds__(THREADS * QT, QT == 1 ? 2 : 1)
attn_fwd_kernel(KParams P) {
  constexpr int NT = THREADS * QT, NW = 4 * QT;
  constexpr int PCOPY = FWD_POS_COPY<QT>, PLEN = FWD_POS_LEN<QT>;
  __shared__ FwdSmem<D, QT> sm;
  extern __shared__ float dyn[];              // time tables (see item_time_slot)
  const int n_items = P.ctrl[QT == 1 ? CTRL_N_ENTRIES : CTRL_N_PAIRS] * P.H;
  int cur = blockIdx.x;
  // second static item: the list's next G items paired in reverse, so the
  // work-group with the longest first item gets the shortest second one
  int nxt = 2 * gridDim.x - 1 - blockIdx.x;
  if (cur >= n_items) return;
  const int tid0 = threadIdx.x;
  if (tid0 < 3) sm.flag[tid0] = 0;
  int phase = 0;

  Item it = load_item(P, cur);
  int item_no = 0;                            // items done by this work-group
  int64_t ts_start = 0, ts_i = 0, ts_k = 0;
  PosEntry pos_v{0.0f, false};
  bf16x8 qreg[D / 16];
  {
    const int lane = tid0 & 63, g = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid0 >> 6);
    const int i_loc = 32 * (w & 1) + l32, sub = w >> 2;
    fwd_item_start<D, POS, TIME, QT>(P, it, sm.tile[0][0], sm.tile[0][1], w, lane, tid0, i_loc,
                                     sub, P.H * D, ts_start, ts_i, ts_k, pos_v);
    const int qt0 = QT * it.tile + sub;
    load_stationary<D>(P.q + ((it.start + (int64_t)qt0 * TILE) * P.H + it.h) * D, i_loc,
                       it.len - qt0 * TILE, P.H * D, g, qreg);
  }
  // the tables after the first item's loads: both latencies overlap
  if (TIME) stage_all_heads<8, NT>(P, dyn, tid0, L2E);

  for (;;) {
    // Lane-derived values are rebuilt per item from an opaque copy of the
    // thread index: otherwise the compiler hoists dozens of per-lane
    // addresses out of the persistent loop and pins their registers.
    int tid = tid0;
    asm volatile("" : "+v"(tid));
    int row_stride = P.H * D;
    asm volatile("" : "+s"(row_stride));
    const int lane = tid & 63, g = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wi = w & 1, wj = (w >> 1) & 1, sub = w >> 2;   // query half, key half, tile
    const int qt = QT * it.tile + sub, h = it.h;
    const int q_valid = it.len - qt * TILE;
    const int i_loc = 32 * wi + l32;
    const int qt_hi = QT * it.tile + QT - 1;                  // the slice's reference tile
    // Per-lane byte offsets from a tile's base of this wave's K reads (one
    // per 16-column step) and V transpose reads (per 32-column block, its
    // rows and rows + 8; the second 16 keys lie 16 rows further, which both
    // keys map to a fixed distance, as the rows-of-8 key does for rows + 8
    // at d=64), kept opaque so that every read is one add of the buffer's
    // base plus an immediate, not a re-derived address
    constexpr bool V_HI = D == 128;           // rows + 8: an offset of its own
    uint32_t koff[D / 16], voff[D / 32], vofh[V_HI ? D / 32 : 1];
#pragma unroll
    for (int ks = 0; ks < D / 16; ++ks) {
      koff[ks] = 2u * (uint32_t)swz<D, FWD_SWZ<D>>(32 * wj + l32, 2 * ks + g);
      asm volatile("" : "+v"(koff[ks]));
    }
    {
      const int c = lane & 15;
      const int vrow = 32 * wj + 4 * g + (c >> 2);
#pragma unroll
      for (int db = 0; db < D / 32; ++db) {
        const int col = 32 * db + ((lane >> 4) & 1) * 16 + 4 * (c & 3);
        voff[db] = 2u * (uint32_t)(swz<D, FWD_SWZ<D>>(vrow, col >> 3) + (col & 7));
        asm volatile("" : "+v"(voff[db]));
        if constexpr (V_HI) {
          vofh[db] = 2u * (uint32_t)(swz<D, FWD_SWZ<D>>(vrow + 8, col >> 3) + (col & 7));
          asm volatile("" : "+v"(vofh[db]));
        }
      }
    }
    const int kt_end = min(qt_hi, (it.len - 1) / TILE);       // the item's last key tile
    const int pos_x = TILE - 1 + TILE * (QT - 1 - sub);       // slice entry of offset 0
    // this lane's bias-slice reads (4 consecutive entries of one copy, see
    // pos_lane) at a per-item byte offset from the slice buffer, kept opaque
    // like the tile offsets
    uint32_t poff = 0;
    if (POS) {
      const int x0 = 32 * wj + 4 * g - i_loc + pos_x;
      poff = 4u * (uint32_t)((x0 & 3) * PCOPY + (x0 - (x0 & 3)));
      asm volatile("" : "+v"(poff));
    }

    float ts_i32 = 0.0f;
    bool q_far = false;
    float *ktab = dyn;
    if (TIME) {
      const int64_t rel = ts_i - ts_start;
      ts_i32 = (float)(int32_t)rel;
      q_far = rel >= NEAR || rel <= -NEAR;
      ktab = item_time_slot<NT>(P, dyn, h, tid, L2E);
    }
    const int64_t ts_i_item = ts_i, ts_start_item = ts_start;
    // the item's K and V rows of head h: one source each for its tiles
    const uint32_t seq_bytes = 2u * (uint32_t)it.len * (uint32_t)row_stride;
    const uint32_t tile_bytes = 2u * (uint32_t)TILE * (uint32_t)row_stride;
    const i32x4 rs_k = rsrc_words(P.k + (it.start * P.H + h) * D, seq_bytes);
    const i32x4 rs_v = rsrc_words(P.v + (it.start * P.H + h) * D, seq_bytes);
    const __amdgpu_buffer_rsrc_t rs_pos = pos_source(P, POS ? h : 0);

    int nxt2 = 0;
    const bool has_next = nxt < n_items;
    Item nit = it;
    if (has_next) nit = load_item(P, nxt);

    f32x16 oacc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) oacc[db][r] = 0.0f;

    for (int kt = 0; kt <= kt_end; ++kt, ++phase) {
      const int pb = phase & 1, fs = phase % 3;
      const bool last = kt == kt_end;          // the item's last step
      const bool diag = kt == qt;              // this wave's diagonal tile
      const bool active = kt <= qt;            // this wave has work in the step
      if (POS) pos_store<false, PCOPY, PLEN>(pos_v, P.inv_alpha, sm.pos[pb], tid);
      if (TIME) {
        bool far = q_far;
        if (tid < TILE) {
          const int64_t rel = ts_k - ts_start_item;
          sm.ts32[pb][tid] = (float)(int32_t)rel;
          sm.ts64[pb][tid] = ts_k;
          far |= rel >= NEAR || rel <= -NEAR;
        }
        if (far) sm.flag[fs] = 1;
      }
      wait_vm();
      lds_barrier();
      const bool slow = TIME && sm.flag[fs] != 0;
      if (TIME && tid == 0) sm.flag[(phase + 2) % 3] = 0;
      // pop the item after next one step before the last (as late as the
      // atomic's latency allows), older than this step's loads, so that no
      // wait for them also waits for the atomic
      if (kt == (kt_end > 0 ? kt_end - 1 : 0) && tid == 0)
        nxt2 = atomicAdd(P.pop, 1);     // + 2 gridDim.x where it is published
      if (!last) {         // stream the next key tile into the other buffer
        const int k_valid = it.len - (kt + 1) * TILE;
        const int64_t r0 = it.start + (int64_t)(kt + 1) * TILE;
        dma_tile_at<D, FWD_SWZ<D>, NW>(rs_k, (uint32_t)(kt + 1) * tile_bytes, row_stride,
                                       sm.tile[pb ^ 1][0], w, lane);
        dma_tile_at<D, FWD_SWZ<D>, NW>(rs_v, (uint32_t)(kt + 1) * tile_bytes, row_stride,
                                       sm.tile[pb ^ 1][1], w, lane);
        if (TIME && tid < TILE)
          ts_k = P.ts[r0 + (tid < k_valid ? tid : k_valid - 1)];
        if (POS) pos_v = pos_fetch(rs_pos, P.N, qt_hi, kt + 1, tid, PLEN);
      } else if (has_next) {   // ... or the next item's first one
        fwd_item_start<D, POS, TIME, QT>(P, nit, sm.tile[pb ^ 1][0], sm.tile[pb ^ 1][1], w,
                                         lane, tid, i_loc, sub, row_stride, ts_start, ts_i,
                                         ts_k, pos_v);
      }
      issue_fence();
      const u16 *kt_lds = sm.tile[pb][0];
      const u16 *vt_lds = sm.tile[pb][1];

      // S^T quadrant [32 keys x 32 queries] = K_wj Q_wi^T, with the position
      // bias as the accumulator's initial value; this lane's keys sit at
      // 32 wj + 4 g + 8 q4 + c
      const int kb = 32 * wj + 4 * g;
      f32x16 s;
      if (active) {
#pragma unroll
        for (int r = 0; r < 16; ++r) s[r] = 0.0f;
        if (POS) {
          const float *pl = (const float *)((const char *)sm.pos[pb] + poff);
#pragma unroll
          for (int q4 = 0; q4 < 4; ++q4) {
            const float4 pbv = *(const float4 *)(pl + 8 * q4);
            s[4 * q4 + 0] = pbv.x; s[4 * q4 + 1] = pbv.y;
            s[4 * q4 + 2] = pbv.z; s[4 * q4 + 3] = pbv.w;
          }
        }
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks)
          s = mfma32(*(const bf16x8 *)((const char *)kt_lds + koff[ks]), qreg[ks], s);
      }
      if (last && has_next) {  // the query rows are free: fetch the next item's
        const int nqt = QT * nit.tile + sub;
        load_stationary<D>(P.q + ((nit.start + (int64_t)nqt * TILE) * P.H + nit.h) * D, i_loc,
                           nit.len - nqt * TILE, row_stride, g, qreg);
      }
      if (!active) continue;

      // x' = (s + pos/alpha) alpha log2e + time bias', A = silu(x)/N, then
      // O_wi += A V, one 16-key half at a time (half the temporaries live at
      // once)
      const float nl = (float)P.N * L2E;
      const float al2e = P.alpha * L2E;
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        float x[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = s[8 * hh + e] * al2e;
        if (TIME) {
          if (!slow) {
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              const float4 t4 = *(const float4 *)(sm.ts32[pb] + kb + 8 * (2 * hh + q));
              x[4 * q + 0] += ktab[time_index(ts_i32 - t4.x)];
              x[4 * q + 1] += ktab[time_index(ts_i32 - t4.y)];
              x[4 * q + 2] += ktab[time_index(ts_i32 - t4.z)];
              x[4 * q + 3] += ktab[time_index(ts_i32 - t4.w)];
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              x[e] += ktab[KTAB + time_bucket(ts_i_item - sm.ts64[pb][kb + c_row(8 * hh + e, 0)],
                                              P.nb)];
          }
        }
        float av[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) av[e] = silu2_over_n(x[e], nl);
        // the diagonal tile is the only one with keys past the query (and
        // the only one that can hold rows past the sequence, zero rows that
        // the same mask removes)
        if (diag) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (kb + c_row(8 * hh + e, 0) > i_loc) av[e] = 0.0f;
        }
        uint4 pk;
        pk.x = pack2(av[0], av[1]);
        pk.y = pack2(av[2], av[3]);
        pk.z = pack2(av[4], av[5]);
        pk.w = pack2(av[6], av[7]);
        const bf16x8 pa = as_bf16x8(pk);
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
          oacc[db] = mfma32(pa,
                            sread_tr_at(vt_lds, voff[db] + hh * 16 * D * 2,
                                        (V_HI ? vofh[V_HI ? db : 0] : voff[db] + 8 * D * 2) +
                                            hh * 16 * D * 2),
                            oacc[db]);
      }
    }

    // the popped index goes out through the epilogue's barriers; sum the
    // two key halves of each query tile in the last tile's buffer, store O
    // (bf16)
    if (tid == 0) sm.next[item_no & 1] = nxt2 + 2 * (int)gridDim.x;
#pragma unroll
    for (int sq = 0; sq < QT; ++sq) {
      const int tq = QT * it.tile + sq;
      fwd_store_o<D, NT>((float *)sm.tile[(phase - 1) & 1], oacc, sub == sq, wj == 0, wi, g,
                         l32, tid, P.out0 + ((it.start + (int64_t)tq * TILE) * P.H + h) * D,
                         row_stride, it.len - tq * TILE);
    }
    if (!has_next) break;
    cur = nxt;
    it = nit;
    nxt = sm.next[item_no & 1];
    ++item_no;
  }
}

// ------------------------------------------------------------ backward
// The backward kernel stages its streamed tiles through registers into a
// padded row-major LDS tile (measured faster here than the forward's
// DMA-filled buffers: the backward is register-bound and the staging
// overlaps with its longer tile step) and works in natural units on N A and
// N dS, with 1/N applied to the accumulated results.

// A 64-row tile of one head, D bf16 per row, moved global -> registers ->
// LDS in 16-byte chunks; rows at or beyond `valid` are zeros, so padded
// keys/queries contribute exact zeros to every product.
template <int D>
struct TileRegs {
  static constexpr int CPT = TILE_CHUNKS<D>;   // chunks per thread
  uint4 c[CPT];

  // Rows at or beyond `valid` read as zeros: the loads go through a buffer
  // resource that ends after row valid-1, so the per-thread offsets are the
  // same for every tile of a given row stride (one register per chunk).
  __device__ __forceinline__ void load(const u16 *__restrict__ tile_base,
                                       int valid, int row_stride, int tid) {
    const int rows = valid < TILE ? (valid > 0 ? valid : 0) : TILE;
    const __amdgpu_buffer_rsrc_t rs =
        make_rsrc(tile_base, 2u * (uint32_t)rows * (uint32_t)row_stride);
#pragma unroll
    for (int x = 0; x < CPT; ++x) {
      const int ch = tid + THREADS * x;
      c[x] = buf_load16(rs, 2u * (uint32_t)((ch / (D / 8)) * row_stride + (ch % (D / 8)) * 8));
    }
  }
  // The 64-row tile `row0_bytes` bytes into a sequence-wide source `rs`
  // (one head's rows of a whole sequence, built once per item; rows at or
  // beyond the sequence's length read as zeros), with no per-tile
  // descriptor: the tile's offset is added to each lane's offset.  Sizes
  // and offsets fit 32 bits: a sequence's rows span at most 2 * 65536 *
  // (64 * 128) bytes = 2^30 under the library's limits on max_len, H, d.
  __device__ __forceinline__ void load_at(__amdgpu_buffer_rsrc_t rs, uint32_t row0_bytes,
                                          int row_stride, int tid) {
#pragma unroll
    for (int x = 0; x < CPT; ++x) {
      const int ch = tid + THREADS * x;
      c[x] = buf_load16(rs, row0_bytes + 2u * (uint32_t)((ch / (D / 8)) * row_stride +
                                                         (ch % (D / 8)) * 8));
    }
  }
  __device__ __forceinline__ void store(u16 *lds, int tid) const {
#pragma unroll
    for (int x = 0; x < CPT; ++x) {
      const int ch = tid + THREADS * x;
      *(uint4 *)(lds + (ch / (D / 8)) * (D + RM_PAD) + (ch % (D / 8)) * 8) = c[x];
    }
  }
};

// 8 consecutive bf16 of row `row` of a row-major LDS tile, from column col.
__device__ __forceinline__ bf16x8 read_rm(const u16 *lds, int stride, int row, int col) {
  return *(const bf16x8 *)(lds + row * stride + col);
}

// Operand holding, for lane l, column ncol + (l & 31) of rows krow .. krow+3
// and krow+8 .. krow+11 of a row-major LDS tile (krow already includes this
// lane's 4*(l/32)), via two LDS transpose loads.  Within a 16-lane group,
// lane c addresses row (c>>2), columns 4*(c&3)..+3 of its group's 16-column
// slab; the transpose hands lane i the column slab+i of the four rows.
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
  alignas(16) float ts32[TILE];          // streamed-tile timestamps - ts_start (exact
                                         // floats on the fast path, |value| < 2^23)
  int64_t ts64[TILE];                    // raw streamed-tile timestamps
  int flag[2];                           // "some timestamp is far" (parity-buffered)
  int item;
};

// Per-lane running sum of d_time contributions (dS multiplied by log2e, as
// the dK/dV items carry it; the table partials keep that factor, which the
// finalize pass divides out) over one float-exponent time index (the lane's
// pairs visit non-decreasing indices when timestamps are ordered, so a run
// ends only when its index changes); a finished run goes to its bucket of
// the work-group's histogram `hist`.  A run is opened by
// the first index of the item's first tile (start), so adding needs no test
// for an empty run.
template <typename A>
struct TimeRun {
  typedef typename A::L L;
  float sum = 0.0f;
  int cur = -1;
  __device__ __forceinline__ void start(int k) { cur = cur < 0 ? k : cur; }
  __device__ __forceinline__ void add(L *hist, int nb, int k, float v) {
    const bool change = k != cur;
    if (change) atomicAdd(&hist[bucket_of_index(cur, nb)], A::lds(sum));
    sum = change ? v : sum + v;
    cur = k;
  }
  __device__ __forceinline__ void flush(L *hist, int nb) {
    if (cur >= 0) atomicAdd(&hist[bucket_of_index(cur, nb)], A::lds(sum));
    cur = -1;
    sum = 0.0f;
  }
};


// The backward kernels work with N dS and N A (the 1/N of both is applied
// once, to the accumulated dQ, dK, dV tiles at their store and to the table
// gradients when they are finalized).

// Table-gradient accumulation types: LDS sums in double and global partials
// in float, or (deterministic mode) both as 64-bit fixed point, whose
// integer additions give the same result in any order.
template <bool DET> struct TabAcc {
  typedef double L;
  typedef float G;
  static __device__ __forceinline__ L lds(float v) { return (double)v; }
  static __device__ __forceinline__ G glob(L v) { return (float)v; }
};
template <> struct TabAcc<true> {
  typedef unsigned long long L;
  typedef unsigned long long G;
  static __device__ __forceinline__ L lds(float v) { return to_fix(v); }
  static __device__ __forceinline__ G glob(L v) { return v; }
};

// The backward kernels' persistent loop: a work-group's first item is
// static (its block index in the longest-first list) and every item pops the
// one after it at its last tile step, so the atomic's latency hides behind
// that step instead of separating items, while a work-group still takes its
// next item only when it is nearly free (greedy longest-first assignment).
// The popped index travels through `nxt` (thread 0) and `slot`.
// The pop's raw return is kept until take_next adds the grid size (the
// first gridDim.x items are static), so that no arithmetic on it sits next
// to the atomic.
__device__ __forceinline__ void pop_next(const KParams &P, int tid, int &nxt) {
  if (tid == 0) nxt = atomicAdd(P.pop, 1);
}

__device__ __forceinline__ int take_next(int *slot, int tid, int nxt) {
  if (tid == 0) *slot = nxt + (int)gridDim.x;
  lds_barrier();
  return *slot;
}

// A work-list entry carries its sequence's start and length.
__device__ __forceinline__ SeqInfo entry_seq(const WorkEntry &e) {
  SeqInfo si;
  si.start = e.start;
  si.len = e.len;
  si.ntiles = (e.len + TILE - 1) / TILE;
  return si;
}

// --------------------------------------------------------------------- dQ
// One q-stationary item: dQ_i = sum_{j<=i} dS_ij k_j for a 64-row query tile
// of one head, recomputing S and dA = dO V^T tile by tile.
template <int D, bool POS, bool TIME>
__device__ __forceinline__ void dq_item(const KParams &P, StreamSmem<D> &sm, float *dyn,
                                        const int tid0, const WorkEntry e, const int h,
                                        int &phase, int &nxt) {
  constexpr int ST = D + RM_PAD;
    int tid = tid0;
    asm volatile("" : "+v"(tid));
    int row_stride = P.H * D;
    asm volatile("" : "+s"(row_stride));
    const int lane = tid & 63, g = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wi = w & 1, wj = w >> 1;

    const SeqInfo si = entry_seq(e);
    const int qt = e.tile;
    const int q_valid = si.len - qt * TILE;
    const int i_loc = 32 * wi + l32;
    const int64_t qoff = ((si.start + (int64_t)qt * TILE) * P.H + h) * D;
    const int64_t ooff = (si.start + (int64_t)qt * TILE) * P.out_stride + h * D;
    const bool fuse = P.h_dq != nullptr;

    // every load of the item's start is issued before any of them is used,
    // so the start costs one memory latency; timestamps of rows past the
    // sequence repeat its last row (those rows are always masked)
    bf16x8 qreg[D / 16], doreg[D / 16];
    load_stationary<D>(P.q + qoff, i_loc, q_valid, row_stride, g, qreg);
    load_stationary<D>(P.dO + qoff, i_loc, q_valid, row_stride, g, doreg);
    // the sequence's K and V rows of head h, each one source for the item
    const uint32_t seq_bytes = 2u * (uint32_t)si.len * (uint32_t)row_stride;
    const __amdgpu_buffer_rsrc_t rs_k = make_rsrc(P.k + (si.start * P.H + h) * D, seq_bytes);
    const __amdgpu_buffer_rsrc_t rs_v = make_rsrc(P.v + (si.start * P.H + h) * D, seq_bytes);
    const uint32_t tile_bytes = 2u * (uint32_t)TILE * (uint32_t)row_stride;
    TileRegs<D> kr, vr;
    kr.load_at(rs_k, 0u, row_stride, tid);
    vr.load_at(rs_v, 0u, row_stride, tid);
    int64_t ts_start = 0, ts_i = 0, ts_k = 0;
    if (TIME) {
      ts_start = P.ts[si.start];
      ts_i = P.ts[si.start + (int64_t)qt * TILE + (i_loc < q_valid ? i_loc : q_valid - 1)];
      if (tid < TILE) ts_k = P.ts[si.start + (tid < si.len ? tid : si.len - 1)];
    }
    const __amdgpu_buffer_rsrc_t rs_pos = pos_source(P, POS ? h : 0);
    PosEntry pos_v = POS ? pos_fetch(rs_pos, P.N, qt, 0, tid) : PosEntry{0.0f, false};

    float ts_i32 = 0.0f;
    bool q_far = false;
    float *ktab = dyn;
    if (TIME) {
      // the work-group's tables, staged at its first item after that item's
      // loads (both latencies overlap)
      if (phase == 0) stage_all_heads<D == 64 ? 8 : 1>(P, dyn, tid, P.inv_alpha);
      const int64_t rel = ts_i - ts_start;
      ts_i32 = (float)(int32_t)rel;
      q_far = rel >= NEAR || rel <= -NEAR;
      ktab = item_time_slot(P, dyn, h, tid, P.inv_alpha);
    }

    f32x16 acc[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[db][r] = 0.0f;

    for (int kt = 0; kt <= qt; ++kt, ++phase) {
      lds_barrier();
      kr.store(sm.t.a, tid);
      vr.store(sm.t.b, tid);
      if (POS) pos_store<false>(pos_v, P.inv_alpha, sm.pos, tid);
      if (TIME) {
        bool far = q_far;
        if (tid < TILE) {
          const int64_t rel = ts_k - ts_start;
          sm.ts32[tid] = (float)(int32_t)rel;
          sm.ts64[tid] = ts_k;
          far |= rel >= NEAR || rel <= -NEAR;
        }
        if (far) sm.flag[phase & 1] = 1;
      }
      lds_barrier();
      const bool slow = TIME && sm.flag[phase & 1] != 0;
      if (TIME && tid == 0) sm.flag[(phase + 1) & 1] = 0;
      if (kt == qt) {
        pop_next(P, tid, nxt);
        // K, V registers are free from here: they take the h chunks of the
        // fused silu' store (d=64; at d=128 they are loaded after the loop,
        // which keeps them out of the loop's register peak)
        if (D == 64 && fuse) kr.load(P.h_dq + ooff, q_valid, P.out_stride, tid);
      }
      if (kt < qt) {
        const int k_valid = si.len - (kt + 1) * TILE;
        const int64_t r0 = si.start + (int64_t)(kt + 1) * TILE;
        kr.load_at(rs_k, (uint32_t)(kt + 1) * tile_bytes, row_stride, tid);
        vr.load_at(rs_v, (uint32_t)(kt + 1) * tile_bytes, row_stride, tid);
        if (TIME && tid < TILE) ts_k = P.ts[r0 + (tid < k_valid ? tid : k_valid - 1)];
        if (POS) pos_v = pos_fetch(rs_pos, P.N, qt, kt + 1, tid);
      }
      issue_fence();

      // S^T quadrant with the position bias as the accumulator's initial
      // value, and dA^T
      const int kb = 32 * wj + 4 * g;
      f32x16 s, da;
#pragma unroll
      for (int r = 0; r < 16; ++r) { s[r] = 0.0f; da[r] = 0.0f; }
      if (POS) {
        const float *pl = pos_lane(sm.pos, kb - i_loc + (TILE - 1));
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float4 pb = *(const float4 *)(pl + 8 * q4);
          s[4 * q4 + 0] = pb.x; s[4 * q4 + 1] = pb.y;
          s[4 * q4 + 2] = pb.z; s[4 * q4 + 3] = pb.w;
        }
      }
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        s = mfma32(read_rm(sm.t.a, ST, 32 * wj + l32, 16 * ks + 8 * g), qreg[ks], s);
        da = mfma32(read_rm(sm.t.b, ST, 32 * wj + l32, 16 * ks + 8 * g), doreg[ks], da);
      }

      // dS = dA silu'(x), then dQ += dS K, one 16-key half at a time (half the
      // temporaries live at once)
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        float x[8], sg[8], dsv[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = s[8 * hh + e];
        if (TIME) {
          if (!slow) {
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              const float4 t4 = *(const float4 *)(sm.ts32 + kb + 8 * (2 * hh + q));
              x[4 * q + 0] += ktab[time_index(ts_i32 - t4.x)];
              x[4 * q + 1] += ktab[time_index(ts_i32 - t4.y)];
              x[4 * q + 2] += ktab[time_index(ts_i32 - t4.z)];
              x[4 * q + 3] += ktab[time_index(ts_i32 - t4.w)];
            }
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e)
              x[e] += ktab[KTAB + time_bucket(ts_i - sm.ts64[kb + c_row(8 * hh + e, 0)], P.nb)];
          }
        }
        // the score is alpha x: sigma(alpha x), silu'(alpha x) =
        // sigma (1 + x (alpha - alpha sigma))
#pragma unroll
        for (int e = 0; e < 8; ++e) sg[e] = __builtin_amdgcn_exp2f(x[e] * P.neg_al2e);
#pragma unroll
        for (int e = 0; e < 8; ++e) sg[e] = __builtin_amdgcn_rcpf(1.0f + sg[e]);
#pragma unroll
        for (int e = 0; e < 8; ++e)
          dsv[e] = (sg[e] * da[8 * hh + e]) *
                   __builtin_fmaf(x[e], __builtin_fmaf(-P.alpha, sg[e], P.alpha), 1.0f);
        if (kt == qt) {
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (kb + c_row(8 * hh + e, 0) > i_loc) dsv[e] = 0.0f;
        }
        uint4 pk;
        pk.x = pack2(dsv[0], dsv[1]);
        pk.y = pack2(dsv[2], dsv[3]);
        pk.z = pack2(dsv[4], dsv[5]);
        pk.w = pack2(dsv[6], dsv[7]);
        const bf16x8 pa = as_bf16x8(pk);
#pragma unroll
        for (int db = 0; db < D / 32; ++db)
          acc[db] = mfma32(pa, read_tr(sm.t.a, ST, 32 * wj + 16 * hh + 4 * g, 32 * db, lane),
                           acc[db]);
      }
    }

    if (D != 64 && fuse) kr.load(P.h_dq + ooff, q_valid, P.out_stride, tid);
    sum_store_tile<D>(&sm.red[0][0], acc, wj == 0, wi, g, l32, tid, P.dq_out + ooff,
                      P.out_stride, q_valid, P.dqk_scale, fuse, kr.c);
}

// ------------------------------------------------------------------ dK/dV
// d_pos of a k-stationary item by diagonal, summed in LDS double windows
// with the LDS f64 add atomic.  Slot x of the window of tile pair (qt, kt)
// holds diagonal m = i - j = (qt - kt)*64 + x - 63, i.e. x = i_loc - j_loc
// + 63, so a lane's 16 elements sit at fixed offsets from one address; one
// copy per lane group g keeps the 64 lanes of each atomic on distinct
// slots.  Tile pairs alternate between two windows.  Once the next tile
// pair's first barrier has passed, slots x < 64 of the previous window are
// final (no later tile pair reaches those diagonals) and go to the
// sequence's global partial, slots x >= 64 carry into slot x - 64 of the
// current window, and the previous window is cleared for reuse.
template <int D, bool POS, bool DET>
struct DkvSmem {
  StreamSmem<D> s;
  typename TabAcc<DET>::L pwin[POS ? 2 : 1][POS ? 2 : 1][POS ? 2 * TILE : 1];   // [window][g][slot]
  // At d=64 the item's stationary K and V tiles live here (swizzled, filled
  // by global-to-LDS loads) instead of in registers, which lets the kernel
  // run three waves per SIMD without the time bias (two with it).
  // At d=128 only the V tile does (the LDS of two work-groups per CU has
  // no room for both).
  alignas(16) u16 kst[D == 64 ? TILE * D : 8];
  alignas(16) u16 vst[TILE * D];
  // At d=128 each wave accumulates only one of dV, dK (its query half picks
  // which), and the waves exchange their step's packed A and dS operands
  // here: [A or dS][key half][query half][16-query half][lane], 16 KB.
  alignas(16) uint4 xbuf[D == 128 ? 2 * 2 * 2 * 2 : 1][64];
};

// Slot x (< 127) of the finished window `prev` of tile offset dt = qt - kt:
// the two copies are summed and cleared; a final diagonal m is returned
// through (dst, val) for a deferred global atomic into dp[m * H] (dp: this
// sequence's and head's partials), a carried one is added into `cur`.
template <typename A>
__device__ __forceinline__ void dpos_retire(typename A::L (*prev)[2 * TILE],
                                            typename A::L (*cur)[2 * TILE], int x, int dt,
                                            bool last, int len, typename A::G *dp, int H,
                                            typename A::G *&dst, typename A::G &val) {
  const typename A::L v = prev[0][x] + prev[1][x];
  prev[0][x] = 0;
  prev[1][x] = 0;
  if (x < TILE || last) {
    const int m = dt * TILE + x - (TILE - 1);
    if (v != 0 && m >= 0 && m < len) {
      dst = dp + m * H;
      val = A::glob(v);
    }
  } else if (v != 0) {
    atomicAdd(&cur[0][x - TILE], v);
  }
}

// dQ block (query half wi, columns 32 wj ..) of a sequence's first q-tile
// at d=64: its tile pair's dS read transposed out of dsb, K columns out of
// the stationary K tile, all 64 keys.
template <int D>
__device__ __forceinline__ f32x16 dq0_block(const u16 *dsb, const u16 *kst, int wi, int wj, int g,
                                            int lane) {
  f32x16 dq;
#pragma unroll
  for (int r = 0; r < 16; ++r) dq[r] = 0.0f;
#pragma unroll
  for (int kk = 0; kk < TILE / 16; ++kk)
    dq = mfma32(read_tr(dsb, DS_STRIDE, 16 * kk + 4 * g, 32 * wi, lane),
                sread_tr<D, SWZ_CF>(kst, 16 * kk + 4 * g, 32 * wj, lane), dq);
  return dq;
}

// One k-stationary item: dV_j, dK_j for a 64-row key tile of one head over
// its query tiles, with the table gradients (d_pos through the sheared tile
// and the rolling diagonal window, d_time through per-lane index runs).
template <int D, bool POS, bool TIME, bool DET, bool KV_LDS>
__device__ __forceinline__ void dkv_item(const KParams &P, DkvSmem<D, POS, DET> &smx,
                                         float *dyn, typename TabAcc<DET>::L *tacc,
                                         const int tid0, const WorkEntry e, const int h,
                                         int &phase, typename TabAcc<DET>::G *&pend_p,
                                         typename TabAcc<DET>::G &pend_v, int &nxt,
                                         u16 *dsb = nullptr) {
  typedef TabAcc<DET> A;
  constexpr int ST = D + RM_PAD;
  StreamSmem<D> &sm = smx.s;
    int tid = tid0;
    asm volatile("" : "+v"(tid));
    int row_stride = P.H * D;
    asm volatile("" : "+s"(row_stride));
    const int lane = tid & 63, g = lane >> 5, l32 = lane & 31;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int wj = w & 1, wi = w >> 1;        // key half (stationary), query half

    const SeqInfo si = entry_seq(e);
    const int kt = e.tile;
    const int k_valid = si.len - kt * TILE;
    const int j_loc = 32 * wj + l32;
    const int64_t koff = ((si.start + (int64_t)kt * TILE) * P.H + h) * D;
    const int64_t ooff = (si.start + (int64_t)kt * TILE) * P.out_stride + h * D;
    const bool fuse = P.h_dk != nullptr;

    // stationary K, V rows: registers, or (d=64) LDS tiles whose rows past
    // the sequence repeat its last row -- those keys only occur in the last
    // key tile's diagonal step, where the causal mask removes them, and
    // query rows past the sequence carry dO = 0
    // dQ of a sequence's first q-tile comes from its tile pair (0, 0) alone:
    // with `dsb` given, the item of k-tile 0 stages that pair's dS^T in
    // `dsb` ([key][query], stride DS_STRIDE) and computes dQ = dS K against
    // the stationary K tile at the item's end (both stay untouched until then).
    const bool with_dq = KV_LDS && dsb != nullptr && kt == 0;
    constexpr bool V_LDS = true;              // V stationary in LDS at both d
    bf16x8 kreg[KV_LDS ? 1 : D / 16];
    {
      // (lane made opaque: the loads' offsets are recomputed here rather
      // than kept in registers across the whole item loop)
      int ln = lane;
      asm volatile("" : "+v"(ln));
      if constexpr (KV_LDS) dma_tile<D, SWZ_CF>(P.k + koff, k_valid, row_stride, smx.kst, w, ln);
      dma_tile<D, SWZ_CF>(P.v + koff, k_valid, row_stride, smx.vst, w, ln);
    }
    if constexpr (!KV_LDS) load_stationary<D>(P.k + koff, j_loc, k_valid, row_stride, g, kreg);

    // every load of the item's start is issued before any of them is used
    // (one memory latency); timestamps of rows past the sequence repeat its
    // last row (those rows are always masked)
    // the sequence's Q and dO rows of head h, each one source for the item
    const uint32_t seq_bytes = 2u * (uint32_t)si.len * (uint32_t)row_stride;
    const __amdgpu_buffer_rsrc_t rs_q = make_rsrc(P.q + (si.start * P.H + h) * D, seq_bytes);
    const __amdgpu_buffer_rsrc_t rs_o = make_rsrc(P.dO + (si.start * P.H + h) * D, seq_bytes);
    const uint32_t tile_bytes = 2u * (uint32_t)TILE * (uint32_t)row_stride;
    TileRegs<D> qr, dr;
    TileRegs<D> hq;                       // h chunks of the first tile's dQ (fused store)
    const int64_t r0k = si.start + (int64_t)kt * TILE;
    qr.load_at(rs_q, (uint32_t)kt * tile_bytes, row_stride, tid);
    dr.load_at(rs_o, (uint32_t)kt * tile_bytes, row_stride, tid);
    int64_t ts_start = 0, ts_j = 0, ts_q = 0;
    if (TIME) {
      ts_start = P.ts[si.start];
      ts_j = P.ts[r0k + (j_loc < k_valid ? j_loc : k_valid - 1)];
      if (tid < TILE) ts_q = P.ts[r0k + (tid < k_valid ? tid : k_valid - 1)];
    }
    const __amdgpu_buffer_rsrc_t rs_pos = pos_source(P, POS ? h : 0);
    PosEntry pos_v = POS ? pos_fetch(rs_pos, P.N, kt, kt, tid) : PosEntry{0.0f, false};

    float ts_j32 = 0.0f;
    bool k_far = false;
    float *ktab = dyn;
    if (TIME) {
      if (phase == 0) stage_all_heads<D == 64 ? 8 : 1>(P, dyn, tid, P.inv_alpha);   // as in dq_item
      const int64_t rel = ts_j - ts_start;
      ts_j32 = (float)(int32_t)rel;
      k_far = rel >= NEAR || rel <= -NEAR;
      ktab = item_time_slot(P, dyn, h, tid, P.inv_alpha);
    }
    TimeRun<A> run;                           // fast path: by float-exponent index
    typename A::L *my_t = TIME ? tacc + h * P.nb : nullptr;
    typename A::G *dp_item = POS ? (typename A::G *)P.dpos_part + si.start * P.H + h : nullptr;

    // At d=128 (SPLIT) a wave's dK and dV accumulators together would take
    // 128 registers and hold the kernel to one wave per SIMD: there each
    // wave keeps one of them for its key half -- dV in the waves of query
    // half 0, dK in those of half 1 -- in `dv`, over both query halves,
    // whose packed A and dS operands the waves exchange through LDS.
    constexpr bool SPLIT = D == 128;
    f32x16 dk[SPLIT ? 1 : D / 32], dv[D / 32];
#pragma unroll
    for (int db = 0; db < D / 32; ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) dv[db][r] = 0.0f;
#pragma unroll
    for (int db = 0; db < (SPLIT ? 1 : D / 32); ++db)
#pragma unroll
      for (int r = 0; r < 16; ++r) dk[db][r] = 0.0f;
    if constexpr (V_LDS) wait_vm();     // the first step's barriers publish the tiles

    for (int qt = kt; qt < si.ntiles; ++qt, ++phase) {
      lds_barrier();
      qr.store(sm.t.a, tid);
      dr.store(sm.t.b, tid);
      if constexpr (POS) {
        pos_store<true>(pos_v, P.inv_alpha, sm.pos, tid);
        if (pend_p) atomicAdd(pend_p, pend_v);
        pend_p = nullptr;
        if (qt > kt && tid < 2 * TILE - 1) {
          dpos_retire<A>(smx.pwin[(phase - 1) & 1], smx.pwin[phase & 1], tid, qt - 1 - kt,
                         false, si.len, dp_item, P.H, pend_p, pend_v);
          if (pend_p) atomicAdd(pend_p, pend_v);
          pend_p = nullptr;
        }
      }
      if (TIME) {
        bool far = k_far;
        if (tid < TILE) {
          const int64_t rel = ts_q - ts_start;
          sm.ts32[tid] = (float)(int32_t)rel;
          sm.ts64[tid] = ts_q;
          far |= rel >= NEAR || rel <= -NEAR;
        }
        if (far) sm.flag[phase & 1] = 1;
      }
      lds_barrier();
      const bool slow = TIME && sm.flag[phase & 1] != 0;
      if (TIME && tid == 0) sm.flag[(phase + 1) & 1] = 0;
      if (qt + 1 == si.ntiles) {
        pop_next(P, tid, nxt);
        // Q, dO registers are free from here: they take the h chunks of
        // the fused silu' stores
        if (fuse) {
          qr.load(P.h_dk + ooff, k_valid, P.out_stride, tid);
          dr.load(P.h_dv + ooff, k_valid, P.out_stride, tid);
          if (with_dq) hq.load(P.h_dq + ooff, k_valid, P.out_stride, tid);
        }
      }
      if (qt + 1 < si.ntiles) {
        const int nv = si.len - (qt + 1) * TILE;
        const int64_t r0 = si.start + (int64_t)(qt + 1) * TILE;
        qr.load_at(rs_q, (uint32_t)(qt + 1) * tile_bytes, row_stride, tid);
        dr.load_at(rs_o, (uint32_t)(qt + 1) * tile_bytes, row_stride, tid);
        if (TIME && tid < TILE) ts_q = P.ts[r0 + (tid < nv ? tid : nv - 1)];
        if (POS) pos_v = pos_fetch(rs_pos, P.N, qt + 1, kt, tid);
      }
      issue_fence();

      // this lane's queries sit at ib + 8 q4 + c, ib = 32 wi + 4 g; offset
      // j - i = j_loc - ib - i_rel walks the slice downwards, i.e. the
      // reversed copies upwards from 126 - x0
      const int ib = 32 * wi + 4 * g;
      const int x0 = j_loc - ib + (TILE - 1);
      // S and dA quadrants [32 queries x 32 keys]; lane holds key j_loc.  The
      // position bias is the score accumulator's initial value.
      f32x16 s, da;
#pragma unroll
      for (int r = 0; r < 16; ++r) { s[r] = 0.0f; da[r] = 0.0f; }
      if (POS) {
        const float *pl = pos_lane(sm.pos, 2 * TILE - 2 - x0);
#pragma unroll
        for (int q4 = 0; q4 < 4; ++q4) {
          const float4 pb = *(const float4 *)(pl + 8 * q4);
          s[4 * q4 + 0] = pb.x; s[4 * q4 + 1] = pb.y;
          s[4 * q4 + 2] = pb.z; s[4 * q4 + 3] = pb.w;
        }
      }
      // At d=128 the S products go first, so that the pointwise chain on S
      // (exp, rcp, A) runs under the dA products (measured 1.7% faster
      // there, 2.4% slower at d=64, where the two chains stay interleaved)
      constexpr bool S_FIRST = D == 128;
#pragma unroll
      for (int ks = 0; ks < D / 16; ++ks) {
        const bf16x8 kop =
            KV_LDS ? sread_rm<D, SWZ_CF>(smx.kst, j_loc, 16 * ks + 8 * g) : kreg[KV_LDS ? 0 : ks];
        s = mfma32(read_rm(sm.t.a, ST, 32 * wi + l32, 16 * ks + 8 * g), kop, s);
        if constexpr (!S_FIRST) {
          const bf16x8 vop = sread_rm<D, SWZ_CF>(smx.vst, j_loc, 16 * ks + 8 * g);
          da = mfma32(read_rm(sm.t.b, ST, 32 * wi + l32, 16 * ks + 8 * g), vop, da);
        }
      }
      if constexpr (S_FIRST) {
#pragma unroll
        for (int ks = 0; ks < D / 16; ++ks) {
          const bf16x8 vop = sread_rm<D, SWZ_CF>(smx.vst, j_loc, 16 * ks + 8 * g);
          da = mfma32(read_rm(sm.t.b, ST, 32 * wi + l32, 16 * ks + 8 * g), vop, da);
        }
      }

      // a = silu(x)/N, dS = dA silu'(x)/N = dA (sg + a (1 - sg))/N with
      // a = x sg, the table gradients, then dV += A^T dO and dK += dS^T Q,
      // one 16-query half at a time (half the temporaries live at once).
      // Both are carried multiplied by log2e (A' = u sg with u = x log2e,
      // dS' = dA (sg log2e + A' (1 - sg))): one multiply per element fewer
      // than natural units; the stores divide it out, and the table
      // partials keep it until the finalize pass.
      // Query rows past the sequence have dO = 0, hence dA = 0 and dS = 0,
      // and contribute a * 0 to dV: only the diagonal tile needs a mask (the
      // causal one).
      float carry = 0.0f;       // d_pos: a quad's row-head sums for the next quad
#pragma unroll
      for (int hh = 0; hh < 2; ++hh) {
        float x[8], sg[8], av[8], dsv[8];
        int tk[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) x[e] = s[8 * hh + e];
        if (TIME) {
          if (!slow) {
#pragma unroll
            for (int q = 0; q < 2; ++q) {
              const float4 t4 = *(const float4 *)(sm.ts32 + ib + 8 * (2 * hh + q));
              tk[4 * q + 0] = time_index(t4.x - ts_j32);
              tk[4 * q + 1] = time_index(t4.y - ts_j32);
              tk[4 * q + 2] = time_index(t4.z - ts_j32);
              tk[4 * q + 3] = time_index(t4.w - ts_j32);
            }
#pragma unroll
            for (int e = 0; e < 8; ++e) x[e] += ktab[tk[e]];
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              tk[e] = time_bucket(sm.ts64[ib + c_row(8 * hh + e, 0)] - ts_j, P.nb);
              x[e] += ktab[KTAB + tk[e]];
            }
          }
        }
        // the score is alpha x (biases staged divided by alpha)
        float u[8];
#pragma unroll
        for (int e = 0; e < 8; ++e) u[e] = x[e] * P.al2e;
#pragma unroll
        for (int e = 0; e < 8; ++e) sg[e] = __builtin_amdgcn_exp2f(-u[e]);
#pragma unroll
        for (int e = 0; e < 8; ++e) sg[e] = __builtin_amdgcn_rcpf(1.0f + sg[e]);
#pragma unroll
        for (int e = 0; e < 8; ++e) {
          const float a1 = u[e] * sg[e];
          av[e] = a1;
          dsv[e] = da[8 * hh + e] * __builtin_fmaf(-a1, sg[e], __builtin_fmaf(sg[e], L2E, a1));
        }
        if (qt == kt) {
          // a real branch: selected without it, the mask's compares and
          // selects would run on every step
          asm volatile("");
#pragma unroll
          for (int e = 0; e < 8; ++e)
            if (ib + c_row(8 * hh + e, 0) < j_loc) { av[e] = 0.0f; dsv[e] = 0.0f; }
        }
        if constexpr (POS) {
          // element (i, j) -> slot i_loc - j_loc + 63, i_loc = ib + c_row(r, 0).
          // A register quad holds rows i0 .. i0+3 of the lane's key, so
          // element (i0 + k) of lane l+k lies on the diagonal of element i0
          // of lane l: each quad is summed along its diagonals inside the
          // 16-lane row first (band: lane l adds lanes l+k, k = 0..3, one
          // atomic per lane).  The six elements of a row's first three lanes
          // that no band reaches (head: lanes m = 0..2 sum them along the
          // diagonals of rows i0+3 of lane m) lie on the band diagonals of
          // lanes 5..7 of the next quad (8 rows further), which adds them;
          // only the step's last quad flushes its heads itself.  Five LDS
          // atomics per lane and step instead of sixteen.
          typename A::L *pw = &smx.pwin[phase & 1][g][ib - j_loc + (TILE - 1)];
          const bool row_head = (lane & 15) < 3;
#pragma unroll
          for (int q = 0; q < 2; ++q) {
            const float *v = dsv + 4 * q;
            const float b4 =
                ((v[0] + row_shl<1>(v[1])) + row_shl<2>(v[2])) + row_shl<3>(v[3]);
            const float band = hh == 0 && q == 0 ? b4 : b4 + carry;   // first quad: none
            const float head = (v[3] + row_shr<1>(v[2])) + row_shr<2>(v[1]);
            const int at = 16 * hh + 8 * q;             // c_row(8 hh + 4 q, 0)
            atomicAdd(pw + at, A::lds(band));
            if (hh == 1 && q == 1) {
              if (row_head) atomicAdd(pw + at + 3, A::lds(head));
            } else {
              carry = row_shr<5>(row_head ? head : 0.0f);
            }
          }
        }
        if (TIME) {
          // slow tiles accumulate by bucket straight into the work-group
          // histogram; fast tiles by float-exponent index, folded per item
          if (!slow) {
            if (hh == 0) run.start(tk[0]);
#pragma unroll
            for (int e = 0; e < 8; ++e) run.add(my_t, P.nb, tk[e], dsv[e]);
          } else {
#pragma unroll
            for (int e = 0; e < 8; ++e) {
              // converted here, not shared with the d_pos atomics: a shared
              // conversion would keep the doubles live across this branch
              float v = dsv[e];
              asm volatile("" : "+v"(v));
              if (v != 0.0f) atomicAdd(&my_t[tk[e]], A::lds(v));
            }
          }
        }
        uint4 pa, pd;
        pa.x = pack2(av[0], av[1]);
        pa.y = pack2(av[2], av[3]);
        pa.z = pack2(av[4], av[5]);
        pa.w = pack2(av[6], av[7]);
        pd.x = pack2(dsv[0], dsv[1]);
        pd.y = pack2(dsv[2], dsv[3]);
        pd.z = pack2(dsv[4], dsv[5]);
        pd.w = pack2(dsv[6], dsv[7]);
        const bf16x8 a8 = as_bf16x8(pa), d8 = as_bf16x8(pd);
        const int krow = 32 * wi + 16 * hh + 4 * g;
        if (with_dq && qt == kt) {
          // this lane's key row; its 8 queries are krow .. +3 and krow+8 .. +11
          u16 *row = dsb + j_loc * DS_STRIDE + krow;
          *(uint2 *)row = make_uint2(pd.x, pd.y);
          *(uint2 *)(row + 8) = make_uint2(pd.z, pd.w);
        }
        if constexpr (SPLIT) {
          smx.xbuf[((0 * 2 + wj) * 2 + wi) * 2 + hh][lane] = pa;
          smx.xbuf[((1 * 2 + wj) * 2 + wi) * 2 + hh][lane] = pd;
        } else {
#pragma unroll
          for (int db = 0; db < D / 32; ++db) {
            dv[db] = mfma32(a8, read_tr(sm.t.b, ST, krow, 32 * db, lane), dv[db]);
            dk[db] = mfma32(d8, read_tr(sm.t.a, ST, krow, 32 * db, lane), dk[db]);
          }
        }
      }
      if constexpr (SPLIT) {
        // this wave's role (wi): dV += A^T dO or dK += dS^T Q over both
        // query halves, from the operands of the two waves of its key half
        lds_barrier();
        const u16 *src = wi ? sm.t.a : sm.t.b;
#pragma unroll
        for (int qh = 0; qh < 2; ++qh)
#pragma unroll
          for (int hh = 0; hh < 2; ++hh) {
            const bf16x8 op = as_bf16x8(smx.xbuf[((wi * 2 + wj) * 2 + qh) * 2 + hh][lane]);
            const int krow = 32 * qh + 16 * hh + 4 * g;
#pragma unroll
            for (int db = 0; db < D / 32; ++db)
              dv[db] = mfma32(op, read_tr(src, ST, krow, 32 * db, lane), dv[db]);
          }
      }
    }

    // close the d_time runs; sum the two query halves, store dK, dV (bf16)
    if (TIME) run.flush(my_t, P.nb);
    lds_barrier();
    if constexpr (POS) {   // every diagonal of the last window is final
      if (tid < 2 * TILE - 1)
        dpos_retire<A>(smx.pwin[(phase - 1) & 1], smx.pwin[phase & 1], tid,
                       si.ntiles - 1 - kt, true, si.len, dp_item, P.H, pend_p, pend_v);
    }
    if constexpr (KV_LDS) {
      if (with_dq)
        quad_store_tile<D>(&sm.red[0][0], dq0_block<D>(dsb, smx.kst, wi, wj, g, lane), wi, wj,
                           g, l32, tid, P.dq_out + ooff, P.out_stride, k_valid, P.dk_scale_l2,
                           fuse, hq.c);
    }
    if constexpr (SPLIT) {
      sum_store_tile<D, false>(&sm.red[0][0], dv, wi == 1, wj, g, l32, tid, P.out0 + ooff,
                               P.out_stride, k_valid, P.dk_scale_l2, fuse, qr.c);
      sum_store_tile<D, false>(&sm.red[0][0], dv, wi == 0, wj, g, l32, tid, P.out1 + ooff,
                               P.out_stride, k_valid, P.dv_scale_l2, fuse, dr.c);
    } else {
      sum_store_tile<D>(&sm.red[0][0], dk, wi == 0, wj, g, l32, tid, P.out0 + ooff,
                        P.out_stride, k_valid, P.dk_scale_l2, fuse, qr.c);
      sum_store_tile<D>(&sm.red[0][0], dv, wi == 0, wj, g, l32, tid, P.out1 + ooff,
                        P.out_stride, k_valid, P.dv_scale_l2, fuse, dr.c);
    }
}

// Work-group start of the kernels that run dK/dV items: zeroed d_time
// histogram, cleared flags and d_pos windows (the
// time tables are staged by the first item).
template <int D, bool POS, bool TIME, bool DET>
__device__ __forceinline__ void dkv_kernel_init(const KParams &P, DkvSmem<D, POS, DET> &smx,
                                                typename TabAcc<DET>::L *tacc, float *dyn,
                                                int tid0) {
  if (TIME) {
    for (int x = tid0; x < P.H * P.nb; x += THREADS) tacc[x] = 0;
  }
  if (tid0 < 2) smx.s.flag[tid0] = 0;
  if constexpr (POS)
    for (int x = tid0; x < 2 * 2 * 2 * TILE; x += THREADS) (&smx.pwin[0][0][0])[x] = 0;
}

// Work-group end: the last deferred d_pos sum (a finished diagonal is sent
// one tile later, after the next wait for the prefetched tiles, because that
// wait also counts atomics), then this work-group's d_time histogram folded
// into one of DTIME_BINS partials.
template <int D, bool POS, bool TIME, bool DET>
__device__ __forceinline__ void dkv_kernel_fini(const KParams &P, typename TabAcc<DET>::L *tacc,
                                                int tid0, typename TabAcc<DET>::G *pend_p,
                                                typename TabAcc<DET>::G pend_v) {
  typedef TabAcc<DET> A;
  if (POS && pend_p) atomicAdd(pend_p, pend_v);
  if (TIME) {
    lds_barrier();
    typename A::G *part =
        (typename A::G *)P.dtime_part + (int64_t)(blockIdx.x % DTIME_BINS) * P.H * P.nb;
    for (int x = tid0; x < P.H * P.nb; x += THREADS)
      if (tacc[x] != 0) atomicAdd(&part[x], A::glob(tacc[x]));
  }
}

// Backward, both item kinds in one launch over the combined list, whose
// entries are dK/dV items (k-stationary) and dQ items (flagged,
// q-stationary) in one longest-first order.
template <int D, bool POS, bool TIME, bool DET>
__global__ void __launch_bounds__(THREADS, 2)
attn_bwd_kernel(KParams P) {
  typedef TabAcc<DET> A;
  __shared__ DkvSmem<D, POS, DET> smx;
  // dS^T of a first tile pair (d=64, see dkv_item)
  __shared__ __attribute__((aligned(16))) u16 dsb[D == 64 ? TILE * DS_STRIDE : 8];
  StreamSmem<D> &sm = smx.s;
  // dynamic LDS: [H][nb] d_time (double), then the time tables
  extern __shared__ double dyn_k[];
  typename A::L *tacc = (typename A::L *)dyn_k;
  float *dyn = (float *)(dyn_k + P.H * P.nb);
  const int tid0 = threadIdx.x;
  const int n_items = P.ctrl[CTRL_N_BWD] * P.H;
  dkv_kernel_init<D, POS, TIME, DET>(P, smx, tacc, dyn, tid0);
  lds_barrier();
  int phase = 0;
  typename A::G *pend_p = nullptr;
  typename A::G pend_v = 0;
  int nxt = 0;
  for (int item = blockIdx.x; item < n_items; item = take_next(&sm.item, tid0, nxt)) {
    WorkEntry e = P.list[item / P.H];
    const int h = item % P.H;
    if (e.tile & BWD_DQ_FLAG) {
      e.tile &= ~BWD_DQ_FLAG;
      dq_item<D, POS, TIME>(P, sm, dyn, tid0, e, h, phase, nxt);
    } else {
      dkv_item<D, POS, TIME, DET, D == 64>(P, smx, dyn, tacc, tid0, e, h, phase, pend_p, pend_v,
                                           nxt, P.fuse_dq0 ? dsb : nullptr);
    }
  }
  dkv_kernel_fini<D, POS, TIME, DET>(P, tacc, tid0, pend_p, pend_v);
}

// Backward, dQ: persistent work-groups pop q-tile items longest first.
template <int D, bool POS, bool TIME>
__global__ void __launch_bounds__(THREADS, D == 64 ? (TIME ? 2 : 3) : 2)
attn_bwd_dq_kernel(KParams P) {
  __shared__ StreamSmem<D> sm;
  extern __shared__ float dyn_q[];            // time tables
  const int tid0 = threadIdx.x;
  const int n_items = P.ctrl[CTRL_N_ENTRIES] * P.H;
  if (tid0 < 2) sm.flag[tid0] = 0;
  lds_barrier();
  int phase = 0;
  int nxt = 0;
  for (int item = blockIdx.x; item < n_items; item = take_next(&sm.item, tid0, nxt))
    dq_item<D, POS, TIME>(P, sm, dyn_q, tid0, P.list[item / P.H], item % P.H, phase, nxt);
}

// Backward, dK/dV and the table gradients: persistent work-groups pop k-tile
// items longest first.
template <int D, bool POS, bool TIME, bool DET>
__global__ void __launch_bounds__(THREADS, D == 64 ? (TIME ? 2 : 3) : 2)
attn_bwd_dkv_kernel(KParams P) {
  typedef TabAcc<DET> A;
  __shared__ DkvSmem<D, POS, DET> smx;
  StreamSmem<D> &sm = smx.s;
  extern __shared__ double dyn_k[];
  typename A::L *tacc = (typename A::L *)dyn_k;
  float *dyn = (float *)(dyn_k + P.H * P.nb);
  const int tid0 = threadIdx.x;
  const int n_items = P.ctrl[CTRL_N_ENTRIES] * P.H;
  dkv_kernel_init<D, POS, TIME, DET>(P, smx, tacc, dyn, tid0);
  lds_barrier();
  int phase = 0;
  typename A::G *pend_p = nullptr;
  typename A::G pend_v = 0;
  int nxt = 0;
  for (int item = blockIdx.x; item < n_items; item = take_next(&sm.item, tid0, nxt))
    // K, V stationary in LDS at d=64 (in registers the kernel measured
    // 5-10% slower on the Zipf batch of 1024 sequences)
    dkv_item<D, POS, TIME, DET, D == 64>(P, smx, dyn, tacc, tid0, P.list[item / P.H],
                                         item % P.H, phase, pend_p, pend_v, nxt);
  dkv_kernel_fini<D, POS, TIME, DET>(P, tacc, tid0, pend_p, pend_v);
}

// ------------------------------------------------------------- launchers
template <typename K>
int persistent_grid(K kernel, size_t dyn, int64_t items, int dev, int block = THREADS) {
  int occ = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&occ, kernel, block, dyn) != hipSuccess ||
      occ < 1)
    occ = 1;
  const int64_t cap = (int64_t)device_info(dev).num_cu * occ;
  return (int)std::max<int64_t>(1, std::min<int64_t>(cap, items));
}

// Time tables: one slot of KTAB + nb floats per head when all heads fit in
// this budget (staged once per work-group), else a single per-item slot.
constexpr size_t ALL_HEADS_BUDGET = 32 * 1024;
bool all_heads(const Problem &p) {
  const size_t budget = p.d == 64 ? ALL_HEADS_BUDGET : ALL_HEADS_BUDGET / 4;
  return p.has_time && sizeof(float) * (size_t)p.H * (KTAB + p.nb) <= budget;
}
size_t slots_bytes(const Problem &p) {
  if (!p.has_time) return 0;
  return sizeof(float) * (size_t)(all_heads(p) ? p.H : 1) * (KTAB + p.nb);
}
size_t q_dyn_bytes(const Problem &p) { return slots_bytes(p); }
size_t k_dyn_bytes(const Problem &p) {
  return p.has_time ? slots_bytes(p) + sizeof(double) * (size_t)p.nb * p.H : 0;
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
  P.alpha = a.p.alpha;
  P.inv_alpha = 1.0f / a.p.alpha;
  P.neg_al2e = -a.p.alpha * L2E;
  P.dqk_scale = a.p.alpha / (float)a.p.N;
  P.al2e = a.p.alpha * L2E;
  P.dk_scale_l2 = P.dqk_scale / L2E;
  P.dv_scale_l2 = P.inv_n / L2E;
  P.all_heads = all_heads(a.p) ? 1 : 0;
  P.out_stride = a.p.H * a.p.d;
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

// As HSTU_DISPATCH, with a fourth template argument QT (forward items of QT
// query tiles).
#define HSTU_DISPATCH_Q(KERNEL, D, POS, TIME, QT, ...)                              \
  do {                                                                              \
    if (D == 64) {                                                                  \
      if (POS && TIME) { auto kfn = KERNEL<64, true, true, QT>; __VA_ARGS__; }      \
      else if (POS) { auto kfn = KERNEL<64, true, false, QT>; __VA_ARGS__; }       \
      else if (TIME) { auto kfn = KERNEL<64, false, true, QT>; __VA_ARGS__; }      \
      else { auto kfn = KERNEL<64, false, false, QT>; __VA_ARGS__; }               \
    } else {                                                                        \
      if (POS && TIME) { auto kfn = KERNEL<128, true, true, QT>; __VA_ARGS__; }     \
      else if (POS) { auto kfn = KERNEL<128, true, false, QT>; __VA_ARGS__; }      \
      else if (TIME) { auto kfn = KERNEL<128, false, true, QT>; __VA_ARGS__; }     \
      else { auto kfn = KERNEL<128, false, false, QT>; __VA_ARGS__; }              \
    }                                                                               \
  } while (0)

// As HSTU_DISPATCH, for the kernels that accumulate the table gradients
// (a fourth template argument: the deterministic fixed-point mode).
#define HSTU_DISPATCH_TAB(KERNEL, D, POS, TIME, DET, ...)                             \
  do {                                                                                \
    if (DET) {                                                                        \
      if (D == 64) {                                                                  \
        if (POS && TIME) { auto kfn = KERNEL<64, true, true, true>; __VA_ARGS__; }    \
        else if (POS) { auto kfn = KERNEL<64, true, false, true>; __VA_ARGS__; }     \
        else if (TIME) { auto kfn = KERNEL<64, false, true, true>; __VA_ARGS__; }    \
        else { auto kfn = KERNEL<64, false, false, true>; __VA_ARGS__; }             \
      } else {                                                                        \
        if (POS && TIME) { auto kfn = KERNEL<128, true, true, true>; __VA_ARGS__; }   \
        else if (POS) { auto kfn = KERNEL<128, true, false, true>; __VA_ARGS__; }    \
        else if (TIME) { auto kfn = KERNEL<128, false, true, true>; __VA_ARGS__; }   \
        else { auto kfn = KERNEL<128, false, false, true>; __VA_ARGS__; }            \
      }                                                                               \
    } else {                                                                          \
      if (D == 64) {                                                                  \
        if (POS && TIME) { auto kfn = KERNEL<64, true, true, false>; __VA_ARGS__; }   \
        else if (POS) { auto kfn = KERNEL<64, true, false, false>; __VA_ARGS__; }    \
        else if (TIME) { auto kfn = KERNEL<64, false, true, false>; __VA_ARGS__; }   \
        else { auto kfn = KERNEL<64, false, false, false>; __VA_ARGS__; }            \
      } else {                                                                        \
        if (POS && TIME) { auto kfn = KERNEL<128, true, true, false>; __VA_ARGS__; }  \
        else if (POS) { auto kfn = KERNEL<128, true, false, false>; __VA_ARGS__; }   \
        else if (TIME) { auto kfn = KERNEL<128, false, true, false>; __VA_ARGS__; }  \
        else { auto kfn = KERNEL<128, false, false, false>; __VA_ARGS__; }           \
      }                                                                               \
    }                                                                                 \
  } while (0)

int current_dev() {
  int dev = 0;
  (void)hipGetDevice(&dev);
  return dev;
}


}  // namespace

bool fwd_pairs(const Problem &p) {
  return p.dtype == HSTU_BF16 && p.d == 64 && p.T >= FWD_PAIR_MIN_AVG_LEN * (int64_t)p.B;
}

int attn_fwd_grid(const Problem &p, int dev) {
  int grid = 1;
  if (fwd_pairs(p))
    HSTU_DISPATCH_Q(attn_fwd_kernel, p.d, p.has_pos, p.has_time, 2,
                    grid = persistent_grid(kfn, q_dyn_bytes(p), p.max_entries * p.H, dev,
                                           2 * THREADS));
  else
    HSTU_DISPATCH_Q(attn_fwd_kernel, p.d, p.has_pos, p.has_time, 1,
                    grid = persistent_grid(kfn, q_dyn_bytes(p), p.max_entries * p.H, dev));
  return grid;
}

int attn_bwd_grid(const Problem &p, int dev) {
  int grid = 1;
  HSTU_DISPATCH_TAB(attn_bwd_kernel, p.d, p.has_pos, p.has_time, p.deterministic,
                    grid = persistent_grid(kfn, k_dyn_bytes(p), 2 * p.max_entries * p.H, dev));
  return grid;
}

int attn_bwd_dq_grid(const Problem &p, int dev) {
  int grid = 1;
  HSTU_DISPATCH(attn_bwd_dq_kernel, p.d, p.has_pos, p.has_time,
                grid = persistent_grid(kfn, q_dyn_bytes(p), p.max_entries * p.H, dev));
  return grid;
}

int attn_bwd_dkv_grid(const Problem &p, int dev) {
  int grid = 1;
  HSTU_DISPATCH_TAB(attn_bwd_dkv_kernel, p.d, p.has_pos, p.has_time, p.deterministic,
                    grid = persistent_grid(kfn, k_dyn_bytes(p), p.max_entries * p.H, dev));
  return grid;
}

hipError_t launch_attn_fwd_bf16(const AttnArgs &a, void *o, hipStream_t s) {
  const char *ws = (const char *)a.ws;
  const Problem &p = a.p;
  const bool pairs = fwd_pairs(p);
  KParams P = make_params(a, (int32_t *)(ws + a.L.ctrl) + CTRL_POP_FWD,
                          (const WorkEntry *)(ws + (pairs ? a.L.list_p : a.L.list_q)));
  P.out0 = (u16 *)o;
  const int grid = attn_fwd_grid(p, current_dev());
  if (pairs)
    HSTU_DISPATCH_Q(attn_fwd_kernel, p.d, p.has_pos, p.has_time, 2,
                    hipLaunchKernelGGL(kfn, dim3(grid), dim3(2 * THREADS), q_dyn_bytes(p), s, P));
  else
    HSTU_DISPATCH_Q(attn_fwd_kernel, p.d, p.has_pos, p.has_time, 1,
                    hipLaunchKernelGGL(kfn, dim3(grid), dim3(THREADS), q_dyn_bytes(p), s, P));
  return hipGetLastError();
}

hipError_t launch_attn_bwd_bf16(const AttnArgs &a, const void *dO, void *dq, void *dk,
                                void *dv, const GradOut *go, hipStream_t s) {
  const char *ws = (const char *)a.ws;
  const Problem &p = a.p;
  auto outputs = [&](KParams &P) {
    P.dO = (const u16 *)dO;
    P.out0 = (u16 *)dk;
    P.out1 = (u16 *)dv;
    P.dq_out = (u16 *)dq;
    if (go) {
      P.out_stride = go->stride;
      P.h_dq = (const u16 *)go->h_dq;
      P.h_dk = (const u16 *)go->h_dk;
      P.h_dv = (const u16 *)go->h_dv;
    }
  };
  if (a.L.bwd_combined) {
    prof::Scope ps("attn_bwd", s);
    KParams P = make_params(a, (int32_t *)(ws + a.L.ctrl) + CTRL_POP_BWD,
                            (const WorkEntry *)(ws + a.L.list_b));
    outputs(P);
    P.dpos_part = a.L.dpos_part ? (void *)(ws + a.L.dpos_part) : nullptr;
    P.dtime_part = a.L.dtime_part ? (void *)(ws + a.L.dtime_part) : nullptr;
    // must match the scheduler's choice (sched_args)
    P.fuse_dq0 = p.d == 64 ? 1 : 0;
    HSTU_DISPATCH_TAB(attn_bwd_kernel, p.d, p.has_pos, p.has_time, p.deterministic,
                      hipLaunchKernelGGL(kfn, dim3(a.L.bwd_grid_both), dim3(THREADS),
                                         k_dyn_bytes(p), s, P));
    return hipGetLastError();
  }
  {
    prof::Scope ps("attn_bwd_dkv", s);
    KParams P = make_params(a, (int32_t *)(ws + a.L.ctrl) + CTRL_POP_DKV,
                            (const WorkEntry *)(ws + a.L.list_k));
    outputs(P);
    P.dpos_part = a.L.dpos_part ? (void *)(ws + a.L.dpos_part) : nullptr;
    P.dtime_part = a.L.dtime_part ? (void *)(ws + a.L.dtime_part) : nullptr;
    HSTU_DISPATCH_TAB(attn_bwd_dkv_kernel, p.d, p.has_pos, p.has_time, p.deterministic,
                      hipLaunchKernelGGL(kfn, dim3(a.L.bwd_grid_dkv), dim3(THREADS),
                                         k_dyn_bytes(p), s, P));
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return e;
  }
  prof::Scope ps("attn_bwd_dq", s);
  KParams P = make_params(a, (int32_t *)(ws + a.L.ctrl) + CTRL_POP_DQ,
                          (const WorkEntry *)(ws + a.L.list_q));
  outputs(P);
  HSTU_DISPATCH(attn_bwd_dq_kernel, p.d, p.has_pos, p.has_time,
                hipLaunchKernelGGL(kfn, dim3(a.L.bwd_grid_dq), dim3(THREADS), q_dyn_bytes(p),
                                   s, P));
  return hipGetLastError();
}

}  // namespace hstu
