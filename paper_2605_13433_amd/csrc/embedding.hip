// Jagged multi-table embedding lookup for gfx950 (Sec. 4.1.2, "Jagged
// Embedding Lookup Acceleration"): explicit jagged indices (table offsets,
// no padding ids) and table-grouped work distribution.
//
// Forward: a gather of 16-byte row chunks.  The ids are table-major and
// every work-group takes a contiguous run of them, so the grid sweeps the
// tables one after the other and all compute units work on the same one or
// two tables at any time: a hot table's rows are fetched into each XCD's L2
// once and reused by every work-group there.  Rows land either flat
// ([num_ids][D]) or straight in the token-major concatenated layout
// ([T][F*D]) that a sequence model consumes, so no conversion pass follows.
//
// Backward: deterministic sparse gradient.  Each id becomes its global row
// key (row_offsets[t] + id; invalid ids get a sentinel that sorts last); a
// stable radix sort orders the positions by key; a head-flag scan numbers
// the distinct rows; then fixed 32-position chunks of the sorted order sum
// the output-gradient rows of each distinct key in position order, writing
// rows that start and end inside a chunk directly and chunk-boundary pieces
// as partials that a fix-up pass joins in chunk order.  Every sum has a
// fixed order, so the result is bitwise reproducible (no float atomics),
// and a hot row that occurs thousands of times is summed by many chunks in
// parallel instead of by one serial loop.
#include <rocprim/device/device_radix_sort.hpp>
#include <rocprim/device/device_scan.hpp>

#include <algorithm>

#include "internal.h"
#include "device.h"
#include "../../include/hstu_embedding.h"

namespace hstu {
namespace {

constexpr int ET = 256;             // threads per work-group
constexpr int FWD_UNROLL = 4;       // 16-byte chunks in flight per thread
constexpr int CHUNK = 32;           // sorted positions per backward chunk
constexpr int MAX_TABLES = 1024;
constexpr int BWD_UNROLL = 8;       // gradient rows in flight per thread
constexpr int MAX_CPB = 16;         // backward chunks per work-group

// Threads per chunk and chunks per work-group of the backward chunk pass
// for `cpr` 16-byte slices per row (host and device agree on this).
__host__ __device__ __forceinline__ int chunk_tpc(int cpr) { return cpr < ET ? cpr : ET; }
__host__ __device__ __forceinline__ int chunk_cpb(int cpr) {
  const int c = ET / chunk_tpc(cpr);
  return c < MAX_CPB ? c : MAX_CPB;
}

// 16-byte vector of the row element type: 4 floats or 8 bf16.
template <typename T> struct Elt;
template <> struct Elt<float> { static constexpr int N = 4; };
template <> struct Elt<u16> { static constexpr int N = 8; };

__device__ __forceinline__ void add_chunk(float *acc, const uint4 &v, float) {
  acc[0] += __uint_as_float(v.x);
  acc[1] += __uint_as_float(v.y);
  acc[2] += __uint_as_float(v.z);
  acc[3] += __uint_as_float(v.w);
}
__device__ __forceinline__ void add_chunk(float *acc, const uint4 &v, u16) {
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    acc[2 * i] += __uint_as_float(w[i] << 16);
    acc[2 * i + 1] += __uint_as_float(w[i] & 0xffff0000u);
  }
}

// Table of id position r: the last t with id_offsets[t] <= r (empty tables
// are skipped because their successor has the same offset).
__device__ __forceinline__ int table_of(const int64_t *io, int F, int64_t r) {
  int lo = 0, hi = F - 1;
  while (lo < hi) {
    const int mid = (lo + hi + 1) >> 1;
    if (io[mid] <= r) lo = mid; else hi = mid - 1;
  }
  return lo;
}

// Table of id position r under the call's layout: in the token layout every
// table holds per_table ids, so the table follows from r alone (never from
// the offsets array, which keeps every output address in bounds whatever
// that array holds).
__device__ __forceinline__ int table_at(bool token, const int64_t *io, int F, int64_t r,
                                        int64_t per_table) {
  // (32-bit: num_ids < 2^31)
  return token ? (int)((uint32_t)r / (uint32_t)per_table) : table_of(io, F, r);
}

// Global row of id `id` in table t, or -1 if the id lies outside its table
// (or the table outside the weight matrix).
__device__ __forceinline__ int64_t global_row(const int64_t *ro, int t, int64_t id,
                                              int64_t total_rows) {
  const int64_t g = ro[t] + id;
  return (id >= 0 && id < ro[t + 1] - ro[t] && ro[t] >= 0 && g < total_rows) ? g : -1;
}

// Where row chunk c of id position r (table t) goes in the output layout.
__device__ __forceinline__ int64_t out_elem(bool token, int64_t r, int t, const int64_t *io,
                                            int F, int D, int64_t per_table, int c, int n_e) {
  return token ? (r - (int64_t)t * per_table) * ((int64_t)F * D) + (int64_t)t * D + c * n_e
               : r * D + c * n_e;
}

struct FwdArgs {
  const void *w;
  const int64_t *ro, *io, *ids;
  void *out;
  int64_t n, per_table, total_rows;
  int F, D, rows_per_block;
  bool token;
};

// Block b gathers id positions [b*RB, (b+1)*RB): thread x handles local
// chunks x, x+ET, ... of those rows (chunk = 16 bytes of a row).
template <typename T>
__global__ void __launch_bounds__(ET) emb_fwd_kernel(FwdArgs a) {
  __shared__ int64_t s_io[MAX_TABLES + 1], s_ro[MAX_TABLES + 1];
  constexpr int NE = Elt<T>::N;
  for (int i = threadIdx.x; i <= a.F; i += ET) {
    s_io[i] = a.io[i];
    s_ro[i] = a.ro[i];
  }
  __syncthreads();
  const int cpr = a.D / NE;
  const int64_t r0 = (int64_t)blockIdx.x * a.rows_per_block;
  const int local = a.rows_per_block * cpr;
  const T *W = (const T *)a.w;
  T *out = (T *)a.out;
  uint4 v[FWD_UNROLL];
  int64_t dst[FWD_UNROLL];
#pragma unroll
  for (int k = 0; k < FWD_UNROLL; ++k) {
    const int x = threadIdx.x + k * ET;
    dst[k] = -1;
    v[k] = make_uint4(0, 0, 0, 0);
    if (x < local) {
      const int64_t r = r0 + x / cpr;
      const int c = x % cpr;
      if (r < a.n) {
        const int t = table_at(a.token, s_io, a.F, r, a.per_table);
        const int64_t g = global_row(s_ro, t, a.ids[r], a.total_rows);
        if (g >= 0) v[k] = *(const uint4 *)(W + g * a.D + c * NE);
        dst[k] = out_elem(a.token, r, t, s_io, a.F, a.D, a.per_table, c, NE);
      }
    }
  }
#pragma unroll
  for (int k = 0; k < FWD_UNROLL; ++k)
    if (dst[k] >= 0) *(uint4 *)(out + dst[k]) = v[k];
}

// ---------------------------------------------------------------- backward
struct BwdArgs {
  const int64_t *ro, *io, *ids;
  const void *dout;
  float *grad;
  int64_t *unique_rows;
  int32_t *num_unique;
  uint64_t *keys_in, *keys;
  uint32_t *pos_in, *pos;
  uint32_t *flag, *runid;
  uint32_t *run_start;               // [num_ids]: first sorted position of each row
  uint32_t *last_valid;              // [1]: last sorted position with a valid key
  float *part;                       // [nchunks][2][D]
  uint64_t sentinel;                 // total_rows
  int64_t n, per_table;
  int F, D, nchunks;
  bool token;
};

__global__ void __launch_bounds__(ET) emb_keys_kernel(BwdArgs a) {
  __shared__ int64_t s_io[MAX_TABLES + 1], s_ro[MAX_TABLES + 1];
  for (int i = threadIdx.x; i <= a.F; i += ET) {
    s_io[i] = a.io[i];
    s_ro[i] = a.ro[i];
  }
  __syncthreads();
  const int64_t r = (int64_t)blockIdx.x * ET + threadIdx.x;
  if (r >= a.n) return;
  const int t = table_at(a.token, s_io, a.F, r, a.per_table);
  const int64_t g = global_row(s_ro, t, a.ids[r], (int64_t)a.sentinel);
  a.keys_in[r] = g >= 0 ? (uint64_t)g : a.sentinel;
  a.pos_in[r] = (uint32_t)r;
}

__global__ void __launch_bounds__(ET) emb_heads_kernel(BwdArgs a) {
  const int64_t p = (int64_t)blockIdx.x * ET + threadIdx.x;
  if (p >= a.n) return;
  const uint64_t k = a.keys[p];
  a.flag[p] = (k != a.sentinel && (p == 0 || a.keys[p - 1] != k)) ? 1u : 0u;
  if (k != a.sentinel && (p + 1 == a.n || a.keys[p + 1] == a.sentinel))
    *a.last_valid = (uint32_t)p;
}

// Output-gradient element offset of chunk c of id position r.
__device__ __forceinline__ int64_t dout_elem(const BwdArgs &a, uint32_t r, int c, int n_e) {
  if (!a.token) return (int64_t)r * a.D + c * n_e;
  const uint32_t t = r / (uint32_t)a.per_table;       // num_ids < 2^31
  return (int64_t)(r - t * (uint32_t)a.per_table) * ((int64_t)a.F * a.D) +
         (int64_t)t * a.D + c * n_e;
}

// One chunk of CHUNK sorted positions per group of `tpc` threads; a thread
// sums its 16-byte column slices over the chunk's pieces (runs of equal
// key) in position order.
template <typename T>
__global__ void __launch_bounds__(ET) emb_chunk_kernel(BwdArgs a) {
  constexpr int NE = Elt<T>::N;
  const int cpr = a.D / NE;
  const int tpc = chunk_tpc(cpr), cpb = chunk_cpb(cpr);
  __shared__ uint64_t s_key[MAX_CPB * CHUNK];
  __shared__ uint32_t s_pos[MAX_CPB * CHUNK];
  const int g = threadIdx.x / tpc, lt = threadIdx.x % tpc;
  const int64_t chunk = (int64_t)blockIdx.x * cpb + g;
  const int64_t p0 = chunk * CHUNK;
  // stage the keys and positions of this block's chunks
  for (int i = threadIdx.x; i < cpb * CHUNK; i += ET) {
    const int64_t p = (int64_t)blockIdx.x * cpb * CHUNK + i;
    s_key[i] = p < a.n ? a.keys[p] : a.sentinel;
    s_pos[i] = p < a.n ? a.pos[p] : 0u;
  }
  __syncthreads();
  if (g >= cpb || chunk >= a.nchunks) return;
  const uint64_t *key = s_key + g * CHUNK;
  const uint32_t *pos = s_pos + g * CHUNK;
  int pe = (int)std::min<int64_t>(CHUNK, a.n - p0);
  // sorted: the sentinel keys (invalid ids) form the array's tail
  int valid = 0;
  while (valid < pe && key[valid] != a.sentinel) ++valid;
  if (valid == 0) return;
  const T *G = (const T *)a.dout;
  const bool prev_same = p0 > 0 && a.keys[p0 - 1] == key[0];
  const bool next_same = valid == pe && p0 + pe < a.n && a.keys[p0 + pe] == key[pe - 1];
  for (int c = lt; c < cpr; c += tpc) {
    float acc[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) acc[e] = 0.0f;
    int start = 0;
    for (int q0 = 0; q0 < valid; q0 += BWD_UNROLL) {
      uint4 v[BWD_UNROLL];
#pragma unroll
      for (int u = 0; u < BWD_UNROLL; ++u)
        v[u] = q0 + u < valid ? *(const uint4 *)(G + dout_elem(a, pos[q0 + u], c, NE))
                              : make_uint4(0, 0, 0, 0);
#pragma unroll
      for (int u = 0; u < BWD_UNROLL; ++u) {
        const int q = q0 + u;
        if (q >= valid) break;
        add_chunk(acc, v[u], T{});
        const uint64_t k = key[q];
        if (q + 1 < valid && key[q + 1] == k) continue;
        // piece [start, q] of key k ends here
        const bool first = start > 0 || !prev_same;
        const bool last = q + 1 < valid || !next_same;
        float *dst;
        if (first && last) dst = a.grad + k * (uint64_t)a.D;
        else if (!first) dst = a.part + (chunk * 2 + 0) * a.D;
        else dst = a.part + (chunk * 2 + 1) * a.D;
#pragma unroll
        for (int e = 0; e < NE; e += 4)
          *(float4 *)(dst + c * NE + e) = make_float4(acc[e], acc[e + 1], acc[e + 2], acc[e + 3]);
        if (first && c == 0) {
          const uint32_t u = a.runid[p0 + start] - 1;
          a.run_start[u] = (uint32_t)(p0 + start);
          if (a.unique_rows) a.unique_rows[u] = (int64_t)k;
        }
#pragma unroll
        for (int e = 0; e < NE; ++e) acc[e] = 0.0f;
        start = q + 1;
      }
    }
  }
}

// Joins the pieces of rows that cross chunk boundaries.  Work-group b
// serves the row (if any) whose first position lies in chunk b and whose
// last lies in a later chunk: it finds that later chunk by binary search on
// the sorted keys, splits the chunks in between into one contiguous range
// per thread group, sums each range in chunk order, and adds the group sums
// to chunk b's own piece in group order -- a fixed order for a given batch,
// with a hot row's thousands of chunks shared by the whole work-group.
// Work-group 0 also publishes the distinct-row count.
template <typename T>
__global__ void __launch_bounds__(ET) emb_fixup_kernel(BwdArgs a) {
  constexpr int NE = Elt<T>::N;
  const int cpr = a.D / NE;
  const int tpc = chunk_tpc(cpr), groups = ET / tpc;
  __shared__ float s_sum[ET * NE];
  if (blockIdx.x == 0 && threadIdx.x == 0 && a.num_unique)
    *a.num_unique = a.n > 0 ? (int32_t)a.runid[a.n - 1] : 0;
  const int64_t chunk = blockIdx.x;
  const int64_t p0 = chunk * CHUNK;
  const int64_t pl = std::min<int64_t>(p0 + CHUNK, a.n) - 1;
  const uint64_t k = a.keys[pl];
  if (k == a.sentinel || pl + 1 >= a.n || a.keys[pl + 1] != k) return;
  if (p0 > 0 && a.keys[p0 - 1] == k && a.keys[p0] == k) return;   // starts earlier
  // last position of key k: just before the next row's first position
  const uint32_t u = a.runid[pl];                   // 1-based: this row is u-1
  const uint32_t nruns = a.runid[a.n - 1];
  const int64_t last = u < nruns ? (int64_t)a.run_start[u] - 1 : (int64_t)*a.last_valid;
  const int64_t c_end = last / CHUNK;               // last chunk holding key k
  const int64_t nparts = c_end - chunk;             // chunks chunk+1 .. c_end
  const int g = threadIdx.x / tpc, lt = threadIdx.x % tpc;
  const int64_t per = (nparts + groups - 1) / groups;
  const int64_t c_lo = chunk + 1 + g * per;
  const int64_t c_hi = std::min<int64_t>(c_lo + per, c_end + 1);
  // every thread runs the same number of slice rounds (the barriers inside)
  const int rounds = (cpr + tpc - 1) / tpc;
  for (int m = 0; m < rounds; ++m) {
    const int c = lt + m * tpc;
    const bool mine = g < groups && c < cpr;
    float acc[NE];
#pragma unroll
    for (int e = 0; e < NE; ++e) acc[e] = 0.0f;
    if (mine) {
      // loads of 4 chunks in flight, added in chunk order
      for (int64_t c0 = c_lo; c0 < c_hi; c0 += 4) {
        float4 x[4][NE / 4];
#pragma unroll
        for (int j = 0; j < 4; ++j)
#pragma unroll
          for (int e = 0; e < NE / 4; ++e)
            x[j][e] = c0 + j < c_hi
                          ? *(const float4 *)(a.part + ((c0 + j) * 2 + 0) * a.D + c * NE + 4 * e)
                          : make_float4(0.0f, 0.0f, 0.0f, 0.0f);
#pragma unroll
        for (int j = 0; j < 4; ++j) {
          if (c0 + j >= c_hi) break;
#pragma unroll
          for (int e = 0; e < NE / 4; ++e) {
            acc[4 * e] += x[j][e].x; acc[4 * e + 1] += x[j][e].y;
            acc[4 * e + 2] += x[j][e].z; acc[4 * e + 3] += x[j][e].w;
          }
        }
      }
    }
    __syncthreads();
    if (mine) {
#pragma unroll
      for (int e = 0; e < NE; ++e) s_sum[(g * tpc + lt) * NE + e] = acc[e];
    }
    __syncthreads();
    if (g == 0 && c < cpr) {
      const float *src = a.part + (chunk * 2 + 1) * a.D + c * NE;
#pragma unroll
      for (int e = 0; e < NE; ++e) acc[e] = src[e];
      for (int gi = 0; gi < groups; ++gi)
#pragma unroll
        for (int e = 0; e < NE; ++e) acc[e] += s_sum[(gi * tpc + lt) * NE + e];
      float *dst = a.grad + k * (uint64_t)a.D + c * NE;
#pragma unroll
      for (int e = 0; e < NE; e += 4)
        *(float4 *)(dst + e) = make_float4(acc[e], acc[e + 1], acc[e + 2], acc[e + 3]);
    }
  }
}

__global__ void emb_count_zero_kernel(int32_t *num_unique) { *num_unique = 0; }

// ------------------------------------------------------------------- host
int check_desc(const hstu_emb_desc *d) {
  if (!d) return fail(HSTU_EINVAL, "desc is NULL");
  if (d->dtype != HSTU_F32 && d->dtype != HSTU_BF16)
    return fail(HSTU_EINVAL, "dtype %d is not HSTU_F32 or HSTU_BF16", (int)d->dtype);
  if (d->num_tables < 0 || d->num_tables > MAX_TABLES)
    return fail(HSTU_EINVAL, "num_tables = %d outside [0, %d]", d->num_tables, MAX_TABLES);
  if (d->dim < 8 || d->dim > 4096 || d->dim % 8)
    return fail(HSTU_EINVAL, "dim = %d is not a multiple of 8 in [8, 4096]", d->dim);
  if (d->num_ids < 0 || d->num_ids >= (int64_t)1 << 31)
    return fail(HSTU_EINVAL, "num_ids = %lld outside [0, 2^31)", (long long)d->num_ids);
  if (d->total_rows < 0 || d->total_rows >= (int64_t)1 << 40)
    return fail(HSTU_EINVAL, "total_rows = %lld outside [0, 2^40)", (long long)d->total_rows);
  if (d->layout != HSTU_EMB_FLAT && d->layout != HSTU_EMB_TOKEN)
    return fail(HSTU_EINVAL, "layout %d is not HSTU_EMB_FLAT or HSTU_EMB_TOKEN",
                (int)d->layout);
  if (d->num_ids > 0 && d->num_tables == 0)
    return fail(HSTU_EINVAL, "num_ids = %lld with no tables", (long long)d->num_ids);
  if (d->layout == HSTU_EMB_TOKEN && d->num_tables > 0 && d->num_ids % d->num_tables)
    return fail(HSTU_EINVAL, "token layout: num_ids = %lld is not a multiple of %d tables",
                (long long)d->num_ids, d->num_tables);
  if (d->num_tables > 0 && (!d->row_offsets || !d->id_offsets))
    return fail(HSTU_EINVAL, "row_offsets and id_offsets must be non-null");
  return HSTU_OK;
}

int elt_n(const hstu_emb_desc *d) { return d->dtype == HSTU_F32 ? 4 : 8; }

struct BwdLayout {
  size_t keys_in, keys, pos_in, pos, flag, runid, run_start, last_valid, part, tmp, tmp_bytes,
      total;
};

BwdLayout bwd_layout(const hstu_emb_desc *d, size_t tmp_bytes) {
  const size_t n = (size_t)d->num_ids;
  const size_t nch = (n + CHUNK - 1) / CHUNK;
  BwdLayout L{};
  size_t o = 0;
  auto take = [&](size_t bytes) { const size_t at = o; o = align_up(o + bytes); return at; };
  L.keys_in = take(8 * n);
  L.keys = take(8 * n);
  L.pos_in = take(4 * n);
  L.pos = take(4 * n);
  L.flag = take(4 * n);
  L.runid = take(4 * n);
  L.run_start = take(4 * n);
  L.last_valid = take(4);
  L.part = take(sizeof(float) * 2 * nch * d->dim);
  L.tmp = take(tmp_bytes);
  L.tmp_bytes = tmp_bytes;
  L.total = o;
  return L;
}

// The sort runs the onesweep radix algorithm at every size above a single
// block (its merge-sort path for mid-size inputs is some twenty small
// launches, latency-bound at the batch sizes here).
using SortConfig = rocprim::radix_sort_config<rocprim::default_config, rocprim::default_config,
                                              rocprim::default_config, 0>;

unsigned key_bits(int64_t total_rows) {
  unsigned b = 1;
  while (b < 63 && ((uint64_t)1 << b) <= (uint64_t)total_rows) ++b;
  return b;                          // keys (and the sentinel) are < 2^b
}

// Temporary bytes of the sort and the scan (the larger of the two; they
// run one after the other on the stream).
hipError_t lib_tmp_bytes(int64_t n, int64_t total_rows, size_t *bytes) {
  size_t s1 = 0, s2 = 0;
  hipError_t e = rocprim::radix_sort_pairs<SortConfig>(nullptr, s1, (uint64_t *)nullptr,
                                           (uint64_t *)nullptr, (uint32_t *)nullptr,
                                           (uint32_t *)nullptr, (unsigned)n, 0,
                                           key_bits(total_rows));
  if (e != hipSuccess) return e;
  e = rocprim::inclusive_scan(nullptr, s2, (uint32_t *)nullptr, (uint32_t *)nullptr,
                              (size_t)n, rocprim::plus<uint32_t>());
  if (e != hipSuccess) return e;
  *bytes = std::max(s1, s2);
  return hipSuccess;
}

}  // namespace
}  // namespace hstu

using namespace hstu;

extern "C" int hstu_jagged_embedding_fwd(const hstu_emb_desc *desc, const void *weights,
                                         const int64_t *ids, void *out, void *stream) {
  clear_last_error();
  int rc = check_desc(desc);
  if (rc) return rc;
  if (desc->num_ids == 0) return HSTU_OK;
  if (!weights || !ids || !out) return fail(HSTU_EINVAL, "weights, ids and out must be non-null");
  const hipStream_t s = (hipStream_t)stream;
  FwdArgs a{};
  a.w = weights;
  a.ro = desc->row_offsets;
  a.io = desc->id_offsets;
  a.ids = ids;
  a.out = out;
  a.n = desc->num_ids;
  a.F = desc->num_tables;
  a.D = desc->dim;
  a.token = desc->layout == HSTU_EMB_TOKEN;
  a.per_table = a.token ? a.n / a.F : 0;
  a.total_rows = desc->total_rows;
  const int cpr = a.D / elt_n(desc);
  a.rows_per_block = std::max(1, ET * FWD_UNROLL / cpr);
  if (a.rows_per_block == 1 && cpr > ET * FWD_UNROLL)
    return fail(HSTU_ENOTSUP, "dim %d: a row exceeds one work-group's chunks", a.D);
  const int64_t grid = (a.n + a.rows_per_block - 1) / a.rows_per_block;
  {
    prof::Scope ps("emb_fwd", s);
    if (desc->dtype == HSTU_F32)
      hipLaunchKernelGGL(emb_fwd_kernel<float>, dim3((unsigned)grid), dim3(ET), 0, s, a);
    else
      hipLaunchKernelGGL(emb_fwd_kernel<u16>, dim3((unsigned)grid), dim3(ET), 0, s, a);
  }
  const hipError_t e = hipGetLastError();
  return e == hipSuccess ? HSTU_OK : hip_fail(e, "embedding forward launch");
}

extern "C" size_t hstu_jagged_embedding_bwd_workspace_bytes(const hstu_emb_desc *desc) {
  clear_last_error();
  if (check_desc(desc)) return 0;
  size_t tmp = 0;
  const hipError_t e = lib_tmp_bytes(desc->num_ids, desc->total_rows, &tmp);
  if (e != hipSuccess) {
    hip_fail(e, "sort/scan workspace query");
    return 0;
  }
  return bwd_layout(desc, tmp).total;
}

extern "C" int hstu_jagged_embedding_bwd(const hstu_emb_desc *desc, const int64_t *ids,
                                         const void *dout, float *grad_weights,
                                         int64_t *unique_rows, int32_t *num_unique,
                                         void *workspace, size_t workspace_bytes,
                                         void *stream) {
  clear_last_error();
  int rc = check_desc(desc);
  if (rc) return rc;
  const hipStream_t s = (hipStream_t)stream;
  const int64_t n = desc->num_ids;
  if (n == 0) {
    if (num_unique) {
      hipLaunchKernelGGL(emb_count_zero_kernel, dim3(1), dim3(1), 0, s, num_unique);
      const hipError_t e = hipGetLastError();
      if (e != hipSuccess) return hip_fail(e, "embedding backward launch");
    }
    return HSTU_OK;
  }
  if (!ids || !dout || !grad_weights)
    return fail(HSTU_EINVAL, "ids, dout and grad_weights must be non-null");
  size_t tmp = 0;
  hipError_t e = lib_tmp_bytes(n, desc->total_rows, &tmp);
  if (e != hipSuccess) return hip_fail(e, "sort/scan workspace query");
  const BwdLayout L = bwd_layout(desc, tmp);
  rc = check_workspace_bytes(L.total, workspace, workspace_bytes);
  if (rc) return rc;
  char *ws = (char *)workspace;
  BwdArgs a{};
  a.ro = desc->row_offsets;
  a.io = desc->id_offsets;
  a.ids = ids;
  a.dout = dout;
  a.grad = grad_weights;
  a.unique_rows = unique_rows;
  a.num_unique = num_unique;
  a.keys_in = (uint64_t *)(ws + L.keys_in);
  a.keys = (uint64_t *)(ws + L.keys);
  a.pos_in = (uint32_t *)(ws + L.pos_in);
  a.pos = (uint32_t *)(ws + L.pos);
  a.flag = (uint32_t *)(ws + L.flag);
  a.runid = (uint32_t *)(ws + L.runid);
  a.run_start = (uint32_t *)(ws + L.run_start);
  a.last_valid = (uint32_t *)(ws + L.last_valid);
  a.part = (float *)(ws + L.part);
  a.sentinel = (uint64_t)desc->total_rows;
  a.n = n;
  a.F = desc->num_tables;
  a.D = desc->dim;
  a.token = desc->layout == HSTU_EMB_TOKEN;
  a.per_table = a.token ? n / a.F : 0;
  a.nchunks = (int)((n + CHUNK - 1) / CHUNK);
  const int cpr = a.D / elt_n(desc);
  const int cpb = chunk_cpb(cpr);
  const unsigned grid_n = (unsigned)((n + ET - 1) / ET);
  prof::Scope ps("emb_bwd", s);
  hipLaunchKernelGGL(emb_keys_kernel, dim3(grid_n), dim3(ET), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "embedding key launch");
  size_t tb = L.tmp_bytes;
  e = rocprim::radix_sort_pairs<SortConfig>(ws + L.tmp, tb, a.keys_in, a.keys, a.pos_in, a.pos,
                                (unsigned)n, 0, key_bits(desc->total_rows), s);
  if (e != hipSuccess) return hip_fail(e, "embedding key sort");
  hipLaunchKernelGGL(emb_heads_kernel, dim3(grid_n), dim3(ET), 0, s, a);
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "embedding head launch");
  tb = L.tmp_bytes;
  e = rocprim::inclusive_scan(ws + L.tmp, tb, a.flag, a.runid, (size_t)n,
                              rocprim::plus<uint32_t>(), s);
  if (e != hipSuccess) return hip_fail(e, "embedding head scan");
  const unsigned grid_c = (unsigned)((a.nchunks + cpb - 1) / cpb);
  const unsigned grid_f = (unsigned)a.nchunks;
  if (desc->dtype == HSTU_F32) {
    hipLaunchKernelGGL(emb_chunk_kernel<float>, dim3(grid_c), dim3(ET), 0, s, a);
    hipLaunchKernelGGL(emb_fixup_kernel<float>, dim3(grid_f), dim3(ET), 0, s, a);
  } else {
    hipLaunchKernelGGL(emb_chunk_kernel<u16>, dim3(grid_c), dim3(ET), 0, s, a);
    hipLaunchKernelGGL(emb_fixup_kernel<u16>, dim3(grid_f), dim3(ET), 0, s, a);
  }
  if ((e = hipGetLastError()) != hipSuccess) return hip_fail(e, "embedding chunk launch");
  return HSTU_OK;
}
