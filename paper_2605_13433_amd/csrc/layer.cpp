// C ABI of the HSTU layer shell: f1 GEMM, SiLU + split, the jagged attention
// calls, f2 GEMM, and the backward through the same steps.
//
// The GEMMs are plain dense products over all T tokens (the jagged structure
// only matters inside the attention), so they go to hipBLASLt: bf16 operands
// and results, float32 accumulation.  Row-major products are issued as the
// column-major product of the transposes (C^T = op(B)^T op(A)^T), which
// hipBLASLt takes with the operands swapped and the same transpose flags.
#include <hip/hip_runtime.h>
#include <hipblaslt/hipblaslt.h>

#include <map>
#include <mutex>
#include <tuple>
#include <vector>

#include "internal.h"

namespace hstu {
namespace {

// hipBLASLt scratch carved from the caller's workspace for each GEMM.
constexpr size_t GEMM_WS_BYTES = size_t(32) << 20;
// Plans cached per device before the cache is flushed (one per distinct
// GEMM shape; the token count T is part of every shape).
constexpr size_t MAX_PLANS = 512;

int blas_fail(hipblasStatus_t st, const char *what) {
  return fail(HSTU_EHIP, "hipBLASLt %s failed (status %d)", what, (int)st);
}

// Row-major C[M][N] (ldc) = op(A)[M][K] . op(B)[K][N], A and B bf16, C bf16
// or (c32) float32; `batch` products at element strides sa, sb, sc.
struct GemmShape {
  bool ta, tb;
  int64_t M, N, K, lda, ldb, ldc;
  int32_t batch = 1;
  int64_t sa = 0, sb = 0, sc = 0;
  bool c32 = false;
  bool operator<(const GemmShape &o) const {
    return std::tie(ta, tb, M, N, K, lda, ldb, ldc, batch, sa, sb, sc, c32) <
           std::tie(o.ta, o.tb, o.M, o.N, o.K, o.lda, o.ldb, o.ldc, o.batch, o.sa, o.sb,
                    o.sc, o.c32);
  }
};

struct GemmPlan {
  hipblasLtMatmulDesc_t op = nullptr;
  hipblasLtMatrixLayout_t la = nullptr, lb = nullptr, lc = nullptr;
  hipblasLtMatmulAlgo_t algo;
  size_t ws = 0;
  // The heuristic's candidates; the first call of the shape outside graph
  // capture times them and keeps the fastest.
  std::vector<hipblasLtMatmulAlgo_t> cands;
  bool tuned = false;
};

void destroy(GemmPlan &g) {
  if (g.la) hipblasLtMatrixLayoutDestroy(g.la);
  if (g.lb) hipblasLtMatrixLayoutDestroy(g.lb);
  if (g.lc) hipblasLtMatrixLayoutDestroy(g.lc);
  if (g.op) hipblasLtMatmulDescDestroy(g.op);
  g = GemmPlan{};
}

struct DevBlas {
  hipblasLtHandle_t handle = nullptr;
  std::map<GemmShape, GemmPlan> plans;
};

std::mutex g_blas_mu;
std::vector<DevBlas> g_blas;

// Builds (or finds) the plan of one shape on device `dev`.  Caller holds
// g_blas_mu.
int get_plan(int dev, const GemmShape &g, GemmPlan **out) {
  if ((int)g_blas.size() <= dev) g_blas.resize(dev + 1);
  DevBlas &db = g_blas[dev];
  if (!db.handle) {
    hipblasStatus_t st = hipblasLtCreate(&db.handle);
    if (st != HIPBLAS_STATUS_SUCCESS) {
      db.handle = nullptr;
      return blas_fail(st, "handle creation");
    }
  }
  auto it = db.plans.find(g);
  if (it != db.plans.end()) {
    *out = &it->second;
    return HSTU_OK;
  }
  if (db.plans.size() >= MAX_PLANS) {
    for (auto &kv : db.plans) destroy(kv.second);
    db.plans.clear();
  }
  // Column-major view: D'[N x M] = op_b(B') [N x K] . op_a(A') [K x M].
  GemmPlan p;
  const hipblasOperation_t opa = g.tb ? HIPBLAS_OP_T : HIPBLAS_OP_N;  // on B
  const hipblasOperation_t opb = g.ta ? HIPBLAS_OP_T : HIPBLAS_OP_N;  // on A
  hipblasStatus_t st =
      hipblasLtMatmulDescCreate(&p.op, HIPBLAS_COMPUTE_32F, HIP_R_32F);
  if (st == HIPBLAS_STATUS_SUCCESS)
    st = hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_TRANSA,
                                         &opa, sizeof(int32_t));
  if (st == HIPBLAS_STATUS_SUCCESS)
    st = hipblasLtMatmulDescSetAttribute(p.op, HIPBLASLT_MATMUL_DESC_TRANSB,
                                         &opb, sizeof(int32_t));
  // Stored shapes in column-major terms (rows, cols, ld).
  if (st == HIPBLAS_STATUS_SUCCESS)
    st = hipblasLtMatrixLayoutCreate(&p.la, HIP_R_16BF, g.tb ? g.K : g.N,
                                     g.tb ? g.N : g.K, g.ldb);
  if (st == HIPBLAS_STATUS_SUCCESS)
    st = hipblasLtMatrixLayoutCreate(&p.lb, HIP_R_16BF, g.ta ? g.M : g.K,
                                     g.ta ? g.K : g.M, g.lda);
  if (st == HIPBLAS_STATUS_SUCCESS)
    st = hipblasLtMatrixLayoutCreate(&p.lc, g.c32 ? HIP_R_32F : HIP_R_16BF, g.N, g.M, g.ldc);
  if (g.batch > 1) {
    const int32_t n = g.batch;
    const hipblasLtMatrixLayout_t lay[3] = {p.la, p.lb, p.lc};
    const int64_t stride[3] = {g.sb, g.sa, g.sc};
    for (int i = 0; i < 3 && st == HIPBLAS_STATUS_SUCCESS; ++i) {
      st = hipblasLtMatrixLayoutSetAttribute(lay[i], HIPBLASLT_MATRIX_LAYOUT_BATCH_COUNT, &n,
                                             sizeof(n));
      if (st == HIPBLAS_STATUS_SUCCESS)
        st = hipblasLtMatrixLayoutSetAttribute(
            lay[i], HIPBLASLT_MATRIX_LAYOUT_STRIDED_BATCH_OFFSET, &stride[i], sizeof(int64_t));
    }
  }
  if (st != HIPBLAS_STATUS_SUCCESS) {
    destroy(p);
    return blas_fail(st, "descriptor creation");
  }
  hipblasLtMatmulPreference_t pref = nullptr;
  st = hipblasLtMatmulPreferenceCreate(&pref);
  uint64_t max_ws = GEMM_WS_BYTES;
  if (st == HIPBLAS_STATUS_SUCCESS)
    st = hipblasLtMatmulPreferenceSetAttribute(
        pref, HIPBLASLT_MATMUL_PREF_MAX_WORKSPACE_BYTES, &max_ws, sizeof(max_ws));
  constexpr int NRES = 16;
  hipblasLtMatmulHeuristicResult_t res[NRES];
  int n = 0;
  if (st == HIPBLAS_STATUS_SUCCESS)
    st = hipblasLtMatmulAlgoGetHeuristic(db.handle, p.op, p.la, p.lb, p.lc,
                                         p.lc, pref, NRES, res, &n);
  if (pref) hipblasLtMatmulPreferenceDestroy(pref);
  int pick = -1;
  for (int i = 0; st == HIPBLAS_STATUS_SUCCESS && i < n && pick < 0; ++i)
    if (res[i].state == HIPBLAS_STATUS_SUCCESS && res[i].workspaceSize <= GEMM_WS_BYTES)
      pick = i;
  if (st != HIPBLAS_STATUS_SUCCESS || pick < 0) {
    destroy(p);
    if (st != HIPBLAS_STATUS_SUCCESS) return blas_fail(st, "algorithm query");
    return fail(HSTU_ENOTSUP,
                "hipBLASLt has no algorithm for a %lld x %lld x %lld bf16 GEMM "
                "(ta=%d tb=%d; %d candidates, first state %d, workspace %zu)",
                (long long)g.M, (long long)g.N, (long long)g.K, (int)g.ta, (int)g.tb,
                n, n > 0 ? (int)res[0].state : -1, n > 0 ? res[0].workspaceSize : 0);
  }
  p.algo = res[pick].algo;
  p.ws = res[pick].workspaceSize;
  for (int i = pick; i < n; ++i)
    if (res[i].state == HIPBLAS_STATUS_SUCCESS && res[i].workspaceSize <= GEMM_WS_BYTES)
      p.cands.push_back(res[i].algo);
  *out = &db.plans.emplace(g, p).first->second;
  return HSTU_OK;
}

// Times every candidate algorithm of plan `p` on the call's own operands
// (two runs each, the second timed; C is rewritten by the call that
// follows) and keeps the fastest.  Skipped while `s` is being captured into
// a graph (no synchronisation is allowed there): the heuristic's first
// choice stays until an uncaptured call.  Returns false on a HIP error.
bool tune_plan(int dev, GemmPlan *p, const void *A, const void *B, void *C, void *ws,
               hipStream_t s) {
  hipStreamCaptureStatus cs = hipStreamCaptureStatusNone;
  if (hipStreamIsCapturing(s, &cs) != hipSuccess) return false;
  if (cs != hipStreamCaptureStatusNone || p->cands.size() < 2) {
    p->tuned = cs == hipStreamCaptureStatusNone;
    return true;
  }
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (hipEventCreate(&e0) != hipSuccess || hipEventCreate(&e1) != hipSuccess) {
    if (e0) hipEventDestroy(e0);
    return false;
  }
  const float alpha = 1.0f, beta = 0.0f;
  float best_ms = 0.0f;
  int best = -1;
  for (size_t i = 0; i < p->cands.size(); ++i) {
    bool ok = true;
    for (int rep = 0; rep < 2 && ok; ++rep) {
      if (rep == 1) ok = hipEventRecord(e0, s) == hipSuccess;
      ok = ok && hipblasLtMatmul(g_blas[dev].handle, p->op, &alpha, B, p->la, A, p->lb,
                                 &beta, C, p->lc, C, p->lc, &p->cands[i], ws,
                                 GEMM_WS_BYTES, s) == HIPBLAS_STATUS_SUCCESS;
      if (rep == 1) ok = ok && hipEventRecord(e1, s) == hipSuccess;
    }
    float ms = 0.0f;
    if (ok && hipEventSynchronize(e1) == hipSuccess &&
        hipEventElapsedTime(&ms, e0, e1) == hipSuccess && (best < 0 || ms < best_ms)) {
      best = (int)i;
      best_ms = ms;
    }
  }
  hipEventDestroy(e0);
  hipEventDestroy(e1);
  if (best >= 0) p->algo = p->cands[best];
  p->tuned = true;
  (void)hipGetLastError();   // a candidate that failed to launch left no state
  return true;
}

// Row-major C = op(A) . op(B) on `s`; `ws` holds GEMM_WS_BYTES.  `name`
// labels the profiler scope (none when NULL).
int gemm(int dev, const GemmShape &g, const void *A, const void *B, void *C,
         void *ws, hipStream_t s, const char *name) {
  std::lock_guard<std::mutex> lock(g_blas_mu);
  GemmPlan *p = nullptr;
  int rc = get_plan(dev, g, &p);
  if (rc != HSTU_OK) return rc;
  if (!p->tuned && !tune_plan(dev, p, A, B, C, ws, s))
    return fail(HSTU_EHIP, "GEMM algorithm timing failed (%s)", name ? name : "split part");
  const float alpha = 1.0f, beta = 0.0f;
  prof::Scope ps(name, s);
  hipblasStatus_t st = hipblasLtMatmul(g_blas[dev].handle, p->op, &alpha, B,
                                       p->la, A, p->lb, &beta, C, p->lc, C,
                                       p->lc, &p->algo, ws, GEMM_WS_BYTES, s);
  if (st != HIPBLAS_STATUS_SUCCESS) return blas_fail(st, name ? name : "split part");
  return HSTU_OK;
}

GemmShape rm(bool ta, bool tb, int64_t M, int64_t N, int64_t K, int64_t lda,
             int64_t ldb, int64_t ldc) {
  return GemmShape{ta, tb, M, N, K, lda, ldb, ldc};
}

// Weight gradients (K = T, small M x N) as split-K products: `parts`
// float32 partials of M x N, summed into the bf16 result.
constexpr int64_t SPLITK_MIN_ROWS = 1024;   // rows of T per part, at least
int splitk_parts(int64_t M, int64_t N, int64_t T) {
  const int64_t tiles = ((M + 127) / 128) * ((N + 127) / 128);
  int64_t s = std::min<int64_t>(16, std::max<int64_t>(1, 256 / std::max<int64_t>(tiles, 1)));
  while (s > 1 && T / s < SPLITK_MIN_ROWS) s /= 2;
  return (int)s;
}
// float32 partials of one split-K product (a remainder part included).
size_t splitk_bytes(int64_t M, int64_t N, int64_t T) {
  const int s = splitk_parts(M, N, T);
  return s > 1 ? sizeof(float) * (size_t)(M * N) * (size_t)(s + 1) : 0;
}

// Row-major C[M][N] (bf16, ldc = N) = A^T B with A [T][M] (lda) and B
// [T][N] (ldb) bf16: for `parts` > 1, `parts` equal row blocks of T as one
// strided batch of float32 products into `part`, the remaining rows as one
// more, then their sum.  `name` labels the whole operation.
int gemm_wgrad(int dev, int64_t M, int64_t N, int64_t T, const void *A, int64_t lda,
               const void *B, int64_t ldb, void *C, float *part, void *ws, hipStream_t s,
               const char *name) {
  const int parts = splitk_parts(M, N, T);
  if (parts <= 1) return gemm(dev, rm(true, false, M, N, T, lda, ldb, N), A, B, C, ws, s, name);
  prof::Scope ps(name, s);
  const int64_t rows = T / parts, rest = T - rows * parts;
  GemmShape g = rm(true, false, M, N, rows, lda, ldb, N);
  g.batch = parts;
  g.sa = rows * lda;
  g.sb = rows * ldb;
  g.sc = M * N;
  g.c32 = true;
  int rc = gemm(dev, g, A, B, part, ws, s, nullptr);
  if (rc != HSTU_OK) return rc;
  if (rest > 0) {
    GemmShape r = rm(true, false, M, N, rest, lda, ldb, N);
    r.c32 = true;
    rc = gemm(dev, r, (const char *)A + 2 * rows * parts * lda,
              (const char *)B + 2 * rows * parts * ldb, part + (size_t)parts * M * N, ws, s,
              nullptr);
    if (rc != HSTU_OK) return rc;
  }
  const hipError_t e = launch_sum_parts(part, C, M * N, parts + (rest > 0 ? 1 : 0), dev, s);
  return e == hipSuccess ? HSTU_OK : hip_fail(e, "split-K sum launch");
}

struct LayerLayout {
  size_t attn, gemm, dy, dh, part, total;
  size_t attn_bytes;
};

LayerLayout layer_layout(const Problem &p, int64_t D, bool for_bwd, int dev) {
  LayerLayout L{};
  size_t at = 0;
  auto take = [&](size_t bytes) {
    size_t off = at;
    at += align_up(bytes);
    return off;
  };
  const size_t C = (size_t)p.H * p.d;
  L.attn_bytes = make_layout(p, for_bwd, dev).total;
  L.attn = take(L.attn_bytes);
  L.gemm = take(GEMM_WS_BYTES);
  if (for_bwd) {
    L.dy = take(2 * (size_t)p.T * C);
    L.dh = take(2 * 4 * (size_t)p.T * C);
    // dW2 [C][D] and dW1 [D][4C] run one after the other: one partial area
    L.part = take(std::max(splitk_bytes(C, D, p.T), splitk_bytes(D, 4 * C, p.T)));
  }
  L.total = at;
  return L;
}

int validate_layer(const void *x, const void *w1, const void *w2,
                   const int64_t *off, int32_t B, int32_t N, int32_t H,
                   int32_t d, int32_t D, const hstu_rab *rab, hstu_dtype dtype,
                   int64_t T, const void *z, Problem *p) {
  if (dtype != HSTU_BF16)
    return fail(HSTU_ENOTSUP, "the layer calls support HSTU_BF16 only");
  if (D < 1 || D > 65536 || D % 8)
    return fail(HSTU_EINVAL, "d_model = %d must be in [8, 65536] and a multiple of 8", D);
  int rc = validate(z, z, z, z, off, B, N, H, d, rab, dtype, T, p);
  if (rc != HSTU_OK) return rc;
  if (T > 0 && (!x || !w1 || !w2))
    return fail(HSTU_EINVAL, "x, w1 and w2 must be non-null when total_tokens > 0");
  return HSTU_OK;
}

}  // namespace
}  // namespace hstu

using namespace hstu;

extern "C" {

size_t hstu_layer_workspace_bytes(int32_t B, int32_t max_len, int32_t H,
                                  int32_t d, int32_t d_model,
                                  int64_t total_tokens, int32_t for_bwd,
                                  hstu_dtype dtype, const hstu_rab *rab) {
  clear_last_error();
  static const char dummy = 0;
  Problem p;
  if (validate_layer(&dummy, &dummy, &dummy, (const int64_t *)&dummy, B,
                     max_len, H, d, d_model, rab, dtype, total_tokens, &dummy,
                     &p) != HSTU_OK)
    return 0;
  int dev = 0;
  if (current_device(&dev) != HSTU_OK) return 0;
  return layer_layout(p, d_model, for_bwd != 0, dev).total;
}

int hstu_layer_fwd(const void *x, const void *w1, const void *w2,
                   const int64_t *seq_offsets, int32_t B, int32_t max_len,
                   int32_t H, int32_t d, int32_t d_model, const hstu_rab *rab,
                   hstu_layer_fwd_out *out, void *stream) {
  clear_last_error();
  if (!out) return fail(HSTU_EINVAL, "out is NULL");
  Problem p;
  int rc = validate_layer(x, w1, w2, seq_offsets, B, max_len, H, d, d_model,
                          rab, out->dtype, out->total_tokens, out->z, &p);
  if (rc != HSTU_OK) return rc;
  const int64_t T = p.T;
  if (T > 0 && (!out->out || !out->h || !out->y || !out->o || !out->ln_mean ||
                !out->ln_rstd))
    return fail(HSTU_EINVAL, "out->out, h, z, y, o, ln_mean, ln_rstd must be non-null");
  if (T == 0) return HSTU_OK;
  int dev = 0;
  if ((rc = current_device(&dev)) != HSTU_OK) return rc;
  const LayerLayout L = layer_layout(p, d_model, false, dev);
  if ((rc = check_workspace_bytes(L.total, out->workspace, out->workspace_bytes)) != HSTU_OK)
    return rc;
  hipStream_t s = (hipStream_t)stream;
  char *ws = (char *)out->workspace;
  const int64_t C = (int64_t)H * d, D = d_model;
  char *z = (char *)out->z;
  const size_t plane = 2 * (size_t)T * C;

  hipError_t e;
  if (gemm_f1_silu_supported(4 * C, D)) {
    // h = x . w1 and the U, V, Q, K planes silu(h) from one hand-written
    // kernel (the split is the epilogue's store address)
    prof::Scope ps("gemm_f1_silu", s);
    e = launch_gemm_f1_silu(x, w1, out->h, z, T, (int32_t)(4 * C), D, s);
    if (e != hipSuccess) return hip_fail(e, "f1 launch");
  } else {
    // h = x . w1 on hipBLASLt, then the SiLU + split pass
    if ((rc = gemm(dev, rm(false, false, T, 4 * C, D, D, 4 * C, 4 * C), x, w1,
                   out->h, ws + L.gemm, s, "gemm_f1")) != HSTU_OK)
      return rc;
    prof::Scope ps("silu_split", s);
    e = launch_silu_split(out->h, z, T, (int32_t)C, dev, s);
    if (e != hipSuccess) return hip_fail(e, "silu split launch");
  }
  hstu_fwd_out fo{HSTU_BF16, T, out->y, out->o, out->ln_mean, out->ln_rstd,
                  ws + L.attn, L.attn_bytes};
  rc = hstu_jagged_attn_fwd(z + 2 * plane, z + 3 * plane, z + plane, z,
                            seq_offsets, B, max_len, H, d, rab, &fo, stream);
  if (rc != HSTU_OK) return rc;
  // out = y . w2
  return gemm(dev, rm(false, false, T, D, C, C, D, D), out->y, w2, out->out,
              ws + L.gemm, s, "gemm_f2");
}

int hstu_layer_bwd(const void *x, const void *w1, const void *w2,
                   const int64_t *seq_offsets, int32_t B, int32_t max_len,
                   int32_t H, int32_t d, int32_t d_model, const hstu_rab *rab,
                   hstu_layer_bwd_io *io, void *stream) {
  clear_last_error();
  if (!io) return fail(HSTU_EINVAL, "io is NULL");
  Problem p;
  int rc = validate_layer(x, w1, w2, seq_offsets, B, max_len, H, d, d_model,
                          rab, io->dtype, io->total_tokens, io->z, &p);
  if (rc != HSTU_OK) return rc;
  const int64_t T = p.T;
  if (T > 0 && (!io->dout || !io->h || !io->y || !io->o || !io->ln_mean ||
                !io->ln_rstd || !io->dx))
    return fail(HSTU_EINVAL, "io->dout, h, z, y, o, ln_mean, ln_rstd, dx must be non-null");
  if (!io->dw1 || !io->dw2) return fail(HSTU_EINVAL, "io->dw1 and dw2 must be non-null");
  if (p.has_pos && !io->d_pos_w)
    return fail(HSTU_EINVAL, "rab->pos_w given but io->d_pos_w is NULL");
  if (p.has_time && !io->d_time_w)
    return fail(HSTU_EINVAL, "rab->time_w given but io->d_time_w is NULL");
  int dev = 0;
  if ((rc = current_device(&dev)) != HSTU_OK) return rc;
  const LayerLayout L = layer_layout(p, d_model, true, dev);
  if ((rc = check_workspace_bytes(L.total, io->workspace, io->workspace_bytes)) != HSTU_OK)
    return rc;
  hipStream_t s = (hipStream_t)stream;
  char *ws = (char *)io->workspace;
  const int64_t C = (int64_t)H * d, D = d_model;
  const char *z = (const char *)io->z;
  const uint16_t *h = (const uint16_t *)io->h;
  uint16_t *dh = (uint16_t *)(ws + L.dh);   // bf16 elements
  const size_t plane = 2 * (size_t)T * C;
  hipError_t e;

  if (T == 0) {
    prof::Scope ps("zero_fill", s);
    e = launch_zero(io->dw1, 2 * (size_t)D * 4 * C, dev, s);
    if (e == hipSuccess) e = launch_zero(io->dw2, 2 * (size_t)C * D, dev, s);
    if (e != hipSuccess) return hip_fail(e, "zero fill launch");
  } else {
    // dy = dout . w2^T ;  dw2 = y^T . dout
    if ((rc = gemm(dev, rm(false, true, T, C, D, D, D, C), io->dout, w2,
                   ws + L.dy, ws + L.gemm, s, "gemm_dy")) != HSTU_OK)
      return rc;
    if ((rc = gemm_wgrad(dev, C, D, T, io->y, C, io->dout, D, io->dw2,
                         (float *)(ws + L.part), ws + L.gemm, s, "gemm_dw2")) != HSTU_OK)
      return rc;
  }
  // Attention backward straight into dh [T][4C]: every gradient of the
  // U, V, Q, K planes is multiplied by silu'(h) at its store, so the planes
  // dz are never written.  Also writes the table gradients (zeros when
  // T = 0).
  hstu_bwd_io bo{HSTU_BF16, T, ws + L.dy, io->o, io->ln_mean, io->ln_rstd,
                 dh + 2 * C, dh + 3 * C, dh + C, dh,
                 io->d_pos_w, io->d_time_w, ws + L.attn, L.attn_bytes};
  const GradOut go{(int32_t)(4 * C), h + 2 * C, h + 3 * C, h + C, h};
  rc = attn_bwd_call(z + 2 * plane, z + 3 * plane, z + plane, z, seq_offsets, B, max_len, H,
                     d, rab, &bo, stream, &go);
  if (rc != HSTU_OK || T == 0) return rc;
  // dx = dh . w1^T ;  dw1 = x^T . dh
  if ((rc = gemm(dev, rm(false, true, T, D, 4 * C, 4 * C, 4 * C, D), ws + L.dh,
                 w1, io->dx, ws + L.gemm, s, "gemm_dx")) != HSTU_OK)
    return rc;
  return gemm_wgrad(dev, D, 4 * C, T, x, D, ws + L.dh, 4 * C, io->dw1,
                    (float *)(ws + L.part), ws + L.gemm, s, "gemm_dw1");
}

}  // extern "C"
