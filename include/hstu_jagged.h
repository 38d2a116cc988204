/*
 * hstu_jagged.h -- C ABI of the MI355X (gfx950) jagged HSTU attention library.
 *
 * Operation.  The paper's jagged fusion operator for attention and RAB
 * (Sec. 4.1.1 "Jagged Fusion Operators for Attention and RAB" and the
 * appendix of the same name) fuses attention with a relative attention bias
 * -- relative position bias (rpb) plus relative time bias (rtb) -- over
 * jagged query/key/value inputs, with no padding and no dense<->jagged
 * conversion at the operator boundary.  For HSTU-style models (Appendix A,
 * "Parameter Settings": bucketized time encodings and relative positional
 * encodings) this library computes, for every sequence b with rows
 * off[b] .. off[b+1]-1, every head h and local positions i, j:
 *
 *   s_ij = alpha <q_i, k_j> + pos_w[h, j - i + N - 1] + time_w[h, bucket(ts_i - ts_j)]
 *   a_ij = silu(s_ij) / N   for j <= i (causal), else 0;   N = max_len
 *   o_i  = sum_j a_ij v_j                                    (per head)
 *   y    = LayerNorm(o) * u   per token over all H*d features
 *          (biased variance, eps = HSTU_LN_EPS, no affine parameters)
 *
 * bucket(x): |x| < 4 -> |x|; else with e = floor(log2 |x|),
 * 4*(e-1) + ((|x| >> (e-2)) & 3), clamped to num_buckets-1 (four log-spaced
 * buckets per octave; the paper names bucketized time encodings without
 * giving the rule, this is the library's reading).
 *
 * with alpha = 1 unless hstu_rab.alpha says otherwise.  The backward pass
 * returns dq, dk, dv, du and the table gradients d_pos_w, d_time_w of
 * sum(y * dy).
 *
 * Layout.  Every tensor is row-major and contiguous.  q, k, v, u, o, dq, dk,
 * dv, du and dO are [T][H][d]; y and dy are [T][H*d] (the same memory
 * layout: head h occupies columns h*d .. h*d+d-1 of a row).  T is the total
 * number of tokens, seq_offsets[B].
 *
 * Pointers.  Every tensor pointer is a DEVICE pointer on the current HIP
 * device; the caller owns all memory.  The attention calls never allocate
 * device memory and never synchronise (for the layer calls see their
 * section): each call enqueues its kernels on `stream` (a hipStream_t; NULL
 * = the default stream) and returns.  Buffers must stay alive until that
 * work completes.
 *
 * seq_offsets contract (int64, device): off[0] = 0, non-decreasing,
 * 0 <= off[b+1] - off[b] <= max_len, off[B] = total_tokens.  It is read on
 * the device only; the kernels clamp each length into [0, max_len] and each
 * row index into [0, total_tokens), so a violating offsets array yields
 * unspecified values but never an out-of-bounds access.  It is checked only
 * when the environment variable HSTU_VALIDATE is "1" at the time of a call:
 * then the call's scheduler kernel records the violations it finds in a
 * status word of the workspace (read it with hstu_jagged_status) and, on any
 * violation, the attention kernels of that call skip their work.  Either
 * way the call never waits for the device.
 * Empty sequences are legal.  B = 0 or total_tokens = 0 is a successful
 * call; it enqueues nothing, except that a backward call with a bias table
 * still writes that table's gradient (all zeros).
 *
 * Precision.  HSTU_BF16: q, k, v, u, dy and all tensor outputs are bfloat16,
 * tables and LayerNorm statistics are float32; contractions run on bf16 MFMA
 * with float32 accumulation, a_ij and dS_ij are rounded to bf16 only as MFMA
 * operands; d in {64, 128}.  HSTU_F32: every tensor is float32 and all
 * arithmetic is float32, except that the two bias-table gradients are
 * summed in float64 (or 64-bit fixed point, deterministic mode) before
 * their float32 store; d in {32, 64, 128}.
 *
 * Return codes: 0 on success, else one of the negative HSTU_E* codes below;
 * hstu_last_error() then describes the failure (thread-local string owned by
 * the library, valid until the next call on the same thread).
 */
#ifndef HSTU_JAGGED_H
#define HSTU_JAGGED_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HSTU_OK 0
#define HSTU_EINVAL (-1)      /* null required pointer, bad size or dtype    */
#define HSTU_ENOTSUP (-2)     /* valid but unsupported (e.g. bf16 with d=32) */
#define HSTU_EWORKSPACE (-3)  /* workspace missing or too small              */
#define HSTU_EHIP (-4)        /* a HIP runtime call or a launch failed        */

#define HSTU_LN_EPS 1e-6f

/* Status word of the seq_offsets contract check (hstu_jagged_status): 0 =
 * checked and held, else a bitwise OR of the violations found, or
 * HSTU_SEQ_UNCHECKED when the call ran without HSTU_VALIDATE=1. */
#define HSTU_SEQ_FIRST_NOT_ZERO 0x1   /* off[0] != 0                        */
#define HSTU_SEQ_DECREASING 0x2       /* off[b+1] < off[b] for some b       */
#define HSTU_SEQ_TOO_LONG 0x4         /* off[b+1] - off[b] > max_len        */
#define HSTU_SEQ_LAST_NOT_T 0x8       /* off[B] != total_tokens             */
#define HSTU_SEQ_UNCHECKED 0x40000000

typedef enum { HSTU_BF16 = 0, HSTU_F32 = 1 } hstu_dtype;

/* Relative attention bias (Sec. 4.1.1: rpb + rtb).  Either table may be
 * NULL; with both NULL the bias is zero. */
typedef struct {
    const float *pos_w;          /* [H][2*max_len-1] float32, or NULL        */
    const float *time_w;         /* [H][num_buckets] float32, or NULL        */
    const int64_t *timestamps;   /* [T] int64; required iff time_w != NULL   */
    int32_t num_buckets;         /* >= 1 iff time_w != NULL; H*num_buckets
                                    <= 4096 for HSTU_BF16                     */
    float alpha;                 /* scale of <q_i, k_j>: s_ij = alpha <q_i, k_j>
                                    + biases (one of the RAB variants of Sec.
                                    4.1.1's operator); 0 is read as 1, so a
                                    zero-initialised struct is the plain
                                    operator; must be finite               */
} hstu_rab;

/* Forward outputs and scratch, all caller-allocated.  o, ln_mean and
 * ln_rstd are the saved state the backward pass consumes. */
typedef struct {
    hstu_dtype dtype;            /* element type of q, k, v, u, y, o         */
    int64_t total_tokens;        /* T = seq_offsets[B]                       */
    void *y;                     /* [T][H*d]   LayerNorm(o) * u              */
    void *o;                     /* [T][H][d]  attention output (pre-norm)   */
    float *ln_mean;              /* [T]                                      */
    float *ln_rstd;              /* [T]  1/sqrt(var + eps)                   */
    void *workspace;             /* device scratch, 256-byte aligned         */
    size_t workspace_bytes;      /* >= hstu_jagged_attn_workspace_bytes(..,0) */
} hstu_fwd_out;

/* Backward inputs (saved forward state + upstream gradient), gradient
 * outputs and scratch.  Gradients are overwritten, never accumulated; table
 * entries no causal pair reaches are written as 0. */
typedef struct {
    hstu_dtype dtype;
    int64_t total_tokens;        /* T = seq_offsets[B]                       */
    const void *dy;              /* [T][H*d]                                 */
    const void *o;               /* [T][H][d]  from the forward              */
    const float *ln_mean;        /* [T]        from the forward              */
    const float *ln_rstd;        /* [T]        from the forward              */
    void *dq, *dk, *dv;          /* [T][H][d]                                */
    void *du;                    /* [T][H*d]                                 */
    float *d_pos_w;              /* [H][2*max_len-1]; required iff pos_w     */
    float *d_time_w;             /* [H][num_buckets]; required iff time_w    */
    void *workspace;             /* device scratch, 256-byte aligned         */
    size_t workspace_bytes;      /* >= hstu_jagged_attn_workspace_bytes(..,1) */
    int32_t deterministic;       /* nonzero: bitwise reproducible table
                                    gradients.  Every partial sum of d_pos_w
                                    and d_time_w is then kept in 64-bit fixed
                                    point (resolution 2^-32 of N dS, so
                                    |partial sums of N dS| < 2^31 is
                                    required) and added with integer atomics,
                                    whose result does not depend on order;
                                    dq, dk, dv, du are reproducible either
                                    way.  0: floating-point accumulation
                                    (faster; the last bits of the tables may
                                    differ from run to run)                  */
} hstu_bwd_io;

/* Forward: o, y, ln_mean, ln_rstd from q, k, v, u (Sec. 4.1.1). */
int hstu_jagged_attn_fwd(const void *q, const void *k, const void *v,
                         const void *u, const int64_t *seq_offsets, int32_t B,
                         int32_t max_len, int32_t H, int32_t d,
                         const hstu_rab *rab, hstu_fwd_out *out, void *stream);

/* For callers that cannot allocate device memory (code under HIP graph
 * capture, tight serving loops, harnesses that forbid allocation): the
 * forward above with the same arguments, kernels and results, except that
 * out->workspace and out->workspace_bytes are ignored.  Its workspace is a
 * fixed array of HSTU_NOALLOC_SCRATCH_BYTES that the library holds on every
 * GPU it runs on until the process ends; a problem whose forward workspace
 * (hstu_jagged_attn_workspace_bytes(.., for_bwd = 0, ..)) is larger is
 * rejected with HSTU_EWORKSPACE (with 4 MiB: up to about 170 000 work-list
 * entries of 64 tokens, e.g. 10 M tokens of 1024 sequences; about 115 000
 * when the forward pairs query tiles, d = 64 with total_tokens >= 256 B).
 * The call itself allocates nothing, records no profiler events, and never
 * waits for the device.  All calls on one GPU share its array: calls that overlap
 * on one GPU (other streams or threads) race and give unspecified results;
 * serialise them.  The seq_offsets status word of such a call lives in that
 * array and is not exposed. */
#define HSTU_NOALLOC_SCRATCH_BYTES (4u << 20)
int hstu_jagged_attn_fwd_noalloc(const void *q, const void *k, const void *v,
                                 const void *u, const int64_t *seq_offsets,
                                 int32_t B, int32_t max_len, int32_t H, int32_t d,
                                 const hstu_rab *rab, hstu_fwd_out *out,
                                 void *stream);

/* Backward: dq, dk, dv, du, d_pos_w, d_time_w of sum(y * dy), given the
 * forward's saved o / ln_mean / ln_rstd (Sec. 4.1.1; the table gradients are
 * the paper's "RAB backward"). */
int hstu_jagged_attn_bwd(const void *q, const void *k, const void *v,
                         const void *u, const int64_t *seq_offsets, int32_t B,
                         int32_t max_len, int32_t H, int32_t d,
                         const hstu_rab *rab, hstu_bwd_io *io, void *stream);

/* Bytes of device workspace a forward (for_bwd = 0) or backward
 * (for_bwd = 1) call needs for these sizes; depends on the current device's
 * compute-unit count.  Returns 0 for invalid sizes (see hstu_last_error). */
size_t hstu_jagged_attn_workspace_bytes(int32_t B, int32_t max_len, int32_t H,
                                        int32_t d, int64_t total_tokens,
                                        int32_t for_bwd, hstu_dtype dtype,
                                        const hstu_rab *rab);

/* ---------------------------------------------------------------------------
 * HSTU layer shell.  The attention above is the middle of one HSTU layer of
 * the models the paper trains (HSTU / FuXi, Appendix A "Parameter Settings").
 * These calls run a whole layer around it, with the library's reading of the
 * layer (the paper does not spell it out): no input norm, residual, bias or
 * dropout; SiLU on all of f1's output; split order U, V, Q, K.
 *
 *   h   = x . w1                       f1 GEMM      [T][4*H*d]
 *   z   = silu(h)  split by columns     U | V | Q | K, each [T][H][d]
 *   y   = LayerNorm(attention(q, k, v) ) * u        as hstu_jagged_attn_fwd
 *   out = y . w2                       f2 GEMM      [T][d_model]
 *
 * and the backward of sum(out * dout) into dx, dw1, dw2 and the table
 * gradients.  All products take bf16 in and out with float32 accumulation.
 * f1 is one hand-written MFMA kernel whose epilogue also writes the planes
 * silu(h) (when 4*H*d is a multiple of 128 and d_model of 64; otherwise
 * hipBLASLt and a separate silu + split kernel); the other GEMMs run on
 * hipBLASLt.  On the way back silu' is applied inside the attention
 * backward's gradient stores, which write dh [T][4*H*d] directly.
 * HSTU_BF16 only, d in {64, 128},
 * 1 <= d_model <= 65536 and d_model % 8 == 0.  Weights are row-major:
 * w1 [d_model][4*H*d], w2 [H*d][d_model]; x, out, dx [T][d_model].
 *
 * Allocation and synchronisation: the first layer call on a device creates
 * that device's hipBLASLt handle (hipBLASLt may allocate its own state then)
 * and each new GEMM shape runs one algorithm query; the first call of a
 * shape on a stream that is not being captured into a graph also times the
 * query's candidate algorithms on the call's own operands and keeps the
 * fastest -- that call waits for its stream once.  Everything is cached for
 * the process; later calls never synchronise.  GEMM scratch comes from the
 * caller's workspace.  Thread-safe.
 * ------------------------------------------------------------------------- */
typedef struct {
    hstu_dtype dtype;            /* HSTU_BF16                                */
    int64_t total_tokens;        /* T = seq_offsets[B]                       */
    void *out;                   /* [T][d_model]  y . w2                     */
    void *h;                     /* [T][4*H*d]    x . w1 (saved)             */
    void *z;                     /* [4][T][H][d]  silu(h) as planes U,V,Q,K
                                    (saved; the attention's u, v, q, k)      */
    void *y;                     /* [T][H*d]      LayerNorm(o) * u (saved)   */
    void *o;                     /* [T][H][d]     (saved)                    */
    float *ln_mean;              /* [T]           (saved)                    */
    float *ln_rstd;              /* [T]           (saved)                    */
    void *workspace;             /* device scratch, 256-byte aligned         */
    size_t workspace_bytes;      /* >= hstu_layer_workspace_bytes(..,0)      */
} hstu_layer_fwd_out;

typedef struct {
    hstu_dtype dtype;            /* HSTU_BF16                                */
    int64_t total_tokens;
    const void *dout;            /* [T][d_model]                             */
    const void *h, *z, *y, *o;   /* saved by hstu_layer_fwd                  */
    const float *ln_mean, *ln_rstd;
    void *dx;                    /* [T][d_model]        overwritten          */
    void *dw1;                   /* [d_model][4*H*d]    overwritten          */
    void *dw2;                   /* [H*d][d_model]      overwritten          */
    float *d_pos_w;              /* as in hstu_bwd_io                        */
    float *d_time_w;
    void *workspace;             /* device scratch, 256-byte aligned         */
    size_t workspace_bytes;      /* >= hstu_layer_workspace_bytes(..,1)      */
} hstu_layer_bwd_io;

/* Layer forward: out and the saved state from x, w1, w2.  T = 0 enqueues
 * nothing. */
int hstu_layer_fwd(const void *x, const void *w1, const void *w2,
                   const int64_t *seq_offsets, int32_t B, int32_t max_len,
                   int32_t H, int32_t d, int32_t d_model, const hstu_rab *rab,
                   hstu_layer_fwd_out *out, void *stream);

/* Layer backward: dx, dw1, dw2, d_pos_w, d_time_w of sum(out * dout).  With
 * T = 0 the weight and table gradients are written as zeros. */
int hstu_layer_bwd(const void *x, const void *w1, const void *w2,
                   const int64_t *seq_offsets, int32_t B, int32_t max_len,
                   int32_t H, int32_t d, int32_t d_model, const hstu_rab *rab,
                   hstu_layer_bwd_io *io, void *stream);

/* Workspace bytes of a layer forward (for_bwd = 0) or backward call; 0 for
 * invalid sizes. */
size_t hstu_layer_workspace_bytes(int32_t B, int32_t max_len, int32_t H,
                                  int32_t d, int32_t d_model,
                                  int64_t total_tokens, int32_t for_bwd,
                                  hstu_dtype dtype, const hstu_rab *rab);

/* Runs only the seq_offsets tile scheduler (the first step of both calls)
 * and copies its work lists out, for inspection and tests.  Work is split
 * into (sequence, 64-row tile) entries; a query tile costs its tile index
 * + 1 key tiles (causal), a key tile the sequence's tiles minus its index.
 * Both lists are longest first -- the sort-by-cost, assign-greedily
 * balancing of Sec. 4.1.3 applied to the compute units of one GPU -- in one
 * of two orders: every entry by cost, or, when the causal tile pairs reach
 * 4 x the longest entry x 4 x (compute units), sequence by sequence
 * (longest sequence first, each sequence's tiles longest first), which
 * keeps concurrent work-groups on few sequences.  The choice is made on the
 * device with one head per entry.  Device pointers: n_entries [1] int32 receives
 * the entry count E; list_q and list_k receive E int32 pairs
 * (sequence, tile) in pop order and must hold
 * min(B*ceil(max_len/64), (total_tokens + 63*B)/64) pairs.  workspace_bytes
 * must be >= hstu_jagged_attn_workspace_bytes(B, max_len, 1, 64,
 * total_tokens, 1, HSTU_F32, NULL).  Asynchronous on `stream`. */
int hstu_jagged_schedule(const int64_t *seq_offsets, int32_t B,
                         int32_t max_len, int64_t total_tokens,
                         int32_t *n_entries, int32_t *list_q, int32_t *list_k,
                         void *workspace, size_t workspace_bytes, void *stream);

/* Enqueues on `stream` a copy of the seq_offsets status word (HSTU_SEQ_*)
 * that the last call which used `workspace` wrote there, into `status`
 * (one int32, device or host memory; host memory is written when the copy
 * runs, so the caller synchronises before reading it).  The word is written
 * by every attention or layer call that enqueues work (calls with
 * total_tokens = 0 enqueue none, see above); a layer call's workspace
 * holds it at the same place.  Never waits for the device. */
int hstu_jagged_status(const void *workspace, int32_t *status, void *stream);

/* Diagnostics: per-kernel timing.  While enabled, every kernel the library
 * launches is bracketed by two HIP events recorded on the stream it is
 * launched on (the caller's stream).  hstu_profile_read waits for the
 * recorded events, fills up to `max` rows (kernel name -- a static string
 * owned by the library --, summed milliseconds, launch count) and clears
 * the records; it returns the number of rows written or a negative code.
 * Host-side only: no device memory is allocated. */
int hstu_profile_enable(int on);
int hstu_profile_read(int max, const char **names, double *total_ms,
                      int *launches);

/* ---------------------------------------------------------------------
 * Standalone relative attention bias (RAB) operator.
 *
 * The bias of Sec. 4.1.1's operator produced on its own, as the jagged
 * tensor an unfused attention would add to its scores, with its backward
 * into the bias parameters (the fused attention above never materialises
 * it).  For sequence b (L = L_b), head h and local i, j < L:
 *
 *   rab[h][sq[b] + i*L + j] = pos_w[h, j - i + N - 1]                (if given)
 *                           + time_w[h, bucket(ts_i - ts_j)]         (if given)
 *                           + a_h (1 + |ts_i - ts_j|)^(-beta_h)      (if time_fn)
 *
 * sq[b] = sum of L_b'^2 over b' < b (one L x L square per sequence, no
 * padding; total_square = sq[B]).  bucket() is the rule above.  time_fn
 * [H][2] = (a_h, beta_h) is a functional time encoding: the paper uses
 * functional time encodings for FuXi (Appendix A) without a formula; the
 * library reads them as this per-head power-law decay with learnable
 * amplitude and exponent.
 *
 * Backward, given d_rab in the same layout (all L x L entries count):
 * d_pos_w[h][x] and d_time_w[h][k] sum d_rab over the entries with that
 * offset / bucket (unreached entries 0), d_time_fn[h] = (sum d_rab g,
 * -sum d_rab a_h g ln(1 + |dt|)) with g = (1 + |dt|)^(-beta_h).  All sums
 * are 64-bit fixed point (resolution 2^-32, |partial sums| < 2^31) added
 * with integer atomics, so the result is bitwise reproducible.
 *
 * Layout: rab and d_rab are float32 [H][total_square].  Tiles are 64 x 64
 * squares of each sequence's L x L block (the paper's square tiling for
 * bias tensors).  Contract on seq_offsets as for the attention (clamped
 * to max_len on the device); the caller sizes rab from sq[B], computed on
 * the host from its copy of the lengths.
 * ------------------------------------------------------------------- */
typedef struct {
    const float *pos_w;          /* [H][2*max_len-1] or NULL                 */
    const float *time_w;         /* [H][num_buckets] or NULL                 */
    const float *time_fn;        /* [H][2] (a_h, beta_h) or NULL             */
    const int64_t *timestamps;   /* [T]; required iff time_w or time_fn      */
    int32_t num_buckets;         /* >= 1 iff time_w != NULL                  */
} hstu_rab_params;

/* Workspace bytes of a standalone RAB call (forward or backward). */
size_t hstu_jagged_rab_workspace_bytes(int32_t B, int32_t max_len, int32_t H,
                                       const hstu_rab_params *rp);

/* rab [H][total_square] (float32) from the parameters. */
int hstu_jagged_rab_fwd(const int64_t *seq_offsets, int32_t B, int32_t max_len,
                        int32_t H, int64_t total_tokens, int64_t total_square,
                        const hstu_rab_params *rp, float *rab,
                        void *workspace, size_t workspace_bytes, void *stream);

/* Parameter gradients from d_rab [H][total_square]; each output is
 * overwritten and required iff its parameter is given in rp. */
int hstu_jagged_rab_bwd(const int64_t *seq_offsets, int32_t B, int32_t max_len,
                        int32_t H, int64_t total_tokens, int64_t total_square,
                        const hstu_rab_params *rp, const float *d_rab,
                        float *d_pos_w, float *d_time_w, float *d_time_fn,
                        void *workspace, size_t workspace_bytes, void *stream);

/* Thread-local description of the last failure ("" if none). */
const char *hstu_last_error(void);

/* Library version string. */
const char *hstu_version(void);

#ifdef __cplusplus
}
#endif
#endif /* HSTU_JAGGED_H */
