/*
 * CPU oracle for jagged HSTU pointwise attention, forward and backward.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing on the product path may link, load or
 * call this file: it exists so that tests, the smoke check and the CPU
 * baseline leg of the benchmark can compare the HIP kernels against a plain,
 * slow, obviously correct computation.  It shares no code, header, table or
 * helper with the HIP library.
 *
 * What it computes.  The paper (Sec. 4.1.1 "Jagged Fusion Operators for
 * Attention and RAB", and its appendix of the same name) fuses attention with
 * a relative attention bias (RAB = relative position bias + relative time
 * bias) over jagged inputs without padding, for HSTU-style models
 * (Appendix A, "Parameter Settings": bucketized time encodings plus relative
 * positional encodings).  The paper does not print the arithmetic; the
 * definition used here is HSTU's pointwise attention as the operator is
 * specified for this library:
 *
 *   for every sequence b (rows off[b] .. off[b+1]-1), head h, local i, j:
 *     s_ij = alpha <q_i, k_j> + w_pos[h, j - i + N - 1] + w_time[h, bucket(ts_i - ts_j)]
 *     a_ij = silu(s_ij) / N  if j <= i, else 0          (N = max_len)
 *     o_i  = sum_j a_ij v_j
 *   per token: z = concat_h o[h]; n = (z - mean z) / sqrt(var z + eps)
 *     (biased variance, no affine); y = n * u.
 *
 * alpha is an optional scale of the query-key product (1 gives the plain
 * operator; the paper's RAB variants include such a scale, unstated in
 * value, so the library reads it as a caller-chosen constant).
 *
 * Everything is double precision; inputs are the exact values of whatever
 * lower precision the caller used.  Loops run in the plainest order
 * (sequence, head, i, j, e) with no blocking or reordering, parallelised over
 * (sequence, head) pairs only.
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

/* Time-difference bucket: |delta| below 4 is its own bucket; above, four
 * buckets per octave, i.e. with e = floor(log2 x) the bucket is
 * 4(e-1) + (the two bits of x just below its leading one); clamped to nb-1.
 * (The paper names 32 log buckets for HSTU without giving the rule; this is
 * the reading the library adopts, an integer rule so that CPU and GPU agree
 * bit for bit.) */
int hstu_oracle_time_bucket(int64_t delta, int32_t nb)
{
    uint64_t x = delta < 0 ? (uint64_t)0 - (uint64_t)delta : (uint64_t)delta;
    int64_t bkt;
    if (x < 4) {
        bkt = (int64_t)x;
    } else {
        int e = 0;                       /* floor(log2 x) by repeated halving */
        while ((x >> (e + 1)) != 0) e++;
        int m = (int)((x >> (e - 2)) & 3u);
        bkt = 4 * (int64_t)(e - 1) + m;
    }
    if (bkt > nb - 1) bkt = nb - 1;
    return (int)bkt;
}

static double silu(double x) { return x / (1.0 + exp(-x)); }

static double sigmoid(double x) { return 1.0 / (1.0 + exp(-x)); }

/* Bias added to score (i, j) of head h; i, j are local positions, r, c the
 * global rows of the query and the key. */
static double rab(const double *pos_w, const double *time_w,
                  const int64_t *ts, int32_t nb, int32_t N, int32_t h,
                  int64_t i, int64_t j, int64_t r, int64_t c)
{
    double b = 0.0;
    if (pos_w) b += pos_w[(int64_t)h * (2 * N - 1) + (j - i + N - 1)];
    if (time_w) b += time_w[(int64_t)h * nb + hstu_oracle_time_bucket(ts[r] - ts[c], nb)];
    return b;
}

static int check_args(const int64_t *off, int32_t B, int32_t N, int32_t H,
                      int32_t d, const double *time_w, const int64_t *ts,
                      int32_t nb)
{
    if (B < 0 || N < 1 || H < 1 || d < 1) return -1;
    if (time_w && (!ts || nb < 1)) return -1;
    if (off[0] != 0) return -1;
    for (int32_t b = 0; b < B; ++b) {
        int64_t L = off[b + 1] - off[b];
        if (L < 0 || L > N) return -1;
    }
    return 0;
}

/* Attention output o[T][H][d] only (step 2 of the definition). */
static void attention(const double *q, const double *k, const double *v,
                      const int64_t *off, int32_t B, int32_t N, int32_t H,
                      int32_t d, const double *pos_w, const double *time_w,
                      const int64_t *ts, int32_t nb, double alpha, double *o)
{
    const int64_t row = (int64_t)H * d;
    const int64_t nbh = (int64_t)B * H;
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t bh = 0; bh < nbh; ++bh) {
        const int32_t b = (int32_t)(bh / H), h = (int32_t)(bh % H);
        const int64_t o0 = off[b], L = off[b + 1] - off[b];
        for (int64_t i = 0; i < L; ++i) {
            const int64_t r = o0 + i;
            double *oi = o + r * row + (int64_t)h * d;
            for (int32_t e = 0; e < d; ++e) oi[e] = 0.0;
            for (int64_t j = 0; j <= i; ++j) {
                const int64_t c = o0 + j;
                const double *qi = q + r * row + (int64_t)h * d;
                const double *kj = k + c * row + (int64_t)h * d;
                const double *vj = v + c * row + (int64_t)h * d;
                double s = 0.0;
                for (int32_t e = 0; e < d; ++e) s += qi[e] * kj[e];
                s = alpha * s + rab(pos_w, time_w, ts, nb, N, h, i, j, r, c);
                const double a = silu(s) / (double)N;
                for (int32_t e = 0; e < d; ++e) oi[e] += a * vj[e];
            }
        }
    }
}

/* Per-token LayerNorm statistics over all H*d features (step 3). */
static void ln_stats(const double *o, int64_t T, int64_t row, double eps,
                     double *mean, double *rstd)
{
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < T; ++r) {
        const double *z = o + r * row;
        double mu = 0.0;
        for (int64_t f = 0; f < row; ++f) mu += z[f];
        mu /= (double)row;
        double var = 0.0;
        for (int64_t f = 0; f < row; ++f) var += (z[f] - mu) * (z[f] - mu);
        var /= (double)row;
        mean[r] = mu;
        rstd[r] = 1.0 / sqrt(var + eps);
    }
}

/*
 * Forward.  Outputs: o [T][H][d], y [T][H*d], ln_mean [T], ln_rstd [T]
 * (y = (o - mean) * rstd * u).  pos_w [H][2N-1] and time_w [H][nb] may be
 * NULL; timestamps are required when time_w is given.  Returns 0, or -1 on
 * inconsistent arguments.
 */
int hstu_oracle_fwd(const double *q, const double *k, const double *v,
                    const double *u, const int64_t *seq_offsets, int32_t B,
                    int32_t max_len, int32_t H, int32_t d,
                    const double *pos_w, const double *time_w,
                    const int64_t *timestamps, int32_t num_buckets, double eps,
                    double alpha, double *o, double *y, double *ln_mean, double *ln_rstd)
{
    if (check_args(seq_offsets, B, max_len, H, d, time_w, timestamps, num_buckets))
        return -1;
    const int64_t T = seq_offsets[B], row = (int64_t)H * d;
    attention(q, k, v, seq_offsets, B, max_len, H, d, pos_w, time_w,
              timestamps, num_buckets, alpha, o);
    ln_stats(o, T, row, eps, ln_mean, ln_rstd);
    for (int64_t r = 0; r < T; ++r)
        for (int64_t f = 0; f < row; ++f)
            y[r * row + f] = (o[r * row + f] - ln_mean[r]) * ln_rstd[r] * u[r * row + f];
    return 0;
}

/*
 * Backward.  Recomputes the forward in double, then, given dy [T][H*d]:
 *   du = n * dy;  g = dy * u;
 *   do = rstd * (g - mean(g) - n * mean(g * n))            (LayerNorm backward)
 *   dA_ij = <do_i, v_j>;  dS_ij = dA_ij * silu'(s_ij) / N   (j <= i)
 *   dv_j += a_ij do_i;  dq_i += alpha dS_ij k_j;  dk_j += alpha dS_ij q_i;
 *   d_pos[h, j-i+N-1] += dS_ij;  d_time[h, bucket] += dS_ij
 * with silu'(x) = sigma(x) (1 + x (1 - sigma(x))).  All gradients are
 * overwritten.  d_pos_w / d_time_w are required iff the matching table is
 * given.  Returns 0, -1 on inconsistent arguments, -2 on allocation failure.
 */
int hstu_oracle_bwd(const double *q, const double *k, const double *v,
                    const double *u, const int64_t *seq_offsets, int32_t B,
                    int32_t max_len, int32_t H, int32_t d,
                    const double *pos_w, const double *time_w,
                    const int64_t *timestamps, int32_t num_buckets, double eps,
                    double alpha, const double *dy, double *dq, double *dk, double *dv,
                    double *du, double *d_pos_w, double *d_time_w)
{
    if (check_args(seq_offsets, B, max_len, H, d, time_w, timestamps, num_buckets))
        return -1;
    if ((pos_w && !d_pos_w) || (time_w && !d_time_w)) return -1;
    const int32_t N = max_len, nb = num_buckets;
    const int64_t T = seq_offsets[B], row = (int64_t)H * d;
    const int64_t npos = (int64_t)H * (2 * N - 1), ntime = time_w ? (int64_t)H * nb : 0;

    double *o = malloc(sizeof(double) * (size_t)(T * row + 1));
    double *dO = malloc(sizeof(double) * (size_t)(T * row + 1));
    double *mean = malloc(sizeof(double) * (size_t)(T + 1));
    double *rstd = malloc(sizeof(double) * (size_t)(T + 1));
    if (!o || !dO || !mean || !rstd) {
        free(o); free(dO); free(mean); free(rstd);
        return -2;
    }
    attention(q, k, v, seq_offsets, B, N, H, d, pos_w, time_w, timestamps, nb, alpha, o);
    ln_stats(o, T, row, eps, mean, rstd);

    /* LayerNorm + gate backward, per token. */
#pragma omp parallel for schedule(static)
    for (int64_t r = 0; r < T; ++r) {
        const double *z = o + r * row, *dyr = dy + r * row, *ur = u + r * row;
        double mg = 0.0, mgn = 0.0;
        for (int64_t f = 0; f < row; ++f) {
            const double n = (z[f] - mean[r]) * rstd[r];
            const double g = dyr[f] * ur[f];
            du[r * row + f] = n * dyr[f];
            mg += g;
            mgn += g * n;
        }
        mg /= (double)row;
        mgn /= (double)row;
        for (int64_t f = 0; f < row; ++f) {
            const double n = (z[f] - mean[r]) * rstd[r];
            const double g = dyr[f] * ur[f];
            dO[r * row + f] = rstd[r] * (g - mg - n * mgn);
        }
    }

    memset(dq, 0, sizeof(double) * (size_t)(T * row));
    memset(dk, 0, sizeof(double) * (size_t)(T * row));
    memset(dv, 0, sizeof(double) * (size_t)(T * row));

    /* Table gradients: one private copy per thread, summed in thread order. */
    int nthreads = 1;
#ifdef _OPENMP
    nthreads = omp_get_max_threads();
#endif
    const int64_t ntab = npos + ntime;
    double *tab = calloc((size_t)(ntab * nthreads + 1), sizeof(double));
    if (!tab) {
        free(o); free(dO); free(mean); free(rstd);
        return -2;
    }

    const int64_t nbh = (int64_t)B * H;
#pragma omp parallel
    {
        int tid = 0;
#ifdef _OPENMP
        tid = omp_get_thread_num();
#endif
        double *my_pos = tab + (int64_t)tid * ntab;
        double *my_time = my_pos + npos;
#pragma omp for schedule(dynamic, 1)
        for (int64_t bh = 0; bh < nbh; ++bh) {
            const int32_t b = (int32_t)(bh / H), h = (int32_t)(bh % H);
            const int64_t o0 = seq_offsets[b], L = seq_offsets[b + 1] - seq_offsets[b];
            for (int64_t i = 0; i < L; ++i) {
                const int64_t r = o0 + i;
                const double *qi = q + r * row + (int64_t)h * d;
                const double *doi = dO + r * row + (int64_t)h * d;
                double *dqi = dq + r * row + (int64_t)h * d;
                for (int64_t j = 0; j <= i; ++j) {
                    const int64_t c = o0 + j;
                    const double *kj = k + c * row + (int64_t)h * d;
                    const double *vj = v + c * row + (int64_t)h * d;
                    double *dkj = dk + c * row + (int64_t)h * d;
                    double *dvj = dv + c * row + (int64_t)h * d;
                    double s = 0.0, dA = 0.0;
                    for (int32_t e = 0; e < d; ++e) s += qi[e] * kj[e];
                    s = alpha * s + rab(pos_w, time_w, timestamps, nb, N, h, i, j, r, c);
                    for (int32_t e = 0; e < d; ++e) dA += doi[e] * vj[e];
                    const double sg = sigmoid(s);
                    const double a = silu(s) / (double)N;
                    const double dS = dA * sg * (1.0 + s * (1.0 - sg)) / (double)N;
                    for (int32_t e = 0; e < d; ++e) {
                        dvj[e] += a * doi[e];
                        dqi[e] += alpha * dS * kj[e];
                        dkj[e] += alpha * dS * qi[e];
                    }
                    if (pos_w) my_pos[(int64_t)h * (2 * N - 1) + (j - i + N - 1)] += dS;
                    if (time_w)
                        my_time[(int64_t)h * nb +
                                hstu_oracle_time_bucket(timestamps[r] - timestamps[c], nb)] += dS;
                }
            }
        }
    }
    if (d_pos_w) {
        memset(d_pos_w, 0, sizeof(double) * (size_t)npos);
        for (int t = 0; t < nthreads; ++t)
            for (int64_t x = 0; x < npos; ++x) d_pos_w[x] += tab[(int64_t)t * ntab + x];
    }
    if (d_time_w) {
        memset(d_time_w, 0, sizeof(double) * (size_t)ntime);
        for (int t = 0; t < nthreads; ++t)
            for (int64_t x = 0; x < ntime; ++x)
                d_time_w[x] += tab[(int64_t)t * ntab + npos + x];
    }
    free(tab);
    free(o); free(dO); free(mean); free(rstd);
    return 0;
}

/* Number of OpenMP threads the oracle runs with (1 without OpenMP). */
int hstu_oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}
