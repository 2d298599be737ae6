/*
 * dp_oracle.c -- TEST INFRASTRUCTURE, NOT PRODUCT CODE.
 *
 * A plain, slow, double-precision CPU statement of the DP-SGD gradient step
 * that Opacus (Yousefpour et al., arXiv 2109.12298) vectorizes.  Only the test
 * suite, the smoke check and the benchmark's CPU-baseline leg load this file's
 * library; the product path never does.  It shares no code, header, table or
 * constant generator with the HIP library.
 *
 * Every per-sample gradient here is the plain definition: the gradient, with
 * respect to one layer's parameters, of sample n's own loss, which the
 * micro-batch method of the paper's appendix ("Micro-Batching") obtains with a
 * batch of one.  Given the layer's input A_n and the backprop B_n = dl_n/dY_n
 * at its output, the chain rule ("Vectorized Computation", the per-sample
 * equation) gives dl_n/dW_ij = B_n,i * A_n,j, summed over any extra (sequence
 * or spatial) dimension.  The scale s multiplies every backprop: s = 1 reads B
 * as backprops of the summed per-sample losses.
 *
 * All arithmetic is fp64; loops run in the obvious order; OpenMP only splits
 * independent samples (or independent output elements), so each result's
 * summation order is fixed.
 */
#include <math.h>
#include <omp.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* Number of OpenMP threads the parallel loops below use. */
int dpo_num_threads(void) { return omp_get_max_threads(); }

/* Set that number (the single-threaded timing of the oracle uses 1). */
void dpo_set_num_threads(int n) { omp_set_num_threads(n > 0 ? n : 1); }

/* ---------------------------------------------------------------------------
 * Per-sample gradients
 * ------------------------------------------------------------------------- */

/* Linear y_t = W x_t + b over T positions ("Vectorized Computation": the
 * einsum n...i,n...j->nij sums the extra dimensions).
 *   A  [N][T][din], B [N][T][dout]
 *   gW [N][dout][din] = s * sum_t B[n][t][i] * A[n][t][j]
 *   gb [N][dout]      = s * sum_t B[n][t][i]            (gb may be NULL)   */
void dpo_linear(const double *A, const double *B, long N, long T, long din,
                long dout, double s, double *gW, double *gb)
{
#pragma omp parallel for schedule(dynamic)
    for (long n = 0; n < N; n++) {
        const double *An = A + n * T * din;
        const double *Bn = B + n * T * dout;
        for (long i = 0; i < dout; i++) {
            double *row = gW + (n * dout + i) * din;
            for (long j = 0; j < din; j++) {
                double acc = 0.0;
                for (long t = 0; t < T; t++)
                    acc += Bn[t * dout + i] * An[t * din + j];
                row[j] = s * acc;
            }
            if (gb) {
                double acc = 0.0;
                for (long t = 0; t < T; t++)
                    acc += Bn[t * dout + i];
                gb[n * dout + i] = s * acc;
            }
        }
    }
}

/* Conv2d, groups = 1, dilation = 1, zero padding (cross-correlation):
 *   Y[co][oh][ow] = b[co] + sum_{ci,u,v} W[co][ci][u][v] * X[ci][oh*sh+u-ph][ow*sw+v-pw]
 * so dl_n/dW[co][ci][u][v] = sum_{oh,ow} GY[n][co][oh][ow] * X[n][ci][oh*sh+u-ph][ow*sw+v-pw]
 * (terms whose input index falls in the padding are zero) and
 * dl_n/db[co] = sum_{oh,ow} GY[n][co][oh][ow].  Direct loops, no unfold.
 *   X [N][Cin][H][W], GY [N][Cout][Ho][Wo], gW [N][Cout][Cin][kh][kw], gb [N][Cout] */
void dpo_conv2d(const double *X, const double *GY, long N, long Cin, long H,
                long W, long Cout, long Ho, long Wo, long kh, long kw, long sh,
                long sw, long ph, long pw, double s, double *gW, double *gb)
{
#pragma omp parallel for schedule(dynamic)
    for (long n = 0; n < N; n++) {
        const double *Xn = X + n * Cin * H * W;
        const double *Gn = GY + n * Cout * Ho * Wo;
        for (long co = 0; co < Cout; co++) {
            const double *g = Gn + co * Ho * Wo;
            for (long ci = 0; ci < Cin; ci++) {
                const double *x = Xn + ci * H * W;
                for (long u = 0; u < kh; u++) {
                    for (long v = 0; v < kw; v++) {
                        double acc = 0.0;
                        for (long oh = 0; oh < Ho; oh++) {
                            long ih = oh * sh + u - ph;
                            if (ih < 0 || ih >= H) continue;
                            for (long ow = 0; ow < Wo; ow++) {
                                long iw = ow * sw + v - pw;
                                if (iw < 0 || iw >= W) continue;
                                acc += g[oh * Wo + ow] * x[ih * W + iw];
                            }
                        }
                        gW[(((n * Cout + co) * Cin + ci) * kh + u) * kw + v] = s * acc;
                    }
                }
            }
            if (gb) {
                double acc = 0.0;
                for (long p = 0; p < Ho * Wo; p++)
                    acc += g[p];
                gb[n * Cout + co] = s * acc;
            }
        }
    }
}

static int cmp_i64(const void *a, const void *b)
{
    int64_t x = *(const int64_t *)a, y = *(const int64_t *)b;
    return (x > y) - (x < y);
}

/* Embedding y_t = E[ids_t]: dl_n/dE[v] = sum over the positions t of sample n
 * whose id is v of B[n][t][:], and zero for every other row.  The non-zero rows
 * are returned sample by sample in CSR form: for sample n, the distinct ids in
 * ascending order are uniq[row_ptr[n] .. row_ptr[n+1]), each with its summed
 * row (positions added in ascending t).
 * Returns the number of stored rows, -1 if it would exceed cap, -2 if an id is
 * outside [0, V).                                                            */
long dpo_embedding(const int64_t *ids, const double *B, long N, long T, long V,
                   long D, double s, int64_t *row_ptr, int64_t *uniq,
                   double *rows, long cap)
{
    for (long i = 0; i < N * T; i++)
        if (ids[i] < 0 || ids[i] >= V)
            return -2;
    int64_t *tmp = (int64_t *)malloc(sizeof(int64_t) * (T > 0 ? T : 1));
    long nnz = 0;
    row_ptr[0] = 0;
    for (long n = 0; n < N; n++) {
        /* distinct ids of sample n, ascending (library sort, then dedupe) */
        memcpy(tmp, ids + n * T, sizeof(int64_t) * T);
        qsort(tmp, T, sizeof(int64_t), cmp_i64);
        long u = 0;
        for (long t = 0; t < T; t++)
            if (t == 0 || tmp[t] != tmp[t - 1])
                tmp[u++] = tmp[t];
        if (nnz + u > cap) {
            free(tmp);
            return -1;
        }
        for (long k = 0; k < u; k++) {
            int64_t v = tmp[k];
            uniq[nnz + k] = v;
            double *r = rows + (nnz + k) * D;
            for (long d = 0; d < D; d++)
                r[d] = 0.0;
            for (long t = 0; t < T; t++)
                if (ids[n * T + t] == v)
                    for (long d = 0; d < D; d++)
                        r[d] += B[(n * T + t) * D + d];
            for (long d = 0; d < D; d++)
                r[d] *= s;
        }
        nnz += u;
        row_ptr[n + 1] = nnz;
    }
    free(tmp);
    return nnz;
}

/* LayerNorm's affine part y = gamma * xhat + beta (per feature k), over T
 * positions: dl_n/dgamma[k] = sum_t B[n][t][k] * xhat[n][t][k],
 * dl_n/dbeta[k] = sum_t B[n][t][k].                                        */
void dpo_layernorm(const double *xhat, const double *B, long N, long T, long D,
                   double s, double *ggamma, double *gbeta)
{
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; n++) {
        for (long k = 0; k < D; k++) {
            double ag = 0.0, ab = 0.0;
            for (long t = 0; t < T; t++) {
                double b = B[(n * T + t) * D + k];
                ag += b * xhat[(n * T + t) * D + k];
                ab += b;
            }
            ggamma[n * D + k] = s * ag;
            gbeta[n * D + k] = s * ab;
        }
    }
}

/* GroupNorm's / InstanceNorm's per-channel affine y = gamma[c] * xhat + beta[c]
 * over the channel's P spatial positions: dl_n/dgamma[c] = sum_p B[n][c][p] *
 * xhat[n][c][p], dl_n/dbeta[c] = sum_p B[n][c][p].                          */
void dpo_groupnorm(const double *xhat, const double *B, long N, long C, long P,
                   double s, double *ggamma, double *gbeta)
{
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; n++) {
        for (long c = 0; c < C; c++) {
            double ag = 0.0, ab = 0.0;
            for (long p = 0; p < P; p++) {
                double b = B[(n * C + c) * P + p];
                ag += b * xhat[(n * C + c) * P + p];
                ab += b;
            }
            ggamma[n * C + c] = s * ag;
            gbeta[n * C + c] = s * ab;
        }
    }
}

/* ---------------------------------------------------------------------------
 * The LSTM's recurrence (the paper's DPLSTM module: a recurrent layer whose
 * per-sample gradients need its backward through time; its weights act as a
 * Linear layer on the input x_t and one on the previous hidden state h_{t-1},
 * both fed the same gate backprop).  Gate order i, f, g, o, as in PyTorch's
 * LSTM; zero initial state.
 * ------------------------------------------------------------------------- */

static double sigmoid(double z) { return 1.0 / (1.0 + exp(-z)); }

/* Forward over T steps (used by the tests to produce consistent activations):
 *   z_t = W_ih x_t + b_ih + W_hh h_{t-1} + b_hh                 [4H]
 *   i = sig(z_i), f = sig(z_f), g = tanh(z_g), o = sig(z_o)
 *   c_t = f * c_{t-1} + i * g,   h_t = o * tanh(c_t),   h_{-1} = c_{-1} = 0
 * x [N][T][D], W_ih [4H][D], W_hh [4H][H], b_* [4H] (may be NULL);
 * gates [N][T][4H] (i, f, g, o after their nonlinearities), c, h [N][T][H]. */
void dpo_lstm_forward(const double *x, const double *W_ih, const double *W_hh, const double *b_ih,
                      const double *b_hh, long N, long T, long D, long H, double *gates, double *c,
                      double *h)
{
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; n++) {
        for (long t = 0; t < T; t++) {
            double *gt = gates + (n * T + t) * 4 * H;
            for (long r = 0; r < 4 * H; r++) {
                double z = (b_ih ? b_ih[r] : 0.0) + (b_hh ? b_hh[r] : 0.0);
                for (long d = 0; d < D; d++)
                    z += W_ih[r * D + d] * x[(n * T + t) * D + d];
                if (t > 0)
                    for (long k = 0; k < H; k++)
                        z += W_hh[r * H + k] * h[(n * T + t - 1) * H + k];
                gt[r] = (r >= 2 * H && r < 3 * H) ? tanh(z) : sigmoid(z);
            }
            for (long k = 0; k < H; k++) {
                double cp = t > 0 ? c[(n * T + t - 1) * H + k] : 0.0;
                double ct = gt[H + k] * cp + gt[k] * gt[2 * H + k];
                c[(n * T + t) * H + k] = ct;
                h[(n * T + t) * H + k] = gt[3 * H + k] * tanh(ct);
            }
        }
    }
}

/* Backward through time: the gradient of sample n's loss with respect to the
 * gate pre-activations z_t (the backprop B that both weight matrices' per-
 * sample gradients take), from the stored gate activations and cell states
 * and the loss gradient arriving at the hidden states (dh_out[n][t][k], or
 * NULL for none, plus dh_last[n][k] at the last step, or NULL).  For t from
 * T-1 down to 0, with dh_rec = W_hh^T delta_{t+1} (0 at t = T-1), dc_{T} = 0,
 * f_{T} = 0 and c_{-1} = 0, by the chain rule through the equations above:
 *   dh      = dh_out_t (+ dh_last at T-1) + dh_rec
 *   dc_t    = dh * o * (1 - tanh(c_t)^2) + dc_{t+1} * f_{t+1}
 *   delta_i = dc_t * g * i (1 - i)          delta_f = dc_t * c_{t-1} * f (1 - f)
 *   delta_g = dc_t * i * (1 - g^2)          delta_o = dh * tanh(c_t) * o (1 - o)
 * gates [N][T][4H], c [N][T][H], W_hh [4H][H]; delta [N][T][4H].            */
void dpo_lstm_backward(const double *gates, const double *c, const double *W_hh, const double *dh_out,
                       const double *dh_last, long N, long T, long H, double *delta)
{
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; n++) {
        double *dc_next = calloc((size_t)H, sizeof(double));
        double *f_next = calloc((size_t)H, sizeof(double));
        for (long t = T - 1; t >= 0; t--) {
            const double *gt = gates + (n * T + t) * 4 * H;
            double *dt = delta + (n * T + t) * 4 * H;
            for (long k = 0; k < H; k++) {
                double dh = dh_out ? dh_out[(n * T + t) * H + k] : 0.0;
                if (t == T - 1 && dh_last)
                    dh += dh_last[n * H + k];
                if (t < T - 1) {
                    const double *dn = delta + (n * T + t + 1) * 4 * H;
                    for (long r = 0; r < 4 * H; r++)
                        dh += W_hh[r * H + k] * dn[r];
                }
                double i = gt[k], f = gt[H + k], g = gt[2 * H + k], o = gt[3 * H + k];
                double ct = c[(n * T + t) * H + k];
                double cp = t > 0 ? c[(n * T + t - 1) * H + k] : 0.0;
                double tc = tanh(ct);
                double dc = dh * o * (1.0 - tc * tc) + dc_next[k] * f_next[k];
                dt[k] = dc * g * i * (1.0 - i);
                dt[H + k] = dc * cp * f * (1.0 - f);
                dt[2 * H + k] = dc * i * (1.0 - g * g);
                dt[3 * H + k] = dh * tc * o * (1.0 - o);
                dc_next[k] = dc;
                f_next[k] = f;
            }
        }
        free(dc_next);
        free(f_next);
    }
}

/* ---------------------------------------------------------------------------
 * Norms, clipping, clipped sum (the DP-SGD step of section 1, figure 1)
 * ------------------------------------------------------------------------- */

/* sq[n] += sum_e G[n][e]^2 : one parameter tensor's share of sample n's
 * squared l2 norm over all parameters.                                      */
void dpo_sqnorm_accumulate(const double *G, long N, long numel, double *sq)
{
#pragma omp parallel for schedule(static)
    for (long n = 0; n < N; n++) {
        double acc = 0.0;
        for (long e = 0; e < numel; e++)
            acc += G[n * numel + e] * G[n * numel + e];
        sq[n] += acc;
    }
}

/* norm[n] = sqrt(sq[n]). */
void dpo_norms(const double *sq, long N, double *norm)
{
    for (long n = 0; n < N; n++)
        norm[n] = sqrt(sq[n]);
}

/* Clip factor c_n = min(1, C / (norm_n + 1e-6)).
 * C = +inf gives c = 1 (no clipping); a non-finite norm gives c = NaN so the
 * sample poisons the sum instead of passing unclipped.  A negative norm is
 * not a norm: it marks a row of a variable-size batch that holds no sample
 * (the batch size changes from step to step under Poisson sampling), and its
 * factor is 0, so the row adds nothing to the clipped sum.                 */
void dpo_clip_factors(const double *norm, long N, double C, double *c)
{
    for (long n = 0; n < N; n++) {
        double x = norm[n];
        if (isnan(x) || isinf(x)) {
            c[n] = NAN;
        } else if (x < 0.0) {
            c[n] = 0.0;
        } else if (isinf(C)) {
            c[n] = 1.0;
        } else {
            double q = C / (x + 1e-6);
            c[n] = q < 1.0 ? q : 1.0;
        }
    }
}

/* S[e] = sum_n c_n * G[n][e], n ascending ("summed_grad": clipped and summed
 * over the batch, no noise; appendix "Tracking Gradients").                */
void dpo_clip_sum(const double *G, const double *c, long N, long numel, double *S)
{
#pragma omp parallel for schedule(static)
    for (long e = 0; e < numel; e++) {
        double acc = 0.0;
        for (long n = 0; n < N; n++)
            acc += c[n] * G[n * numel + e];
        S[e] = acc;
    }
}

/* Dense clipped sum of a CSR embedding gradient: S[V][D] = sum_n c_n * g_n,
 * where g_n is zero outside the rows sample n touched.  n ascending.        */
void dpo_clip_sum_embedding(const int64_t *row_ptr, const int64_t *uniq,
                            const double *rows, const double *c, long N, long V,
                            long D, double *S)
{
    for (long e = 0; e < V * D; e++)
        S[e] = 0.0;
    for (long n = 0; n < N; n++)
        for (int64_t k = row_ptr[n]; k < row_ptr[n + 1]; k++) {
            int64_t v = uniq[k];
            for (long d = 0; d < D; d++)
                S[v * D + d] += c[n] * rows[k * D + d];
        }
}

/* ---------------------------------------------------------------------------
 * Gaussian noise: Philox4x32-10 (Salmon, Moraes, Dror, Shaw, "Parallel Random
 * Numbers: As Easy as 1, 2, 3", SC'11) followed by the Box-Muller transform.
 * ------------------------------------------------------------------------- */

/* One Philox4x32 bijection, 10 rounds.  A round multiplies words 0 and 2 by
 * the two round multipliers, keeping both halves of each 64-bit product; the
 * new words are (hi(x2*M1) ^ x1 ^ k0, lo(x2*M1), hi(x0*M0) ^ x3 ^ k1,
 * lo(x0*M0)).  Between rounds the key is advanced by the two Weyl constants.
 * The four constants are the ones the SC'11 paper gives for Philox4x32.    */
void dpo_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    const uint32_t M0 = 0xD2511F53u, M1 = 0xCD9E8D57u;
    const uint32_t W0 = 0x9E3779B9u, W1 = 0xBB67AE85u;
    uint32_t x0 = ctr[0], x1 = ctr[1], x2 = ctr[2], x3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int r = 0; r < 10; r++) {
        if (r > 0) {
            k0 += W0;
            k1 += W1;
        }
        uint64_t p0 = (uint64_t)M0 * (uint64_t)x0;
        uint64_t p1 = (uint64_t)M1 * (uint64_t)x2;
        uint32_t hi0 = (uint32_t)(p0 >> 32), lo0 = (uint32_t)p0;
        uint32_t hi1 = (uint32_t)(p1 >> 32), lo1 = (uint32_t)p1;
        x0 = hi1 ^ x1 ^ k0;
        x1 = lo1;
        x2 = hi0 ^ x3 ^ k1;
        x3 = lo0;
    }
    out[0] = x0;
    out[1] = x1;
    out[2] = x2;
    out[3] = x3;
}

/* The noise stream of one parameter tensor.  Element e takes word e mod 4 of
 * the Philox block with key (seed_lo, seed_hi) and counter
 * (e div 4, param_index, step_lo, step_hi).  Words (w0, w1) and (w2, w3) are
 * turned into two normals each by Box-Muller:
 *   u1 = (floor(wa / 256) + 1) / 2^24  in (0, 1]
 *   u2 =  floor(wb / 256)      / 2^24  in [0, 1)
 *   za = sqrt(-2 ln u1) cos(2 pi u2),  zb = sqrt(-2 ln u1) sin(2 pi u2).
 * raw (numel words) and z (numel normals) may each be NULL.                */
void dpo_philox_normals(long numel, uint64_t seed, uint64_t step,
                        uint32_t param_index, uint32_t *raw, double *z)
{
    const double two_pi = 6.283185307179586476925286766559;
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    long nblk = (numel + 3) / 4;
#pragma omp parallel for schedule(static)
    for (long q = 0; q < nblk; q++) {
        uint32_t ctr[4] = {(uint32_t)q, param_index, (uint32_t)step, (uint32_t)(step >> 32)};
        uint32_t w[4];
        double zz[4];
        dpo_philox4x32_10(ctr, key, w);
        for (int p = 0; p < 2; p++) {
            double u1 = ((double)(w[2 * p] >> 8) + 1.0) / 16777216.0;
            double u2 = (double)(w[2 * p + 1] >> 8) / 16777216.0;
            double r = sqrt(-2.0 * log(u1));
            zz[2 * p] = r * cos(two_pi * u2);
            zz[2 * p + 1] = r * sin(two_pi * u2);
        }
        for (int k = 0; k < 4; k++) {
            long e = 4 * q + k;
            if (e >= numel) break;
            if (raw) raw[e] = w[k];
            if (z) z[e] = zz[k];
        }
    }
}

/* Final gradient of one parameter tensor: out = (S + sigma * C * z) / denom
 * (clipped, noised and averaged; "grad" in appendix "Tracking Gradients").
 * sigma = 0 adds nothing (also when C is infinite).                        */
void dpo_add_noise(const double *S, long numel, uint64_t seed, uint64_t step,
                   uint32_t param_index, double sigma, double C, double denom,
                   double *out)
{
    if (sigma == 0.0) {
        for (long e = 0; e < numel; e++)
            out[e] = S[e] / denom;
        return;
    }
    double *z = (double *)malloc(sizeof(double) * (numel > 0 ? numel : 1));
    dpo_philox_normals(numel, seed, step, param_index, NULL, z);
    for (long e = 0; e < numel; e++)
        out[e] = (S[e] + sigma * C * z[e]) / denom;
    free(z);
}
