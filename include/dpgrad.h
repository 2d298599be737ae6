/*
 * dpgrad.h -- C ABI of libdpgrad.so: the DP-SGD gradient step on one AMD
 * Instinct MI355X (gfx950), in hand-written HIP kernels.
 *
 * The step (Opacus, arXiv 2109.12298, section 1 and figure 1): compute every
 * sample's gradient, clip each sample's l2 norm (taken over all parameters)
 * to C, add the clipped gradients over the batch, add Gaussian noise of
 * standard deviation sigma*C, and divide by the batch size.  The per-sample
 * gradients come from each layer's stored input activations A and the
 * backprops B at its output ("highway gradients"; appendix "Vectorized
 * Computation"), and the fields the paper's appendix "Tracking Gradients"
 * names map onto these outputs: grad_sample -> the per-sample gradients,
 * summed_grad -> the clipped sum, grad -> the noised average.
 *
 * Conventions shared by every entry point
 *  - Return a dp_status.  Arguments are validated on the host before anything
 *    is enqueued; an invalid call enqueues nothing and returns DP_EINVAL,
 *    DP_EDTYPE or DP_EUNSUPPORTED.  DP_EHIP means a kernel launch failed.
 *    Nothing throws across the ABI.
 *  - No entry point allocates, frees or synchronizes.  Every pointer is a
 *    caller-owned device pointer (unless stated) to a dense row-major array;
 *    all work is enqueued on the caller's `stream` (NULL = default stream),
 *    so results are ready when the caller's own synchronization says so.
 *  - Scratch memory: entry points taking `ws` need a caller-owned device
 *    workspace of at least the size reported by the matching
 *    *_workspace_bytes() query (which is host-only and may be called at any
 *    time); `ws` may be NULL only when that size is 0.  The workspace holds
 *    nothing between calls.
 *  - Input dtype: DP_F32 or DP_BF16 for activations/backprops.  Per-sample
 *    gradients, norms, sums and outputs are always fp32, accumulated in fp32.
 *  - `scale` (s) multiplies every backprop: s = 1 takes B as backprops of the
 *    summed per-sample losses, so each result is the gradient of that
 *    sample's own loss; callers holding backprops of a batch-mean loss pass
 *    s = N.
 *  - Device-side conditions are OR-ed into `*status` (a caller-owned device
 *    int32, zeroed by the caller; may be NULL to ignore them):
 *    DP_FLAG_BAD_INDEX (a token id outside [0, V)), DP_FLAG_NONFINITE (a
 *    per-sample norm that is NaN or infinite), DP_FLAG_CAP (CSR capacity
 *    exceeded), DP_FLAG_WAIT (a bounded wait of one workgroup for another
 *    ran out: an internal error, the outputs are not to be trusted).  The
 *    caller reads the word after its own synchronization.
 *  - Results are deterministic: no floating-point atomics, every reduction
 *    has a fixed order, so the same inputs give the same bits run to run.
 *  - Entry points are stateless and re-entrant; calls on different streams
 *    with disjoint outputs and workspaces may overlap.  One exception:
 *    dp_conv2d_set_path is a process-wide switch of the convolution kernel
 *    (a test and tuning aid, to be set while no call is in flight; every
 *    choice gives the same results to rounding), and
 *    dp_grad_sample_linear_noalloc shares one scratch array per GPU.
 */
#ifndef DPGRAD_H
#define DPGRAD_H

#include <stddef.h>
#include <stdint.h>
#include <hip/hip_runtime_api.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum dp_status {
    DP_OK = 0,
    DP_EINVAL = 1,       /* a null required pointer, a bad size, a too-small workspace */
    DP_EDTYPE = 2,       /* an unknown dp_dtype */
    DP_EUNSUPPORTED = 3, /* a valid request this library does not implement (e.g. groups != 1) */
    DP_ECAP = 4,         /* a host-checkable capacity is too small */
    DP_EHIP = 5          /* a HIP launch failed */
} dp_status;

typedef enum dp_dtype { DP_F32 = 0, DP_BF16 = 1 } dp_dtype;

enum {
    DP_FLAG_BAD_INDEX = 1,
    DP_FLAG_NONFINITE = 2,
    DP_FLAG_CAP = 4,
    DP_FLAG_WAIT = 8
};

/* Human-readable text for a status code (static storage; never NULL). */
const char *dp_status_string(dp_status s);

/* ABI version of this header; bumped on any incompatible change. */
int dp_abi_version(void);

/* ---------------------------------------------------------------------------
 * Per-sample gradients (row a of the step: grad_sample)
 * ------------------------------------------------------------------------- */

/* Linear layer y_t = W x_t + b applied at T positions per sample.  Per the
 * per-sample equation of the appendix "Vectorized Computation" (the einsum
 * "n...i,n...j->nij" of B and A, extra dimensions summed):
 *   gW[n][i][j] = s * sum_t B[n][t][i] * A[n][t][j]
 *   gb[n][i]    = s * sum_t B[n][t][i]
 *   sqnorm[n]   = sum_ij gW[n][i][j]^2 + sum_i gb[n][i]^2   (overwritten)
 * A: [N][T][d_in] of `dt`;  B: [N][T][d_out] of `dt`  (T = 1: [N][d_in], [N][d_out]).
 * gW: fp32 [N][d_out][d_in] (required); gb: fp32 [N][d_out] or NULL (no bias);
 * sqnorm: fp32 [N] or NULL.  N >= 0, T >= 0 (T = 0 gives zeros), d_in, d_out >= 1.
 * T = 1 runs a bandwidth-bound outer product; T > 1 a per-sample MFMA GEMM
 * with K = T. */
size_t dp_grad_sample_linear_workspace_bytes(int64_t N, int64_t T, int64_t d_in,
                                             int64_t d_out, dp_dtype dt);
dp_status dp_grad_sample_linear(const void *A, const void *B, dp_dtype dt, int64_t N,
                                int64_t T, int64_t d_in, int64_t d_out, float scale,
                                float *gW, float *gb, float *sqnorm, int32_t *status,
                                void *ws, size_t ws_bytes, hipStream_t stream);

/* dp_grad_sample_linear for callers that cannot allocate device memory (code
 * under HIP graph capture, tight serving loops, harnesses that forbid
 * allocation): the same arguments and results without `ws`, the scratch
 * being a fixed array inside the library (8 MiB on each GPU it runs on, held
 * until the process ends; dp_grad_sample_linear_noalloc_max_bytes() returns
 * the size).  A call whose dp_grad_sample_linear_workspace_bytes() exceeds it
 * returns DP_ECAP and enqueues nothing.  Allocates and frees nothing.  Every
 * call on one GPU uses that GPU's one array (each call overwrites what it
 * reads; nothing there needs to start at zero), so calls that may overlap on
 * one GPU (different streams, or graphs replayed concurrently) race and must
 * be serialized by the caller; the stream's device picks the array. */
size_t dp_grad_sample_linear_noalloc_max_bytes(void);
dp_status dp_grad_sample_linear_noalloc(const void *A, const void *B, dp_dtype dt, int64_t N,
                                        int64_t T, int64_t d_in, int64_t d_out, float scale,
                                        float *gW, float *gb, float *sqnorm, int32_t *status,
                                        hipStream_t stream);

/* Conv2d (cross-correlation, zero padding) with groups = 1 and dilation = 1.
 * The paper defers this layer's formula to its tutorials; it is the weight
 * gradient of the convolution restricted to one sample:
 *   gW[n][co][ci][u][v] = s * sum_{oh,ow} GY[n][co][oh][ow] * X[n][ci][oh*sh+u-ph][ow*sw+v-pw]
 *   gb[n][co]           = s * sum_{oh,ow} GY[n][co][oh][ow]
 * (input positions inside the padding contribute zero), i.e. the product of
 * GY_n [Cout][Ho*Wo] with the transposed unfold (im2col) of X_n, whose rows are
 * ordered (ci, u, v) like the weight.  The unfold is never materialized.
 * X: [N][Cin][H][W] of `dt`; GY: [N][Cout][Ho][Wo] of `dt`, where Ho and Wo
 * must equal (H + 2ph - kh)/sh + 1 and (W + 2pw - kw)/sw + 1 (else DP_EINVAL).
 * gW fp32 [N][Cout][Cin][kh][kw]; gb fp32 [N][Cout] or NULL; sqnorm fp32 [N]
 * or NULL (overwritten with the layer's squared norm).
 * dh, dw != 1 or groups != 1 return DP_EUNSUPPORTED. */
size_t dp_grad_sample_conv2d_workspace_bytes(int64_t N, int64_t Cin, int64_t H, int64_t W,
                                             int64_t Cout, int64_t kh, int64_t kw, int64_t sh,
                                             int64_t sw, int64_t ph, int64_t pw);
dp_status dp_grad_sample_conv2d(const void *X, const void *GY, dp_dtype dt, int64_t N,
                                int64_t Cin, int64_t H, int64_t W, int64_t Cout,
                                int64_t Ho, int64_t Wo, int64_t kh, int64_t kw, int64_t sh,
                                int64_t sw, int64_t ph, int64_t pw, int64_t dh, int64_t dw,
                                int64_t groups, float scale, float *gW, float *gb,
                                float *sqnorm, int32_t *status, void *ws, size_t ws_bytes,
                                hipStream_t stream);

/* Kernel choice of dp_grad_sample_conv2d, process-wide.  DP_CONV_AUTO (the
 * default): a sample whose padded input planes and backprop fit one
 * workgroup's LDS (48 KB), with Cout <= 256 and a weight gradient of at most
 * 32 blocks of 16 (Cin*kh*kw) x 16 (Cout), runs one workgroup per sample;
 * other shapes with at least 97 weight columns (Cin*kh*kw) run by output
 * row chunks (a workgroup per sample and tile of up to 288 weight columns x
 * 64 channels) when one output row's inputs fit its LDS, else the tiled
 * kernel.  DP_CONV_ROWS: the row-chunked kernel
 * wherever it applies, else the tiled one.  DP_CONV_TILED: always the tiled
 * kernel.  All give the same results to rounding.  Returns the previous choice, or -1 (choice unchanged)
 * for an unknown value.  Not synchronized with calls in flight on other host
 * threads: set it before enqueueing. */
enum { DP_CONV_AUTO = 0, DP_CONV_TILED = 1, DP_CONV_ROWS = 2 };
int dp_conv2d_set_path(int path);

/* Which kernel dp_grad_sample_conv2d would run for this shape under the
 * choice in force (dp_conv2d_set_path), for reports and tests:
 * DP_CONV_KERNEL_SMALL (one workgroup per sample), _ROWS (row chunks),
 * _TILED; -1 for a shape the call would refuse. */
enum { DP_CONV_KERNEL_SMALL = 0, DP_CONV_KERNEL_ROWS = 1, DP_CONV_KERNEL_TILED = 2 };
int32_t dp_conv2d_kernel_choice(int64_t N, int64_t Cin, int64_t H, int64_t W, int64_t Cout, int64_t kh,
                                int64_t kw, int64_t sh, int64_t sw, int64_t ph, int64_t pw);

/* One layer of dp_grad_sample_many: the arguments of dp_grad_sample_linear
 * (kind DP_LAYER_LINEAR: A, B, T, d_in, d_out) or dp_grad_sample_conv2d
 * (kind DP_LAYER_CONV2D: A = X, B = GY, Cin .. pw; groups = dilation = 1),
 * with the same meaning, layouts and outputs (gW, gb or NULL, sqnorm or NULL;
 * all fp32, overwritten).  The caller owns every buffer. */
enum { DP_LAYER_LINEAR = 0, DP_LAYER_CONV2D = 1 };
typedef struct dp_layer_grad {
    int32_t kind;
    const void *A;
    const void *B;
    int64_t T, d_in, d_out;
    int64_t Cin, H, W, Cout, Ho, Wo, kh, kw, sh, sw, ph, pw;
    float scale;
    float *gW;
    float *gb;
    float *sqnorm;
} dp_layer_grad;

/* The per-sample gradients of `count` layers that share N and the dtype, as
 * by one dp_grad_sample_linear / dp_grad_sample_conv2d call per layer (same
 * formulas; results equal to rounding order, and bit for bit for the bf16
 * and fp32 sequence layers), in grouped launches for the layers that qualify
 * (dp_grad_sample_many_grouped), so that the layers' fixed costs (launch,
 * load round trip) and their last, partly idle rounds of workgroups overlap
 * instead of adding up:
 *  - small layers (a Linear layer with T = 1; a Conv2d layer whose sample
 *    fits one workgroup, as for DP_CONV_AUTO, while that choice is in force):
 *    one workgroup per sample and layer, up to 8 layers per launch;
 *  - bf16 Linear layers over a sequence that dp_grad_sample_linear runs on
 *    its staged kernel (T a multiple of 32, d_in and d_out multiples of 8,
 *    16-byte aligned A, B, gW): runs of consecutive samples per 256 x 128
 *    tile, the run length balanced over all of them, up to 16 layers per
 *    launch, plus one launch adding each layer's squared-norm partials;
 *  - fp32 Linear layers over a sequence that dp_grad_sample_linear runs on
 *    its staged kernel (T a multiple of 16, d_in and d_out multiples of 4,
 *    16-byte aligned A, B, gW): up to 16 layers per launch, each workgroup
 *    taking one 64 x 64 tile of one sample, a sample's tiles of all the
 *    layers together (layers that read the same B, as an LSTM's two weight
 *    matrices do, read it while it is cached), plus one launch adding each
 *    layer's squared-norm partials.
 * The other layers run through the single-layer entry points inside this
 * call, one after the other on `stream`, sharing `ws`.  Arguments are
 * checked as the single-layer calls check them; the first invalid layer's
 * status is returned before anything is enqueued.  count in [0, 64].
 * dp_grad_sample_many_grouped: 1 if the layer goes into a grouped launch,
 * else 0. */
int32_t dp_grad_sample_many_grouped(const dp_layer_grad *item, dp_dtype dt, int64_t N);
size_t dp_grad_sample_many_workspace_bytes(const dp_layer_grad *items, int32_t count, dp_dtype dt,
                                           int64_t N);
dp_status dp_grad_sample_many(const dp_layer_grad *items, int32_t count, dp_dtype dt, int64_t N,
                              int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream);

/* Embedding y_t = E[ids[n][t]] over a [V][D] table.  Sample n's gradient is
 * zero except on the rows of the ids it holds; row v is s * sum of B[n][t][:]
 * over the positions t with ids[n][t] = v.  Returned sparse, as CSR over the
 * batch (a dense [N][V][D] gradient is never formed):
 *   row_ptr[n] .. row_ptr[n+1]   the stored rows of sample n
 *   uniq_ids[k]                  the id of stored row k; ascending within a sample
 *   rows[k][:]                   its gradient row (positions added in ascending t; a long
 *                                segment is added in consecutive pieces, each in ascending
 *                                t, the pieces then added in t order: a fixed order)
 *   sqnorm[n]                    sum of the squares of sample n's rows (overwritten)
 * ids: int64 [N][T]; B: [N][T][D] of `dt`; row_ptr int64 [N+1]; uniq_ids int64
 * [cap]; rows fp32 [cap][D]; sqnorm fp32 [N] or NULL.  cap >= N*T always
 * suffices; a smaller cap that the data overflows sets DP_FLAG_CAP, row_ptr
 * still holds the true counts and rows past cap are not written.  An id
 * outside [0, V) sets DP_FLAG_BAD_INDEX and its position is left out.
 * Needs T <= 4096 and N*T < 2^31 (else DP_EUNSUPPORTED) and V < 2^31.
 * For T <= 512 the call is one kernel (after a small clearing launch): a
 * workgroup per sample, each taking its first CSR row from the distinct
 * counts that the earlier samples' workgroups publish (a bounded wait; past
 * the bound DP_FLAG_WAIT is raised and the result is not to be trusted).
 * Workspace: dp_grad_sample_embedding_workspace_bytes(N, T) bytes, contents
 * arbitrary on entry. */
size_t dp_grad_sample_embedding_workspace_bytes(int64_t N, int64_t T);
dp_status dp_grad_sample_embedding(const int64_t *ids, const void *B, dp_dtype dt, int64_t N,
                                   int64_t T, int64_t V, int64_t D, float scale,
                                   int64_t *row_ptr, int64_t *uniq_ids, float *rows,
                                   int64_t cap, float *sqnorm, int32_t *status, void *ws,
                                   size_t ws_bytes, hipStream_t stream);

/* LayerNorm's elementwise affine y = gamma * xhat + beta over D features at T
 * positions (the paper lists normalization layers among those supported):
 *   ggamma[n][k] = s * sum_t B[n][t][k] * xhat[n][t][k]
 *   gbeta[n][k]  = s * sum_t B[n][t][k]
 * xhat, B: [N][T][D] of `dt`; ggamma, gbeta fp32 [N][D]; sqnorm fp32 [N] or NULL. */
size_t dp_grad_sample_layernorm_workspace_bytes(int64_t N, int64_t T, int64_t D);
dp_status dp_grad_sample_layernorm(const void *xhat, const void *B, dp_dtype dt, int64_t N,
                                   int64_t T, int64_t D, float scale, float *ggamma,
                                   float *gbeta, float *sqnorm, int32_t *status, void *ws,
                                   size_t ws_bytes, hipStream_t stream);

/* One layer of dp_grad_sample_layernorm_many: the arguments of
 * dp_grad_sample_layernorm (xhat, B, T, D, scale, ggamma, gbeta, sqnorm or
 * NULL) with the same meaning and layouts.  The caller owns every buffer. */
typedef struct dp_layernorm_layer {
    const void *xhat;
    const void *B;
    int64_t T, D;
    float scale;
    float *ggamma;
    float *gbeta;
    float *sqnorm;
} dp_layernorm_layer;

/* The LayerNorm affine gradients of `count` layers that share N and the
 * dtype, as by one dp_grad_sample_layernorm call per layer (same formulas;
 * equal up to rounding order), in one launch over every layer's (sample,
 * 128-byte feature chunk) pairs, each adding all T positions in a fixed
 * order, and one more adding each sample's chunk partials of the squared
 * norm in chunk order (layers whose D is not a multiple of 16 bytes' worth
 * of elements, or whose xhat or B is not 16-byte aligned, take a launch of
 * their own with element loads; up to 16 layers per launch).  Arguments are
 * checked as dp_grad_sample_layernorm checks them; the first invalid layer's
 * status is returned before anything is enqueued.  count in [0, 64].
 * Workspace: dp_grad_sample_layernorm_many_workspace_bytes(items, count, N,
 * dt) bytes (one float per sample and chunk of each layer with more than one
 * chunk, in item order). */
size_t dp_grad_sample_layernorm_many_workspace_bytes(const dp_layernorm_layer *items, int32_t count,
                                                     int64_t N, dp_dtype dt);
dp_status dp_grad_sample_layernorm_many(const dp_layernorm_layer *items, int32_t count, dp_dtype dt,
                                        int64_t N, int32_t *status, void *ws, size_t ws_bytes,
                                        hipStream_t stream);

/* GroupNorm's and InstanceNorm's per-channel affine y = gamma[c] * xhat +
 * beta[c] over a channel's P spatial positions (normalization layers are
 * among the predefined layer types of section "Design Principles and
 * Features"; these two normalize within each sample, so, unlike BatchNorm,
 * their per-sample gradients exist):
 *   ggamma[n][c] = s * sum_p B[n][c][p] * xhat[n][c][p]
 *   gbeta[n][c]  = s * sum_p B[n][c][p]
 * xhat (the normalized input), B: [N][C][P] of `dt` (P = the product of the
 * spatial sizes, contiguous); ggamma fp32 [N][C]; gbeta fp32 [N][C] or NULL
 * (no bias); sqnorm fp32 [N] or NULL (overwritten with |ggamma_n|^2 +
 * |gbeta_n|^2).  ws: dp_grad_sample_groupnorm_workspace_bytes(N, C, P)
 * bytes (non-zero when C > 16), else DP_EINVAL.  Sums are deterministic. */
size_t dp_grad_sample_groupnorm_workspace_bytes(int64_t N, int64_t C, int64_t P);
dp_status dp_grad_sample_groupnorm(const void *xhat, const void *B, dp_dtype dt, int64_t N, int64_t C,
                                   int64_t P, float scale, float *ggamma, float *gbeta, float *sqnorm,
                                   int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream);

/* Backward through time of an LSTM layer (the paper's DPLSTM: its recurrent
 * modules are the layers whose per-sample gradients cost it most): the
 * gradient of each sample's loss with respect to the gate pre-activations,
 * delta, which the per-sample gradients of W_ih (A = x_t) and W_hh
 * (A = h_{t-1}) and of both biases take as B (dp_grad_sample_linear with
 * T positions).  PyTorch's gate order i, f, g, o; zero initial state.  For t
 * = T-1 down to 0, with dc_T = 0, f_T = 0, c_{-1} = 0:
 *   dh      = dh_out[t] (+ dh_last at T-1) + W_hh^T delta_{t+1}   (no term at T-1)
 *   dc_t    = dh * o * (1 - tanh(c_t)^2) + dc_{t+1} * f_{t+1}
 *   delta_i = dc_t * g * i * (1 - i)        delta_f = dc_t * c_{t-1} * f * (1 - f)
 *   delta_g = dc_t * i * (1 - g^2)          delta_o = dh * tanh(c_t) * o * (1 - o)
 * gates fp32 [N][T][4H]: i, f, g, o after their nonlinearities (as stored by
 * the forward); c fp32 [N][T][H]: cell states; W_hh fp32 [4H][H]; dh_out fp32
 * [N][T][H] or NULL (loss gradient at every hidden state); dh_last fp32 [N][H]
 * or NULL (at the last one); delta fp32 [N][T][4H] (written).  Needs
 * 1 <= H <= 128 (else DP_EINVAL / DP_EUNSUPPORTED); N < 2^31. */
dp_status dp_lstm_backward(const float *gates, const float *c, const float *W_hh, const float *dh_out,
                           const float *dh_last, int64_t N, int64_t T, int64_t H, float *delta,
                           int32_t *status, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Norms and clipping
 * ------------------------------------------------------------------------- */

/* norm[n] = sqrt(sum_l sqnorm[l][n]), layers added in ascending l: the l2
 * norm of sample n's gradient over all parameters (section 1: clip each
 * per-sample gradient's l2 norm).  sqnorm fp32 [n_layers][N]; norm fp32 [N].
 * A NaN or infinite norm sets DP_FLAG_NONFINITE. */
dp_status dp_per_sample_norms(const float *sqnorm, int32_t n_layers, int64_t N, float *norm,
                              int32_t *status, hipStream_t stream);

/* dp_per_sample_norms over a batch of variable size held in N rows (section
 * "Design Principles and Features": with Poisson sampling the batch size
 * changes from step to step).  n_active: one int64 in device memory, read
 * while the launch runs, so a captured graph follows it from replay to
 * replay; rows n >= *n_active are padding and get norm[n] = -1 with no flag.
 * Every clip factor of this library is 0 for a negative norm, so padding rows
 * add nothing to any clipped sum that takes these norms (their per-sample
 * gradients must still be finite: 0 times a non-finite value is NaN).
 * n_active NULL: every row is active, as dp_per_sample_norms. */
dp_status dp_per_sample_norms_active(const float *sqnorm, int32_t n_layers, int64_t N,
                                     const int64_t *n_active, float *norm, int32_t *status,
                                     hipStream_t stream);

/* Ghost norm of a Linear layer: its per-sample squared gradient norm without
 * forming the per-sample gradient.  The related-work section ("Gradient
 * Clipping") describes computing only each sample's gradient norm (exact for
 * fully connected layers, extended to sequential inputs by ghost clipping).
 * With the Gram matrices G_A = A_n A_n^T and G_B = B_n B_n^T (T x T):
 *   sqnorm[n] = s^2 * sum_{t,t'} G_B[t][t'] * (G_A[t][t'] + (bias ? 1 : 0))
 * which equals |gW_n|^2 + |gb_n|^2 of dp_grad_sample_linear on the same
 * inputs (up to rounding).  Worth it when 2 T^2 < d_in * d_out.
 * A: [N][T][d_in] of `dt`; B: [N][T][d_out] of `dt`; sqnorm fp32 [N]
 * (overwritten, required when N > 0).  N >= 0, T >= 0 (T = 0 gives zeros),
 * d_in, d_out >= 1, T < 2^20, T * max(d_in, d_out) < 2^31
 * (DP_EUNSUPPORTED beyond).  Workspace:
 * dp_ghost_norm_linear_workspace_bytes(N, T, d_in, d_out) bytes (one float
 * per sample and 64 x 64 tile pair of the Grams when T > 64, and, when the
 * call has too few of those to fill the GPU, the partial Gram tiles of the
 * feature chunks it then splits each pair into: 32 KB per sample, pair and
 * chunk; zero when N or T is 0).  The same as dp_ghost_norm_linear_many
 * with one layer. */
size_t dp_ghost_norm_linear_workspace_bytes(int64_t N, int64_t T, int64_t d_in, int64_t d_out);
dp_status dp_ghost_norm_linear(const void *A, const void *B, dp_dtype dt, int64_t N, int64_t T,
                               int64_t d_in, int64_t d_out, float scale, int32_t bias,
                               float *sqnorm, int32_t *status, void *ws, size_t ws_bytes,
                               hipStream_t stream);

/* One layer of dp_ghost_norm_linear_many: the arguments of
 * dp_ghost_norm_linear (A, B, T, d_in, d_out, scale, bias, sqnorm) with the
 * same meaning and layouts.  The caller owns every buffer. */
typedef struct dp_ghost_layer {
    const void *A;
    const void *B;
    int64_t T, d_in, d_out;
    float scale;
    int32_t bias;
    float *sqnorm;
} dp_ghost_layer;

/* The ghost norms of `count` Linear layers that share N and the dtype, as by
 * one dp_ghost_norm_linear call per layer (same formula; equal up to
 * rounding order, and bit for bit when both split the layer's features into
 * the same number of chunks), in one launch over all the layers' (sample,
 * tile pair) units, one more adding each layer's pairs when T > 64, and one
 * adding the feature chunks when the units are too few to fill the GPU (up
 * to 16 layers per launch; layers whose d_in or d_out is not a multiple of 16
 * bytes' worth of elements, or whose A or B is not 16-byte aligned, take a
 * launch of their own with element loads).  Arguments are checked as
 * dp_ghost_norm_linear checks them; the first invalid layer's status is
 * returned before anything is enqueued.  count in [0, 64].  Workspace:
 * dp_ghost_norm_linear_many_workspace_bytes(items, count, N) bytes (the
 * layers' pair values and chunk tiles, in item order). */
size_t dp_ghost_norm_linear_many_workspace_bytes(const dp_ghost_layer *items, int32_t count, int64_t N);
dp_status dp_ghost_norm_linear_many(const dp_ghost_layer *items, int32_t count, dp_dtype dt, int64_t N,
                                    int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream);

/* sqnorm[n] = sum_e G[n][e]^2 for an already materialized per-sample gradient
 * G fp32 [N][numel] (overwritten). */
dp_status dp_sqnorm_from_grads(const float *G, int64_t N, int64_t numel, float *sqnorm,
                               int32_t *status, hipStream_t stream);

/* Clip factors c[n] = min(1, C / (norm[n] + 1e-6)), computed in fp32.
 * C = +inf gives 1; a NaN or infinite norm gives NaN (and DP_FLAG_NONFINITE)
 * so a broken sample poisons the sum rather than passing unclipped.  A
 * negative norm (a padding row, see dp_per_sample_norms_active) gives 0; the
 * same rule holds wherever a clipped sum takes norms.
 * C must be > 0 (else DP_EINVAL). */
dp_status dp_clip_factors(const float *norm, int64_t N, float C, float *c, int32_t *status,
                          hipStream_t stream);

/* Clipped sum of a materialized per-sample gradient (summed_grad):
 *   sum[e] = sum_n c_n * G[n][e], n ascending, c_n as in dp_clip_factors.
 * G fp32 [N][numel]; norm fp32 [N]; sum fp32 [numel] (N = 0 writes zeros);
 * c_out fp32 [N] or NULL receives the factors. */
size_t dp_clip_accumulate_workspace_bytes(int64_t N, int64_t numel);
dp_status dp_clip_accumulate(const float *G, const float *norm, float C, int64_t N,
                             int64_t numel, float *sum, float *c_out, int32_t *status,
                             void *ws, size_t ws_bytes, hipStream_t stream);

/* Clipped sum of a Linear layer computed from A and B without reading the
 * per-sample gradients: with c_n as above,
 *   sumW = s * sum_n c_n * B_n^T A_n  (one GEMM with K = N*T: B^T diag(c) A)
 *   sumb = s * sum_n c_n * sum_t B[n][t][:]
 * Same A/B layout as dp_grad_sample_linear; sumW fp32 [d_out][d_in]; sumb fp32
 * [d_out] or NULL.  The K range is split over workgroups and the partial sums
 * are added in a fixed order in a second pass. */
size_t dp_clip_accumulate_linear_workspace_bytes(int64_t N, int64_t T, int64_t d_in,
                                                 int64_t d_out, dp_dtype dt);
dp_status dp_clip_accumulate_linear(const void *A, const void *B, dp_dtype dt, int64_t N,
                                    int64_t T, int64_t d_in, int64_t d_out, float scale,
                                    const float *norm, float C, float *sumW, float *sumb,
                                    int32_t *status, void *ws, size_t ws_bytes,
                                    hipStream_t stream);

/* One Linear layer of dp_clip_accumulate_linear_many: the arguments of
 * dp_clip_accumulate_linear that differ between layers. */
typedef struct dp_linear_clip {
    const void *A;       /* activations [N][T][d_in] */
    const void *B;       /* backprops [N][T][d_out] */
    int64_t T, d_in, d_out;
    float scale;         /* s */
    float *sumW;         /* fp32 [d_out][d_in] clipped sum of the weight gradients */
    float *sumb;         /* fp32 [d_out] clipped sum of the bias gradients, or NULL */
} dp_linear_clip;

/* dp_clip_accumulate_linear for `count` layers that share N, the norms, C
 * and dtype (items: a host array read during the call only), with the same
 * results: sumW = s * sum_n c_n * B_n^T A_n, sumb = s * sum_n c_n * sum_t
 * B_n[t] (section 1: clip each sample's gradient, then add).  bf16 layers
 * with T a multiple of 32, d_in and d_out multiples of 8, and 16-byte aligned
 * A, B, sumW share one launch (at most 16 layers per launch; each workgroup
 * holds a 256 x 128 output tile over the whole N*T sum, with the clip factor
 * applied in fp32 sample by sample, so no partial sums are written); every
 * other layer runs dp_clip_accumulate_linear's kernels, one after another on
 * `stream`, sharing the workspace.  Validation as dp_clip_accumulate_linear;
 * the workspace is the size dp_clip_accumulate_linear_many_workspace_bytes
 * reports for the same items (0 when every layer takes the grouped launch). */
size_t dp_clip_accumulate_linear_many_workspace_bytes(const dp_linear_clip *items, int32_t count,
                                                      dp_dtype dt, int64_t N);
dp_status dp_clip_accumulate_linear_many(const dp_linear_clip *items, int32_t count, dp_dtype dt,
                                         int64_t N, const float *norm, float C, int32_t *status,
                                         void *ws, size_t ws_bytes, hipStream_t stream);

/* Dense clipped sum of CSR embedding gradients (as dp_grad_sample_embedding
 * writes them): sum[v][:] = sum_n c_n * (sample n's row for id v, if any),
 * n ascending; rows no sample touched are written as zeros.
 * row_ptr int64 [N+1]; uniq_ids int64 [cap]; rows fp32 [cap][D] (the arrays
 * and cap given to dp_grad_sample_embedding); sum fp32 [V][D].  Stored rows
 * at index cap or beyond are left out and set DP_FLAG_CAP; stored ids outside
 * [0, V) set DP_FLAG_BAD_INDEX and are left out.  Needs 64 * V < 2^31 and
 * cap < 2^31 (else DP_EUNSUPPORTED).  The workspace (16-byte aligned) holds
 * an inverted index of 64 samples at a time. */
size_t dp_clip_accumulate_embedding_workspace_bytes(int64_t N, int64_t V);
dp_status dp_clip_accumulate_embedding(const int64_t *row_ptr, const int64_t *uniq_ids,
                                       const float *rows, int64_t cap, const float *norm, float C,
                                       int64_t N, int64_t V, int64_t D, float *sum,
                                       int32_t *status, void *ws, size_t ws_bytes,
                                       hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Grouped clipped sums and noise over many parameter tensors
 * ------------------------------------------------------------------------- */

/* One parameter tensor of dp_clip_noise_many. */
typedef struct dp_param {
    const float *grad_sample; /* fp32 [N][numel] per-sample gradients (used with DP_PARAM_REDUCE;
                                 may be NULL when N = 0) */
    float *sum;               /* fp32 [numel] clipped sum (summed_grad): written with
                                 DP_PARAM_REDUCE, read otherwise (fused routes formed it) */
    float *out;               /* fp32 [numel] noised average (grad), or NULL for no output */
    int64_t numel;
    uint32_t param_index;     /* index of the tensor's noise stream (see dp_add_noise) */
    uint32_t flags;           /* DP_PARAM_REDUCE or 0; other bits must be 0 */
    float *accum;             /* fp32 [numel] running clipped sum over the physical batches of
                                 a logical batch (virtual steps), or NULL */
} dp_param;

enum { DP_PARAM_REDUCE = 1 };

/* For every tensor of `params` (a host array of `count` entries, read during
 * the call only): with DP_PARAM_REDUCE, sum = sum_n c_n * grad_sample[n]
 * with c_n = min(1, C / (norm[n] + 1e-6)) as dp_clip_accumulate (n ascending;
 * N = 0 gives zeros); then, if accum is given, accum += sum (virtual steps:
 * the paper's section on Opacus' features decouples the physical batch,
 * bounded by memory, from the logical batch that one noised step covers;
 * the caller zeroes accum before the first physical batch) and the output
 * below is formed from accum instead of sum; then, if out is given (the last
 * physical batch), out = (sum + sigma*C*z) / denom
 * with z the tensor's stream as in dp_add_noise at step
 * step + (*step_dev if step_dev is not NULL, read on the device).  The device
 * step lets one captured graph replay the call at an advancing step (see
 * dp_step_advance).  This is the optimizer part of the step (clip, sum,
 * noise, average) in two launches for all tensors, with the same results as
 * dp_clip_accumulate followed by dp_add_noise.  Workspace from
 * dp_clip_noise_many_workspace_bytes (same params, count and N). */
size_t dp_clip_noise_many_workspace_bytes(const dp_param *params, int32_t count, int64_t N);
dp_status dp_clip_noise_many(const dp_param *params, int32_t count, int64_t N, const float *norm,
                             float C, uint64_t seed, uint64_t step, const uint64_t *step_dev,
                             float sigma, float denom, int32_t *status, void *ws, size_t ws_bytes,
                             hipStream_t stream);

/* dp_per_sample_norms followed by dp_clip_noise_many, in one launch per
 * group of up to 40 tensors: with sqnorm given, norm[n] = sqrt(sum_l
 * sqnorm[l][n]) is computed and written as dp_per_sample_norms does
 * (DP_FLAG_NONFINITE included); with sqnorm NULL, norm is an input.  Then,
 * for every tensor, the clipped sum, noise and division of
 * dp_clip_noise_many.  A workgroup reduces a run of consecutive elements of
 * a tensor over the whole batch: KG contiguous sample ranges, each added in
 * ascending n, then the KG range sums in range order, so the results are
 * deterministic (they match dp_clip_noise_many to rounding, which groups
 * the samples differently).  KG is 4, 8 or 16, the fewest that still give
 * 256 such workgroups for the call's tensors; it depends only on the
 * tensors' sizes and alignment.  No workspace is needed (the size query returns
 * 0; ws may be NULL). */
size_t dp_norms_clip_noise_workspace_bytes(const dp_param *params, int32_t count, int64_t N);
dp_status dp_norms_clip_noise(const float *sqnorm, int32_t n_layers, const dp_param *params,
                              int32_t count, int64_t N, float *norm, float C, uint64_t seed,
                              uint64_t step, const uint64_t *step_dev, float sigma, float denom,
                              int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream);

/* dp_norms_clip_noise with a noise schedule (section "Design Principles and
 * Features", "Noise scheduler and variable batch size": the noise multiplier
 * evolves during training by a predefined schedule, such as exponential,
 * step or a custom function; the table holds any such schedule, evaluated
 * by the caller): the noise multiplier of step t (t = step + *step_dev, the
 * same step the noise stream is keyed by) is
 * sigma_table[min(t, table_len - 1)], read on the device, so a captured graph
 * follows the schedule from replay to replay.  sigma_table: table_len >= 1
 * floats in device memory, owned by the caller and read while the launch
 * runs; each entry must be finite and >= 0 (an entry that is not raises
 * DP_FLAG_NONFINITE in *status and turns that step's noised outputs to NaN).
 * A NULL table, table_len < 1 or an infinite C returns DP_EINVAL.
 * n_active (device int64, may be NULL): the batch of variable size of
 * dp_per_sample_norms_active; rows n >= *n_active (clamped to [0, N]) are
 * left out of every column sum (they are not read), and, with sqnorm given,
 * get norm[n] = -1; the sample ranges are still those of N rows, so a sum
 * matches a call with N = *n_active to rounding.  Everything else is as
 * dp_norms_clip_noise; with a table of one entry s and n_active NULL it
 * gives the same results as dp_norms_clip_noise with sigma = s. */
dp_status dp_norms_clip_noise_sched(const float *sqnorm, int32_t n_layers, const dp_param *params,
                                    int32_t count, int64_t N, float *norm, float C, uint64_t seed,
                                    uint64_t step, const uint64_t *step_dev, const float *sigma_table,
                                    int64_t table_len, const int64_t *n_active, float denom,
                                    int32_t *status, void *ws, size_t ws_bytes, hipStream_t stream);

/* *step_dev += by, on the device (one tiny kernel): advances the step counter
 * a captured graph reads through dp_clip_noise_many. */
dp_status dp_step_advance(uint64_t *step_dev, uint64_t by, hipStream_t stream);

/* ---------------------------------------------------------------------------
 * Noise and averaging (grad)
 * ------------------------------------------------------------------------- */

/* out[e] = (sum[e] + sigma * C * z[e]) / denom for one parameter tensor.
 * z[e] is element e of the tensor's normal stream: Philox4x32-10 (Salmon et
 * al., SC'11) with key (seed_lo, seed_hi) and counter (e/4, param_index,
 * step_lo, step_hi); each 4-word block gives four normals by Box-Muller on
 * word pairs (w0,w1) and (w2,w3) with u1 = (w>>8)+1)/2^24, u2 = (w>>8)/2^24,
 * z = sqrt(-2 ln u1) * (cos, sin)(2 pi u2).  Element e takes normal e mod 4.
 * The noise is a pure function of (seed, step, param_index, e), so a resumed
 * run reproduces it and every data-parallel rank would draw the same values.
 * sigma = 0 adds nothing (also for C = +inf); sigma > 0 with C = +inf, or
 * denom <= 0, or sigma < 0 is DP_EINVAL.  out may equal sum (in place).
 * sum, out: fp32 [numel]. */
dp_status dp_add_noise(const float *sum, float *out, int64_t numel, uint64_t seed, uint64_t step,
                       uint32_t param_index, float sigma, float C, float denom,
                       int32_t *status, hipStream_t stream);

/* The raw stream behind dp_add_noise: z fp32 [numel] (or NULL) receives the
 * normals, raw uint32 [numel] (or NULL) the Philox words. */
dp_status dp_philox_normals(float *z, uint32_t *raw, int64_t numel, uint64_t seed,
                            uint64_t step, uint32_t param_index, hipStream_t stream);

#ifdef __cplusplus
}
#endif

#endif /* DPGRAD_H */
