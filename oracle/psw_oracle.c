/*
 * psw_oracle.c -- plain CPU oracle for pipelined CNN training with stale
 * weights (Zhang & Abdelrahman, "Pipelined Training with Stale Weights of
 * Deep Convolutional Neural Networks", ICLR 2020 submission, arXiv 1912.12675).
 *
 * TEST INFRASTRUCTURE ONLY.  This file is the slow, obviously-correct
 * reference that the HIP path is checked against.  Only the test suite, the
 * smoke check and the CPU-baseline leg of the benchmark may load it.  It shares
 * no code, header, table or helper with the GPU library.
 *
 * Precision: every value is stored and accumulated in IEEE double.  Inputs
 * arrive as float32 (the harness draws them in float32) and are widened.
 * The optional "bf16" switch emulates a GPU mode in which the two operands of
 * every convolution / fully-connected product are rounded to bfloat16 (round
 * to nearest even, via float32) before being multiplied; accumulation stays
 * in double.
 *
 * Layout: NCHW activations, KCRS convolution weights, [out][in] FC weights,
 * i.e. the layout in which the operations are usually written down.
 *
 * What is computed (paper section in brackets):
 *   - per-layer forward and backward of conv / BN(+residual)+ReLU / max-pool /
 *     global average pool / fully connected / softmax cross-entropy, and the
 *     SGD-momentum update  [Sec. 2, backpropagation; App. A/B hyperparameters]
 *   - dropout (App. A: VGG-16 trains with dropout), its masks drawn from a
 *     counter-based generator (Philox4x32-10) so that the backward pass of a
 *     mini-batch recomputes the mask its forward pass used
 *   - the stale-weight schedule  [Sec. 3, pipelined backpropagation]:
 *     every stage s keeps its FULL weight history W_s^(0), W_s^(1), ...;
 *     the forward pass of mini-batch t reads W_s^(max(0, t - d_s)), the
 *     backward pass (data gradients) reads the current W_s^(t), the weight
 *     gradients use the activations saved by that forward pass, and the
 *     update produces W_s^(t+1) from W_s^(t).  With every d_s = 0 this is
 *     ordinary mini-batch SGD [Sec. 2].
 *
 * Parity status of each part is recorded in the test suite: layer maths are
 * pinned to torch.nn.functional in float64, brute force and finite
 * differences; the schedule is pinned to an independent register/cycle
 * simulator written from Sec. 3; architectures are pinned by the weight
 * column of the memory-usage table (Table 6).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#ifdef _OPENMP
#include <omp.h>
#endif

/* ------------------------------------------------------------------------ */
/* Philox4x32-10 (Salmon, Moraes, Dror and Shaw, "Parallel random numbers:   */
/* as easy as 1, 2, 3", SC 2011): a 4 x 32-bit counter is transformed by ten */
/* rounds under a 2 x 32-bit key.  A round multiplies counter words 0 and 2  */
/* by the two round constants (full 64-bit products), and forms the new     */
/* counter from the high halves xor-ed with the other two words and the key, */
/* and the low halves; the key grows by the two Weyl constants between      */
/* rounds.                                                                  */
/* ------------------------------------------------------------------------ */
void orc_philox4x32_10(const uint32_t ctr[4], const uint32_t key[2], uint32_t out[4])
{
    uint32_t c0 = ctr[0], c1 = ctr[1], c2 = ctr[2], c3 = ctr[3];
    uint32_t k0 = key[0], k1 = key[1];
    for (int round = 0; round < 10; ++round) {
        if (round > 0) {
            k0 += 0x9E3779B9u;
            k1 += 0xBB67AE85u;
        }
        const uint64_t a = (uint64_t)0xD2511F53u * c0;
        const uint64_t b = (uint64_t)0xCD9E8D57u * c2;
        const uint32_t n0 = (uint32_t)(b >> 32) ^ c1 ^ k0;
        const uint32_t n1 = (uint32_t)b;
        const uint32_t n2 = (uint32_t)(a >> 32) ^ c3 ^ k1;
        const uint32_t n3 = (uint32_t)a;
        c0 = n0;
        c1 = n1;
        c2 = n2;
        c3 = n3;
    }
    out[0] = c0;
    out[1] = c1;
    out[2] = c2;
    out[3] = c3;
}

/* Dropout mask of the tensor written by operation `op` in mini-batch t: an
 * element with flat NCHW index j is kept iff the top 24 bits of word j % 4 of
 * Philox4x32-10(counter (j / 4, op, t mod 2^32, t / 2^32), key (seed mod
 * 2^32, seed / 2^32)) are >= p24, i.e. it is dropped with probability
 * p24 / 2^24.  Kept elements are scaled by 2^24 / (2^24 - p24) (inverted
 * dropout: the expectation of the output is the input). */
static int dropout_keep(int64_t j, int op, int64_t t, uint64_t seed, int p24)
{
    const uint32_t ctr[4] = {(uint32_t)(j / 4), (uint32_t)op, (uint32_t)t, (uint32_t)((uint64_t)t >> 32)};
    const uint32_t key[2] = {(uint32_t)seed, (uint32_t)(seed >> 32)};
    uint32_t r[4];
    orc_philox4x32_10(ctr, key, r);
    return (int)(r[j % 4] >> 8) >= p24;
}

void orc_dropout_fwd(int64_t n, const double *x, double *y, int p24, uint64_t seed, int op, int64_t t)
{
    const double scale = 16777216.0 / (16777216.0 - p24);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j) y[j] = dropout_keep(j, op, t, seed, p24) ? x[j] * scale : 0.0;
}

/* dx += mask * scale * dy (accumulates, as every data gradient here) */
void orc_dropout_bwd(int64_t n, const double *dy, double *dx, int p24, uint64_t seed, int op, int64_t t)
{
    const double scale = 16777216.0 / (16777216.0 - p24);
#pragma omp parallel for schedule(static)
    for (int64_t j = 0; j < n; ++j)
        if (dropout_keep(j, op, t, seed, p24)) dx[j] += dy[j] * scale;
}

/* ------------------------------------------------------------------------ */
/* bf16 operand rounding (emulation of the GPU's bf16-in / fp32-acc mode).   */
/* fp64 -> fp32 (RNE, by the C cast) -> bf16 (RNE on the upper 16 bits).     */
/* ------------------------------------------------------------------------ */
static double to_bf16(double v)
{
    float f = (float)v;
    uint32_t u;
    memcpy(&u, &f, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) { /* inf / nan: truncate */
        u &= 0xffff0000u;
    } else {
        uint32_t lsb = (u >> 16) & 1u;
        u += 0x7fffu + lsb;
        u &= 0xffff0000u;
    }
    memcpy(&f, &u, 4);
    return (double)f;
}

static double *rounded_copy(const double *src, int64_t n, int bf16)
{
    double *dst = (double *)malloc(sizeof(double) * (size_t)(n > 0 ? n : 1));
    for (int64_t i = 0; i < n; ++i) dst[i] = bf16 ? to_bf16(src[i]) : src[i];
    return dst;
}

int orc_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

void orc_set_num_threads(int n)
{
#ifdef _OPENMP
    if (n > 0) omp_set_num_threads(n);
#else
    (void)n;
#endif
}

/* ------------------------------------------------------------------------ */
/* Convolution [Sec. 2: x^(l) from x^(l-1) and W^(l)]                       */
/*   y[n,k,p,q] = b[k] + sum_{c,r,s} w[k,c,r,s] * x[n,c, p*st+r-pad, q*st+s-pad] */
/* (out-of-range input positions contribute zero: zero padding)             */
/* ------------------------------------------------------------------------ */
static int out_dim(int in, int k, int stride, int pad) { return (in + 2 * pad - k) / stride + 1; }

void orc_conv_fwd(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                  const double *x, const double *w, const double *b, double *y, int bf16)
{
    const int P = out_dim(H, R, stride, pad), Q = out_dim(W, S, stride, pad);
    double *xr = rounded_copy(x, (int64_t)N * C * H * W, bf16);
    double *wr = rounded_copy(w, (int64_t)K * C * R * S, bf16);
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int k = 0; k < K; ++k) {
            double *yp = y + ((int64_t)n * K + k) * P * Q;
            for (int i = 0; i < P * Q; ++i) yp[i] = b ? b[k] : 0.0;
            for (int c = 0; c < C; ++c)
                for (int r = 0; r < R; ++r)
                    for (int s = 0; s < S; ++s) {
                        const double wv = wr[(((int64_t)k * C + c) * R + r) * S + s];
                        for (int p = 0; p < P; ++p) {
                            const int ih = p * stride + r - pad;
                            if (ih < 0 || ih >= H) continue;
                            const double *xrow = xr + (((int64_t)n * C + c) * H + ih) * W;
                            for (int q = 0; q < Q; ++q) {
                                const int iw = q * stride + s - pad;
                                if (iw < 0 || iw >= W) continue;
                                yp[p * Q + q] += wv * xrow[iw];
                            }
                        }
                    }
        }
    free(xr);
    free(wr);
}

/* Backward data [Sec. 2: delta^(l-1) from delta^(l) and W]: the adjoint of
 * the forward map,  dx[n,c,ih,iw] += sum over (k,r,s,p,q) with
 * ih = p*st+r-pad, iw = q*st+s-pad of dy[n,k,p,q] * w[k,c,r,s].
 * ACCUMULATES into dx. */
void orc_conv_bwd_data(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                       const double *w, const double *dy, double *dx, int bf16)
{
    const int P = out_dim(H, R, stride, pad), Q = out_dim(W, S, stride, pad);
    double *dyr = rounded_copy(dy, (int64_t)N * K * P * Q, bf16);
    double *wr = rounded_copy(w, (int64_t)K * C * R * S, bf16);
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int c = 0; c < C; ++c) {
            double *dxp = dx + ((int64_t)n * C + c) * H * W;
            for (int k = 0; k < K; ++k)
                for (int r = 0; r < R; ++r)
                    for (int s = 0; s < S; ++s) {
                        const double wv = wr[(((int64_t)k * C + c) * R + r) * S + s];
                        const double *dyp = dyr + ((int64_t)n * K + k) * P * Q;
                        for (int p = 0; p < P; ++p) {
                            const int ih = p * stride + r - pad;
                            if (ih < 0 || ih >= H) continue;
                            for (int q = 0; q < Q; ++q) {
                                const int iw = q * stride + s - pad;
                                if (iw < 0 || iw >= W) continue;
                                dxp[ih * W + iw] += wv * dyp[p * Q + q];
                            }
                        }
                    }
        }
    free(dyr);
    free(wr);
}

/* Backward weight [Sec. 2: dE/dW^(l) from x^(l-1) and delta^(l)]:
 *   dw[k,c,r,s] = sum_{n,p,q} dy[n,k,p,q] * x[n,c,p*st+r-pad,q*st+s-pad]
 *   db[k]       = sum_{n,p,q} dy[n,k,p,q]         (db may be NULL)
 * OVERWRITES dw and db. */
void orc_conv_bwd_weight(int N, int C, int H, int W, int K, int R, int S, int stride, int pad,
                         const double *x, const double *dy, double *dw, double *db, int bf16)
{
    const int P = out_dim(H, R, stride, pad), Q = out_dim(W, S, stride, pad);
    double *xr = rounded_copy(x, (int64_t)N * C * H * W, bf16);
    double *dyr = rounded_copy(dy, (int64_t)N * K * P * Q, bf16);
#pragma omp parallel for collapse(2) schedule(static)
    for (int k = 0; k < K; ++k)
        for (int c = 0; c < C; ++c)
            for (int r = 0; r < R; ++r)
                for (int s = 0; s < S; ++s) {
                    double acc = 0.0;
                    for (int n = 0; n < N; ++n) {
                        const double *dyp = dyr + ((int64_t)n * K + k) * P * Q;
                        const double *xp = xr + ((int64_t)n * C + c) * H * W;
                        for (int p = 0; p < P; ++p) {
                            const int ih = p * stride + r - pad;
                            if (ih < 0 || ih >= H) continue;
                            for (int q = 0; q < Q; ++q) {
                                const int iw = q * stride + s - pad;
                                if (iw < 0 || iw >= W) continue;
                                acc += dyp[p * Q + q] * xp[ih * W + iw];
                            }
                        }
                    }
                    dw[(((int64_t)k * C + c) * R + r) * S + s] = acc;
                }
    if (db) {
        for (int k = 0; k < K; ++k) {
            double acc = 0.0;
            for (int n = 0; n < N; ++n)
                for (int i = 0; i < P * Q; ++i) acc += dy[((int64_t)n * K + k) * P * Q + i];
            db[k] = acc; /* bias gradient uses the unrounded dy: the bias add is not a product */
        }
    }
    free(xr);
    free(dyr);
}

/* ------------------------------------------------------------------------ */
/* Batch normalisation (training mode) + optional residual + optional ReLU. */
/*   mean_c = (1/M) sum y,  var_c = (1/M) sum (y-mean)^2  (biased),          */
/*   xhat = (y-mean)/sqrt(var+eps),  z = gamma*xhat + beta [+ sc(res)],     */
/*   z = max(z, 0) if relu.  M = N*H*W.                                      */
/* sc(res) is the identity (same shape) or the "option A" shortcut of the   */
/* CIFAR ResNets: spatial subsample by Hr/H (even positions) and zero        */
/* channels padded equally on both sides, (C - Cr)/2 each.                  */
/* Running statistics: rm = (1-m) rm + m mean, rv = (1-m) rv + m var*M/(M-1) */
/* ------------------------------------------------------------------------ */
static double shortcut_value(const double *res, int n, int c, int h, int w,
                             int C, int H, int W, int Cr, int Hr, int Wr)
{
    if (Cr == C && Hr == H && Wr == W)
        return res[(((int64_t)n * Cr + c) * Hr + h) * Wr + w];
    const int lo = (C - Cr) / 2;
    const int cc = c - lo;
    if (cc < 0 || cc >= Cr) return 0.0;
    const int sh = Hr / H, sw = Wr / W;
    return res[(((int64_t)n * Cr + cc) * Hr + h * sh) * Wr + w * sw];
}

void orc_bn_fwd(int N, int C, int H, int W, const double *y, const double *gamma,
                const double *beta, const double *res, int Cr, int Hr, int Wr, int relu,
                double eps, double *z, double *save_mean, double *save_invstd,
                double *run_mean, double *run_var, double momentum)
{
    const int64_t HW = (int64_t)H * W, M = (int64_t)N * HW;
#pragma omp parallel for schedule(static)
    for (int c = 0; c < C; ++c) {
        double sum = 0.0;
        for (int n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) sum += y[((int64_t)n * C + c) * HW + i];
        const double mean = sum / (double)M;
        double sq = 0.0;
        for (int n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const double d = y[((int64_t)n * C + c) * HW + i] - mean;
                sq += d * d;
            }
        const double var = sq / (double)M;
        const double invstd = 1.0 / sqrt(var + eps);
        save_mean[c] = mean;
        save_invstd[c] = invstd;
        if (run_mean) run_mean[c] = (1.0 - momentum) * run_mean[c] + momentum * mean;
        if (run_var)
            run_var[c] = (1.0 - momentum) * run_var[c] +
                         momentum * (M > 1 ? var * (double)M / (double)(M - 1) : var);
        for (int n = 0; n < N; ++n)
            for (int h = 0; h < H; ++h)
                for (int w = 0; w < W; ++w) {
                    const int64_t idx = (((int64_t)n * C + c) * H + h) * W + w;
                    double v = gamma[c] * (y[idx] - mean) * invstd + beta[c];
                    if (res) v += shortcut_value(res, n, c, h, w, C, H, W, Cr, Hr, Wr);
                    if (relu && !(v > 0.0)) v = 0.0;
                    z[idx] = v;
                }
    }
}

/* Backward of the above.  g = dz * [z > 0] (if relu) ;
 *   dbeta = sum g ; dgamma = sum g*xhat ;
 *   dy = gamma * invstd * (g - dbeta/M - xhat * dgamma/M)   (OVERWRITES dy)
 *   dres += sc^T(g)   (ACCUMULATES; NULL when there is no residual)
 * gamma is whatever version the caller passes (the schedule passes W^(t)). */
void orc_bn_bwd(int N, int C, int H, int W, const double *dz, const double *z, const double *y,
                const double *gamma, const double *save_mean, const double *save_invstd, int relu,
                double *dy, double *dgamma, double *dbeta, double *dres, int Cr, int Hr, int Wr)
{
    const int64_t HW = (int64_t)H * W, M = (int64_t)N * HW;
#pragma omp parallel for schedule(static)
    for (int c = 0; c < C; ++c) {
        const double mean = save_mean[c], invstd = save_invstd[c];
        double sg = 0.0, sgx = 0.0;
        for (int n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const int64_t idx = ((int64_t)n * C + c) * HW + i;
                const double g = (relu && !(z[idx] > 0.0)) ? 0.0 : dz[idx];
                sg += g;
                sgx += g * (y[idx] - mean) * invstd;
            }
        dbeta[c] = sg;
        dgamma[c] = sgx;
        for (int n = 0; n < N; ++n)
            for (int64_t i = 0; i < HW; ++i) {
                const int64_t idx = ((int64_t)n * C + c) * HW + i;
                const double g = (relu && !(z[idx] > 0.0)) ? 0.0 : dz[idx];
                const double xhat = (y[idx] - mean) * invstd;
                dy[idx] = gamma[c] * invstd * (g - sg / (double)M - xhat * sgx / (double)M);
            }
    }
    if (dres) {
        const int identity = (Cr == C && Hr == H && Wr == W);
        const int lo = (C - Cr) / 2;
        const int sh = identity ? 1 : Hr / H, sw = identity ? 1 : Wr / W;
        /* each residual element receives from at most one output element */
#pragma omp parallel for schedule(static)
        for (int c = 0; c < C; ++c) {
            const int cc = identity ? c : c - lo;
            if (cc < 0 || cc >= Cr) continue;
            for (int n = 0; n < N; ++n)
                for (int h = 0; h < H; ++h)
                    for (int w = 0; w < W; ++w) {
                        const int64_t idx = (((int64_t)n * C + c) * H + h) * W + w;
                        const double g = (relu && !(z[idx] > 0.0)) ? 0.0 : dz[idx];
                        dres[(((int64_t)n * Cr + cc) * Hr + h * sh) * Wr + w * sw] += g;
                    }
        }
    }
}

/* ------------------------------------------------------------------------ */
/* ReLU on a whole tensor and its backward (mask taken from the output).    */
/* ------------------------------------------------------------------------ */
void orc_relu_inplace(int64_t n, double *z)
{
    for (int64_t i = 0; i < n; ++i)
        if (!(z[i] > 0.0)) z[i] = 0.0;
}

/* ------------------------------------------------------------------------ */
/* Max pooling, window k x k, stride st, no padding, floor mode.            */
/* argmax = flat index (ih*W+iw) inside the input plane of the FIRST        */
/* maximum in row-major window order.                                       */
/* ------------------------------------------------------------------------ */
void orc_maxpool_fwd(int N, int C, int H, int W, int k, int st, const double *x, double *y,
                     int32_t *argmax)
{
    const int P = (H - k) / st + 1, Q = (W - k) / st + 1;
    for (int64_t nc = 0; nc < (int64_t)N * C; ++nc)
        for (int p = 0; p < P; ++p)
            for (int q = 0; q < Q; ++q) {
                double best = 0.0;
                int bi = -1;
                for (int r = 0; r < k; ++r)
                    for (int s = 0; s < k; ++s) {
                        const int ih = p * st + r, iw = q * st + s;
                        const double v = x[nc * H * W + ih * W + iw];
                        if (bi < 0 || v > best) {
                            best = v;
                            bi = ih * W + iw;
                        }
                    }
                y[nc * P * Q + p * Q + q] = best;
                argmax[nc * P * Q + p * Q + q] = bi;
            }
}

/* dx[argmax] += dy  (ACCUMULATES) */
void orc_maxpool_bwd(int N, int C, int H, int W, int k, int st, const double *dy,
                     const int32_t *argmax, double *dx)
{
    const int P = (H - k) / st + 1, Q = (W - k) / st + 1;
    for (int64_t nc = 0; nc < (int64_t)N * C; ++nc)
        for (int i = 0; i < P * Q; ++i) dx[nc * H * W + argmax[nc * P * Q + i]] += dy[nc * P * Q + i];
}

/* Global average pool: y[n,c] = (1/HW) sum x[n,c,:,:]; backward broadcasts
 * dy/HW (ACCUMULATES). */
void orc_gavgpool_fwd(int N, int C, int H, int W, const double *x, double *y)
{
    const int64_t HW = (int64_t)H * W;
    for (int64_t nc = 0; nc < (int64_t)N * C; ++nc) {
        double s = 0.0;
        for (int64_t i = 0; i < HW; ++i) s += x[nc * HW + i];
        y[nc] = s / (double)HW;
    }
}

void orc_gavgpool_bwd(int N, int C, int H, int W, const double *dy, double *dx)
{
    const int64_t HW = (int64_t)H * W;
    for (int64_t nc = 0; nc < (int64_t)N * C; ++nc)
        for (int64_t i = 0; i < HW; ++i) dx[nc * HW + i] += dy[nc] / (double)HW;
}

/* ------------------------------------------------------------------------ */
/* Fully connected: y[n,o] = b[o] + sum_i x[n,i] w[o,i]   (w is [out][in])  */
/* ------------------------------------------------------------------------ */
void orc_fc_fwd(int N, int In, int Out, const double *x, const double *w, const double *b,
                double *y, int bf16)
{
    double *xr = rounded_copy(x, (int64_t)N * In, bf16);
    double *wr = rounded_copy(w, (int64_t)Out * In, bf16);
#pragma omp parallel for collapse(2) schedule(static)
    for (int n = 0; n < N; ++n)
        for (int o = 0; o < Out; ++o) {
            double acc = b ? b[o] : 0.0;
            for (int i = 0; i < In; ++i) acc += xr[(int64_t)n * In + i] * wr[(int64_t)o * In + i];
            y[(int64_t)n * Out + o] = acc;
        }
    free(xr);
    free(wr);
}

/* dx[n,i] += sum_o dy[n,o] w[o,i]  (ACCUMULATES; dx may be NULL)
 * dw[o,i]  = sum_n dy[n,o] x[n,i] ;  db[o] = sum_n dy[n,o]   (OVERWRITE) */
void orc_fc_bwd(int N, int In, int Out, const double *x, const double *w, const double *dy,
                double *dx, double *dw, double *db, int bf16)
{
    double *xr = rounded_copy(x, (int64_t)N * In, bf16);
    double *wr = rounded_copy(w, (int64_t)Out * In, bf16);
    double *dyr = rounded_copy(dy, (int64_t)N * Out, bf16);
    if (dx) {
#pragma omp parallel for collapse(2) schedule(static)
        for (int n = 0; n < N; ++n)
            for (int i = 0; i < In; ++i) {
                double acc = 0.0;
                for (int o = 0; o < Out; ++o) acc += dyr[(int64_t)n * Out + o] * wr[(int64_t)o * In + i];
                dx[(int64_t)n * In + i] += acc;
            }
    }
#pragma omp parallel for collapse(2) schedule(static)
    for (int o = 0; o < Out; ++o)
        for (int i = 0; i < In; ++i) {
            double acc = 0.0;
            for (int n = 0; n < N; ++n) acc += dyr[(int64_t)n * Out + o] * xr[(int64_t)n * In + i];
            dw[(int64_t)o * In + i] = acc;
        }
    if (db)
        for (int o = 0; o < Out; ++o) {
            double acc = 0.0;
            for (int n = 0; n < N; ++n) acc += dy[(int64_t)n * Out + o];
            db[o] = acc;
        }
    free(xr);
    free(wr);
    free(dyr);
}

/* ------------------------------------------------------------------------ */
/* Softmax cross-entropy, mean over the mini-batch (the training error e of */
/* Sec. 2).  loss = (1/N) sum_n [ log sum_j exp z[n,j] - z[n,y_n] ]         */
/* dz[n,j] = (softmax(z_n)_j - [j == y_n]) / N.                             */
/* ------------------------------------------------------------------------ */
double orc_softmax_xent(int N, int Cls, const double *z, const int32_t *labels, double *dz)
{
    double total = 0.0;
    for (int n = 0; n < N; ++n) {
        const double *zn = z + (int64_t)n * Cls;
        double mx = zn[0];
        for (int j = 1; j < Cls; ++j)
            if (zn[j] > mx) mx = zn[j];
        double se = 0.0;
        for (int j = 0; j < Cls; ++j) se += exp(zn[j] - mx);
        const double lse = mx + log(se);
        total += lse - zn[labels[n]];
        if (dz)
            for (int j = 0; j < Cls; ++j)
                dz[(int64_t)n * Cls + j] = (exp(zn[j] - lse) - (j == labels[n] ? 1.0 : 0.0)) / (double)N;
    }
    return total / (double)N;
}

/* ------------------------------------------------------------------------ */
/* SGD with momentum (App. A/B: momentum 0.9, optional weight decay and     */
/* Nesterov):  d = g + wd*w ;  v = mom*v + d ;                               */
/*   w_new = w - lr * (nesterov ? d + mom*v : v)                            */
/* w_out may alias w_in.                                                    */
/* ------------------------------------------------------------------------ */
void orc_sgd(int64_t n, const double *w_in, double *w_out, double *v, const double *g, double lr,
             double mom, double wd, int nesterov)
{
    for (int64_t i = 0; i < n; ++i) {
        const double d = g[i] + wd * w_in[i];
        v[i] = mom * v[i] + d;
        const double step = nesterov ? d + mom * v[i] : v[i];
        w_out[i] = w_in[i] - lr * step;
    }
}

/* ======================================================================== */
/* Network description.  A network is a list of operations; tensor 0 is the */
/* mini-batch input and operation i writes tensor i+1.  Each operation is   */
/* nine int32 values:                                                       */
/*   kind, in0, in1, cin, cout, k, stride, pad, flags                       */
/* kind: 1 conv, 2 batch-norm, 3 max-pool, 4 global avg-pool, 5 fc,        */
/*       6 dropout (k: drop probability in units of 2^-24)                  */
/* in1 : residual tensor of a batch-norm (-1: none)                         */
/* flags: bit0 bias (conv, fc), bit1 ReLU (conv, bn, fc)                    */
/* A stage split is given as stage_end[s] = one past the last operation of  */
/* stage s; the parameters of a stage are the concatenation, in operation   */
/* order, of conv (weight, bias), bn (gamma, beta), fc (weight, bias).      */
/* ======================================================================== */
enum { OP_CONV = 1, OP_BN = 2, OP_MAXPOOL = 3, OP_GAVG = 4, OP_FC = 5, OP_DROPOUT = 6 };
enum { F_BIAS = 1, F_RELU = 2 };

typedef struct {
    int kind, in0, in1, cin, cout, k, stride, pad, flags;
} orc_op;

typedef struct {
    int n, c, h, w;
} orc_shape;

typedef struct {
    int n_ops, n_stages;
    orc_op *ops;
    orc_shape *shape;   /* n_ops + 1 tensors */
    int *stage_of;      /* per op */
    int64_t *poff;      /* per op: offset of its parameters inside its stage */
    int64_t *pcount;    /* per op: number of parameters */
    int64_t *stage_np;  /* per stage: number of parameters */
    int *stage_begin, *stage_end;
    int n_bn;           /* number of BN ops */
    int *bn_index;      /* per op: BN ordinal or -1 */
    int64_t *bn_off;    /* per BN ordinal: offset into running-stat arrays */
    int64_t bn_total;
} orc_net;

static void net_free(orc_net *net)
{
    free(net->ops);
    free(net->shape);
    free(net->stage_of);
    free(net->poff);
    free(net->pcount);
    free(net->stage_np);
    free(net->stage_begin);
    free(net->stage_end);
    free(net->bn_index);
    free(net->bn_off);
}

static int64_t shape_numel_(orc_shape s) { return (int64_t)s.n * s.c * s.h * s.w; }

/* returns 0 on success, a negative number naming the first bad op otherwise */
static int net_build(orc_net *net, int n_ops, const int32_t *desc, int N, int C0, int H0, int W0,
                     int n_stages, const int32_t *stage_end)
{
    memset(net, 0, sizeof(*net));
    net->n_ops = n_ops;
    net->n_stages = n_stages;
    net->ops = (orc_op *)calloc((size_t)n_ops, sizeof(orc_op));
    net->shape = (orc_shape *)calloc((size_t)n_ops + 1, sizeof(orc_shape));
    net->stage_of = (int *)calloc((size_t)n_ops, sizeof(int));
    net->poff = (int64_t *)calloc((size_t)n_ops, sizeof(int64_t));
    net->pcount = (int64_t *)calloc((size_t)n_ops, sizeof(int64_t));
    net->stage_np = (int64_t *)calloc((size_t)n_stages, sizeof(int64_t));
    net->stage_begin = (int *)calloc((size_t)n_stages, sizeof(int));
    net->stage_end = (int *)calloc((size_t)n_stages, sizeof(int));
    net->bn_index = (int *)calloc((size_t)n_ops, sizeof(int));
    net->bn_off = (int64_t *)calloc((size_t)n_ops + 1, sizeof(int64_t));
    net->shape[0] = (orc_shape){N, C0, H0, W0};
    int prev = 0;
    for (int s = 0; s < n_stages; ++s) {
        if (stage_end[s] <= prev || stage_end[s] > n_ops) return -1000 - s;
        net->stage_begin[s] = prev;
        net->stage_end[s] = stage_end[s];
        for (int i = prev; i < stage_end[s]; ++i) net->stage_of[i] = s;
        prev = stage_end[s];
    }
    if (prev != n_ops) return -999;
    for (int i = 0; i < n_ops; ++i) {
        const int32_t *d = desc + 9 * i;
        orc_op o = {d[0], d[1], d[2], d[3], d[4], d[5], d[6], d[7], d[8]};
        net->ops[i] = o;
        if (o.in0 < 0 || o.in0 > i) return -(i + 1);
        if (o.in1 > i) return -(i + 1);
        const orc_shape a = net->shape[o.in0];
        orc_shape out = a;
        int64_t np = 0;
        net->bn_index[i] = -1;
        switch (o.kind) {
        case OP_CONV:
            if (a.c != o.cin) return -(i + 1);
            out.c = o.cout;
            out.h = out_dim(a.h, o.k, o.stride, o.pad);
            out.w = out_dim(a.w, o.k, o.stride, o.pad);
            np = (int64_t)o.cout * o.cin * o.k * o.k + ((o.flags & F_BIAS) ? o.cout : 0);
            break;
        case OP_BN:
            if (a.c != o.cin || o.cout != o.cin) return -(i + 1);
            np = 2 * (int64_t)o.cin;
            net->bn_index[i] = net->n_bn;
            net->bn_off[net->n_bn + 1] = net->bn_off[net->n_bn] + o.cin;
            net->n_bn++;
            break;
        case OP_MAXPOOL:
            out.h = (a.h - o.k) / o.stride + 1;
            out.w = (a.w - o.k) / o.stride + 1;
            break;
        case OP_GAVG:
            out.h = out.w = 1;
            break;
        case OP_FC:
            if ((int64_t)a.c * a.h * a.w != o.cin) return -(i + 1);
            out.c = o.cout;
            out.h = out.w = 1;
            np = (int64_t)o.cout * o.cin + ((o.flags & F_BIAS) ? o.cout : 0);
            break;
        case OP_DROPOUT: /* k = drop probability in units of 2^-24 */
            if (a.c != o.cin || o.cout != o.cin || o.k <= 0 || o.k >= (1 << 24)) return -(i + 1);
            if (shape_numel_(a) / 4 > (int64_t)UINT32_MAX) return -(i + 1);
            break;
        default:
            return -(i + 1);
        }
        const int s = net->stage_of[i];
        net->poff[i] = net->stage_np[s];
        net->pcount[i] = np;
        net->stage_np[s] += np;
        net->shape[i + 1] = out;
    }
    net->bn_total = net->bn_off[net->n_bn];
    return 0;
}

static int64_t shape_numel(orc_shape s) { return (int64_t)s.n * s.c * s.h * s.w; }

/* Parameter count of each stage for a description (no computation).
 * Returns 0 or a negative error code (see net_build). */
int orc_param_counts(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
                     const int32_t *stage_end, int64_t *out_counts)
{
    orc_net net;
    int rc = net_build(&net, n_ops, desc, N, C0, H0, W0, n_stages, stage_end);
    if (rc == 0)
        for (int s = 0; s < n_stages; ++s) out_counts[s] = net.stage_np[s];
    net_free(&net);
    return rc;
}

/* Output shape of every tensor (n_ops+1 rows of n,c,h,w). */
int orc_shapes(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
               const int32_t *stage_end, int32_t *out_shapes)
{
    orc_net net;
    int rc = net_build(&net, n_ops, desc, N, C0, H0, W0, n_stages, stage_end);
    if (rc == 0)
        for (int t = 0; t <= n_ops; ++t) {
            out_shapes[4 * t + 0] = net.shape[t].n;
            out_shapes[4 * t + 1] = net.shape[t].c;
            out_shapes[4 * t + 2] = net.shape[t].h;
            out_shapes[4 * t + 3] = net.shape[t].w;
        }
    net_free(&net);
    return rc;
}

/* State of one forward pass that the backward pass needs. */
typedef struct {
    double **act;       /* n_ops+1 tensors */
    double **bn_mean, **bn_invstd; /* per op (BN only) */
    int32_t **argmax;   /* per op (max-pool only) */
} orc_fwd_state;

/* Forward pass of one mini-batch.  wfor[s] points at the parameter vector
 * that stage s uses for this forward pass.  Returns the loss; writes dlogits
 * (gradient of the loss w.r.t. the last tensor) into *dlogits_out. */
static double forward(const orc_net *net, double *const *wfor, const float *x, const int32_t *labels,
                      orc_fwd_state *st, double *run_mean, double *run_var, double bn_eps,
                      double bn_mom, int bf16, double *dlogits, uint64_t seed, int64_t t)
{
    const int n_ops = net->n_ops;
    const int64_t n0 = shape_numel(net->shape[0]);
    st->act[0] = (double *)malloc(sizeof(double) * (size_t)n0);
    for (int64_t i = 0; i < n0; ++i) st->act[0][i] = (double)x[i];
    for (int i = 0; i < n_ops; ++i) {
        const orc_op o = net->ops[i];
        const orc_shape a = net->shape[o.in0], out = net->shape[i + 1];
        const double *p = wfor[net->stage_of[i]] + net->poff[i];
        double *y = (double *)calloc((size_t)shape_numel(out), sizeof(double));
        st->act[i + 1] = y;
        switch (o.kind) {
        case OP_CONV:
            orc_conv_fwd(a.n, a.c, a.h, a.w, o.cout, o.k, o.k, o.stride, o.pad, st->act[o.in0], p,
                         (o.flags & F_BIAS) ? p + (int64_t)o.cout * o.cin * o.k * o.k : NULL, y, bf16);
            if (o.flags & F_RELU) orc_relu_inplace(shape_numel(out), y);
            break;
        case OP_BN: {
            const int b = net->bn_index[i];
            st->bn_mean[i] = (double *)malloc(sizeof(double) * (size_t)a.c);
            st->bn_invstd[i] = (double *)malloc(sizeof(double) * (size_t)a.c);
            const double *res = NULL;
            orc_shape rs = {0, 0, 0, 0};
            if (o.in1 >= 0) {
                res = st->act[o.in1];
                rs = net->shape[o.in1];
            }
            orc_bn_fwd(a.n, a.c, a.h, a.w, st->act[o.in0], p, p + o.cin, res, rs.c, rs.h, rs.w,
                       (o.flags & F_RELU) != 0, bn_eps, y, st->bn_mean[i], st->bn_invstd[i],
                       run_mean ? run_mean + net->bn_off[b] : NULL,
                       run_var ? run_var + net->bn_off[b] : NULL, bn_mom);
            break;
        }
        case OP_MAXPOOL:
            st->argmax[i] = (int32_t *)malloc(sizeof(int32_t) * (size_t)shape_numel(out));
            orc_maxpool_fwd(a.n, a.c, a.h, a.w, o.k, o.stride, st->act[o.in0], y, st->argmax[i]);
            break;
        case OP_GAVG:
            orc_gavgpool_fwd(a.n, a.c, a.h, a.w, st->act[o.in0], y);
            break;
        case OP_FC:
            orc_fc_fwd(a.n, o.cin, o.cout, st->act[o.in0], p,
                       (o.flags & F_BIAS) ? p + (int64_t)o.cout * o.cin : NULL, y, bf16);
            if (o.flags & F_RELU) orc_relu_inplace(shape_numel(out), y);
            break;
        case OP_DROPOUT:
            orc_dropout_fwd(shape_numel(out), st->act[o.in0], y, o.k, seed, i, t);
            break;
        }
    }
    const orc_shape last = net->shape[n_ops];
    return orc_softmax_xent(last.n, last.c * last.h * last.w, st->act[n_ops], labels, dlogits);
}

/* Backward pass.  wcur[s] is the parameter vector used for data gradients
 * (the schedule passes the current version W_s^(t)); weight gradients use
 * the saved forward activations.  grads[s] receives stage s's gradient. */
static void backward(const orc_net *net, double *const *wcur, const orc_fwd_state *st,
                     const double *dlogits, double *const *grads, int bf16, uint64_t seed, int64_t t)
{
    const int n_ops = net->n_ops;
    double **d = (double **)calloc((size_t)n_ops + 1, sizeof(double *));
    for (int t = 1; t <= n_ops; ++t) d[t] = (double *)calloc((size_t)shape_numel(net->shape[t]), sizeof(double));
    memcpy(d[n_ops], dlogits, sizeof(double) * (size_t)shape_numel(net->shape[n_ops]));
    for (int i = n_ops - 1; i >= 0; --i) {
        const orc_op o = net->ops[i];
        const orc_shape a = net->shape[o.in0], out = net->shape[i + 1];
        const double *p = wcur[net->stage_of[i]] + net->poff[i];
        double *g = grads[net->stage_of[i]] + net->poff[i];
        double *dout = d[i + 1];
        double *din = o.in0 > 0 ? d[o.in0] : NULL; /* no gradient for the input batch */
        switch (o.kind) {
        case OP_CONV: {
            if (o.flags & F_RELU) {
                const double *z = st->act[i + 1];
                for (int64_t j = 0; j < shape_numel(out); ++j)
                    if (!(z[j] > 0.0)) dout[j] = 0.0;
            }
            const int64_t nw = (int64_t)o.cout * o.cin * o.k * o.k;
            orc_conv_bwd_weight(a.n, a.c, a.h, a.w, o.cout, o.k, o.k, o.stride, o.pad, st->act[o.in0],
                                dout, g, (o.flags & F_BIAS) ? g + nw : NULL, bf16);
            if (din)
                orc_conv_bwd_data(a.n, a.c, a.h, a.w, o.cout, o.k, o.k, o.stride, o.pad, p, dout, din, bf16);
            break;
        }
        case OP_BN: {
            double *dy = (double *)malloc(sizeof(double) * (size_t)shape_numel(a));
            double *dres = NULL;
            orc_shape rs = {0, 0, 0, 0};
            if (o.in1 >= 0) {
                rs = net->shape[o.in1];
                dres = o.in1 > 0 ? d[o.in1] : NULL;
            }
            orc_bn_bwd(a.n, a.c, a.h, a.w, dout, st->act[i + 1], st->act[o.in0], p, st->bn_mean[i],
                       st->bn_invstd[i], (o.flags & F_RELU) != 0, dy, g, g + o.cin, dres, rs.c, rs.h, rs.w);
            if (din)
                for (int64_t j = 0; j < shape_numel(a); ++j) din[j] += dy[j];
            free(dy);
            break;
        }
        case OP_MAXPOOL:
            if (din) orc_maxpool_bwd(a.n, a.c, a.h, a.w, o.k, o.stride, dout, st->argmax[i], din);
            break;
        case OP_GAVG:
            if (din) orc_gavgpool_bwd(a.n, a.c, a.h, a.w, dout, din);
            break;
        case OP_FC: {
            if (o.flags & F_RELU) {
                const double *z = st->act[i + 1];
                for (int64_t j = 0; j < shape_numel(out); ++j)
                    if (!(z[j] > 0.0)) dout[j] = 0.0;
            }
            const int64_t nw = (int64_t)o.cout * o.cin;
            orc_fc_bwd(a.n, o.cin, o.cout, st->act[o.in0], p, dout, din, g,
                       (o.flags & F_BIAS) ? g + nw : NULL, bf16);
            break;
        }
        case OP_DROPOUT: /* the mask of this mini-batch's forward pass, recomputed */
            if (din) orc_dropout_bwd(shape_numel(out), dout, din, o.k, seed, i, t);
            break;
        }
    }
    for (int t = 1; t <= n_ops; ++t) free(d[t]);
    free(d);
}

static void state_alloc(orc_fwd_state *st, int n_ops)
{
    st->act = (double **)calloc((size_t)n_ops + 1, sizeof(double *));
    st->bn_mean = (double **)calloc((size_t)n_ops, sizeof(double *));
    st->bn_invstd = (double **)calloc((size_t)n_ops, sizeof(double *));
    st->argmax = (int32_t **)calloc((size_t)n_ops, sizeof(int32_t *));
}

static void state_free(orc_fwd_state *st, int n_ops)
{
    for (int t = 0; t <= n_ops; ++t) free(st->act[t]);
    for (int i = 0; i < n_ops; ++i) {
        free(st->bn_mean[i]);
        free(st->bn_invstd[i]);
        free(st->argmax[i]);
    }
    free(st->act);
    free(st->bn_mean);
    free(st->bn_invstd);
    free(st->argmax);
}

/* One forward + backward of one mini-batch with a single parameter set
 * (no update).  params: concatenated stage vectors.  grads_out: same layout.
 * acts_out (optional): receives every tensor, concatenated, in order
 * 0..n_ops.  Returns 0 or a negative error code; *loss receives the loss. */
int orc_loss_and_grad(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
                      const int32_t *stage_end, const double *params, const float *x,
                      const int32_t *labels, double bn_eps, int bf16, double *loss, double *grads_out,
                      double *acts_out, uint64_t dropout_seed, int64_t step)
{
    orc_net net;
    int rc = net_build(&net, n_ops, desc, N, C0, H0, W0, n_stages, stage_end);
    if (rc != 0) {
        net_free(&net);
        return rc;
    }
    double **wv = (double **)calloc((size_t)n_stages, sizeof(double *));
    double **gv = (double **)calloc((size_t)n_stages, sizeof(double *));
    int64_t off = 0;
    for (int s = 0; s < n_stages; ++s) {
        wv[s] = (double *)params + off;
        gv[s] = grads_out + off;
        off += net.stage_np[s];
    }
    orc_fwd_state st;
    state_alloc(&st, n_ops);
    const orc_shape last = net.shape[n_ops];
    double *dlog = (double *)malloc(sizeof(double) * (size_t)shape_numel(last));
    *loss = forward(&net, wv, x, labels, &st, NULL, NULL, bn_eps, 0.1, bf16, dlog, dropout_seed, step);
    backward(&net, wv, &st, dlog, gv, bf16, dropout_seed, step);
    if (acts_out) {
        int64_t o2 = 0;
        for (int t = 0; t <= n_ops; ++t) {
            const int64_t ne = shape_numel(net.shape[t]);
            memcpy(acts_out + o2, st.act[t], sizeof(double) * (size_t)ne);
            o2 += ne;
        }
    }
    free(dlog);
    state_free(&st, n_ops);
    free(wv);
    free(gv);
    net_free(&net);
    return 0;
}

/* ======================================================================== */
/* Training under the stale-weight schedule [Sec. 3, Sec. 4].                */
/*                                                                          */
/* For t = t0 .. t0+T-1, with d_s = staleness[(t-t0)*S + s]:                */
/*   r_s = max(0, t - d_s)                  (version read by the forward)   */
/*   forward with W_s^(r_s) for every stage s, saving activations;           */
/*   loss and its gradient;                                                  */
/*   backward: data gradients with W_s^(t), weight gradients from the saved  */
/*   activations;                                                           */
/*   (stash != 0: data gradients with W_s^(r_s) instead, the weight-stashing */
/*   scheme that the paper contrasts its own with, Sec. 6.7 and Sec. 7)     */
/*   update:  W_s^(t+1) = SGD(W_s^(t), grad_s)  for every stage s.           */
/* Every version produced is kept (no ring): version v of stage s is         */
/* history[s][v].  The hybrid schedule of Sec. 4 is expressed by giving      */
/* d_s = 0 from step n_p on.                                                */
/*                                                                          */
/* The run may start from a checkpoint at step t0 >= 0:                     */
/* depth     : versions given per stage (>= 1)                              */
/* hist0     : stage by stage, `depth` packed parameter vectors holding      */
/*             W_s^(t0-depth+1) .. W_s^(t0) in that order; vectors of        */
/*             versions below 0 are present but ignored                     */
/* mom0      : momentum buffers at t0, concatenated (NULL: zero)            */
/* bn_in     : 0 -> running statistics start at mean 0, var 1; else         */
/*             run_mean / run_var hold the checkpoint's values on entry     */
/* xs        : T mini-batches, float32, NCHW  (step t0+i uses batch i)      */
/* labels    : T x N int32                                                  */
/* staleness : T x S int32 (>= 0)                                           */
/* lr        : T x S learning rates (per step, for the schedules of App. A  */
/*             and B, and per stage, cf. the per-stage rate of Table 7)     */
/* outputs   : hist_out: stage by stage, `out_depth` vectors                */
/*             W_s^(t0+T-out_depth+1) .. W_s^(t0+T) (versions below 0 are   */
/*             left untouched); mom_out (momentum buffers); grad_out (the  */
/*             gradient of the last step, may be NULL); run_mean/run_var    */
/*             (BN running stats, concatenated over BN ops; may be NULL);   */
/*             losses (T); versions (T x S: r_s)                            */
/* Returns 0, or -2000 for a negative staleness, -2001 when a forward pass   */
/* would read a version older than the checkpoint holds, -2002 for bad      */
/* t0 / depth / out_depth.                                                  */
/* ======================================================================== */
int orc_train_from(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
                   const int32_t *stage_end, int64_t t0, int depth, const double *hist0,
                   const double *mom0, int bn_in, int T, const float *xs, const int32_t *labels,
                   const int32_t *staleness, const double *lr, double mom, double wd, int nesterov,
                   double bn_eps, double bn_mom, int bf16, int stash, int out_depth, double *hist_out,
                   double *mom_out, double *grad_out, double *run_mean, double *run_var,
                   double *losses, int32_t *versions, uint64_t dropout_seed)
{
    if (t0 < 0 || depth < 1 || out_depth < 1 || T < 0) return -2002;
    orc_net net;
    int rc = net_build(&net, n_ops, desc, N, C0, H0, W0, n_stages, stage_end);
    if (rc != 0) {
        net_free(&net);
        return rc;
    }
    const int S = n_stages;
    const int64_t oldest = t0 - depth + 1 > 0 ? t0 - depth + 1 : 0; /* oldest version held */
    for (int i = 0; i < T; ++i)
        for (int s = 0; s < S; ++s) {
            const int d = staleness[(int64_t)i * S + s];
            if (d < 0) {
                net_free(&net);
                return -2000;
            }
            const int64_t t = t0 + i;
            if ((t - d > 0 ? t - d : 0) < oldest) {
                net_free(&net);
                return -2001;
            }
        }
    /* history[s][v], v = 0 .. t0+T; only versions >= oldest are allocated */
    const int64_t nv = t0 + T + 1;
    double ***hist = (double ***)calloc((size_t)S, sizeof(double **));
    double **vel = (double **)calloc((size_t)S, sizeof(double *));
    double **grad = (double **)calloc((size_t)S, sizeof(double *));
    int64_t off = 0;
    for (int s = 0; s < S; ++s) {
        const int64_t np = net.stage_np[s];
        hist[s] = (double **)calloc((size_t)nv, sizeof(double *));
        for (int k = 0; k < depth; ++k) {
            const int64_t v = t0 - depth + 1 + k;
            if (v < 0) continue;
            hist[s][v] = (double *)malloc(sizeof(double) * (size_t)(np > 0 ? np : 1));
            memcpy(hist[s][v], hist0 + (int64_t)depth * off + (int64_t)k * np, sizeof(double) * (size_t)np);
        }
        vel[s] = (double *)calloc((size_t)(np > 0 ? np : 1), sizeof(double));
        if (mom0) memcpy(vel[s], mom0 + off, sizeof(double) * (size_t)np);
        grad[s] = (double *)calloc((size_t)(np > 0 ? np : 1), sizeof(double));
        off += np;
    }
    if (!bn_in) {
        if (run_mean)
            for (int64_t i = 0; i < net.bn_total; ++i) run_mean[i] = 0.0;
        if (run_var)
            for (int64_t i = 0; i < net.bn_total; ++i) run_var[i] = 1.0;
    }

    const int64_t in_numel = shape_numel(net.shape[0]);
    const orc_shape last = net.shape[n_ops];
    double *dlog = (double *)malloc(sizeof(double) * (size_t)shape_numel(last));
    double **wfor = (double **)calloc((size_t)S, sizeof(double *));
    double **wcur = (double **)calloc((size_t)S, sizeof(double *));

    for (int i = 0; i < T; ++i) {
        const int64_t t = t0 + i;
        for (int s = 0; s < S; ++s) {
            const int d = staleness[(int64_t)i * S + s];
            const int64_t r = t - d > 0 ? t - d : 0;
            versions[(int64_t)i * S + s] = (int32_t)r;
            wfor[s] = hist[s][r];
            wcur[s] = stash ? hist[s][r] : hist[s][t];
        }
        orc_fwd_state st;
        state_alloc(&st, n_ops);
        losses[i] = forward(&net, wfor, xs + (int64_t)i * in_numel, labels + (int64_t)i * N, &st,
                            run_mean, run_var, bn_eps, bn_mom, bf16, dlog, dropout_seed, t);
        backward(&net, wcur, &st, dlog, grad, bf16, dropout_seed, t);
        state_free(&st, n_ops);
        for (int s = 0; s < S; ++s) {
            const int64_t np = net.stage_np[s];
            hist[s][t + 1] = (double *)malloc(sizeof(double) * (size_t)(np > 0 ? np : 1));
            orc_sgd(np, hist[s][t], hist[s][t + 1], vel[s], grad[s], lr[(int64_t)i * S + s], mom, wd, nesterov);
        }
    }
    off = 0;
    for (int s = 0; s < S; ++s) {
        const int64_t np = net.stage_np[s];
        for (int k = 0; k < out_depth; ++k) {
            const int64_t v = t0 + T - out_depth + 1 + k;
            if (v >= 0 && hist[s][v])
                memcpy(hist_out + (int64_t)out_depth * off + (int64_t)k * np, hist[s][v], sizeof(double) * (size_t)np);
        }
        if (mom_out) memcpy(mom_out + off, vel[s], sizeof(double) * (size_t)np);
        if (grad_out) memcpy(grad_out + off, grad[s], sizeof(double) * (size_t)np);
        off += np;
        for (int64_t v = 0; v < nv; ++v) free(hist[s][v]);
        free(hist[s]);
        free(vel[s]);
        free(grad[s]);
    }
    free(hist);
    free(vel);
    free(grad);
    free(dlog);
    free(wfor);
    free(wcur);
    net_free(&net);
    return 0;
}

/* The run from step 0: W_s^(0) = params0 (concatenated, stage by stage),
 * momentum zero, running statistics mean 0 / var 1; params_out receives
 * W_s^(T).  Arguments otherwise as orc_train_from. */
int orc_train(int n_ops, const int32_t *desc, int N, int C0, int H0, int W0, int n_stages,
              const int32_t *stage_end, const double *params0, int T, const float *xs,
              const int32_t *labels, const int32_t *staleness, const double *lr, double mom,
              double wd, int nesterov, double bn_eps, double bn_mom, int bf16, int stash, double *params_out,
              double *mom_out, double *run_mean, double *run_var, double *losses, int32_t *versions,
              uint64_t dropout_seed)
{
    return orc_train_from(n_ops, desc, N, C0, H0, W0, n_stages, stage_end, 0, 1, params0, NULL, 0, T, xs,
                          labels, staleness, lr, mom, wd, nesterov, bn_eps, bn_mom, bf16, stash, 1, params_out,
                          mom_out, NULL, run_mean, run_var, losses, versions, dropout_seed);
}
