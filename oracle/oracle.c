/*
 * CPU oracle for the stage math of one HetPipe pipeline stage.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the library under paper_2005_14038_amd/
 * may include, link or call this file; only tests/, the smoke check and the
 * benchmark's CPU-baseline leg use it.
 *
 * Every routine is the textbook definition of the operator written out as
 * plain loops over the output elements, accumulating in double precision.
 * There is no blocking, tiling or reordering: each output element is computed
 * on its own by the formula, and the "_at" entry points evaluate the same
 * formula at a caller-chosen list of output elements (used to check sampled
 * outputs of full-size problems).  OpenMP only distributes independent output
 * elements over threads.
 *
 * The paper (HetPipe, Sec. 2 "Background", training of a DNN layer by layer;
 * Sec. 5 on the ImageNet CNNs VGG-19 and ResNet-152 it trains) relies on these
 * operators without restating them; the definitions are the standard ones:
 *
 *   tensors are NHWC, convolution weights are [K][R][S][C], FC weights are
 *   [out][in];
 *   conv:  y[n,p,q,k] = b[k] + sum_{r,s,c} x[n, p*st-pad+r, q*st-pad+s, c] w[k,r,s,c]
 *          (cross-correlation, zero padding, P = (H + 2 pad - R)/st + 1);
 *   dgrad: dx[n,h,w,c] = sum over (p,q,k,r,s) with p*st-pad+r = h and
 *          q*st-pad+s = w of dy[n,p,q,k] w[k,r,s,c];
 *   wgrad: dw[k,r,s,c] = sum_{n,p,q} dy[n,p,q,k] x[n, p*st-pad+r, q*st-pad+s, c],
 *          db[k] = sum_{n,p,q} dy[n,p,q,k];
 *   FC:    y = x W^T + b, dx = dy W, dW = dy^T x, db = column sums of dy;
 *   max-pool: maximum over the in-range window taps; the backward routes
 *          dy to the first maximum in row-major window order;
 *   batch-norm (training mode): biased per-channel batch statistics over
 *          (n, h, w), x_hat = (x - mu) / sqrt(var + eps), y = gamma x_hat + beta;
 *   softmax cross-entropy: mean over the batch of logsumexp(z) - z[label],
 *          gradient (softmax(z) - onehot) / B.
 */
#include <math.h>
#include <stdint.h>
#include <stddef.h>

/* ------------------------------------------------------------------ conv */

static double conv_fwd_elem(const double *x, int H, int W, int C,
                            const double *w, const double *b, int R, int S,
                            int st, int pad, int n, int p, int q, int k)
{
    double acc = b ? b[k] : 0.0;
    for (int r = 0; r < R; ++r) {
        int h = p * st - pad + r;
        if (h < 0 || h >= H) continue;
        for (int s = 0; s < S; ++s) {
            int ww = q * st - pad + s;
            if (ww < 0 || ww >= W) continue;
            const double *xp = x + (((size_t)n * H + h) * W + ww) * C;
            const double *wp = w + (((size_t)k * R + r) * S + s) * C;
            for (int c = 0; c < C; ++c) acc += xp[c] * wp[c];
        }
    }
    return acc;
}

/* y has shape [N][P][Q][K] */
void oc_conv_fwd(const double *x, int N, int H, int W, int C,
                 const double *w, const double *b, int K, int R, int S,
                 int st, int pad, int P, int Q, double *y)
{
    long total = (long)N * P * Q * K;
#pragma omp parallel for schedule(static)
    for (long i = 0; i < total; ++i) {
        int k = (int)(i % K);
        long t = i / K;
        int q = (int)(t % Q); t /= Q;
        int p = (int)(t % P);
        int n = (int)(t / P);
        y[i] = conv_fwd_elem(x, H, W, C, w, b, R, S, st, pad, n, p, q, k);
    }
}

void oc_conv_fwd_at(const double *x, int N, int H, int W, int C,
                    const double *w, const double *b, int K, int R, int S,
                    int st, int pad, int P, int Q,
                    const int64_t *idx, long nidx, double *out)
{
    (void)N;
#pragma omp parallel for schedule(dynamic, 16)
    for (long j = 0; j < nidx; ++j) {
        long i = idx[j];
        int k = (int)(i % K);
        long t = i / K;
        int q = (int)(t % Q); t /= Q;
        int p = (int)(t % P);
        int n = (int)(t / P);
        out[j] = conv_fwd_elem(x, H, W, C, w, b, R, S, st, pad, n, p, q, k);
    }
}

static double conv_dgrad_elem(const double *dy, int P, int Q, int K,
                              const double *w, int R, int S, int C,
                              int st, int pad, int n, int h, int ww, int c)
{
    double acc = 0.0;
    for (int r = 0; r < R; ++r) {
        int tp = h + pad - r;               /* = p * st */
        if (tp < 0 || tp % st) continue;
        int p = tp / st;
        if (p >= P) continue;
        for (int s = 0; s < S; ++s) {
            int tq = ww + pad - s;
            if (tq < 0 || tq % st) continue;
            int q = tq / st;
            if (q >= Q) continue;
            const double *dyp = dy + (((size_t)n * P + p) * Q + q) * K;
            for (int k = 0; k < K; ++k)
                acc += dyp[k] * w[(((size_t)k * R + r) * S + s) * C + c];
        }
    }
    return acc;
}

/* dx has shape [N][H][W][C] */
void oc_conv_dgrad(const double *dy, int N, int P, int Q, int K,
                   const double *w, int R, int S, int C, int st, int pad,
                   int H, int W, double *dx)
{
    long total = (long)N * H * W * C;
#pragma omp parallel for schedule(static)
    for (long i = 0; i < total; ++i) {
        int c = (int)(i % C);
        long t = i / C;
        int ww = (int)(t % W); t /= W;
        int h = (int)(t % H);
        int n = (int)(t / H);
        dx[i] = conv_dgrad_elem(dy, P, Q, K, w, R, S, C, st, pad, n, h, ww, c);
    }
}

void oc_conv_dgrad_at(const double *dy, int N, int P, int Q, int K,
                      const double *w, int R, int S, int C, int st, int pad,
                      int H, int W, const int64_t *idx, long nidx, double *out)
{
    (void)N;
#pragma omp parallel for schedule(dynamic, 16)
    for (long j = 0; j < nidx; ++j) {
        long i = idx[j];
        int c = (int)(i % C);
        long t = i / C;
        int ww = (int)(t % W); t /= W;
        int h = (int)(t % H);
        int n = (int)(t / H);
        out[j] = conv_dgrad_elem(dy, P, Q, K, w, R, S, C, st, pad, n, h, ww, c);
    }
}

static double conv_wgrad_elem(const double *x, int N, int H, int W, int C,
                              const double *dy, int P, int Q, int K,
                              int st, int pad, int k, int r, int s, int c)
{
    double acc = 0.0;
    for (int n = 0; n < N; ++n)
        for (int p = 0; p < P; ++p) {
            int h = p * st - pad + r;
            if (h < 0 || h >= H) continue;
            for (int q = 0; q < Q; ++q) {
                int ww = q * st - pad + s;
                if (ww < 0 || ww >= W) continue;
                acc += dy[(((size_t)n * P + p) * Q + q) * K + k] *
                       x[(((size_t)n * H + h) * W + ww) * C + c];
            }
        }
    return acc;
}

/* dw has shape [K][R][S][C]; db (optional) has shape [K] */
void oc_conv_wgrad(const double *x, int N, int H, int W, int C,
                   const double *dy, int P, int Q, int K, int R, int S,
                   int st, int pad, double *dw, double *db)
{
    long total = (long)K * R * S * C;
#pragma omp parallel for schedule(static)
    for (long i = 0; i < total; ++i) {
        int c = (int)(i % C);
        long t = i / C;
        int s = (int)(t % S); t /= S;
        int r = (int)(t % R);
        int k = (int)(t / R);
        dw[i] = conv_wgrad_elem(x, N, H, W, C, dy, P, Q, K, st, pad, k, r, s, c);
    }
    if (db) {
#pragma omp parallel for schedule(static)
        for (int k = 0; k < K; ++k) {
            double acc = 0.0;
            for (long m = 0; m < (long)N * P * Q; ++m) acc += dy[m * K + k];
            db[k] = acc;
        }
    }
}

void oc_conv_wgrad_at(const double *x, int N, int H, int W, int C,
                      const double *dy, int P, int Q, int K, int R, int S,
                      int st, int pad, const int64_t *idx, long nidx, double *out)
{
#pragma omp parallel for schedule(dynamic, 1)
    for (long j = 0; j < nidx; ++j) {
        long i = idx[j];
        int c = (int)(i % C);
        long t = i / C;
        int s = (int)(t % S); t /= S;
        int r = (int)(t % R);
        int k = (int)(t / R);
        out[j] = conv_wgrad_elem(x, N, H, W, C, dy, P, Q, K, st, pad, k, r, s, c);
    }
}

/* -------------------------------------------------------------------- FC */

/* x [B][IN], w [OUT][IN], b [OUT] (optional), y [B][OUT] */
void oc_fc_fwd(const double *x, int B, int IN, const double *w, const double *b,
               int OUT, double *y)
{
#pragma omp parallel for schedule(static)
    for (long i = 0; i < (long)B * OUT; ++i) {
        int o = (int)(i % OUT), n = (int)(i / OUT);
        double acc = b ? b[o] : 0.0;
        for (int j = 0; j < IN; ++j) acc += x[(size_t)n * IN + j] * w[(size_t)o * IN + j];
        y[i] = acc;
    }
}

/* dx [B][IN] = dy [B][OUT] . w [OUT][IN] */
void oc_fc_dgrad(const double *dy, int B, int OUT, const double *w, int IN, double *dx)
{
#pragma omp parallel for schedule(static)
    for (long i = 0; i < (long)B * IN; ++i) {
        int j = (int)(i % IN), n = (int)(i / IN);
        double acc = 0.0;
        for (int o = 0; o < OUT; ++o) acc += dy[(size_t)n * OUT + o] * w[(size_t)o * IN + j];
        dx[i] = acc;
    }
}

/* dw [OUT][IN] = dy^T x ; db [OUT] = sum_n dy */
void oc_fc_wgrad(const double *x, int B, int IN, const double *dy, int OUT,
                 double *dw, double *db)
{
#pragma omp parallel for schedule(static)
    for (long i = 0; i < (long)OUT * IN; ++i) {
        int j = (int)(i % IN), o = (int)(i / IN);
        double acc = 0.0;
        for (int n = 0; n < B; ++n) acc += dy[(size_t)n * OUT + o] * x[(size_t)n * IN + j];
        dw[i] = acc;
    }
    if (db) {
        for (int o = 0; o < OUT; ++o) {
            double acc = 0.0;
            for (int n = 0; n < B; ++n) acc += dy[(size_t)n * OUT + o];
            db[o] = acc;
        }
    }
}

/* -------------------------------------------------------------- max-pool */

/* Position (row-major tap index r*S+s) of the first maximum of one window, or
 * -1 when the window has no in-range tap. */
static int pool_first_argmax(const double *x, int H, int W, int C, int R, int S,
                             int st, int pad, int n, int p, int q, int c,
                             double *maxval)
{
    int best = -1;
    double m = -INFINITY;
    for (int r = 0; r < R; ++r) {
        int h = p * st - pad + r;
        if (h < 0 || h >= H) continue;
        for (int s = 0; s < S; ++s) {
            int ww = q * st - pad + s;
            if (ww < 0 || ww >= W) continue;
            double v = x[(((size_t)n * H + h) * W + ww) * C + c];
            if (best < 0 || v > m) { m = v; best = r * S + s; }
        }
    }
    if (maxval) *maxval = m;
    return best;
}

void oc_maxpool_fwd(const double *x, int N, int H, int W, int C, int R, int S,
                    int st, int pad, int P, int Q, double *y)
{
#pragma omp parallel for schedule(static)
    for (long i = 0; i < (long)N * P * Q * C; ++i) {
        int c = (int)(i % C);
        long t = i / C;
        int q = (int)(t % Q); t /= Q;
        int p = (int)(t % P);
        int n = (int)(t / P);
        double m;
        pool_first_argmax(x, H, W, C, R, S, st, pad, n, p, q, c, &m);
        y[i] = m;
    }
}

/* dx[n,h,w,c] = sum of dy over the windows whose first maximum sits at (h,w) */
void oc_maxpool_bwd(const double *x, int N, int H, int W, int C, int R, int S,
                    int st, int pad, int P, int Q, const double *dy, double *dx)
{
#pragma omp parallel for schedule(static)
    for (long i = 0; i < (long)N * H * W * C; ++i) {
        int c = (int)(i % C);
        long t = i / C;
        int ww = (int)(t % W); t /= W;
        int h = (int)(t % H);
        int n = (int)(t / H);
        double acc = 0.0;
        for (int r = 0; r < R; ++r) {
            int tp = h + pad - r;
            if (tp < 0 || tp % st) continue;
            int p = tp / st;
            if (p >= P) continue;
            for (int s = 0; s < S; ++s) {
                int tq = ww + pad - s;
                if (tq < 0 || tq % st) continue;
                int q = tq / st;
                if (q >= Q) continue;
                if (pool_first_argmax(x, H, W, C, R, S, st, pad, n, p, q, c, NULL) == r * S + s)
                    acc += dy[(((size_t)n * P + p) * Q + q) * C + c];
            }
        }
        dx[i] = acc;
    }
}

/* ------------------------------------------------------------ batch-norm */

/* x, y: [M][C] with M = N*H*W.  Writes per-channel mean and 1/sqrt(var+eps). */
void oc_bn_fwd(const double *x, long M, int C, const double *gamma,
               const double *beta, double eps, double *y, double *mean,
               double *invstd)
{
#pragma omp parallel for schedule(static)
    for (int c = 0; c < C; ++c) {
        double s = 0.0;
        for (long m = 0; m < M; ++m) s += x[m * C + c];
        double mu = s / (double)M;
        double v = 0.0;
        for (long m = 0; m < M; ++m) {
            double d = x[m * C + c] - mu;
            v += d * d;
        }
        v /= (double)M;
        double is = 1.0 / sqrt(v + eps);
        mean[c] = mu;
        invstd[c] = is;
        for (long m = 0; m < M; ++m)
            y[m * C + c] = gamma[c] * ((x[m * C + c] - mu) * is) + beta[c];
    }
}

/* Backward of oc_bn_fwd given the saved mean and invstd:
 *   dbeta = sum dy, dgamma = sum dy * x_hat,
 *   dx = gamma * invstd * (dy - dbeta/M - x_hat * dgamma/M). */
void oc_bn_bwd(const double *x, const double *dy, long M, int C,
               const double *gamma, const double *mean, const double *invstd,
               double *dx, double *dgamma, double *dbeta)
{
#pragma omp parallel for schedule(static)
    for (int c = 0; c < C; ++c) {
        double sdy = 0.0, sdyx = 0.0;
        for (long m = 0; m < M; ++m) {
            double xh = (x[m * C + c] - mean[c]) * invstd[c];
            sdy += dy[m * C + c];
            sdyx += dy[m * C + c] * xh;
        }
        dgamma[c] = sdyx;
        dbeta[c] = sdy;
        double k = gamma[c] * invstd[c];
        for (long m = 0; m < M; ++m) {
            double xh = (x[m * C + c] - mean[c]) * invstd[c];
            dx[m * C + c] = k * (dy[m * C + c] - sdy / (double)M - xh * sdyx / (double)M);
        }
    }
}

/* ------------------------------------------------- softmax cross-entropy */

/* z [B][K] logits, labels [B].  loss = mean_n (logsumexp(z_n) - z_n[label_n]);
 * dz = (softmax(z) - onehot(label)) / B.  Returns the loss. */
double oc_softmax_ce(const double *z, int B, int K, const int32_t *labels, double *dz)
{
    double total = 0.0;
    for (int n = 0; n < B; ++n) {
        const double *zr = z + (size_t)n * K;
        double m = zr[0];
        for (int k = 1; k < K; ++k) if (zr[k] > m) m = zr[k];
        double s = 0.0;
        for (int k = 0; k < K; ++k) s += exp(zr[k] - m);
        double lse = m + log(s);
        total += lse - zr[labels[n]];
        for (int k = 0; k < K; ++k) {
            double pk = exp(zr[k] - lse);
            dz[(size_t)n * K + k] = (pk - (k == labels[n] ? 1.0 : 0.0)) / (double)B;
        }
    }
    return total / (double)B;
}
