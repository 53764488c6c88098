/*
 * cfref.c -- plain fp64 CPU oracle for the ConvFirst residual block.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file or the library built from it; only the tests, the smoke
 * check and the CPU-baseline leg of the benchmark do.  It shares no code,
 * header, constant or helper with the GPU library.
 *
 * Every quantity is a double.  Callers pass the exact (widened) values of the
 * fp16/bf16 tensors the GPU consumes.  No blocking, no fusion, no reordering:
 * each function is the definition it cites, written as loops.
 *
 * Paper: A. Lavin, "On the Efficiency of Convolutional Neural Networks",
 * arXiv:2404.03617.
 *
 * Layouts (all row-major, channels fastest):
 *   x, y, d     [N][H][W][C]           activations (NHWC), Sec. 4.1.1
 *   dw_w        [k][k][C]              depth-wise taps, one k x k filter per channel
 *   w1          [E*C][C]               expand weights, row r = hidden channel r
 *   w2          [C][E*C]               project weights, row c = output channel c
 *   wd          [Cout][2][2][Cin]      2x2 stride-2 down-sampling conv
 *   scale/bias  per output channel; a NULL scale means 1, a NULL bias means 0
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#include <unistd.h>

#define CFREF_ACT_GELU_ERF 0
#define CFREF_ACT_RELU 1
#define CFREF_ACT_IDENTITY 2

int cfref_version(void) { return 1; }

/* ------------------------------------------------------------------------ */
/* Element-wise activation phi of the FFN (Sec. 5.2, eq. e:ffn).
 * GELU uses the exact Gaussian-CDF form u * Phi(u), Phi(u) = (1 + erf(u/sqrt2))/2,
 * with the C library's double-precision erf. */
double cfref_act(double u, int act)
{
    if (act == CFREF_ACT_GELU_ERF)
        return 0.5 * u * (1.0 + erf(u / sqrt(2.0)));
    if (act == CFREF_ACT_RELU)
        return u > 0.0 ? u : 0.0;
    return u;
}

/* ------------------------------------------------------------------------ */
/* Depth-wise convolution, K = C (Sec. 4.1.1, eq. f:depth-wise-conv2d), with the
 * implicit zero padding of floor(k/2) on every border (Sec. 4.1.1, text after
 * eq. f:conv2d), taps centred on the output pixel, cross-correlation (no flip):
 *   D[n,h,w,c] = s0[c] * sum_{i<k} sum_{j<k} A[i][j][c] * X[n, h+i-k/2, w+j-k/2, c] + b0[c]
 * One output pixel. */
static void dw_pixel(const double *x, const double *dw_w, const double *s0, const double *b0,
                     int H, int W, int C, int k, int n, int h, int w, double *out /*[C]*/)
{
    int pad = k / 2;
    for (int c = 0; c < C; c++) {
        double acc = 0.0;
        for (int i = 0; i < k; i++) {
            int hh = h + i - pad;
            if (hh < 0 || hh >= H)
                continue; /* zero padding */
            for (int j = 0; j < k; j++) {
                int ww = w + j - pad;
                if (ww < 0 || ww >= W)
                    continue; /* zero padding */
                double xv = x[(((int64_t)n * H + hh) * W + ww) * C + c];
                double av = dw_w[((int64_t)i * k + j) * C + c];
                acc += av * xv;
            }
        }
        out[c] = (s0 ? s0[c] : 1.0) * acc + (b0 ? b0[c] : 0.0);
    }
}

/* Point-wise convolution as a matrix product over the unfolded pixel index
 * (Sec. 4.1.1, eq. f:pointwise-matrix-conv2d):
 *   Y[p,o] = s[o] * sum_i A[o][i] * X[p,i] + b[o]         for one pixel p. */
static void pw_pixel(const double *xin /*[Cin]*/, const double *a /*[Cout][Cin]*/,
                     const double *s, const double *b, int Cin, int Cout, double *out /*[Cout]*/)
{
    for (int o = 0; o < Cout; o++) {
        double acc = 0.0;
        for (int i = 0; i < Cin; i++)
            acc += a[(int64_t)o * Cin + i] * xin[i];
        out[o] = (s ? s[o] : 1.0) * acc + (b ? b[o] : 0.0);
    }
}

/* ------------------------------------------------------------------------ */
/* Row-parallel driver: the work items are the N*H output rows (n, h). */
typedef struct job job;
typedef void (*row_fn)(const job *J, int n, int h, double *scratch);
struct job {
    row_fn fn;
    int N, H, W, C, E, k, act, Cout, gw;
    const double *x, *dw_w, *s0, *b0, *w1, *s1, *b1, *w2, *s2, *b2;
    double *y;
    size_t scratch_doubles;
    int64_t next_row; /* shared counter, taken under the lock */
    pthread_mutex_t lock;
};

static void *worker(void *arg)
{
    job *J = (job *)arg;
    double *scratch = (double *)malloc(J->scratch_doubles * sizeof(double) + 16);
    int64_t rows = (int64_t)J->N * J->H;
    for (;;) {
        pthread_mutex_lock(&J->lock);
        int64_t r = J->next_row++;
        pthread_mutex_unlock(&J->lock);
        if (r >= rows)
            break;
        J->fn(J, (int)(r / J->H), (int)(r % J->H), scratch);
    }
    free(scratch);
    return NULL;
}

int cfref_default_threads(void)
{
    long n = sysconf(_SC_NPROCESSORS_ONLN);
    return n > 0 ? (int)n : 1;
}

/* Runs J->fn over all rows on `nthreads` threads (<= 0: one per online CPU).
 * Returns the number of threads actually used. */
static int run_rows(job *J, int nthreads)
{
    if (nthreads <= 0)
        nthreads = cfref_default_threads();
    int64_t rows = (int64_t)J->N * J->H;
    if (nthreads > rows)
        nthreads = rows > 0 ? (int)rows : 1;
    J->next_row = 0;
    pthread_mutex_init(&J->lock, NULL);
    pthread_t *t = (pthread_t *)malloc(sizeof(pthread_t) * nthreads);
    for (int i = 0; i < nthreads; i++)
        pthread_create(&t[i], NULL, worker, J);
    for (int i = 0; i < nthreads; i++)
        pthread_join(t[i], NULL);
    free(t);
    pthread_mutex_destroy(&J->lock);
    return nthreads;
}

/* ------------------------------------------------------------------------ */
/* Depth-wise layer alone. */
static void dw_row(const job *J, int n, int h, double *scratch)
{
    (void)scratch;
    for (int w = 0; w < J->W; w++)
        dw_pixel(J->x, J->dw_w, J->s0, J->b0, J->H, J->W, J->C, J->k, n, h, w,
                 J->y + (((int64_t)n * J->H + h) * J->W + w) * J->C);
}

int cfref_depthwise(const double *x, const double *dw_w, const double *s0, const double *b0,
                    int N, int H, int W, int C, int k, double *d, int nthreads)
{
    job J;
    memset(&J, 0, sizeof J);
    J.fn = dw_row;
    J.N = N; J.H = H; J.W = W; J.C = C; J.k = k;
    J.x = x; J.dw_w = dw_w; J.s0 = s0; J.b0 = b0; J.y = d;
    J.scratch_doubles = 1;
    return run_rows(&J, nthreads);
}

/* Point-wise layer alone over P = N*H*W pixels (rows are taken as 1 x P). */
static void pw_row(const job *J, int n, int h, double *scratch)
{
    (void)scratch;
    int64_t p = (int64_t)n * J->H + h; /* here H is the pixel count, N == 1 */
    pw_pixel(J->x + p * J->C, J->w1, J->s1, J->b1, J->C, J->Cout, J->y + p * J->Cout);
}

int cfref_pointwise(const double *x, const double *a, const double *s, const double *b,
                    int64_t P, int Cin, int Cout, double *y, int nthreads)
{
    job J;
    memset(&J, 0, sizeof J);
    J.fn = pw_row;
    J.N = 1; J.H = (int)P; J.W = 1; J.C = Cin; J.Cout = Cout;
    J.x = x; J.w1 = a; J.s1 = s; J.b1 = b; J.y = y;
    J.scratch_doubles = 1;
    return run_rows(&J, nthreads);
}

/* ------------------------------------------------------------------------ */
/* The ConvFirst block, layer by layer (Sec. 5.3 and Sec. 5.3.1: grouped conv
 * first -- here its depth-wise case -- then the FFN of eq. e:ffn, then the
 * residual shortcut; every batch norm folded into a per-channel scale and
 * bias after its linear layer):
 *   D = s0 * dwconv(X) + b0
 *   U = s1 * (D W1^T) + b1          hidden layer, E*C channels
 *   G = phi(U)
 *   Z = s2 * (G W2^T) + b2
 *   Y = X + Z
 * The hidden layer of a whole row of pixels is materialised here on purpose:
 * this is the direct layer-by-layer algorithm. */
static void block_row(const job *J, int n, int h, double *scratch)
{
    int W = J->W, C = J->C, EC = J->E * J->C;
    double *D = scratch;              /* [W][C]  */
    double *U = D + (size_t)W * C;    /* [W][EC] */
    double *G = U + (size_t)W * EC;   /* [W][EC] */
    double *Z = G + (size_t)W * EC;   /* [W][C]  */
    for (int w = 0; w < W; w++)
        dw_pixel(J->x, J->dw_w, J->s0, J->b0, J->H, W, C, J->k, n, h, w, D + (size_t)w * C);
    for (int w = 0; w < W; w++)
        pw_pixel(D + (size_t)w * C, J->w1, J->s1, J->b1, C, EC, U + (size_t)w * EC);
    for (size_t e = 0; e < (size_t)W * EC; e++)
        G[e] = cfref_act(U[e], J->act);
    for (int w = 0; w < W; w++)
        pw_pixel(G + (size_t)w * EC, J->w2, J->s2, J->b2, EC, C, Z + (size_t)w * C);
    for (int w = 0; w < W; w++) {
        int64_t base = (((int64_t)n * J->H + h) * W + w) * C;
        for (int c = 0; c < C; c++)
            J->y[base + c] = J->x[base + c] + Z[(size_t)w * C + c];
    }
}

/* The same block with the FFN evaluated in the loop-fused order of
 * eq. e:ffn-eff: one hidden channel r at a time, produced by column r of the
 * expand and immediately consumed by row r of the project,
 *   Z = sum_r phi(D U^r + a_r) V_r + b,
 * with the output accumulator initialised from the block input (the residual
 * shortcut, Sec. 5.3.1).  It must equal block_row up to rounding order; the
 * tests use the pair to check eq. e:ffn-eff against eq. e:ffn. */
static void block_row_loopfused(const job *J, int n, int h, double *scratch)
{
    int W = J->W, C = J->C, EC = J->E * J->C;
    double *D = scratch;            /* [C] one pixel of the conv output */
    double *Z = D + C;              /* [C] projected sum for that pixel */
    for (int w = 0; w < W; w++) {
        int64_t base = (((int64_t)n * J->H + h) * W + w) * C;
        dw_pixel(J->x, J->dw_w, J->s0, J->b0, J->H, W, C, J->k, n, h, w, D);
        for (int c = 0; c < C; c++)
            Z[c] = 0.0;
        for (int r = 0; r < EC; r++) {
            double u = 0.0;
            for (int c = 0; c < C; c++)
                u += J->w1[(int64_t)r * C + c] * D[c];
            u = (J->s1 ? J->s1[r] : 1.0) * u + (J->b1 ? J->b1[r] : 0.0);
            double g = cfref_act(u, J->act);
            for (int c = 0; c < C; c++)
                Z[c] += J->w2[(int64_t)c * EC + r] * g;
        }
        for (int c = 0; c < C; c++)
            J->y[base + c] = J->x[base + c] + (J->s2 ? J->s2[c] : 1.0) * Z[c] + (J->b2 ? J->b2[c] : 0.0);
    }
}

static int block_common(row_fn fn, size_t scratch, const double *x, const double *dw_w,
                        const double *s0, const double *b0, const double *w1, const double *s1,
                        const double *b1, const double *w2, const double *s2, const double *b2,
                        int N, int H, int W, int C, int E, int k, int act, double *y, int nthreads)
{
    job J;
    memset(&J, 0, sizeof J);
    J.fn = fn;
    J.N = N; J.H = H; J.W = W; J.C = C; J.E = E; J.k = k; J.act = act;
    J.x = x; J.dw_w = dw_w; J.s0 = s0; J.b0 = b0;
    J.w1 = w1; J.s1 = s1; J.b1 = b1; J.w2 = w2; J.s2 = s2; J.b2 = b2;
    J.y = y;
    J.scratch_doubles = scratch;
    return run_rows(&J, nthreads);
}

int cfref_block_forward(const double *x, const double *dw_w, const double *s0, const double *b0,
                        const double *w1, const double *s1, const double *b1,
                        const double *w2, const double *s2, const double *b2,
                        int N, int H, int W, int C, int E, int k, int act, double *y, int nthreads)
{
    size_t scratch = (size_t)W * C * 2 + (size_t)W * E * C * 2;
    return block_common(block_row, scratch, x, dw_w, s0, b0, w1, s1, b1, w2, s2, b2,
                        N, H, W, C, E, k, act, y, nthreads);
}

int cfref_block_forward_loopfused(const double *x, const double *dw_w, const double *s0,
                                  const double *b0, const double *w1, const double *s1,
                                  const double *b1, const double *w2, const double *s2,
                                  const double *b2, int N, int H, int W, int C, int E, int k,
                                  int act, double *y, int nthreads)
{
    return block_common(block_row_loopfused, (size_t)C * 2, x, dw_w, s0, b0, w1, s1, b1, w2,
                        s2, b2, N, H, W, C, E, k, act, y, nthreads);
}

/* ------------------------------------------------------------------------ */
/* 2x2 stride-2 down-sampling convolution (the conv2d of eq. f:conv2d with
 * R = S = 2, stride 2, no padding):
 *   Yd[n,i,j,o] = sd[o] * sum_{a<2} sum_{b<2} sum_c Wd[o][a][b][c] * X[n, 2i+a, 2j+b, c] + bd[o]
 * H and W must be even; the output is H/2 x W/2 x Cout. */
static void down_row(const job *J, int n, int i, double *scratch)
{
    (void)scratch;
    int H = J->H * 2, W = J->W * 2, Cin = J->C, Cout = J->Cout;
    for (int j = 0; j < J->W; j++) {
        double *out = J->y + (((int64_t)n * J->H + i) * J->W + j) * Cout;
        for (int o = 0; o < Cout; o++) {
            double acc = 0.0;
            for (int a = 0; a < 2; a++)
                for (int b = 0; b < 2; b++)
                    for (int c = 0; c < Cin; c++)
                        acc += J->w1[(((int64_t)o * 2 + a) * 2 + b) * Cin + c] *
                               J->x[(((int64_t)n * H + 2 * i + a) * W + 2 * j + b) * Cin + c];
            out[o] = (J->s1 ? J->s1[o] : 1.0) * acc + (J->b1 ? J->b1[o] : 0.0);
        }
    }
}

int cfref_downsample(const double *x, const double *wd, const double *sd, const double *bd,
                     int N, int H, int W, int Cin, int Cout, double *y, int nthreads)
{
    if ((H % 2) || (W % 2))
        return -1;
    job J;
    memset(&J, 0, sizeof J);
    J.fn = down_row;
    J.N = N; J.H = H / 2; J.W = W / 2; J.C = Cin; J.Cout = Cout;
    J.x = x; J.w1 = wd; J.s1 = sd; J.b1 = bd; J.y = y;
    J.scratch_doubles = 1;
    return run_rows(&J, nthreads);
}

/* ------------------------------------------------------------------------ */
/* Grouped convolution, eq. f:grouped-conv2d (Sec. 4.1.1), in the paper's own
 * index order: weights A[K][R][S][T], T = C / G input channels per group,
 * group index g(k) = floor(k * C / (K * T)).  Zero padding `pad` on every
 * border and a stride, taps not flipped:
 *   Y[n,ho,wo,k] = sum_{r<R} sum_{s<S} sum_{t<T} A[k][r][s][t] *
 *                  X[n, ho*stride + r - pad, wo*stride + s - pad, g(k)*T + t]
 * Output size Ho = (H + 2 pad - R) / stride + 1, Wo likewise (R = S).
 * Serial; used on small inputs to cross-check the block's grouped layer
 * against the paper's definition.  Returns -1 on inconsistent sizes. */
int cfref_grouped_conv(const double *x, const double *a, int N, int H, int W, int C, int K, int R,
                       int T, int stride, int pad, double *y)
{
    if (T <= 0 || C % T || R <= 0 || stride <= 0 || pad < 0)
        return -1;
    int Ho = (H + 2 * pad - R) / stride + 1;
    int Wo = (W + 2 * pad - R) / stride + 1;
    if (Ho <= 0 || Wo <= 0)
        return -1;
    for (int n = 0; n < N; n++)
        for (int ho = 0; ho < Ho; ho++)
            for (int wo = 0; wo < Wo; wo++)
                for (int k = 0; k < K; k++) {
                    int g = (int)(((int64_t)k * C) / ((int64_t)K * T));
                    double acc = 0.0;
                    for (int r = 0; r < R; r++) {
                        int hh = ho * stride + r - pad;
                        if (hh < 0 || hh >= H)
                            continue;
                        for (int q = 0; q < R; q++) {
                            int ww = wo * stride + q - pad;
                            if (ww < 0 || ww >= W)
                                continue;
                            for (int t = 0; t < T; t++)
                                acc += a[(((int64_t)k * R + r) * R + q) * T + t] *
                                       x[(((int64_t)n * H + hh) * W + ww) * C + (int64_t)g * T + t];
                        }
                    }
                    y[(((int64_t)n * Ho + ho) * Wo + wo) * K + k] = acc;
                }
    return 0;
}

/* ------------------------------------------------------------------------ */
/* The ConvFirst block as the paper defines it (Sec. 5.3): a k x k grouped
 * convolution of group width gw with C input and C output channels, then the
 * FFN, then the residual shortcut, each batch norm folded into a per-channel
 * scale and bias.  Grouped taps in the library's layout A[i][j][c][t]
 * (tap-major, then output channel, then the input channel within the output
 * channel's group); output channel c reads input channels
 * floor(c / gw) * gw + t (eq. f:grouped-conv2d with K = C, T = gw):
 *   D[n,h,w,c] = s0[c] * sum_{i<k} sum_{j<k} sum_{t<gw} A[i][j][c][t] *
 *                X[n, h+i-k/2, w+j-k/2, floor(c/gw)*gw + t] + b0[c]
 * One output pixel. */
static void gconv_pixel(const double *x, const double *a, const double *s0, const double *b0,
                        int H, int W, int C, int k, int gw, int n, int h, int w, double *out /*[C]*/)
{
    int pad = k / 2;
    for (int c = 0; c < C; c++) {
        int first = (c / gw) * gw;
        double acc = 0.0;
        for (int i = 0; i < k; i++) {
            int hh = h + i - pad;
            if (hh < 0 || hh >= H)
                continue; /* zero padding */
            for (int j = 0; j < k; j++) {
                int ww = w + j - pad;
                if (ww < 0 || ww >= W)
                    continue; /* zero padding */
                for (int t = 0; t < gw; t++)
                    acc += a[(((int64_t)i * k + j) * C + c) * gw + t] *
                           x[(((int64_t)n * H + hh) * W + ww) * C + first + t];
            }
        }
        out[c] = (s0 ? s0[c] : 1.0) * acc + (b0 ? b0[c] : 0.0);
    }
}

/* Grouped layer alone. */
static void gconv_row(const job *J, int n, int h, double *scratch)
{
    (void)scratch;
    for (int w = 0; w < J->W; w++)
        gconv_pixel(J->x, J->dw_w, J->s0, J->b0, J->H, J->W, J->C, J->k, J->gw, n, h, w,
                    J->y + (((int64_t)n * J->H + h) * J->W + w) * J->C);
}

int cfref_gconv(const double *x, const double *a, const double *s0, const double *b0,
                int N, int H, int W, int C, int k, int gw, double *d, int nthreads)
{
    if (gw <= 0 || C % gw)
        return -1;
    job J;
    memset(&J, 0, sizeof J);
    J.fn = gconv_row;
    J.N = N; J.H = H; J.W = W; J.C = C; J.k = k; J.gw = gw;
    J.x = x; J.dw_w = a; J.s0 = s0; J.b0 = b0; J.y = d;
    J.scratch_doubles = 1;
    return run_rows(&J, nthreads);
}

/* The grouped block layer by layer: D (grouped conv), U = s1 (D W1^T) + b1,
 * G = phi(U), Z = s2 (G W2^T) + b2, Y = X + Z (eq. e:ffn, Sec. 5.3). */
static void gblock_row(const job *J, int n, int h, double *scratch)
{
    int W = J->W, C = J->C, EC = J->E * J->C;
    double *D = scratch;              /* [W][C]  */
    double *U = D + (size_t)W * C;    /* [W][EC] */
    double *G = U + (size_t)W * EC;   /* [W][EC] */
    double *Z = G + (size_t)W * EC;   /* [W][C]  */
    for (int w = 0; w < W; w++)
        gconv_pixel(J->x, J->dw_w, J->s0, J->b0, J->H, W, C, J->k, J->gw, n, h, w, D + (size_t)w * C);
    for (int w = 0; w < W; w++)
        pw_pixel(D + (size_t)w * C, J->w1, J->s1, J->b1, C, EC, U + (size_t)w * EC);
    for (size_t e = 0; e < (size_t)W * EC; e++)
        G[e] = cfref_act(U[e], J->act);
    for (int w = 0; w < W; w++)
        pw_pixel(G + (size_t)w * EC, J->w2, J->s2, J->b2, EC, C, Z + (size_t)w * C);
    for (int w = 0; w < W; w++) {
        int64_t base = (((int64_t)n * J->H + h) * W + w) * C;
        for (int c = 0; c < C; c++)
            J->y[base + c] = J->x[base + c] + Z[(size_t)w * C + c];
    }
}

int cfref_gblock_forward(const double *x, const double *a, const double *s0, const double *b0,
                         const double *w1, const double *s1, const double *b1,
                         const double *w2, const double *s2, const double *b2,
                         int N, int H, int W, int C, int E, int k, int gw, int act, double *y,
                         int nthreads)
{
    if (gw <= 0 || C % gw)
        return -1;
    job J;
    memset(&J, 0, sizeof J);
    J.fn = gblock_row;
    J.N = N; J.H = H; J.W = W; J.C = C; J.E = E; J.k = k; J.gw = gw; J.act = act;
    J.x = x; J.dw_w = a; J.s0 = s0; J.b0 = b0;
    J.w1 = w1; J.s1 = s1; J.b1 = b1; J.w2 = w2; J.s2 = s2; J.b2 = b2;
    J.y = y;
    J.scratch_doubles = (size_t)W * C * 2 + (size_t)W * E * C * 2;
    return run_rows(&J, nthreads);
}

/* ------------------------------------------------------------------------ */
/* The MBConv block with Squeeze & Excitation in the paper's variant
 * (Sec. 5.4 and the kernel description of Sec. 5.4.1): the depth-wise conv of
 * MBConv replaced by a grouped conv of group width gw; batch norm after each
 * conv folded into a per-channel scale and bias; SiLU after the expand and
 * after the grouped conv; the SE layer squeezes the global average of each
 * hidden channel to R values with ReLU and expands them back with a sigmoid,
 * whose output gates the hidden channels; then the project and the residual.
 * Hidden width EC = E * C.
 *   U  = SiLU(s1 * (X W1^T) + b1)                          [N,H,W,EC]
 *   V  = SiLU(s2 * gconv_k(U) + b2)                        [N,H,W,EC]
 *   sq[n,c] = (1 / (H W)) sum_{h,w} V[n,h,w,c]
 *   z[n,r]  = ReLU(sum_c Wr[r][c] sq[n,c] + br[r])         r < R
 *   g[n,c]  = sigmoid(sum_r We[c][r] z[n,r] + be[c])
 *   Y  = X + s3 * ((V * g) W2^T) + b3
 * Layouts: w1 [EC][C], gwt [k][k][EC][gw], wr [R][EC], we [EC][R],
 * w2 [C][EC] (stride 2: [K][EC]).  Serial over images (each image's SE couples all its pixels);
 * for the small late-stage shapes the block is used at. */
static double silu(double u) { return u / (1.0 + exp(-u)); }
static double sigmoid(double u) { return 1.0 / (1.0 + exp(-u)); }

/* BlurPool with the Triangle-3 filter (Sec. 5.4: the down-sampling layer of
 * the stride-2 MBConv block, after the grouped convolution), on one image
 * [H][W][Ch]: a per-channel low-pass with the separable taps [1, 2, 1] / 4
 * in each direction, then every second pixel:
 *   Vd[i][j][c] = sum_{a<3} sum_{b<3} t[a] t[b] V[r(2i + a - 1)][r(2j + b - 1)][c]
 * with one pixel of reflect padding, r(-1) = 1, r(H) = H - 2 (H, W >= 2).
 * Output ceil(H/2) x ceil(W/2). */
static void blurpool_tri3(const double *V, int H, int W, int Ch, double *Vd)
{
    static const double t[3] = {0.25, 0.5, 0.25};
    const int Ho = (H + 1) / 2, Wo = (W + 1) / 2;
    for (int i = 0; i < Ho; i++)
        for (int j = 0; j < Wo; j++)
            for (int c = 0; c < Ch; c++) {
                double acc = 0.0;
                for (int a = 0; a < 3; a++) {
                    int r = 2 * i + a - 1;
                    r = r < 0 ? -r : (r >= H ? 2 * (H - 1) - r : r);
                    for (int b = 0; b < 3; b++) {
                        int q = 2 * j + b - 1;
                        q = q < 0 ? -q : (q >= W ? 2 * (W - 1) - q : q);
                        acc += t[a] * t[b] * V[((size_t)r * W + q) * Ch + c];
                    }
                }
                Vd[((size_t)i * Wo + j) * Ch + c] = acc;
            }
}

int cfref_blurpool_tri3(const double *x, int N, int H, int W, int Ch, double *y)
{
    if (H < 2 || W < 2 || Ch <= 0)
        return -1;
    const size_t in = (size_t)H * W * Ch, out = (size_t)((H + 1) / 2) * ((W + 1) / 2) * Ch;
    for (int n = 0; n < N; n++)
        blurpool_tri3(x + n * in, H, W, Ch, y + n * out);
    return 0;
}

/* The block for stride 1 (K = C, residual) and stride 2 (BlurPool after the
 * grouped conv's activation, the squeeze over the down-sampled map, the
 * project to K channels, no residual: the output has another shape). */
static int mbconv_core(const double *x, const double *w1, const double *s1, const double *b1,
                       const double *gwt, const double *s2, const double *b2,
                       const double *wr, const double *br, const double *we, const double *be,
                       const double *w2, const double *s3, const double *b3,
                       int N, int H, int W, int C, int E, int R, int k, int gw, int stride, int K, double *y)
{
    const int EC = E * C;
    if (gw <= 0 || EC % gw || R <= 0 || k % 2 == 0 || K <= 0 || (stride == 1 && K != C) ||
        (stride != 1 && stride != 2) || (stride == 2 && (H < 2 || W < 2)))
        return -1;
    const size_t P = (size_t)H * W;
    const int Ho = stride == 2 ? (H + 1) / 2 : H, Wo = stride == 2 ? (W + 1) / 2 : W;
    const size_t Po = (size_t)Ho * Wo;
    double *U = (double *)malloc(sizeof(double) * P * EC);
    double *V = (double *)malloc(sizeof(double) * P * EC);
    double *Vd = stride == 2 ? (double *)malloc(sizeof(double) * Po * EC) : V;
    double *sq = (double *)malloc(sizeof(double) * EC);
    double *z = (double *)malloc(sizeof(double) * R);
    double *g = (double *)malloc(sizeof(double) * EC);
    if (!U || !V || !Vd || !sq || !z || !g) {
        free(U); free(V); if (Vd != V) free(Vd); free(sq); free(z); free(g);
        return -2;
    }
    const int pad = k / 2;
    for (int n = 0; n < N; n++) {
        const double *xn = x + (size_t)n * P * C;
        /* expand, folded norm, SiLU */
        for (size_t p = 0; p < P; p++)
            for (int r = 0; r < EC; r++) {
                double acc = 0.0;
                for (int c = 0; c < C; c++)
                    acc += w1[(size_t)r * C + c] * xn[p * C + c];
                U[p * EC + r] = silu((s1 ? s1[r] : 1.0) * acc + (b1 ? b1[r] : 0.0));
            }
        /* grouped conv over the hidden channels (eq. f:grouped-conv2d, K = C = EC,
         * T = gw), zero padding, folded norm, SiLU */
        for (int h = 0; h < H; h++)
            for (int w = 0; w < W; w++)
                for (int c = 0; c < EC; c++) {
                    const int first = (c / gw) * gw;
                    double acc = 0.0;
                    for (int i = 0; i < k; i++) {
                        const int hh = h + i - pad;
                        if (hh < 0 || hh >= H)
                            continue;
                        for (int j = 0; j < k; j++) {
                            const int ww = w + j - pad;
                            if (ww < 0 || ww >= W)
                                continue;
                            for (int t = 0; t < gw; t++)
                                acc += gwt[(((size_t)i * k + j) * EC + c) * gw + t] *
                                       U[((size_t)hh * W + ww) * EC + first + t];
                        }
                    }
                    V[((size_t)h * W + w) * EC + c] = silu((s2 ? s2[c] : 1.0) * acc + (b2 ? b2[c] : 0.0));
                }
        if (stride == 2)
            blurpool_tri3(V, H, W, EC, Vd);
        /* squeeze: global average, reduce to R with ReLU, expand with sigmoid */
        for (int c = 0; c < EC; c++) {
            double acc = 0.0;
            for (size_t p = 0; p < Po; p++)
                acc += Vd[p * EC + c];
            sq[c] = acc / (double)Po;
        }
        for (int r = 0; r < R; r++) {
            double acc = 0.0;
            for (int c = 0; c < EC; c++)
                acc += wr[(size_t)r * EC + c] * sq[c];
            acc += br ? br[r] : 0.0;
            z[r] = acc > 0.0 ? acc : 0.0;
        }
        for (int c = 0; c < EC; c++) {
            double acc = 0.0;
            for (int r = 0; r < R; r++)
                acc += we[(size_t)c * R + r] * z[r];
            g[c] = sigmoid(acc + (be ? be[c] : 0.0));
        }
        /* gate, project, folded norm, residual (stride 1) */
        for (size_t p = 0; p < Po; p++)
            for (int o = 0; o < K; o++) {
                double acc = 0.0;
                for (int c = 0; c < EC; c++)
                    acc += w2[(size_t)o * EC + c] * (Vd[p * EC + c] * g[c]);
                y[((size_t)n * Po + p) * K + o] =
                    (stride == 1 ? xn[p * C + o] : 0.0) + (s3 ? s3[o] : 1.0) * acc + (b3 ? b3[o] : 0.0);
            }
    }
    free(U); free(V); if (Vd != V) free(Vd); free(sq); free(z); free(g);
    return 0;
}

int cfref_mbconv_forward(const double *x, const double *w1, const double *s1, const double *b1,
                         const double *gwt, const double *s2, const double *b2,
                         const double *wr, const double *br, const double *we, const double *be,
                         const double *w2, const double *s3, const double *b3,
                         int N, int H, int W, int C, int E, int R, int k, int gw, double *y)
{
    return mbconv_core(x, w1, s1, b1, gwt, s2, b2, wr, br, we, be, w2, s3, b3, N, H, W, C, E, R, k, gw, 1, C, y);
}

/* The stride-2 MBConv block (Fig. f:mbconv, stride 2; Sec. 5.4): y is
 * [N][ceil(H/2)][ceil(W/2)][K], w2 [K][E*C], s3, b3 [K]. */
int cfref_mbconv_s2_forward(const double *x, const double *w1, const double *s1, const double *b1,
                            const double *gwt, const double *s2, const double *b2,
                            const double *wr, const double *br, const double *we, const double *be,
                            const double *w2, const double *s3, const double *b3,
                            int N, int H, int W, int C, int E, int R, int K, int k, int gw, double *y)
{
    return mbconv_core(x, w1, s1, b1, gwt, s2, b2, wr, br, we, be, w2, s3, b3, N, H, W, C, E, R, k, gw, 2, K, y);
}

/* ------------------------------------------------------------------------ */
/* The stride-2 ConvFirst block (Fig. f:convfirst-block (c): the variant that
 * down-samples with BlurPool, Triangle-3).  Reading taken (the figure is not
 * in the text): the grouped k x k conv C -> C at the input size with its
 * folded norm, D = s0 * gconv(X) + b0; BlurPool of D and of the block input
 * X; the two down-sampled maps concatenated along channels, Z = [bp(D),
 * bp(X)] (2C channels, D's first); then the FFN at the output size,
 *   U = phi(s1 * (W1 Z) + b1),  Y = s2 * (W2 U) + b2,
 * with no residual (the output has K channels on a ceil(H/2) x ceil(W/2)
 * map).  Per image this counts 2 H W C k^2 gw (conv), 2 Ho Wo 2C R (expand)
 * and 2 Ho Wo R K (project) operations, the Conv, Exp and Prj columns of
 * the stride-2 ConvFirst rows of the speed-projection tables (App. A).
 *   x [N][H][W][C], gwt [k][k][C][gw], w1 [R][2C], w2 [K][R]; s0, b0 [C];
 *   s1, b1 [R]; s2, b2 [K]; y [N][ceil(H/2)][ceil(W/2)][K]; H, W >= 2. */
int cfref_convfirst_s2_forward(const double *x, const double *gwt, const double *s0, const double *b0,
                               const double *w1, const double *s1, const double *b1, const double *w2,
                               const double *s2, const double *b2, int N, int H, int W, int C, int R,
                               int K, int k, int gw, int act, double *y)
{
    if (N < 0 || H < 2 || W < 2 || C <= 0 || R <= 0 || K <= 0 || k <= 0 || k % 2 == 0 || gw <= 0 || C % gw)
        return -1;
    const int Ho = (H + 1) / 2, Wo = (W + 1) / 2, C2 = 2 * C;
    const size_t P = (size_t)H * W, Po = (size_t)Ho * Wo;
    double *D = malloc(sizeof(double) * P * C);
    double *Dd = malloc(sizeof(double) * Po * C);
    double *Xd = malloc(sizeof(double) * Po * C);
    double *Z = malloc(sizeof(double) * C2);
    double *U = malloc(sizeof(double) * R);
    if (!D || !Dd || !Xd || !Z || !U) {
        free(D); free(Dd); free(Xd); free(Z); free(U);
        return -1;
    }
    for (int n = 0; n < N; n++) {
        /* the grouped conv and its norm at the input size */
        for (int h = 0; h < H; h++)
            for (int w = 0; w < W; w++)
                gconv_pixel(x, gwt, s0, b0, H, W, C, k, gw, n, h, w, D + ((size_t)h * W + w) * C);
        /* both maps down-sampled */
        blurpool_tri3(D, H, W, C, Dd);
        blurpool_tri3(x + (size_t)n * P * C, H, W, C, Xd);
        for (size_t p = 0; p < Po; p++) {
            for (int c = 0; c < C; c++) {
                Z[c] = Dd[p * C + c];
                Z[C + c] = Xd[p * C + c];
            }
            /* expand, norm, activation */
            for (int r = 0; r < R; r++) {
                double acc = 0.0;
                for (int c = 0; c < C2; c++)
                    acc += w1[(size_t)r * C2 + c] * Z[c];
                U[r] = cfref_act((s1 ? s1[r] : 1.0) * acc + (b1 ? b1[r] : 0.0), act);
            }
            /* project and norm */
            for (int o = 0; o < K; o++) {
                double acc = 0.0;
                for (int r = 0; r < R; r++)
                    acc += w2[(size_t)o * R + r] * U[r];
                y[((size_t)n * Po + p) * K + o] = (s2 ? s2[o] : 1.0) * acc + (b2 ? b2[o] : 0.0);
            }
        }
    }
    free(D); free(Dd); free(Xd); free(Z); free(U);
    return 0;
}
