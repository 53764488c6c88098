/* Driver for the oracle under AddressSanitizer and UndefinedBehaviorSanitizer
 * (built and run by test_sanitize_cpu.py; host code only).  Every tensor is
 * its own heap allocation of exactly the size the function's contract
 * states, so a read or write past any of them, an uninitialised size
 * computation that overflows, or a data race on shared scratch in the
 * row-parallel paths shows up as a sanitizer report and a non-zero exit.
 * The shapes cover the edge cases of the oracle's loops: one pixel, images
 * smaller than the kernel, k = 7, odd sizes, several images and threads, and
 * NULL scales and biases (the row-parallel functions return the number of
 * threads they ran, the serial ones 0, and -1 for inconsistent sizes).  Two cross-checks guard against a driver that
 * calls functions without exercising them: the loop-fused block equals the
 * layer-by-layer one, and the grouped block with group width 1 equals the
 * depth-wise block. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>
#include <string.h>

int cfref_depthwise(const double *x, const double *dw_w, const double *s0, const double *b0, int N, int H, int W,
                    int C, int k, double *d, int nthreads);
int cfref_pointwise(const double *x, const double *a, const double *s, const double *b, int64_t P, int Cin,
                    int Cout, double *y, int nthreads);
int cfref_block_forward(const double *x, const double *dw_w, const double *s0, const double *b0, const double *w1,
                        const double *s1, const double *b1, const double *w2, const double *s2, const double *b2,
                        int N, int H, int W, int C, int E, int k, int act, double *y, int nthreads);
int cfref_block_forward_loopfused(const double *x, const double *dw_w, const double *s0, const double *b0,
                                  const double *w1, const double *s1, const double *b1, const double *w2,
                                  const double *s2, const double *b2, int N, int H, int W, int C, int E, int k,
                                  int act, double *y, int nthreads);
int cfref_downsample(const double *x, const double *wd, const double *sd, const double *bd, int N, int H, int W,
                     int Cin, int Cout, double *y, int nthreads);
int cfref_grouped_conv(const double *x, const double *a, int N, int H, int W, int C, int K, int R, int T,
                       int stride, int pad, double *y);
int cfref_gconv(const double *x, const double *a, const double *s0, const double *b0, int N, int H, int W, int C,
                int k, int gw, double *d, int nthreads);
int cfref_gblock_forward(const double *x, const double *a, const double *s0, const double *b0, const double *w1,
                         const double *s1, const double *b1, const double *w2, const double *s2, const double *b2,
                         int N, int H, int W, int C, int E, int k, int gw, int act, double *y, int nthreads);
int cfref_mbconv_forward(const double *x, const double *w1, const double *s1, const double *b1, const double *gwt,
                         const double *s2, const double *b2, const double *wr, const double *br, const double *we,
                         const double *be, const double *w2, const double *s3, const double *b3, int N, int H,
                         int W, int C, int E, int R, int k, int gw, double *y);
int cfref_convfirst_s2_forward(const double *x, const double *gwt, const double *s0, const double *b0,
                               const double *w1, const double *s1, const double *b1, const double *w2,
                               const double *s2, const double *b2, int N, int H, int W, int C, int R,
                               int K, int k, int gw, int act, double *y);

static uint64_t rng = 0x9e3779b97f4a7c15ull;

static double *buf(size_t n)
{
    double *p = (double *)malloc(sizeof(double) * (n ? n : 1));
    if (!p) {
        fprintf(stderr, "out of memory\n");
        exit(2);
    }
    for (size_t i = 0; i < n; i++) {
        rng = rng * 6364136223846793005ull + 1442695040888963407ull;
        p[i] = ((double)(rng >> 11) / 9007199254740992.0 - 0.5) * 0.5;
    }
    return p;
}

static int fails = 0;

static void expect(int cond, const char *what)
{
    if (!cond) {
        fprintf(stderr, "FAILED: %s\n", what);
        fails++;
    }
}

static double maxdiff(const double *a, const double *b, size_t n)
{
    double m = 0.0;
    for (size_t i = 0; i < n; i++)
        if (fabs(a[i] - b[i]) > m)
            m = fabs(a[i] - b[i]);
    return m;
}

/* the depth-wise block both ways, and the grouped block with group width 1 */
static void block_case(int N, int H, int W, int C, int E, int k, int act, int with_vectors, int nthreads)
{
    const size_t P = (size_t)N * H * W, EC = (size_t)E * C;
    double *x = buf(P * C), *dw = buf((size_t)k * k * C), *w1 = buf(EC * C), *w2 = buf((size_t)C * EC);
    double *s0 = with_vectors ? buf(C) : NULL, *b0 = with_vectors ? buf(C) : NULL;
    double *s1 = with_vectors ? buf(EC) : NULL, *b1 = with_vectors ? buf(EC) : NULL;
    double *s2 = with_vectors ? buf(C) : NULL, *b2 = with_vectors ? buf(C) : NULL;
    double *y = buf(P * C), *yf = buf(P * C), *yg = buf(P * C), *d = buf(P * C);
    char what[160];
    snprintf(what, sizeof what, "block N%d %dx%d C%d E%d k%d act%d vec%d t%d", N, H, W, C, E, k, act, with_vectors,
             nthreads);
    expect(cfref_block_forward(x, dw, s0, b0, w1, s1, b1, w2, s2, b2, N, H, W, C, E, k, act, y, nthreads) >= 0,
           what);
    expect(cfref_block_forward_loopfused(x, dw, s0, b0, w1, s1, b1, w2, s2, b2, N, H, W, C, E, k, act, yf,
                                         nthreads) >= 0,
           what);
    expect(maxdiff(y, yf, P * C) < 1e-12, "loop-fused block equals the layer-by-layer block");
    /* group width 1: the grouped taps [k][k][C][1] are the depth-wise taps */
    expect(cfref_gblock_forward(x, dw, s0, b0, w1, s1, b1, w2, s2, b2, N, H, W, C, E, k, 1, act, yg, nthreads) >= 0,
           what);
    expect(maxdiff(y, yg, P * C) == 0.0, "grouped block with group width 1 equals the depth-wise block");
    expect(cfref_depthwise(x, dw, s0, b0, N, H, W, C, k, d, nthreads) >= 0, what);
    free(x); free(dw); free(w1); free(w2); free(s0); free(b0); free(s1); free(b1); free(s2); free(b2);
    free(y); free(yf); free(yg); free(d);
}

static void grouped_case(int N, int H, int W, int C, int E, int k, int gw, int nthreads)
{
    const size_t P = (size_t)N * H * W, EC = (size_t)E * C;
    double *x = buf(P * C), *a = buf((size_t)k * k * C * gw), *w1 = buf(EC * C), *w2 = buf((size_t)C * EC);
    double *s0 = buf(C), *b0 = buf(C), *y = buf(P * C), *d = buf(P * C);
    expect(cfref_gconv(x, a, s0, b0, N, H, W, C, k, gw, d, nthreads) >= 0, "gconv");
    expect(cfref_gblock_forward(x, a, s0, b0, w1, NULL, NULL, w2, NULL, NULL, N, H, W, C, E, k, gw, 1, y,
                                nthreads) >= 0,
           "gblock");
    expect(cfref_gconv(x, a, s0, b0, N, H, W, C, k, 3, d, nthreads) < 0 || C % 3 == 0, "gconv rejects C % gw");
    free(x); free(a); free(w1); free(w2); free(s0); free(b0); free(y); free(d);
}

static void conv_case(int N, int H, int W, int C, int K, int R, int T, int stride, int pad)
{
    const int Ho = (H + 2 * pad - R) / stride + 1, Wo = (W + 2 * pad - R) / stride + 1;
    double *x = buf((size_t)N * H * W * C), *a = buf((size_t)K * R * R * T);
    double *y = buf((size_t)N * (Ho > 0 ? Ho : 1) * (Wo > 0 ? Wo : 1) * K);
    expect(cfref_grouped_conv(x, a, N, H, W, C, K, R, T, stride, pad, y) >= 0, "grouped_conv");
    free(x); free(a); free(y);
}

static void mbconv_case(int N, int H, int W, int C, int E, int R, int k, int with_vectors)
{
    const size_t P = (size_t)N * H * W, EC = (size_t)E * C;
    const int gw = 8;
    double *x = buf(P * C), *w1 = buf(EC * C), *gwt = buf((size_t)k * k * EC * gw), *wr = buf((size_t)R * EC);
    double *we = buf(EC * R), *w2 = buf((size_t)C * EC), *y = buf(P * C);
    double *s1 = with_vectors ? buf(EC) : NULL, *b1 = with_vectors ? buf(EC) : NULL;
    double *s2 = with_vectors ? buf(EC) : NULL, *b2 = with_vectors ? buf(EC) : NULL;
    double *br = with_vectors ? buf(R) : NULL, *be = with_vectors ? buf(EC) : NULL;
    double *s3 = with_vectors ? buf(C) : NULL, *b3 = with_vectors ? buf(C) : NULL;
    expect(cfref_mbconv_forward(x, w1, s1, b1, gwt, s2, b2, wr, br, we, be, w2, s3, b3, N, H, W, C, E, R, k, gw, y) >= 0,
           "mbconv");
    free(x); free(w1); free(gwt); free(wr); free(we); free(w2); free(y);
    free(s1); free(b1); free(s2); free(b2); free(br); free(be); free(s3); free(b3);
}

static void convfirst_s2_case(int N, int H, int W, int C, int R, int K, int with_vectors)
{
    const int Ho = (H + 1) / 2, Wo = (W + 1) / 2;
    double *x = buf((size_t)N * H * W * C), *gwt = buf((size_t)9 * C * 8), *w1 = buf((size_t)R * 2 * C);
    double *w2 = buf((size_t)K * R), *y = buf((size_t)N * Ho * Wo * K);
    double *s0 = with_vectors ? buf(C) : NULL, *b0 = with_vectors ? buf(C) : NULL;
    double *s1 = with_vectors ? buf(R) : NULL, *b1 = with_vectors ? buf(R) : NULL;
    double *s2 = with_vectors ? buf(K) : NULL, *b2 = with_vectors ? buf(K) : NULL;
    expect(cfref_convfirst_s2_forward(x, gwt, s0, b0, w1, s1, b1, w2, s2, b2, N, H, W, C, R, K, 3, 8, 1, y) == 0,
           "convfirst_s2");
    expect(cfref_convfirst_s2_forward(x, gwt, s0, b0, w1, s1, b1, w2, s2, b2, N, 1, W, C, R, K, 3, 8, 1, y) < 0,
           "convfirst_s2 rejects H < 2");
    free(x); free(gwt); free(w1); free(w2); free(y);
    free(s0); free(b0); free(s1); free(b1); free(s2); free(b2);
}

int main(void)
{
    /* depth-wise block: one pixel, H, W < k, odd sizes, several images and threads */
    block_case(1, 1, 1, 8, 2, 3, 0, 1, 1);
    block_case(2, 3, 2, 16, 1, 7, 1, 0, 3);
    block_case(3, 5, 7, 8, 4, 5, 2, 1, 4);
    block_case(1, 9, 4, 24, 2, 1, 0, 1, 2);
    block_case(2, 6, 6, 16, 3, 3, 0, 1, 16);
    /* grouped block and conv, group width 8 */
    grouped_case(2, 4, 5, 16, 3, 3, 8, 2);
    grouped_case(1, 1, 1, 8, 2, 5, 8, 1);
    grouped_case(1, 3, 9, 24, 1, 7, 8, 3);
    /* the paper's grouped conv equation: stride 2, dense, K != C */
    conv_case(2, 7, 6, 8, 12, 3, 8, 2, 1);
    conv_case(1, 5, 5, 16, 16, 3, 2, 1, 1);
    conv_case(1, 2, 3, 3, 16, 3, 3, 2, 1);
    /* point-wise and down-sampling layers */
    {
        double *x = buf(13 * 24), *a = buf(40 * 24), *s = buf(40), *y = buf(13 * 40);
        expect(cfref_pointwise(x, a, s, NULL, 13, 24, 40, y, 3) >= 0, "pointwise");
        free(x); free(a); free(s); free(y);
        double *xd = buf(2 * 6 * 4 * 8), *wd = buf(12 * 2 * 2 * 8), *yd = buf(2 * 3 * 2 * 12);
        expect(cfref_downsample(xd, wd, NULL, NULL, 2, 6, 4, 8, 12, yd, 2) >= 0, "downsample");
        expect(cfref_downsample(xd, wd, NULL, NULL, 2, 5, 4, 8, 12, yd, 2) < 0, "downsample rejects odd H");
        free(xd); free(wd); free(yd);
    }
    /* MBConv + SE: one pixel, odd sizes, several images, NULL vectors */
    mbconv_case(1, 1, 1, 16, 1, 4, 3, 1);
    mbconv_case(2, 3, 5, 16, 2, 8, 3, 0);
    mbconv_case(1, 4, 4, 8, 4, 1, 5, 1);
    /* stride-2 ConvFirst: the smallest image, odd sizes, NULL vectors */
    convfirst_s2_case(1, 2, 2, 8, 16, 8, 1);
    convfirst_s2_case(2, 5, 7, 16, 24, 16, 0);
    convfirst_s2_case(1, 9, 4, 24, 32, 8, 1);
    if (fails) {
        fprintf(stderr, "%d check(s) failed\n", fails);
        return 1;
    }
    printf("sanitize_oracle: ok\n");
    return 0;
}
