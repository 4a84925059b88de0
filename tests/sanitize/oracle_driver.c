/* Exercises every oracle entry point on small tensors held in exactly sized
 * heap buffers, so that AddressSanitizer and UndefinedBehaviorSanitizer see
 * any out-of-bounds access or undefined operation (test infrastructure). */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

double oracle_round(double x, int dtype);
void oracle_round_array(const double* x, int64_t n, int dtype, float* y);
int oracle_out_dim(int in, int k, int s, int p);
void oracle_conv2d(const float* x, int N, int C, int H, int W, const float* w, int Co, int KH,
                   int KW, int stride, int pad, int groups, const float* bias,
                   const float* gamma, const float* beta, const float* mean, const float* var,
                   double eps, const float* res, int act, int dtype, float* y);
void oracle_maxpool2d(const float* x, int N, int C, int H, int W, int k, int stride, int pad,
                      int dtype, float* y);
void oracle_global_avgpool(const float* x, int N, int C, int H, int W, int dtype, float* y);
void oracle_linear(const float* x, int N, int K, const float* w, int O, const float* bias,
                   int act, int softmax, int dtype, float* y);

static uint64_t st = 0x9e3779b97f4a7c15ull;
static float rnd(void)
{
    st ^= st << 13; st ^= st >> 7; st ^= st << 17;
    return (float)((st >> 11) * (1.0 / 9007199254740992.0)) * 2.0f - 1.0f;
}
static float* buf(size_t n)
{
    float* p = (float*)malloc(n * sizeof(float));
    for (size_t i = 0; i < n; ++i) p[i] = rnd();
    return p;
}

int main(void)
{
    int checked = 0;
    for (int dt = 0; dt < 3; ++dt) {
        /* convolutions: k, stride, pad, groups (1, 2, depthwise), BN, residual, act */
        const int cases[][6] = {{3, 1, 1, 1, 1, 1}, {3, 2, 1, 2, 0, 2}, {1, 1, 0, 1, 1, 0},
                                {7, 2, 3, 1, 1, 1}, {3, 2, 1, 4, 1, 2}, {5, 1, 2, 1, 0, 0}};
        for (size_t c = 0; c < sizeof cases / sizeof cases[0]; ++c) {
            const int k = cases[c][0], s = cases[c][1], p = cases[c][2];
            const int N = 2, C = 4, H = 9, W = 7;
            const int g = cases[c][3] == 4 ? C : cases[c][3], Co = g == C ? C : 6;
            const int Ho = oracle_out_dim(H, k, s, p), Wo = oracle_out_dim(W, k, s, p);
            float* x = buf((size_t)N * C * H * W);
            float* w = buf((size_t)Co * (C / g) * k * k);
            float* b = buf(Co);
            float *ga = buf(Co), *be = buf(Co), *mu = buf(Co), *va = buf(Co);
            for (int i = 0; i < Co; ++i) va[i] = 1.0f + 0.5f * va[i];
            float* r = cases[c][4] ? buf((size_t)N * Co * Ho * Wo) : NULL;
            float* y = (float*)malloc((size_t)N * Co * Ho * Wo * sizeof(float));
            oracle_conv2d(x, N, C, H, W, w, Co, k, k, s, p, g, c % 2 ? b : NULL,
                          c % 3 ? ga : NULL, be, mu, va, 1e-5, r, cases[c][5], dt, y);
            for (int i = 0; i < N * Co * Ho * Wo; ++i) checked += isfinite(y[i]) ? 1 : 0;
            free(x); free(w); free(b); free(ga); free(be); free(mu); free(va); free(r); free(y);
        }
        /* pooling: 3x3 s2 p1, 2x2 s2 p0 */
        for (int q = 0; q < 2; ++q) {
            const int k = q ? 2 : 3, s = 2, p = q ? 0 : 1, N = 2, C = 3, H = 7, W = 8;
            const int Ho = oracle_out_dim(H, k, s, p), Wo = oracle_out_dim(W, k, s, p);
            float* x = buf((size_t)N * C * H * W);
            float* y = (float*)malloc((size_t)N * C * Ho * Wo * sizeof(float));
            oracle_maxpool2d(x, N, C, H, W, k, s, p, dt, y);
            float* z = (float*)malloc((size_t)N * C * sizeof(float));
            oracle_global_avgpool(x, N, C, H, W, dt, z);
            checked += (int)(y[0] == y[0]) + (int)(z[0] == z[0]);
            free(x); free(y); free(z);
        }
        /* fully connected, with ReLU and with softmax */
        for (int sm = 0; sm < 2; ++sm) {
            const int N = 3, K = 37, O = 11;
            float *x = buf((size_t)N * K), *w = buf((size_t)O * K), *b = buf(O);
            float* y = (float*)malloc((size_t)N * O * sizeof(float));
            oracle_linear(x, N, K, w, O, b, sm ? 0 : 1, sm, dt, y);
            checked += (int)(y[0] == y[0]);
            free(x); free(w); free(b); free(y);
        }
        /* rounding at the edges of each format */
        const double edge[] = {0.0, -0.0, 65504.0, 65520.0, 1e-8, 3.0e38, -1e-45, NAN, INFINITY};
        float out[9];
        oracle_round_array(edge, 9, dt, out);
        for (int i = 0; i < 9; ++i) checked += (int)(oracle_round(edge[i], dt) == out[i] ||
                                                      (isnan(out[i]) && isnan(edge[i])));
    }
    printf("oracle sanitizer driver: %d values checked\n", checked);
    return checked > 0 ? 0 : 1;
}
