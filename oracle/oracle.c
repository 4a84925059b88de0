/*
 * CPU oracle for the batched forward pass of a CNN partition.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the GPU library links, includes or
 * calls this file; only the test suite, the smoke check and the benchmark's
 * CPU-baseline leg load it.  It shares no code, header or table with the GPU
 * path.
 *
 * What it computes is the plain definition of each fused layer's forward pass
 * (the computation whose per-layer latency L_kbi and partition latency C_ldbij
 * the paper's planner consumes, Appendix A.1, table of MILP inputs):
 *   - 2-D cross-correlation over NCHW tensors, grouped (groups = C gives the
 *     depthwise case), zero padding, floor-mode output size;
 *   - batch norm written out unfolded, (v - mean) / sqrt(var + eps) * gamma + beta;
 *   - residual add, then ReLU or ReLU6;
 *   - max pooling with -inf padding, global average pooling;
 *   - fully connected layer over the NCHW flattening, softmax.
 * Every sum is accumulated in fp64 from the stored values.  Every stored layer
 * output is rounded once, to nearest with ties to even, from fp64 to the
 * partition's storage dtype (fp32, fp16 or bf16) and held in a float
 * container.  Softmax probabilities are returned as fp32.
 *
 * Layout NCHW (the GPU path uses NHWC), plain loops, OpenMP over (n, c).
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>
#ifdef _OPENMP
#include <omp.h>
#endif

enum { OR_F32 = 0, OR_F16 = 1, OR_BF16 = 2 };
enum { OR_ACT_NONE = 0, OR_ACT_RELU = 1, OR_ACT_RELU6 = 2 };

/* Round x to the nearest value of a binary floating-point format with a p-bit
 * significand and minimum normal exponent emin, ties to even, overflow to
 * infinity, subnormals kept.  The quantum (unit in the last place) of the
 * binade that holds x is 2^(e - (p-1)) with e = max(floor(log2|x|), emin);
 * x / quantum is exact and rint() rounds it to an integer under the default
 * round-to-nearest-even mode. */
static double round_binary(double x, int p, int emin, double max_finite)
{
    if (x == 0.0 || isnan(x) || isinf(x))
        return x;
    int e2;
    frexp(x, &e2);              /* |x| = m * 2^e2 with m in [0.5, 1) */
    int e = e2 - 1;             /* exponent of the leading bit */
    if (e < emin)
        e = emin;
    double q = ldexp(1.0, e - (p - 1));
    double r = rint(x / q) * q;
    if (fabs(r) > max_finite)
        return copysign(INFINITY, x);
    return r;
}

double oracle_round(double x, int dtype)
{
    switch (dtype) {
    case OR_F32:  return round_binary(x, 24, -126, 3.4028234663852886e38);
    case OR_F16:  return round_binary(x, 11, -14, 65504.0);
    case OR_BF16: return round_binary(x, 8, -126, 3.3895313892515355e38);
    default:      return NAN;
    }
}

void oracle_round_array(const double* x, int64_t n, int dtype, float* y)
{
    for (int64_t i = 0; i < n; ++i)
        y[i] = (float)oracle_round(x[i], dtype);
}

int oracle_num_threads(void)
{
#ifdef _OPENMP
    return omp_get_max_threads();
#else
    return 1;
#endif
}

/* Floor-mode output extent of a window of size k, stride s, padding p. */
int oracle_out_dim(int in, int k, int s, int p)
{
    return (in + 2 * p - k) / s + 1;
}

static double apply_act(double v, int act)
{
    if (act == OR_ACT_RELU)
        return v > 0.0 ? v : 0.0;
    if (act == OR_ACT_RELU6)
        return v < 0.0 ? 0.0 : (v > 6.0 ? 6.0 : v);
    return v;
}

/* First and one-past-last output index o whose input index o*s - p + t falls
 * inside [0, in).  Linear scans: slow but plainly right. */
static void valid_range(int out, int in, int s, int p, int t, int* lo, int* hi)
{
    int a = 0;
    while (a < out && a * s - p + t < 0)
        ++a;
    int b = out;
    while (b > a && (b - 1) * s - p + t >= in)
        --b;
    *lo = a;
    *hi = b;
}

/*
 * y[n][co][ho][wo] = act( BN( sum_{ci in group(co), kh, kw}
 *                               x[n][ci][ho*s - p + kh][wo*s - p + kw] * w[co][ci'][kh][kw]
 *                             + bias[co] ) + res[n][co][ho][wo] )
 * Out-of-range taps contribute zero.  bias, the four BN arrays and res may be
 * NULL (the BN arrays are either all present or all NULL).
 */
void oracle_conv2d(const float* x, int N, int C, int H, int W,
                   const float* w, int Co, int KH, int KW, int stride, int pad,
                   int groups, const float* bias,
                   const float* gamma, const float* beta, const float* mean,
                   const float* var, double eps,
                   const float* res, int act, int dtype, float* y)
{
    const int Ho = oracle_out_dim(H, KH, stride, pad);
    const int Wo = oracle_out_dim(W, KW, stride, pad);
    const int cig = C / groups, cog = Co / groups;
#pragma omp parallel for collapse(2) schedule(dynamic)
    for (int n = 0; n < N; ++n) {
        for (int co = 0; co < Co; ++co) {
            double* acc = (double*)calloc((size_t)Ho * Wo, sizeof(double));
            const int g = co / cog;
            for (int cl = 0; cl < cig; ++cl) {
                const int ci = g * cig + cl;
                const float* xp = x + ((size_t)n * C + ci) * H * W;
                for (int kh = 0; kh < KH; ++kh) {
                    int ho_lo, ho_hi;
                    valid_range(Ho, H, stride, pad, kh, &ho_lo, &ho_hi);
                    for (int kw = 0; kw < KW; ++kw) {
                        int wo_lo, wo_hi;
                        valid_range(Wo, W, stride, pad, kw, &wo_lo, &wo_hi);
                        const double wv = w[(((size_t)co * cig + cl) * KH + kh) * KW + kw];
                        for (int ho = ho_lo; ho < ho_hi; ++ho) {
                            const float* xr = xp + (size_t)(ho * stride - pad + kh) * W;
                            double* ar = acc + (size_t)ho * Wo;
                            for (int wo = wo_lo; wo < wo_hi; ++wo)
                                ar[wo] += (double)xr[wo * stride - pad + kw] * wv;
                        }
                    }
                }
            }
            const size_t obase = ((size_t)n * Co + co) * Ho * Wo;
            for (int i = 0; i < Ho * Wo; ++i) {
                double v = acc[i];
                if (bias)
                    v += bias[co];
                if (gamma)
                    v = (v - mean[co]) / sqrt((double)var[co] + eps) * gamma[co] + beta[co];
                if (res)
                    v += res[obase + i];
                y[obase + i] = (float)oracle_round(apply_act(v, act), dtype);
            }
            free(acc);
        }
    }
}

/* Max over the in-range taps of each window (padding behaves as -inf). */
void oracle_maxpool2d(const float* x, int N, int C, int H, int W,
                      int k, int stride, int pad, int dtype, float* y)
{
    const int Ho = oracle_out_dim(H, k, stride, pad);
    const int Wo = oracle_out_dim(W, k, stride, pad);
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n) {
        for (int c = 0; c < C; ++c) {
            const float* xp = x + ((size_t)n * C + c) * H * W;
            float* yp = y + ((size_t)n * C + c) * Ho * Wo;
            for (int ho = 0; ho < Ho; ++ho) {
                for (int wo = 0; wo < Wo; ++wo) {
                    double m = -INFINITY;
                    for (int kh = 0; kh < k; ++kh) {
                        const int hi = ho * stride - pad + kh;
                        if (hi < 0 || hi >= H)
                            continue;
                        for (int kw = 0; kw < k; ++kw) {
                            const int wi = wo * stride - pad + kw;
                            if (wi < 0 || wi >= W)
                                continue;
                            if (xp[hi * W + wi] > m)
                                m = xp[hi * W + wi];
                        }
                    }
                    yp[ho * Wo + wo] = (float)oracle_round(m, dtype);
                }
            }
        }
    }
}

/* y[n][c] = mean over (h, w) of x[n][c][h][w]. */
void oracle_global_avgpool(const float* x, int N, int C, int H, int W,
                           int dtype, float* y)
{
#pragma omp parallel for collapse(2)
    for (int n = 0; n < N; ++n) {
        for (int c = 0; c < C; ++c) {
            const float* xp = x + ((size_t)n * C + c) * H * W;
            double s = 0.0;
            for (int i = 0; i < H * W; ++i)
                s += xp[i];
            y[(size_t)n * C + c] = (float)oracle_round(s / (double)(H * W), dtype);
        }
    }
}

/*
 * Fully connected layer on x[N][K], the NCHW flattening (index c*H*W + h*W + w)
 * of the producer's output: z[n][o] = sum_k w[o][k] * x[n][k] + bias[o].
 * softmax == 0: y[n][o] = round_dtype(act(z)).
 * softmax != 0: y[n][o] = exp(z[n][o] - max_o z) / sum_o exp(z[n][o] - max_o z),
 *               computed in fp64 and stored as fp32 (act is ignored).
 */
void oracle_linear(const float* x, int N, int K, const float* w, int O,
                   const float* bias, int act, int softmax, int dtype, float* y)
{
    for (int n = 0; n < N; ++n) {
        double* z = (double*)malloc((size_t)O * sizeof(double));
        const float* xn = x + (size_t)n * K;
#pragma omp parallel for
        for (int o = 0; o < O; ++o) {
            const float* wo = w + (size_t)o * K;
            double s = 0.0;
            for (int k = 0; k < K; ++k)
                s += (double)wo[k] * (double)xn[k];
            if (bias)
                s += bias[o];
            z[o] = s;
        }
        if (softmax) {
            double zmax = -INFINITY;
            for (int o = 0; o < O; ++o)
                if (z[o] > zmax)
                    zmax = z[o];
            double sum = 0.0;
            for (int o = 0; o < O; ++o) {
                z[o] = exp(z[o] - zmax);
                sum += z[o];
            }
            for (int o = 0; o < O; ++o)
                y[(size_t)n * O + o] = (float)oracle_round(z[o] / sum, OR_F32);
        } else {
            for (int o = 0; o < O; ++o)
                y[(size_t)n * O + o] = (float)oracle_round(apply_act(z[o], act), dtype);
        }
        free(z);
    }
}
