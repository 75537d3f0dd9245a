/*
 * fso.c -- plain, slow CPU oracle for the ensemble-inference path.
 *
 * TEST INFRASTRUCTURE ONLY.  Nothing in the product path may call, link or
 * load this file; only the tests, the smoke check and the CPU baseline of the
 * benchmark do.  It shares no code, header, table or helper with the HIP
 * library.
 *
 * What it computes (FlexServe, Fig. 1 caption and Sec. 2.2-2.3): one data
 * transformation of a batch of images shared by every model, the forward
 * pass of each CNN of the ensemble on that one tensor, a softmax per model,
 * and the per-image combination of the models' outputs.  The paper fixes no
 * arithmetic; the definitions below are the textbook ones:
 *
 *   resize     bilinear, half-pixel centres, no antialias, border clamp
 *   normalise  x = (v/255 - mean_c)/std_c
 *   conv       y = act(sum_{ky,kx,ci} in*w + bias (+ residual)), zero padding;
 *              a block's projection shortcut (1x1 conv) summed into the
 *              block's last conv before its one storage point (fso_conv2d_proj)
 *   max pool   max over the taps inside the image
 *   avg pool   mean over all H*W positions
 *   fc         z = b + W f
 *   softmax    p_j = exp(z_j - max z) / sum_k exp(z_k - max z)
 *   combine    S = sum over models of p, mean = S/N, vote = argmax S;
 *              or, from the models' top-1 classes, plurality or detection
 *              of one class by at least k models (fso_vote_policy)
 *
 * Arithmetic: every sum is accumulated in double precision, and each value
 * the GPU path *stores* is rounded to the storage type at that point:
 * prec 0 = fp32, prec 1 = bf16 (round to nearest, ties to even).  The
 * storage points are: the normalised input, each conv output after its full
 * epilogue (except a projection shortcut, whose sum goes straight into the
 * block's last conv), the average-pool output, hidden FC outputs, and the
 * weights once after the batch-norm fold.  Logits, probabilities and sums
 * stay fp32.
 *
 * Layout: activations are NHWC (batch, row, column, channel), row-major.
 * Parallelism: OpenMP over independent outputs only; each output's
 * summation order is fixed, so results do not depend on the thread count.
 *
 * Build: gcc -O2 -fopenmp -fno-fast-math -shared -fPIC fso.c -lm
 */
#include <math.h>
#include <stdint.h>
#include <string.h>
#include <float.h>

/* Accumulation switch: 0 = double (default), 1 = float, sequential.  The
 * float mode exists only to measure the oracle's own summation-order noise. */
static int g_acc32 = 0;
void fso_set_acc32(int on) { g_acc32 = on ? 1 : 0; }

/* ---------------------------------------------------------------- rounding */

/* Round a float to the nearest bfloat16 (8 significand bits), ties to even,
 * returned as a float.  NaN stays NaN, infinities stay infinite. */
float fso_round_bf16(float x)
{
    uint32_t u;
    memcpy(&u, &x, 4);
    if ((u & 0x7f800000u) == 0x7f800000u) {        /* inf or nan */
        if (u & 0x007fffffu) u = (u & 0xffff0000u) | 0x00400000u;   /* quiet nan */
        else u &= 0xffff0000u;                                          /* +-inf */
    } else {
        uint32_t lsb = (u >> 16) & 1u;                 /* ties go to the even neighbour */
        u += 0x7fffu + lsb;
        u &= 0xffff0000u;
    }
    float r;
    memcpy(&r, &u, 4);
    return r;
}

/* The storage rounding: double -> fp32 (round to nearest), then for bf16 a
 * second rounding fp32 -> bf16, exactly as a kernel that accumulates in fp32
 * and stores bf16 would see it. */
static float store(double v, int prec)
{
    float f = (float)v;
    return prec ? fso_round_bf16(f) : f;
}

void fso_round_array(const float *x, int64_t n, int prec, float *out)
{
    for (int64_t i = 0; i < n; ++i) out[i] = prec ? fso_round_bf16(x[i]) : x[i];
}

/* ------------------------------------------------------ resize + normalise */

/* One image: uint8 HWC RGB (h rows, w columns, row_stride bytes per row) to
 * a [out_h][out_w][3] float tensor: bilinear resize with half-pixel centres
 * (source coordinate s = (o + 1/2) * in/out - 1/2, clamped below at 0, the
 * upper neighbour clamped at the last row/column), then (v/255 - mean)/std
 * per channel, stored in precision prec. */
void fso_preprocess(const uint8_t *img, int h, int w, int row_stride,
                    int out_h, int out_w, const float *mean, const float *stdv,
                    int prec, float *out)
{
    const double sh = (double)h / (double)out_h;
    const double sw = (double)w / (double)out_w;
    #pragma omp parallel for schedule(static)
    for (int oy = 0; oy < out_h; ++oy) {
        double sy = (oy + 0.5) * sh - 0.5;
        if (sy < 0) sy = 0;
        int y0 = (int)floor(sy);
        if (y0 > h - 1) y0 = h - 1;
        int y1 = y0 + 1 < h ? y0 + 1 : h - 1;
        double ly = sy - y0, hy = 1.0 - ly;
        for (int ox = 0; ox < out_w; ++ox) {
            double sx = (ox + 0.5) * sw - 0.5;
            if (sx < 0) sx = 0;
            int x0 = (int)floor(sx);
            if (x0 > w - 1) x0 = w - 1;
            int x1 = x0 + 1 < w ? x0 + 1 : w - 1;
            double lx = sx - x0, hx = 1.0 - lx;
            for (int c = 0; c < 3; ++c) {
                double v00 = img[(int64_t)y0 * row_stride + x0 * 3 + c];
                double v01 = img[(int64_t)y0 * row_stride + x1 * 3 + c];
                double v10 = img[(int64_t)y1 * row_stride + x0 * 3 + c];
                double v11 = img[(int64_t)y1 * row_stride + x1 * 3 + c];
                double v = hy * (hx * v00 + lx * v01) + ly * (hx * v10 + lx * v11);
                double x = (v / 255.0 - (double)mean[c]) / (double)stdv[c];
                out[((int64_t)oy * out_w + ox) * 3 + c] = store(x, prec);
            }
        }
    }
}

/* ------------------------------------------------------------- BN folding */

/* w'[co][...] = w[co][...] * scale[co] as a single-precision product, then
 * stored in precision prec; b'[co] = shift[co] (or bias, or 0). */
void fso_fold_bn(const float *w, int cout, int64_t per_out, const float *scale,
                 const float *shift, const float *bias, int prec,
                 float *w_out, float *b_out)
{
    for (int co = 0; co < cout; ++co) {
        float s = scale ? scale[co] : 1.0f;
        for (int64_t i = 0; i < per_out; ++i) {
            float p = scale ? (float)((double)w[co * per_out + i] * (double)s)
                            : w[co * per_out + i];
            w_out[co * per_out + i] = prec ? fso_round_bf16(p) : p;
        }
        b_out[co] = shift ? shift[co] : (bias ? bias[co] : 0.0f);
    }
}

/* ------------------------------------------------------------ convolution */

/* in  [B][H][W][Cin], w [Cout][kh][kw][Cin], bias [Cout] or NULL,
 * res [B][Ho][Wo][Cout] or NULL, out [B][Ho][Wo][Cout] with
 * Ho = (H + 2 pad - kh)/stride + 1 (likewise Wo).
 * out = store(relu?(sum + bias + res)).  Taps outside the image contribute
 * zero.  absacc, if not NULL, receives sum |in*w| per output (for the
 * rounding bound of a reordered fp32 sum). */
void fso_conv2d(const float *in, int B, int H, int W, int Cin,
                const float *w, const float *bias, const float *res,
                int Cout, int kh, int kw, int stride, int pad, int relu,
                int prec, float *out, float *absacc)
{
    const int Ho = (H + 2 * pad - kh) / stride + 1;
    const int Wo = (W + 2 * pad - kw) / stride + 1;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int oy = 0; oy < Ho; ++oy) {
            for (int ox = 0; ox < Wo; ++ox) {
                for (int co = 0; co < Cout; ++co) {
                    double acc = 0.0, aabs = 0.0;
                    float acc32 = 0.0f;
                    for (int ky = 0; ky < kh; ++ky) {
                        int iy = oy * stride - pad + ky;
                        if (iy < 0 || iy >= H) continue;
                        for (int kx = 0; kx < kw; ++kx) {
                            int ix = ox * stride - pad + kx;
                            if (ix < 0 || ix >= W) continue;
                            const float *xp = in + (((int64_t)b * H + iy) * W + ix) * Cin;
                            const float *wp = w + (((int64_t)co * kh + ky) * kw + kx) * Cin;
                            for (int ci = 0; ci < Cin; ++ci) {
                                double p = (double)xp[ci] * (double)wp[ci];
                                acc += p;
                                aabs += fabs(p);
                                if (g_acc32) acc32 = acc32 + xp[ci] * wp[ci];
                            }
                        }
                    }
                    if (g_acc32) acc = acc32;
                    double y = acc + (bias ? (double)bias[co] : 0.0);
                    int64_t o = (((int64_t)b * Ho + oy) * Wo + ox) * Cout + co;
                    if (res) y += (double)res[o];
                    if (relu && y < 0) y = 0;
                    out[o] = store(y, prec);
                    if (absacc) absacc[o] = (float)aabs;
                }
            }
        }
    }
}

/* The last conv of a residual block whose shortcut is a projection (a 1x1
 * conv of the block input with stride s2, no activation; He et al.'s
 * ResNets, the kind of CNN the ensemble serves): the projection is not
 * stored on its own; its products join the conv's sum,
 *   y = store(relu?(sum_{ky,kx,ci} in*w + sum_{c2} in2[b][oy*s2][ox*s2][c2]*w2[co][c2]
 *                   + bias + bias2)),
 * in  [B][H][W][Cin], w [Cout][kh][kw][Cin], in2 [B][H2][W2][C2],
 * w2 [Cout][C2], bias / bias2 [Cout] or NULL.  The main conv's terms are
 * summed first, then the projection's, in ascending c2.  absacc as in
 * fso_conv2d (over both sets of products). */
void fso_conv2d_proj(const float *in, int B, int H, int W, int Cin, const float *w, const float *bias,
                     const float *in2, int H2, int W2, int C2, const float *w2, const float *bias2, int s2,
                     int Cout, int kh, int kw, int stride, int pad, int relu, int prec,
                     float *out, float *absacc)
{
    const int Ho = (H + 2 * pad - kh) / stride + 1;
    const int Wo = (W + 2 * pad - kw) / stride + 1;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b) {
        for (int oy = 0; oy < Ho; ++oy) {
            for (int ox = 0; ox < Wo; ++ox) {
                const float *x2 = in2 + (((int64_t)b * H2 + (int64_t)oy * s2) * W2 + (int64_t)ox * s2) * C2;
                for (int co = 0; co < Cout; ++co) {
                    double acc = 0.0, aabs = 0.0;
                    float acc32 = 0.0f;
                    for (int ky = 0; ky < kh; ++ky) {
                        int iy = oy * stride - pad + ky;
                        if (iy < 0 || iy >= H) continue;
                        for (int kx = 0; kx < kw; ++kx) {
                            int ix = ox * stride - pad + kx;
                            if (ix < 0 || ix >= W) continue;
                            const float *xp = in + (((int64_t)b * H + iy) * W + ix) * Cin;
                            const float *wp = w + (((int64_t)co * kh + ky) * kw + kx) * Cin;
                            for (int ci = 0; ci < Cin; ++ci) {
                                double p = (double)xp[ci] * (double)wp[ci];
                                acc += p;
                                aabs += fabs(p);
                                if (g_acc32) acc32 = acc32 + xp[ci] * wp[ci];
                            }
                        }
                    }
                    const float *w2p = w2 + (int64_t)co * C2;
                    for (int c2 = 0; c2 < C2; ++c2) {
                        double p = (double)x2[c2] * (double)w2p[c2];
                        acc += p;
                        aabs += fabs(p);
                        if (g_acc32) acc32 = acc32 + x2[c2] * w2p[c2];
                    }
                    if (g_acc32) acc = acc32;
                    double y = acc + (bias ? (double)bias[co] : 0.0) + (bias2 ? (double)bias2[co] : 0.0);
                    if (relu && y < 0) y = 0;
                    int64_t o = (((int64_t)b * Ho + oy) * Wo + ox) * Cout + co;
                    out[o] = store(y, prec);
                    if (absacc) absacc[o] = (float)aabs;
                }
            }
        }
    }
}

/* --------------------------------------------------------------- pooling */

/* Max over the k x k taps of each window that fall inside the image.  No
 * rounding: the result is one of the inputs. */
void fso_maxpool(const float *in, int B, int H, int W, int C, int k, int stride,
                 int pad, float *out)
{
    const int Ho = (H + 2 * pad - k) / stride + 1;
    const int Wo = (W + 2 * pad - k) / stride + 1;
    #pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b)
        for (int oy = 0; oy < Ho; ++oy)
            for (int ox = 0; ox < Wo; ++ox)
                for (int c = 0; c < C; ++c) {
                    float m = -INFINITY;
                    for (int ky = 0; ky < k; ++ky) {
                        int iy = oy * stride - pad + ky;
                        if (iy < 0 || iy >= H) continue;
                        for (int kx = 0; kx < k; ++kx) {
                            int ix = ox * stride - pad + kx;
                            if (ix < 0 || ix >= W) continue;
                            float v = in[(((int64_t)b * H + iy) * W + ix) * C + c];
                            if (v > m) m = v;
                        }
                    }
                    out[(((int64_t)b * Ho + oy) * Wo + ox) * C + c] = m;
                }
}

/* Global average: out[b][c] = store(sum_{y,x} in[b][y][x][c] / (H*W)). */
void fso_gap(const float *in, int B, int H, int W, int C, int prec, float *out)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b)
        for (int c = 0; c < C; ++c) {
            double s = 0.0;
            for (int i = 0; i < H * W; ++i) s += in[((int64_t)b * H * W + i) * C + c];
            out[(int64_t)b * C + c] = store(s / (double)(H * W), prec);
        }
}

/* ------------------------------------------------------------------- FC */

/* Flatten an NHWC map to the channel-major order c*H*W + y*W + x. */
void fso_flatten_nchw(const float *in, int B, int H, int W, int C, float *out)
{
    for (int b = 0; b < B; ++b)
        for (int c = 0; c < C; ++c)
            for (int y = 0; y < H; ++y)
                for (int x = 0; x < W; ++x)
                    out[(int64_t)b * C * H * W + ((int64_t)c * H + y) * W + x] =
                        in[(((int64_t)b * H + y) * W + x) * C + c];
}

/* out[b][n] = store(relu?(bias[n] + sum_k in[b][k] * w[n][k])); the final
 * layer passes prec 0 so its logits stay fp32. */
void fso_fc(const float *in, int B, int K, const float *w, const float *bias, int N,
            int relu, int prec, float *out)
{
    #pragma omp parallel for collapse(2) schedule(static)
    for (int b = 0; b < B; ++b)
        for (int n = 0; n < N; ++n) {
            double acc = 0.0;
            float acc32 = 0.0f;
            for (int k = 0; k < K; ++k) {
                acc += (double)in[(int64_t)b * K + k] * (double)w[(int64_t)n * K + k];
                if (g_acc32) acc32 = acc32 + in[(int64_t)b * K + k] * w[(int64_t)n * K + k];
            }
            if (g_acc32) acc = acc32;
            double y = acc + (bias ? (double)bias[n] : 0.0);
            if (relu && y < 0) y = 0;
            out[(int64_t)b * N + n] = store(y, prec);
        }
}

/* --------------------------------------------------- softmax and combine */

/* Row-wise softmax of z [R][C]: subtract the row max, exponentiate, divide by
 * the sum (all in double), store fp32. */
void fso_softmax(const float *z, int R, int C, float *p)
{
    for (int r = 0; r < R; ++r) {
        const float *zr = z + (int64_t)r * C;
        double m = -INFINITY;
        for (int j = 0; j < C; ++j) if (zr[j] > m) m = zr[j];
        double d = 0.0;
        for (int j = 0; j < C; ++j) d += exp((double)zr[j] - m);
        for (int j = 0; j < C; ++j)
            p[(int64_t)r * C + j] = (float)(exp((double)zr[j] - m) / d);
    }
}

/* Smallest index attaining the maximum of x[0..n). */
int fso_argmax(const float *x, int n)
{
    int best = 0;
    for (int j = 1; j < n; ++j) if (x[j] > x[best]) best = j;
    return best;
}

/* Ensemble combination of per-model probabilities p [N][B][C]:
 *   S[b][c] = sum_i p[i][b][c] (double, rounded to fp32),
 *   mean    = S / N,
 *   vote[b] = smallest c maximising S[b][c],
 * and per-model top-1 from the logits z [N][B][C] (smallest maximising c). */
void fso_combine(const float *p, const float *z, int N, int B, int C,
                 float *S, float *mean, int32_t *vote, int32_t *top1)
{
    for (int b = 0; b < B; ++b) {
        for (int c = 0; c < C; ++c) {
            double s = 0.0;
            for (int i = 0; i < N; ++i) s += p[((int64_t)i * B + b) * C + c];
            S[(int64_t)b * C + c] = (float)s;
            if (mean) mean[(int64_t)b * C + c] = (float)(s / N);
        }
        vote[b] = fso_argmax(S + (int64_t)b * C, C);
        if (z && top1)
            for (int i = 0; i < N; ++i)
                top1[(int64_t)i * B + b] = fso_argmax(z + ((int64_t)i * B + b) * C, C);
    }
}

/* Combined result from the models' top-1 classes top1 [N][B] (Sec. 2.1: the
 * consumer combines the outputs by its own policy).
 *   policy 1, plurality: out[b] = the class named top-1 by the most models,
 *     the smallest such class when several are named equally often; found
 *     by counting the votes of every class 0..C-1.
 *   policy 2, detection of class pos: model i reports y_i = 1 when its top-1
 *     class is pos; out[b] = 1 when at least k of the y_i are 1.  k = 1 is
 *     y_1 | y_2 | ... | y_N, the maximum-sensitivity policy. */
void fso_vote_policy(const int32_t *top1, int N, int B, int C, int policy, int pos, int k, int32_t *out)
{
    for (int b = 0; b < B; ++b) {
        if (policy == 2) {
            int yes = 0;
            for (int i = 0; i < N; ++i) yes += top1[(int64_t)i * B + b] == pos;
            out[b] = yes >= k;
        } else {
            int best = 0, best_votes = -1;
            for (int c = 0; c < C; ++c) {
                int votes = 0;
                for (int i = 0; i < N; ++i) votes += top1[(int64_t)i * B + b] == c;
                if (votes > best_votes) { best_votes = votes; best = c; }
            }
            out[b] = best;
        }
    }
}
