/* Host driver of the CPU oracle (oracle/fso.c) for sanitizer builds: every
 * exported function on small, odd-sized inputs (ragged borders, strides,
 * padding, residuals, both storage types), so out-of-bounds accesses and
 * undefined behaviour in the oracle's loops show up under ASan/UBSan. */
#include <math.h>
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

float fso_round_bf16(float x);
void fso_round_array(const float* x, int64_t n, int prec, float* out);
void fso_set_acc32(int on);
void fso_preprocess(const uint8_t* img, int h, int w, int stride, int oh, int ow, const float* mean,
                    const float* std, int prec, float* out);
void fso_fold_bn(const float* w, int cout, int64_t per, const float* scale, const float* shift,
                 const float* bias, int prec, float* wo, float* bo);
void fso_conv2d(const float* x, int B, int H, int W, int Cin, const float* w, const float* b, const float* res,
                int Cout, int kh, int kw, int stride, int pad, int relu, int prec, float* out, float* absacc);
void fso_maxpool(const float* x, int B, int H, int W, int C, int k, int stride, int pad, float* out);
void fso_gap(const float* x, int B, int H, int W, int C, int prec, float* out);
void fso_flatten_nchw(const float* x, int B, int H, int W, int C, float* out);
void fso_fc(const float* x, int B, int K, const float* w, const float* b, int N, int relu, int prec, float* out);
void fso_softmax(const float* z, int rows, int C, float* out);
int fso_argmax(const float* x, int n);
void fso_combine(const float* p, const float* z, int N, int B, int C, float* S, float* mean, int32_t* vote,
                 int32_t* top1);
void fso_vote_policy(const int32_t* top1, int N, int B, int C, int policy, int pos, int k, int32_t* out);

static float* rnd(size_t n, unsigned* s) {
  float* a = malloc(n * sizeof(float));
  for (size_t i = 0; i < n; ++i) {
    *s = *s * 1103515245u + 12345u;
    a[i] = ((*s >> 8) & 0xffff) / 32768.0f - 1.0f;
  }
  return a;
}

int main(void) {
  unsigned s = 7;
  const float mean[3] = {0.485f, 0.456f, 0.406f}, sd[3] = {0.229f, 0.224f, 0.225f};
  uint8_t img[7 * 40 * 3];
  for (int i = 0; i < 7 * 40 * 3; ++i) img[i] = (uint8_t)(i * 37);
  float pre[9 * 5 * 3];
  for (int prec = 0; prec < 2; ++prec) fso_preprocess(img, 7, 11, 40 * 3 / 3 * 3, 9, 5, mean, sd, prec, pre);
  for (int acc = 0; acc < 2; ++acc) {
    fso_set_acc32(acc);
    for (int prec = 0; prec < 2; ++prec) {
      const int B = 2, H = 7, W = 5, Ci = 3, Co = 4;
      float *x = rnd((size_t)B * H * W * Ci, &s), *w = rnd((size_t)Co * 3 * 3 * Ci, &s), *b = rnd(Co, &s);
      float *sc = rnd(Co, &s), *sh = rnd(Co, &s), *wo = malloc(sizeof(float) * Co * 9 * Ci), *bo = malloc(sizeof(float) * Co);
      fso_fold_bn(w, Co, 9 * Ci, sc, sh, NULL, prec, wo, bo);
      fso_fold_bn(w, Co, 9 * Ci, NULL, NULL, b, prec, wo, bo);
      for (int st = 1; st <= 2; ++st)
        for (int pd = 0; pd <= 2; ++pd) {
          const int Ho = (H + 2 * pd - 3) / st + 1, Wo = (W + 2 * pd - 3) / st + 1;
          float *y = malloc(sizeof(float) * B * Ho * Wo * Co), *ab = malloc(sizeof(float) * B * Ho * Wo * Co);
          float* r = rnd((size_t)B * Ho * Wo * Co, &s);
          fso_conv2d(x, B, H, W, Ci, wo, bo, r, Co, 3, 3, st, pd, 1, prec, y, ab);
          fso_conv2d(x, B, H, W, Ci, wo, NULL, NULL, Co, 3, 3, st, pd, 0, prec, y, NULL);
          const int Hp = (Ho + 2 - 3) / 2 + 1, Wp = (Wo + 2 - 3) / 2 + 1;
          float* p = malloc(sizeof(float) * B * Hp * Wp * Co);
          fso_maxpool(y, B, Ho, Wo, Co, 3, 2, 1, p);
          float* g = malloc(sizeof(float) * B * Co);
          fso_gap(y, B, Ho, Wo, Co, prec, g);
          float* f = malloc(sizeof(float) * B * Ho * Wo * Co);
          fso_flatten_nchw(y, B, Ho, Wo, Co, f);
          float *fw = rnd((size_t)6 * Ho * Wo * Co, &s), *fo = malloc(sizeof(float) * B * 6);
          fso_fc(f, B, Ho * Wo * Co, fw, NULL, 6, 1, prec, fo);
          free(y), free(ab), free(r), free(p), free(g), free(f), free(fw), free(fo);
        }
      free(x), free(w), free(b), free(sc), free(sh), free(wo), free(bo);
    }
  }
  fso_set_acc32(0);
  const int N = 3, B = 4, C = 7;
  float *z = rnd((size_t)N * B * C, &s), *pr = malloc(sizeof(float) * N * B * C);
  float *S = malloc(sizeof(float) * B * C), *mn = malloc(sizeof(float) * B * C);
  int32_t vote[4], top1[12], out[4];
  fso_softmax(z, N * B, C, pr);
  fso_combine(pr, z, N, B, C, S, mn, vote, top1);
  fso_combine(pr, NULL, N, B, C, S, mn, vote, NULL);
  for (int pol = 1; pol <= 2; ++pol) fso_vote_policy(top1, N, B, C, pol, 2, 2, out);
  float r16[5] = {1.0f, 1.00390625f, -3.5e-39f, INFINITY, NAN}, o16[5];
  fso_round_array(r16, 5, 1, o16);
  (void)fso_round_bf16(1.5f);
  (void)fso_argmax(z, C);
  free(z), free(pr), free(S), free(mn);
  printf("oracle driver ok\n");
  return 0;
}
