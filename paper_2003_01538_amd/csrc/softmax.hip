// Softmax of every model's logits and the ensemble combination, one
// workgroup per image (FlexServe returns every model's output for every
// image together with a combined result: Fig. 1 caption, Sec. 2.1, 2.3).
//
// For image b the workgroup walks the N models in order: a block-wide
// (max, first argmax) reduction gives the row maximum and the model's top-1
// class, a block-wide sum of exp(z - max) gives the denominator, and the
// probabilities are written and added into per-thread running sums S[c]
// (fp32, model order).  After the last model the same reduction picks the
// vote = smallest c maximising S, and mean = S / N is written.  One launch,
// logits read once, probabilities written once.  The other combine
// policies decide vote from the models' top-1 classes, gathered in LDS:
// plurality (the class most models rank first, the smallest among equally
// many) or detection of one class by at least k models (k = 1: the
// maximum-sensitivity OR of Sec. 2.1).
#include "common.hpp"
#include "device.hpp"

#include "flexserve.h"

namespace fs {

// vote of a top-1 policy from the N models' top-1 classes (one thread)
__device__ int policy_vote(const SoftmaxArgs& a, const int* tops) {
  if (a.policy == FS_COMBINE_ANY) {
    int n = 0;
    for (int m = 0; m < a.N; ++m) n += tops[m] == a.pos_class ? 1 : 0;
    return n >= a.min_votes ? 1 : 0;
  }
  int best = a.C, best_n = 0;  // FS_COMBINE_PLURALITY
  for (int m = 0; m < a.N; ++m) {
    int n = 0;
    for (int k = 0; k < a.N; ++k) n += tops[k] == tops[m] ? 1 : 0;
    if (n > best_n || (n == best_n && tops[m] < best)) { best_n = n; best = tops[m]; }
  }
  return best;
}

constexpr int SM_T = 256;
constexpr int SM_PER = SOFTMAX_MAX_C / SM_T;  // classes per thread, upper bound

__device__ __forceinline__ void block_argmax(float& v, int& i, float* sv, int* si) {
  wave_argmax(v, i);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) { sv[wave] = v; si[wave] = i; }
  __syncthreads();
  v = sv[0]; i = si[0];
#pragma unroll
  for (int w = 1; w < SM_T / 64; ++w)
    if (sv[w] > v || (sv[w] == v && si[w] < i)) { v = sv[w]; i = si[w]; }
}

__device__ __forceinline__ float block_sum(float v, float* sv) {
  v = wave_sum(v);
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  __syncthreads();
  if (lane == 0) sv[wave] = v;
  __syncthreads();
  float s = 0.f;
#pragma unroll
  for (int w = 0; w < SM_T / 64; ++w) s += sv[w];
  return s;
}

template <int PER>
__global__ void __launch_bounds__(SM_T) k_softmax_combine(SoftmaxArgs a) {
  __shared__ float sv[SM_T / 64];
  __shared__ int si[SM_T / 64];
  __shared__ int tops[COMBINE_MAX_PLURALITY];
  int n_pos = 0;  // models whose top-1 is the designated class (thread 0)
  const int b = blockIdx.x, tid = threadIdx.x;
  float S[PER], z[PER];
#pragma unroll
  for (int j = 0; j < PER; ++j) S[j] = 0.f;

  for (int m = 0; m < a.N; ++m) {
    const float* row = a.logits + ((int64_t)m * a.B + b) * a.C;
    float best = -INFINITY;
    int bi = a.C;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int c = tid + j * SM_T;
      z[j] = c < a.C ? row[c] : -INFINITY;
      if (c < a.C && (z[j] > best || (z[j] == best && c < bi))) { best = z[j]; bi = c; }
    }
    block_argmax(best, bi, sv, si);
    if (a.top1 && tid == 0) a.top1[(int64_t)m * a.B + b] = bi;
    if (tid == 0) {
      if (m < COMBINE_MAX_PLURALITY) tops[m] = bi;
      n_pos += bi == a.pos_class ? 1 : 0;
    }
    float e[PER], part = 0.f;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      e[j] = (tid + j * SM_T) < a.C ? expf(z[j] - best) : 0.f;
      part += e[j];
    }
    const float d = block_sum(part, sv);
    float* prow = a.probs + ((int64_t)m * a.B + b) * a.C;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int c = tid + j * SM_T;
      if (c < a.C) {
        const float p = e[j] / d;
        prow[c] = p;
        S[j] += p;
      }
    }
  }

  float best = -INFINITY;
  int bi = a.C;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int c = tid + j * SM_T;
    if (c < a.C && (S[j] > best || (S[j] == best && c < bi))) { best = S[j]; bi = c; }
  }
  block_argmax(best, bi, sv, si);
  if (tid == 0) {
    if (a.policy == FS_COMBINE_ANY) a.vote[b] = n_pos >= a.min_votes ? 1 : 0;
    else if (a.policy == FS_COMBINE_PLURALITY) a.vote[b] = policy_vote(a, tops);
    else a.vote[b] = bi;
  }
  if (a.mean) {
    const float invn = (float)a.N;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int c = tid + j * SM_T;
      if (c < a.C) a.mean[(int64_t)b * a.C + c] = S[j] / invn;
    }
  }
}

// Up to 8 models of up to 1024 classes: the models of one image run side by
// side, TPM threads each, and meet once in LDS for the combination: S[c] =
// p_0[c] + p_1[c] + ... in model order.  The chain of dependent steps is one
// model long instead of N.  With TPM = 256 (up to 4 models) the class-to-
// thread map and the reductions are those of the kernel above (so the same
// bits); 5 to 8 models take TPM = 128 (8 classes per thread, two waves per
// model), whose sums of exponentials run in another order.
template <int NG, int TPM = SM_T>
__global__ void __launch_bounds__(TPM * NG) k_softmax_combine_mg(SoftmaxArgs a) {
  constexpr int PER = 1024 / TPM, W = TPM / 64;  // classes per thread, waves per model
  __shared__ float ps[NG][PER * TPM];
  __shared__ float sv[NG * W];
  __shared__ int si[NG * W];
  __shared__ int tops[NG];
  const int b = blockIdx.x, tid = threadIdx.x;
  const int g = tid / TPM, t = tid - g * TPM, lane = tid & 63, wave = tid >> 6;
  const bool live = g < a.N;
  const float* row = a.logits + ((int64_t)(live ? g : 0) * a.B + b) * a.C;
  float z[PER], best = -INFINITY;
  int bi = a.C;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int c = t + j * TPM;
    z[j] = (live && c < a.C) ? row[c] : -INFINITY;
    if (live && c < a.C && (z[j] > best || (z[j] == best && c < bi))) { best = z[j]; bi = c; }
  }
  wave_argmax(best, bi);
  if (lane == 0) { sv[wave] = best; si[wave] = bi; }
  __syncthreads();
  best = sv[g * W]; bi = si[g * W];
#pragma unroll
  for (int w = 1; w < W; ++w)
    if (sv[g * W + w] > best || (sv[g * W + w] == best && si[g * W + w] < bi)) { best = sv[g * W + w]; bi = si[g * W + w]; }
  if (live && a.top1 && t == 0) a.top1[(int64_t)g * a.B + b] = bi;
  if (live && t == 0) tops[g] = bi;  // read after the barriers below
  float e[PER], part = 0.f;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    e[j] = (live && (t + j * TPM) < a.C) ? expf(z[j] - best) : 0.f;
    part += e[j];
  }
  part = wave_sum(part);
  __syncthreads();  // every group has read its maxima
  if (lane == 0) sv[wave] = part;
  __syncthreads();
  float d = 0.f;
#pragma unroll
  for (int w = 0; w < W; ++w) d += sv[g * W + w];
  float* prow = a.probs + ((int64_t)(live ? g : 0) * a.B + b) * a.C;
#pragma unroll
  for (int j = 0; j < PER; ++j) {
    const int c = t + j * TPM;
    if (live && c < a.C) {
      const float p = e[j] / d;
      prow[c] = p;
      ps[g][c] = p;
    }
  }
  __syncthreads();
  // combination over the classes, every thread of the block
  float cb = -INFINITY;
  int ci = a.C;
  const float invn = (float)a.N;
  for (int c = tid; c < a.C; c += TPM * NG) {
    float S = 0.f;
    for (int m = 0; m < a.N; ++m) S += ps[m][c];
    if (a.mean) a.mean[(int64_t)b * a.C + c] = S / invn;
    if (S > cb || (S == cb && c < ci)) { cb = S; ci = c; }
  }
  wave_argmax(cb, ci);
  __syncthreads();
  if (lane == 0) { sv[wave] = cb; si[wave] = ci; }
  __syncthreads();
  if (tid == 0) {
    float v = sv[0];
    int i = si[0];
    for (int w = 1; w < NG * W; ++w)
      if (sv[w] > v || (sv[w] == v && si[w] < i)) { v = sv[w]; i = si[w]; }
    a.vote[b] = a.policy == FS_COMBINE_MEAN ? i : policy_vote(a, tops);
  }
}

void launch_softmax_combine(const SoftmaxArgs& a, hipStream_t s) {
  const int per = (a.C + SM_T - 1) / SM_T;
  dim3 grid(a.B), block(SM_T);
  if (per <= 4 && a.N <= 4) {
    switch (a.N) {
      case 1: hipLaunchKernelGGL(k_softmax_combine_mg<1>, grid, dim3(SM_T * 1), 0, s, a); return;
      case 2: hipLaunchKernelGGL(k_softmax_combine_mg<2>, grid, dim3(SM_T * 2), 0, s, a); return;
      case 3: hipLaunchKernelGGL(k_softmax_combine_mg<3>, grid, dim3(SM_T * 3), 0, s, a); return;
      default: hipLaunchKernelGGL(k_softmax_combine_mg<4>, grid, dim3(SM_T * 4), 0, s, a); return;
    }
  }
  if (per <= 4 && a.N <= 8) {
    switch (a.N) {
      case 5: hipLaunchKernelGGL((k_softmax_combine_mg<5, 128>), grid, dim3(128 * 5), 0, s, a); return;
      case 6: hipLaunchKernelGGL((k_softmax_combine_mg<6, 128>), grid, dim3(128 * 6), 0, s, a); return;
      case 7: hipLaunchKernelGGL((k_softmax_combine_mg<7, 128>), grid, dim3(128 * 7), 0, s, a); return;
      default: hipLaunchKernelGGL((k_softmax_combine_mg<8, 128>), grid, dim3(128 * 8), 0, s, a); return;
    }
  }
  if (per <= 1) hipLaunchKernelGGL(k_softmax_combine<1>, grid, block, 0, s, a);
  else if (per <= 4) hipLaunchKernelGGL(k_softmax_combine<4>, grid, block, 0, s, a);
  else hipLaunchKernelGGL(k_softmax_combine<SM_PER>, grid, block, 0, s, a);
}

}  // namespace fs
