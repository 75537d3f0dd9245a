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
// logits read once, probabilities written once.
#include "common.hpp"
#include "device.hpp"

namespace fs {

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
  if (tid == 0) a.vote[b] = bi;
  if (a.mean) {
    const float invn = (float)a.N;
#pragma unroll
    for (int j = 0; j < PER; ++j) {
      const int c = tid + j * SM_T;
      if (c < a.C) a.mean[(int64_t)b * a.C + c] = S[j] / invn;
    }
  }
}

void launch_softmax_combine(const SoftmaxArgs& a, hipStream_t s) {
  const int per = (a.C + SM_T - 1) / SM_T;
  dim3 grid(a.B), block(SM_T);
  if (per <= 1) hipLaunchKernelGGL(k_softmax_combine<1>, grid, block, 0, s, a);
  else if (per <= 4) hipLaunchKernelGGL(k_softmax_combine<4>, grid, block, 0, s, a);
  else hipLaunchKernelGGL(k_softmax_combine<SM_PER>, grid, block, 0, s, a);
}

}  // namespace fs
