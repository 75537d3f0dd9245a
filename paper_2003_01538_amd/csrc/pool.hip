// Pooling on NHWC tensors: max pool over the taps inside the image, and the
// global average pool (fp32 sum over H*W in a fixed order, divided by H*W,
// rounded once to the storage type).  Both are HBM-bound: each thread owns
// 8 (bf16) or 4 (fp32) consecutive channels, so neighbouring threads touch
// neighbouring 16-byte words.  grid.y runs over the Z models of a group.
#include "common.hpp"
#include "device.hpp"

namespace fs {

template <bool BF16>
__global__ void __launch_bounds__(256) k_maxpool(PoolArgs a) {
  constexpr int V = BF16 ? 8 : 4;
  const int CV = a.C / V;
  const int64_t total = (int64_t)a.B * a.Ho * a.Wo * CV;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int z = blockIdx.y;
  const int cv = (int)(i % CV);
  const int64_t pix = i / CV;
  const int ox = (int)(pix % a.Wo);
  const int64_t t = pix / a.Wo;
  const int oy = (int)(t % a.Ho);
  const int b = (int)(t / a.Ho);
  float m[V];
#pragma unroll
  for (int e = 0; e < V; ++e) m[e] = -INFINITY;
  for (int ky = 0; ky < a.k; ++ky) {
    const int iy = oy * a.stride - a.pad + ky;
    if ((unsigned)iy >= (unsigned)a.H) continue;
    for (int kx = 0; kx < a.k; ++kx) {
      const int ix = ox * a.stride - a.pad + kx;
      if ((unsigned)ix >= (unsigned)a.W) continue;
      const int64_t off = (((int64_t)b * a.H + iy) * a.W + ix) * a.C + cv * V;
      float v[V];
      if (BF16) {
        const uint16_t* x = reinterpret_cast<const uint16_t*>(a.x) + z * a.x_mstride;
        bf8_to_f8(*reinterpret_cast<const uint4*>(x + off), v);
      } else {
        const float* x = reinterpret_cast<const float*>(a.x) + z * a.x_mstride;
        float4 q = *reinterpret_cast<const float4*>(x + off);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
      }
#pragma unroll
      for (int e = 0; e < V; ++e) m[e] = fmaxf(m[e], v[e]);
    }
  }
  const int64_t o = pix * a.C + cv * V;
  if (BF16) {
    uint16_t* y = reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride;
    *reinterpret_cast<uint4*>(y + o) = f8_to_bf8(m);  // exact: each m is a stored bf16
  } else {
    float* y = reinterpret_cast<float*>(a.y) + z * a.y_mstride;
    *reinterpret_cast<float4*>(y + o) = make_float4(m[0], m[1], m[2], m[3]);
  }
}

// Global average pool: a workgroup owns 16 channel vectors of one image; its
// 16 pixel lanes per vector sum pixels p = lane, lane + 16, ... and the 16
// partial sums are combined in LDS in a fixed order (deterministic).
constexpr int GAP_CV = 16, GAP_PL = 16;

template <bool BF16>
__global__ void __launch_bounds__(256) k_gap(PoolArgs a) {
  constexpr int V = BF16 ? 8 : 4;
  __shared__ float part[GAP_PL][GAP_CV][V];
  const int CV = a.C / V;
  const int cv = blockIdx.x % ((CV + GAP_CV - 1) / GAP_CV) * GAP_CV + (threadIdx.x % GAP_CV);
  const int b = blockIdx.x / ((CV + GAP_CV - 1) / GAP_CV);
  const int pl = threadIdx.x / GAP_CV, lc = threadIdx.x % GAP_CV;
  const int z = blockIdx.y;
  const int HW = a.H * a.W;
  float s[V];
#pragma unroll
  for (int e = 0; e < V; ++e) s[e] = 0.f;
  if (cv < CV) {
    for (int p = pl; p < HW; p += GAP_PL) {
      const int64_t off = ((int64_t)b * HW + p) * a.C + cv * V;
      float v[V];
      if (BF16) {
        const uint16_t* x = reinterpret_cast<const uint16_t*>(a.x) + z * a.x_mstride;
        bf8_to_f8(*reinterpret_cast<const uint4*>(x + off), v);
      } else {
        const float* x = reinterpret_cast<const float*>(a.x) + z * a.x_mstride;
        float4 q = *reinterpret_cast<const float4*>(x + off);
        v[0] = q.x; v[1] = q.y; v[2] = q.z; v[3] = q.w;
      }
#pragma unroll
      for (int e = 0; e < V; ++e) s[e] += v[e];
    }
  }
#pragma unroll
  for (int e = 0; e < V; ++e) part[pl][lc][e] = s[e];
  __syncthreads();
  if (pl != 0 || cv >= CV) return;
  float t[V];
#pragma unroll
  for (int e = 0; e < V; ++e) t[e] = part[0][lc][e];
  for (int q = 1; q < GAP_PL; ++q)
#pragma unroll
    for (int e = 0; e < V; ++e) t[e] += part[q][lc][e];
  const float hw = (float)HW;
#pragma unroll
  for (int e = 0; e < V; ++e) t[e] = t[e] / hw;
  const int64_t o = (int64_t)b * a.C + cv * V;
  if (BF16) {
    uint16_t* y = reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride;
    *reinterpret_cast<uint4*>(y + o) = f8_to_bf8(t);
  } else {
    float* y = reinterpret_cast<float*>(a.y) + z * a.y_mstride;
    *reinterpret_cast<float4*>(y + o) = make_float4(t[0], t[1], t[2], t[3]);
  }
}

void launch_maxpool(const PoolArgs& a, Prec p, hipStream_t s) {
  const int V = p == BF16 ? 8 : 4;
  const int64_t total = (int64_t)a.B * a.Ho * a.Wo * (a.C / V);
  dim3 grid((unsigned)((total + 255) / 256), a.Z);
  if (p == BF16)
    hipLaunchKernelGGL(k_maxpool<true>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k_maxpool<false>, grid, dim3(256), 0, s, a);
}

void launch_gap(const PoolArgs& a, Prec p, hipStream_t s) {
  const int V = p == BF16 ? 8 : 4;
  const int groups = (a.C / V + GAP_CV - 1) / GAP_CV;
  dim3 grid(a.B * groups, a.Z);
  if (p == BF16)
    hipLaunchKernelGGL(k_gap<true>, grid, dim3(256), 0, s, a);
  else
    hipLaunchKernelGGL(k_gap<false>, grid, dim3(256), 0, s, a);
}

}  // namespace fs
