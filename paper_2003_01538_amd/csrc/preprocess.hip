// The one data transformation shared by every model of the ensemble
// (FlexServe, Fig. 1 caption; Sec. 2.2): bilinear resize of each uint8 HWC
// image to out_h x out_w (half-pixel centres, no antialias, the upper
// neighbour clamped at the border), then (v/255 - mean)/std per channel,
// written once as NHWC with the channel dimension padded to 4 (the padding
// channel is 0) so that the first convolution loads one aligned 8- or
// 16-byte vector per pixel, and/or in a space-to-depth layout (2x2 pixel
// blocks of 3 channels, padded to 16) that turns a stride-2 first
// convolution into a stride-1 one with 64-element filter rows.
//
// One thread per output pixel, 256 consecutive pixels of one image per
// workgroup: the stores are fully coalesced; the four taps are gathered
// through the cache (HBM-bound on the output for upscaling, on the input for
// downscaling).  Ragged batches need no host work: each image's size comes
// from its device-side descriptor.
#include "common.hpp"
#include "device.hpp"

namespace fs {

// Transformed value of output pixel (oy, ox), channels 0..2, of image d.
__device__ __forceinline__ void transform_pixel(const PreArgs& a, const ImageDesc& d, int oy, int ox, float* o) {
  const uint8_t* img = a.pixels + d.offset;
  // Source coordinate s = ((2o + 1) * in - out) / (2 * out), clamped at 0:
  // the integer part and the fraction come from exact integer arithmetic,
  // so only the fraction itself is rounded (relative error 2^-24).
  const int ny = (2 * oy + 1) * d.h - a.out_h, dy = 2 * a.out_h;
  const int nx = (2 * ox + 1) * d.w - a.out_w, dx = 2 * a.out_w;
  int y0 = 0, x0 = 0;
  float ly = 0.f, lx = 0.f;
  if (ny > 0) { y0 = ny / dy; ly = (float)(ny - y0 * dy) / (float)dy; }
  if (nx > 0) { x0 = nx / dx; lx = (float)(nx - x0 * dx) / (float)dx; }
  y0 = min(y0, d.h - 1);
  x0 = min(x0, d.w - 1);
  const int y1 = min(y0 + 1, d.h - 1), x1 = min(x0 + 1, d.w - 1);
  const float hy = 1.0f - ly, hx = 1.0f - lx;
  const uint8_t* r0 = img + (int64_t)y0 * d.row_stride;
  const uint8_t* r1 = img + (int64_t)y1 * d.row_stride;
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    float v00 = r0[x0 * 3 + c], v01 = r0[x1 * 3 + c];
    float v10 = r1[x0 * 3 + c], v11 = r1[x1 * 3 + c];
    float v = hy * (hx * v00 + lx * v01) + ly * (hx * v10 + lx * v11);
    o[c] = (v / 255.0f - a.mean[c]) / a.std_[c];
  }
}

template <bool BF16>
__global__ void __launch_bounds__(256) k_preprocess(PreArgs a) {
  const int b = blockIdx.y;
  const int pix = blockIdx.x * 256 + threadIdx.x;
  if (pix >= a.out_h * a.out_w) return;
  const int oy = pix / a.out_w, ox = pix - oy * a.out_w;
  const ImageDesc d = a.desc[b];
  float o[4];
  transform_pixel(a, d, oy, ox, o);
  o[3] = 0.0f;
  const int64_t idx = ((int64_t)b * a.out_h * a.out_w + pix);
  if (BF16) {
    floatx4 f = {o[0], o[1], o[2], o[3]};
    bf16x4 h = __builtin_convertvector(f, bf16x4);
    reinterpret_cast<uint2*>(a.out)[idx] = __builtin_bit_cast(uint2, h);
  } else {
    reinterpret_cast<float4*>(a.out)[idx] = make_float4(o[0], o[1], o[2], o[3]);
  }
}

// Space-to-depth layout for a stride-2 first convolution: one thread per 2x2
// block of output pixels, 32 bytes written.
__global__ void __launch_bounds__(256) k_preprocess_s2d(PreArgs a) {
  const int b = blockIdx.y;
  const int hs = a.out_h / 2, ws = a.out_w / 2;
  const int pix = blockIdx.x * 256 + threadIdx.x;
  if (pix >= hs * ws) return;
  const int Y = pix / ws, X = pix - Y * ws;
  const ImageDesc d = a.desc[b];
  float o[16];
#pragma unroll
  for (int s = 0; s < 4; ++s) transform_pixel(a, d, 2 * Y + (s >> 1), 2 * X + (s & 1), o + 3 * s);
#pragma unroll
  for (int e = 12; e < 16; ++e) o[e] = 0.f;
  uint4* dst = reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.out_s2d) + ((int64_t)b * hs * ws + pix) * 16);
  dst[0] = f8_to_bf8(o);
  dst[1] = f8_to_bf8(o + 8);
}

void launch_preprocess(const PreArgs& a, Prec p, hipStream_t s) {
  if (a.out) {
    dim3 grid((a.out_h * a.out_w + 255) / 256, a.B);
    if (p == BF16)
      hipLaunchKernelGGL(k_preprocess<true>, grid, dim3(256), 0, s, a);
    else
      hipLaunchKernelGGL(k_preprocess<false>, grid, dim3(256), 0, s, a);
  }
  if (a.out_s2d) {
    dim3 grid(((a.out_h / 2) * (a.out_w / 2) + 255) / 256, a.B);
    hipLaunchKernelGGL(k_preprocess_s2d, grid, dim3(256), 0, s, a);
  }
}

}  // namespace fs
