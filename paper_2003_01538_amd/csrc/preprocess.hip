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
// One thread per output pixel (per 2x2 block in the space-to-depth layout),
// 256 consecutive ones of one image per workgroup: the stores are fully
// coalesced and the four taps are gathered through the cache.  At 224x224
// the kernel is bound by its vector instructions rather than by HBM (a wave
// instruction holds a 16-lane SIMD for four cycles), so the per-pixel
// arithmetic is kept short: tap positions from float reciprocals where that
// is exact, each row's and column's taps computed once per block, and the
// normalisation as one fused multiply-add and one multiply.  Ragged batches
// need no host work: each image's size comes from its device-side
// descriptor.
#include "common.hpp"
#include "device.hpp"

namespace fs {

// Source taps of output coordinate o along one axis of `in` input and
// `out` output samples: s = ((2o + 1) in - out) / (2 out), clamped at 0,
// lower tap i0 = floor(s), upper tap i1 = min(i0 + 1, in - 1), weight of the
// upper tap l.  The numerator n and the denominator 2 out are exact
// integers.  With n + 1 < 2^22 (`fast`, checked per image) the quotient
// comes from a float reciprocal: n + 0.5 is exact, the product carries a
// relative error below 2^-23, and (n + 0.5) / d lies at least 0.5 / d from
// an integer, so truncating it gives floor(n / d) exactly; otherwise an
// integer division.  The fraction is the exact remainder times 1/d (within
// an ulp of the rounded quotient).
struct Tap {
  int i0, i1;
  float l;
};
__device__ __forceinline__ Tap source_tap(int o, int in, int out, bool fast, float inv_d) {
  const int d = 2 * out;
  const int n = (2 * o + 1) * in - out;
  Tap t{0, 0, 0.f};
  if (n > 0) {
    t.i0 = fast ? (int)(((float)n + 0.5f) * inv_d) : n / d;
    t.l = (float)(n - t.i0 * d) * inv_d;
  }
  t.i0 = min(t.i0, in - 1);
  t.i1 = min(t.i0 + 1, in - 1);
  return t;
}

// Transformed channels 0..2 of the output pixel with row taps ty and column
// taps tx of image d: bilinear blend of the four taps on the 0..255 values,
// then (v/255 - mean) / std as one fused multiply-add and one multiply.
__device__ __forceinline__ void transform_pixel(const PreArgs& a, const uint8_t* img, int64_t row_stride,
                                                const Tap& ty, const Tap& tx, float* o) {
  const uint8_t* r0 = img + (int64_t)ty.i0 * row_stride;
  const uint8_t* r1 = img + (int64_t)ty.i1 * row_stride;
  const float hy = 1.0f - ty.l, hx = 1.0f - tx.l;
#pragma unroll
  for (int c = 0; c < 3; ++c) {
    float v00 = r0[tx.i0 * 3 + c], v01 = r0[tx.i1 * 3 + c];
    float v10 = r1[tx.i0 * 3 + c], v11 = r1[tx.i1 * 3 + c];
    float v = hy * (hx * v00 + tx.l * v01) + ty.l * (hx * v10 + tx.l * v11);
    o[c] = __builtin_fmaf(v, 1.0f / 255.0f, -a.mean[c]) * a.inv_std[c];
  }
}

// Per-image constants of the tap computation (uniform over a workgroup).
struct ImageTaps {
  const uint8_t* img;
  int64_t row_stride;
  int h, w;
  bool fast_y, fast_x;
  float inv_dy, inv_dx;
};
__device__ __forceinline__ ImageTaps image_taps(const PreArgs& a, const ImageDesc& d) {
  ImageTaps t;
  t.img = a.pixels + d.offset;
  t.row_stride = d.row_stride;
  t.h = d.h;
  t.w = d.w;
  t.fast_y = (int64_t)2 * a.out_h * d.h < (1 << 22);
  t.fast_x = (int64_t)2 * a.out_w * d.w < (1 << 22);
  t.inv_dy = 1.0f / (float)(2 * a.out_h);
  t.inv_dx = 1.0f / (float)(2 * a.out_w);
  return t;
}

template <bool BF16>
__global__ void __launch_bounds__(256) k_preprocess(PreArgs a) {
  const int b = blockIdx.y;
  const int pix = blockIdx.x * 256 + threadIdx.x;
  if (pix >= a.out_h * a.out_w) return;
  const int oy = pix / a.out_w, ox = pix - oy * a.out_w;
  const ImageTaps it = image_taps(a, a.desc[b]);
  float o[4];
  if (it.h == a.out_h && it.w == a.out_w) {  // same size: the pixel itself, normalised
    const uint8_t* px = it.img + (int64_t)oy * it.row_stride + 3 * ox;
#pragma unroll
    for (int c = 0; c < 3; ++c) o[c] = __builtin_fmaf((float)px[c], 1.0f / 255.0f, -a.mean[c]) * a.inv_std[c];
  } else {
    transform_pixel(a, it.img, it.row_stride, source_tap(oy, it.h, a.out_h, it.fast_y, it.inv_dy),
                    source_tap(ox, it.w, a.out_w, it.fast_x, it.inv_dx), o);
  }
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
  const ImageTaps it = image_taps(a, a.desc[b]);
  float o[16];
  if (it.h == a.out_h && it.w == a.out_w) {
    // same size (uniform over the workgroup): every tap is the pixel itself
    // with weight 1 (the blend returns it exactly), so only the
    // normalisation remains
    const uint8_t* r0 = it.img + (int64_t)(2 * Y) * it.row_stride + 6 * X;
    const uint8_t* r1 = r0 + it.row_stride;
#pragma unroll
    for (int s = 0; s < 4; ++s)
#pragma unroll
      for (int c = 0; c < 3; ++c) {
        const float v = (s < 2 ? r0 : r1)[(s & 1) * 3 + c];
        o[3 * s + c] = __builtin_fmaf(v, 1.0f / 255.0f, -a.mean[c]) * a.inv_std[c];
      }
#pragma unroll
    for (int e = 12; e < 16; ++e) o[e] = 0.f;
    uint4* dst = reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.out_s2d) + ((int64_t)b * hs * ws + pix) * 16);
    dst[0] = f8_to_bf8(o);
    dst[1] = f8_to_bf8(o + 8);
    return;
  }
  // the two rows' and the two columns' taps, each shared by two pixels
  const Tap ty[2] = {source_tap(2 * Y, it.h, a.out_h, it.fast_y, it.inv_dy),
                     source_tap(2 * Y + 1, it.h, a.out_h, it.fast_y, it.inv_dy)};
  const Tap tx[2] = {source_tap(2 * X, it.w, a.out_w, it.fast_x, it.inv_dx),
                     source_tap(2 * X + 1, it.w, a.out_w, it.fast_x, it.inv_dx)};
#pragma unroll
  for (int s = 0; s < 4; ++s) transform_pixel(a, it.img, it.row_stride, ty[s >> 1], tx[s & 1], o + 3 * s);
#pragma unroll
  for (int e = 12; e < 16; ++e) o[e] = 0.f;
  uint4* dst = reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.out_s2d) + ((int64_t)b * hs * ws + pix) * 16);
  dst[0] = f8_to_bf8(o);
  dst[1] = f8_to_bf8(o + 8);
}

void launch_preprocess(const PreArgs& args, Prec p, hipStream_t s) {
  PreArgs a = args;
  for (int c = 0; c < 3; ++c) a.inv_std[c] = 1.0f / a.std_[c];
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
