// Fully connected layer y[b][n] = relu?(bias[n] + sum_k x[b][k] * w[n][k]) on
// the matrix cores.  At serving batch sizes the layer streams its weights
// once (arithmetic intensity = B FLOP per weight byte), so the kernel is
// built to keep HBM busy rather than to tile for reuse: a workgroup owns 16
// output features, its waves read weight rows straight from global memory
// with 16-byte loads (no LDS staging; each weight is used by exactly one
// wave) and multiply them with 16*FB batch columns per MFMA step.  Large K
// is also split over grid.z (split-K) into an fp32 scratch that a second
// small kernel sums in a fixed order, so results do not depend on
// scheduling.
//
// MFMA operands: A = 16 weight rows (features), B = 16 batch rows, so each
// lane's accumulator holds 4 consecutive features of one image.
//
// Long reductions (K >= 1024) take k_fc_stream instead.  There the
// activations, not the weights, limited the kernel above: every 16-feature
// workgroup reads the whole [B][K] input, twice the weight bytes at B = 32,
// in 64-byte pieces of 16 rows, and a probe of that access mix streams the
// weights at 1.9 TB/s against 6.2 TB/s for the weights alone.  k_fc_stream
// gives a workgroup 64 features (16 per wave), stages each 256-wide K chunk
// of its images' activations in LDS once for its four waves, and has each
// wave load its weight rows for the next chunk into registers while the
// current chunk's MFMAs run.  Each wave runs the whole K range of its split,
// so per output the sum runs over K in order within a split, then over the
// splits in order (k_fc_reduce).
#include "common.hpp"
#include "device.hpp"

#include <algorithm>

namespace fs {

template <int P> struct FcT;
template <> struct FcT<BF16> { using T = uint16_t; static constexpr int KSTEP = 32; };
template <> struct FcT<F32> { using T = float; static constexpr int KSTEP = 4; };

constexpr int FC_UNROLL = 4;

// One workgroup = 16 output features x 16*FB images; its 4 waves take
// interleaved quarters of the K steps and their accumulators are added in
// wave order through LDS.  grid.z = split * Z (split-K over workgroups for
// very long K, finished by k_fc_reduce).
template <int P, int FB>
__global__ void __launch_bounds__(256) k_fc(FcArgs a) {
  using T = typename FcT<P>::T;
  constexpr int KSTEP = FcT<P>::KSTEP;
  __shared__ floatx4 red[3][FB][64];
  const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
  const int n0 = blockIdx.x * 16;
  const int b0 = blockIdx.y * 16 * FB;
  const int model = blockIdx.z / a.split, sp = blockIdx.z - model * a.split;
  const T* __restrict__ x = reinterpret_cast<const T*>(a.x) + model * a.x_mstride;
  const T* __restrict__ w = reinterpret_cast<const T*>(a.w) + model * a.w_mstride;

  // K range of this split, in whole MFMA steps
  const int steps = (a.K + KSTEP - 1) / KSTEP;
  const int per = (steps + a.split - 1) / a.split;
  const int kb = sp * per * KSTEP;
  const int ke = min(a.K, kb + per * KSTEP);

  const int row_n = n0 + (lane & 15);
  const bool n_ok = row_n < a.N;
  constexpr int LE = P == BF16 ? 8 : 1;  // elements per lane per step
  const int koff = (lane >> 4) * LE;
  const T* wrow = w + (int64_t)(n_ok ? row_n : 0) * a.K + koff;
  const T* xrow[FB];
  bool b_ok[FB];
#pragma unroll
  for (int f = 0; f < FB; ++f) {
    int bb = b0 + f * 16 + (lane & 15);
    b_ok[f] = bb < a.B;
    xrow[f] = x + (int64_t)(b_ok[f] ? bb : 0) * a.K + koff;
  }

  floatx4 acc[FB];
#pragma unroll
  for (int f = 0; f < FB; ++f) acc[f] = floatx4{0.f, 0.f, 0.f, 0.f};

  // wave w takes steps w, w+4, ... in groups of FC_UNROLL
  for (int k = kb + wave * KSTEP; k < ke; k += 4 * KSTEP * FC_UNROLL) {
    if constexpr (P == BF16) {
      uint4 wa[FC_UNROLL], xb[FC_UNROLL][FB];
#pragma unroll
      for (int u = 0; u < FC_UNROLL; ++u) {
        const int ku = k + u * 4 * KSTEP;
        const bool kin = ku + koff + LE <= ke;
        wa[u] = (kin && n_ok) ? *reinterpret_cast<const uint4*>(wrow + ku) : uint4{0, 0, 0, 0};
#pragma unroll
        for (int f = 0; f < FB; ++f)
          xb[u][f] = (kin && b_ok[f]) ? *reinterpret_cast<const uint4*>(xrow[f] + ku) : uint4{0, 0, 0, 0};
      }
#pragma unroll
      for (int u = 0; u < FC_UNROLL; ++u)
#pragma unroll
        for (int f = 0; f < FB; ++f)
          acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wa[u]),
                                                           __builtin_bit_cast(bf16x8, xb[u][f]),
                                                           acc[f], 0, 0, 0);
    } else {
      float wa[FC_UNROLL], xb[FC_UNROLL][FB];
#pragma unroll
      for (int u = 0; u < FC_UNROLL; ++u) {
        const int ku = k + u * 4 * KSTEP;
        const bool kin = ku + koff < ke;
        wa[u] = (kin && n_ok) ? wrow[ku] : 0.f;
#pragma unroll
        for (int f = 0; f < FB; ++f) xb[u][f] = (kin && b_ok[f]) ? xrow[f][ku] : 0.f;
      }
#pragma unroll
      for (int u = 0; u < FC_UNROLL; ++u)
#pragma unroll
        for (int f = 0; f < FB; ++f)
          acc[f] = __builtin_amdgcn_mfma_f32_16x16x4f32(wa[u], xb[u][f], acc[f], 0, 0, 0);
    }
  }

  // waves 1..3 hand their sums to wave 0, which adds them in wave order
  if (wave > 0)
#pragma unroll
    for (int f = 0; f < FB; ++f) red[wave - 1][f][lane] = acc[f];
  __syncthreads();
  if (wave > 0) return;
#pragma unroll
  for (int f = 0; f < FB; ++f)
#pragma unroll
    for (int q = 0; q < 3; ++q) acc[f] += red[q][f][lane];

  // acc[f][r] = y[b = b0 + 16f + (lane & 15)][n = n0 + 4 (lane >> 4) + r]
  const float* bias = a.bias + model * a.b_mstride;
#pragma unroll
  for (int f = 0; f < FB; ++f) {
    const int bb = b0 + f * 16 + (lane & 15);
    if (bb >= a.B) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int n = n0 + (lane >> 4) * 4 + r;
      if (n >= a.N) continue;
      if (a.split > 1) {
        a.partial[(((int64_t)sp * a.Z + model) * a.B + bb) * a.N + n] = acc[f][r];
      } else {
        float v = acc[f][r] + bias[n];
        if (a.relu) v = v > 0.f ? v : 0.f;
        const int64_t o = (int64_t)bb * a.N + n;
        if (a.out_f32 || P == F32)
          (reinterpret_cast<float*>(a.y) + model * a.y_mstride)[o] = v;
        else
          (reinterpret_cast<uint16_t*>(a.y) + model * a.y_mstride)[o] = f2bf(v);
      }
    }
  }
}

constexpr int FCS_KC = 256;              // K elements per staged chunk
constexpr int FCS_PITCH = FCS_KC + 8;    // LDS row pitch (elements): 16-byte reads of 16 rows hit distinct banks

// Whether the weight-streaming kernel takes the layer (shape only).
static bool fc_stream_ok(Prec p, int K) { return p == BF16 && K >= 1024 && K % 32 == 0; }

// 64 output features x 16*FB images per workgroup, grid.z = split * Z.
template <int FB>
__global__ void __launch_bounds__(256) k_fc_stream(FcArgs a) {
  __shared__ __attribute__((aligned(16))) uint16_t xs[2][16 * FB][FCS_PITCH];
  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int n0 = blockIdx.x * 64 + wave * 16;
  const int b0 = blockIdx.y * 16 * FB;
  const int model = blockIdx.z / a.split, sp = blockIdx.z - model * a.split;
  const uint16_t* __restrict__ x = reinterpret_cast<const uint16_t*>(a.x) + model * a.x_mstride;
  const uint16_t* __restrict__ w = reinterpret_cast<const uint16_t*>(a.w) + model * a.w_mstride;

  // this split's K range, in whole 32-wide steps (K is a multiple of 32)
  const int steps = a.K / 32;
  const int per = (steps + a.split - 1) / a.split;
  const int kb = min(a.K, sp * per * 32), ke = min(a.K, kb + per * 32);
  const int nchunks = (ke - kb + FCS_KC - 1) / FCS_KC;

  const int row_n = n0 + (lane & 15);
  const bool n_ok = row_n < a.N;
  const uint16_t* wrow = w + (int64_t)(n_ok ? row_n : 0) * a.K + (lane >> 4) * 8;

  // the chunk's activations: (16 FB rows) x (32 pieces of 16 bytes), 2 FB
  // pieces per thread, 32 consecutive threads per row
  constexpr int XP = 2 * FB;
  auto load_x = [&](int k0, uint4 (&v)[XP]) {
#pragma unroll
    for (int i = 0; i < XP; ++i) {
      const int pc = tid + i * 256, r = pc >> 5, c = pc & 31;
      const int bb = b0 + r, k = k0 + c * 8;
      v[i] = (bb < a.B && k < ke) ? *reinterpret_cast<const uint4*>(x + (int64_t)bb * a.K + k) : uint4{0, 0, 0, 0};
    }
  };
  auto store_x = [&](int buf, const uint4 (&v)[XP]) {
#pragma unroll
    for (int i = 0; i < XP; ++i) {
      const int pc = tid + i * 256, r = pc >> 5, c = pc & 31;
      *reinterpret_cast<uint4*>(&xs[buf][r][c * 8]) = v[i];
    }
  };
  // this lane's weight pieces of the chunk's eight 32-wide steps
  auto load_w = [&](int k0, uint4 (&v)[8]) {
#pragma unroll
    for (int s = 0; s < 8; ++s) {
      const int k = k0 + s * 32;
      v[s] = (n_ok && k < ke) ? *reinterpret_cast<const uint4*>(wrow + k) : uint4{0, 0, 0, 0};
    }
  };

  floatx4 acc[FB];
#pragma unroll
  for (int f = 0; f < FB; ++f) acc[f] = floatx4{0.f, 0.f, 0.f, 0.f};

  uint4 wc[8], wn[8], xn[XP];
  if (nchunks > 0) {
    load_w(kb, wc);
    load_x(kb, xn);
    store_x(0, xn);
  }
  __syncthreads();
  for (int c = 0; c < nchunks; ++c) {
    const int k0 = kb + c * FCS_KC;
    const bool more = c + 1 < nchunks;
    if (more) {  // next chunk in flight during this one's MFMAs
      load_w(k0 + FCS_KC, wn);
      load_x(k0 + FCS_KC, xn);
    }
    const int buf = c & 1;
#pragma unroll
    for (int s = 0; s < 8; ++s)
#pragma unroll
      for (int f = 0; f < FB; ++f) {
        const uint4 xb = *reinterpret_cast<const uint4*>(&xs[buf][f * 16 + (lane & 15)][s * 32 + (lane >> 4) * 8]);
        acc[f] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wc[s]),
                                                         __builtin_bit_cast(bf16x8, xb), acc[f], 0, 0, 0);
      }
    if (more) {
      store_x(buf ^ 1, xn);  // every wave finished reading that buffer before the last barrier
#pragma unroll
      for (int s = 0; s < 8; ++s) wc[s] = wn[s];
    }
    __syncthreads();
  }

  // acc[f][r] = y[b = b0 + 16f + (lane & 15)][n = n0 + 4 (lane >> 4) + r]
  const float* bias = a.bias + model * a.b_mstride;
#pragma unroll
  for (int f = 0; f < FB; ++f) {
    const int bb = b0 + f * 16 + (lane & 15);
    if (bb >= a.B) continue;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
      const int n = n0 + (lane >> 4) * 4 + r;
      if (n >= a.N) continue;
      if (a.split > 1) {
        a.partial[(((int64_t)sp * a.Z + model) * a.B + bb) * a.N + n] = acc[f][r];
      } else {
        float v = acc[f][r] + bias[n];
        if (a.relu) v = v > 0.f ? v : 0.f;
        const int64_t o = (int64_t)bb * a.N + n;
        if (a.out_f32)
          (reinterpret_cast<float*>(a.y) + model * a.y_mstride)[o] = v;
        else
          (reinterpret_cast<uint16_t*>(a.y) + model * a.y_mstride)[o] = f2bf(v);
      }
    }
  }
}

// Sum of the split-K partials in split order, then bias, ReLU and the store.
__global__ void __launch_bounds__(256) k_fc_reduce(FcArgs a, int out_bf16) {
  const int64_t total = (int64_t)a.Z * a.B * a.N;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int n = (int)(i % a.N);
  const int64_t t = i / a.N;
  const int bb = (int)(t % a.B), model = (int)(t / a.B);
  float v = 0.f;
  for (int sp = 0; sp < a.split; ++sp)
    v += a.partial[(((int64_t)sp * a.Z + model) * a.B + bb) * a.N + n];
  v += a.bias[model * a.b_mstride + n];
  if (a.relu) v = v > 0.f ? v : 0.f;
  const int64_t o = (int64_t)bb * a.N + n;
  if (out_bf16)
    (reinterpret_cast<uint16_t*>(a.y) + model * a.y_mstride)[o] = f2bf(v);
  else
    (reinterpret_cast<float*>(a.y) + model * a.y_mstride)[o] = v;
}

static int fc_fb(int B) { return B > 32 ? 4 : (B > 16 ? 2 : 1); }

int fc_pick_split(Prec p, int B, int K, int N, int Z, int num_cus) {
  const int fb = fc_fb(B);
  if (fc_stream_ok(p, K)) {
    // about four workgroups per CU, each split at least two chunks long
    const int wgs = ((N + 63) / 64) * ((B + 16 * fb - 1) / (16 * fb)) * Z;
    const int max_split = std::max(1, K / (2 * FCS_KC));
    const int split = (4 * num_cus + wgs - 1) / wgs;
    return std::max(1, std::min(split, std::min(max_split, 32)));
  }
  const int wgs = ((N + 15) / 16) * ((B + 16 * fb - 1) / (16 * fb)) * Z;
  const int kstep = p == BF16 ? 32 : 4;
  // each split keeps >= 4 unrolled step groups for every one of the 4 waves
  const int max_split = std::max(1, K / (kstep * FC_UNROLL * 4 * 4));
  int split = (2 * num_cus + wgs - 1) / wgs;
  return std::max(1, std::min(split, std::min(max_split, 32)));
}

size_t fc_partial_floats(int B, int N, int split, int Z) {
  return split > 1 ? (size_t)split * Z * B * N : 0;
}

int fc_launches(int split) { return split > 1 ? 2 : 1; }

template <int P, int FB>
static void launch_fc_t(const FcArgs& a, hipStream_t s) {
  dim3 grid((a.N + 15) / 16, (a.B + 16 * FB - 1) / (16 * FB), a.split * a.Z);
  hipLaunchKernelGGL((k_fc<P, FB>), grid, dim3(256), 0, s, a);
}

void launch_fc(const FcArgs& a, Prec p, hipStream_t s) {
  const int fb = fc_fb(a.B);
  if (fc_stream_ok(p, a.K)) {
    dim3 grid((a.N + 63) / 64, (a.B + 16 * fb - 1) / (16 * fb), a.split * a.Z);
    if (fb == 4) hipLaunchKernelGGL(k_fc_stream<4>, grid, dim3(256), 0, s, a);
    else if (fb == 2) hipLaunchKernelGGL(k_fc_stream<2>, grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL(k_fc_stream<1>, grid, dim3(256), 0, s, a);
  } else if (p == BF16) {
    if (fb == 4) launch_fc_t<BF16, 4>(a, s);
    else if (fb == 2) launch_fc_t<BF16, 2>(a, s);
    else launch_fc_t<BF16, 1>(a, s);
  } else {
    if (fb == 4) launch_fc_t<F32, 4>(a, s);
    else if (fb == 2) launch_fc_t<F32, 2>(a, s);
    else launch_fc_t<F32, 1>(a, s);
  }
  if (a.split > 1) {
    const int64_t total = (int64_t)a.Z * a.B * a.N;
    const int out_bf16 = (p == BF16 && !a.out_f32) ? 1 : 0;
    hipLaunchKernelGGL(k_fc_reduce, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a, out_bf16);
  }
}

}  // namespace fs
