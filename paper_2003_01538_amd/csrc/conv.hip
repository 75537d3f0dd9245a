// Convolution as an implicit GEMM on the CDNA4 matrix cores, with the
// epilogue fused: y = relu?(conv(x, w) + bias + residual), stored once.
//
// GEMM view (NHWC activations): rows m = (b, oy, ox) of the output, columns
// n = output channel, reduction k = (ky, kx, ci) with ci fastest.  The
// A tile (BM x BK) is gathered on the fly from the input (zero outside the
// image), the B tile (BN x BK) is a slice of the packed weights
// [Cout][Kp].  Both are staged through two LDS buffers fed from two
// register sets: the global loads of tile k+2 are in flight while the MFMAs
// consume tile k from LDS and tile k+1 waits in registers.  The
// fp32 accumulators are written to LDS after the reduction and read back
// row-contiguous, so bias, residual, ReLU and the rounding store are done
// with 16-byte coalesced accesses.
//
// bf16: v_mfma_f32_16x16x32_bf16, BK = 64.  fp32: v_mfma_f32_16x16x4_f32,
// BK = 32.  Four waves per workgroup in a 2 x 2 arrangement.  One launch
// covers all Z models of a homogeneous group (the models' tensors sit at a
// fixed stride), and the workgroup -> tile mapping keeps the N-tiles of an
// M-tile on one XCD so that the A rows are re-read from that XCD's L2.
#include "common.hpp"
#include "device.hpp"

#include <algorithm>

namespace fs {

template <int P> struct PT;
template <> struct PT<BF16> {
  using T = uint16_t;
  static constexpr int BK = 64, KSTEP = 32;
};
template <> struct PT<F32> {
  using T = float;
  static constexpr int BK = 32, KSTEP = 4;
};

template <int BYTES> struct VecT;
template <> struct VecT<16> { using T = uint4; };
template <> struct VecT<8> { using T = uint2; };

constexpr int NT = 256;          // threads per workgroup (4 waves)
constexpr int ROWB = 128 + 16;   // LDS bytes per tile row: 128 B of data + 16 B pad

constexpr uint32_t OOB = 0x80000000u;  // buffer offset past every tensor: loads return 0
constexpr int RSRC_DW3 = 0x00020000;    // raw (untyped) buffer resource, gfx9 family

__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, RSRC_DW3);
}
template <int BYTES>
__device__ __forceinline__ typename VecT<BYTES>::T buf_load(__amdgpu_buffer_rsrc_t r, uint32_t off) {
  if constexpr (BYTES == 16)
    return __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, 0));
  else
    return __builtin_bit_cast(uint2, __builtin_amdgcn_raw_buffer_load_b64(r, off, 0, 0));
}

// FAST: Cin is a multiple of BK, so every K-tile lies inside one filter tap
// (ky, kx) and a contiguous channel range: the tap is wave-uniform.
template <int P, int BM, int BN, int VEC, bool FAST>
__global__ void __launch_bounds__(NT, BM >= 256 ? 1 : 2) k_conv(ConvArgs a) {
  using T = typename PT<P>::T;
  constexpr int BK = PT<P>::BK, KSTEP = PT<P>::KSTEP;
  constexpr int ES = sizeof(T);
  constexpr int RE = ROWB / ES;              // LDS row stride in elements
  constexpr int TM = BM / 2, TN = BN / 2;    // wave tile
  constexpr int FM = TM / 16, FN = TN / 16;  // 16x16 fragments per wave
  // A loads: VEC elements per vector
  constexpr int AVB = VEC * ES;
  using AV = typename VecT<AVB>::T;
  constexpr int AKV = BK / VEC, ARPP = NT / AKV, AP = BM / ARPP;
  // B loads: 16-byte vectors
  constexpr int BVE = 16 / ES;
  constexpr int BKV = BK / BVE, BRPP = NT / BKV, BP = (BN + BRPP - 1) / BRPP;
  static_assert(BM % ARPP == 0, "A tile rows");
  constexpr int STAGE = (BM + BN) * ROWB;
  constexpr int CS = BM * (BN + 4) * 4;
  constexpr int SMEM = (2 * STAGE > CS) ? 2 * STAGE : CS;
  __shared__ __attribute__((aligned(16))) char smem[SMEM];

  const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
  const int wm = wave >> 1, wn = wave & 1;

  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.Cout + BN - 1) / BN;
  const int tiles = tiles_m * tiles_n;
  const int id = xcd_remap(blockIdx.x, tiles * a.Z);
  const int z = id / tiles, tile = id - z * tiles;
  const int mt = tile / tiles_n, ntile = tile - mt * tiles_n;
  const int m0 = mt * BM, n0 = ntile * BN;

  // Buffer resources: out-of-range offsets (padding taps, rows past M,
  // columns past Cout) read as zero without a branch.
  const __amdgpu_buffer_rsrc_t rx = make_rsrc(reinterpret_cast<const T*>(a.x) + z * a.x_mstride,
                                              (uint32_t)((int64_t)a.B * a.H * a.W * a.Cin * ES));
  const __amdgpu_buffer_rsrc_t rw = make_rsrc(reinterpret_cast<const T*>(a.w) + z * a.w_mstride,
                                              (uint32_t)((int64_t)a.Cout * a.Kp * ES));

  // ---- per-thread A rows: fixed for the whole reduction
  const int aj = tid % AKV;           // which vector of the row
  int a_off[AP], a_iy[AP], a_ix[AP];  // offset of (b, iy0, ix0) + this thread's channels; top-left tap
  const int HoWo = a.Ho * a.Wo;
#pragma unroll
  for (int p = 0; p < AP; ++p) {
    int m = m0 + p * ARPP + tid / AKV;
    if (m < a.M) {
      int b = m / HoWo, r = m - b * HoWo;
      int oy = r / a.Wo, ox = r - oy * a.Wo;
      a_iy[p] = oy * a.stride - a.pad;
      a_ix[p] = ox * a.stride - a.pad;
      a_off[p] = ((b * a.H + a_iy[p]) * a.W + a_ix[p]) * a.Cin + aj * VEC;
    } else {
      a_off[p] = 0;
      a_iy[p] = -(1 << 28);  // never inside the image
      a_ix[p] = 0;
    }
  }
  // reduction position of this thread's vector: k = (ky*kw + kx)*Cin + ci
  int ci, kx, ky;
  {
    int k = aj * VEC;
    int tap = k / a.Cin;
    ci = k - tap * a.Cin;
    ky = tap / a.kw;
    kx = tap - ky * a.kw;
  }
  // ---- B rows
  const int bj = tid % BKV;
  uint32_t b_off[BP];  // byte offset of this thread's weight vector, OOB past Cout
#pragma unroll
  for (int p = 0; p < BP; ++p) {
    int n = n0 + p * BRPP + tid / BKV;
    b_off[p] = (n < a.Cout) ? (uint32_t)((n * a.Kp + bj * BVE) * ES) : OOB;
  }

  // Two register staging sets: the global loads of tile k+2 are in flight
  // while tile k is consumed from LDS and tile k+1 waits in registers.
  AV ra0[AP], ra1[AP];
  uint4 rb0[BP], rb1[BP];
  auto load_tiles = [&](AV* ra, uint4* rb, int kt) {
    int tky, tkx, tci;
    if constexpr (FAST) {  // wave-uniform tap of this K-tile
      const int k0 = kt * BK;
      const int tap = k0 / a.Cin;
      tci = k0 - tap * a.Cin;
      tky = tap / a.kw;
      tkx = tap - tky * a.kw;
    } else {
      tky = ky; tkx = kx; tci = ci - aj * VEC;
    }
    const bool kvalid = tky < a.kh;
    const int tap_off = (tky * a.W + tkx) * a.Cin + tci;
#pragma unroll
    for (int p = 0; p < AP; ++p) {
      const int iy = a_iy[p] + tky, ix = a_ix[p] + tkx;
      const bool ok = kvalid && (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
      ra[p] = buf_load<AVB>(rx, ok ? (uint32_t)((a_off[p] + tap_off) * ES) : OOB);
    }
#pragma unroll
    for (int p = 0; p < BP; ++p)
      rb[p] = buf_load<16>(rw, b_off[p] == OOB ? OOB : b_off[p] + (uint32_t)(kt * BK * ES));
  };
  auto advance_k = [&]() {
    if constexpr (!FAST) {
      ci += BK;
      while (ci >= a.Cin) {
        ci -= a.Cin;
        if (++kx == a.kw) { kx = 0; ++ky; }
      }
    }
  };
  auto store_tiles = [&](int buf, const AV* ra, const uint4* rb) {
    char* As = smem + buf * STAGE;
    char* Bs = As + BM * ROWB;
#pragma unroll
    for (int p = 0; p < AP; ++p)
      *reinterpret_cast<AV*>(As + (p * ARPP + tid / AKV) * ROWB + aj * AVB) = ra[p];
#pragma unroll
    for (int p = 0; p < BP; ++p)
      if (p * BRPP + tid / BKV < BN)
        *reinterpret_cast<uint4*>(Bs + (p * BRPP + tid / BKV) * ROWB + bj * 16) = rb[p];
  };

  floatx4 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j) acc[i][j] = floatx4{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](int buf) {
    const T* As = reinterpret_cast<const T*>(smem + buf * STAGE);
    const T* Bs = reinterpret_cast<const T*>(smem + buf * STAGE + BM * ROWB);
#pragma unroll
    for (int ks = 0; ks < BK / KSTEP; ++ks) {
      if constexpr (P == BF16) {
        bf16x8 af[FM], bfr[FN];
        const int col = ks * KSTEP + (lane >> 4) * 8;
#pragma unroll
        for (int i = 0; i < FM; ++i)
          af[i] = *reinterpret_cast<const bf16x8*>(As + (wm * TM + i * 16 + (lane & 15)) * RE + col);
#pragma unroll
        for (int j = 0; j < FN; ++j)
          bfr[j] = *reinterpret_cast<const bf16x8*>(Bs + (wn * TN + j * 16 + (lane & 15)) * RE + col);
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(af[i], bfr[j], acc[i][j], 0, 0, 0);
      } else {
        float af[FM], bfr[FN];
        const int col = ks * KSTEP + (lane >> 4);
#pragma unroll
        for (int i = 0; i < FM; ++i) af[i] = As[(wm * TM + i * 16 + (lane & 15)) * RE + col];
#pragma unroll
        for (int j = 0; j < FN; ++j) bfr[j] = Bs[(wn * TN + j * 16 + (lane & 15)) * RE + col];
#pragma unroll
        for (int i = 0; i < FM; ++i)
#pragma unroll
          for (int j = 0; j < FN; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_16x16x4f32(af[i], bfr[j], acc[i][j], 0, 0, 0);
      }
    }
  };

  // ---- main loop: two LDS buffers, two register sets (prefetch distance 2)
  const int nk = a.Kp / BK;
  load_tiles(ra0, rb0, 0);
  advance_k();
  if (nk > 1) {
    load_tiles(ra1, rb1, 1);
    advance_k();
  }
  store_tiles(0, ra0, rb0);
  __syncthreads();
  // iteration kt: LDS[kt & 1] holds tile kt, registers set (kt+1) & 1 hold
  // tile kt+1, and set kt & 1 is free for tile kt+2.
  auto iter = [&](int kt, AV* ra_free, uint4* rb_free, const AV* ra_next, const uint4* rb_next) {
    if (kt + 2 < nk) {
      load_tiles(ra_free, rb_free, kt + 2);
      advance_k();
    }
    compute(kt & 1);
    if (kt + 1 < nk) store_tiles((kt + 1) & 1, ra_next, rb_next);
    __syncthreads();
  };
  for (int kt = 0; kt < nk; kt += 2) {
    iter(kt, ra0, rb0, ra1, rb1);
    if (kt + 1 < nk) iter(kt + 1, ra1, rb1, ra0, rb0);
  }

  // ---- epilogue: accumulators -> LDS -> coalesced rows
  float* Cs = reinterpret_cast<float*>(smem);
  constexpr int CSTR = BN + 4;
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int r = 0; r < 4; ++r)
        Cs[(wm * TM + i * 16 + (lane >> 4) * 4 + r) * CSTR + wn * TN + j * 16 + (lane & 15)] = acc[i][j][r];
  __syncthreads();

  const float* __restrict__ bias = a.bias + z * a.b_mstride;
  const T* __restrict__ res = a.res ? reinterpret_cast<const T*>(a.res) + z * a.res_mstride : nullptr;
  T* __restrict__ y = reinterpret_cast<T*>(a.y) + z * a.y_mstride;
  constexpr int CPR = BN / 8;
  for (int idx = tid; idx < BM * CPR; idx += NT) {
    const int row = idx / CPR, c8 = idx - row * CPR;
    const int m = m0 + row, n = n0 + c8 * 8;
    if (m >= a.M || n >= a.Cout) continue;
    float v[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = Cs[row * CSTR + c8 * 8 + e] + bias[n + e];
    const int64_t o = (int64_t)m * a.Cout + n;
    if constexpr (P == BF16) {
      if (res) {
        float r[8];
        bf8_to_f8(*reinterpret_cast<const uint4*>(res + o), r);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += r[e];
      }
      if (a.relu)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
      *reinterpret_cast<uint4*>(y + o) = f8_to_bf8(v);
    } else {
      if (res) {
        float4 r0 = *reinterpret_cast<const float4*>(res + o);
        float4 r1 = *reinterpret_cast<const float4*>(res + o + 4);
        v[0] += r0.x; v[1] += r0.y; v[2] += r0.z; v[3] += r0.w;
        v[4] += r1.x; v[5] += r1.y; v[6] += r1.z; v[7] += r1.w;
      }
      if (a.relu)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
      *reinterpret_cast<float4*>(y + o) = make_float4(v[0], v[1], v[2], v[3]);
      *reinterpret_cast<float4*>(y + o + 4) = make_float4(v[4], v[5], v[6], v[7]);
    }
  }
}

// ------------------------------------------------------------- tile table
static const ConvTile kTilesBF16[] = {
    {128, 128, 8, "bf16_128x128_v8"},
    {128, 64, 8, "bf16_128x64_v8"},
    {64, 64, 8, "bf16_64x64_v8"},
    {128, 64, 4, "bf16_128x64_v4"},
    {64, 64, 4, "bf16_64x64_v4"},
    {256, 64, 8, "bf16_256x64_v8"},
    {128, 128, 8, "bf16dma2_128x128_w4_v8", 2, 4, 2},
    {128, 64, 8, "bf16dma3_128x64_w4_v8", 3, 4, 2},
    {64, 128, 8, "bf16dma3_64x128_w4_v8", 3, 4, 2},
    {64, 64, 8, "bf16dma3_64x64_w4_v8", 3, 4, 2},
    {256, 128, 8, "bf16dma3_256x128_w8_v8", 3, 8, 4},
    {256, 64, 8, "bf16dma3_256x64_w8_v8", 3, 8, 4},
    {128, 64, 8, "bf16dma2_128x64_w4_v8", 2, 4, 2},
    {64, 128, 8, "bf16dma2_64x128_w4_v8", 2, 4, 2},
    {256, 64, 8, "bf16dma2_256x64_w4m4_v8", 2, 4, 4},
    {224, 64, 8, "bf16halo_4x56_n64_v8", 0, 7, 7, 1, 4, 56},
    {128, 128, 8, "bf16hs_128x128_w4_v8", 0, 4, 2, 2},
    {128, 128, 8, "bf16dma1_128x128_w4_v8", 1, 4, 2},
    {128, 64, 8, "bf16dma1_128x64_w4_v8", 1, 4, 2},
    {64, 128, 8, "bf16dma1_64x128_w4_v8", 1, 4, 2},
    {256, 128, 8, "bf16dma2_256x128_w4_v8", 2, 4, 2},
    {256, 128, 8, "bf16dma3_256x128_w4_v8", 3, 4, 2},
    {128, 256, 8, "bf16dma2_128x256_w4_v8", 2, 4, 2},
    {256, 256, 8, "bf16dma2_256x256_w8_v8", 2, 8, 2},
    {128, 128, 8, "bf16dma3_128x128_w4_v8", 3, 4, 2},
    {160, 128, 8, "bf16dma2_160x128_w4m1_v8", 2, 4, 1},
    {96, 128, 8, "bf16dma2_96x128_w4m1_v8", 2, 4, 1},
    {96, 128, 8, "bf16dma1_96x128_w4m1_v8", 1, 4, 1},
    {160, 128, 8, "bf16hr_160x128_w4m1_v8", 0, 4, 1, 3},
    {96, 128, 8, "bf16hr_96x128_w4m1_v8", 0, 4, 1, 3},
};
static const ConvTile kTilesF32[] = {
    {64, 64, 4, "f32_64x64_v4"},
    {64, 32, 4, "f32_64x32_v4"},
};

int conv_num_tiles(Prec p) {
  return p == BF16 ? (int)(sizeof(kTilesBF16) / sizeof(ConvTile))
                   : (int)(sizeof(kTilesF32) / sizeof(ConvTile));
}
const ConvTile& conv_tile(Prec p, int t) { return p == BF16 ? kTilesBF16[t] : kTilesF32[t]; }

bool conv_tile_ok(Prec p, int t, const ConvArgs& a) {
  if (t < 0 || t >= conv_num_tiles(p)) return false;
  const ConvTile& c = conv_tile(p, t);
  if (c.halo == 3) return p == BF16 && conv_hr_ok(a, c.bm);
  if (c.halo == 2) return p == BF16 && conv_hs_ok(a);
  if (c.halo) return p == BF16 && conv_halo_ok(a, c.th, c.tw, c.bn);
  if (conv_tile_direct(c)) return p == BF16 && conv_dma_ok(a);
  if (a.split > 1 || a.x2) return false;  // only the LDS-DMA kernels split K or take a projection
  return a.Cin % c.vec == 0 && a.Kp % CONV_KPAD == 0 && a.Cout % 8 == 0;
}

// Whether tile t is among the layer's automatic choices (see conv_hs_chosen
// for the streamed-weight halo kernel).
bool conv_tile_candidate(Prec p, int t, const ConvArgs& a) {
  if (!conv_tile_ok(p, t, a)) return false;
  return conv_tile(p, t).halo < 2 || conv_hs_chosen(a);
}

// Largest useful tile: prefer tiles that keep >= 2 workgroups per CU busy,
// then the least padding waste, then the larger tile (more reuse per byte).
int conv_pick_tile(Prec p, const ConvArgs& a, int num_cus) {
  int fam = -1;
  for (int t = 0; t < conv_num_tiles(p); ++t)
    if (conv_tile_candidate(p, t, a)) fam = std::max(fam, conv_tile_family(conv_tile(p, t)));
  int best = -1;
  double best_score = -1;
  for (int t = 0; t < conv_num_tiles(p); ++t) {
    if (!conv_tile_candidate(p, t, a) || conv_tile_family(conv_tile(p, t)) != fam) continue;
    const ConvTile& c = conv_tile(p, t);
    const double tm = (a.M + c.bm - 1) / c.bm, tn = (a.Cout + c.bn - 1) / c.bn;
    const double wgs = tm * tn * a.Z;
    const double useful = (double)a.M * a.Cout / (tm * c.bm * tn * c.bn);
    const double fill = wgs >= 2.0 * num_cus ? 1.0 : wgs / (2.0 * num_cus);
    const double reuse = (double)c.bm * c.bn / (c.bm + c.bn) / 64.0;  // 1.0 for 128x128
    const double score = useful * (0.35 + 0.65 * fill) * (0.6 + 0.4 * reuse) * (c.vec == 8 || p == F32 ? 1.0 : 0.9);
    if (score > best_score) { best_score = score; best = t; }
  }
  return best;
}

template <int P, int BM, int BN, int VEC>
static void launch_t(const ConvArgs& a, hipStream_t s) {
  const int tiles = ((a.M + BM - 1) / BM) * ((a.Cout + BN - 1) / BN) * a.Z;
  if (a.Cin % PT<P>::BK == 0)
    hipLaunchKernelGGL((k_conv<P, BM, BN, VEC, true>), dim3(tiles), dim3(NT), 0, s, a);
  else
    hipLaunchKernelGGL((k_conv<P, BM, BN, VEC, false>), dim3(tiles), dim3(NT), 0, s, a);
}

void launch_conv(const ConvArgs& a, Prec p, int tile, hipStream_t s, bool reduce) {
  if (p == BF16 && conv_tile(p, tile).halo == 3) {
    launch_conv_hr(a, conv_tile(p, tile).bm, s);
    return;
  }
  if (p == BF16 && conv_tile(p, tile).halo == 2) {
    launch_conv_hs(a, s);
    return;
  }
  if (p == BF16 && conv_tile(p, tile).halo) {
    const ConvTile& c = conv_tile(p, tile);
    launch_conv_halo(a, c.th, c.tw, c.bn, s);
    return;
  }
  if (p == BF16 && conv_tile_direct(conv_tile(p, tile))) {
    const ConvTile& c = conv_tile(p, tile);
    launch_conv_dma(a, c.bm, c.bn, c.waves, c.wgm, c.dma, s);
    if (a.split > 1 && reduce) launch_conv_splitk_reduce(a, s);
    return;
  }
  if (p == BF16) {
    switch (tile) {
      case 0: launch_t<BF16, 128, 128, 8>(a, s); break;
      case 1: launch_t<BF16, 128, 64, 8>(a, s); break;
      case 2: launch_t<BF16, 64, 64, 8>(a, s); break;
      case 3: launch_t<BF16, 128, 64, 4>(a, s); break;
      case 4: launch_t<BF16, 64, 64, 4>(a, s); break;
      case 5: launch_t<BF16, 256, 64, 8>(a, s); break;
      default: break;
    }
  } else {
    switch (tile) {
      case 0: launch_t<F32, 64, 64, 4>(a, s); break;
      case 1: launch_t<F32, 64, 32, 4>(a, s); break;
      default: break;
    }
  }
}

}  // namespace fs
