// Convolution as an implicit GEMM on the CDNA4 matrix cores, operands fed
// to LDS by direct (LDS-DMA) buffer loads.
//
// Same GEMM view as the register-staged kernel (rows m = (b, oy, ox), columns
// n = output channel, reduction k = (ky, kx, ci) with ci fastest) for layers
// whose 64-wide K-tiles each lie in one filter row (Cin a multiple of 64, or
// kw * Cin a multiple of 64 with Cin dividing 64): the tap is wave-uniform and
// each tile row is one contiguous 128-byte run of input channels/pixels.
//
// Loads: `buffer_load_dwordx4 ... lds` writes lane j's 16 bytes to
// LDS[M0 + 16 j] without touching VGPRs; offsets past the buffer read as
// zero, which supplies the convolution's zero padding and the rows/columns
// past M and N.  A wave instruction fills 8 tile rows (1 KB).  Rows are
// stored unpadded with their eight 16-byte chunks XOR-swizzled by
// swz(row) = (row & 7) ^ ((row >> 3) & 1): an operand read serves 16 lanes
// (16 rows x 16 bytes) per cycle from 64 four-byte banks, and consecutive
// rows alternate between the two 128-byte bank halves, so the 16 rows need
// distinct chunks within each parity class, which (row & 7) alone does not
// give for rows r and r + 8.
//
// Pipeline: STAGES LDS buffers.  Iteration k waits (vmcnt) for its own
// wave's loads of tile k, meets the other waves at one barrier (after which
// tile k is complete in LDS and tile k-1's buffer is free), issues the loads
// of tile k + STAGES - 1, and runs the MFMAs of tile k.
//
// Four or eight waves per workgroup, v_mfma_f32_32x32x16_bf16 (on gfx950
// it sustains ~1.4x the rate of the 16x16x32 form), fp32 accumulators; the
// epilogue (bias, residual, ReLU, bf16 store) works on the accumulators in
// registers, so LDS holds only the operand ring.  One launch covers the Z
// models of a group.
#include "common.hpp"
#include "device.hpp"

namespace fs {

namespace {

typedef __attribute__((address_space(3))) void lds_void;

constexpr int BK = 64;          // bf16 elements per K-tile row (128 bytes)
constexpr int ROW = 128;        // LDS bytes per tile row
constexpr uint32_t OOB = 0x80000000u;

__device__ __forceinline__ int swz(int row) { return (row & 7) ^ ((row >> 3) & 1); }

__device__ __forceinline__ __amdgpu_buffer_rsrc_t rsrc(const void* base, uint32_t bytes) {
  return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes, 0x00020000);
}

// s_waitcnt vmcnt(n) leaving the other counters alone (gfx9 encoding)
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 0xF) | ((N >> 4) << 14) | (0x7 << 4) | (0xF << 8));
}

// Wait until at most `ahead` K-tiles (LPT load instructions each) of this
// wave are still in flight; `ahead` <= A (vmcnt takes an immediate).
template <int A, int LPT>
__device__ __forceinline__ void wait_tiles(int ahead) {
  if constexpr (A <= 0) {
    wait_vmcnt<0>();
  } else {
    if (ahead >= A) wait_vmcnt<A * LPT>();
    else wait_tiles<A - 1, LPT>(ahead);
  }
}

// MFMAs of one 64-wide K-tile for a wave's TM x TN sub-tile (FM x FN blocks of
// 32x32).  32x32x16 operands: lane l supplies row (l & 31), k-group (l >> 5)
// of 8; the weights are the A operand, so block (i, j) accumulates D[n][m].
template <int FM, int FN>
__device__ __forceinline__ void mma_ktile(const char* As, const char* Bs, int row_a, int row_b, int lane,
                                          floatx16 (&acc)[FM][FN]) {
  const int fr = lane & 31, fq = lane >> 5;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh) {  // two halves of the 64-wide K-tile
    bf16x8 af[2][FM], bfr[2][FN];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = (kh * 2 + ks) * 2 + fq;  // logical 16-byte chunk
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int r = row_a + i * 32 + fr;
        af[ks][i] = *reinterpret_cast<const bf16x8*>(As + r * ROW + ((c ^ swz(r)) << 4));
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) {
        const int r = row_b + j * 32 + fr;
        bfr[ks][j] = *reinterpret_cast<const bf16x8*>(Bs + r * ROW + ((c ^ swz(r)) << 4));
      }
    }
#pragma unroll
    for (int ks = 0; ks < 2; ++ks)
#pragma unroll
      for (int i = 0; i < FM; ++i)
#pragma unroll
        for (int j = 0; j < FN; ++j)
          acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[ks][j], af[ks][i], acc[i][j], 0, 0, 0);
  }
}

// Epilogue straight from the accumulators.  The MFMA computes D[n][m]
// (weights as the A operand), so lane l holds pixel m = l & 31 and channels
// 8g + 4q + r (q = l >> 5, r < 4) of each 32x32 block.  One permlane32 swap
// per register pair gives every lane 8 consecutive channels of one pixel:
// lanes 0-31 channels 8g.., lanes 32-63 channels 8(g+1).., for g = 0, 2.
// Bias, residual, ReLU, bf16 rounding and a 16-byte store follow; with a K
// split the raw fp32 sums go to the partial buffer instead.
template <int FM, int FN>
__device__ __forceinline__ void conv_epilogue(const ConvArgs& a, floatx16 (&acc)[FM][FN], int mrow, int ncol,
                                              int z, int sp, int lane) {
  const int fr = lane & 31, fq = lane >> 5;
  const float* __restrict__ bias = a.bias + z * a.b_mstride;
  const uint16_t* __restrict__ res = a.res ? reinterpret_cast<const uint16_t*>(a.res) + z * a.res_mstride : nullptr;
  uint16_t* __restrict__ y = reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = mrow + i * 32 + fr;
#pragma unroll
    for (int j = 0; j < FN; ++j) {
#pragma unroll
      for (int gp = 0; gp < 4; gp += 2) {
        float v[8];
#pragma unroll
        for (int r = 0; r < 4; ++r) {
          const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i][j][gp * 4 + r]),
                                                           __float_as_uint(acc[i][j][(gp + 1) * 4 + r]), false, false);
          v[r] = __uint_as_float(sw[0]);      // channels 8(gp+q) + r
          v[4 + r] = __uint_as_float(sw[1]);  // channels 8(gp+q) + 4 + r
        }
        const int n = ncol + j * 32 + 8 * (gp + fq);
        if (m >= a.M || n >= a.Cout) continue;
        if (a.split > 1) {  // raw partial sums; the reduce kernel finishes
          float4* pp = reinterpret_cast<float4*>(a.partial + (((int64_t)sp * a.Z + z) * a.M + m) * a.Cout + n);
          pp[0] = make_float4(v[0], v[1], v[2], v[3]);
          pp[1] = make_float4(v[4], v[5], v[6], v[7]);
          continue;
        }
        const float4 b0 = *reinterpret_cast<const float4*>(bias + n);
        const float4 b1 = *reinterpret_cast<const float4*>(bias + n + 4);
        v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
        v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
        const int64_t o = (int64_t)m * a.Cout + n;
        if (res) {
          float rr[8];
          bf8_to_f8(*reinterpret_cast<const uint4*>(res + o), rr);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += rr[e];
        }
        if (a.relu)
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = fmaxf(v[e], 0.f);
        *reinterpret_cast<uint4*>(y + o) = f8_to_bf8(v);
      }
    }
  }
}

// Tile of workgroup `bid` among tiles * Z * split, XCD-contiguous.
struct TileCoord {
  int m0, n0, z, sp;
};
template <int BM, int BN>
__device__ __forceinline__ TileCoord tile_coord(const ConvArgs& a, int bid) {
  const int tiles_m = (a.M + BM - 1) / BM, tiles_n = (a.Cout + BN - 1) / BN;
  const int tiles = tiles_m * tiles_n;
  const int id = xcd_remap(bid, tiles * a.Z * a.split);
  const int tile = id % tiles, zs = id / tiles;
  const int mt = tile / tiles_n, nt = tile - mt * tiles_n;
  return TileCoord{mt * BM, nt * BN, zs % a.Z, zs / a.Z};
}

// BM x BN block tile, WGM x WGN waves (wave tile BM/WGM x BN/WGN, multiples
// of 32), v_mfma_f32_32x32x16_bf16.
template <int BM, int BN, int WGM, int WGN, int STAGES>
__global__ void __launch_bounds__(64 * WGM * WGN,
                                  (STAGES * (BM + BN) * 128 > 80 * 1024) ? 1 : 2) k_conv_dma(ConvArgs a) {
  constexpr int NW = WGM * WGN, NTH = 64 * NW;
  constexpr int TM = BM / WGM, TN = BN / WGN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int AP = BM / (8 * NW), BP = BN / (8 * NW);  // DMA instructions per wave per tile
  constexpr int LPT = AP + BP;                             // vmcnt units per tile
  constexpr int STAGE = (BM + BN) * ROW;
  constexpr int SMEM = STAGES * STAGE;
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile");
  static_assert(AP * 8 * NW == BM && BP * 8 * NW == BN, "DMA blocks");
  static_assert(NW % 2 == 0, "the swizzle of a DMA block's rows depends on the wave only");
  __shared__ __attribute__((aligned(1024))) char smem[SMEM];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave / WGN, wn = wave % WGN;

  const TileCoord tc = tile_coord<BM, BN>(a, blockIdx.x);
  const int m0 = tc.m0, n0 = tc.n0, z = tc.z, sp = tc.sp;

  const __amdgpu_buffer_rsrc_t rx = rsrc(reinterpret_cast<const uint16_t*>(a.x) + z * a.x_mstride,
                                         (uint32_t)((int64_t)a.B * a.H * a.W * a.Cin * 2));
  const __amdgpu_buffer_rsrc_t rw = rsrc(reinterpret_cast<const uint16_t*>(a.w) + z * a.w_mstride,
                                         (uint32_t)((int64_t)a.Cout * a.Kp * 2));

  // lane j of a DMA instruction writes LDS row (j >> 3) of its 8-row block
  // (block i * NW + wave, so row bit 3 is the wave's parity), physical chunk
  // (j & 7), which holds logical chunk (j & 7) ^ swz(row)
  const int lr = lane >> 3;
  const int lc = (lane & 7) ^ lr ^ (wave & 1);
  // when Cin < 64 a 64-wide K-tile spans 64 / Cin consecutive pixels of one
  // filter row: this lane's 8 channels belong to pixel kx + dx
  const int dx = (lc * 8) / a.Cin;

  int a_off[AP], a_iy[AP], a_ix[AP];
  const int HoWo = a.Ho * a.Wo;
#pragma unroll
  for (int i = 0; i < AP; ++i) {
    const int m = m0 + (i * NW + wave) * 8 + lr;
    if (m < a.M) {
      const int b = m / HoWo, r = m - b * HoWo;
      const int oy = r / a.Wo, ox = r - oy * a.Wo;
      a_iy[i] = oy * a.stride - a.pad;
      a_ix[i] = ox * a.stride - a.pad;
      a_off[i] = ((b * a.H + a_iy[i]) * a.W + a_ix[i]) * a.Cin + lc * 8;
    } else {
      a_iy[i] = -(1 << 28);
      a_ix[i] = 0;
      a_off[i] = 0;
    }
  }
  uint32_t b_off[BP];
#pragma unroll
  for (int i = 0; i < BP; ++i) {
    const int n = n0 + (i * NW + wave) * 8 + lr;
    b_off[i] = n < a.Cout ? (uint32_t)((n * a.Kp + lc * 8) * 2) : OOB;
  }

  auto issue = [&](int kt, int stage) {
    const int k0 = kt * BK;
    const int tap = k0 / a.Cin;
    const int ci0 = k0 - tap * a.Cin;
    const int ky = tap / a.kw, kx = tap - ky * a.kw;
    const int tap_off = (ky * a.W + kx) * a.Cin + ci0;
    char* base = smem + stage * STAGE;
#pragma unroll
    for (int i = 0; i < AP; ++i) {
      const int iy = a_iy[i] + ky, ix = a_ix[i] + kx + dx;
      const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
      const uint32_t off = ok ? (uint32_t)((a_off[i] + tap_off) * 2) : OOB;
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)(base + (i * NW + wave) * 1024), 16, off, 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < BP; ++i) {
      const uint32_t off = b_off[i] == OOB ? OOB : b_off[i] + (uint32_t)(k0 * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void*)(base + BM * ROW + (i * NW + wave) * 1024), 16,
                                               off, 0, 0, 0);
    }
  };

  floatx16 acc[FM][FN];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;

  auto compute = [&](int stage) {
    const char* As = smem + stage * STAGE;
    mma_ktile<FM, FN>(As, As + BM * ROW, wm * TM, wn * TN, lane, acc);
  };

  // this workgroup's share of the K-tiles (all of them unless split-K)
  const int nk_all = a.Kp / BK;
  const int kb = sp * nk_all / a.split, nk = (sp + 1) * nk_all / a.split - kb;
#pragma unroll
  for (int s = 0; s < STAGES - 1; ++s)
    if (s < nk) issue(kb + s, s);
  for (int kt = 0; kt < nk; ++kt) {
    // tiles issued after kt that may stay in flight
    const int ahead = min(nk - 1, kt + STAGES - 2) - kt;
    wait_tiles<STAGES - 2, LPT>(ahead);
    __builtin_amdgcn_s_barrier();
    if (kt + STAGES - 1 < nk) issue(kb + kt + STAGES - 1, (kt + STAGES - 1) % STAGES);
    compute(kt % STAGES);
  }

  conv_epilogue<FM, FN>(a, acc, m0 + wm * TM, n0 + wn * TN, z, sp, lane);
}

// Split-K completion: partial sums added in split order, then bias,
// residual, ReLU and the bf16 store, 8 channels per thread.
__global__ void __launch_bounds__(256) k_conv_splitk_reduce(ConvArgs a) {
  const int cg = a.Cout / 8;
  const int64_t total = (int64_t)a.Z * a.M * cg;
  const int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  if (i >= total) return;
  const int c8 = (int)(i % cg);
  const int64_t zm = i / cg;
  const int z = (int)(zm / a.M), m = (int)(zm % a.M), n = c8 * 8;
  float v[8];
  const float4* p0 = reinterpret_cast<const float4*>(a.partial + ((int64_t)z * a.M + m) * a.Cout + n);
  float4 q0 = p0[0], q1 = p0[1];
  v[0] = q0.x; v[1] = q0.y; v[2] = q0.z; v[3] = q0.w; v[4] = q1.x; v[5] = q1.y; v[6] = q1.z; v[7] = q1.w;
  for (int sp = 1; sp < a.split; ++sp) {
    const float4* pp =
        reinterpret_cast<const float4*>(a.partial + (((int64_t)sp * a.Z + z) * a.M + m) * a.Cout + n);
    q0 = pp[0]; q1 = pp[1];
    v[0] += q0.x; v[1] += q0.y; v[2] += q0.z; v[3] += q0.w;
    v[4] += q1.x; v[5] += q1.y; v[6] += q1.z; v[7] += q1.w;
  }
  const float* bias = a.bias + z * a.b_mstride + n;
#pragma unroll
  for (int e = 0; e < 8; ++e) v[e] += bias[e];
  const int64_t o = (int64_t)m * a.Cout + n;
  if (a.res) {
    float r[8];
    bf8_to_f8(*reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a.res) + z * a.res_mstride + o), r);
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] += r[e];
  }
  if (a.relu)
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] = fmaxf(v[e], 0.f);
  *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride + o) = f8_to_bf8(v);
}

}  // namespace

void launch_conv_splitk_reduce(const ConvArgs& a, hipStream_t s) {
  const int64_t total = (int64_t)a.Z * a.M * (a.Cout / 8);
  hipLaunchKernelGGL(k_conv_splitk_reduce, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a);
}

size_t conv_partial_floats(const ConvArgs& a) { return a.split > 1 ? (size_t)a.split * a.Z * a.M * a.Cout : 0; }

// K split of a layer: a function of its shape only (never of the tile), so
// every tile of the family still produces identical sums.  Split while the
// layer has fewer than three 64x64 output tiles per CU, keeping >= 8 K-tiles
// per split.
int conv_split(Prec p, const ConvArgs& a, int num_cus) {
  if (p != BF16 || !conv_dma_ok(a)) return 1;
  const int64_t units = (int64_t)((a.M + 63) / 64) * ((a.Cout + 63) / 64) * a.Z;
  const int nk = a.Kp / BK;
  int split = 1;
  while (units * split < 3 * num_cus && split < 4 && nk / (split * 2) >= 8) split *= 2;
  return split;
}

// Every 64-wide K-tile must lie in one filter row and cover whole pixels.
bool conv_dma_ok(const ConvArgs& a) {
  const bool tiles_ok = a.Cin % BK == 0 || (a.Cin % 8 == 0 && BK % a.Cin == 0 && (a.kw * a.Cin) % BK == 0);
  return tiles_ok && a.Kp % BK == 0 && a.K == a.Kp && a.Cout % 8 == 0;
}

void launch_conv_dma(const ConvArgs& a, int bm, int bn, int waves, int wgm, int stages, hipStream_t s) {
  const int tiles = ((a.M + bm - 1) / bm) * ((a.Cout + bn - 1) / bn) * a.Z * a.split;
#define FS_DMA(BMv, BNv, WMv, WNv, Sv)                                                                   \
  if (bm == BMv && bn == BNv && waves == WMv * WNv && stages == Sv && wgm == WMv) {                                    \
    hipLaunchKernelGGL((k_conv_dma<BMv, BNv, WMv, WNv, Sv>), dim3(tiles), dim3(64 * WMv * WNv), 0, s, a); \
    return;                                                                                              \
  }
  FS_DMA(128, 128, 2, 2, 2)
  FS_DMA(128, 64, 2, 2, 3)
  FS_DMA(64, 128, 2, 2, 3)
  FS_DMA(64, 64, 2, 2, 3)
  FS_DMA(256, 128, 4, 2, 3)
  FS_DMA(256, 64, 4, 2, 3)
  FS_DMA(128, 64, 2, 2, 2)
  FS_DMA(64, 128, 2, 2, 2)
  FS_DMA(256, 64, 4, 1, 2)
#undef FS_DMA
}

}  // namespace fs
