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
#include "lds_dma.hpp"

#include <algorithm>
#include <cstring>

namespace fs {

namespace {

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

// Operand fragments of half kh (k16 steps 2kh, 2kh+1) of a 64-wide K-tile.
// ra[i] / rb[j]: the LDS row this lane supplies for A block i / B block j.
// 32x32x16 operands: lane l supplies row (l & 31) of its block, k-group
// (l >> 5) of 8.
template <int FM, int FN>
__device__ __forceinline__ void frags_half(const char* As, const char* Bs, const int (&ra)[FM], const int (&rb)[FN],
                                           int lane, int kh, bf16x8 (&af)[2][FM], bf16x8 (&bf)[2][FN]) {
  const int fq = lane >> 5;
#pragma unroll
  for (int ks = 0; ks < 2; ++ks) {
    const int c = (kh * 2 + ks) * 2 + fq;  // logical 16-byte chunk
#pragma unroll
    for (int i = 0; i < FM; ++i) af[ks][i] = *reinterpret_cast<const bf16x8*>(As + ra[i] * ROW + ((c ^ swz(ra[i])) << 4));
#pragma unroll
    for (int j = 0; j < FN; ++j) bf[ks][j] = *reinterpret_cast<const bf16x8*>(Bs + rb[j] * ROW + ((c ^ swz(rb[j])) << 4));
  }
}

// MFMAs of one half K-tile; the weights are the A operand, so block (i, j)
// accumulates D[n][m].
template <int FM, int FN>
__device__ __forceinline__ void mma_half(const bf16x8 (&af)[2][FM], const bf16x8 (&bf)[2][FN], floatx16 (&acc)[FM][FN]) {
#pragma unroll
  for (int ks = 0; ks < 2; ++ks)
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bf[ks][j], af[ks][i], acc[i][j], 0, 0, 0);
}

// The same with the A rows' swizzles given (sa[i] instead of swz(ra[i])).
template <int FM, int FN>
__device__ __forceinline__ void mma_ktile_rows_sw(const char* As, const char* Bs, const int (&ra)[FM],
                                                  const int (&sa)[FM], const int (&rb)[FN], int lane,
                                                  floatx16 (&acc)[FM][FN]) {
  const int fq = lane >> 5;
#pragma unroll
  for (int kh = 0; kh < 2; ++kh) {
    bf16x8 af[2][FM], bfr[2][FN];
#pragma unroll
    for (int ks = 0; ks < 2; ++ks) {
      const int c = (kh * 2 + ks) * 2 + fq;
#pragma unroll
      for (int i = 0; i < FM; ++i) af[ks][i] = *reinterpret_cast<const bf16x8*>(As + ra[i] * ROW + ((c ^ sa[i]) << 4));
#pragma unroll
      for (int j = 0; j < FN; ++j) bfr[ks][j] = *reinterpret_cast<const bf16x8*>(Bs + rb[j] * ROW + ((c ^ swz(rb[j])) << 4));
    }
    mma_half<FM, FN>(af, bfr, acc);
  }
}

// MFMAs of one 64-wide K-tile for a wave's FM x FN blocks of 32x32; per
// accumulator the k16 steps run 0, 1, 2, 3.
template <int FM, int FN>
__device__ __forceinline__ void mma_ktile_rows(const char* As, const char* Bs, const int (&ra)[FM],
                                               const int (&rb)[FN], int lane, floatx16 (&acc)[FM][FN]) {
#pragma unroll
  for (int kh = 0; kh < 2; ++kh) {
    bf16x8 af[2][FM], bfr[2][FN];
    frags_half<FM, FN>(As, Bs, ra, rb, lane, kh, af, bfr);
    mma_half<FM, FN>(af, bfr, acc);
  }
}

// The same for a wave sub-tile of consecutive rows row_a.., row_b...
template <int FM, int FN>
__device__ __forceinline__ void mma_ktile(const char* As, const char* Bs, int row_a, int row_b, int lane,
                                          floatx16 (&acc)[FM][FN]) {
  const int fr = lane & 31;
  int ra[FM], rb[FN];
#pragma unroll
  for (int i = 0; i < FM; ++i) ra[i] = row_a + i * 32 + fr;
#pragma unroll
  for (int j = 0; j < FN; ++j) rb[j] = row_b + j * 32 + fr;
  mma_ktile_rows<FM, FN>(As, Bs, ra, rb, lane, acc);
}

// Epilogue straight from the accumulators.  The MFMA computes D[n][m]
// (weights as the A operand), so lane l holds pixel m = l & 31 and channels
// 8g + 4q + r (q = l >> 5, r < 4) of each 32x32 block.  One permlane32 swap
// per register pair gives every lane 8 consecutive channels of one pixel:
// lanes 0-31 channels 8g.., lanes 32-63 channels 8(g+1).., for g = 0, 2.
// Bias, residual, ReLU, bf16 rounding and a 16-byte store follow; with a K
// split the raw fp32 sums go to the partial buffer instead.
// mg[i]: the output row m (pixel) this lane holds in block i, or -1.
// PRE: the residual of this lane's outputs is already in registers, rpre
// ([i][j][gp / 2], as loaded by load_residual); otherwise rpre is unused.
// BP: the bias of this lane's channels is already in registers, bpre
// ([j][gp / 2]); otherwise it is read here and bpre is unused.
template <int FM, int FN, bool PRE = false, bool BP = false>
__device__ __forceinline__ void conv_epilogue_m(const ConvArgs& a, floatx16 (&acc)[FM][FN], const int (&mg)[FM],
                                                int ncol, int z, int sp, int lane, const uint4 (&rpre)[FM][FN][2],
                                                const float (&bpre)[FN][2][8]) {
  const int fq = lane >> 5;
  const float* __restrict__ bias = a.bias + z * a.b_mstride;
  const uint16_t* __restrict__ res = a.res ? reinterpret_cast<const uint16_t*>(a.res) + z * a.res_mstride : nullptr;
  uint16_t* __restrict__ y = reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = mg[i];
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
        if (m < 0 || m >= a.M || n >= a.Cout) continue;
        if (a.split > 1) {  // raw partial sums; the reduce kernel finishes
          float4* pp = reinterpret_cast<float4*>(a.partial + (((int64_t)sp * a.Z + z) * a.M + m) * a.Cout + n);
          pp[0] = make_float4(v[0], v[1], v[2], v[3]);
          pp[1] = make_float4(v[4], v[5], v[6], v[7]);
          continue;
        }
        if (BP) {
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += bpre[j][gp >> 1][e];
        } else {
          const float4 b0 = *reinterpret_cast<const float4*>(bias + n);
          const float4 b1 = *reinterpret_cast<const float4*>(bias + n + 4);
          v[0] += b0.x; v[1] += b0.y; v[2] += b0.z; v[3] += b0.w;
          v[4] += b1.x; v[5] += b1.y; v[6] += b1.z; v[7] += b1.w;
        }
        const int64_t o = (int64_t)m * a.Cout + n;
        if (PRE) {
          float rr[8];
          bf8_to_f8(rpre[i][j][gp >> 1], rr);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += rr[e];
        } else if (res) {
          float rr[8];
          bf8_to_f8(*reinterpret_cast<const uint4*>(res + o), rr);
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += rr[e];
        }
        if (a.relu)
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
        *reinterpret_cast<uint4*>(y + o) = f8_to_bf8(v);
      }
    }
  }
}

template <int FM, int FN, bool PRE, bool BP>
__device__ __forceinline__ void conv_epilogue(const ConvArgs& a, floatx16 (&acc)[FM][FN], int mrow, int ncol,
                                              int z, int sp, int lane, const uint4 (&rpre)[FM][FN][2],
                                              const float (&bpre)[FN][2][8]) {
  int mg[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) mg[i] = mrow + i * 32 + (lane & 31);
  conv_epilogue_m<FM, FN, PRE, BP>(a, acc, mg, ncol, z, sp, lane, rpre, bpre);
}

// The bias of the channels this lane stores in conv_epilogue_m (ncol + 32 j
// + 8 (gp + q) .. + 7 for gp = 0, 2), loaded into registers; channels past
// Cout (never stored) read the last eight.
template <int FN>
__device__ __forceinline__ void load_bias(const ConvArgs& a, int ncol, int z, int lane, float (&bp)[FN][2][8]) {
  const float* __restrict__ bias = a.bias + z * a.b_mstride;
  const int fq = lane >> 5;
#pragma unroll
  for (int j = 0; j < FN; ++j)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int n = min(ncol + j * 32 + 8 * (2 * h + fq), a.Cout - 8);
      const float4 b0 = *reinterpret_cast<const float4*>(bias + n);
      const float4 b1 = *reinterpret_cast<const float4*>(bias + n + 4);
      bp[j][h][0] = b0.x; bp[j][h][1] = b0.y; bp[j][h][2] = b0.z; bp[j][h][3] = b0.w;
      bp[j][h][4] = b1.x; bp[j][h][5] = b1.y; bp[j][h][6] = b1.z; bp[j][h][7] = b1.w;
    }
}

// The residual of the outputs this lane stores in conv_epilogue_m (pixel
// mrow + 32 i + (lane & 31), channels ncol + 32 j + 8 (gp + q) .. + 7),
// loaded into registers; past M or Cout the buffer reads zeros, which the
// epilogue never stores.
template <int FM, int FN>
__device__ __forceinline__ void load_residual(const ConvArgs& a, int mrow, int ncol, int z, int lane,
                                              uint4 (&rp)[FM][FN][2]) {
  const __amdgpu_buffer_rsrc_t rr =
      rsrc(reinterpret_cast<const uint16_t*>(a.res) + z * a.res_mstride, (uint32_t)((int64_t)a.M * a.Cout * 2));
  const int fq = lane >> 5;
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = mrow + i * 32 + (lane & 31);
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int n = ncol + j * 32 + 8 * (2 * h + fq);
        const uint32_t off = m < a.M && n < a.Cout ? (uint32_t)(((int64_t)m * a.Cout + n) * 2) : OOB;
        rp[i][j][h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0));
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
// PRE: the layer has a residual and does not split K; its residual is
// loaded into registers before the first operand loads, so the fetch
// overlaps theirs and the MFMAs instead of following them in the epilogue
// (the memory-bound 1x1 convolutions with a residual wait on nothing else).
// BREG (one row of waves, each owning 32 channels, two stages): no wave
// reads another wave's weights, so the weight operand skips LDS: each wave
// loads its fragments for the next K-tile straight into registers from the
// fragment-ordered copy a.wf (one 1 KB load per k16 step) while the current
// K-tile's MFMAs run.  The operand values and the MFMA order are those of
// the LDS path, so the sums are bit-identical.
template <int BM, int BN, int WGM, int WGN, int STAGES, bool PRE, bool BREG>
__global__ void __launch_bounds__(64 * WGM * WGN, STAGES == 1 ? (PRE ? 3 : 4)
                                                  : (STAGES * (BM + BN) * 128 > 80 * 1024) ? 1 : 2) k_conv_dma(ConvArgs a) {
  constexpr int NW = WGM * WGN;
  constexpr int TM = BM / WGM, TN = BN / WGN;
  constexpr int FM = TM / 32, FN = TN / 32;
  constexpr int AP = BM / (8 * NW), BP = BN / (8 * NW);  // DMA instructions per wave per tile
  constexpr int LPT = AP + BP;                             // vmcnt units per tile
  constexpr int STAGE = (BREG ? BM : BM + BN) * ROW;
  constexpr int SMEM = STAGES * STAGE;
  static_assert(TM % 32 == 0 && TN % 32 == 0, "wave tile");
  static_assert(AP * 8 * NW == BM && BP * 8 * NW == BN, "DMA blocks");
  static_assert(NW % 2 == 0, "the swizzle of a DMA block's rows depends on the wave only");
  static_assert(!BREG || (WGM == 1 && FN == 1 && STAGES == 2), "register weights: one row of waves, two stages");
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
  // the projection shortcut's input (an empty resource without one)
  const __amdgpu_buffer_rsrc_t rx2 =
      rsrc(a.x2 ? reinterpret_cast<const uint16_t*>(a.x2) + z * a.x2_mstride : reinterpret_cast<const uint16_t*>(a.x),
           a.x2 ? (uint32_t)((int64_t)a.B * a.H2 * a.W2 * a.Cin2 * 2) : 0u);

  // lane j of a DMA instruction writes LDS row (j >> 3) of its 8-row block
  // (block i * NW + wave, so row bit 3 is the wave's parity), physical chunk
  // (j & 7), which holds logical chunk (j & 7) ^ swz(row)
  const int lr = lane >> 3;
  const int lc = (lane & 7) ^ lr ^ (wave & 1);
  // when Cin < 64 a 64-wide K-tile spans 64 / Cin consecutive pixels of one
  // filter row: this lane's 8 channels belong to pixel kx + dx
  const int dx = (lc * 8) / a.Cin;

  int a_off[AP], a_iy[AP], a_ix[AP];
  uint32_t a2_off[AP];  // projection shortcut: byte offset of (b, oy*s2, ox*s2) + this lane's channels
  const int HoWo = a.Ho * a.Wo;
  // quotients from float reciprocals (fdiv_small) where every dividend is
  // below 2^22, integer division otherwise
  const bool small_m = a.M < (1 << 22);
  const float inv_howo = 1.0f / (float)HoWo, inv_wo = 1.0f / (float)a.Wo;
#pragma unroll
  for (int i = 0; i < AP; ++i) {
    const int m = m0 + (i * NW + wave) * 8 + lr;
    if (m < a.M) {
      const int b = small_m ? fdiv_small(m, inv_howo) : m / HoWo, r = m - b * HoWo;
      const int oy = small_m ? fdiv_small(r, inv_wo) : r / a.Wo, ox = r - oy * a.Wo;
      a_iy[i] = oy * a.stride - a.pad;
      a_ix[i] = ox * a.stride - a.pad;
      a_off[i] = ((b * a.H + a_iy[i]) * a.W + a_ix[i]) * a.Cin + lc * 8;
      a2_off[i] = (uint32_t)((((int64_t)b * a.H2 + oy * a.stride2) * a.W2 + ox * a.stride2) * a.Cin2 + lc * 8) * 2;
    } else {
      a_iy[i] = -(1 << 28);
      a_ix[i] = 0;
      a_off[i] = 0;
      a2_off[i] = OOB;
    }
  }
  uint32_t b_off[BP];
#pragma unroll
  for (int i = 0; i < BP; ++i) {
    const int n = n0 + (i * NW + wave) * 8 + lr;
    b_off[i] = n < a.Cout ? (uint32_t)((n * a.Kp + lc * 8) * 2) : OOB;
  }

  // BREG: this wave's 32 channels are fragment block nb = (n0 + 32 wn) / 32
  // of a.wf; k16 step s of it is 1 KB at (nb * Kp / 16 + s) * 1 KB, lane l
  // reading the 16 bytes at l * 16 (past Cout: out of range, zeros)
  const int nw0 = n0 + wn * TN;
  const uint32_t wf_base =
      BREG && nw0 < a.Cout ? (uint32_t)((int64_t)(nw0 / 32) * (a.Kp / 16) * 1024 + lane * 16) : OOB;
  const __amdgpu_buffer_rsrc_t rwf =
      rsrc(BREG && a.wf ? reinterpret_cast<const uint16_t*>(a.wf) + z * a.wf_mstride : reinterpret_cast<const uint16_t*>(a.w),
           BREG && a.wf ? (uint32_t)((int64_t)a.Cout * a.Kp * 2) : 0u);
  auto load_wfrag = [&](int kt, uint4 (&v)[4]) {
#pragma unroll
    for (int s = 0; s < 4; ++s) {
      const uint32_t off = wf_base == OOB ? OOB : wf_base + (uint32_t)(kt * 4 + s) * 1024u;
      v[s] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rwf, off, 0, 0));
    }
  };

  const float inv_cin = 1.0f / (float)a.Cin, inv_kw = 1.0f / (float)a.kw;
  auto issue = [&](int kt, int stage) {
    const int k0 = kt * BK;
    char* base = smem + stage * STAGE;
    if (a.x2 && k0 >= a.K1) {  // the projection shortcut's 1x1 reduction (wave-uniform)
      const uint32_t c2 = (uint32_t)(k0 - a.K1) * 2;
#pragma unroll
      for (int i = 0; i < AP; ++i) {
        const uint32_t off = a2_off[i] == OOB ? OOB : a2_off[i] + c2;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx2, (lds_void*)(base + (i * NW + wave) * 1024), 16, off, 0, 0, 0);
      }
    } else {
      // k0 < Kp and the tap index stay far below 2^22 (conv_dma_ok)
      const int tap = __builtin_amdgcn_readfirstlane(fdiv_small(k0, inv_cin));
      const int ci0 = k0 - tap * a.Cin;
      const int ky = __builtin_amdgcn_readfirstlane(fdiv_small(tap, inv_kw)), kx = tap - ky * a.kw;
      const int tap_off = (ky * a.W + kx) * a.Cin + ci0;
#pragma unroll
      for (int i = 0; i < AP; ++i) {
        const int iy = a_iy[i] + ky, ix = a_ix[i] + kx + dx;
        const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
        const uint32_t off = ok ? (uint32_t)((a_off[i] + tap_off) * 2) : OOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)(base + (i * NW + wave) * 1024), 16, off, 0, 0, 0);
      }
    }
    if constexpr (!BREG)
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

  // issued before every operand load: vmcnt counts loads in issue order, so
  // the waits for the operand tiles below also cover these
  uint4 rpre[FM][FN][2];
  if constexpr (PRE) load_residual<FM, FN>(a, m0 + wm * TM, n0 + wn * TN, z, lane, rpre);
  // Without a residual in registers (and with a ring: the one-stage tiles
  // keep their registers for occupancy), an unsplit layer's bias is fetched
  // here too, so the epilogue does not wait for it after the last MFMA.
  constexpr bool BIASP = !PRE && STAGES > 1;
  float bpre[FN][2][8];
  if constexpr (BIASP)
    if (a.split == 1) load_bias<FN>(a, n0 + wn * TN, z, lane, bpre);

  // this workgroup's share of the K-tiles (all of them unless split-K)
  const int nk_all = a.Kp / BK;
  const int kb = sp * nk_all / a.split, nk = (sp + 1) * nk_all / a.split - kb;
  // BREG: A fragments from LDS as in mma_ktile, the weight fragment of k16
  // step 2 kh + ks from bv
  auto compute_breg = [&](int stage, const uint4 (&bv)[4]) {
    const char* As = smem + stage * STAGE;
    const int fr = lane & 31;
    int ra[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) ra[i] = wm * TM + i * 32 + fr;
#pragma unroll
    for (int kh = 0; kh < 2; ++kh) {
      bf16x8 af[2][FM], bfr[2][FN];
      const int fq = lane >> 5;
#pragma unroll
      for (int ks = 0; ks < 2; ++ks) {
        const int c = (kh * 2 + ks) * 2 + fq;
#pragma unroll
        for (int i = 0; i < FM; ++i) af[ks][i] = *reinterpret_cast<const bf16x8*>(As + ra[i] * ROW + ((c ^ swz(ra[i])) << 4));
        bfr[ks][0] = __builtin_bit_cast(bf16x8, bv[kh * 2 + ks]);
      }
      mma_half<FM, FN>(af, bfr, acc);
    }
  };
  if constexpr (BREG) {
    // two register sets named by the parity of the K-tile (the loop is
    // unrolled by two), so no copy moves them between K-tiles; the wait
    // before each barrier covers the A tile and the weight fragments alike
    uint4 wa[4], wb[4];
    if (nk > 0) {
      issue(kb, 0);
      load_wfrag(kb, wa);
    }
    auto step = [&](int kt, const uint4 (&cur)[4], uint4 (&nxt)[4]) {
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
      if (kt + 1 < nk) {
        issue(kb + kt + 1, (kt + 1) & 1);
        load_wfrag(kb + kt + 1, nxt);
      }
      compute_breg(kt & 1, cur);
    };
    for (int kt = 0; kt < nk; kt += 2) {
      step(kt, wa, wb);
      if (kt + 1 < nk) step(kt + 1, wb, wa);
    }
  } else if constexpr (STAGES == 1) {
    // one buffer (for layers of one or a few K-tiles, where a deeper ring
    // only costs occupancy): fetch, wait, compute, and meet again before the
    // next fetch overwrites the buffer
    for (int kt = 0; kt < nk; ++kt) {
      if (kt > 0) __builtin_amdgcn_s_barrier();
      issue(kb + kt, 0);
      wait_vmcnt<0>();
      __builtin_amdgcn_s_barrier();
      compute(0);
    }
  } else {
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
  }

  conv_epilogue<FM, FN, PRE, BIASP>(a, acc, m0 + wm * TM, n0 + wn * TN, z, sp, lane, rpre, bpre);
}

// Direct 3x3 / stride 1 / pad 1 convolution with the input halo staged
// once per 64-channel chunk.  The implicit GEMM above fetches every input
// pixel once per filter tap (9 times for a 3x3 filter); here a workgroup
// loads the (TH+2) x (W+2) patch of one 64-channel chunk into LDS once and
// all 9 taps read their shifted A operands from it, while the weights of the
// workgroup's BN output channels stay resident in LDS for its whole life.
// The kernel is persistent: one workgroup per CU, each owning one (model,
// N-tile) group and a contiguous range of its spatial tiles (TH output rows
// x the full output width of one image); steps (tile, chunk) run through a
// double-buffered patch, the next step's patch in flight while this one's
// MFMAs run.  Each wave owns FM blocks of 32 pixels x all BN channels.  The
// bias is loaded once; a tile's residual is loaded when its last step
// starts, so neither waits at the epilogue.  Per output, the sum runs over
// chunks, then taps, then the 64 channels in the same MFMA order as the
// implicit GEMM; with one chunk (Cin = 64) the order, and so every bit, is
// that of the implicit GEMM.  Patch pixel (r, c) (patch row, padded column)
// is swizzled by h = r * TW + c, which runs consecutively over the 16
// outputs an operand read serves per cycle, also across an output row's end
// (where the patch index skips the two padding columns), so the reads are
// free of bank conflicts at every tap.
template <int TH, int TW, int BN, int FM, int WBYTES>
__global__ void __launch_bounds__(64 * (TH * TW / 32) / FM, 1) k_conv_halo(ConvArgs a) {
  constexpr int P = TH * TW, MB = P / 32, NW = MB / FM, FN = BN / 32;
  constexpr int PW = TW + 2, NP = (TH + 2) * PW;  // patch width and pixels
  constexpr int NPB = (NP + 7) / 8;               // 8-pixel load blocks
  constexpr int PATCH = NPB * 8 * ROW;
  constexpr int NIT = (NPB + NW - 1) / NW;        // patch load instructions per wave
  static_assert(P % 32 == 0 && MB % FM == 0 && BN % 32 == 0, "tile");
  __shared__ __attribute__((aligned(1024))) char smem[WBYTES + 2 * PATCH];
  char* const wsm = smem;
  char* const psm = smem + WBYTES;

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane >> 3, fr = lane & 31, fq = lane >> 5;
  const int nkt = a.Kp / BK;

  // ---- this workgroup's group (model z, N-tile) and range of spatial tiles
  const int tiles_h = (a.Ho + TH - 1) / TH, T = a.B * tiles_h;
  const int NT = a.Cout / BN, G = a.Z * NT;
  const int nwg = gridDim.x, base = nwg / G, rem = nwg % G, big = rem * (base + 1);
  const int bx = blockIdx.x;
  const int g = bx < big ? bx / (base + 1) : rem + (bx - big) / base;
  const int gi = bx < big ? bx % (base + 1) : (bx - big) % base;
  const int gsize = base + (g < rem ? 1 : 0);
  const int z = g / NT, n0 = (g - z * NT) * BN;
  const int t_begin = (int)((int64_t)gi * T / gsize), t_end = (int)((int64_t)(gi + 1) * T / gsize);
  if (t_begin >= t_end) return;  // uniform over the workgroup

  const __amdgpu_buffer_rsrc_t rx = rsrc(reinterpret_cast<const uint16_t*>(a.x) + z * a.x_mstride,
                                         (uint32_t)((int64_t)a.B * a.H * a.W * a.Cin * 2));
  const __amdgpu_buffer_rsrc_t rw = rsrc(reinterpret_cast<const uint16_t*>(a.w) + z * a.w_mstride,
                                         (uint32_t)((int64_t)a.Cout * a.Kp * 2));

  // ---- resident weights: LDS row kt * BN + n holds w[n0 + n][kt*64 .. +64]
  {
    const int nblk = nkt * BN / 8;
    for (int blk = wave; blk < nblk; blk += NW) {
      const int r = blk * 8 + lr;
      const int kt = r / BN, n = r - kt * BN;
      const int lc = (lane & 7) ^ swz(r);  // this lane fills physical chunk lane & 7
      const uint32_t off = (uint32_t)((((int64_t)(n0 + n) * a.Kp) + kt * BK + lc * 8) * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void*)(wsm + blk * 1024), 16, off, 0, 0, 0);
    }
  }

  // ---- patch loads: pixel q of the patch is input (oy0 - 1 + q / PW, q % PW - 1).
  // Every wave issues NIT instructions for every patch (a wave past the last
  // block repeats it: the same bytes to the same LDS slot), the step after the
  // last fetches out of range, and the residual loads are unconditional, so
  // each wave's count of vector-memory operations is the same on every path
  // and the compiler's own waits are exact rather than full drains.
  int q_dy[NIT], q_ix[NIT], q_lc[NIT], q_blk[NIT];
#pragma unroll
  for (int it = 0; it < NIT; ++it) {
    const int blk = min(it * NW + wave, NPB - 1);
    q_blk[it] = blk;
    const int q = blk * 8 + lr;
    q_lc[it] = (lane & 7) ^ (((q / PW * TW + q % PW) >> 1) & 7);
    if (blk < NPB && q < NP) {
      const int pr = q / PW;
      q_dy[it] = pr - 1;
      q_ix[it] = q - pr * PW - 1;
    } else {
      q_dy[it] = -(1 << 28);  // never inside the image
      q_ix[it] = 0;
    }
  }
  auto issue_patch = [&](int t, int cc, int buf, bool live) {
    const int img = t / tiles_h, oy0 = (t - img * tiles_h) * TH;
    char* pb = psm + buf * PATCH;
#pragma unroll
    for (int it = 0; it < NIT; ++it) {
      const int iy = oy0 + q_dy[it], ix = q_ix[it];
      const bool ok = live && (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
      const uint32_t keep = 0u - (uint32_t)ok;  // a bitwise blend keeps the load unconditional
      const uint32_t real =
          (uint32_t)(((((int64_t)img * a.H + max(iy, 0)) * a.W + max(ix, 0)) * a.Cin + cc * BK + q_lc[it] * 8) * 2);
      const uint32_t off = (real & keep) | (OOB & ~keep);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)(pb + q_blk[it] * 1024), 16, off, 0, 0, 0);
    }
  };

  // ---- this lane's pixels (block i of the wave is tile block wave * FM + i)
  // and, for the epilogue, its 8-channel groups: after the permlane32 swap a
  // lane holds channels n0 + 32 j + 8 (gp + fq) .. +8 of its pixel, gp = 0, 2
  int q0[FM], h0[FM], pr_[FM], pc_[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int pidx = (wave * FM + i) * 32 + fr;
    pr_[i] = pidx / TW;
    pc_[i] = pidx - pr_[i] * TW;
    q0[i] = pr_[i] * PW + pc_[i];
    h0[i] = pr_[i] * TW + pc_[i];
  }
  float bias_v[FN][2][8];
  {
    const float* __restrict__ bias = a.bias + z * a.b_mstride;
#pragma unroll
    for (int j = 0; j < FN; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int n = n0 + j * 32 + 8 * (2 * h + fq);
        const float4 b0 = *reinterpret_cast<const float4*>(bias + n);
        const float4 b1 = *reinterpret_cast<const float4*>(bias + n + 4);
        bias_v[j][h][0] = b0.x; bias_v[j][h][1] = b0.y; bias_v[j][h][2] = b0.z; bias_v[j][h][3] = b0.w;
        bias_v[j][h][4] = b1.x; bias_v[j][h][5] = b1.y; bias_v[j][h][6] = b1.z; bias_v[j][h][7] = b1.w;
      }
  }
  const bool has_res = a.res != nullptr;
  // residual through a buffer resource (empty without one: every load reads zero)
  const __amdgpu_buffer_rsrc_t rres =
      has_res ? rsrc(reinterpret_cast<const uint16_t*>(a.res) + z * a.res_mstride, (uint32_t)((int64_t)a.M * a.Cout * 2))
              : rsrc(a.y, 0u);

  floatx16 acc[FM][FN];
  auto zero_acc = [&]() {
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
  };
  zero_acc();
  // Two register sets for the tiles' output rows and residuals: a step uses
  // one and fetches the next tile's into the other, so no copy (which the
  // compiler guarded with a full wait) moves them between steps.
  uint4 res_a[FM][FN][2], res_b[FM][FN][2];
  int mg_a[FM], mg_b[FM];

  // outputs through a buffer resource: an epilogue issues exactly NSTORE
  // stores per lane (out-of-range ones are dropped), so the next step waits
  // for its patch without waiting for them
  constexpr int NSTORE = FM * FN * 2;
  const __amdgpu_buffer_rsrc_t ry = rsrc(reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride,
                                         (uint32_t)((int64_t)a.M * a.Cout * 2));
  // a tile's output rows and its residual (into rv), fetched one tile ahead,
  // behind the next tile's patch: the wait for that patch also covers it
  auto tile_rows_res = [&](int t, int (&m_)[FM], uint4 (&rv)[FM][FN][2]) {
    const int img = t / tiles_h, oy0 = (t - img * tiles_h) * TH;
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int oy = oy0 + pr_[i];
      m_[i] = oy < a.Ho ? (img * a.Ho + oy) * a.Wo + pc_[i] : -1;
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int n = n0 + j * 32 + 8 * (2 * h + fq);
          // a bitwise blend, not a select: the compiler turned the select into
          // two branches with a load each, which made the load count vary
          const uint32_t keep = 0u - (uint32_t)(m_[i] >= 0);
          const uint32_t off = ((uint32_t)((max(m_[i], 0) * a.Cout + n) * 2) & keep) |
                               ((OOB + 16u * (uint32_t)((i * FN + j) * 2 + h)) & ~keep);  // distinct: never merged
          rv[i][j][h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rres, off, 0, 0));
        }
    }
  };
  // One 64-channel chunk (conv_halo_ok: the resident weights hold at most
  // 9 x 64 x BN), so a step is a whole tile.
  const int steps = t_end - t_begin;
  issue_patch(t_begin, 0, 0, true);
  tile_rows_res(t_begin, mg_a, res_a);
  dummy_stores<NSTORE>(ry);  // every step starts with NSTORE stores in flight behind its patch
  auto step = [&](int st, const int (&mg)[FM], const uint4 (&res_v)[FM][FN][2], int (&mg_n)[FM],
                  uint4 (&res_n)[FM][FN][2]) {
    wait_vmcnt<NSTORE>();  // the patch and the tile's residual landed; the last step's stores may be in flight
    wg_barrier();
    {  // the next tile's patch (out of range after the last tile) and residual
      const bool live = st + 1 < steps;
      const int tn = t_begin + min(st + 1, steps - 1);
      issue_patch(tn, 0, (st + 1) & 1, live);
      tile_rows_res(tn, mg_n, res_n);
      __builtin_amdgcn_sched_barrier(0);  // issued here, not sunk among the MFMAs: they have the whole step to land
    }
    const char* Pb = psm + (st & 1) * PATCH;
#pragma unroll
    for (int tap = 0; tap < 9; ++tap) {
      const int ky = tap / 3, kx = tap - ky * 3;
      int ra[FM], sa[FM], rb[FN];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        ra[i] = q0[i] + ky * PW + kx;
        sa[i] = ((h0[i] + ky * TW + kx) >> 1) & 7;
      }
#pragma unroll
      for (int j = 0; j < FN; ++j) rb[j] = tap * BN + j * 32 + fr;
      mma_ktile_rows_sw<FM, FN>(Pb, wsm, ra, sa, rb, lane, acc);
    }
    // epilogue: bias, residual, ReLU, bf16, 16-byte stores
#pragma unroll
    for (int i = 0; i < FM; ++i)
#pragma unroll
      for (int j = 0; j < FN; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int gp = 2 * h;
          float v[8], rr[8];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i][j][gp * 4 + r]),
                                                             __float_as_uint(acc[i][j][(gp + 1) * 4 + r]), false, false);
            v[r] = __uint_as_float(sw[0]);
            v[4 + r] = __uint_as_float(sw[1]);
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) v[e] += bias_v[j][h][e];
          if (has_res) {
            bf8_to_f8(res_v[i][j][h], rr);
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] += rr[e];
          }
          if (a.relu)
#pragma unroll
            for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
          const int n = n0 + j * 32 + 8 * (gp + fq);
          const uint32_t keep = 0u - (uint32_t)(mg[i] >= 0);
          const uint32_t off = ((uint32_t)((max(mg[i], 0) * a.Cout + n) * 2) & keep) |
                               ((OOB + 16u * (uint32_t)((i * FN + j) * 2 + h)) & ~keep);  // distinct: never merged
          __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, f8_to_bf8(v)), ry, off, 0, 0);
        }
    zero_acc();
  };
  for (int st = 0; st < steps; st += 2) {
    step(st, mg_a, res_a, mg_b, res_b);
    if (st + 1 < steps) step(st + 1, mg_b, res_b, mg_a, res_a);
  }
  wait_vmcnt<0>();  // the out-of-range fetches after the last step land before the workgroup leaves
}

// The ResNet stem fused: 7x7/2 conv in its space-to-depth form (4x4/1,
// pad 2, on the [B][Hs][Ws][16] tensor, K = 256), bias, ReLU, bf16 rounding,
// then the 3x3/2 max pool (pad 1), writing only the pooled tensor.  Rounding
// before the max is exact: max commutes with a monotone rounding, so the
// result equals the two layers run separately.  After the ReLU every value
// is +0 or positive, whose bf16 bit patterns order like the values, so the
// pool takes packed 16-bit integer maxima; window taps outside the image are
// replaced by in-window neighbours (clamped), which leaves a max unchanged.
//
// Persistent: the workgroups are split evenly over the models, and each
// walks a contiguous run of (image, pooled-row pair) steps of its model with
// that model's 64 x 256 weights resident in LDS.  A step computes 4 conv rows
// (2 pooled rows' worth) from the 7 input rows it needs, staged in LDS as
// 32-byte pixels at a fixed row stride (the two 16-byte halves of pixel x
// are swapped when bit 3 of x is set, so the 16 consecutive pixels an
// operand read touches fall on distinct banks) and double-buffered: the next
// step's rows load while this step's MFMAs run.  Every 16-wide K step is one
// (Ky, Kx) tap, in the MFMA order of the implicit GEMM.  The activated rows
// go to a ring of five LDS row buffers (conv row r in buffer r % 5); the two
// pooled rows of a step are taken from the ring while the next step's MFMAs
// run, and the last conv row stays for the next pair.  A run that starts
// below the top of an image first computes the four conv rows above it.
// 7 waves, each two 32-pixel blocks x 64 channels (4 rows x 112 = 14 blocks).
constexpr int STEM_WMAX = 112;                 // conv output width limit
constexpr int STEM_PW = STEM_WMAX + 3;         // patch pixels per row (fixed stride)
constexpr int STEM_TR = 4;                     // conv rows per step
constexpr int STEM_PR = STEM_TR + 3;           // input rows per step
constexpr int STEM_RING = STEM_TR + 1;         // conv rows kept for pooling
constexpr int STEM_NSLOT = STEM_PR * STEM_PW * 2;  // 16-byte patch slots
constexpr int STEM_PATCH = ((STEM_NSLOT * 16 + 1023) / 1024) * 1024;
constexpr int STEM_FM = 2;                     // 32-pixel blocks per wave
constexpr int STEM_WAVES = (STEM_TR * STEM_WMAX + 32 * STEM_FM - 1) / (32 * STEM_FM);
constexpr int STEM_PBLK = (STEM_NSLOT + 63) / 64;                           // patch load instructions
constexpr int STEM_PIT = (STEM_PBLK + STEM_WAVES - 1) / STEM_WAVES;         // ... per wave
constexpr int STEM_NSTORE = (2 * ((STEM_WMAX - 1) / 2 + 1) * 8 + 64 * STEM_WAVES - 1) / (64 * STEM_WAVES);

typedef unsigned short u16x8 __attribute__((ext_vector_type(8)));

__global__ void __launch_bounds__(64 * STEM_WAVES, 1) k_stem_pool(ConvArgs a) {
  constexpr int WB = 4 * 64 * ROW;             // resident weights
  constexpr int RB = STEM_WMAX * ROW;          // one activated conv row
  // separate arrays (and a step loop unrolled by two, so each step reads one
  // patch buffer and fills the other by name): the compiler can then tell
  // that the LDS reads and writes of a step do not touch the buffer the
  // direct loads are filling, and does not wait for those loads
  __shared__ __attribute__((aligned(1024))) char wsm[WB];
  __shared__ __attribute__((aligned(1024))) char psm0[STEM_PATCH];
  __shared__ __attribute__((aligned(1024))) char psm1[STEM_PATCH];
  __shared__ __attribute__((aligned(1024))) char rsm[STEM_RING * RB];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane >> 3, fr = lane & 31, fq = lane >> 5;
  const int Wc = a.Wo, Hc = a.Ho;              // conv output
  const int Hp = (Hc - 1) / 2 + 1, Wp = (Wc - 1) / 2 + 1;  // 3x3/2/p1 pool output
  const int npair = (Hp + 1) / 2;              // pooled-row pairs per image

  // ---- this workgroup's model and run of (image, pair) steps
  const int nwg = gridDim.x, base = nwg / a.Z, rem = nwg % a.Z, big = rem * (base + 1);
  const int bx = blockIdx.x;
  const int z = bx < big ? bx / (base + 1) : rem + (bx - big) / base;
  const int gi = bx < big ? bx % (base + 1) : (bx - big) % base;
  const int gsize = base + (z < rem ? 1 : 0);
  const int T = a.B * npair;
  const int j0 = (int)((int64_t)gi * T / gsize), j1 = (int)((int64_t)(gi + 1) * T / gsize);
  if (j0 >= j1) return;  // uniform over the workgroup
  const int carry = (j0 % npair) > 0 ? 1 : 0; // the first pair needs the conv rows above it
  const int nsteps = j1 - j0 + carry;
  // step s -> image and top conv row; pools unless it is the carry step
  auto step_img = [&](int s) { return (j0 + max(s - carry, 0)) / npair; };
  auto step_rho = [&](int s) {
    const int j = j0 + max(s - carry, 0);
    return STEM_TR * (j - (j / npair) * npair) - (s < carry ? STEM_TR : 0);
  };

  const __amdgpu_buffer_rsrc_t rx = rsrc(reinterpret_cast<const uint16_t*>(a.x) + z * a.x_mstride,
                                         (uint32_t)((int64_t)a.B * a.H * a.W * 16 * 2));
  const __amdgpu_buffer_rsrc_t rw = rsrc(reinterpret_cast<const uint16_t*>(a.w) + z * a.w_mstride,
                                         (uint32_t)((int64_t)a.Cout * a.Kp * 2));
  // resident weights: LDS row Ky * 64 + n holds w[n][Ky*64 .. +64]
  for (int blk = wave; blk < 4 * 64 / 8; blk += STEM_WAVES) {
    const int r = blk * 8 + lr;
    const int ky = r >> 6, n = r & 63;
    const int lc = (lane & 7) ^ swz(r);
    const uint32_t off = (uint32_t)(((int64_t)n * a.Kp + ky * BK + lc * 8) * 2);
    __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void*)(wsm + blk * 1024), 16, off, 0, 0, 0);
  }
  // patch of the step with top conv row rho0: input rows rho0 - 2 .. rho0 +
  // STEM_TR + 2, columns -2 .. STEM_PW - 3; slot s = 2 * (pr * STEM_PW + pc) +
  // stored half.  Per lane and load instruction the slot's row, column and
  // byte offset within the pixel are fixed: precomputed.
  int q_pr[STEM_PIT], q_ix[STEM_PIT], q_hb[STEM_PIT];
#pragma unroll
  for (int it = 0; it < STEM_PIT; ++it) {
    const int sl = (it * STEM_WAVES + wave) * 64 + lane;
    const int pix = sl >> 1, pr = pix / STEM_PW, pc = pix - pr * STEM_PW;
    const bool ok = sl < STEM_NSLOT && pc - 2 < a.W;
    q_pr[it] = ok ? pr - 2 : -(1 << 28);
    q_ix[it] = pc - 2;
    q_hb[it] = (((sl & 1) ^ ((pc >> 3) & 1)) * 8) * 2;
  }
  auto issue_patch = [&](int b, int rho0, char* pb) {
    const int64_t img = (int64_t)b * a.H;
#pragma unroll
    for (int it = 0; it < STEM_PIT; ++it) {
      const int blk = it * STEM_WAVES + wave;
      if (blk < STEM_PBLK) {
        const int iy = rho0 + q_pr[it], ix = q_ix[it];
        const bool ok = (unsigned)iy < (unsigned)a.H && (unsigned)ix < (unsigned)a.W;
        const uint32_t off = ok ? (uint32_t)(((img + iy) * a.W + ix) * 32 + q_hb[it]) : OOB;
        __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)(pb + blk * 1024), 16, off, 0, 0, 0);
      }
    }
  };

  // ---- this lane's pixels (block i of the wave is step block wave * FM + i)
  // and the byte offsets of its operands: A for (i, kx) at ky = 0 (the ky
  // offset is a constant), B per kx (j and ky are constants)
  int pr0[STEM_FM], pc0[STEM_FM], a_off[STEM_FM][4];
  bool pv[STEM_FM];
#pragma unroll
  for (int i = 0; i < STEM_FM; ++i) {
    const int pidx = (wave * STEM_FM + i) * 32 + fr;
    pv[i] = pidx < STEM_TR * Wc;
    pr0[i] = pv[i] ? pidx / Wc : 0;
    pc0[i] = pv[i] ? pidx - pr0[i] * Wc : 0;
#pragma unroll
    for (int kx = 0; kx < 4; ++kx) {
      const int pc = pc0[i] + kx;
      a_off[i][kx] = (2 * (pr0[i] * STEM_PW + pc) + (fq ^ ((pc >> 3) & 1))) * 16;
    }
  }
  int b_off[4];
#pragma unroll
  for (int kx = 0; kx < 4; ++kx) b_off[kx] = fr * ROW + (((2 * kx + fq) ^ swz(fr)) << 4);
  float bias_v[2][2][8];
  {
    const float* __restrict__ bias = a.bias + z * a.b_mstride;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h)
#pragma unroll
        for (int e = 0; e < 8; ++e) bias_v[j][h][e] = bias[j * 32 + 8 * (2 * h + fq) + e];
  }
  // pooled output through a buffer resource: every thread issues exactly
  // STEM_NSTORE stores per step (out-of-range ones are dropped), so the next
  // step can wait for its input rows without waiting for them
  const __amdgpu_buffer_rsrc_t ry = rsrc(reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride,
                                         (uint32_t)((int64_t)a.B * Hp * Wp * 64 * 2));

  // item u of this thread's share of the two pooled rows of step ps (whose
  // activated rows are in the ring): one 16-byte store, written or dropped
  auto pool_item = [&](int ps, bool live_step, int u) {
    const int b = step_img(ps), rho0 = step_rho(ps);
    {
      const int item = tid + u * 64 * STEM_WAVES;
      const int q = item / (Wp * 8), rest = item - q * (Wp * 8);
      const int px = rest >> 3, ch = rest & 7;
      const int py = rho0 / 2 + q;
      const bool live = live_step && q < 2 && py < Hp;
      u16x8 m = {0, 0, 0, 0, 0, 0, 0, 0};
      if (live) {
#pragma unroll
        for (int dy = -1; dy <= 1; ++dy) {
          const int cr = min(max(2 * py + dy, 0), Hc - 1);
          const char* rowp = rsm + (cr % STEM_RING) * RB;
#pragma unroll
          for (int dx = -1; dx <= 1; ++dx) {
            const int cc = min(max(2 * px + dx, 0), Wc - 1);
            const uint4 v = *reinterpret_cast<const uint4*>(rowp + cc * ROW + ((ch ^ swz(cc)) << 4));
            m = __builtin_elementwise_max(m, __builtin_bit_cast(u16x8, v));
          }
        }
      }
      const uint32_t off = live ? (uint32_t)(((((int64_t)b * Hp + py) * Wp + px) * 64 + ch * 8) * 2)
                                : OOB + 16u * (uint32_t)u;  // distinct: never merged
      __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, m), ry, off, 0, 0);
    }
  };
  auto pool_step = [&](int ps, bool live_step) {
#pragma unroll
    for (int u = 0; u < STEM_NSTORE; ++u) pool_item(ps, live_step, u);
  };

  auto do_step = [&](int st, const char* Pb, char* Pn) __attribute__((always_inline)) {
    const int rho0 = step_rho(st);
    wait_vmcnt<STEM_NSTORE>();  // this step's rows landed; the last step's stores may be in flight
    wait_lgkm0();
    wg_barrier();               // ...and every wave's activated rows of the last step are in the ring
    if (st + 1 < nsteps) issue_patch(step_img(st + 1), step_rho(st + 1), Pn);
    floatx16 acc[STEM_FM][2];
#pragma unroll
    for (int i = 0; i < STEM_FM; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    // the previous step's pooled rows are interleaved with these MFMAs: they
    // read only the ring, so their LDS reads, maxima and stores issue while
    // the matrix cores work
    const int pps = st > 0 ? st - 1 : 0;
    const bool plive = st > 0 && st - 1 >= carry;
#pragma unroll
    for (int ky = 0; ky < 4; ++ky) {
#pragma unroll
      for (int kx = 0; kx < 4; ++kx) {
        constexpr int NTAP = 16;
        const int tap = ky * 4 + kx;
#pragma unroll
        for (int u = 0; u < STEM_NSTORE; ++u)
          if (tap == (u + 1) * NTAP / (STEM_NSTORE + 1)) pool_item(pps, plive, u);
        bf16x8 af[STEM_FM], bfr[2];
#pragma unroll
        for (int i = 0; i < STEM_FM; ++i)
          af[i] = *reinterpret_cast<const bf16x8*>(Pb + a_off[i][kx] + ky * STEM_PW * 32);
#pragma unroll
        for (int j = 0; j < 2; ++j)
          bfr[j] = *reinterpret_cast<const bf16x8*>(wsm + b_off[kx] + (ky * 64 + j * 32) * ROW);
#pragma unroll
        for (int i = 0; i < STEM_FM; ++i)
#pragma unroll
          for (int j = 0; j < 2; ++j)
            acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(bfr[j], af[i], acc[i][j], 0, 0, 0);
      }
    }
    wait_lgkm0();
    wg_barrier();  // the ring rows the pooling read may now be overwritten
    // activated bf16 conv rows into the LDS ring (row rho in buffer rho % 5)
#pragma unroll
    for (int i = 0; i < STEM_FM; ++i) {
      const int rho = rho0 + pr0[i];
      char* rowp = rsm + ((rho + STEM_RING) % STEM_RING) * RB + pc0[i] * ROW;
      const int sw = swz(pc0[i]);
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int h = 0; h < 2; ++h) {
          const int gp = 2 * h;
          float v[8];
#pragma unroll
          for (int r = 0; r < 4; ++r) {
            const auto sw2 = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i][j][gp * 4 + r]),
                                                              __float_as_uint(acc[i][j][(gp + 1) * 4 + r]), false, false);
            v[r] = __uint_as_float(sw2[0]);
            v[4 + r] = __uint_as_float(sw2[1]);
          }
#pragma unroll
          for (int e = 0; e < 8; ++e) {
            const float t = v[e] + bias_v[j][h][e];
            v[e] = t > 0.f ? t : 0.f;  // +0 for every non-positive value
          }
          const int chunk = j * 4 + gp + fq;  // 8-channel group of the 64
          if (pv[i] && rho >= 0 && rho < Hc)
            *reinterpret_cast<uint4*>(rowp + ((chunk ^ sw) << 4)) = f8_to_bf8(v);
        }
    }
  };

  issue_patch(step_img(0), step_rho(0), psm0);
  // STEM_NSTORE dropped stores, so that every step starts with the same count
  // of stores in flight behind its rows
  dummy_stores<STEM_NSTORE>(ry);
  for (int st = 0; st < nsteps; st += 2) {
    do_step(st, psm0, psm1);
    if (st + 1 < nsteps) do_step(st + 1, psm1, psm0);
  }
  wait_lgkm0();
  wg_barrier();
  pool_step(nsteps - 1, nsteps - 1 >= carry);
}

bool stem_pool_ok_impl(const ConvArgs& a) {
  return a.Cin == 16 && a.kh == 4 && a.kw == 4 && a.stride == 1 && a.pad == 2 && a.Cout == 64 && a.Kp == 256 &&
         a.K == 256 && a.Wo <= STEM_WMAX && a.Wo >= 1 && a.Ho >= 1 && a.relu && !a.res && a.Wo == a.W &&
         a.Ho == a.H;
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
    for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
  *reinterpret_cast<uint4*>(reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride + o) = f8_to_bf8(v);
}

// Split-K completion fused with the global average pool that is the conv's
// only reader: a workgroup of 1024 threads owns one (model, image); thread (channel group
// cg, pixel lane pl) finishes pixels pl, pl + PL, ... exactly as the plain
// reduce does (partials in split order, bias, residual, ReLU, bf16 rounding:
// the stored activation) and sums them in fp32; the PL lanes' sums are added
// in lane order, divided by H*W and rounded once.  The activation tensor is
// never written.  y: [B][Cout] per model.
constexpr int RG_T = 1024;  // threads of the fused split-K completion + pool

__global__ void __launch_bounds__(RG_T) k_conv_splitk_reduce_gap(ConvArgs a, uint16_t* gy, int64_t gy_mstride) {
  __shared__ float part[RG_T][8];
  const int CG = a.Cout / 8, PL = RG_T / CG;
  const int z = blockIdx.x / a.B, b = blockIdx.x - z * a.B;
  const int cg = threadIdx.x % CG, pl = threadIdx.x / CG, n = cg * 8;
  const int HW = a.Ho * a.Wo;
  const float* bias = a.bias + z * a.b_mstride + n;
  float bv[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) bv[e] = bias[e];
  float acc[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) acc[e] = 0.f;
  for (int p = pl; p < HW; p += PL) {
    const int64_t m = (int64_t)b * HW + p;
    float v[8];
    const float4* p0 = reinterpret_cast<const float4*>(a.partial + ((int64_t)z * a.M + m) * a.Cout + n);
    float4 q0 = p0[0], q1 = p0[1];
    v[0] = q0.x; v[1] = q0.y; v[2] = q0.z; v[3] = q0.w; v[4] = q1.x; v[5] = q1.y; v[6] = q1.z; v[7] = q1.w;
    for (int sp = 1; sp < a.split; ++sp) {
      const float4* pp = reinterpret_cast<const float4*>(a.partial + (((int64_t)sp * a.Z + z) * a.M + m) * a.Cout + n);
      q0 = pp[0]; q1 = pp[1];
      v[0] += q0.x; v[1] += q0.y; v[2] += q0.z; v[3] += q0.w;
      v[4] += q1.x; v[5] += q1.y; v[6] += q1.z; v[7] += q1.w;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) v[e] += bv[e];
    if (a.res) {
      float r[8];
      bf8_to_f8(*reinterpret_cast<const uint4*>(reinterpret_cast<const uint16_t*>(a.res) + z * a.res_mstride + m * a.Cout + n), r);
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += r[e];
    }
    if (a.relu)
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
    float st[8];
    bf8_to_f8(f8_to_bf8(v), st);  // the stored bf16 activation
#pragma unroll
    for (int e = 0; e < 8; ++e) acc[e] += st[e];
  }
#pragma unroll
  for (int e = 0; e < 8; ++e) part[threadIdx.x][e] = acc[e];
  __syncthreads();
  if (pl != 0) return;
  float t[8];
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = part[cg][e];
  for (int q = 1; q < PL; ++q)
#pragma unroll
    for (int e = 0; e < 8; ++e) t[e] += part[q * CG + cg][e];
  const float hw = (float)HW;
#pragma unroll
  for (int e = 0; e < 8; ++e) t[e] = t[e] / hw;
  *reinterpret_cast<uint4*>(gy + z * gy_mstride + (int64_t)b * a.Cout + n) = f8_to_bf8(t);
}

}  // namespace

void launch_conv_splitk_reduce(const ConvArgs& a, hipStream_t s) {
  const int64_t total = (int64_t)a.Z * a.M * (a.Cout / 8);
  hipLaunchKernelGGL(k_conv_splitk_reduce, dim3((unsigned)((total + 255) / 256)), dim3(256), 0, s, a);
}

bool conv_reduce_gap_ok(const ConvArgs& a) {
  const int cg = a.Cout / 8;
  return a.split > 1 && a.Cout % 8 == 0 && cg >= 1 && cg <= RG_T && RG_T % cg == 0;
}

void launch_conv_splitk_reduce_gap(const ConvArgs& a, void* gy, int64_t gy_mstride, hipStream_t s) {
  hipLaunchKernelGGL(k_conv_splitk_reduce_gap, dim3(a.Z * a.B), dim3(RG_T), 0, s, a, static_cast<uint16_t*>(gy),
                     gy_mstride);
}

size_t conv_partial_floats(const ConvArgs& a) { return a.split > 1 ? (size_t)a.split * a.Z * a.M * a.Cout : 0; }

// K split of a layer: a function of its shape only (never of the tile), so
// every tile of the family still produces identical sums.  Split while the
// layer has fewer than three 64x64 output tiles per CU, keeping >= 8 K-tiles
// per split.
int conv_split(Prec p, const ConvArgs& a, int num_cus) {
  if (p != BF16 || !conv_dma_ok(a) || conv_hs_chosen(a)) return 1;  // the streamed-weight halo kernel never splits
  const int64_t units = (int64_t)((a.M + 63) / 64) * ((a.Cout + 63) / 64) * a.Z;
  const int nk = a.Kp / BK;
  int split = 1;
  while (units * split < 3 * num_cus && split < 4 && nk / (split * 2) >= 8) split *= 2;
  return split;
}

// Every 64-wide K-tile must lie in one filter row and cover whole pixels.
bool conv_dma_ok(const ConvArgs& a) {
  const bool tiles_ok = a.Cin % BK == 0 || (a.Cin % 8 == 0 && BK % a.Cin == 0 && (a.kw * a.Cin) % BK == 0);
  // a projection shortcut: whole K-tiles of the main reduction, then of the 1x1 one
  const bool proj_ok = !a.x2 || (a.K1 % BK == 0 && a.Cin2 % BK == 0 && a.K1 + a.Cin2 == a.K &&
                                 (a.Ho - 1) * a.stride2 < a.H2 && (a.Wo - 1) * a.stride2 < a.W2 &&
                                 (int64_t)a.B * a.H2 * a.W2 * a.Cin2 * 2 < (1ll << 31));
  return tiles_ok && proj_ok && a.Kp % BK == 0 && a.K == a.Kp && a.Cout % 8 == 0 && a.Kp < (1 << 22);
}

// Halo kernel shapes: TH output rows x TW (= the output width) pixels, BN
// output channels, FM M-blocks per wave, resident weights <= 72 KB.
constexpr int HALO_WBYTES = 72 * 1024;

bool conv_halo_ok(const ConvArgs& a, int th, int tw, int bn) {
  return !a.x2 && a.kh == 3 && a.kw == 3 && a.stride == 1 && a.pad == 1 && a.Cin == BK && a.K == a.Kp &&
         a.Wo == tw && a.Ho == a.H && a.Wo == a.W && a.Cout % bn == 0 && a.split == 1 &&
         (int64_t)a.Kp * bn * 2 <= HALO_WBYTES && a.Z * (a.Cout / bn) <= 4096;
}

static int cus_of_current_device() {
  static int cache[64] = {0};
  int dev = 0;
  if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 256;
  if (!cache[dev]) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
    cache[dev] = n;
  }
  return cache[dev];
}

void launch_conv_halo(const ConvArgs& a_in, int th, int tw, int bn, hipStream_t s) {
  ConvArgs a = a_in;  // the halo kernel never splits K: it always writes finished outputs
  a.split = 1;
  a.partial = nullptr;
  const int groups = a.Z * (a.Cout / bn);
  const int tiles = a.B * ((a.Ho + th - 1) / th) * groups;
  const int nwg = std::max(groups, std::min(tiles, cus_of_current_device()));
#define FS_HALO(THv, TWv, BNv, FMv)                                                                            \
  if (th == THv && tw == TWv && bn == BNv) {                                                                   \
    hipLaunchKernelGGL((k_conv_halo<THv, TWv, BNv, FMv, HALO_WBYTES>), dim3(nwg), dim3(64 * (THv * TWv / 32) / FMv), \
                       0, s, a);                                                                               \
    return;                                                                                                    \
  }
  FS_HALO(4, 56, 64, 1)
#undef FS_HALO
}

bool conv_stem_pool_ok(const ConvArgs& a) { return stem_pool_ok_impl(a); }

// y: the pooled [B][Hp][Wp][64] tensor; a.Ho x a.Wo is the conv output size.
void launch_conv_stem_pool(const ConvArgs& a, hipStream_t s) {
  const int Hp = (a.Ho - 1) / 2 + 1;
  const int steps = a.Z * a.B * ((Hp + 1) / 2);
  const int nwg = std::max(a.Z, std::min(steps, cus_of_current_device()));
  hipLaunchKernelGGL(k_stem_pool, dim3(nwg), dim3(64 * STEM_WAVES), 0, s, a);
}

void conv_frag_order(const uint16_t* w, int Cout, int Kp, uint16_t* out) {
  const int S = Kp / 16;
  for (int nb = 0; nb < Cout / 32; ++nb)
    for (int st = 0; st < S; ++st)
      for (int l = 0; l < 64; ++l)
        std::memcpy(out + (((size_t)nb * S + st) * 64 + l) * 8,
                    w + (size_t)(nb * 32 + (l & 31)) * Kp + 16 * st + 8 * (l >> 5), 16);
}

// The weights go to registers (BREG) when the tile has one row of waves of
// 32 channels each and a fragment-ordered copy of the weights exists.
template <int BMv, int BNv, int WMv, int WNv, int Sv>
static void launch_dma_t(const ConvArgs& a, int tiles, bool pre, hipStream_t s) {
  constexpr bool can_breg = WMv == 1 && BNv / WNv == 32 && Sv == 2;
  if constexpr (can_breg) {
    if (a.wf && a.Cout % 32 == 0) {
      if (pre)
        hipLaunchKernelGGL((k_conv_dma<BMv, BNv, WMv, WNv, Sv, true, true>), dim3(tiles), dim3(64 * WMv * WNv), 0, s, a);
      else
        hipLaunchKernelGGL((k_conv_dma<BMv, BNv, WMv, WNv, Sv, false, true>), dim3(tiles), dim3(64 * WMv * WNv), 0, s, a);
      return;
    }
  }
  if (pre)
    hipLaunchKernelGGL((k_conv_dma<BMv, BNv, WMv, WNv, Sv, true, false>), dim3(tiles), dim3(64 * WMv * WNv), 0, s, a);
  else
    hipLaunchKernelGGL((k_conv_dma<BMv, BNv, WMv, WNv, Sv, false, false>), dim3(tiles), dim3(64 * WMv * WNv), 0, s, a);
}

void launch_conv_dma(const ConvArgs& a, int bm, int bn, int waves, int wgm, int stages, hipStream_t s) {
  const int tiles = ((a.M + bm - 1) / bm) * ((a.Cout + bn - 1) / bn) * a.Z * a.split;
  const bool pre = a.res && a.split == 1;
#define FS_DMA(BMv, BNv, WMv, WNv, Sv)                                                                       \
  if (bm == BMv && bn == BNv && waves == WMv * WNv && stages == Sv && wgm == WMv) {                          \
    launch_dma_t<BMv, BNv, WMv, WNv, Sv>(a, tiles, pre, s);                                                  \
    return;                                                                                                  \
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
  FS_DMA(128, 128, 2, 2, 1)
  FS_DMA(128, 64, 2, 2, 1)
  FS_DMA(64, 128, 2, 2, 1)
  FS_DMA(256, 128, 2, 2, 2)
  FS_DMA(256, 128, 2, 2, 3)
  FS_DMA(128, 256, 2, 2, 2)
  FS_DMA(256, 256, 2, 4, 2)
  FS_DMA(128, 128, 2, 2, 3)
  FS_DMA(160, 128, 1, 4, 2)
  FS_DMA(96, 128, 1, 4, 1)
  FS_DMA(96, 128, 1, 4, 2)
#undef FS_DMA
}

}  // namespace fs
