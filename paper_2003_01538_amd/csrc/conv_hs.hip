// Direct 3x3 / stride 1 / pad 1 convolution with the input halo staged once
// per 64-channel chunk and the weights streamed one filter tap at a time, for
// layers with at least two 64-channel chunks (Cin a multiple of 128) and
// Cout a multiple of 128.  Two kernels: k_conv_hs streams the weights
// through LDS (below), k_conv_hr holds them in registers (further down).
//
// Why: the implicit GEMM fetches every input pixel once per filter tap, so a
// 3x3 layer moves its input through L2 nine times per output-channel tile.
// Here a tile's input patch of one 64-channel chunk is loaded into LDS once
// and all nine taps read their shifted operands from it; per (chunk, tap)
// only the 128 x 64 weight slice is streamed in.  Bytes fetched per MFMA
// drop by about 2.4x against a 64 x 128 implicit-GEMM tile, and each wave
// works on a 64 x 64 sub-tile (two operand fragments per MFMA pair instead
// of three).
//
// Tiles are runs of 128 consecutive output pixels in (image, row, column)
// order, so they may start mid-row and run into the next image.  The patch
// is a band of rows of the zero-padded input: in "padded row" coordinates an
// image occupies rows b (H+2) .. b (H+2) + H+1 (first and last all zero) and
// each padded row has PW = W+2 columns (first and last zero).  A tile's
// patch starts one padded row above its first pixel and holds NPB*8 padded
// pixels, enough for its last pixel's bottom-right tap (checked on the host).
// Output pixel (b, y, x) sits at padded (b (H+2) + y + 1, x + 1); its tap
// (ky, kx) reads patch pixel q0 + ky PW + kx, where q0 is its top-left tap.
// Pixels outside the image load as zero (buffer loads past the range).
//
// Work: the workgroups are split evenly over the (model, 128-channel) groups
// and each walks a contiguous run of that group's pixel tiles.  A step is
// one (chunk, tap): 16 MFMAs per wave (2 x 2 blocks of 32 x 32, four
// k16 steps).  Per output the sum runs over chunks, then taps, then the 64
// channels of the chunk in the MFMA order of the implicit GEMM.
//
// Pipeline (per wave, exact vector-memory counts): weights for step s + 3
// are fetched at step s into a ring of three 16 KB slots (slot = tap mod 3,
// fixed at compile time since 9 taps make one chunk), the next chunk's
// patch is fetched in nine slices during the current chunk into the other
// of two patch buffers, and the operand fragments of step s + 1 are read
// from LDS into a second register set while the MFMAs of step s run.  One
// barrier per step: after it, the weights of step s + 1 are visible and the
// slot read by step s is free for the fetch of step s + 3.  A tile's residual
// is fetched at the start of its last chunk and its outputs stored at the
// end; chunks that end no tile issue the same loads and stores out of range
// (dropped), so every step waits on a compile-time count.
#include "common.hpp"
#include "device.hpp"
#include "lds_dma.hpp"

#include <algorithm>
#include <type_traits>

namespace fs {

namespace {

constexpr int HS_BM = 128;                 // output pixels per tile
constexpr int HS_BN = 128;                 // output channels per tile
constexpr int HS_NW = 4;                   // waves: 2 along pixels x 2 along channels
constexpr int HS_WI = HS_BN / 8 / HS_NW;   // weight DMA instructions per wave and step
constexpr int HS_RI = 8;                   // residual loads per lane and tile
constexpr int HS_SI = 8;                   // output stores per lane and tile
constexpr int HS_WSLOT = HS_BN * ROW;      // one tap's weights: 128 rows x 128 bytes

template <int I, int N, class F>
__device__ __forceinline__ void static_for(F&& f) {
  if constexpr (I < N) {
    f(std::integral_constant<int, I>{});
    static_for<I + 1, N>(f);
  }
}

// Patch instructions per wave in slice u of a chunk's nine slices.
template <int NPBW>
constexpr int hs_ps(int u) { return NPBW / 9 + (u < NPBW % 9 ? 1 : 0); }
template <int NPBW>
constexpr int hs_ps_begin(int u) {
  int s = 0;
  for (int v = 0; v < u; ++v) s += hs_ps<NPBW>(v);
  return s;
}

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
  return (uint32_t)(uintptr_t)(const __attribute__((address_space(3))) char*)p;
}

template <int OFF>
__device__ __forceinline__ void ds_read16(bf16x8& f, uint32_t addr) {
  asm volatile("ds_read_b128 %0, %1 offset:%2" : "=v"(f) : "v"(addr), "i"(OFF));
}

struct HsFrags;
__device__ __forceinline__ void lgkm0_tie(HsFrags& F);

// Compiler scheduling fence: no instruction moves across it.
__device__ __forceinline__ void sched_fence() { __builtin_amdgcn_sched_barrier(0); }
// Keeps the order of the vector-memory instructions on either side.
__device__ __forceinline__ void issue_fence() { __asm__ __volatile__("" ::: "memory"); }

struct HsFrags {
  bf16x8 w[4][2];  // weights (MFMA A operand): k16 step, channel block
  bf16x8 p[4][2];  // pixels (MFMA B operand): k16 step, pixel block
};

// Wait for every LDS read of this wave; F's registers are outputs of the
// wait, so no use of them can be scheduled before it.
__device__ __forceinline__ void lgkm0_tie(HsFrags& F) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(F.w[0][0]), "+v"(F.w[0][1]), "+v"(F.p[0][0]), "+v"(F.p[0][1]));
  asm volatile("" : "+v"(F.w[1][0]), "+v"(F.w[1][1]), "+v"(F.p[1][0]), "+v"(F.p[1][1]));
  asm volatile("" : "+v"(F.w[2][0]), "+v"(F.w[2][1]), "+v"(F.p[2][0]), "+v"(F.p[2][1]));
  asm volatile("" : "+v"(F.w[3][0]), "+v"(F.w[3][1]), "+v"(F.p[3][0]), "+v"(F.p[3][1]));
}

template <int NPB>
__global__ void __launch_bounds__(64 * HS_NW, 1) k_conv_hs(ConvArgs a) {
  static_assert(NPB % HS_NW == 0, "patch blocks per wave");
  constexpr int NPBW = NPB / HS_NW;  // patch DMA instructions per wave and chunk
  constexpr int PATCH = NPB * 1024;
  __shared__ __attribute__((aligned(1024))) char ws0[HS_WSLOT];
  __shared__ __attribute__((aligned(1024))) char ws1[HS_WSLOT];
  __shared__ __attribute__((aligned(1024))) char ws2[HS_WSLOT];
  __shared__ __attribute__((aligned(1024))) char ps0[PATCH];
  __shared__ __attribute__((aligned(1024))) char ps1[PATCH];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int wm = wave & 1, wn = wave >> 1;
  const int lr = lane >> 3, fr = lane & 31, fq = lane >> 5;
  const int H = a.H, W = a.W, PW = W + 2, HP = H + 2, HW = H * W;
  const int CH = a.Cin / BK;  // 64-channel chunks (even)
  const float inv_hw = 1.0f / (float)HW, inv_w = 1.0f / (float)W, inv_pw = 1.0f / (float)PW,
              inv_hp = 1.0f / (float)HP;

  // ---- this workgroup's group (model z, channel tile) and run of pixel tiles;
  // workgroups are numbered XCD by XCD so that a group's workgroups share an
  // L2 (and its weights)
  const int tiles_m = (a.M + HS_BM - 1) / HS_BM;
  const int NT = a.Cout / HS_BN, G = a.Z * NT;
  const int nwg = gridDim.x, base = nwg / G, rem = nwg % G, big = rem * (base + 1);
  const int bx = xcd_remap(blockIdx.x, nwg);
  const int g = bx < big ? bx / (base + 1) : rem + (bx - big) / base;
  const int gi = bx < big ? bx % (base + 1) : (bx - big) % base;
  const int gsize = base + (g < rem ? 1 : 0);
  const int z = g / NT, n0 = (g - z * NT) * HS_BN;
  const int t_begin = (int)((int64_t)gi * tiles_m / gsize), t_end = (int)((int64_t)(gi + 1) * tiles_m / gsize);
  if (t_begin >= t_end) return;  // uniform over the workgroup
  const int pairs_per_tile = CH / 2;

  const __amdgpu_buffer_rsrc_t rx = rsrc(reinterpret_cast<const uint16_t*>(a.x) + z * a.x_mstride,
                                         (uint32_t)((int64_t)a.B * HW * a.Cin * 2));
  const __amdgpu_buffer_rsrc_t rw = rsrc(reinterpret_cast<const uint16_t*>(a.w) + z * a.w_mstride,
                                         (uint32_t)((int64_t)a.Cout * a.Kp * 2));
  const __amdgpu_buffer_rsrc_t ry = rsrc(reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride,
                                         (uint32_t)((int64_t)a.M * a.Cout * 2));
  const bool has_res = a.res != nullptr;
  const __amdgpu_buffer_rsrc_t rr =
      has_res ? rsrc(reinterpret_cast<const uint16_t*>(a.res) + z * a.res_mstride, (uint32_t)((int64_t)a.M * a.Cout * 2))
              : rsrc(a.y, 0u);

  // ---- bias of this lane's output channels (after the permlane32 swap a
  // lane holds channels n0 + 64 wn + 32 j + 8 (2 h + fq) .. +8)
  float bias_v[2][2][8];
  {
    const float* __restrict__ bias = a.bias + z * a.b_mstride;
#pragma unroll
    for (int j = 0; j < 2; ++j)
#pragma unroll
      for (int h = 0; h < 2; ++h) {
        const int n = n0 + wn * 64 + j * 32 + 8 * (2 * h + fq);
        const float4 b0 = *reinterpret_cast<const float4*>(bias + n);
        const float4 b1 = *reinterpret_cast<const float4*>(bias + n + 4);
        bias_v[j][h][0] = b0.x; bias_v[j][h][1] = b0.y; bias_v[j][h][2] = b0.z; bias_v[j][h][3] = b0.w;
        bias_v[j][h][4] = b1.x; bias_v[j][h][5] = b1.y; bias_v[j][h][6] = b1.z; bias_v[j][h][7] = b1.w;
      }
  }  // (complete at the prologue's wait, with the first fetches)

  // ---- weight DMA: instruction i of this wave fills slot rows (4 i + wave) * 8 .. +8
  uint32_t wb[HS_WI];
#pragma unroll
  for (int i = 0; i < HS_WI; ++i) {
    const int n = (i * HS_NW + wave) * 8 + lr;
    const int lc = (lane & 7) ^ swz(n);
    wb[i] = (uint32_t)((((int64_t)(n0 + n)) * a.Kp + lc * 8) * 2);
  }
  auto issue_w = [&](char* slot, int kt) {
    const uint32_t koff = (uint32_t)(kt * BK * 2);
#pragma unroll
    for (int i = 0; i < HS_WI; ++i)
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rw, (lds_void*)(slot + (i * HS_NW + wave) * 1024), 16, wb[i] + koff,
                                               0, 0, 0);
  };

  // ---- patch DMA: instruction v of this wave fills patch block v * 4 + wave;
  // lane's patch pixel q = block * 8 + lr sits at padded (R0 + q / PW, q % PW).
  // Patch rows are swizzled by h = (R - 2 b) W + c for padded row R of image
  // b and padded column c, which is m + ky W + kx for the pixel that output
  // m reads at tap (ky, kx): over the 16 consecutive outputs an operand read
  // serves per cycle, h runs consecutively (across image-row ends and image
  // ends), and the LDS row parity alternates with it, so the rows of each
  // parity class take 8 distinct chunks at every tap.
  int q_pr[NPBW], q_pc[NPBW];
#pragma unroll
  for (int v = 0; v < NPBW; ++v) {
    const int q = (v * HS_NW + wave) * 8 + lr;
    q_pr[v] = fdiv_small(q, inv_pw);
    q_pc[v] = q - q_pr[v] * PW;
  }
  // byte offsets (chunk 0) of this lane's patch pixels for tile t; pixels
  // outside the image get an offset past the range for every chunk
  auto patch_offsets = [&](int t, uint32_t (&po)[NPBW]) {
    const int m0 = t * HS_BM;
    const int b0 = fdiv_small(m0, inv_hw), r0 = m0 - b0 * HW, y0 = fdiv_small(r0, inv_w);
    const int R0 = b0 * HP + y0;  // padded row above the first pixel
#pragma unroll
    for (int v = 0; v < NPBW; ++v) {
      const int R = R0 + q_pr[v];
      const int b = fdiv_small(R, inv_hp), yy = R - b * HP - 1, xx = q_pc[v] - 1;
      const int lc = (lane & 7) ^ ((((R - 2 * b) * W + q_pc[v]) >> 1) & 7);
      const bool ok = b < a.B && (unsigned)yy < (unsigned)H && (unsigned)xx < (unsigned)W;
      po[v] = ok ? (uint32_t)(((((int64_t)b * H + yy) * W + xx) * a.Cin + lc * 8) * 2) : OOB;
    }
  };
  auto issue_slice = [&](auto uc, char* pb, const uint32_t (&po)[NPBW], int cc) {
    constexpr int u = decltype(uc)::value;
    constexpr int v0 = hs_ps_begin<NPBW>(u), nv = hs_ps<NPBW>(u);
#pragma unroll
    for (int v = v0; v < v0 + nv; ++v) {
      const uint32_t off = po[v] + (uint32_t)(cc * BK * 2);  // OOB plus a chunk offset stays past the range
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)(pb + (v * HS_NW + wave) * 1024), 16, off, 0, 0, 0);
    }
  };

  // ---- this lane's two pixels (blocks 2 wm + i) of tile t: top-left patch
  // position q0 and its swizzle key h0 = m (both 0 for pixels past M), and
  // the output row m (-1 past M)
  auto pixel_geom = [&](int t, int (&q0)[2], int (&h0)[2], int (&mg)[2]) {
    const int m0 = t * HS_BM;
    const int b0 = fdiv_small(m0, inv_hw), r0 = m0 - b0 * HW, y0 = fdiv_small(r0, inv_w);
    const int R0 = b0 * HP + y0;
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int m = m0 + (wm * 2 + i) * 32 + fr;
      if (m < a.M) {
        const int b = fdiv_small(m, inv_hw), r = m - b * HW, y = fdiv_small(r, inv_w), x = r - y * W;
        const int prow = b * HP + y - R0;  // patch row of the top-left tap
        q0[i] = prow * PW + x;
        h0[i] = m;
        mg[i] = m;
      } else {
        q0[i] = 0;
        h0[i] = 0;
        mg[i] = -1;
      }
    }
  };

  // ---- operand fragments.  Weights: rows 64 wn + 32 j + fr of a slot; the
  // lane's 16-byte chunk 2 kk + fq sits at physical chunk (2 kk + fq) ^ s,
  // i.e. at ((fq ^ s) << 4) ^ (kk << 5) within the 128-byte row.  Block j = 1
  // is 32 rows (4 KB) further with the same swizzle.
  const int rbw = wn * 64 + fr;
  const uint32_t wu = (uint32_t)(((fq ^ swz(rbw)) << 4) + rbw * ROW);
  const uint32_t wa0 = lds_addr(ws0) + wu, wa1 = lds_addr(ws1) + wu, wa2 = lds_addr(ws2) + wu;
  // The reads are inline assembly so that the compiler neither sinks them
  // next to their MFMAs nor adds waits of its own for the LDS fetches in
  // flight: the step waits (lgkmcnt) for them itself, and that wait carries
  // the registers' dependence to the MFMAs.
  auto read_frags = [&](uint32_t wa, const char* pb, const int (&q0)[2], const int (&h0)[2], int dq, int dh,
                        HsFrags& F, int half) {
    uint32_t pa[2];
#pragma unroll
    for (int i = 0; i < 2; ++i) {
      const int s = ((h0[i] + dh) >> 1) & 7;
      pa[i] = (lds_addr(pb) + (uint32_t)((q0[i] + dq) * ROW)) | (uint32_t)((fq ^ s) << 4);
    }
#pragma unroll
    for (int k2 = 0; k2 < 2; ++k2) {
      const int kk = half * 2 + k2;
      const uint32_t x = (uint32_t)(kk << 5);
      ds_read16<0>(F.w[kk][0], wa ^ x);
      ds_read16<32 * ROW>(F.w[kk][1], wa ^ x);
#pragma unroll
      for (int i = 0; i < 2; ++i) ds_read16<0>(F.p[kk][i], pa[i] ^ x);
    }
  };

  floatx16 acc[2][2];
  auto mma = [&](const HsFrags& F, int kk) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
        acc[i][j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(F.w[kk][j], F.p[kk][i], acc[i][j], 0, 0, 0);
  };

  auto wslot = [&](auto sc) -> char* {
    constexpr int s = decltype(sc)::value % 3;
    if constexpr (s == 0) return ws0;
    else if constexpr (s == 1) return ws1;
    else return ws2;
  };
  auto waddr = [&](auto sc) -> uint32_t {
    constexpr int s = decltype(sc)::value % 3;
    if constexpr (s == 0) return wa0;
    else if constexpr (s == 1) return wa1;
    else return wa2;
  };

  // ---- prologue: chunk 0's patch and the weights of steps 0 and 1; F for
  // step 0; then, as a chunk's last step would, slice 0 of chunk 1, the
  // weights of step 2 and (dropped) stores
  int q0c[2], h0c[2], mgc[2];
  pixel_geom(t_begin, q0c, h0c, mgc);
  uint32_t poA[NPBW], poB[NPBW];
  patch_offsets(t_begin, poA);
  static_for<0, 9>([&](auto uc) { issue_slice(uc, ps0, poA, 0); });
  issue_w(ws0, 0 * CH + 0);
  issue_w(ws1, 1 * CH + 0);
  wait_vmcnt<0>();
  wg_barrier();
  HsFrags Fa, Fb;
  read_frags(wa0, ps0, q0c, h0c, 0, 0, Fa, 0);
  read_frags(wa0, ps0, q0c, h0c, 0, 0, Fa, 1);
  issue_slice(std::integral_constant<int, 0>{}, ps1, poA, 1);
  issue_w(ws2, 2 * CH + 0);
  dummy_stores<HS_SI>(ry);

  uint4 res_v[2][2][2];
  int ge = 0;  // even chunk of the current pair, counted over the workgroup's tiles
  for (int tile = t_begin; tile < t_end; ++tile) {
#pragma unroll
    for (int i = 0; i < 2; ++i)
#pragma unroll
      for (int j = 0; j < 2; ++j)
#pragma unroll
        for (int e = 0; e < 16; ++e) acc[i][j][e] = 0.f;
    for (int pp = 0; pp < pairs_per_tile; ++pp, ge += 2) {
      const int cc_e = 2 * pp, cc_o = cc_e + 1;
      const bool last = pp == pairs_per_tile - 1;  // the odd chunk ends the tile
      const int tile_n = last ? tile + 1 : tile, cc_n = last ? 0 : cc_e + 2;  // the next pair's
      int q0n[2], h0n[2], mgn[2];
      if (last) {
        pixel_geom(tile_n, q0n, h0n, mgn);
        patch_offsets(tile_n, poB);
      } else {
#pragma unroll
        for (int i = 0; i < 2; ++i) {
          q0n[i] = q0c[i];
          h0n[i] = h0c[i];
          mgn[i] = mgc[i];
        }
#pragma unroll
        for (int v = 0; v < NPBW; ++v) poB[v] = poA[v];
      }

      // one step: parity P (0 even chunk, 1 odd), tap t; F = this step's
      // fragments, Fn = the next step's
      auto step = [&](auto Pc, auto tc, HsFrags& F, HsFrags& Fn) {
        constexpr int P = decltype(Pc)::value, t = decltype(tc)::value;
        constexpr int PS_T = hs_ps<NPBW>(t % 9), PS_0 = hs_ps<NPBW>(0), PS_1 = hs_ps<NPBW>(1), PS_2 = hs_ps<NPBW>(2);
        constexpr int ALLOW =
            t == 8 ? HS_WI
            : P == 0 ? (t == 0 ? PS_0 + HS_WI + HS_SI : t == 1 ? HS_SI + PS_1 + HS_WI : PS_T + HS_WI)
                     : (t == 0 ? PS_0 + HS_WI : t == 1 ? PS_1 + HS_WI + HS_RI : t == 2 ? HS_RI + PS_2 + HS_WI : PS_T + HS_WI);
        char* const pcur = P == 0 ? ps0 : ps1;   // this chunk's patch
        char* const pnxt = P == 0 ? ps1 : ps0;   // the next chunk's
        lgkm0_tie(F);  // this step's fragments (read during the last step) are in
        sched_fence();
        mma(F, 0);
        sched_fence();
        wait_vmcnt<ALLOW>();
        wg_barrier();
        // fetches, in this order: patch slice (t + 1) % 9 of the next chunk
        // (of the chunk after it at t = 8), the weights of step s + 3, and
        // at the odd chunk's first step the tile's residual
        if constexpr (t < 8) {
          if constexpr (P == 0) issue_slice(std::integral_constant<int, t + 1>{}, pnxt, poA, cc_o);
          else issue_slice(std::integral_constant<int, t + 1>{}, pnxt, poB, cc_n);
        } else {
          if constexpr (P == 0) issue_slice(std::integral_constant<int, 0>{}, pcur, poB, cc_n);
          else issue_slice(std::integral_constant<int, 0>{}, pcur, poB, cc_n + 1);
        }
        issue_fence();
        {
          constexpr int t3 = t + 3;
          const int cc_this = P == 0 ? cc_e : cc_o, cc_next = P == 0 ? cc_o : cc_n;
          const int kt = t3 <= 8 ? t3 * CH + cc_this : (t3 - 9) * CH + cc_next;
          issue_w(wslot(tc), kt);
        }
        issue_fence();
        if constexpr (P == 1 && t == 0) {  // out of range unless the tile ends with this chunk
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int h = 0; h < 2; ++h) {
                const int n = n0 + wn * 64 + j * 32 + 8 * (2 * h + fq);
                const uint32_t off =
                    (has_res && last && mgc[i] >= 0) ? (uint32_t)(((int64_t)mgc[i] * a.Cout + n) * 2) : OOB;
                res_v[i][j][h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0));
              }
          issue_fence();
        }
        // next step's fragments, read in two halves between this step's
        // MFMAs; the second half has 8 MFMAs to land before the next step
        auto read_next = [&](int half) {
          if constexpr (t < 8)
            read_frags(waddr(std::integral_constant<int, t + 1>{}), pcur, q0c, h0c, ((t + 1) / 3) * PW + (t + 1) % 3,
                       ((t + 1) / 3) * W + (t + 1) % 3, Fn, half);
          else if constexpr (P == 0)
            read_frags(wa0, pnxt, q0c, h0c, 0, 0, Fn, half);
          else
            read_frags(wa0, pnxt, q0n, h0n, 0, 0, Fn, half);
        };
        read_next(0);
        mma(F, 1);
        sched_fence();
        read_next(1);
        mma(F, 2);
        mma(F, 3);
        sched_fence();
        if constexpr (P == 1 && t == 8) {  // epilogue: stores out of range unless the tile ends here
#pragma unroll
          for (int i = 0; i < 2; ++i)
#pragma unroll
            for (int j = 0; j < 2; ++j)
#pragma unroll
              for (int h = 0; h < 2; ++h) {
                const int gp = 2 * h;
                float v[8];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                  const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i][j][gp * 4 + r]),
                                                                   __float_as_uint(acc[i][j][(gp + 1) * 4 + r]), false,
                                                                   false);
                  v[r] = __uint_as_float(sw[0]);
                  v[4 + r] = __uint_as_float(sw[1]);
                }
#pragma unroll
                for (int e = 0; e < 8; ++e) v[e] += bias_v[j][h][e];
                if (has_res) {
                  float rv[8];
                  bf8_to_f8(res_v[i][j][h], rv);
#pragma unroll
                  for (int e = 0; e < 8; ++e) v[e] += rv[e];
                }
                if (a.relu)
#pragma unroll
                  for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
                const int n = n0 + wn * 64 + j * 32 + 8 * (gp + fq);
                const uint32_t off = (last && mgc[i] >= 0) ? (uint32_t)(((int64_t)mgc[i] * a.Cout + n) * 2)
                                                           : OOB + 16u * (uint32_t)((i * 2 + j) * 2 + h);  // distinct: never merged
                __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, f8_to_bf8(v)), ry, off, 0, 0);
              }
        }
      };
      // 18 steps; the fragment sets alternate (Fa holds step 0's on entry)
      static_for<0, 9>([&](auto tc) {
        constexpr int t = decltype(tc)::value;
        if constexpr (t % 2 == 0) step(std::integral_constant<int, 0>{}, tc, Fa, Fb);
        else step(std::integral_constant<int, 0>{}, tc, Fb, Fa);
      });
      static_for<0, 9>([&](auto tc) {
        constexpr int t = decltype(tc)::value;
        if constexpr ((t + 9) % 2 == 0) step(std::integral_constant<int, 1>{}, tc, Fa, Fb);
        else step(std::integral_constant<int, 1>{}, tc, Fb, Fa);
      });
#pragma unroll
      for (int v = 0; v < NPBW; ++v) poA[v] = poB[v];
#pragma unroll
      for (int i = 0; i < 2; ++i) {
        q0c[i] = q0n[i];
        h0c[i] = h0n[i];
        mgc[i] = mgn[i];
      }
    }
  }
  (void)ge;
  wait_vmcnt<0>();  // no LDS fetch may land after the workgroup has left
  asm volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
}

// Patch pixels the tiles of BM output pixels of this layer need: for each
// tile, through its last pixel's bottom-right tap, plus the two rows above
// that pixel's row whose band the first pixel's top taps start.
template <int BM>
int64_t patch_px(const ConvArgs& a) {
  const int64_t HW = (int64_t)a.H * a.W, PW = a.W + 2, HP = a.H + 2;
  const int64_t tiles = (a.M + BM - 1) / BM;
  int64_t need = 0;
  for (int64_t t = 0; t < tiles; ++t) {
    const int64_t m0 = t * BM, m1 = std::min<int64_t>(a.M, m0 + BM) - 1;
    const int64_t R0 = (m0 / HW) * HP + (m0 % HW) / a.W;      // padded row above the first pixel
    const int64_t b1 = m1 / HW, y1 = (m1 % HW) / a.W, x1 = (m1 % HW) % a.W;
    const int64_t q = (b1 * HP + y1 - R0) * PW + x1 + 2 * PW + 2;  // last pixel's bottom-right tap
    need = std::max(need, q + 1);
  }
  return need;
}
int64_t hs_patch_px(const ConvArgs& a) { return patch_px<HS_BM>(a); }

constexpr int HS_NPB[] = {32, 40, 48};  // instantiated patch sizes (8-pixel blocks)

// ------------------------------------------------------------------------
// The same convolution with the weights in registers: one workgroup per tile
// of BM consecutive output pixels x 128 channels, its four waves in one row
// (each all BM pixels x 32 channels), so no wave needs another's weights:
// each loads its fragments of the next tap straight into registers from the
// fragment-ordered copy (conv_frag_order; one 1 KB load per k16 step) while
// the current tap's MFMAs run.  The LDS holds only the input patch of a
// 64-channel chunk, double-buffered: the next chunk's patch loads in nine
// slices during this chunk's taps, and the workgroup meets once per chunk.
// At most 80 KB of LDS and 256 VGPRs, so two workgroups share a CU.  Patch
// geometry and swizzle as above; per output the sum runs over chunks, then
// taps, then the 64 channels in MFMA order, as above, so the bits are the
// same.  Each tap issues the next tap's weights and a ninth of the next
// patch, runs its MFMAs and then waits for those loads.
constexpr int HR_BN = 128;
constexpr int HR_NW = 4;
constexpr int HR_NPB[] = {24, 32, 40};  // instantiated patch sizes (8-pixel blocks)

template <int BM, int NPB>
__global__ void __launch_bounds__(64 * HR_NW, 2) k_conv_hr(ConvArgs a) {
  constexpr int FM = BM / 32;
  static_assert(BM % 32 == 0 && NPB % HR_NW == 0, "tile");
  constexpr int NPBW = NPB / HR_NW;  // patch DMA instructions per wave and chunk
  constexpr int PATCH = NPB * 1024;
  __shared__ __attribute__((aligned(1024))) char ps0[PATCH];
  __shared__ __attribute__((aligned(1024))) char ps1[PATCH];

  const int tid = threadIdx.x, lane = tid & 63;
  const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
  const int lr = lane >> 3, fr = lane & 31, fq = lane >> 5;
  const int H = a.H, W = a.W, PW = W + 2, HP = H + 2, HW = H * W;
  const int CH = a.Cin / BK;  // 64-channel chunks (even)
  const float inv_hw = 1.0f / (float)HW, inv_w = 1.0f / (float)W, inv_pw = 1.0f / (float)PW,
              inv_hp = 1.0f / (float)HP;

  // ---- tile: N tiles vary fastest, XCD-contiguous
  const int tiles_m = (a.M + BM - 1) / BM, NT = a.Cout / HR_BN;
  const int id = xcd_remap(blockIdx.x, tiles_m * NT * a.Z);
  const int nt = id % NT, mz = id / NT, mt = mz % tiles_m, z = mz / tiles_m;
  const int m0 = mt * BM, n0 = nt * HR_BN, nw = n0 + wave * 32;

  const __amdgpu_buffer_rsrc_t rx = rsrc(reinterpret_cast<const uint16_t*>(a.x) + z * a.x_mstride,
                                         (uint32_t)((int64_t)a.B * HW * a.Cin * 2));
  const __amdgpu_buffer_rsrc_t rwf = rsrc(reinterpret_cast<const uint16_t*>(a.wf) + z * a.wf_mstride,
                                          (uint32_t)((int64_t)a.Cout * a.Kp * 2));
  const __amdgpu_buffer_rsrc_t ry = rsrc(reinterpret_cast<uint16_t*>(a.y) + z * a.y_mstride,
                                         (uint32_t)((int64_t)a.M * a.Cout * 2));
  const bool has_res = a.res != nullptr;
  const __amdgpu_buffer_rsrc_t rr =
      has_res ? rsrc(reinterpret_cast<const uint16_t*>(a.res) + z * a.res_mstride, (uint32_t)((int64_t)a.M * a.Cout * 2))
              : rsrc(a.y, 0u);

  // ---- this lane's pixels m = m0 + 32 i + fr: top-left patch position q0
  // (the swizzle key and the output row are m itself; 0 / none past M)
  const int b0 = fdiv_small(m0, inv_hw), r0 = m0 - b0 * HW, y0 = fdiv_small(r0, inv_w);
  const int R0 = b0 * HP + y0;  // padded row above the first pixel
  int q0[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i) {
    const int m = m0 + i * 32 + fr;
    if (m < a.M) {
      const int b = fdiv_small(m, inv_hw), r = m - b * HW, y = fdiv_small(r, inv_w), x = r - y * W;
      q0[i] = (b * HP + y - R0) * PW + x;
    } else {
      q0[i] = 0;
    }
  }

  // ---- weights: tap t of chunk c is K-tile t * CH + c; fragment block of
  // this wave's 32 channels, k16 step s of that K-tile: 1 KB at
  // ((nw / 32) * Kp / 16 + 4 kt + s) KB, this lane's 16 bytes at lane * 16
  const uint32_t wbase = (uint32_t)((int64_t)(nw / 32) * (a.Kp / 16) * 1024 + lane * 16);
  auto load_w = [&](int kt, uint4 (&v)[4]) {
#pragma unroll
    for (int k = 0; k < 4; ++k)
      v[k] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rwf, wbase + (uint32_t)(kt * 4 + k) * 1024u, 0, 0));
  };

  // ---- patch DMA: instruction v of this wave fills block v * 4 + wave; the
  // lane's pixel q = block * 8 + lr sits at padded (R0 + q / PW, q % PW)
  uint32_t po[NPBW];
#pragma unroll
  for (int v = 0; v < NPBW; ++v) {
    const int q = (v * HR_NW + wave) * 8 + lr;
    const int pr = fdiv_small(q, inv_pw), pc = q - pr * PW;
    const int R = R0 + pr;
    const int b = fdiv_small(R, inv_hp), yy = R - b * HP - 1, xx = pc - 1;
    const int lc = (lane & 7) ^ ((((R - 2 * b) * W + pc) >> 1) & 7);
    const bool ok = b < a.B && (unsigned)yy < (unsigned)H && (unsigned)xx < (unsigned)W;
    po[v] = ok ? (uint32_t)(((((int64_t)b * H + yy) * W + xx) * a.Cin + lc * 8) * 2) : OOB;
  }
  auto issue_slice = [&](auto uc, char* pb, int cc) {
    constexpr int u = decltype(uc)::value;
    constexpr int v0 = hs_ps_begin<NPBW>(u), nv = hs_ps<NPBW>(u);
#pragma unroll
    for (int v = v0; v < v0 + nv; ++v) {
      const uint32_t off = po[v] == OOB ? OOB : po[v] + (uint32_t)(cc * BK * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx, (lds_void*)(pb + (v * HR_NW + wave) * 1024), 16, off, 0, 0, 0);
    }
  };

  // ---- projection shortcut (a.x2): after the 3x3 reduction, Cin2 / 64 more
  // K-tiles of the 1x1 conv of x2 at (oy s2, ox s2), each a plain tile of BM
  // pixel rows x 64 channels loaded into a patch buffer (instruction i of
  // this wave fills rows (4 i + wave) * 8 .. +8; the lane's 16-byte chunk
  // lands at chunk (lane & 7) of its row, holding channels ((lane & 7) ^
  // swz(row)) * 8 .., as in the implicit GEMM)
  const int NP = a.x2 ? a.Cin2 / BK : 0;
  const __amdgpu_buffer_rsrc_t rx2 =
      rsrc(a.x2 ? reinterpret_cast<const uint16_t*>(a.x2) + z * a.x2_mstride : reinterpret_cast<const uint16_t*>(a.x),
           a.x2 ? (uint32_t)((int64_t)a.B * a.H2 * a.W2 * a.Cin2 * 2) : 0u);
  uint32_t p2[FM];
  if (NP > 0) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const int row = (i * HR_NW + wave) * 8 + lr, m = m0 + row;
      const int lc = (lane & 7) ^ swz(row);
      if (m < a.M) {
        const int b = fdiv_small(m, inv_hw), r = m - b * HW, y = fdiv_small(r, inv_w), x = r - y * W;
        p2[i] = (uint32_t)(((((int64_t)b * a.H2 + y * a.stride2) * a.W2 + x * a.stride2) * a.Cin2 + lc * 8) * 2);
      } else {
        p2[i] = OOB;
      }
    }
  }
  auto issue_proj = [&](char* pb, int j) {
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      const uint32_t off = p2[i] == OOB ? OOB : p2[i] + (uint32_t)(j * BK * 2);
      __builtin_amdgcn_raw_ptr_buffer_load_lds(rx2, (lds_void*)(pb + (i * HR_NW + wave) * 1024), 16, off, 0, 0, 0);
    }
  };

  floatx16 acc[FM];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int e = 0; e < 16; ++e) acc[i][e] = 0.f;

  // one projection K-tile: rows 32 i + fr of the tile, weights from wv
  auto proj_mma = [&](const char* pb, const uint4 (&wv)[4]) {
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 pf[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i) {
        const int row = i * 32 + fr;
        pf[i] = *reinterpret_cast<const bf16x8*>(pb + row * ROW + (((2 * kk + fq) ^ swz(row)) << 4));
      }
#pragma unroll
      for (int i = 0; i < FM; ++i)
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wv[kk]), pf[i], acc[i], 0, 0, 0);
    }
  };

  // one tap: pixel fragments from the patch (row q0 + ky PW + kx, swizzle
  // key h0 + ky W + kx), weight fragments from wv
  auto tap_mma = [&](const char* pb, int t, const uint4 (&wv)[4]) {
    const int ky = t / 3, kx = t - ky * 3;
    const int dq = ky * PW + kx, dh = ky * W + kx;
    // (recomputed per tap: the compiler would otherwise keep all 18 taps'
    // addresses of a chunk pair in registers across the chunk loop)
    uint32_t pa[FM];
#pragma unroll
    for (int i = 0; i < FM; ++i) {
      int q = q0[i], m = m0 + i * 32 + fr;
      asm volatile("" : "+v"(q), "+v"(m));
      const int sw = (((m < a.M ? m : 0) + dh) >> 1) & 7;
      pa[i] = (uint32_t)((q + dq) * ROW) | (uint32_t)((fq ^ sw) << 4);
    }
#pragma unroll
    for (int kk = 0; kk < 4; ++kk) {
      bf16x8 pf[FM];
#pragma unroll
      for (int i = 0; i < FM; ++i) pf[i] = *reinterpret_cast<const bf16x8*>(pb + (pa[i] ^ (uint32_t)(kk << 5)));
#pragma unroll
      for (int i = 0; i < FM; ++i)
        acc[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, wv[kk]), pf[i], acc[i], 0, 0, 0);
    }
  };

  // one chunk: nine taps; at tap t the next tap's weights and slice t of
  // the next chunk's patch are issued (after the last chunk: the first
  // projection K-tile and its weights), then this tap's MFMAs run, then the
  // wave waits for what it issued; the workgroup meets after the last tap
  uint4 wA[4], wB[4];
  auto chunk = [&](int cc, const char* pcur, char* pnxt, auto par) {
    constexpr int P0 = decltype(par)::value;  // register set of tap 0: 0 = wA, 1 = wB
    const bool more = cc + 1 < CH, proj = !more && NP > 0;
    static_for<0, 9>([&](auto tc) {
      constexpr int t = decltype(tc)::value;
      constexpr bool inA = ((P0 + t) & 1) == 0;
      if (more) issue_slice(tc, pnxt, cc + 1);
      if constexpr (t == 0) {
        if (proj) issue_proj(pnxt, 0);
      }
      if (t < 8) {
        if constexpr (inA) load_w((t + 1) * CH + cc, wB);
        else load_w((t + 1) * CH + cc, wA);
      } else if (more || proj) {
        const int kt = more ? cc + 1 : 9 * CH;  // the next chunk's tap 0, or the first projection K-tile
        if constexpr (inA) load_w(kt, wB);
        else load_w(kt, wA);
      }
      if constexpr (inA) tap_mma(pcur, t, wA);
      else tap_mma(pcur, t, wB);
      wait_vmcnt<0>();
    });
    wg_barrier();
  };

  // prologue: chunk 0's patch, tap 0's weights
  static_for<0, 9>([&](auto uc) { issue_slice(uc, ps0, 0); });
  load_w(0, wA);
  wait_vmcnt<0>();
  wg_barrier();
  for (int cc = 0; cc < CH; cc += 2) {  // chunks in pairs: the patch buffers and register sets by name
    chunk(cc, ps0, ps1, std::integral_constant<int, 0>{});
    chunk(cc + 1, ps1, ps0, std::integral_constant<int, 1>{});
  }
  // the projection K-tiles (CH is even: the first is in ps0 and wA), each
  // with the next one's tile and weights in flight; every wave waits for
  // its loads, and the workgroup meets before a tile is read and before its
  // buffer is refilled
  auto pstep = [&](int j, const char* pcur, char* pnxt, const uint4 (&wc)[4], uint4 (&wn)[4]) {
    if (j + 1 < NP) {
      issue_proj(pnxt, j + 1);
      load_w(9 * CH + j + 1, wn);
    }
    proj_mma(pcur, wc);
    wait_vmcnt<0>();
    wg_barrier();
  };
  for (int j = 0; j < NP; j += 2) {
    pstep(j, ps0, ps1, wA, wB);
    if (j + 1 < NP) pstep(j + 1, ps1, ps0, wB, wA);
  }

  // ---- epilogue: bias, residual, ReLU, bf16, 16-byte stores (after the
  // permlane32 swap a lane holds channels nw + 8 (2 h + fq) .. +8 of pixel
  // m0 + 32 i + fr); the residual and the bias are loaded here, every
  // register of the loop being taken by the operands
  uint4 res_v[FM][2];
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int m = m0 + i * 32 + fr, n = nw + 8 * (2 * h + fq);
      const uint32_t off = (has_res && m < a.M) ? (uint32_t)(((int64_t)m * a.Cout + n) * 2) : OOB;
      res_v[i][h] = __builtin_bit_cast(uint4, __builtin_amdgcn_raw_buffer_load_b128(rr, off, 0, 0));
    }
  float bias_v[2][8];
  {
    const float* __restrict__ bias = a.bias + z * a.b_mstride;
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int n = nw + 8 * (2 * h + fq);
      const float4 c0 = *reinterpret_cast<const float4*>(bias + n);
      const float4 c1 = *reinterpret_cast<const float4*>(bias + n + 4);
      bias_v[h][0] = c0.x; bias_v[h][1] = c0.y; bias_v[h][2] = c0.z; bias_v[h][3] = c0.w;
      bias_v[h][4] = c1.x; bias_v[h][5] = c1.y; bias_v[h][6] = c1.z; bias_v[h][7] = c1.w;
    }
  }
#pragma unroll
  for (int i = 0; i < FM; ++i)
#pragma unroll
    for (int h = 0; h < 2; ++h) {
      const int gp = 2 * h;
      const int mgi = m0 + i * 32 + fr;
      float v[8];
#pragma unroll
      for (int r = 0; r < 4; ++r) {
        const auto sw = __builtin_amdgcn_permlane32_swap(__float_as_uint(acc[i][gp * 4 + r]),
                                                         __float_as_uint(acc[i][(gp + 1) * 4 + r]), false, false);
        v[r] = __uint_as_float(sw[0]);
        v[4 + r] = __uint_as_float(sw[1]);
      }
#pragma unroll
      for (int e = 0; e < 8; ++e) v[e] += bias_v[h][e];
      if (has_res) {
        float rv[8];
        bf8_to_f8(res_v[i][h], rv);
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] += rv[e];
      }
      if (a.relu)
#pragma unroll
        for (int e = 0; e < 8; ++e) v[e] = v[e] > 0.f ? v[e] : 0.f;
      const int n = nw + 8 * (gp + fq);
      if (mgi < a.M)
        __builtin_amdgcn_raw_buffer_store_b128(__builtin_bit_cast(v4u, f8_to_bf8(v)), ry,
                                               (uint32_t)(((int64_t)mgi * a.Cout + n) * 2), 0, 0);
    }
}

}  // namespace

// A 3x3/1 layer carrying a projection shortcut, in the register-weight
// form: the 3x3 part as conv_hs_ok requires, then whole 64-channel K-tiles
// of the shortcut's input at (oy s2, ox s2).
static bool hr_proj_shape_ok(const ConvArgs& a) {
  if (!a.x2) return false;
  ConvArgs m = a;  // the 3x3 part alone
  m.x2 = nullptr;
  m.K = m.Kp = a.K1;
  return conv_hs_ok(m) && a.K1 == 9 * a.Cin && a.Cin2 % BK == 0 && a.K1 + a.Cin2 == a.K && a.K == a.Kp &&
         (a.Ho - 1) * a.stride2 < a.H2 && (a.Wo - 1) * a.stride2 < a.W2 &&
         (int64_t)a.B * a.H2 * a.W2 * a.Cin2 * 2 < (1ll << 31) && (int64_t)a.Cout * a.Kp * 2 < (1ll << 31);
}

bool conv_hs_ok(const ConvArgs& a) {
  if (!(!a.x2 && a.kh == 3 && a.kw == 3 && a.stride == 1 && a.pad == 1 && a.Cin % (2 * BK) == 0 && a.K == a.Kp &&
        a.Kp == 9 * a.Cin && a.Ho == a.H && a.Wo == a.W && a.Cout % HS_BN == 0))
    return false;
  if ((int64_t)a.B * (a.H + 2) * (a.W + 2) + 1024 >= (1 << 22)) return false;  // fdiv range
  if ((int64_t)a.B * a.H * a.W * a.Cin * 2 >= (1ll << 31) || (int64_t)a.Cout * a.Kp * 2 >= (1ll << 31)) return false;
  return hs_patch_px(a) <= 8 * HS_NPB[2];
}

// The family (the 128 x 128 tiles above and the register-weight form below)
// takes every 3x3/1 layer it fits: fetching each input pixel once per
// 64-channel chunk rather than once per tap beats the implicit GEMM there.
// Shape-only, so a layer's kernel family, and with it the bits of its
// results, never depends on the device or the batch.
bool conv_hs_chosen(const ConvArgs& a) { return conv_hs_ok(a) || hr_proj_shape_ok(a); }

// The register-weight form needs the fragment-ordered weights and a patch of
// at most 40 KB (two buffers per workgroup, two workgroups per CU); it also
// takes a projection shortcut.
bool conv_hr_ok(const ConvArgs& a, int bm) {
  if (!(conv_hs_ok(a) || hr_proj_shape_ok(a)) || !a.wf) return false;
  const int64_t need = bm == 160 ? patch_px<160>(a) : bm == 96 ? patch_px<96>(a) : -1;
  return need >= 0 && need <= 8 * HR_NPB[2];
}

void launch_conv_hr(const ConvArgs& a_in, int bm, hipStream_t s) {
  ConvArgs a = a_in;
  a.split = 1;
  a.partial = nullptr;
  const int64_t need = bm == 160 ? patch_px<160>(a) : patch_px<96>(a);
  int npb = 0;
  for (int c : HR_NPB)
    if (need <= 8 * c) { npb = c; break; }
  const int wgs = ((a.M + bm - 1) / bm) * (a.Cout / HR_BN) * a.Z;
#define FS_HR(BMv, NPBv)                                                                              \
  if (bm == BMv && npb == NPBv) {                                                                     \
    hipLaunchKernelGGL((k_conv_hr<BMv, NPBv>), dim3(wgs), dim3(64 * HR_NW), 0, s, a);                 \
    return;                                                                                           \
  }
  FS_HR(160, 24) FS_HR(160, 32) FS_HR(160, 40)
  FS_HR(96, 24) FS_HR(96, 32) FS_HR(96, 40)
#undef FS_HR
}

void launch_conv_hs(const ConvArgs& a_in, hipStream_t s) {
  ConvArgs a = a_in;  // outputs are always finished here: no K split
  a.split = 1;
  a.partial = nullptr;
  const int64_t need = hs_patch_px(a);
  int npb = 0;
  for (int c : HS_NPB)
    if (need <= 8 * c) { npb = c; break; }
  const int groups = a.Z * (a.Cout / HS_BN);
  const int tiles = ((a.M + HS_BM - 1) / HS_BM) * groups;
  int dev = 0, cus = 256;
  if (hipGetDevice(&dev) == hipSuccess) {
    int n = 0;
    if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) == hipSuccess && n > 0) cus = n;
  }
  const int nwg = std::max(groups, std::min(tiles, cus));
  switch (npb) {
    case 32: hipLaunchKernelGGL((k_conv_hs<32>), dim3(nwg), dim3(64 * HS_NW), 0, s, a); break;
    case 40: hipLaunchKernelGGL((k_conv_hs<40>), dim3(nwg), dim3(64 * HS_NW), 0, s, a); break;
    case 48: hipLaunchKernelGGL((k_conv_hs<48>), dim3(nwg), dim3(64 * HS_NW), 0, s, a); break;
    default: break;  // conv_hs_ok rejects the layer
  }
}

}  // namespace fs
