// Internal declarations shared by the HIP kernels and the host runtime of the
// ensemble library.  gfx950 (CDNA4) only: 64-lane wavefronts, MFMA, 160 KB LDS.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <stddef.h>

namespace fs {

using bf16_t = uint16_t;  // bfloat16 bits in memory

enum Prec { F32 = 0, BF16 = 1 };

// ---------------------------------------------------------------- preprocess
struct ImageDesc {  // mirrors fs_image_desc
  uint64_t offset;
  int32_t h, w, row_stride, reserved;
};

struct PreArgs {
  const uint8_t* pixels;
  const ImageDesc* desc;
  int B, out_h, out_w;
  float mean[3], std_[3];
  float inv_std[3];  // 1 / std_, set by launch_preprocess
  void* out;      // [B][out_h][out_w][4], bf16 or fp32, or null
  void* out_s2d;  // bf16 [B][out_h/2][out_w/2][16] space-to-depth layout, or null:
                  // channel (sy*2 + sx)*3 + c holds pixel (2Y+sy, 2X+sx), channel c;
                  // channels 12..15 are zero
};
void launch_preprocess(const PreArgs& a, Prec p, hipStream_t s);

// ---------------------------------------------------------------------- conv
// Implicit GEMM: rows m = (b, oy, ox), columns n = output channel,
// reduction k = (ky, kx, ci) with ci fastest.  Z models share a launch; each
// tensor of model z sits at base + z * mstride (elements).
struct ConvArgs {
  const void* x;   int64_t x_mstride;    // [B][H][W][Cin]  (Cin = channel stride)
  const void* w;   int64_t w_mstride;    // packed [Cout][Kp]
  const float* bias; int64_t b_mstride;  // [Cout]
  const void* res; int64_t res_mstride;  // [B][Ho][Wo][Cout] or null
  void* y;         int64_t y_mstride;    // [B][Ho][Wo][Cout]
  int B, H, W, Cin, Ho, Wo, Cout;
  int kh, kw, stride, pad, relu;
  int K, Kp, M, Z;
  int split = 1;            // K split over workgroups (LDS-DMA kernels only)
  float* partial = nullptr; // split > 1: fp32 partial sums [split][Z][M][Cout]
  // A residual block's projection shortcut summed into this conv (bf16
  // LDS-DMA kernels only): reduction indices K1 .. K-1 are the 1x1 conv of
  // x2 [B][H2][W2][Cin2] at pixel (oy * stride2, ox * stride2), channel
  // k - K1; the packed weight rows hold both parts.  x2 == null: none.
  const void* x2 = nullptr; int64_t x2_mstride = 0;
  int H2 = 0, W2 = 0, Cin2 = 0, stride2 = 1, K1 = 0;
  // The packed bf16 weights again in MFMA fragment order (conv_frag_order),
  // for the LDS-DMA tiles that load their weights into registers; null: the
  // kernels stage the weights through LDS.
  const void* wf = nullptr; int64_t wf_mstride = 0;
};
// Fragment order of packed bf16 conv weights w [Cout][Kp] (Cout % 32 == 0,
// Kp % 16 == 0): for 32-channel block nb and k16 step s, 64 lanes x 8 values
// at ((nb * Kp / 16 + s) * 64 + l) * 8, lane l holding w[32 nb + l % 32]
// [16 s + 8 (l / 32) .. +8]: the operand one v_mfma_f32_32x32x16_bf16 lane
// takes for those channels and that k16 step.
void conv_frag_order(const uint16_t* w, int Cout, int Kp, uint16_t* out);
inline bool conv_frag_wanted(Prec p, int Cout, int Kp) { return p == BF16 && Cout % 32 == 0 && Kp % 16 == 0; }
struct ConvTile {
  int bm, bn, vec;   // block tile and A-load vector (elements)
  const char* name;
  int dma = 0;       // 0: register-staged gather kernel; >0: LDS-DMA kernel with this many stages
  int waves = 4;     // LDS-DMA kernel: waves per workgroup
  int wgm = 2;       // LDS-DMA kernel: waves along M
  int halo = 0;      // 1: direct 3x3 kernel with the input halo and the weights in LDS,
  int th = 0, tw = 0;  //    tiles of th output rows x tw (= output width) columns;
                       // 2: direct 3x3 kernel, input halo in LDS, weights streamed per tap
};
// Every LDS-DMA tile shares one MFMA step and K order, so all of them
// produce bit-identical sums.
inline bool conv_tile_direct(const ConvTile& c) { return c.dma > 0; }
// Kernel family of a tile: 3 halo with streamed weights, 2 halo with resident
// weights, 1 LDS-DMA implicit GEMM, 0 register-staged implicit GEMM.  A layer
// always runs in the highest family that fits it, and tiles are only ever
// compared within one family.
inline int conv_tile_family(const ConvTile& c) { return c.halo >= 2 ? 3 : c.halo ? 2 : (c.dma > 0 ? 1 : 0); }
int conv_num_tiles(Prec p);
const ConvTile& conv_tile(Prec p, int t);
int conv_pick_tile(Prec p, const ConvArgs& a, int num_cus);
bool conv_tile_ok(Prec p, int t, const ConvArgs& a);         // the tile's kernel can run the layer
bool conv_tile_candidate(Prec p, int t, const ConvArgs& a);  // ... and is among its automatic choices
bool conv_dma_ok(const ConvArgs& a);
void launch_conv_dma(const ConvArgs& a, int bm, int bn, int waves, int wgm, int stages, hipStream_t s);
bool conv_halo_ok(const ConvArgs& a, int th, int tw, int bn);
bool conv_hs_ok(const ConvArgs& a);      // the streamed-weight halo kernel can run the layer
bool conv_hs_chosen(const ConvArgs& a);  // ... and is its automatic choice
void launch_conv_hs(const ConvArgs& a, hipStream_t s);
bool conv_hr_ok(const ConvArgs& a, int bm);  // ... in its register-weight form, tiles of bm pixels
void launch_conv_hr(const ConvArgs& a, int bm, hipStream_t s);
// Space-to-depth ResNet stem (4x4/1/p2 on 16 channels, 64 outputs, ReLU)
// fused with the following 3x3/2/p1 max pool; y receives the pooled tensor.
bool conv_stem_pool_ok(const ConvArgs& a);
void launch_conv_stem_pool(const ConvArgs& a, hipStream_t s);
void launch_conv_halo(const ConvArgs& a, int th, int tw, int bn, hipStream_t s);
void launch_conv(const ConvArgs& a, Prec p, int tile, hipStream_t s,
                 bool reduce = true);  // 1 or 2 launches (split-K reduce unless !reduce)
// Split-K completion fused with a following global average pool (bf16):
// gy [Z][B][Cout] receives the pooled activations, which are not stored.
bool conv_reduce_gap_ok(const ConvArgs& a);
void launch_conv_splitk_reduce_gap(const ConvArgs& a, void* gy, int64_t gy_mstride, hipStream_t s);
int conv_split(Prec p, const ConvArgs& a, int num_cus);
size_t conv_partial_floats(const ConvArgs& a);
void launch_conv_splitk_reduce(const ConvArgs& a, hipStream_t s);
constexpr int CONV_KPAD = 64;  // packed reduction length is a multiple of this

// ------------------------------------------------------------------- pooling
struct PoolArgs {
  const void* x; int64_t x_mstride;
  void* y;       int64_t y_mstride;
  int B, H, W, C, Ho, Wo, k, stride, pad, Z;
};
void launch_maxpool(const PoolArgs& a, Prec p, hipStream_t s);
void launch_gap(const PoolArgs& a, Prec p, hipStream_t s);

// ------------------------------------------------------------------------ fc
struct FcArgs {
  const void* x;   int64_t x_mstride;    // [B][K] storage type
  const void* w;   int64_t w_mstride;    // [N][K] storage type
  const float* bias; int64_t b_mstride;  // [N]
  void* y;         int64_t y_mstride;    // [B][N]: fp32 if out_f32 else storage type
  float* partial;                        // split-K scratch [split][Z][B][N] fp32
  int B, K, N, relu, out_f32, split, Z;
};
int fc_pick_split(Prec p, int B, int K, int N, int Z, int num_cus);
size_t fc_partial_floats(int B, int N, int split, int Z);
void launch_fc(const FcArgs& a, Prec p, hipStream_t s);  // 1 or 2 launches (split-K reduce)
int fc_launches(int split);

// ------------------------------------------------------- softmax + combine
struct SoftmaxArgs {
  const float* logits;  // [N][B][C]
  float* probs;         // [N][B][C]
  float* mean;          // [B][C] or null
  int32_t* vote;        // [B]
  int32_t* top1;        // [N][B] or null
  int N, B, C;
  int policy = 0;       // fs_combine of vote
  int pos_class = 0;    // FS_COMBINE_ANY: the designated class
  int min_votes = 1;    // FS_COMBINE_ANY: models that must detect it
};
constexpr int SOFTMAX_MAX_C = 4096;
constexpr int COMBINE_MAX_PLURALITY = 64;  // most models FS_COMBINE_PLURALITY takes
void launch_softmax_combine(const SoftmaxArgs& a, hipStream_t s);

}  // namespace fs
