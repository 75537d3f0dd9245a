// Host runtime behind the C ABI: validation, weight preparation (batch-norm
// fold, packing, bf16 conversion, one weight arena), the ensemble plan
// (homogeneous models grouped so one launch per layer serves all of them,
// activation slots reused by liveness), the device pass, host staging, and
// the per-kernel event profiler.
//
// FlexServe (Fig. 1 caption; Sec. 2.2): all models live in one device memory
// and consume ONE transformed copy of the request's images; the batch size
// varies per request (Sec. 2.3); every model's per-image output is returned
// together with a combined result.
#include "flexserve.h"
#include "common.hpp"

#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <functional>
#include <map>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

namespace {

using namespace fs;

struct Error {
  fs_status st;
  std::string msg;
};
[[noreturn]] void fail(fs_status st, const std::string& msg) { throw Error{st, msg}; }

void hipchk(hipError_t e, const char* what) {
  if (e == hipSuccess) return;
  fail(e == hipErrorOutOfMemory ? FS_ERR_OOM : FS_ERR_DEVICE,
       std::string(what) + ": " + hipGetErrorString(e));
}
#define HIPCHK(x) hipchk((x), #x)

thread_local std::string g_thread_error;

// Round to nearest even fp32 -> bf16 on the host (weights).
uint16_t host_bf16(float f) {
  uint32_t u;
  std::memcpy(&u, &f, 4);
  if ((u & 0x7f800000u) == 0x7f800000u) return (u & 0x007fffffu) ? uint16_t((u >> 16) | 0x40) : uint16_t(u >> 16);
  u += 0x7fffu + ((u >> 16) & 1u);
  return uint16_t(u >> 16);
}
float host_bf16_to_f(uint16_t h) {
  uint32_t u = uint32_t(h) << 16;
  float f;
  std::memcpy(&f, &u, 4);
  return f;
}

size_t round_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

// ------------------------------------------------------------ device memory
struct DevBuf {  // owns one device allocation; movable, not copyable
  void* p = nullptr;
  size_t bytes = 0;
  DevBuf() = default;
  DevBuf(const DevBuf&) = delete;
  DevBuf& operator=(const DevBuf&) = delete;
  DevBuf(DevBuf&& o) noexcept : p(o.p), bytes(o.bytes) { o.p = nullptr; o.bytes = 0; }
  DevBuf& operator=(DevBuf&& o) noexcept {
    if (this != &o) {
      release();
      p = o.p; bytes = o.bytes;
      o.p = nullptr; o.bytes = 0;
    }
    return *this;
  }
  void alloc(size_t n) {
    release();
    if (n == 0) return;
    HIPCHK(hipMalloc(&p, n));
    bytes = n;
  }
  void ensure(size_t n) {
    if (n > bytes) alloc(n);
  }
  void release() {
    if (p) (void)hipFree(p);
    p = nullptr;
    bytes = 0;
  }
  ~DevBuf() { release(); }
};

struct HostBuf {  // pinned; not copyable
  void* p = nullptr;
  size_t bytes = 0;
  HostBuf() = default;
  HostBuf(const HostBuf&) = delete;
  HostBuf& operator=(const HostBuf&) = delete;
  void ensure(size_t n) {
    if (n <= bytes) return;
    release();
    HIPCHK(hipHostMalloc(&p, n, hipHostMallocDefault));
    bytes = n;
  }
  void release() {
    if (p) (void)hipHostFree(p);
    p = nullptr;
    bytes = 0;
  }
  ~HostBuf() { release(); }
};

// ------------------------------------------------------------------- plan
struct Shape {
  int H = 0, W = 0, C = 0;
  int64_t elems() const { return (int64_t)H * W * C; }
};

enum { SLOT_INPUT = -2, SLOT_LOGITS = -3 };

struct LayerPlan {
  int op = 0, src = -1, res = -1;
  Shape in, out;
  int cin_p = 0;  // channel stride of the input tensor
  int kh = 1, kw = 1, stride = 1, pad = 0, relu = 0, flatten = 0;
  int K = 0, Kp = 0;
  size_t w_off = 0, b_off = 0;  // bytes into the arena (model 0)
  int64_t w_melems = 0, b_melems = 0;
  size_t wf_off = 0;      // bf16 conv: the weights again in MFMA fragment order (model 0), if has_wf
  bool has_wf = false;
  int in_slot = SLOT_INPUT, res_slot = -1, out_slot = -1;
  bool last = false;
  bool s2d = false;       // first conv rewritten on the space-to-depth input
  bool pool_fused = false;  // conv: also applies the next layer's 3x3/2 max pool, writes the pooled tensor
  bool fused_away = false;  // max pool: done by the conv before it (no launch, shares its slot)
  bool gap_only = false;    // conv whose only reader is the global average pool right after it
  // projection shortcut (bf16): a 1x1 conv read only as the residual of one
  // later conv is computed inside that conv's launch as the tail of its
  // reduction (never stored); proj_into: that conv, on the shortcut;
  // proj: the shortcut, on the conv, with the shortcut's input
  int proj_into = -1, proj = -1;
  int proj_slot = -1, proj_cin = 0, proj_stride = 1;
  Shape proj_in;
  int kreal = 0;          // kh * kw * cin of the layer as specified (FLOP count)
  int in_c_real = 0;      // input channels as specified (byte count)
};

struct Group {
  int first = 0, Z = 1;
  std::vector<LayerPlan> layers;
  std::vector<int64_t> slot_elems;  // per image, per model
  std::vector<DevBuf> slots;        // [Z][max_batch][slot_elems]
  // with one stream per group: the group's own stream, end-of-group event
  // and split-K scratch (groups then run concurrently)
  hipStream_t stream = nullptr;
  hipEvent_t done = nullptr;
  DevBuf conv_partial, fc_partial;
};

enum KClass { K_PRE = 0, K_CONV, K_MAXPOOL, K_GAP, K_FC, K_SOFTMAX, K_NCLASS };
const char* kClassName[K_NCLASS] = {"preprocess", "conv", "maxpool", "gap", "fc", "softmax_combine"};

struct ProfRec {
  int cls;
  hipEvent_t a, b;
  double flops, bytes;
  int launches;
  int group, layer, M, N, K, Z;
  const char* kernel;
};

}  // namespace

namespace fs {
namespace {

// Helper threads for the host side of fs_infer: copying the caller's images
// into the pinned staging buffer (several MB at B = 32) is its largest host
// cost.  run(n, f) calls f(0) .. f(n - 1), each once, spread over the
// helpers and the calling thread, and returns when all have returned; f must
// not throw.  One run at a time (the ensemble's lock is held).
class HostPool {
 public:
  explicit HostPool(int helpers) {
    try {
      for (int i = 0; i < helpers; ++i) th_.emplace_back([this] { work(); });
    } catch (...) {  // fewer helpers (or none): the caller does the rest
    }
  }
  ~HostPool() {
    {
      std::lock_guard<std::mutex> lk(mu_);
      stop_ = true;
    }
    go_.notify_all();
    for (std::thread& t : th_) t.join();
  }
  void run(int n, const std::function<void(int)>& f) {
    std::unique_lock<std::mutex> lk(mu_);
    job_ = &f;
    parts_ = n;
    next_ = done_ = 0;
    ++gen_;
    go_.notify_all();
    take(lk);
    done_cv_.wait(lk, [&] { return done_ == parts_; });
    job_ = nullptr;
    parts_ = next_ = done_ = 0;
  }

 private:
  void take(std::unique_lock<std::mutex>& lk) {
    while (next_ < parts_) {
      const int i = next_++;
      const std::function<void(int)>* f = job_;
      lk.unlock();
      (*f)(i);
      lk.lock();
      if (++done_ == parts_) done_cv_.notify_all();
    }
  }
  void work() {
    std::unique_lock<std::mutex> lk(mu_);
    uint64_t seen = 0;
    for (;;) {
      go_.wait(lk, [&] { return stop_ || (gen_ != seen && next_ < parts_); });
      if (stop_) return;
      seen = gen_;
      take(lk);
    }
  }
  std::vector<std::thread> th_;
  std::mutex mu_;
  std::condition_variable go_, done_cv_;
  const std::function<void(int)>* job_ = nullptr;
  int parts_ = 0, next_ = 0, done_ = 0;
  uint64_t gen_ = 0;
  bool stop_ = false;
};

}  // namespace
}  // namespace fs

struct fs_ensemble {
  std::mutex mu;
  std::string err;
  int device = 0, num_cus = 256;
  Prec prec = BF16;
  int N = 0, C = 0, max_batch = 0;
  int combine = FS_COMBINE_MEAN, pos_class = 0, min_votes = 1;  // policy of vote
  fs_preprocess pre{};
  std::vector<Group> groups;
  double flops_per_image = 0;
  // weights, shared by every handle made from this one with fs_ensemble_share
  std::shared_ptr<DevBuf> arena = std::make_shared<DevBuf>();
  size_t arena_bytes = 0;
  DevBuf input;     // [max_batch][out_h][out_w][4]
  DevBuf input_s2d; // [max_batch][out_h/2][out_w/2][16] bf16
  bool need_plain = false, need_s2d = false;
  DevBuf partial;   // fc split-K scratch
  DevBuf conv_partial;  // conv split-K scratch (grown when a batch bucket is first planned)
  DevBuf logits;    // [N][max_batch][C] fp32
  // host-path staging
  DevBuf d_pixels, d_desc, d_probs, d_mean, d_vote, d_top1;
  HostBuf h_pixels, h_desc, h_out;
  std::unique_ptr<fs::HostPool> pack_pool;  // started by the first fs_infer
  hipStream_t stream = nullptr;
  // groups on streams of their own, forked after the transformation and
  // joined before the softmax, so the layers of different groups share the
  // chip (on by default when there are several groups)
  bool group_streams = true;
  hipEvent_t fork = nullptr;
  // end of the last pass, on the stream it ran on: passes share the
  // workspace, so a pass on another stream first waits for this event
  hipEvent_t pass_done = nullptr;
  hipStream_t pass_stream = nullptr;
  bool pass_pending = false;
  // conv tile per (batch bucket) -> per group -> per layer, measured once
  std::map<int, std::vector<std::vector<int>>> tiles;
  // tile choice: 0 = committed table, else the shape rule (no timing);
  // 1 = time every candidate; 2 (default) = the table, timing what it lacks
  int tune = 2;
  // captured passes, replayed with one launch: key = batch size, stream and
  // every buffer the pass reads or writes (caller's and the ensemble's own);
  // off by default (eager launches measured faster, see fs_graphs_enable)
  bool graphs = false;
  std::map<std::vector<uintptr_t>, hipGraphExec_t> graph_cache;
  // profiler
  bool prof_on = false;
  std::vector<ProfRec> prof;
  std::vector<hipEvent_t> ev_pool;
  int64_t workspace_bytes = 0;
  // every candidate timing of the tile tuner, one line each (fs_tuning_log)
  std::string tune_log;
  // host-side phases of the last fs_infer, ms (summed over its chunks)
  double phase_ms[5] = {0, 0, 0, 0, 0};
  // test-only capture of one image's stored layer outputs (fs_debug_capture)
  int dbg_image = -1;
  DevBuf dbg;
  std::vector<std::vector<int64_t>> dbg_off;  // [model][layer]: byte offset in dbg, -1 = never stored
  std::vector<std::vector<int64_t>> dbg_bytes;
  std::vector<std::vector<char>> dbg_have;     // captured by the last pass
  int64_t dbg_in_off = 0, dbg_in_bytes = 0;
  bool dbg_in_have = false;
};

namespace {

size_t es(Prec p) { return p == BF16 ? 2 : 4; }

// ----------------------------------------------------------- validation
// Checks a combine policy and its parameters for N models of C classes.
void check_combine(int policy, int pos_class, int min_votes, int N, int C) {
  if (policy != FS_COMBINE_MEAN && policy != FS_COMBINE_PLURALITY && policy != FS_COMBINE_ANY)
    fail(FS_ERR_INVALID, "unknown combine policy " + std::to_string(policy));
  if (policy == FS_COMBINE_PLURALITY && N > COMBINE_MAX_PLURALITY)
    fail(FS_ERR_UNSUPPORTED, "FS_COMBINE_PLURALITY takes at most 64 models");
  if (policy == FS_COMBINE_ANY && (pos_class < 0 || pos_class >= C))
    fail(FS_ERR_INVALID, "positive_class must be in 0..num_classes-1");
  if (policy == FS_COMBINE_ANY && (min_votes < 1 || min_votes > N))
    fail(FS_ERR_INVALID, "min_votes must be in 1..num_models");
}

void validate_desc(const fs_ensemble_desc* d) {
  if (!d) fail(FS_ERR_INVALID, "desc is NULL");
  if (d->num_models < 1 || !d->models) fail(FS_ERR_INVALID, "num_models must be >= 1 with a models array");
  if (d->precision != FS_F32 && d->precision != FS_BF16) fail(FS_ERR_INVALID, "precision must be FS_F32 or FS_BF16");
  if (d->combine != FS_COMBINE_MEAN && d->combine != FS_COMBINE_PLURALITY)
    fail(FS_ERR_INVALID, "combine must be FS_COMBINE_MEAN or FS_COMBINE_PLURALITY at create "
                         "(FS_COMBINE_ANY takes its class and count through fs_set_combine)");
  if (d->combine == FS_COMBINE_PLURALITY && d->num_models > COMBINE_MAX_PLURALITY)
    fail(FS_ERR_UNSUPPORTED, "FS_COMBINE_PLURALITY takes at most 64 models");
  if (d->max_batch < 1 || d->max_batch > 4096) fail(FS_ERR_INVALID, "max_batch must be in 1..4096");
  if (d->pre.out_h < 1 || d->pre.out_w < 1 || d->pre.out_h > 4096 || d->pre.out_w > 4096)
    fail(FS_ERR_INVALID, "preprocess output size must be in 1..4096");
  for (int c = 0; c < 3; ++c)
    if (!std::isfinite(d->pre.mean[c]) || !std::isfinite(d->pre.std[c]) || d->pre.std[c] == 0.f)
      fail(FS_ERR_INVALID, "mean/std must be finite and std non-zero");
  const int prec = d->precision;
  const int C = d->models[0].num_classes;
  for (int m = 0; m < d->num_models; ++m) {
    const fs_model_spec& s = d->models[m];
    const std::string pfx = "model " + std::to_string(m) + ": ";
    if (s.num_layers < 1 || !s.layers) fail(FS_ERR_INVALID, pfx + "no layers");
    if (s.num_classes < 1) fail(FS_ERR_INVALID, pfx + "num_classes must be >= 1");
    if (s.num_classes != C) fail(FS_ERR_INVALID, pfx + "num_classes differs between models (the combine needs one class set)");
    if (s.num_classes > SOFTMAX_MAX_C) fail(FS_ERR_UNSUPPORTED, pfx + "more than 4096 classes");
    std::vector<Shape> out(s.num_layers);
    for (int i = 0; i < s.num_layers; ++i) {
      const fs_layer& L = s.layers[i];
      const std::string lp = pfx + "layer " + std::to_string(i) + ": ";
      if (L.src < -1 || L.src >= i) fail(FS_ERR_INVALID, lp + "src must be -1 or an earlier layer");
      Shape in = L.src < 0 ? Shape{d->pre.out_h, d->pre.out_w, 3} : out[L.src];
      const bool last = i == s.num_layers - 1;
      switch (L.op) {
        case FS_OP_CONV: {
          if (!L.weight) fail(FS_ERR_INVALID, lp + "conv weight is NULL");
          if (L.cin != in.C) fail(FS_ERR_INVALID, lp + "conv cin does not match its input channels");
          if (L.cout < 1 || L.kh < 1 || L.kw < 1 || L.stride < 1 || L.pad < 0)
            fail(FS_ERR_INVALID, lp + "conv geometry");
          int Ho = (in.H + 2 * L.pad - L.kh) / L.stride + 1, Wo = (in.W + 2 * L.pad - L.kw) / L.stride + 1;
          if (in.H + 2 * L.pad < L.kh || in.W + 2 * L.pad < L.kw || Ho < 1 || Wo < 1)
            fail(FS_ERR_INVALID, lp + "conv output would be empty");
          if (L.cout % 8) fail(FS_ERR_UNSUPPORTED, lp + "conv cout must be a multiple of 8");
          if (L.src >= 0 && L.cin % 8) fail(FS_ERR_UNSUPPORTED, lp + "conv cin must be a multiple of 8");
          out[i] = Shape{Ho, Wo, L.cout};
          if (L.residual_src != -1) {
            if (L.residual_src < 0 || L.residual_src >= i) fail(FS_ERR_INVALID, lp + "residual_src must be -1 or an earlier layer");
            const Shape& r = out[L.residual_src];
            if (r.H != Ho || r.W != Wo || r.C != L.cout) fail(FS_ERR_INVALID, lp + "residual shape differs from the conv output");
          }
          if (last) fail(FS_ERR_INVALID, lp + "the last layer must be fc");
          break;
        }
        case FS_OP_MAXPOOL: {
          if (L.src < 0) fail(FS_ERR_UNSUPPORTED, lp + "max pool directly on the transformed input");
          if (L.kh < 1 || L.kh != L.kw || L.stride < 1 || L.pad < 0 || L.pad >= L.kh)
            fail(FS_ERR_INVALID, lp + "max pool geometry (square window, 0 <= pad < k)");
          int Ho = (in.H + 2 * L.pad - L.kh) / L.stride + 1, Wo = (in.W + 2 * L.pad - L.kw) / L.stride + 1;
          if (in.H + 2 * L.pad < L.kh || in.W + 2 * L.pad < L.kw || Ho < 1 || Wo < 1)
            fail(FS_ERR_INVALID, lp + "max pool output would be empty");
          out[i] = Shape{Ho, Wo, in.C};
          if (last) fail(FS_ERR_INVALID, lp + "the last layer must be fc");
          break;
        }
        case FS_OP_GAP:
          if (L.src < 0) fail(FS_ERR_UNSUPPORTED, lp + "global pool directly on the transformed input");
          out[i] = Shape{1, 1, in.C};
          if (last) fail(FS_ERR_INVALID, lp + "the last layer must be fc");
          break;
        case FS_OP_FC: {
          if (L.src < 0) fail(FS_ERR_UNSUPPORTED, lp + "fc directly on the transformed input");
          if (!L.weight) fail(FS_ERR_INVALID, lp + "fc weight is NULL");
          if ((int64_t)L.cin != in.elems()) fail(FS_ERR_INVALID, lp + "fc cin does not match the flattened input");
          if (L.cout < 1) fail(FS_ERR_INVALID, lp + "fc cout must be >= 1");
          if (prec == FS_BF16 && L.cin % 8) fail(FS_ERR_UNSUPPORTED, lp + "bf16 fc cin must be a multiple of 8");
          if (!last && L.cout % 8) fail(FS_ERR_UNSUPPORTED, lp + "hidden fc cout must be a multiple of 8");
          if (last && L.cout != s.num_classes) fail(FS_ERR_INVALID, lp + "last fc cout differs from num_classes");
          out[i] = Shape{1, 1, L.cout};
          break;
        }
        default:
          fail(FS_ERR_INVALID, lp + "unknown op");
      }
      if (out[i].elems() * (int64_t)d->max_batch * (prec == FS_BF16 ? 2 : 4) >= (int64_t(1) << 31))
        fail(FS_ERR_UNSUPPORTED, lp + "activation tensor of max_batch images exceeds 2 GiB");
    }
    if (s.layers[s.num_layers - 1].op != FS_OP_FC) fail(FS_ERR_INVALID, pfx + "the last layer must be fc");
  }
  if ((int64_t)d->pre.out_h * d->pre.out_w * 4 * d->max_batch * (prec == FS_BF16 ? 2 : 4) >= (int64_t(1) << 31))
    fail(FS_ERR_UNSUPPORTED, "transformed input of max_batch images exceeds 2 GiB");
}

bool same_structure(const fs_model_spec& a, const fs_model_spec& b) {
  if (a.num_layers != b.num_layers) return false;
  for (int i = 0; i < a.num_layers; ++i) {
    const fs_layer &x = a.layers[i], &y = b.layers[i];
    if (x.op != y.op || x.src != y.src || x.residual_src != y.residual_src || x.cin != y.cin ||
        x.cout != y.cout || x.kh != y.kh || x.kw != y.kw || x.stride != y.stride || x.pad != y.pad ||
        x.relu != y.relu || x.flatten_nchw != y.flatten_nchw)
      return false;
  }
  return true;
}

// ------------------------------------------------------- weight packing
// conv: [Cout][kh][kw][cin] (fp32, BN folded here) -> [Cout][Kp] with
// k = (ky*kw + kx)*cin_p + ci, zeros in padded positions.
void pack_conv(const fs_layer& L, int cin_p, int Kp, Prec p, void* dst_w, float* dst_b) {
  const int taps = L.kh * L.kw;
  for (int co = 0; co < L.cout; ++co) {
    const float s = L.bn_scale ? L.bn_scale[co] : 1.0f;
    for (int k = 0; k < Kp; ++k) {
      float v = 0.f;
      const int tap = k / cin_p, ci = k % cin_p;
      if (tap < taps && ci < L.cin) {
        v = L.weight[((int64_t)co * taps + tap) * L.cin + ci];
        if (L.bn_scale) v = v * s;
      }
      if (p == BF16)
        static_cast<uint16_t*>(dst_w)[(int64_t)co * Kp + k] = host_bf16(v);
      else
        static_cast<float*>(dst_w)[(int64_t)co * Kp + k] = v;
    }
    dst_b[co] = L.bn_shift ? L.bn_shift[co] : (L.bias ? L.bias[co] : 0.f);
  }
}

// fc: [N][K]; with flatten_nchw the columns are permuted from the
// channel-major order c*H*W + y*W + x to the NHWC order (y*W + x)*C + c.
void pack_fc(const fs_layer& L, const Shape& in, Prec p, void* dst_w, float* dst_b) {
  const int K = L.cin, HW = in.H * in.W;
  for (int n = 0; n < L.cout; ++n) {
    for (int k = 0; k < K; ++k) {
      int src_k = k;
      if (L.flatten_nchw) {
        const int pix = k / in.C, c = k % in.C;
        src_k = c * HW + pix;
      }
      const float v = L.weight[(int64_t)n * K + src_k];
      if (p == BF16)
        static_cast<uint16_t*>(dst_w)[(int64_t)n * K + k] = host_bf16(v);
      else
        static_cast<float*>(dst_w)[(int64_t)n * K + k] = v;
    }
    dst_b[n] = L.bias ? L.bias[n] : 0.f;
  }
}

// ------------------------------------------------------ space-to-depth stem
// A k x k, stride-2, pad (k-1)/2 convolution of the 3-channel transformed
// input equals a stride-1 convolution of its space-to-depth form (2x2 pixel
// blocks, channel (sy*2 + sx)*3 + c, padded to 16): input row 2*oy + q maps
// to block row oy + floor(q/2), sub-row q mod 2, for q = ky - (k-1)/2.
struct S2dGeom {
  int ks, pad;
};
int floor_div2(int v) { return v >= 0 ? v / 2 : -((-v + 1) / 2); }
S2dGeom s2d_geom(int k) {
  const int p = (k - 1) / 2;
  const int lo = floor_div2(-p), hi = floor_div2(p);
  return S2dGeom{hi - lo + 1, -lo};
}
bool s2d_eligible(const fs_layer& L, const fs_preprocess& pre, Prec prec) {
  return prec == BF16 && L.op == FS_OP_CONV && L.src < 0 && L.cin == 3 && L.stride == 2 && L.kh == L.kw &&
         (L.kh % 2) == 1 && L.pad == (L.kh - 1) / 2 && pre.out_h % 2 == 0 && pre.out_w % 2 == 0;
}
// w16[co][Ky][Kx][16] from w[co][ky][kx][3]; taps that fall outside the
// original filter are zero.
std::vector<float> s2d_weights(const fs_layer& L) {
  const int k = L.kh, p = (k - 1) / 2;
  const S2dGeom g = s2d_geom(k);
  std::vector<float> w16((size_t)L.cout * g.ks * g.ks * 16, 0.f);
  for (int co = 0; co < L.cout; ++co)
    for (int Ky = 0; Ky < g.ks; ++Ky)
      for (int Kx = 0; Kx < g.ks; ++Kx)
        for (int sy = 0; sy < 2; ++sy)
          for (int sx = 0; sx < 2; ++sx) {
            const int ky = 2 * (Ky - g.pad) + sy + p, kx = 2 * (Kx - g.pad) + sx + p;
            if (ky < 0 || ky >= k || kx < 0 || kx >= k) continue;
            for (int c = 0; c < 3; ++c)
              w16[(((size_t)co * g.ks + Ky) * g.ks + Kx) * 16 + (sy * 2 + sx) * 3 + c] =
                  L.weight[(((size_t)co * k + ky) * k + kx) * 3 + c];
          }
  return w16;
}
// The s2d form of a layer: same output, weights in w16 (caller keeps it alive).
fs_layer s2d_layer(const fs_layer& L, const std::vector<float>& w16) {
  const S2dGeom g = s2d_geom(L.kh);
  fs_layer q = L;
  q.cin = 16;
  q.kh = q.kw = g.ks;
  q.stride = 1;
  q.pad = g.pad;
  q.weight = w16.data();
  return q;
}

// ----------------------------------------------------------- planning
void plan_group(fs_ensemble* e, const fs_ensemble_desc* d, Group& g) {
  const fs_model_spec& s = d->models[g.first];
  const int n = s.num_layers;
  g.layers.resize(n);
  std::vector<Shape> out(n);
  std::vector<int> last_use(n, -1);
  std::vector<int> readers(n, 0);
  for (int i = 0; i < n; ++i) {
    const fs_layer& L = s.layers[i];
    if (L.src >= 0) last_use[L.src] = std::max(last_use[L.src], i);
    if (L.op == FS_OP_CONV && L.residual_src >= 0) last_use[L.residual_src] = std::max(last_use[L.residual_src], i);
    if (L.src >= 0) ++readers[L.src];
    if (L.op == FS_OP_CONV && L.residual_src >= 0) ++readers[L.residual_src];
  }
  // projection shortcuts summed into their block's last conv: a 1x1 conv
  // (no padding, no ReLU) whose only reader takes it as its residual, both
  // on 64-channel multiples so that the implicit GEMM runs the two
  // reductions back to back (bf16 only: in fp32 the shortcut's storage is
  // exact to fp32 rounding anyway)
  std::vector<int> proj_of(n, -1), folded_into(n, -1);
  if (e->prec == BF16)
    for (int i = 0; i < n; ++i) {
      const fs_layer& L = s.layers[i];
      if (L.op != FS_OP_CONV || L.residual_src < 0 || L.src < 0 || L.cin % 64) continue;
      const int dd = L.residual_src;
      const fs_layer& D = s.layers[dd];
      if (D.op != FS_OP_CONV || D.kh != 1 || D.kw != 1 || D.pad != 0 || D.relu || D.src < 0 || D.cin % 64 ||
          readers[dd] != 1 || D.cout != L.cout)
        continue;
      proj_of[i] = dd;
      folded_into[dd] = i;
      last_use[D.src] = std::max(last_use[D.src], i);  // read by the conv itself now
    }
  // slots: greedy reuse of freed buffers
  std::vector<int> slot_busy_until;  // layer index of last reader, per slot
  std::vector<int64_t>& slot_elems = g.slot_elems;
  std::vector<int> layer_slot(n, -1);
  for (int i = 0; i < n; ++i) {
    const fs_layer& L = s.layers[i];
    LayerPlan& P = g.layers[i];
    P.op = L.op;
    P.src = L.src;
    P.res = L.op == FS_OP_CONV ? L.residual_src : -1;
    P.in = L.src < 0 ? Shape{d->pre.out_h, d->pre.out_w, 3} : out[L.src];
    P.cin_p = L.src < 0 ? 4 : P.in.C;
    P.kh = L.kh; P.kw = L.kw; P.stride = L.stride; P.pad = L.pad;
    P.relu = L.relu ? 1 : 0;
    P.flatten = L.flatten_nchw ? 1 : 0;
    P.last = i == n - 1;
    P.in_c_real = P.in.C;
    switch (L.op) {
      case FS_OP_CONV:
        P.out = Shape{(P.in.H + 2 * L.pad - L.kh) / L.stride + 1, (P.in.W + 2 * L.pad - L.kw) / L.stride + 1, L.cout};
        P.K = L.kh * L.kw * P.cin_p;
        P.Kp = (int)round_up(P.K, CONV_KPAD);
        P.kreal = L.kh * L.kw * L.cin;
        e->flops_per_image += 2.0 * P.out.H * P.out.W * L.cout * (double)P.kreal * g.Z;
        if (s2d_eligible(L, d->pre, e->prec)) {  // launch geometry of the s2d form
          const S2dGeom sg = s2d_geom(L.kh);
          P.s2d = true;
          P.in = Shape{d->pre.out_h / 2, d->pre.out_w / 2, 16};
          P.cin_p = 16;
          P.kh = P.kw = sg.ks;
          P.stride = 1;
          P.pad = sg.pad;
          P.K = P.Kp = sg.ks * sg.ks * 16;
          e->need_s2d = true;
        } else if (L.src < 0) {
          e->need_plain = true;
        }
        if (i + 2 < n && s.layers[i + 1].op == FS_OP_GAP && s.layers[i + 1].src == i && last_use[i] == i + 1)
          P.gap_only = true;  // the split-K completion may also do the average pool
        if (P.s2d && L.relu && L.residual_src < 0 && L.cout == 64 && P.kh == 4 && P.pad == 2 && P.Kp == 256 &&
            P.out.W <= 112 && P.out.H == P.in.H && P.out.W == P.in.W && i + 1 < n - 1) {
          const fs_layer& Nx = s.layers[i + 1];  // a max pool that is the conv's only reader
          P.pool_fused = Nx.op == FS_OP_MAXPOOL && Nx.src == i && Nx.kh == 3 && Nx.kw == 3 && Nx.stride == 2 &&
                         Nx.pad == 1 && last_use[i] == i + 1;
        }
        break;
      case FS_OP_MAXPOOL:
        P.out = Shape{(P.in.H + 2 * L.pad - L.kh) / L.stride + 1, (P.in.W + 2 * L.pad - L.kw) / L.stride + 1, P.in.C};
        break;
      case FS_OP_GAP:
        P.out = Shape{1, 1, P.in.C};
        break;
      case FS_OP_FC:
        P.out = Shape{1, 1, L.cout};
        P.K = L.cin;
        e->flops_per_image += 2.0 * L.cin * L.cout * g.Z;
        break;
    }
    out[i] = P.out;
    P.in_slot = L.src < 0 ? SLOT_INPUT : layer_slot[L.src];
    if (folded_into[i] >= 0) {  // computed inside its block's last conv: no launch, no tensor
      P.proj_into = folded_into[i];
      P.out_slot = -1;
      continue;
    }
    if (proj_of[i] >= 0) {
      const fs_layer& D = s.layers[proj_of[i]];
      P.proj = proj_of[i];
      P.res = -1;
      P.proj_slot = layer_slot[D.src];
      P.proj_in = out[D.src];
      P.proj_cin = D.cin;
      P.proj_stride = D.stride;
      P.K += D.cin;
      P.Kp = (int)round_up(P.K, CONV_KPAD);
      P.kreal += D.cin;
    }
    P.res_slot = P.res >= 0 ? layer_slot[P.res] : -1;
    // free slots whose readers are all at or before this layer... but not
    // before this layer has read them: release after assigning the output.
    if (P.op == FS_OP_MAXPOOL && L.src == i - 1 && i > 0 && g.layers[i - 1].pool_fused) {
      // computed by the conv before it, straight into that conv's slot
      P.fused_away = true;
      const int slot = g.layers[i - 1].out_slot;
      P.out_slot = slot;
      layer_slot[i] = slot;
      slot_elems[slot] = std::max(slot_elems[slot], P.out.elems());
      slot_busy_until[slot] = std::max(slot_busy_until[slot], std::max(last_use[i], i));
    } else if (P.last) {
      P.out_slot = SLOT_LOGITS;
    } else {
      const int64_t need = P.pool_fused ? (int64_t)((P.out.H - 1) / 2 + 1) * ((P.out.W - 1) / 2 + 1) * P.out.C
                                        : P.out.elems();
      int pick = -1;
      for (size_t sidx = 0; sidx < slot_busy_until.size(); ++sidx) {
        if (slot_busy_until[sidx] < i) {  // free: its last reader ran before layer i
          if (pick < 0 || std::llabs(slot_elems[sidx] - need) < std::llabs(slot_elems[pick] - need)) pick = (int)sidx;
        }
      }
      if (pick < 0) {
        slot_elems.push_back(need);
        slot_busy_until.push_back(0);
        pick = (int)slot_elems.size() - 1;
      }
      slot_elems[pick] = std::max(slot_elems[pick], need);
      slot_busy_until[pick] = std::max(last_use[i], i);
      layer_slot[i] = pick;
      P.out_slot = pick;
    }
  }
}

int num_cus_of(int dev) {
  int n = 0;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) n = 256;
  return n;
}

void set_device(int dev) {
  int count = 0;
  hipError_t err = hipGetDeviceCount(&count);
  if (err != hipSuccess || count <= 0) fail(FS_ERR_DEVICE, std::string("no HIP device available: ") + hipGetErrorString(err));
  if (dev < 0 || dev >= count) fail(FS_ERR_DEVICE, "device ordinal " + std::to_string(dev) + " out of range");
  HIPCHK(hipSetDevice(dev));
}

void alloc_workspace(fs_ensemble* e);
ConvArgs conv_args(fs_ensemble* e, Group& g, const LayerPlan& P, int B, void* y, int64_t y_ms);

void build(fs_ensemble* e, const fs_ensemble_desc* d) {
  e->prec = d->precision == FS_BF16 ? BF16 : F32;
  e->N = d->num_models;
  e->combine = d->combine;
  e->C = d->models[0].num_classes;
  e->max_batch = d->max_batch;
  e->pre = d->pre;
  e->device = d->device;
  if (const char* t = std::getenv("FS_TUNE")) e->tune = std::atoi(t);
  if (const char* t = std::getenv("FS_GROUP_STREAMS")) e->group_streams = std::atoi(t) != 0;
  // groups of consecutive structurally identical models
  for (int m = 0; m < e->N;) {
    int z = 1;
    while (m + z < e->N && same_structure(d->models[m], d->models[m + z])) ++z;
    Group g;
    g.first = m;
    g.Z = z;
    e->groups.push_back(std::move(g));
    m += z;
  }
  for (Group& g : e->groups) plan_group(e, d, g);

  // weight arena layout
  const size_t esz = es(e->prec);
  size_t off = 0;
  for (Group& g : e->groups) {
    for (LayerPlan& P : g.layers) {
      if ((P.op == FS_OP_CONV && P.proj_into < 0) || P.op == FS_OP_FC) {
        const int64_t welems = P.op == FS_OP_CONV ? (int64_t)P.out.C * P.Kp : (int64_t)P.out.C * P.K;
        P.w_melems = (int64_t)round_up(welems, 128);
        P.b_melems = (int64_t)round_up(P.out.C, 64);
        P.w_off = off;
        off += (size_t)P.w_melems * esz * g.Z;
        P.b_off = off;
        off += (size_t)P.b_melems * 4 * g.Z;
        off = round_up(off, 256);
        // the implicit GEMM's one-row tiles load their weights into
        // registers from a fragment-ordered copy (the stem's fused kernel
        // keeps its weights in LDS)
        P.has_wf = P.op == FS_OP_CONV && !P.pool_fused && conv_frag_wanted(e->prec, P.out.C, P.Kp);
        if (P.has_wf) {
          P.wf_off = off;
          off = round_up(off + (size_t)P.w_melems * esz * g.Z, 256);
        }
      }
    }
  }
  e->arena_bytes = off;
  std::vector<char> host(off, 0);
  for (Group& g : e->groups) {
    for (int li = 0; li < (int)g.layers.size(); ++li) {
      LayerPlan& P = g.layers[li];
      if ((P.op != FS_OP_CONV || P.proj_into >= 0) && P.op != FS_OP_FC) continue;
      for (int z = 0; z < g.Z; ++z) {
        const fs_layer& L = d->models[g.first + z].layers[li];
        void* wdst = host.data() + P.w_off + (size_t)z * P.w_melems * esz;
        float* bdst = reinterpret_cast<float*>(host.data() + P.b_off + (size_t)z * P.b_melems * 4);
        if (P.op == FS_OP_CONV && P.s2d) {
          const std::vector<float> w16 = s2d_weights(L);
          pack_conv(s2d_layer(L, w16), P.cin_p, P.Kp, e->prec, wdst, bdst);
        } else if (P.op == FS_OP_CONV && P.proj >= 0) {
          // rows [main conv (K1) | projection shortcut (Cin2)], biases added
          const fs_layer& D = d->models[g.first + z].layers[P.proj];
          const int K1 = P.Kp - P.proj_cin;
          std::vector<char> w1((size_t)P.out.C * K1 * esz), w2((size_t)P.out.C * P.proj_cin * esz);
          std::vector<float> b1(P.out.C), b2(P.out.C);
          pack_conv(L, P.cin_p, K1, e->prec, w1.data(), b1.data());
          pack_conv(D, P.proj_cin, P.proj_cin, e->prec, w2.data(), b2.data());
          for (int co = 0; co < P.out.C; ++co) {
            std::memcpy(static_cast<char*>(wdst) + (size_t)co * P.Kp * esz, w1.data() + (size_t)co * K1 * esz, K1 * esz);
            std::memcpy(static_cast<char*>(wdst) + ((size_t)co * P.Kp + K1) * esz,
                        w2.data() + (size_t)co * P.proj_cin * esz, P.proj_cin * esz);
            bdst[co] = b1[co] + b2[co];
          }
        } else if (P.op == FS_OP_CONV) {
          pack_conv(L, P.cin_p, P.Kp, e->prec, wdst, bdst);
        } else {
          pack_fc(L, P.in, e->prec, wdst, bdst);
        }
        if (P.has_wf)
          conv_frag_order(static_cast<const uint16_t*>(wdst), P.out.C, P.Kp,
                          reinterpret_cast<uint16_t*>(host.data() + P.wf_off + (size_t)z * P.w_melems * esz));
      }
    }
  }

  set_device(e->device);
  e->num_cus = num_cus_of(e->device);
  HIPCHK(hipStreamCreateWithFlags(&e->stream, hipStreamNonBlocking));
  e->arena->alloc(std::max<size_t>(off, 256));
  HIPCHK(hipMemcpy(e->arena->p, host.data(), off, hipMemcpyHostToDevice));
  alloc_workspace(e);
}

// Activation slots, split-K scratch, transformed-input and logit buffers of
// one handle, for its max_batch.
void alloc_workspace(fs_ensemble* e) {
  const size_t esz = es(e->prec);
  const int Bm = e->max_batch;
  int64_t ws = 0;
  for (Group& g : e->groups) {
    g.slots.resize(g.slot_elems.size());
    for (size_t sidx = 0; sidx < g.slot_elems.size(); ++sidx) {
      const size_t bytes = round_up((size_t)g.slot_elems[sidx] * Bm * g.Z * esz, 256);
      g.slots[sidx].alloc(bytes);
      ws += bytes;
    }
  }
  // split-K scratch of the FC layers: the split depends on B, so size it
  // for the worst case over every batch size a pass can see
  size_t pf_all = 0;
  for (Group& g : e->groups)
    for (LayerPlan& P : g.layers)
      if (P.op == FS_OP_FC)
        for (int B = 1; B <= Bm; ++B)
          pf_all = std::max(pf_all, fc_partial_floats(B, P.out.C, fc_pick_split(e->prec, B, P.K, P.out.C, g.Z, e->num_cus), g.Z));
  e->partial.alloc(round_up(std::max<size_t>(pf_all, 1) * 4, 256));
  if (e->group_streams && e->groups.size() > 1) {
    // concurrent groups cannot share split-K scratch: one set per group
    for (Group& g : e->groups) {
      size_t pf = 0, cf = 0;
      for (LayerPlan& P : g.layers)
        for (int B = 1; B <= Bm; ++B) {
          if (P.op == FS_OP_FC)
            pf = std::max(pf, fc_partial_floats(B, P.out.C, fc_pick_split(e->prec, B, P.K, P.out.C, g.Z, e->num_cus), g.Z));
          else if (P.op == FS_OP_CONV && !P.pool_fused && P.proj_into < 0)
            cf = std::max(cf, conv_partial_floats(conv_args(e, g, P, B, nullptr, 0)));
        }
      g.fc_partial.alloc(round_up(std::max<size_t>(pf, 1) * 4, 256));
      g.conv_partial.alloc(round_up(std::max<size_t>(cf, 1) * 4, 256));
      ws += g.fc_partial.bytes + g.conv_partial.bytes;
      HIPCHK(hipStreamCreateWithFlags(&g.stream, hipStreamNonBlocking));
      HIPCHK(hipEventCreateWithFlags(&g.done, hipEventDisableTiming));
    }
    HIPCHK(hipEventCreateWithFlags(&e->fork, hipEventDisableTiming));
  }
  // split-K scratch of the conv layers, likewise for every batch size: a
  // layer's K split grows as its M shrinks, so a batch below its bucket's
  // size can need more than the bucket size itself
  size_t cf_all = 0;
  for (Group& g : e->groups)
    for (LayerPlan& P : g.layers)
      if (P.op == FS_OP_CONV && !P.pool_fused && P.proj_into < 0)
        for (int B = 1; B <= Bm; ++B) cf_all = std::max(cf_all, conv_partial_floats(conv_args(e, g, P, B, nullptr, 0)));
  if (cf_all) e->conv_partial.alloc(round_up(cf_all * 4, 256));
  ws += e->conv_partial.bytes;
  if (e->need_plain) e->input.alloc(round_up((size_t)Bm * e->pre.out_h * e->pre.out_w * 4 * esz, 256));
  if (e->need_s2d) e->input_s2d.alloc(round_up((size_t)Bm * e->pre.out_h * e->pre.out_w * 4 * 2, 256));
  e->logits.alloc(round_up((size_t)e->N * Bm * e->C * 4, 256));
  ws += e->partial.bytes + e->input.bytes + e->input_s2d.bytes + e->logits.bytes;
  e->workspace_bytes = ws;
}

// ------------------------------------------------------------- profiler
struct Launcher {
  fs_ensemble* e;
  hipStream_t s;
  int group = -1, layer = -1, M = 0, N = 0, K = 0, Z = 1;
  const char* kernel = "";
  template <class F>
  void operator()(int cls, double flops, double bytes, int launches, F&& fn) {
    if (!e->prof_on) {
      fn();
      return;
    }
    auto take = [&]() {
      hipEvent_t ev;
      if (!e->ev_pool.empty()) {
        ev = e->ev_pool.back();
        e->ev_pool.pop_back();
      } else {
        HIPCHK(hipEventCreate(&ev));
      }
      return ev;
    };
    ProfRec r{cls, take(), take(), flops, bytes, launches, group, layer, M, N, K, Z, kernel};
    HIPCHK(hipEventRecord(r.a, s));
    fn();
    HIPCHK(hipEventRecord(r.b, s));
    e->prof.push_back(r);
  }
};

void prof_clear(fs_ensemble* e) {
  for (ProfRec& r : e->prof) {
    e->ev_pool.push_back(r.a);
    e->ev_pool.push_back(r.b);
  }
  e->prof.clear();
}

// ------------------------------------------------------------ device pass
void* slot_ptr(Group& g, int slot) { return g.slots[slot].p; }

ConvArgs conv_args(fs_ensemble* e, Group& g, const LayerPlan& P, int B, void* y, int64_t y_ms) {
  const int Bm = e->max_batch;
  char* arena = static_cast<char*>(e->arena->p);
  ConvArgs a{};
  a.x = P.in_slot == SLOT_INPUT ? (P.s2d ? e->input_s2d.p : e->input.p) : slot_ptr(g, P.in_slot);
  a.x_mstride = P.in_slot == SLOT_INPUT ? 0 : (int64_t)g.slot_elems[P.in_slot] * Bm;
  a.w = arena + P.w_off; a.w_mstride = P.w_melems;
  if (P.has_wf) { a.wf = arena + P.wf_off; a.wf_mstride = P.w_melems; }
  a.bias = reinterpret_cast<const float*>(arena + P.b_off); a.b_mstride = P.b_melems;
  a.res = P.res_slot >= 0 ? slot_ptr(g, P.res_slot) : nullptr;
  a.res_mstride = P.res_slot >= 0 ? (int64_t)g.slot_elems[P.res_slot] * Bm : 0;
  a.y = y; a.y_mstride = y_ms;
  a.B = B; a.H = P.in.H; a.W = P.in.W; a.Cin = P.cin_p;
  a.Ho = P.out.H; a.Wo = P.out.W; a.Cout = P.out.C;
  a.kh = P.kh; a.kw = P.kw; a.stride = P.stride; a.pad = P.pad; a.relu = P.relu;
  a.K = P.K; a.Kp = P.Kp; a.M = B * P.out.H * P.out.W; a.Z = g.Z;
  if (P.proj >= 0) {
    a.x2 = slot_ptr(g, P.proj_slot);
    a.x2_mstride = (int64_t)g.slot_elems[P.proj_slot] * Bm;
    a.H2 = P.proj_in.H; a.W2 = P.proj_in.W; a.Cin2 = P.proj_cin; a.stride2 = P.proj_stride;
    a.K1 = P.Kp - P.proj_cin;
  }
  a.split = conv_split(e->prec, a, e->num_cus);
  a.partial = static_cast<float*>(g.conv_partial.p ? g.conv_partial.p : e->conv_partial.p);
  return a;
}

int batch_bucket(int B, int max_batch) {
  int b = 1;
  while (b < B) b <<= 1;
  return std::min(b, max_batch);
}

// Conv tiles for one batch bucket.  With tuning on, every candidate tile
// of a layer is timed (HIP events, two launches after a warm-up) on the
// layer's own buffers and the fastest kept.  Candidates are restricted to one
// kernel family per layer (the highest that fits it, a rule on the shape
// alone): within a family every tile sums each output in the same order, so
// the choice never changes the results.
// The committed tile table: layer shape, batch bucket and models per launch
// -> tile name.
struct TileEntry {
  int bucket, prec, kh, kw, stride, pad, cin, cout, h, w, z, proj_cin, proj_stride;
  const char* tile;
};
const TileEntry kTileTable[] = {
#include "tile_table.inc"
    {0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, 0, nullptr}};

// The table's tile for this layer at this bucket, or -1 (also when the
// entry names a tile outside the layer's kernel family fam, e.g. a table
// written under another family rule: the layer is then timed afresh).
int table_tile(const fs_ensemble* e, const ConvArgs& a, int bucket, int fam) {
  for (const TileEntry& t : kTileTable) {
    if (!t.tile) break;
    if (t.bucket == bucket && t.prec == (e->prec == BF16 ? 1 : 0) && t.kh == a.kh && t.kw == a.kw &&
        t.stride == a.stride && t.pad == a.pad && t.cin == a.Cin && t.cout == a.Cout && t.h == a.H && t.w == a.W &&
        t.z == a.Z && t.proj_cin == (a.x2 ? a.Cin2 : 0) && t.proj_stride == (a.x2 ? a.stride2 : 0)) {
      for (int i = 0; i < conv_num_tiles(e->prec); ++i)
        if (std::strcmp(conv_tile(e->prec, i).name, t.tile) == 0)
          return conv_tile_candidate(e->prec, i, a) && conv_tile_family(conv_tile(e->prec, i)) == fam ? i : -1;
      return -1;
    }
  }
  return -1;
}

const std::vector<std::vector<int>>& tiles_for(fs_ensemble* e, int B, hipStream_t s) {
  const int bucket = batch_bucket(B, e->max_batch);
  auto it = e->tiles.find(bucket);
  if (it != e->tiles.end()) return it->second;
  std::vector<std::vector<int>> choice(e->groups.size());
  hipEvent_t e0 = nullptr, e1 = nullptr;
  if (e->tune) {  // created lazily enough: events are cheap
    HIPCHK(hipEventCreate(&e0));
    HIPCHK(hipEventCreate(&e1));
  }
  for (size_t gi = 0; gi < e->groups.size(); ++gi) {
    Group& g = e->groups[gi];
    choice[gi].assign(g.layers.size(), -1);
    for (size_t li = 0; li < g.layers.size(); ++li) {
      LayerPlan& P = g.layers[li];
      if (P.op != FS_OP_CONV || P.pool_fused || P.proj_into >= 0) continue;
      ConvArgs a = conv_args(e, g, P, bucket, slot_ptr(g, P.out_slot), (int64_t)g.slot_elems[P.out_slot] * e->max_batch);
      const size_t need = conv_partial_floats(a) * 4;
      if (need > (g.conv_partial.p ? g.conv_partial.bytes : e->conv_partial.bytes))
        fail(FS_ERR_INTERNAL, "split-K scratch too small for this batch size");
      if (need > e->conv_partial.bytes) {  // split-K scratch for this bucket
        HIPCHK(hipStreamSynchronize(s));
        e->conv_partial.alloc(round_up(need, 256));
        e->workspace_bytes += (int64_t)e->conv_partial.bytes;
        a.partial = static_cast<float*>(e->conv_partial.p);
      }
      int fam = -1;  // the layer runs in the highest kernel family among its candidates
      for (int t = 0; t < conv_num_tiles(e->prec); ++t)
        if (conv_tile_candidate(e->prec, t, a)) fam = std::max(fam, conv_tile_family(conv_tile(e->prec, t)));
      int best = conv_pick_tile(e->prec, a, e->num_cus);
      const int from_table = e->tune == 1 ? -1 : table_tile(e, a, bucket, fam);
      if (from_table >= 0) best = from_table;
      if (e->tune == 1 || e->tune == 3 || (e->tune == 2 && from_table < 0)) {
        // re-timing against the table (3): its tile is timed first, so that
        // another candidate replaces it only by winning by the margin below
        std::vector<int> order;
        if (e->tune == 3 && from_table >= 0) order.push_back(from_table);
        for (int t = 0; t < conv_num_tiles(e->prec); ++t)
          if (conv_tile_candidate(e->prec, t, a) && conv_tile_family(conv_tile(e->prec, t)) == fam &&
              !(e->tune == 3 && t == from_table))
            order.push_back(t);
        float best_ms = 1e30f;
        for (int t : order) {
          launch_conv(a, e->prec, t, s);
          HIPCHK(hipEventRecord(e0, s));
          launch_conv(a, e->prec, t, s);
          launch_conv(a, e->prec, t, s);
          HIPCHK(hipEventRecord(e1, s));
          HIPCHK(hipEventSynchronize(e1));
          float ms = 0.f;
          HIPCHK(hipEventElapsedTime(&ms, e0, e1));
          // a later candidate must win by 3%: timing noise alone does not
          // flip the choice between near-equal tiles from run to run
          if (ms < best_ms * 0.97f) { best_ms = ms; best = t; }
          char line[160];
          std::snprintf(line, sizeof(line), "bucket %d group %zu layer %zu M %d N %d K %d Z %d split %d tile %s us %.2f\n",
                        bucket, gi, li, a.M, a.Cout, a.K, a.Z, a.split, conv_tile(e->prec, t).name, ms * 500.0f);
          e->tune_log += line;
        }
        HIPCHK(hipGetLastError());
        char line[200];
        std::snprintf(line, sizeof(line),
                      "choice bucket %d group %zu layer %zu prec %d kh %d kw %d stride %d pad %d cin %d cout %d "
                      "h %d w %d z %d proj_cin %d proj_stride %d tile %s\n",
                      bucket, gi, li, e->prec == BF16 ? 1 : 0, a.kh, a.kw, a.stride, a.pad, a.Cin, a.Cout, a.H, a.W, a.Z,
                      a.x2 ? a.Cin2 : 0, a.x2 ? a.stride2 : 0, conv_tile(e->prec, best).name);
        e->tune_log += line;
      }
      if (best < 0) fail(FS_ERR_INTERNAL, "no conv tile fits a planned layer");
      choice[gi][li] = best;
    }
  }
  if (e0) (void)hipEventDestroy(e0);
  if (e1) (void)hipEventDestroy(e1);
  return e->tiles.emplace(bucket, std::move(choice)).first->second;
}

// Test-only: copy image e->dbg_image of layer li's stored output, for every
// model of group g, into the capture buffer (y: the output tensor of model 0,
// y_ms: its per-model stride in elements, elems: elements per image, esz:
// bytes per element).
void dbg_capture(fs_ensemble* e, const Group& g, int li, const void* y, int64_t y_ms, int64_t elems, size_t esz,
                 int B, hipStream_t s) {
  if (e->dbg_image < 0 || e->dbg_image >= B) return;
  for (int z = 0; z < g.Z; ++z) {
    const int m = g.first + z;
    const int64_t off = e->dbg_off[m][li];
    if (off < 0 || e->dbg_bytes[m][li] != elems * (int64_t)esz) continue;
    const char* src = static_cast<const char*>(y) + ((int64_t)z * y_ms + (int64_t)e->dbg_image * elems) * esz;
    HIPCHK(hipMemcpyAsync(static_cast<char*>(e->dbg.p) + off, src, elems * esz, hipMemcpyDeviceToDevice, s));
    e->dbg_have[m][li] = 1;
  }
}

void run_pass(fs_ensemble* e, const uint8_t* d_pixels, const ImageDesc* d_desc, int B, float* d_probs,
              float* d_mean, int32_t* d_vote, int32_t* d_top1, float* d_logits, hipStream_t s) {
  Launcher launch{e, s};
  const Prec p = e->prec;
  const size_t esz = es(p);
  const int oh = e->pre.out_h, ow = e->pre.out_w;
  const int Bm = e->max_batch;
  float* logits = d_logits ? d_logits : static_cast<float*>(e->logits.p);

  PreArgs pa{};
  pa.pixels = d_pixels;
  pa.desc = d_desc;
  pa.B = B;
  pa.out_h = oh;
  pa.out_w = ow;
  for (int c = 0; c < 3; ++c) {
    pa.mean[c] = e->pre.mean[c];
    pa.std_[c] = e->pre.std[c];
  }
  pa.out = e->need_plain ? e->input.p : nullptr;
  pa.out_s2d = e->need_s2d ? e->input_s2d.p : nullptr;
  launch(K_PRE, 0.0, (double)B * oh * ow * 3 * esz * ((e->need_plain ? 1 : 0) + (e->need_s2d ? 1 : 0)),
         (e->need_plain ? 1 : 0) + (e->need_s2d ? 1 : 0), [&] { launch_preprocess(pa, p, s); });
  if (e->dbg_image >= 0) {
    for (auto& v : e->dbg_have) std::fill(v.begin(), v.end(), 0);
    e->dbg_in_have = false;
    if (e->dbg_image < B) {
      const void* src = e->need_plain ? e->input.p : e->input_s2d.p;
      HIPCHK(hipMemcpyAsync(static_cast<char*>(e->dbg.p) + e->dbg_in_off,
                            static_cast<const char*>(src) + (int64_t)e->dbg_image * e->dbg_in_bytes, e->dbg_in_bytes,
                            hipMemcpyDeviceToDevice, s));
      e->dbg_in_have = true;
    }
  }

  char* arena = static_cast<char*>(e->arena->p);
  const std::vector<std::vector<int>>& tiles = tiles_for(e, B, s);
  const hipStream_t s_main = s;
  const bool multi = e->fork != nullptr;
  if (multi) HIPCHK(hipEventRecord(e->fork, s_main));
  for (size_t gi = 0; gi < e->groups.size(); ++gi) {
    Group& g = e->groups[gi];
    // the group's launches go to its own stream when groups run concurrently
    const hipStream_t s = multi ? g.stream : s_main;
    if (multi) HIPCHK(hipStreamWaitEvent(s, e->fork, 0));
    launch.s = s;
    bool skip_next = false;  // the layer was done by the launch before it
    for (size_t li = 0; li < g.layers.size(); ++li) {
      LayerPlan& P = g.layers[li];
      if (skip_next) {
        skip_next = false;
        continue;
      }
      launch.group = (int)gi;
      launch.layer = (int)li;
      launch.Z = g.Z;
      launch.kernel = "";
      const void* x = P.in_slot == SLOT_INPUT ? (P.s2d ? e->input_s2d.p : e->input.p) : slot_ptr(g, P.in_slot);
      const int64_t x_ms = P.in_slot == SLOT_INPUT ? 0 : (int64_t)g.slot_elems[P.in_slot] * Bm;
      void* y = nullptr;
      int64_t y_ms = 0;
      if (P.out_slot == SLOT_LOGITS) {
        y = logits + (int64_t)g.first * B * e->C;
        y_ms = (int64_t)B * e->C;
      } else {
        y = slot_ptr(g, P.out_slot);
        y_ms = (int64_t)g.slot_elems[P.out_slot] * Bm;
      }
      switch (P.op) {
        case FS_OP_CONV: {
          if (P.proj_into >= 0) break;  // runs inside its block's last conv
          const ConvArgs a = conv_args(e, g, P, B, y, y_ms);
          if (conv_partial_floats(a) * 4 > (g.conv_partial.p ? g.conv_partial.bytes : e->conv_partial.bytes))
            fail(FS_ERR_INTERNAL, "split-K scratch too small for this batch size");
          const int tile = tiles[gi][li];
          launch.M = a.M; launch.N = a.Cout; launch.K = P.kreal;
          launch.kernel = P.pool_fused ? "stem_s2d_conv_maxpool" : conv_tile(p, tile).name;
          const double kreal = (double)P.kreal;
          const double flops = 2.0 * a.M * a.Cout * kreal * g.Z;
          const double in_b = (double)B * P.in.H * P.in.W * P.in_c_real * (P.s2d ? 4 : 1) * esz *
                              (P.in_slot == SLOT_INPUT ? 1 : g.Z);
          const double out_px = P.pool_fused ? (double)B * ((P.out.H - 1) / 2 + 1) * ((P.out.W - 1) / 2 + 1) : a.M;
          const double proj_b = P.proj >= 0 ? (double)B * P.proj_in.elems() * esz * g.Z : 0.0;
          const double bytes = in_b + proj_b + ((double)a.Cout * kreal * esz + out_px * a.Cout * esz * (a.res ? 2 : 1)) * g.Z;
          const size_t yes = P.last ? 4 : esz;
          if (P.pool_fused) {
            launch(K_CONV, flops, bytes, 1, [&] { launch_conv_stem_pool(a, s); });
            dbg_capture(e, g, (int)li + 1, y, y_ms, g.layers[li + 1].out.elems(), esz, B, s);
          } else if (P.gap_only && p == BF16 && conv_tile_direct(conv_tile(p, tile)) && conv_reduce_gap_ok(a)) {
            // the split-K completion also takes the average pool of the next layer
            const LayerPlan& G = g.layers[li + 1];
            void* gy = slot_ptr(g, G.out_slot);
            const int64_t gy_ms = (int64_t)g.slot_elems[G.out_slot] * Bm;
            launch(K_CONV, flops, bytes, 2, [&] {
              launch_conv(a, p, tile, s, false);
              launch_conv_splitk_reduce_gap(a, gy, gy_ms, s);
            });
            dbg_capture(e, g, (int)li + 1, gy, gy_ms, G.out.elems(), esz, B, s);
            skip_next = true;
          } else {
            launch(K_CONV, flops, bytes, a.split > 1 ? 2 : 1, [&] { launch_conv(a, p, tile, s); });
            dbg_capture(e, g, (int)li, y, y_ms, P.last ? e->C : P.out.elems(), yes, B, s);
          }
          break;
        }
        case FS_OP_MAXPOOL:
        case FS_OP_GAP: {
          if (P.fused_away) break;
          PoolArgs a{};
          a.x = x; a.x_mstride = x_ms; a.y = y; a.y_mstride = y_ms;
          a.B = B; a.H = P.in.H; a.W = P.in.W; a.C = P.in.C;
          a.Ho = P.out.H; a.Wo = P.out.W; a.k = P.kh; a.stride = P.stride; a.pad = P.pad; a.Z = g.Z;
          const double bytes = ((double)B * P.in.elems() + (double)B * P.out.elems()) * esz * g.Z;
          if (P.op == FS_OP_MAXPOOL)
            launch(K_MAXPOOL, 0.0, bytes, 1, [&] { launch_maxpool(a, p, s); });
          else
            launch(K_GAP, 0.0, bytes, 1, [&] { launch_gap(a, p, s); });
          dbg_capture(e, g, (int)li, y, y_ms, P.out.elems(), esz, B, s);
          break;
        }
        case FS_OP_FC: {
          FcArgs a{};
          a.x = x; a.x_mstride = x_ms;
          a.w = arena + P.w_off; a.w_mstride = P.w_melems;
          a.bias = reinterpret_cast<const float*>(arena + P.b_off); a.b_mstride = P.b_melems;
          a.y = y; a.y_mstride = y_ms;
          a.partial = static_cast<float*>(g.fc_partial.p ? g.fc_partial.p : e->partial.p);
          a.B = B; a.K = P.K; a.N = P.out.C; a.relu = P.relu; a.out_f32 = P.last ? 1 : 0;
          a.Z = g.Z;
          a.split = fc_pick_split(p, B, a.K, a.N, g.Z, e->num_cus);
          launch.M = B; launch.N = a.N; launch.K = a.K;
          launch.kernel = a.split > 1 ? "fc_splitk" : "fc";
          const double flops = 2.0 * B * a.N * (double)a.K * g.Z;
          const double bytes = ((double)a.N * a.K * esz + (double)B * a.K * esz +
                                (double)B * a.N * (a.out_f32 ? 4 : esz)) * g.Z;
          launch(K_FC, flops, bytes, fc_launches(a.split), [&] { launch_fc(a, p, s); });
          dbg_capture(e, g, (int)li, y, y_ms, a.N, a.out_f32 ? 4 : esz, B, s);
          break;
        }
      }
    }
    if (multi) HIPCHK(hipEventRecord(g.done, s));
  }
  launch.s = s_main;
  if (multi)
    for (Group& g : e->groups) HIPCHK(hipStreamWaitEvent(s_main, g.done, 0));

  launch.group = launch.layer = -1;
  launch.kernel = "";
  SoftmaxArgs sa{};
  sa.logits = logits;
  sa.probs = d_probs;
  sa.mean = d_mean;
  sa.vote = d_vote;
  sa.top1 = d_top1;
  sa.N = e->N;
  sa.B = B;
  sa.C = e->C;
  sa.policy = e->combine;
  sa.pos_class = e->pos_class;
  sa.min_votes = e->min_votes;
  const double sbytes = (double)e->N * B * e->C * 8 + (d_mean ? (double)B * e->C * 4 : 0) + B * 4.0;
  launch(K_SOFTMAX, 0.0, sbytes, 1, [&] { launch_softmax_combine(sa, s_main); });
  HIPCHK(hipGetLastError());
}

int launches_per_pass(fs_ensemble* e) {
  int n = 1 + (e->need_plain ? 1 : 0) + (e->need_s2d ? 1 : 0);  // preprocess + softmax/combine
  for (Group& g : e->groups) {
    const std::vector<std::vector<int>>* tl = nullptr;
    auto it = e->tiles.find(batch_bucket(e->max_batch, e->max_batch));
    if (it != e->tiles.end()) tl = &it->second;
    bool skip_next = false;
    for (size_t li = 0; li < g.layers.size(); ++li) {
      LayerPlan& P = g.layers[li];
      if (skip_next) { skip_next = false; continue; }
      if (P.op == FS_OP_FC) {
        n += fc_launches(fc_pick_split(e->prec, e->max_batch, P.K, P.out.C, g.Z, e->num_cus));
      } else if (P.op == FS_OP_CONV && P.proj_into < 0) {
        const ConvArgs a = conv_args(e, g, P, e->max_batch, nullptr, 0);
        n += (!P.pool_fused && a.split > 1) ? 2 : 1;
        const int gi = (int)(&g - e->groups.data());
        const int tile = tl ? (*tl)[gi][li] : conv_pick_tile(e->prec, a, e->num_cus);
        if (P.gap_only && e->prec == BF16 && tile >= 0 && conv_tile_direct(conv_tile(e->prec, tile)) &&
            conv_reduce_gap_ok(a))
          skip_next = true;
      } else if (!P.fused_away && P.op != FS_OP_CONV) {
        n += 1;
      }
    }
  }
  return n;
}

template <class F>
fs_status guarded(fs_ensemble* e, F&& fn) {
  try {
    fn();
    if (e) e->err.clear();
    return FS_OK;
  } catch (const Error& x) {
    if (e) e->err = x.msg; else g_thread_error = x.msg;
    return x.st;
  } catch (const std::bad_alloc&) {
    const char* m = "host allocation failed";
    if (e) e->err = m; else g_thread_error = m;
    return FS_ERR_OOM;
  } catch (const std::exception& x) {
    if (e) e->err = x.what(); else g_thread_error = x.what();
    return FS_ERR_INTERNAL;
  } catch (...) {
    if (e) e->err = "unknown error"; else g_thread_error = "unknown error";
    return FS_ERR_INTERNAL;
  }
}

void clear_graphs(fs_ensemble* e) {
  for (auto& kv : e->graph_cache) (void)hipGraphExecDestroy(kv.second);
  e->graph_cache.clear();
}

// One pass.  With graphs on (and the profiler off), the pass is captured the
// first time this exact batch size meets these buffers on this stream and
// replayed from then on; the tile plan of the batch bucket (which may time
// candidates and grow the split-K scratch) is made before the capture, so
// only kernel launches are recorded.  A capture that fails turns graphs off
// for the ensemble and the pass runs eagerly.
void run_pass_ordered(fs_ensemble* e, const uint8_t* d_pixels, const ImageDesc* d_desc, int B, float* d_probs,
                      float* d_mean, int32_t* d_vote, int32_t* d_top1, float* d_logits, hipStream_t s);

// Every pass of a handle uses the handle's one workspace (transformed
// input, activation slots, split-K scratch, logits), so passes issued on
// different streams must not overlap: a pass on a stream other than the
// previous pass's first waits (on the device) for the previous pass's end.
void run_pass_cached(fs_ensemble* e, const uint8_t* d_pixels, const ImageDesc* d_desc, int B, float* d_probs,
                     float* d_mean, int32_t* d_vote, int32_t* d_top1, float* d_logits, hipStream_t s) {
  if (e->pass_pending && e->pass_stream != s) HIPCHK(hipStreamWaitEvent(s, e->pass_done, 0));
  if (!e->pass_done) HIPCHK(hipEventCreateWithFlags(&e->pass_done, hipEventDisableTiming));
  run_pass_ordered(e, d_pixels, d_desc, B, d_probs, d_mean, d_vote, d_top1, d_logits, s);
  HIPCHK(hipEventRecord(e->pass_done, s));
  e->pass_stream = s;
  e->pass_pending = true;
}

void run_pass_ordered(fs_ensemble* e, const uint8_t* d_pixels, const ImageDesc* d_desc, int B, float* d_probs,
                      float* d_mean, int32_t* d_vote, int32_t* d_top1, float* d_logits, hipStream_t s) {
  if (!e->graphs || e->prof_on || e->dbg_image >= 0 || s == nullptr) {
    run_pass(e, d_pixels, d_desc, B, d_probs, d_mean, d_vote, d_top1, d_logits, s);
    return;
  }
  tiles_for(e, B, s);
  const std::vector<uintptr_t> key = {
      (uintptr_t)B, (uintptr_t)s, (uintptr_t)d_pixels, (uintptr_t)d_desc, (uintptr_t)d_probs, (uintptr_t)d_mean,
      (uintptr_t)d_vote, (uintptr_t)d_top1, (uintptr_t)d_logits, (uintptr_t)e->logits.p,
      (uintptr_t)e->conv_partial.p, (uintptr_t)e->partial.p};
  auto it = e->graph_cache.find(key);
  if (it == e->graph_cache.end()) {
    if (e->graph_cache.size() >= 64) clear_graphs(e);
    hipGraph_t g = nullptr;
    hipGraphExec_t x = nullptr;
    bool ok = hipStreamBeginCapture(s, hipStreamCaptureModeThreadLocal) == hipSuccess;
    if (ok) {
      try {
        run_pass(e, d_pixels, d_desc, B, d_probs, d_mean, d_vote, d_top1, d_logits, s);
      } catch (...) {
        if (hipStreamEndCapture(s, &g) == hipSuccess && g) (void)hipGraphDestroy(g);
        throw;
      }
      ok = hipStreamEndCapture(s, &g) == hipSuccess && g;
      ok = ok && hipGraphInstantiate(&x, g, nullptr, nullptr, 0) == hipSuccess;
      if (g) (void)hipGraphDestroy(g);
    }
    if (!ok) {
      (void)hipGetLastError();
      e->graphs = false;
      run_pass(e, d_pixels, d_desc, B, d_probs, d_mean, d_vote, d_top1, d_logits, s);
      return;
    }
    it = e->graph_cache.emplace(key, x).first;
  }
  HIPCHK(hipGraphLaunch(it->second, s));
}

void destroy_impl(fs_ensemble* e) {
  if (!e) return;
  if (hipSetDevice(e->device) == hipSuccess) {
    if (e->pass_pending) (void)hipEventSynchronize(e->pass_done);
    if (e->pass_done) (void)hipEventDestroy(e->pass_done);
    for (Group& g : e->groups) {
      if (g.stream) (void)hipStreamSynchronize(g.stream);
      if (g.stream) (void)hipStreamDestroy(g.stream);
      if (g.done) (void)hipEventDestroy(g.done);
    }
    if (e->fork) (void)hipEventDestroy(e->fork);
    if (e->stream) (void)hipStreamSynchronize(e->stream);
    clear_graphs(e);
    prof_clear(e);
    for (hipEvent_t ev : e->ev_pool) (void)hipEventDestroy(ev);
    e->ev_pool.clear();
    if (e->stream) (void)hipStreamDestroy(e->stream);
  }
  delete e;
}

// ------------------------------------------------------ test-entry helpers
struct TmpDev {
  std::vector<void*> ptrs;
  void* alloc(size_t n) {
    void* p = nullptr;
    HIPCHK(hipMalloc(&p, std::max<size_t>(n, 16)));
    ptrs.push_back(p);
    return p;
  }
  ~TmpDev() {
    for (void* p : ptrs) (void)hipFree(p);
  }
};

// host fp32 -> device storage type
void* upload_as(TmpDev& t, const float* src, int64_t n, Prec p) {
  void* d = t.alloc((size_t)n * es(p));
  if (p == BF16) {
    std::vector<uint16_t> h(n);
    for (int64_t i = 0; i < n; ++i) h[i] = host_bf16(src[i]);
    HIPCHK(hipMemcpy(d, h.data(), n * 2, hipMemcpyHostToDevice));
  } else {
    HIPCHK(hipMemcpy(d, src, n * 4, hipMemcpyHostToDevice));
  }
  return d;
}

void download_as(float* dst, const void* d, int64_t n, Prec p) {
  if (p == BF16) {
    std::vector<uint16_t> h(n);
    HIPCHK(hipMemcpy(h.data(), d, n * 2, hipMemcpyDeviceToHost));
    for (int64_t i = 0; i < n; ++i) dst[i] = host_bf16_to_f(h[i]);
  } else {
    HIPCHK(hipMemcpy(dst, d, n * 4, hipMemcpyDeviceToHost));
  }
}

Prec prec_of(int32_t precision) {
  if (precision != FS_F32 && precision != FS_BF16) fail(FS_ERR_INVALID, "precision must be FS_F32 or FS_BF16");
  return precision == FS_BF16 ? BF16 : F32;
}

void check_images(const fs_image* imgs, int B) {
  if (B < 0) fail(FS_ERR_INVALID, "B must be >= 0");
  if (B > 0 && !imgs) fail(FS_ERR_INVALID, "images array is NULL");
  for (int b = 0; b < B; ++b) {
    const fs_image& im = imgs[b];
    if (!im.data) fail(FS_ERR_INVALID, "image " + std::to_string(b) + " has no data");
    if (im.h < 1 || im.w < 1) fail(FS_ERR_INVALID, "image " + std::to_string(b) + " has zero size");
    if (im.w > 32768 || im.h > 32768) fail(FS_ERR_INVALID, "image " + std::to_string(b) + " is larger than 32768 pixels a side");
    if (im.row_stride < 3 * im.w) fail(FS_ERR_INVALID, "image " + std::to_string(b) + " row_stride < 3*w");
  }
}

// pack images densely into host memory and descriptors
size_t packed_size(const fs_image* imgs, int b0, int nb) {
  size_t n = 0;
  for (int b = b0; b < b0 + nb; ++b) n += round_up((size_t)imgs[b].h * imgs[b].w * 3, 16);
  return n;
}
void pack_images(const fs_image* imgs, int b0, int nb, uint8_t* dst, ImageDesc* desc) {
  size_t off = 0;
  for (int b = b0; b < b0 + nb; ++b) {
    const fs_image& im = imgs[b];
    const size_t row = (size_t)im.w * 3;
    for (int y = 0; y < im.h; ++y) std::memcpy(dst + off + y * row, im.data + (size_t)y * im.row_stride, row);
    desc[b - b0] = ImageDesc{off, im.h, im.w, (int32_t)row, 0};
    off += round_up(row * im.h, 16);
  }
}

// The same packing, staged for an overlapped upload: descriptors first, then
// the bytes in `pieces` parts of about equal size, each copied by the pool
// (in units of at most ~256 KB: whole images, or row blocks of a large one)
// and handed to `piece_done(begin, end)` (a byte range of dst) before the
// next part is copied.  A contiguous image (row_stride = 3w) is one memcpy.
void pack_images_staged(const fs_image* imgs, int b0, int nb, uint8_t* dst, ImageDesc* desc, HostPool& pool,
                        int pieces, const std::function<void(size_t, size_t)>& piece_done) {
  struct Unit {
    int b, y0, y1;
  };
  size_t off = 0;
  for (int b = b0; b < b0 + nb; ++b) {
    const fs_image& im = imgs[b];
    const size_t row = (size_t)im.w * 3;
    desc[b - b0] = ImageDesc{off, im.h, im.w, (int32_t)row, 0};
    off += round_up(row * im.h, 16);
  }
  const size_t total = off;
  constexpr size_t UNIT = 256 << 10;
  std::vector<Unit> units;
  int b = b0;
  size_t done = 0;  // bytes of dst handed over so far
  for (int p = 0; p < pieces && b < b0 + nb; ++p) {
    // whole images up to this piece's share of the bytes (at least one)
    const size_t goal = total * (size_t)(p + 1) / (size_t)pieces;
    units.clear();
    do {
      const fs_image& im = imgs[b];
      const size_t row = (size_t)im.w * 3;
      const int rows = (int)std::max<size_t>(1, UNIT / row);
      for (int y = 0; y < im.h; y += rows) units.push_back(Unit{b, y, std::min(im.h, y + rows)});
      ++b;
    } while (b < b0 + nb && desc[b - b0].offset < goal);
    pool.run((int)units.size(), [&](int u) {
      const Unit& t = units[u];
      const fs_image& im = imgs[t.b];
      const size_t row = (size_t)im.w * 3;
      uint8_t* d = dst + desc[t.b - b0].offset + (size_t)t.y0 * row;
      if ((size_t)im.row_stride == row) {
        std::memcpy(d, im.data + (size_t)t.y0 * row, (size_t)(t.y1 - t.y0) * row);
      } else {
        for (int y = t.y0; y < t.y1; ++y) std::memcpy(d + (size_t)(y - t.y0) * row, im.data + (size_t)y * im.row_stride, row);
      }
    });
    const size_t end = b < b0 + nb ? (size_t)desc[b - b0].offset : total;
    piece_done(done, end);
    done = end;
  }
}

// ------------------------------------------- allocation-free convolution
// The split-K partial sums of fs_conv_bf16_device_noalloc live in this
// library-static device array: every GPU the library runs on holds its own
// copy until the process ends.  In host code the name is only a stand-in;
// its device address comes from hipGetSymbolAddress, once per device, and
// only that address is passed to kernels.
constexpr size_t kNoallocScratchFloats = (size_t)FS_NOALLOC_SCRATCH_BYTES / 4;
static __device__ __align__(256) float scratch[kNoallocScratchFloats];

constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
float* g_scratch_ptr[kMaxDevices] = {};

// The current device's copy of `scratch` (looked up on its first use there).
float* noalloc_scratch(int dev) {
  if (dev < 0 || dev >= kMaxDevices) fail(FS_ERR_DEVICE, "device ordinal outside 0..63");
  std::lock_guard<std::mutex> lk(g_scratch_mu);
  if (!g_scratch_ptr[dev]) {
    void* p = nullptr;
    HIPCHK(hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)));
    if (!p) fail(FS_ERR_DEVICE, "no device address for the scratch array");
    g_scratch_ptr[dev] = static_cast<float*>(p);
  }
  return g_scratch_ptr[dev];
}

}  // namespace

// ==================================================================== ABI
extern "C" {

fs_status fs_conv_bf16_device_noalloc(const void* d_in, int32_t B, int32_t H, int32_t W, int32_t Cin, const void* d_w,
                                      const float* d_bias, const void* d_res, int32_t Cout, int32_t kh, int32_t kw,
                                      int32_t stride, int32_t pad, int32_t relu, void* d_out, void* stream) {
  return guarded(nullptr, [&] {
    if (!d_in || !d_w || !d_bias || !d_out) fail(FS_ERR_INVALID, "input, weight, bias and output are required");
    if (B < 1 || H < 1 || W < 1 || Cin < 1 || Cout < 1 || kh < 1 || kw < 1 || stride < 1 || pad < 0)
      fail(FS_ERR_INVALID, "bad conv arguments");
    if (H + 2 * pad < kh || W + 2 * pad < kw) fail(FS_ERR_INVALID, "conv output would be empty");
    if (Cin % 64) fail(FS_ERR_UNSUPPORTED, "Cin must be a multiple of 64");
    if (Cout % 8) fail(FS_ERR_UNSUPPORTED, "Cout must be a multiple of 8");
    const int Ho = (H + 2 * pad - kh) / stride + 1, Wo = (W + 2 * pad - kw) / stride + 1;
    if ((int64_t)B * H * W * Cin * 2 >= (int64_t(1) << 31) || (int64_t)B * Ho * Wo * Cout * 2 >= (int64_t(1) << 31))
      fail(FS_ERR_UNSUPPORTED, "tensor exceeds 2 GiB");
    int dev = 0;
    HIPCHK(hipGetDevice(&dev));
    ConvArgs a{};
    a.x = d_in; a.w = d_w; a.bias = d_bias; a.res = d_res; a.y = d_out;
    a.B = B; a.H = H; a.W = W; a.Cin = Cin; a.Ho = Ho; a.Wo = Wo; a.Cout = Cout;
    a.kh = kh; a.kw = kw; a.stride = stride; a.pad = pad; a.relu = relu ? 1 : 0;
    a.K = kh * kw * Cin; a.Kp = a.K; a.M = B * Ho * Wo; a.Z = 1;
    const int cus = num_cus_of(dev);
    const int tl = conv_pick_tile(BF16, a, cus);
    if (tl < 0 || !conv_tile_ok(BF16, tl, a)) fail(FS_ERR_UNSUPPORTED, "no conv kernel takes this shape");
    if (conv_tile_direct(conv_tile(BF16, tl))) {
      a.split = conv_split(BF16, a, cus);
      if (a.split > 1) {
        if (conv_partial_floats(a) > kNoallocScratchFloats)
          fail(FS_ERR_UNSUPPORTED, "the split-K partial sums of this shape (" +
                                       std::to_string(conv_partial_floats(a) * 4) + " bytes) exceed the " +
                                       std::to_string(FS_NOALLOC_SCRATCH_BYTES) + "-byte scratch array");
        a.partial = noalloc_scratch(dev);
      }
    }
    launch_conv(a, BF16, tl, static_cast<hipStream_t>(stream));
    HIPCHK(hipGetLastError());
  });
}

fs_status fs_ensemble_create(const fs_ensemble_desc* desc, fs_ensemble** out) {
  if (out) *out = nullptr;
  fs_ensemble* e = nullptr;
  fs_status st = guarded(nullptr, [&] {
    if (!out) fail(FS_ERR_INVALID, "out is NULL");
    validate_desc(desc);
    e = new fs_ensemble();
    try {
      build(e, desc);
    } catch (...) {
      destroy_impl(e);
      e = nullptr;
      throw;
    }
  });
  if (st == FS_OK) *out = e;
  return st;
}

fs_status fs_ensemble_share(fs_ensemble* src, fs_ensemble** out) {
  if (out) *out = nullptr;
  if (!src || !out) {
    g_thread_error = "ensemble or out is NULL";
    return FS_ERR_INVALID;
  }
  fs_ensemble* e = nullptr;
  fs_status st = guarded(nullptr, [&] {
    std::lock_guard<std::mutex> lk(src->mu);
    e = new fs_ensemble();
    try {
      e->device = src->device;
      e->num_cus = src->num_cus;
      e->prec = src->prec;
      e->N = src->N; e->C = src->C; e->max_batch = src->max_batch;
      e->combine = src->combine; e->pos_class = src->pos_class; e->min_votes = src->min_votes;
      e->pre = src->pre;
      e->groups.resize(src->groups.size());
      for (size_t i = 0; i < src->groups.size(); ++i) {  // the plan; slots are the new handle's own
        e->groups[i].first = src->groups[i].first;
        e->groups[i].Z = src->groups[i].Z;
        e->groups[i].layers = src->groups[i].layers;
        e->groups[i].slot_elems = src->groups[i].slot_elems;
      }
      e->flops_per_image = src->flops_per_image;
      e->arena = src->arena;
      e->arena_bytes = src->arena_bytes;
      e->need_plain = src->need_plain;
      e->need_s2d = src->need_s2d;
      e->tiles = src->tiles;
      e->tune = src->tune;
      e->group_streams = src->group_streams;
      e->graphs = src->graphs;
      set_device(e->device);
      HIPCHK(hipStreamCreateWithFlags(&e->stream, hipStreamNonBlocking));
      alloc_workspace(e);
    } catch (...) {
      destroy_impl(e);
      e = nullptr;
      throw;
    }
  });
  if (st == FS_OK) *out = e;
  return st;
}

fs_status fs_infer_device(fs_ensemble* e, const uint8_t* d_pixels, const fs_image_desc* d_desc, int32_t B,
                          float* d_probs, float* d_mean_probs, int32_t* d_vote, int32_t* d_top1,
                          float* d_logits, void* stream) {
  if (!e) {
    g_thread_error = "ensemble is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    if (B < 1 || B > e->max_batch) fail(FS_ERR_INVALID, "B must be in 1..max_batch for the device path");
    if (!d_pixels || !d_desc || !d_probs || !d_vote) fail(FS_ERR_INVALID, "required device pointer is NULL");
    HIPCHK(hipSetDevice(e->device));
    hipStream_t s = stream ? static_cast<hipStream_t>(stream) : e->stream;
    run_pass_cached(e, d_pixels, reinterpret_cast<const ImageDesc*>(d_desc), B, d_probs, d_mean_probs, d_vote,
                    d_top1, d_logits, s);
  });
}

fs_status fs_infer(fs_ensemble* e, const fs_image* imgs, int32_t B, float* probs, float* mean_probs,
                   int32_t* vote, int32_t* top1, float* logits) {
  if (!e) {
    g_thread_error = "ensemble is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    check_images(imgs, B);
    if (B == 0) return;
    if (!probs || !vote) fail(FS_ERR_INVALID, "probs and vote are required");
    HIPCHK(hipSetDevice(e->device));
    const int N = e->N, C = e->C, Bm = e->max_batch;
    hipStream_t s = e->stream;
    e->d_probs.ensure((size_t)N * Bm * C * 4);
    e->d_mean.ensure((size_t)Bm * C * 4);
    e->d_vote.ensure((size_t)Bm * 4);
    e->d_top1.ensure((size_t)N * Bm * 4);
    e->d_desc.ensure((size_t)Bm * sizeof(ImageDesc));
    e->h_desc.ensure((size_t)Bm * sizeof(ImageDesc));
    const size_t out_floats = (size_t)N * Bm * C * 2 + (size_t)Bm * C;
    e->h_out.ensure(out_floats * 4 + ((size_t)N + 1) * Bm * 4);
    using clk = std::chrono::steady_clock;
    auto lap = [](clk::time_point& t) {
      const clk::time_point n = clk::now();
      const double ms = std::chrono::duration<double, std::milli>(n - t).count();
      t = n;
      return ms;
    };
    for (double& v : e->phase_ms) v = 0;
    clk::time_point t = clk::now();
    for (int b0 = 0; b0 < B; b0 += Bm) {
      const int nb = std::min(Bm, B - b0);
      const size_t pbytes = packed_size(imgs, b0, nb);
      e->h_pixels.ensure(pbytes);
      e->d_pixels.ensure(pbytes);
      ImageDesc* hd = static_cast<ImageDesc*>(e->h_desc.p);
      if (!e->pack_pool) {
        const unsigned hw = std::thread::hardware_concurrency();
        e->pack_pool = std::make_unique<HostPool>((int)std::min(3u, hw > 1 ? hw - 1 : 0u));
      }
      // the first part's upload overlaps the copying of the second
      uint8_t* hpix = static_cast<uint8_t*>(e->h_pixels.p);
      uint8_t* dpix = static_cast<uint8_t*>(e->d_pixels.p);
      pack_images_staged(imgs, b0, nb, hpix, hd, *e->pack_pool, 2, [&](size_t lo, size_t hi) {
        if (hi > lo) HIPCHK(hipMemcpyAsync(dpix + lo, hpix + lo, hi - lo, hipMemcpyHostToDevice, s));
      });
      HIPCHK(hipMemcpyAsync(e->d_desc.p, hd, nb * sizeof(ImageDesc), hipMemcpyHostToDevice, s));
      e->phase_ms[0] += lap(t);
      float* dlog = static_cast<float*>(e->logits.p);
      run_pass_cached(e, static_cast<const uint8_t*>(e->d_pixels.p), static_cast<const ImageDesc*>(e->d_desc.p),
                      nb, static_cast<float*>(e->d_probs.p), mean_probs ? static_cast<float*>(e->d_mean.p) : nullptr,
                      static_cast<int32_t*>(e->d_vote.p), static_cast<int32_t*>(e->d_top1.p), dlog, s);
      e->phase_ms[1] += lap(t);
      float* hp = static_cast<float*>(e->h_out.p);
      float* hl = hp + (size_t)N * Bm * C;
      float* hm = hl + (size_t)N * Bm * C;
      int32_t* hv = reinterpret_cast<int32_t*>(hm + (size_t)Bm * C);
      int32_t* ht = hv + Bm;
      const size_t nbc = (size_t)N * nb * C;
      HIPCHK(hipMemcpyAsync(hp, e->d_probs.p, nbc * 4, hipMemcpyDeviceToHost, s));
      if (logits) HIPCHK(hipMemcpyAsync(hl, dlog, nbc * 4, hipMemcpyDeviceToHost, s));
      if (mean_probs) HIPCHK(hipMemcpyAsync(hm, e->d_mean.p, (size_t)nb * C * 4, hipMemcpyDeviceToHost, s));
      HIPCHK(hipMemcpyAsync(hv, e->d_vote.p, (size_t)nb * 4, hipMemcpyDeviceToHost, s));
      HIPCHK(hipMemcpyAsync(ht, e->d_top1.p, (size_t)N * nb * 4, hipMemcpyDeviceToHost, s));
      e->phase_ms[2] += lap(t);
      HIPCHK(hipStreamSynchronize(s));
      e->phase_ms[3] += lap(t);
      for (int i = 0; i < N; ++i) {
        std::memcpy(probs + ((size_t)i * B + b0) * C, hp + (size_t)i * nb * C, (size_t)nb * C * 4);
        if (logits) std::memcpy(logits + ((size_t)i * B + b0) * C, hl + (size_t)i * nb * C, (size_t)nb * C * 4);
        if (top1) std::memcpy(top1 + (size_t)i * B + b0, ht + (size_t)i * nb, (size_t)nb * 4);
      }
      if (mean_probs) std::memcpy(mean_probs + (size_t)b0 * C, hm, (size_t)nb * C * 4);
      std::memcpy(vote + b0, hv, (size_t)nb * 4);
      e->phase_ms[4] += lap(t);
    }
  });
}

void fs_destroy(fs_ensemble* e) {
  try {
    destroy_impl(e);
  } catch (...) {
  }
}

const char* fs_last_error(const fs_ensemble* e) { return e ? e->err.c_str() : g_thread_error.c_str(); }

fs_status fs_query(const fs_ensemble* ce, fs_info* info) {
  fs_ensemble* e = const_cast<fs_ensemble*>(ce);
  if (!e || !info) {
    g_thread_error = "NULL argument";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    info->num_models = e->N;
    info->num_classes = e->C;
    info->max_batch = e->max_batch;
    info->precision = e->prec == BF16 ? FS_BF16 : FS_F32;
    info->num_groups = (int32_t)e->groups.size();
    info->launches_per_pass = launches_per_pass(e);
    info->weight_bytes = (int64_t)e->arena_bytes;
    info->workspace_bytes = e->workspace_bytes;
    info->flops_per_image = e->flops_per_image;
  });
}

fs_status fs_graphs_enable(fs_ensemble* e, int32_t enable) {
  if (!e) {
    g_thread_error = "ensemble is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    HIPCHK(hipSetDevice(e->device));
    HIPCHK(hipStreamSynchronize(e->stream));
    if (e->pass_pending) HIPCHK(hipEventSynchronize(e->pass_done));
    clear_graphs(e);
    e->graphs = enable != 0;
  });
}

fs_status fs_set_combine(fs_ensemble* e, int32_t policy, int32_t positive_class, int32_t min_votes) {
  if (!e) {
    g_thread_error = "ensemble is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    check_combine(policy, positive_class, min_votes, e->N, e->C);
    HIPCHK(hipSetDevice(e->device));
    HIPCHK(hipStreamSynchronize(e->stream));
    if (e->pass_pending) HIPCHK(hipEventSynchronize(e->pass_done));
    clear_graphs(e);  // the recorded passes carry the old policy's arguments
    e->combine = policy;
    e->pos_class = policy == FS_COMBINE_ANY ? positive_class : 0;
    e->min_votes = policy == FS_COMBINE_ANY ? min_votes : 1;
  });
}

fs_status fs_profile_enable(fs_ensemble* e, int32_t enable) {
  if (!e) {
    g_thread_error = "ensemble is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    HIPCHK(hipSetDevice(e->device));
    HIPCHK(hipDeviceSynchronize());
    prof_clear(e);
    e->prof_on = enable != 0;
  });
}

fs_status fs_profile_read(fs_ensemble* e, fs_kernel_stat* stats, int32_t max_stats, int32_t* n_stats) {
  if (!e || !stats || !n_stats) {
    g_thread_error = "NULL argument";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    HIPCHK(hipSetDevice(e->device));
    fs_kernel_stat acc[K_NCLASS];
    std::memset(acc, 0, sizeof(acc));
    for (int c = 0; c < K_NCLASS; ++c) std::snprintf(acc[c].name, sizeof(acc[c].name), "%s", kClassName[c]);
    for (ProfRec& r : e->prof) {
      HIPCHK(hipEventSynchronize(r.b));
      float ms = 0.f;
      HIPCHK(hipEventElapsedTime(&ms, r.a, r.b));
      acc[r.cls].launches += r.launches;
      acc[r.cls].total_ms += ms;
      acc[r.cls].flops += r.flops;
      acc[r.cls].bytes += r.bytes;
    }
    int n = 0;
    for (int c = 0; c < K_NCLASS && n < max_stats; ++c)
      if (acc[c].launches) stats[n++] = acc[c];
    *n_stats = n;
  });
}

fs_status fs_profile_launches(fs_ensemble* e, fs_launch_stat* out, int32_t max_out, int32_t* n_out) {
  if (!e || !out || !n_out) {
    g_thread_error = "NULL argument";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    HIPCHK(hipSetDevice(e->device));
    int n = 0;
    for (ProfRec& r : e->prof) {
      if (n >= max_out) break;
      HIPCHK(hipEventSynchronize(r.b));
      float ms = 0.f;
      HIPCHK(hipEventElapsedTime(&ms, r.a, r.b));
      fs_launch_stat& o = out[n++];
      std::memset(&o, 0, sizeof(o));
      std::snprintf(o.kclass, sizeof(o.kclass), "%s", kClassName[r.cls]);
      std::snprintf(o.kernel, sizeof(o.kernel), "%s", r.kernel ? r.kernel : "");
      o.group = r.group; o.layer = r.layer; o.M = r.M; o.N = r.N; o.K = r.K; o.Z = r.Z;
      o.ms = ms; o.flops = r.flops; o.bytes = r.bytes;
    }
    *n_out = n;
  });
}

fs_status fs_tuning_log(fs_ensemble* e, char* buf, int64_t n, int64_t* needed) {
  if (!e) {
    g_thread_error = "ensemble is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  if (needed) *needed = (int64_t)e->tune_log.size() + 1;
  if (buf && n > 0) {
    const size_t k = std::min<size_t>((size_t)n - 1, e->tune_log.size());
    std::memcpy(buf, e->tune_log.data(), k);
    buf[k] = 0;
  }
  return FS_OK;
}

fs_status fs_infer_phases(fs_ensemble* e, double* ms) {
  if (!e || !ms) {
    g_thread_error = "ensemble or ms is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  for (int i = 0; i < 5; ++i) ms[i] = e->phase_ms[i];
  return FS_OK;
}

fs_status fs_debug_capture(fs_ensemble* e, int32_t image) {
  if (!e) {
    g_thread_error = "ensemble is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    if (image < -1 || image >= e->max_batch) fail(FS_ERR_INVALID, "image must be -1 or in 0..max_batch-1");
    HIPCHK(hipSetDevice(e->device));
    HIPCHK(hipStreamSynchronize(e->stream));
    if (e->pass_pending) HIPCHK(hipEventSynchronize(e->pass_done));
    e->dbg_image = -1;
    e->dbg_off.assign(e->N, {});
    e->dbg_bytes.assign(e->N, {});
    e->dbg_have.assign(e->N, {});
    e->dbg_in_have = false;
    if (image < 0) {
      e->dbg.release();
      return;
    }
    const size_t esz = es(e->prec);
    int64_t off = 0;
    e->dbg_in_off = 0;
    e->dbg_in_bytes = e->need_plain ? (int64_t)e->pre.out_h * e->pre.out_w * 4 * esz
                                    : (int64_t)(e->pre.out_h / 2) * (e->pre.out_w / 2) * 16 * 2;
    off = (int64_t)round_up(e->dbg_in_bytes, 256);
    for (const Group& g : e->groups) {
      for (int z = 0; z < g.Z; ++z) {
        const int m = g.first + z;
        e->dbg_off[m].assign(g.layers.size(), -1);
        e->dbg_bytes[m].assign(g.layers.size(), 0);
        e->dbg_have[m].assign(g.layers.size(), 0);
        for (size_t li = 0; li < g.layers.size(); ++li) {
          const LayerPlan& P = g.layers[li];
          if (P.op == FS_OP_CONV && (P.pool_fused || P.proj_into >= 0)) continue;  // never stored
          const int64_t elems = P.last ? e->C : P.out.elems();
          e->dbg_off[m][li] = off;
          e->dbg_bytes[m][li] = elems * (int64_t)(P.last ? 4 : esz);
          off += (int64_t)round_up(e->dbg_bytes[m][li], 256);
        }
      }
    }
    e->dbg.alloc(std::max<int64_t>(off, 256));
    e->dbg_image = image;
  });
}

fs_status fs_debug_layer(fs_ensemble* e, int32_t model, int32_t layer, float* out, int64_t n) {
  if (!e || !out) {
    g_thread_error = "ensemble or out is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(e->mu);
  return guarded(e, [&] {
    if (e->dbg_image < 0) fail(FS_ERR_INVALID, "no capture armed (fs_debug_capture)");
    if (model < 0 || model >= e->N) fail(FS_ERR_INVALID, "model out of range");
    HIPCHK(hipSetDevice(e->device));
    HIPCHK(hipStreamSynchronize(e->stream));
    if (e->pass_pending) HIPCHK(hipEventSynchronize(e->pass_done));
    const size_t esz = es(e->prec);
    if (layer == -1) {
      if (!e->dbg_in_have) fail(FS_ERR_INVALID, "the last pass captured no input");
      const int oh = e->pre.out_h, ow = e->pre.out_w;
      if (n != (int64_t)oh * ow * 3) fail(FS_ERR_INVALID, "n must be out_h * out_w * 3 for the input");
      std::vector<float> raw;
      const int64_t ne = e->dbg_in_bytes / (e->need_plain ? (int64_t)esz : 2);
      raw.resize(ne);
      download_as(raw.data(), static_cast<char*>(e->dbg.p) + e->dbg_in_off, ne, e->need_plain ? e->prec : BF16);
      for (int y = 0; y < oh; ++y)
        for (int x = 0; x < ow; ++x)
          for (int c = 0; c < 3; ++c)
            out[((int64_t)y * ow + x) * 3 + c] =
                e->need_plain ? raw[((int64_t)y * ow + x) * 4 + c]
                              : raw[((int64_t)(y / 2) * (ow / 2) + x / 2) * 16 + ((y & 1) * 2 + (x & 1)) * 3 + c];
      return;
    }
    if (layer < 0 || layer >= (int32_t)e->dbg_off[model].size()) fail(FS_ERR_INVALID, "layer out of range");
    if (e->dbg_off[model][layer] < 0) fail(FS_ERR_UNSUPPORTED, "this layer's output is never stored (fused)");
    if (!e->dbg_have[model][layer]) fail(FS_ERR_UNSUPPORTED, "the last pass stored no copy of this layer");
    int gi = 0;
    while (!(e->groups[gi].first <= model && model < e->groups[gi].first + e->groups[gi].Z)) ++gi;
    const LayerPlan& P = e->groups[gi].layers[layer];
    const int64_t elems = P.last ? e->C : P.out.elems();
    if (n != elems) fail(FS_ERR_INVALID, "n must be the layer's H * W * C");
    download_as(out, static_cast<char*>(e->dbg.p) + e->dbg_off[model][layer], elems, P.last ? F32 : e->prec);
  });
}

// ---------------------------------------------------------- test entries
fs_status fs_test_preprocess(const fs_image* imgs, int32_t B, int32_t out_h, int32_t out_w, const float mean[3],
                             const float std_[3], int32_t precision, int32_t layout, float* out, int32_t device) {
  return guarded(nullptr, [&] {
    Prec p = prec_of(precision);
    check_images(imgs, B);
    if (B == 0) return;
    if (out_h < 1 || out_w < 1 || !mean || !std_ || !out) fail(FS_ERR_INVALID, "bad preprocess arguments");
    if (layout != 0 && layout != 1) fail(FS_ERR_INVALID, "layout must be 0 (NHWC4) or 1 (space-to-depth)");
    if (layout == 1 && (p != BF16 || out_h % 2 || out_w % 2))
      fail(FS_ERR_UNSUPPORTED, "space-to-depth output needs bf16 and an even output size");
    set_device(device);
    TmpDev t;
    const size_t pb = packed_size(imgs, 0, B);
    std::vector<uint8_t> hp(pb);
    std::vector<ImageDesc> hd(B);
    pack_images(imgs, 0, B, hp.data(), hd.data());
    void* dp = t.alloc(pb);
    void* dd = t.alloc(B * sizeof(ImageDesc));
    const int64_t n = (int64_t)B * out_h * out_w * 4;
    void* dout = t.alloc(n * es(p));
    HIPCHK(hipMemcpy(dp, hp.data(), pb, hipMemcpyHostToDevice));
    HIPCHK(hipMemcpy(dd, hd.data(), B * sizeof(ImageDesc), hipMemcpyHostToDevice));
    PreArgs a{};
    a.pixels = static_cast<const uint8_t*>(dp);
    a.desc = static_cast<const ImageDesc*>(dd);
    a.B = B; a.out_h = out_h; a.out_w = out_w;
    for (int c = 0; c < 3; ++c) { a.mean[c] = mean[c]; a.std_[c] = std_[c]; }
    a.out = layout == 0 ? dout : nullptr;
    a.out_s2d = layout == 1 ? dout : nullptr;
    launch_preprocess(a, p, nullptr);
    HIPCHK(hipGetLastError());
    HIPCHK(hipDeviceSynchronize());
    download_as(out, dout, n, p);
  });
}

// One conv on host tensors; with stem_pool the space-to-depth stem kernel
// that also applies the 3x3/2/p1 max pool runs instead, and out receives
// the pooled tensor.
static void run_test_conv(const float* in, int32_t B, int32_t H, int32_t W, int32_t Cin, const float* w,
                          const float* bias, const float* res, int32_t Cout, int32_t kh, int32_t kw, int32_t stride,
                          int32_t pad, int32_t relu, int32_t precision, int32_t tile, float* out, int32_t device,
                          bool stem_pool) {
  {
    Prec p = prec_of(precision);
    if (!in || !w || !out || B < 1 || H < 1 || W < 1 || Cin < 1 || Cout < 1 || kh < 1 || kw < 1 || stride < 1 ||
        pad < 0)
      fail(FS_ERR_INVALID, "bad conv arguments");
    if (H + 2 * pad < kh || W + 2 * pad < kw) fail(FS_ERR_INVALID, "conv output would be empty");
    if (Cout % 8) fail(FS_ERR_UNSUPPORTED, "Cout must be a multiple of 8");
    const int cin_p = Cin == 3 ? 4 : Cin;
    if (Cin != 3 && Cin % (p == BF16 ? 8 : 4)) fail(FS_ERR_UNSUPPORTED, "Cin must be 3 or a multiple of the vector width");
    const int Ho = (H + 2 * pad - kh) / stride + 1, Wo = (W + 2 * pad - kw) / stride + 1;
    if ((int64_t)B * H * W * cin_p * es(p) >= (int64_t(1) << 31) ||
        (int64_t)B * Ho * Wo * Cout * es(p) >= (int64_t(1) << 31))
      fail(FS_ERR_UNSUPPORTED, "tensor exceeds 2 GiB");
    set_device(device);
    TmpDev t;
    fs_layer L{};
    L.op = FS_OP_CONV; L.src = -1; L.cin = Cin; L.cout = Cout; L.kh = kh; L.kw = kw; L.stride = stride; L.pad = pad;
    L.weight = w; L.bias = bias;
    fs_preprocess pre{};
    pre.out_h = H; pre.out_w = W;
    // the space-to-depth form whenever the requested tile cannot gather
    // 4-channel pixels (as the ensemble does for a stride-2 first conv)
    const bool use_s2d = s2d_eligible(L, pre, p) && (tile < 0 || conv_tile(p, tile).vec == 8);
    std::vector<float> xin, w16;
    const float* xsrc = in;
    int gH = H, gW = W, gC = cin_p, gk = kh, gs = stride, gp = pad;
    if (use_s2d) {
      gH = H / 2; gW = W / 2; gC = 16;
      xin.assign((size_t)B * gH * gW * 16, 0.f);
      for (int b = 0; b < B; ++b)
        for (int y = 0; y < H; ++y)
          for (int x = 0; x < W; ++x)
            for (int c = 0; c < 3; ++c)
              xin[(((size_t)b * gH + y / 2) * gW + x / 2) * 16 + ((y & 1) * 2 + (x & 1)) * 3 + c] =
                  in[(((size_t)b * H + y) * W + x) * 3 + c];
      xsrc = xin.data();
      w16 = s2d_weights(L);
      L = s2d_layer(L, w16);
      gk = L.kh; gs = 1; gp = L.pad;
    } else if (cin_p != Cin) {  // pad the channel dimension with zeros
      xin.assign((size_t)B * H * W * cin_p, 0.f);
      for (int64_t px = 0; px < (int64_t)B * H * W; ++px)
        for (int c = 0; c < Cin; ++c) xin[px * cin_p + c] = in[px * Cin + c];
      xsrc = xin.data();
    }
    void* dx = upload_as(t, xsrc, (int64_t)B * gH * gW * gC, p);
    const int K = gk * gk * gC, Kp = (int)round_up(K, CONV_KPAD);
    std::vector<char> wp((size_t)Cout * Kp * es(p));
    std::vector<float> bp(Cout);
    pack_conv(L, gC, Kp, p, wp.data(), bp.data());
    void* dw = t.alloc(wp.size());
    HIPCHK(hipMemcpy(dw, wp.data(), wp.size(), hipMemcpyHostToDevice));
    void* dwf = nullptr;
    if (conv_frag_wanted(p, Cout, Kp)) {  // as the ensemble keeps for its bf16 conv layers
      std::vector<char> wf(wp.size());
      conv_frag_order(reinterpret_cast<const uint16_t*>(wp.data()), Cout, Kp, reinterpret_cast<uint16_t*>(wf.data()));
      dwf = t.alloc(wf.size());
      HIPCHK(hipMemcpy(dwf, wf.data(), wf.size(), hipMemcpyHostToDevice));
    }
    void* db = t.alloc(Cout * 4);
    HIPCHK(hipMemcpy(db, bp.data(), Cout * 4, hipMemcpyHostToDevice));
    const int64_t no = (int64_t)B * Ho * Wo * Cout;
    void* dr = res ? upload_as(t, res, no, p) : nullptr;
    void* dy = t.alloc(no * es(p));
    ConvArgs a{};
    a.x = dx; a.w = dw; a.wf = dwf; a.bias = static_cast<const float*>(db); a.res = dr; a.y = dy;
    a.B = B; a.H = gH; a.W = gW; a.Cin = gC; a.Ho = Ho; a.Wo = Wo; a.Cout = Cout;
    a.kh = gk; a.kw = gk; a.stride = gs; a.pad = gp; a.relu = relu ? 1 : 0;
    a.K = K; a.Kp = Kp; a.M = B * Ho * Wo; a.Z = 1;
    if (stem_pool) {
      if (!use_s2d || !conv_stem_pool_ok(a)) fail(FS_ERR_UNSUPPORTED, "not a space-to-depth stem the fused kernel takes");
      const int64_t npool = (int64_t)B * ((Ho - 1) / 2 + 1) * ((Wo - 1) / 2 + 1) * Cout;
      launch_conv_stem_pool(a, nullptr);
      HIPCHK(hipGetLastError());
      HIPCHK(hipDeviceSynchronize());
      download_as(out, dy, npool, p);
      return;
    }
    int tl = tile;
    if (tl < 0) tl = conv_pick_tile(p, a, num_cus_of(device));
    if (!conv_tile_ok(p, tl, a)) fail(FS_ERR_UNSUPPORTED, "tile " + std::to_string(tile) + " does not fit this conv");
    if (conv_tile_direct(conv_tile(p, tl))) {  // the ensemble's split rule, so split-K is exercised too
      a.split = conv_split(p, a, num_cus_of(device));
      if (a.split > 1) a.partial = static_cast<float*>(t.alloc(conv_partial_floats(a) * 4));
    }
    launch_conv(a, p, tl, nullptr);
    HIPCHK(hipGetLastError());
    HIPCHK(hipDeviceSynchronize());
    download_as(out, dy, no, p);
  }
}

fs_status fs_test_conv(const float* in, int32_t B, int32_t H, int32_t W, int32_t Cin, const float* w,
                       const float* bias, const float* res, int32_t Cout, int32_t kh, int32_t kw, int32_t stride,
                       int32_t pad, int32_t relu, int32_t precision, int32_t tile, float* out, int32_t device) {
  return guarded(nullptr, [&] {
    run_test_conv(in, B, H, W, Cin, w, bias, res, Cout, kh, kw, stride, pad, relu, precision, tile, out, device,
                  false);
  });
}

fs_status fs_test_stem_pool(const float* in, int32_t B, int32_t H, int32_t W, const float* w, const float* bias,
                            float* out, int32_t device) {
  return guarded(nullptr, [&] {
    if (H % 2 || W % 2) fail(FS_ERR_UNSUPPORTED, "the space-to-depth stem needs even H and W");
    run_test_conv(in, B, H, W, 3, w, bias, nullptr, 64, 7, 7, 2, 3, 1, FS_BF16, -1, out, device, true);
  });
}

fs_status fs_test_maxpool(const float* in, int32_t B, int32_t H, int32_t W, int32_t C, int32_t k, int32_t stride,
                          int32_t pad, int32_t precision, float* out, int32_t device) {
  return guarded(nullptr, [&] {
    Prec p = prec_of(precision);
    if (!in || !out || B < 1 || H < 1 || W < 1 || C < 1 || k < 1 || stride < 1 || pad < 0 || pad >= k)
      fail(FS_ERR_INVALID, "bad maxpool arguments");
    if (C % (p == BF16 ? 8 : 4)) fail(FS_ERR_UNSUPPORTED, "C must be a multiple of the vector width");
    if (H + 2 * pad < k || W + 2 * pad < k) fail(FS_ERR_INVALID, "pool output would be empty");
    const int Ho = (H + 2 * pad - k) / stride + 1, Wo = (W + 2 * pad - k) / stride + 1;
    set_device(device);
    TmpDev t;
    void* dx = upload_as(t, in, (int64_t)B * H * W * C, p);
    const int64_t no = (int64_t)B * Ho * Wo * C;
    void* dy = t.alloc(no * es(p));
    PoolArgs a{};
    a.x = dx; a.y = dy; a.B = B; a.H = H; a.W = W; a.C = C; a.Ho = Ho; a.Wo = Wo;
    a.k = k; a.stride = stride; a.pad = pad; a.Z = 1;
    launch_maxpool(a, p, nullptr);
    HIPCHK(hipGetLastError());
    HIPCHK(hipDeviceSynchronize());
    download_as(out, dy, no, p);
  });
}

fs_status fs_test_gap(const float* in, int32_t B, int32_t H, int32_t W, int32_t C, int32_t precision, float* out,
                      int32_t device) {
  return guarded(nullptr, [&] {
    Prec p = prec_of(precision);
    if (!in || !out || B < 1 || H < 1 || W < 1 || C < 1) fail(FS_ERR_INVALID, "bad gap arguments");
    if (C % (p == BF16 ? 8 : 4)) fail(FS_ERR_UNSUPPORTED, "C must be a multiple of the vector width");
    set_device(device);
    TmpDev t;
    void* dx = upload_as(t, in, (int64_t)B * H * W * C, p);
    void* dy = t.alloc((size_t)B * C * es(p));
    PoolArgs a{};
    a.x = dx; a.y = dy; a.B = B; a.H = H; a.W = W; a.C = C; a.Ho = 1; a.Wo = 1; a.Z = 1;
    launch_gap(a, p, nullptr);
    HIPCHK(hipGetLastError());
    HIPCHK(hipDeviceSynchronize());
    download_as(out, dy, (int64_t)B * C, p);
  });
}

fs_status fs_test_fc(const float* in, int32_t B, int32_t K, const float* w, const float* bias, int32_t N,
                     int32_t relu, int32_t precision, int32_t out_storage, float* out, int32_t device) {
  return guarded(nullptr, [&] {
    Prec p = prec_of(precision);
    if (!in || !w || !out || B < 1 || K < 1 || N < 1) fail(FS_ERR_INVALID, "bad fc arguments");
    if (p == BF16 && K % 8) fail(FS_ERR_UNSUPPORTED, "bf16 K must be a multiple of 8");
    set_device(device);
    const int cus = num_cus_of(device);
    TmpDev t;
    void* dx = upload_as(t, in, (int64_t)B * K, p);
    void* dw = upload_as(t, w, (int64_t)N * K, p);
    std::vector<float> b(N, 0.f);
    if (bias) std::copy(bias, bias + N, b.begin());
    void* db = t.alloc(N * 4);
    HIPCHK(hipMemcpy(db, b.data(), N * 4, hipMemcpyHostToDevice));
    const bool f32out = !out_storage || p == F32;
    void* dy = t.alloc((size_t)B * N * (f32out ? 4 : es(p)));
    FcArgs a{};
    a.x = dx; a.w = dw; a.bias = static_cast<const float*>(db); a.y = dy;
    a.B = B; a.K = K; a.N = N; a.relu = relu ? 1 : 0; a.out_f32 = f32out ? 1 : 0; a.Z = 1;
    a.split = fc_pick_split(p, B, K, N, 1, cus);
    a.partial = static_cast<float*>(t.alloc(std::max<size_t>(fc_partial_floats(B, N, a.split, 1), 1) * 4));
    launch_fc(a, p, nullptr);
    HIPCHK(hipGetLastError());
    HIPCHK(hipDeviceSynchronize());
    download_as(out, dy, (int64_t)B * N, f32out ? F32 : p);
  });
}

fs_status fs_test_softmax_combine(const float* logits, int32_t N, int32_t B, int32_t C, float* probs, float* mean,
                                  int32_t* vote, int32_t* top1, int32_t device) {
  return fs_test_softmax_combine_policy(logits, N, B, C, FS_COMBINE_MEAN, 0, 1, probs, mean, vote, top1, device);
}

fs_status fs_test_softmax_combine_policy(const float* logits, int32_t N, int32_t B, int32_t C, int32_t policy,
                                         int32_t positive_class, int32_t min_votes, float* probs, float* mean,
                                         int32_t* vote, int32_t* top1, int32_t device) {
  return guarded(nullptr, [&] {
    if (!logits || !probs || !vote || N < 1 || B < 1 || C < 1) fail(FS_ERR_INVALID, "bad softmax arguments");
    if (C > SOFTMAX_MAX_C) fail(FS_ERR_UNSUPPORTED, "more than 4096 classes");
    check_combine(policy, positive_class, min_votes, N, C);
    set_device(device);
    TmpDev t;
    const size_t n = (size_t)N * B * C;
    void* dz = t.alloc(n * 4);
    HIPCHK(hipMemcpy(dz, logits, n * 4, hipMemcpyHostToDevice));
    void* dp = t.alloc(n * 4);
    void* dm = t.alloc((size_t)B * C * 4);
    void* dv = t.alloc((size_t)B * 4);
    void* dt = t.alloc((size_t)N * B * 4);
    SoftmaxArgs a{};
    a.logits = static_cast<const float*>(dz);
    a.probs = static_cast<float*>(dp);
    a.mean = mean ? static_cast<float*>(dm) : nullptr;
    a.vote = static_cast<int32_t*>(dv);
    a.top1 = top1 ? static_cast<int32_t*>(dt) : nullptr;
    a.N = N; a.B = B; a.C = C;
    a.policy = policy; a.pos_class = positive_class; a.min_votes = min_votes;
    launch_softmax_combine(a, nullptr);
    HIPCHK(hipGetLastError());
    HIPCHK(hipDeviceSynchronize());
    HIPCHK(hipMemcpy(probs, dp, n * 4, hipMemcpyDeviceToHost));
    if (mean) HIPCHK(hipMemcpy(mean, dm, (size_t)B * C * 4, hipMemcpyDeviceToHost));
    HIPCHK(hipMemcpy(vote, dv, (size_t)B * 4, hipMemcpyDeviceToHost));
    if (top1) HIPCHK(hipMemcpy(top1, dt, (size_t)N * B * 4, hipMemcpyDeviceToHost));
  });
}

fs_status fs_bench_conv(int32_t B, int32_t H, int32_t W, int32_t Cin, int32_t Cout, int32_t kh, int32_t kw,
                        int32_t stride, int32_t pad, int32_t relu, int32_t residual, int32_t precision, int32_t tile,
                        int32_t Z, int32_t iters, double* avg_ms, int32_t* tile_used, int32_t device) {
  return guarded(nullptr, [&] {
    Prec p = prec_of(precision);
    if (!avg_ms || B < 1 || H < 1 || W < 1 || Cin < 1 || Cout < 1 || kh < 1 || kw < 1 || stride < 1 || pad < 0 ||
        Z < 1 || iters < 1)
      fail(FS_ERR_INVALID, "bad bench arguments");
    if (H + 2 * pad < kh || W + 2 * pad < kw) fail(FS_ERR_INVALID, "conv output would be empty");
    if (Cout % 8) fail(FS_ERR_UNSUPPORTED, "Cout must be a multiple of 8");
    const int cin_p = Cin == 3 ? 4 : Cin;
    if (Cin != 3 && Cin % (p == BF16 ? 8 : 4)) fail(FS_ERR_UNSUPPORTED, "Cin must be 3 or a multiple of the vector width");
    const int Ho = (H + 2 * pad - kh) / stride + 1, Wo = (W + 2 * pad - kw) / stride + 1;
    const int64_t nx = (int64_t)B * H * W * cin_p, ny = (int64_t)B * Ho * Wo * Cout;
    if (nx * es(p) >= (int64_t(1) << 31) || ny * es(p) >= (int64_t(1) << 31))
      fail(FS_ERR_UNSUPPORTED, "tensor exceeds 2 GiB");
    set_device(device);
    fs_layer L{};
    L.op = FS_OP_CONV; L.src = -1; L.cin = Cin; L.cout = Cout; L.kh = kh; L.kw = kw; L.stride = stride; L.pad = pad;
    fs_preprocess pre{};
    pre.out_h = H; pre.out_w = W;
    int gH = H, gW = W, gC = cin_p, gk = kh, gs = stride, gp = pad;
    if (s2d_eligible(L, pre, p) && (tile < 0 || conv_tile(p, tile).vec == 8)) {
      const S2dGeom g = s2d_geom(kh);
      gH = H / 2; gW = W / 2; gC = 16; gk = g.ks; gs = 1; gp = g.pad;
    }
    const int K = gk * gk * gC, Kp = (int)round_up(K, CONV_KPAD);
    const int64_t nxg = (int64_t)B * gH * gW * gC;
    TmpDev t;
    const size_t e = es(p);
    void* dx = t.alloc(nxg * e);
    void* dw = t.alloc((size_t)Z * Cout * Kp * e);
    void* db = t.alloc((size_t)Z * Cout * 4);
    void* dr = residual ? t.alloc((size_t)Z * ny * e) : nullptr;
    void* dy = t.alloc((size_t)Z * ny * e);
    void* dwf = conv_frag_wanted(p, Cout, Kp) ? t.alloc((size_t)Z * Cout * Kp * e) : nullptr;
    // small finite values everywhere (0x3c00 = 2^-7 in bf16; constant
    // weights are their own fragment order)
    HIPCHK(hipMemsetD16(reinterpret_cast<hipDeviceptr_t>(dx), 0x3c00, nxg * e / 2));
    HIPCHK(hipMemsetD16(reinterpret_cast<hipDeviceptr_t>(dw), 0x3c00, (size_t)Z * Cout * Kp * e / 2));
    if (dwf) HIPCHK(hipMemsetD16(reinterpret_cast<hipDeviceptr_t>(dwf), 0x3c00, (size_t)Z * Cout * Kp * e / 2));
    HIPCHK(hipMemset(db, 0, (size_t)Z * Cout * 4));
    if (dr) HIPCHK(hipMemset(dr, 0, (size_t)Z * ny * e));
    ConvArgs a{};
    a.x = dx; a.x_mstride = 0;
    a.w = dw; a.w_mstride = (int64_t)Cout * Kp;
    a.wf = dwf; a.wf_mstride = (int64_t)Cout * Kp;
    a.bias = static_cast<const float*>(db); a.b_mstride = Cout;
    a.res = dr; a.res_mstride = ny;
    a.y = dy; a.y_mstride = ny;
    a.B = B; a.H = gH; a.W = gW; a.Cin = gC; a.Ho = Ho; a.Wo = Wo; a.Cout = Cout;
    a.kh = gk; a.kw = gk; a.stride = gs; a.pad = gp; a.relu = relu ? 1 : 0;
    a.K = K; a.Kp = Kp; a.M = B * Ho * Wo; a.Z = Z;
    int tl = tile < 0 ? conv_pick_tile(p, a, num_cus_of(device)) : tile;
    if (!conv_tile_ok(p, tl, a)) fail(FS_ERR_UNSUPPORTED, "tile does not fit this conv");
    if (conv_tile_direct(conv_tile(p, tl))) {
      a.split = conv_split(p, a, num_cus_of(device));
      if (a.split > 1) a.partial = static_cast<float*>(t.alloc(conv_partial_floats(a) * 4));
    }
    if (tile_used) *tile_used = tl;
    hipStream_t s = nullptr;
    for (int i = 0; i < 3; ++i) launch_conv(a, p, tl, s);
    HIPCHK(hipGetLastError());
    hipEvent_t e0, e1;
    HIPCHK(hipEventCreate(&e0));
    HIPCHK(hipEventCreate(&e1));
    HIPCHK(hipEventRecord(e0, s));
    for (int i = 0; i < iters; ++i) launch_conv(a, p, tl, s);
    HIPCHK(hipEventRecord(e1, s));
    HIPCHK(hipEventSynchronize(e1));
    float ms = 0.f;
    HIPCHK(hipEventElapsedTime(&ms, e0, e1));
    (void)hipEventDestroy(e0);
    (void)hipEventDestroy(e1);
    HIPCHK(hipGetLastError());
    *avg_ms = ms / iters;
  });
}

int32_t fs_conv_num_tiles(int32_t precision) {
  if (precision != FS_F32 && precision != FS_BF16) return 0;
  return conv_num_tiles(precision == FS_BF16 ? BF16 : F32);
}

const char* fs_conv_tile_name(int32_t precision, int32_t tile) {
  if (precision != FS_F32 && precision != FS_BF16) return nullptr;
  const Prec p = precision == FS_BF16 ? BF16 : F32;
  if (tile < 0 || tile >= conv_num_tiles(p)) return nullptr;
  return conv_tile(p, tile).name;
}

}  // extern "C"
