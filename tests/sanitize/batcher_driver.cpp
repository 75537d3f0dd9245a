// Host-only driver of the request batcher (csrc/batcher.cpp) for sanitizer
// builds: the ensemble entry points the batcher calls are replaced by a stub
// whose "pass" writes outputs derived from each image's first byte, so every
// caller can check it got its own images' results.  Exercises concurrent
// callers, coalescing, and destroying the batcher while requests are queued
// and callers are still waking up.
#include "flexserve.h"

#include <atomic>
#include <chrono>
#include <cstdio>
#include <cstdlib>
#include <cstring>
#include <thread>
#include <vector>

namespace {
constexpr int N = 2, C = 5, MAXB = 16;
std::atomic<int> g_passes{0};
int g_pass_sleep_ms = 1;
}  // namespace

extern "C" {
struct fs_ensemble {
  int id;
};

fs_status fs_infer(fs_ensemble*, const fs_image* imgs, int32_t B, float* probs, float* mean, int32_t* vote,
                   int32_t* top1, float* logits) {
  std::this_thread::sleep_for(std::chrono::milliseconds(g_pass_sleep_ms));
  for (int b = 0; b < B; ++b) {
    const float v = imgs[b].data[0];
    for (int i = 0; i < N; ++i)
      for (int c = 0; c < C; ++c) {
        probs[((size_t)i * B + b) * C + c] = v + i + c;
        if (logits) logits[((size_t)i * B + b) * C + c] = -v;
      }
    if (mean)
      for (int c = 0; c < C; ++c) mean[(size_t)b * C + c] = v;
    vote[b] = (int)v;
    if (top1)
      for (int i = 0; i < N; ++i) top1[(size_t)i * B + b] = (int)v + i;
  }
  ++g_passes;
  return FS_OK;
}

fs_status fs_query(const fs_ensemble*, fs_info* info) {
  std::memset(info, 0, sizeof(*info));
  info->num_models = N;
  info->num_classes = C;
  info->max_batch = MAXB;
  info->weight_bytes = 1;
  return FS_OK;
}

const char* fs_last_error(const fs_ensemble*) { return "stub"; }
}

static bool request(fs_batcher* b, int tag, int B) {
  std::vector<uint8_t> px(B * 3);
  std::vector<fs_image> im(B);
  for (int k = 0; k < B; ++k) {
    px[k * 3] = (uint8_t)((tag + k) & 0xff);
    im[k] = fs_image{&px[k * 3], 1, 1, 3};
  }
  std::vector<float> probs((size_t)N * B * C), mean((size_t)B * C);
  std::vector<int32_t> vote(B), top1((size_t)N * B);
  if (fs_batcher_infer(b, im.data(), B, probs.data(), mean.data(), vote.data(), top1.data(), nullptr) != FS_OK)
    return false;
  for (int k = 0; k < B; ++k) {
    const int v = (tag + k) & 0xff;
    if (vote[k] != v || top1[(size_t)1 * B + k] != v + 1 || probs[((size_t)1 * B + k) * C + 4] != v + 5.0f ||
        mean[(size_t)k * C] != (float)v)
      return false;
  }
  return true;
}

int main() {
  fs_ensemble h0{0}, h1{1};
  fs_ensemble* hs[2] = {&h0, &h1};
  // 1. many concurrent callers, two workers
  {
    fs_batcher* b = nullptr;
    if (fs_batcher_create(hs, 2, 200, &b) != FS_OK) return 1;
    std::atomic<int> bad{0};
    std::vector<std::thread> ts;
    for (int t = 0; t < 8; ++t)
      ts.emplace_back([&, t] {
        for (int r = 0; r < 40; ++r)
          if (!request(b, t * 31 + r, 1 + (t * 7 + r) % 20)) ++bad;  // some above max_batch
      });
    for (auto& t : ts) t.join();
    int64_t passes = 0, reqs = 0, imgs = 0;
    fs_batcher_stats(b, &passes, &reqs, &imgs);
    fs_batcher_destroy(b);
    if (bad || reqs != 320) {
      std::printf("concurrent callers: %d bad results, %lld requests\n", bad.load(), (long long)reqs);
      return 1;
    }
  }
  // 2. destroy while requests are queued and their callers blocked
  for (int round = 0; round < 20; ++round) {
    g_pass_sleep_ms = 5;
    fs_batcher* b = nullptr;
    if (fs_batcher_create(hs, 1, 1000, &b) != FS_OK) return 1;
    std::atomic<int> entered{0}, bad{0};
    std::vector<std::thread> ts;
    for (int t = 0; t < 6; ++t)
      ts.emplace_back([&, t] {
        ++entered;
        if (!request(b, t * 13 + round, 3 + t)) ++bad;
      });
    while (entered.load() < 6) std::this_thread::yield();
    std::this_thread::sleep_for(std::chrono::milliseconds(20));
    fs_batcher_destroy(b);  // serves the queue, returns once every caller has left
    for (auto& t : ts) t.join();
    if (bad) {
      std::printf("destroy with queued requests: %d bad results\n", bad.load());
      return 1;
    }
  }
  std::printf("batcher driver ok (%d passes)\n", g_passes.load());
  return 0;
}
