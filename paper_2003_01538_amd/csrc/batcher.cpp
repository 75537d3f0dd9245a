// Cross-request coalescing for one ensemble.
//
// FlexServe takes batches of any size per request (Sec. 2.3) and scales
// over concurrent clients with server workers (Sec. 2.2).  On one GPU, small
// requests from concurrent clients waste most of a pass: the layers of a
// batch of 2 run at a fraction of the chip.  The batcher queues the requests
// of every calling thread; a worker thread takes whole requests in arrival
// order, up to max_batch images (a single larger request alone, which
// fs_infer chunks), waiting at most max_wait_us after the first for more to
// arrive, runs them as ONE fs_infer, and hands every caller its own slice of
// the outputs.  There is one worker per handle given, each handle one of the
// same ensemble (fs_ensemble_share: same weights, own workspace and
// stream), so one worker's host staging and copies overlap another's device
// pass.  Each
// image's result depends only on the image and on the total batch size of
// the pass it ran in (never on its neighbours or its position), so a
// coalesced request gets the bits that fs_infer gives for the same images in
// a batch of that size.
#include "flexserve.h"

#include <algorithm>
#include <chrono>
#include <condition_variable>
#include <cstring>
#include <deque>
#include <mutex>
#include <new>
#include <string>
#include <thread>
#include <vector>

namespace {

struct Request {
  const fs_image* imgs;
  int32_t B;
  float* probs;
  float* mean;
  int32_t* vote;
  int32_t* top1;
  float* logits;
  fs_status st = FS_OK;
  std::string err;
  bool done = false;
};

thread_local std::string g_batcher_error;

}  // namespace

struct Worker {
  fs_ensemble* e = nullptr;  // the caller's handle this worker runs its passes on
  std::thread th;
  // host outputs of one coalesced pass, [N][Bt][C] model-major like fs_infer
  std::vector<float> probs, mean, logits;
  std::vector<int32_t> vote, top1;
  std::vector<fs_image> imgs;
};

struct fs_batcher {
  int32_t N = 0, C = 0, max_batch = 0;
  std::chrono::microseconds max_wait{0};
  std::mutex mu;
  std::condition_variable cv_work, cv_done, cv_idle;
  std::deque<Request*> queue;
  int64_t queued_images = 0;
  int64_t callers = 0;  // threads inside fs_batcher_infer with a queued request
  bool stop = false;
  bool gathering = false;  // a worker is collecting the next pass
  int64_t passes = 0, requests = 0, images = 0;
  std::vector<Worker> workers;

  void run(Worker& w);
  void pass(Worker& w, std::vector<Request*>& batch);
  void shutdown();
};

void fs_batcher::pass(Worker& wk, std::vector<Request*>& batch) {
  fs_ensemble* e = wk.e;
  std::vector<float>& probs = wk.probs;
  std::vector<float>& mean = wk.mean;
  std::vector<float>& logits = wk.logits;
  std::vector<int32_t>& vote = wk.vote;
  std::vector<int32_t>& top1 = wk.top1;
  std::vector<fs_image>& imgs = wk.imgs;
  int64_t Bt = 0;
  bool want_mean = false, want_top1 = false, want_logits = false;
  for (Request* r : batch) {
    Bt += r->B;
    want_mean |= r->mean != nullptr;
    want_top1 |= r->top1 != nullptr;
    want_logits |= r->logits != nullptr;
  }
  imgs.clear();
  for (Request* r : batch) imgs.insert(imgs.end(), r->imgs, r->imgs + r->B);
  probs.resize((size_t)N * Bt * C);
  vote.resize((size_t)Bt);
  if (want_mean) mean.resize((size_t)Bt * C);
  if (want_top1) top1.resize((size_t)N * Bt);
  if (want_logits) logits.resize((size_t)N * Bt * C);
  const fs_status st = fs_infer(e, imgs.data(), (int32_t)Bt, probs.data(), want_mean ? mean.data() : nullptr,
                                vote.data(), want_top1 ? top1.data() : nullptr,
                                want_logits ? logits.data() : nullptr);
  const std::string err = st == FS_OK ? std::string() : std::string(fs_last_error(e));
  int64_t o = 0;  // the request's first image in the pass
  for (Request* r : batch) {
    r->st = st;
    r->err = err;
    if (st == FS_OK) {
      const size_t b = (size_t)r->B;
      for (int32_t i = 0; i < N; ++i) {
        std::memcpy(r->probs + (size_t)i * b * C, probs.data() + ((size_t)i * Bt + o) * C, b * C * 4);
        if (r->logits)
          std::memcpy(r->logits + (size_t)i * b * C, logits.data() + ((size_t)i * Bt + o) * C, b * C * 4);
        if (r->top1) std::memcpy(r->top1 + (size_t)i * b, top1.data() + (size_t)i * Bt + o, b * 4);
      }
      std::memcpy(r->vote, vote.data() + o, b * 4);
      if (r->mean) std::memcpy(r->mean, mean.data() + (size_t)o * C, b * C * 4);
    }
    o += r->B;
  }
}

// One worker at a time gathers the next pass (the others are running theirs
// or waiting their turn), so gathering overlaps the passes in flight.
void fs_batcher::run(Worker& wk) {
  std::unique_lock<std::mutex> lk(mu);
  for (;;) {
    cv_work.wait(lk, [&] { return (stop && queue.empty()) || (!gathering && !queue.empty()); });
    if (queue.empty()) break;  // stop requested and nothing left
    gathering = true;
    // give concurrent callers until the deadline to fill the pass
    const auto deadline = std::chrono::steady_clock::now() + max_wait;
    while (!stop && queued_images < max_batch)
      if (cv_work.wait_until(lk, deadline) == std::cv_status::timeout) break;
    std::vector<Request*> batch;
    int64_t total = 0;
    while (!queue.empty() && (batch.empty() || total + queue.front()->B <= max_batch)) {
      batch.push_back(queue.front());
      total += queue.front()->B;
      queue.pop_front();
    }
    queued_images -= total;
    gathering = false;
    cv_work.notify_all();  // the next worker may gather
    lk.unlock();
    try {
      pass(wk, batch);
    } catch (...) {  // host buffers of the pass could not grow: the requests fail, the worker lives on
      for (Request* r : batch) {
        r->st = FS_ERR_OOM;
        r->err = "batcher: host allocation failed";
      }
    }
    lk.lock();
    ++passes;
    requests += (int64_t)batch.size();
    images += total;
    for (Request* r : batch) r->done = true;
    cv_done.notify_all();
  }
}

// Stops the workers once the queue is empty, then waits until every caller
// whose request was served has woken and left fs_batcher_infer, so the
// mutex and condition variables are no longer in use when the batcher is
// freed.
void fs_batcher::shutdown() {
  {
    std::lock_guard<std::mutex> lk(mu);
    stop = true;
  }
  cv_work.notify_all();
  for (Worker& w : workers)
    if (w.th.joinable()) w.th.join();
  workers.clear();
  std::unique_lock<std::mutex> lk(mu);
  cv_idle.wait(lk, [&] { return callers == 0; });
}

extern "C" {

fs_status fs_batcher_create(fs_ensemble* const* handles, int32_t n_handles, int32_t max_wait_us,
                            fs_batcher** out) {
  if (out) *out = nullptr;
  if (!handles || !out || n_handles < 1 || n_handles > 16 || max_wait_us < 0) {
    g_batcher_error = "handles or out is NULL, n_handles outside 1..16, or max_wait_us < 0";
    return FS_ERR_INVALID;
  }
  fs_info first{};
  for (int32_t i = 0; i < n_handles; ++i) {
    fs_info info{};
    const fs_status st = handles[i] ? fs_query(handles[i], &info) : FS_ERR_INVALID;
    if (st != FS_OK) {
      g_batcher_error = "handle " + std::to_string(i) + " is not a valid ensemble";
      return FS_ERR_INVALID;
    }
    if (i == 0) first = info;
    if (info.num_models != first.num_models || info.num_classes != first.num_classes ||
        info.max_batch != first.max_batch || info.weight_bytes != first.weight_bytes) {
      g_batcher_error = "handle " + std::to_string(i) + " is not a handle of the first one's ensemble";
      return FS_ERR_INVALID;
    }
  }
  fs_batcher* b = new (std::nothrow) fs_batcher();
  if (!b) return FS_ERR_OOM;
  b->N = first.num_models;
  b->C = first.num_classes;
  b->max_batch = first.max_batch;
  b->max_wait = std::chrono::microseconds(max_wait_us);
  b->workers.resize(n_handles);
  for (int32_t i = 0; i < n_handles; ++i) b->workers[i].e = handles[i];
  try {
    for (Worker& w : b->workers) w.th = std::thread([b, &w] { b->run(w); });
  } catch (...) {
    b->shutdown();
    delete b;
    g_batcher_error = "cannot start the batcher threads";
    return FS_ERR_INTERNAL;
  }
  *out = b;
  return FS_OK;
}

fs_status fs_batcher_infer(fs_batcher* b, const fs_image* imgs, int32_t B, float* probs, float* mean_probs,
                           int32_t* vote, int32_t* top1, float* logits) {
  if (!b) {
    g_batcher_error = "batcher is NULL";
    return FS_ERR_INVALID;
  }
  if (B < 0 || (B > 0 && !imgs)) {
    g_batcher_error = "B must be >= 0 with an image array";
    return FS_ERR_INVALID;
  }
  if (B == 0) return FS_OK;
  if (!probs || !vote) {
    g_batcher_error = "probs and vote are required";
    return FS_ERR_INVALID;
  }
  for (int32_t i = 0; i < B; ++i) {  // checked here, so a bad request never fails the others of its pass
    const fs_image& im = imgs[i];
    if (!im.data || im.h < 1 || im.w < 1 || im.h > 32768 || im.w > 32768 || im.row_stride < 3 * im.w) {
      g_batcher_error = "image " + std::to_string(i) + ": needs data, 1 <= h, w <= 32768 and row_stride >= 3*w";
      return FS_ERR_INVALID;
    }
  }
  Request r{imgs, B, probs, mean_probs, vote, top1, logits};
  {
    std::unique_lock<std::mutex> lk(b->mu);
    if (b->stop) {
      g_batcher_error = "batcher is shutting down";
      return FS_ERR_INVALID;
    }
    try {
      b->queue.push_back(&r);
    } catch (...) {
      g_batcher_error = "batcher: host allocation failed";
      return FS_ERR_OOM;
    }
    b->queued_images += B;
    ++b->callers;
    b->cv_work.notify_all();  // the gathering worker re-checks its fill
    b->cv_done.wait(lk, [&] { return r.done; });
    if (--b->callers == 0) b->cv_idle.notify_all();
  }
  if (r.st != FS_OK) g_batcher_error = r.err;
  return r.st;
}

fs_status fs_batcher_stats(fs_batcher* b, int64_t* passes, int64_t* requests, int64_t* images) {
  if (!b) {
    g_batcher_error = "batcher is NULL";
    return FS_ERR_INVALID;
  }
  std::lock_guard<std::mutex> lk(b->mu);
  if (passes) *passes = b->passes;
  if (requests) *requests = b->requests;
  if (images) *images = b->images;
  return FS_OK;
}

const char* fs_batcher_last_error(void) { return g_batcher_error.c_str(); }

void fs_batcher_destroy(fs_batcher* b) {
  if (!b) return;
  b->shutdown();  // the queue is drained first
  delete b;
}

}  // extern "C"
