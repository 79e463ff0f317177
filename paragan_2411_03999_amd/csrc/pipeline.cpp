// Congestion-aware host data pipeline (Implementation, "Congestion-Aware
// Data Pipelining"): host threads fetch batches into caller-provided slots
// ahead of the consumer, and a controller driven by a sliding window of
// fetch latencies adds a thread and a slot of prefetch depth while the
// window's mean is above a threshold and gives one of each back while it is
// at or below it.  Host code only: no HIP call, usable without a GPU.
//
// Also the seeded synthetic batch source used in place of the image
// dataset: every value is a function of (seed, batch, index) through the
// SplitMix64 finaliser, so a batch is the same whichever thread makes it.
#include <algorithm>
#include <cstdint>
#include <chrono>
#include <condition_variable>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "../../include/paragan.h"

namespace {

using Clock = std::chrono::steady_clock;

double ms_since(Clock::time_point t0) {
  return std::chrono::duration<double, std::milli>(Clock::now() - t0).count();
}

// ------------------------------------------------------------ controller
// The sliding window and the grow/release rule, kept apart from the
// threading so that it is a plain state machine.
struct Controller {
  paragan_pipeline_cfg cfg;
  std::vector<double> win;     // ring of the last cfg.window latencies
  int64_t n = 0;               // samples seen
  int64_t since_change = 0;    // samples since the last adjustment
  double sum = 0.0;
  int threads, depth;
  int64_t grows = 0, shrinks = 0;

  explicit Controller(const paragan_pipeline_cfg& c)
      : cfg(c), win((size_t)c.window, 0.0), threads(c.min_threads), depth(c.min_depth) {}

  double mean() const {
    const int64_t k = std::min<int64_t>(n, cfg.window);
    return k ? sum / (double)k : 0.0;
  }
  // Adds one latency sample; returns true if threads or depth changed.
  bool add(double ms) {
    const size_t i = (size_t)(n % cfg.window);
    if (n >= cfg.window) sum -= win[i];
    win[i] = ms;
    sum += ms;
    ++n;
    ++since_change;
    // decide only on a full window of samples taken since the last change
    if (n < cfg.window || since_change < cfg.window) return false;
    const double m = mean();
    if (m > cfg.threshold_ms) {
      if (threads >= cfg.max_threads && depth >= cfg.max_depth) return false;
      threads = std::min(threads + 1, (int)cfg.max_threads);
      depth = std::min(depth + 1, (int)cfg.max_depth);
      ++grows;
    } else {
      if (threads <= cfg.min_threads && depth <= cfg.min_depth) return false;
      threads = std::max(threads - 1, (int)cfg.min_threads);
      depth = std::max(depth - 1, (int)cfg.min_depth);
      ++shrinks;
    }
    since_change = 0;
    return true;
  }
};

}  // namespace

struct paragan_pipeline {
  paragan_fetch_fn fetch = nullptr;
  void* user = nullptr;
  std::vector<void*> slots;
  size_t slot_bytes = 0;

  std::mutex mu;
  std::condition_variable cv_work;    // workers: a batch may be claimed, or a thread should retire
  std::condition_variable cv_ready;   // consumer: a batch became ready, or an error
  Controller ctl;
  enum SlotState { kFree, kFetching, kReady, kHeld };
  std::vector<int> free_slots;
  std::vector<SlotState> state;       // per slot
  std::vector<int64_t> ready_seq;     // per slot: the seq it holds once ready, -1 otherwise
  int64_t next_claim = 0;             // next seq a worker will fetch
  int64_t next_deliver = 0;           // next seq the consumer will receive
  int64_t outstanding = 0;            // slots fetching, ready or held by the consumer
  int64_t fetched = 0, delivered = 0;
  double wait_ms = 0.0;
  int live_threads = 0;               // running workers
  bool stop = false;
  std::string err;                    // the failure of the lowest failed batch (sticky)
  int64_t err_seq = INT64_MAX;        // that batch; the batches before it are still delivered
  std::string last_err;               // last failed call's message
  std::vector<std::thread> workers;

  explicit paragan_pipeline(const paragan_pipeline_cfg& c) : ctl(c) {}

  void spawn_locked() {
    ++live_threads;
    workers.emplace_back([this] { run(); });
  }

  void run() {
    std::unique_lock<std::mutex> lk(mu);
    for (;;) {
      cv_work.wait(lk, [this] {
        return stop || live_threads > ctl.threads ||
               (err.empty() && outstanding < ctl.depth && !free_slots.empty());
      });
      if (stop || live_threads > ctl.threads) break;
      const int64_t seq = next_claim++;
      const int slot = free_slots.back();
      free_slots.pop_back();
      state[(size_t)slot] = kFetching;
      ++outstanding;
      lk.unlock();
      const auto t0 = Clock::now();
      const int rc = fetch(user, seq, slots[(size_t)slot], slot_bytes);
      const double ms = ms_since(t0);
      lk.lock();
      if (rc != 0) {
        // every batch before seq was claimed before it, so those still
        // arrive and are delivered; nothing after it is claimed any more
        if (seq < err_seq) {
          err_seq = seq;
          err = "fetch callback returned " + std::to_string(rc) + " for batch " + std::to_string(seq);
        }
        state[(size_t)slot] = kFree;
        free_slots.push_back(slot);
        --outstanding;
        cv_ready.notify_all();
        continue;
      }
      ++fetched;
      ready_seq[(size_t)slot] = seq;
      state[(size_t)slot] = kReady;
      const int old_threads = ctl.threads;
      // no thread is started once destruction has begun
      if (!stop && ctl.add(ms)) {
        while (live_threads < ctl.threads) spawn_locked();
        if (ctl.threads < old_threads) cv_work.notify_all();   // one retires
      }
      cv_ready.notify_all();
      cv_work.notify_all();   // depth may have grown
    }
    --live_threads;
  }

  int find_ready_locked(int64_t seq) const {
    for (size_t s = 0; s < ready_seq.size(); ++s)
      if (ready_seq[s] == seq) return (int)s;
    return -1;
  }
};

namespace {

int bad(paragan_pipeline* p, const std::string& m) {
  if (p) p->last_err = m;
  return PARAGAN_EINVAL;
}

std::string g_create_err;

}  // namespace

extern "C" {

int paragan_pipeline_create(paragan_pipeline** out, const paragan_pipeline_cfg* cfg, paragan_fetch_fn fetch,
                            void* user, void* const* slots, int32_t n_slots, size_t slot_bytes) {
  auto fail = [](const char* m) {
    g_create_err = m;
    return PARAGAN_EINVAL;
  };
  if (!out || !cfg || !fetch || !slots) return fail("pipeline_create: null argument");
  if (n_slots < 1 || n_slots > 4096) return fail("pipeline_create: n_slots must be in [1, 4096]");
  for (int i = 0; i < n_slots; ++i)
    if (!slots[i]) return fail("pipeline_create: null slot");
  if (slot_bytes == 0) return fail("pipeline_create: slot_bytes must be > 0");
  if (cfg->min_threads < 1 || cfg->max_threads < cfg->min_threads || cfg->max_threads > 64)
    return fail("pipeline_create: need 1 <= min_threads <= max_threads <= 64");
  if (cfg->min_depth < 1 || cfg->max_depth < cfg->min_depth || cfg->max_depth > n_slots)
    return fail("pipeline_create: need 1 <= min_depth <= max_depth <= n_slots");
  if (cfg->window < 1 || cfg->window > 100000) return fail("pipeline_create: window must be in [1, 100000]");
  if (!(cfg->threshold_ms > 0.0)) return fail("pipeline_create: threshold_ms must be > 0");
  paragan_pipeline* p = nullptr;
  try {
    p = new paragan_pipeline(*cfg);
    p->fetch = fetch;
    p->user = user;
    p->slots.assign(slots, slots + n_slots);
    p->slot_bytes = slot_bytes;
    p->ready_seq.assign((size_t)n_slots, -1);
    p->state.assign((size_t)n_slots, paragan_pipeline::kFree);
    for (int i = n_slots - 1; i >= 0; --i) p->free_slots.push_back(i);
    std::lock_guard<std::mutex> lk(p->mu);
    for (int i = 0; i < cfg->min_threads; ++i) p->spawn_locked();
  } catch (const std::exception& e) {
    g_create_err = std::string("pipeline_create: ") + e.what();
    if (p) paragan_pipeline_destroy(p);
    return PARAGAN_EINVAL;
  }
  *out = p;
  return PARAGAN_OK;
}

int paragan_pipeline_next(paragan_pipeline* p, int64_t* seq, int32_t* slot, int32_t timeout_ms) {
  if (!p) return PARAGAN_EINVAL;
  if (!seq || !slot) return bad(p, "pipeline_next: null output");
  std::unique_lock<std::mutex> lk(p->mu);
  const auto t0 = Clock::now();
  int s = -1;
  auto ready = [&] {
    s = p->find_ready_locked(p->next_deliver);
    return s >= 0 || p->err_seq <= p->next_deliver;
  };
  bool ok;
  if (timeout_ms < 0) {
    p->cv_ready.wait(lk, ready);
    ok = true;
  } else {
    ok = p->cv_ready.wait_for(lk, std::chrono::milliseconds(timeout_ms), ready);
  }
  p->wait_ms += ms_since(t0);
  if (s < 0 && p->err_seq <= p->next_deliver) return bad(p, "pipeline_next: " + p->err);
  if (!ok || s < 0) {
    p->last_err = "pipeline_next: no batch within the timeout";
    return PARAGAN_ETIMEOUT;
  }
  p->ready_seq[(size_t)s] = -1;
  p->state[(size_t)s] = paragan_pipeline::kHeld;
  *seq = p->next_deliver++;
  *slot = s;
  ++p->delivered;
  return PARAGAN_OK;
}

int paragan_pipeline_release(paragan_pipeline* p, int32_t slot) {
  if (!p) return PARAGAN_EINVAL;
  std::lock_guard<std::mutex> lk(p->mu);
  if (slot < 0 || slot >= (int32_t)p->slots.size()) return bad(p, "pipeline_release: slot out of range");
  if (p->state[(size_t)slot] != paragan_pipeline::kHeld)
    return bad(p, "pipeline_release: slot " + std::to_string(slot) + " is not held by the consumer");
  p->state[(size_t)slot] = paragan_pipeline::kFree;
  p->free_slots.push_back(slot);
  --p->outstanding;
  p->cv_work.notify_all();
  return PARAGAN_OK;
}

int paragan_pipeline_get_stats(paragan_pipeline* p, paragan_pipeline_stats* out) {
  if (!p) return PARAGAN_EINVAL;
  if (!out) return bad(p, "pipeline_get_stats: null output");
  std::lock_guard<std::mutex> lk(p->mu);
  out->threads = p->ctl.threads;
  out->depth = p->ctl.depth;
  out->window_mean_ms = p->ctl.mean();
  out->fetched = p->fetched;
  out->delivered = p->delivered;
  out->grows = p->ctl.grows;
  out->shrinks = p->ctl.shrinks;
  out->consumer_wait_ms = p->wait_ms;
  return PARAGAN_OK;
}

const char* paragan_pipeline_error(const paragan_pipeline* p) {
  return p ? p->last_err.c_str() : g_create_err.c_str();
}

void paragan_pipeline_destroy(paragan_pipeline* p) {
  if (!p) return;
  {
    std::lock_guard<std::mutex> lk(p->mu);
    p->stop = true;
  }
  p->cv_work.notify_all();
  for (auto& t : p->workers)
    if (t.joinable()) t.join();
  delete p;
}

// ------------------------------------------------------------ synthetic source
static inline uint64_t splitmix64(uint64_t x) {
  x += 0x9E3779B97F4A7C15ull;
  x = (x ^ (x >> 30)) * 0xBF58476D1CE4E5B9ull;
  x = (x ^ (x >> 27)) * 0x94D049BB133111EBull;
  return x ^ (x >> 31);
}

size_t paragan_synth_batch_bytes(const paragan_synth_source* s) {
  if (!s || s->B < 1 || s->img < 1) return 0;
  return (size_t)s->B * s->img * s->img * 3 * sizeof(float) + (size_t)s->B * sizeof(int32_t);
}

int paragan_synth_fetch(void* user, int64_t seq, void* slot, size_t slot_bytes) {
  const auto* s = (const paragan_synth_source*)user;
  if (!s || !slot || seq < 0 || s->n_classes < 1) return 1;
  const size_t need = paragan_synth_batch_bytes(s);
  if (need == 0 || slot_bytes < need) return 2;
  const auto t0 = Clock::now();
  const int64_t n = (int64_t)s->B * s->img * s->img * 3;
  float* img = (float*)slot;
  int32_t* lab = (int32_t*)(img + n);
  // image value i of batch seq: the top 24 bits of
  // splitmix64(seed + 2^40 seq + i) as u in [0, 1), mapped to 2u - 1;
  // label b: splitmix64(seed + 2^40 seq + 2^39 + b) mod n_classes
  const uint64_t base = s->seed + ((uint64_t)seq << 40);
  for (int64_t i = 0; i < n; ++i)
    img[i] = (float)(splitmix64(base + (uint64_t)i) >> 40) * (2.0f / 16777216.0f) - 1.0f;
  for (int b = 0; b < s->B; ++b)
    lab[b] = (int32_t)(splitmix64(base + (1ull << 39) + (uint64_t)b) % (uint64_t)s->n_classes);
  if (s->latency_ms && s->n_latency > 0) {
    const double want = s->latency_ms[seq % s->n_latency];
    const double left = want - ms_since(t0);
    if (left > 0) std::this_thread::sleep_for(std::chrono::duration<double, std::milli>(left));
  }
  return 0;
}

}  // extern "C"
