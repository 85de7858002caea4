// Library-wide entry points: error text, version and kernel timing.
#include <atomic>
#include <cstring>
#include <map>
#include <mutex>
#include <string>

#include "cel_internal.h"

namespace cel {
const char *last_error_text();

namespace {
std::atomic<int> g_timing{0};
std::mutex g_mu;
struct Tot {
  long long launches = 0;
  double ms = 0.0;
};
std::map<std::string, Tot> &totals() {
  static std::map<std::string, Tot> t;
  return t;
}
struct Pending {
  const char *name;
  hipEvent_t a, b;
};
// Event pairs of timed launches, resolved lazily (when statistics are read or
// when many are pending) so that a timed call pays only for recording them.
std::vector<Pending> g_pending;
std::vector<hipEvent_t> g_pool;
constexpr size_t kMaxPending = 4096;

hipEvent_t take_event() {  // g_mu held
  if (!g_pool.empty()) {
    hipEvent_t e = g_pool.back();
    g_pool.pop_back();
    return e;
  }
  hipEvent_t e = nullptr;
  if (hipEventCreate(&e) != hipSuccess) return nullptr;
  return e;
}

void collect_locked() {
  for (const Pending &p : g_pending) {
    float ms = 0.f;
    if (hipEventSynchronize(p.b) == hipSuccess && hipEventElapsedTime(&ms, p.a, p.b) == hipSuccess) {
      Tot &t = totals()[p.name];
      t.launches++;
      t.ms += ms;
    }
    g_pool.push_back(p.a);
    g_pool.push_back(p.b);
  }
  g_pending.clear();
}
}  // namespace

KTimer::KTimer(hipStream_t s, const char *name) : s_(s), name_(name) {
  if (!g_timing.load(std::memory_order_relaxed)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  a_ = take_event();
  b_ = take_event();
  if (a_ && b_) (void)hipEventRecord(a_, s_);
}

KTimer::~KTimer() {
  if (!a_ || !b_) return;
  (void)hipEventRecord(b_, s_);
  std::lock_guard<std::mutex> lk(g_mu);
  g_pending.push_back(Pending{name_, a_, b_});
  if (g_pending.size() >= kMaxPending) collect_locked();
}

}  // namespace cel


extern "C" const char *cel_last_error(void) { return cel::last_error_text(); }

extern "C" int cel_version(void) { return 100; /* 0.1.0 */ }

extern "C" int cel_timing(int enable) { return cel::g_timing.exchange(enable ? 1 : 0); }

extern "C" int cel_kernel_stats(char *buf, int buflen, int reset) {
  std::lock_guard<std::mutex> lk(cel::g_mu);
  cel::collect_locked();
  std::string out;
  int count = 0;
  for (auto &kv : cel::totals()) {
    char line[256];
    snprintf(line, sizeof line, "%s %lld %.6f\n", kv.first.c_str(), kv.second.launches, kv.second.ms);
    out += line;
    count++;
  }
  if (buf && buflen > 0) {
    size_t k = out.size() < (size_t)(buflen - 1) ? out.size() : (size_t)(buflen - 1);
    memcpy(buf, out.data(), k);
    buf[k] = 0;
  }
  if (reset) cel::totals().clear();
  return count;
}
