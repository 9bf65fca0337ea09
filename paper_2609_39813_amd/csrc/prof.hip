// Kernel timing instrumentation: when enabled, a pair of HIP events is recorded on the
// launch stream around each instrumented kernel launch; bs_profile_read() waits for the
// events and sums the elapsed time per kernel name. Off by default (no events recorded): a
// launch then reads one atomic flag and takes no lock.
#include <atomic>
#include <mutex>
#include <string>
#include <vector>

#include "bsp_kernels.h"

namespace bsp {

namespace {
struct Rec {
  std::string name;
  hipEvent_t a, b;
  double work, exec;
};
std::mutex g_mu;
std::atomic<bool> g_on{false};
std::vector<hipEvent_t> g_pool;
size_t g_next = 0;
std::vector<Rec> g_recs;
constexpr size_t kPool = 16384;

void release_all() {
  for (auto e : g_pool) hipEventDestroy(e);
  g_pool.clear();
  g_recs.clear();
  g_next = 0;
}
}  // namespace

ProfScope::ProfScope(const char* name, hipStream_t st, double work, double exec)
    : name_(name), st_(st), work_(work), exec_(exec), a_(nullptr), b_(nullptr) {
  if (!g_on.load(std::memory_order_acquire)) return;
  std::lock_guard<std::mutex> lk(g_mu);
  if (!g_on.load(std::memory_order_relaxed) || g_next + 2 > g_pool.size()) return;
  a_ = g_pool[g_next++];
  b_ = g_pool[g_next++];
  hipEventRecord(a_, st_);
}

ProfScope::~ProfScope() {
  if (!a_) return;
  hipEventRecord(b_, st_);
  std::lock_guard<std::mutex> lk(g_mu);
  g_recs.push_back({name_, a_, b_, work_, exec_});
}

}  // namespace bsp

extern "C" {

int bs_profile_enable(int on) {
  using namespace bsp;
  std::lock_guard<std::mutex> lk(g_mu);
  g_on.store(false, std::memory_order_release);
  release_all();
  if (on != 0) {
    g_pool.resize(kPool);
    for (auto& e : g_pool)
      if (hipEventCreate(&e) != hipSuccess) return BS_EHIP;
    g_on.store(true, std::memory_order_release);
  }
  return BS_OK;
}

int bs_profile_read(const char* kernel, double* total_ms, int* launches) {
  using namespace bsp;
  std::lock_guard<std::mutex> lk(g_mu);
  double tot = 0.0;
  int n = 0;
  for (auto& r : g_recs) {
    if (kernel && r.name != kernel) continue;
    if (hipEventSynchronize(r.b) != hipSuccess) return BS_EHIP;
    float ms = 0.0f;
    if (hipEventElapsedTime(&ms, r.a, r.b) != hipSuccess) return BS_EHIP;
    tot += ms;
    ++n;
  }
  if (total_ms) *total_ms = tot;
  if (launches) *launches = n;
  return BS_OK;
}

int bs_profile_work(const char* kernel, double* work, double* exec) {
  using namespace bsp;
  std::lock_guard<std::mutex> lk(g_mu);
  double tot = 0.0, ex = 0.0;
  for (auto& r : g_recs)
    if (!kernel || r.name == kernel) {
      tot += r.work;
      ex += r.exec;
    }
  if (work) *work = tot;
  if (exec) *exec = ex;
  return BS_OK;
}

}  // extern "C"
