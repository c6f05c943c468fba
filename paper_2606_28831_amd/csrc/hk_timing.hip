// Optional per-kernel timing: HIP events recorded on the launch stream around the launches
// of the kernels named in hk_timed_kernel.  Off by default; a measurement harness turns it
// on, runs its timed region, then reads the summed durations.  Host code only.
#include <mutex>
#include <vector>

#include "hk_internal.h"

namespace hk {
namespace {

struct Pair {
  hipEvent_t start, stop;
};

std::mutex g_mu;
uint32_t g_mask = 0;   // bit k: time kernel k
std::vector<Pair> g_pool;
std::vector<Pair> g_pending[HK_TK_COUNT];

bool take(Pair& p) {
  if (!g_pool.empty()) {
    p = g_pool.back();
    g_pool.pop_back();
    return true;
  }
  // timing-only events: no system-scope fence at record (a default event writes back and
  // invalidates the caches there, which costs the timed stream time of its own)
  if (hipEventCreateWithFlags(&p.start, hipEventDisableSystemFence) != hipSuccess) return false;
  if (hipEventCreateWithFlags(&p.stop, hipEventDisableSystemFence) != hipSuccess) {
    (void)hipEventDestroy(p.start);
    return false;
  }
  return true;
}

}  // namespace

TimedLaunch::TimedLaunch(int kernel, hipStream_t st) : kernel_(kernel), st_(st), active_(false) {
  std::lock_guard<std::mutex> lk(g_mu);
  if (kernel < 0 || kernel >= HK_TK_COUNT || !((g_mask >> kernel) & 1u)) return;
  Pair p;
  if (!take(p)) return;
  if (hipEventRecord(p.start, st) != hipSuccess) {
    g_pool.push_back(p);
    return;
  }
  g_pending[kernel].push_back(p);
  active_ = true;
}

TimedLaunch::~TimedLaunch() {
  if (!active_) return;
  std::lock_guard<std::mutex> lk(g_mu);
  (void)hipEventRecord(g_pending[kernel_].back().stop, st_);
}

}  // namespace hk

extern "C" {

hk_status hk_timing_enable(uint32_t kernel_mask) {
  std::lock_guard<std::mutex> lk(hk::g_mu);
  hk::g_mask = kernel_mask & ((1u << HK_TK_COUNT) - 1u);
  return HK_OK;
}

hk_status hk_timing_read(int32_t kernel, double* total_ms, int64_t* launches) {
  if (kernel < 0 || kernel >= HK_TK_COUNT || !total_ms || !launches) return HK_ERR_ARG;
  std::vector<hk::Pair> pend;
  {
    std::lock_guard<std::mutex> lk(hk::g_mu);
    pend.swap(hk::g_pending[kernel]);
  }
  double sum = 0.0;
  hk_status rc = HK_OK;
  for (const hk::Pair& p : pend) {
    float ms = 0.f;
    if (hipEventSynchronize(p.stop) != hipSuccess ||
        hipEventElapsedTime(&ms, p.start, p.stop) != hipSuccess)
      rc = HK_ERR_HIP;
    sum += ms;
  }
  {
    std::lock_guard<std::mutex> lk(hk::g_mu);
    hk::g_pool.insert(hk::g_pool.end(), pend.begin(), pend.end());
  }
  *total_ms = sum;
  *launches = (int64_t)pend.size();
  return rc;
}

}  // extern "C"
