// Launch timer: events around each GEMM kernel launch, so that a caller can
// read the kernels' own durations (for measurement; not on any compute path).
#include <hip/hip_runtime.h>

#include <mutex>
#include <vector>

#include "../../include/dqt.h"
#include "dqt_launch.h"

namespace dqt {
namespace {

std::mutex g_mu;
std::vector<hipEvent_t> g_ev;   // begin and end of each slot
int g_cap = 0, g_used = 0;
bool g_on = false;

void destroy_events() {
  for (hipEvent_t e : g_ev) (void)hipEventDestroy(e);
  g_ev.clear();
  g_cap = g_used = 0;
  g_on = false;
}

}  // namespace

hipError_t launch_timer_begin(hipStream_t s, int* slot) {
  std::lock_guard<std::mutex> lock(g_mu);
  *slot = -1;
  if (!g_on || g_used >= g_cap) return hipSuccess;
  const int k = g_used++;
  *slot = k;
  return hipEventRecord(g_ev[2 * k], s);
}

hipError_t launch_timer_end(int slot, hipStream_t s) {
  if (slot < 0) return hipSuccess;
  std::lock_guard<std::mutex> lock(g_mu);
  if (!g_on || slot >= g_used) return hipSuccess;
  return hipEventRecord(g_ev[2 * slot + 1], s);
}

}  // namespace dqt

extern "C" {

dqt_status dqt_launch_timer_start(int32_t max_launches) {
  if (max_launches < 1 || max_launches > DQT_LAUNCH_TIMER_MAX) return DQT_ERR_SHAPE;
  std::lock_guard<std::mutex> lock(dqt::g_mu);
  if (dqt::g_on) return DQT_ERR_UNSUPPORTED;
  dqt::g_ev.assign(2 * (size_t)max_launches, nullptr);
  for (hipEvent_t& e : dqt::g_ev)
    if (hipEventCreate(&e) != hipSuccess) {
      e = nullptr;
      for (hipEvent_t& f : dqt::g_ev)
        if (f != nullptr) (void)hipEventDestroy(f);
      dqt::g_ev.clear();
      return DQT_ERR_HIP;
    }
  dqt::g_cap = max_launches;
  dqt::g_used = 0;
  dqt::g_on = true;
  return DQT_OK;
}

dqt_status dqt_launch_timer_stop(float* ms, int32_t max, int32_t* count) {
  std::lock_guard<std::mutex> lock(dqt::g_mu);
  if (!dqt::g_on) return DQT_ERR_UNSUPPORTED;
  // arguments checked before anything changes: the timer keeps running
  if (max < 0) return DQT_ERR_SHAPE;
  if (count == nullptr || (ms == nullptr && max > 0)) return DQT_ERR_NULL;
  dqt_status st = DQT_OK;
  for (int k = 0; k < dqt::g_used; ++k) {
    float t = 0.f;
    if (hipEventSynchronize(dqt::g_ev[2 * k + 1]) != hipSuccess ||
        hipEventElapsedTime(&t, dqt::g_ev[2 * k], dqt::g_ev[2 * k + 1]) != hipSuccess) {
      st = DQT_ERR_HIP;
      break;
    }
    if (k < max) ms[k] = t;
  }
  *count = dqt::g_used;
  dqt::destroy_events();
  return st;
}

}  // extern "C"
