// Measurement helpers (not on any compute path): the launch timer, events
// around each GEMM kernel launch so that a caller can read the kernels' own
// durations; and a plain streaming read, the achievable HBM read rate that
// the streaming kernels are compared with.
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

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// Grid-stride read of n16 16-byte words, 8 non-temporal loads in flight per
// lane; each wave's xor of what it read goes to sink[4 * block + wave].
__global__ __launch_bounds__(256) void read_stream_kernel(const u32x4_t* __restrict__ p, int64_t n16,
                                                          uint32_t* __restrict__ sink) {
  const int64_t stride = (int64_t)gridDim.x * 256;
  int64_t i = (int64_t)blockIdx.x * 256 + threadIdx.x;
  uint32_t acc = 0;
  for (; i + 7 * stride < n16; i += 8 * stride) {
    u32x4_t v[8];
#pragma unroll
    for (int u = 0; u < 8; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
    for (int u = 0; u < 8; ++u) acc ^= v[u].x ^ v[u].y ^ v[u].z ^ v[u].w;
  }
  for (; i < n16; i += stride) {
    const u32x4_t v = __builtin_nontemporal_load(p + i);
    acc ^= v.x ^ v.y ^ v.z ^ v.w;
  }
#pragma unroll
  for (int o = 32; o > 0; o >>= 1) acc ^= (uint32_t)__shfl_xor((int)acc, o, 64);
  if ((threadIdx.x & 63) == 0) sink[4 * blockIdx.x + (threadIdx.x >> 6)] = acc;
}

}  // namespace dqt

extern "C" {

dqt_status dqt_read_stream(const void* src, size_t bytes, uint32_t* sink, void* stream) {
  if (bytes == 0) return DQT_OK;
  if (src == nullptr || sink == nullptr) return DQT_ERR_NULL;
  if (bytes % 16 != 0) return DQT_ERR_SHAPE;
  if (reinterpret_cast<uintptr_t>(src) % 16 != 0 || reinterpret_cast<uintptr_t>(sink) % 16 != 0)
    return DQT_ERR_ALIGN;
  constexpr int kBlocks = DQT_READ_STREAM_SINK_WORDS / 4;
  const hipError_t e = dqt::launch_kernel(dqt::read_stream_kernel, dim3(kBlocks), dim3(256),
                                          static_cast<hipStream_t>(stream),
                                          static_cast<const dqt::u32x4_t*>(src),
                                          static_cast<int64_t>(bytes / 16), sink);
  return e == hipSuccess ? DQT_OK : DQT_ERR_HIP;
}

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
