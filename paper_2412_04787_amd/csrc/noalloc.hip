// The batched forward without a caller workspace, for callers that cannot
// allocate device memory (code under graph capture, serving loops, harnesses
// that forbid allocation).  Its scratch -- the persistent GEMM's tile
// counters and, when they fit, the operand bytes the codes are expanded
// into -- lives in one static device array per GPU, kept for the life of the
// process.
#include <mutex>

#include "../../include/dqt.h"
#include "dqt_launch.h"

namespace {

// File-scope device array: every GPU the library runs on holds its own copy.
// Host code never names it except through HIP_SYMBOL to find its address.
static __device__ __align__(256) uint8_t scratch[DQT_NOALLOC_SCRATCH_BYTES];

constexpr int kMaxDevices = 64;
std::mutex g_mu;
uint8_t* g_scratch[kMaxDevices];   // device address of `scratch` on device d

// The current device's copy of the array: looked up once per device (with
// that device current) and remembered.
dqt_status scratch_of_current_device(uint8_t** out) {
  int dev = -1;
  if (hipGetDevice(&dev) != hipSuccess) return DQT_ERR_HIP;
  if (dev < 0 || dev >= kMaxDevices) return DQT_ERR_UNSUPPORTED;
  std::lock_guard<std::mutex> lock(g_mu);
  if (g_scratch[dev] == nullptr) {
    void* p = nullptr;
    if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || p == nullptr) return DQT_ERR_HIP;
    g_scratch[dev] = static_cast<uint8_t*>(p);
  }
  *out = g_scratch[dev];
  return DQT_OK;
}

}  // namespace

extern "C" dqt_status dqt_linear_fwd_batch_noalloc(int32_t n, const dqt_linear_io* io, int64_t M,
                                                   int32_t act_q, int32_t y_t, void* stream) {
  // every check is dqt_linear_fwd_batch's, made before anything is
  // enqueued: a batch whose smallest workspace exceeds the scratch is refused
  // (DQT_ERR_WORKSPACE); ternary codes whose expansion does not fit run from
  // the packed codes
  uint8_t* ws = nullptr;
  const dqt_status st = scratch_of_current_device(&ws);
  if (st != DQT_OK) return st;
  return dqt_linear_fwd_batch(n, io, M, act_q, y_t, ws, (size_t)DQT_NOALLOC_SCRATCH_BYTES, stream);
}
