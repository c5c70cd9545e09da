// Internal launcher interface between the C ABI (abi.hip) and the kernels.
// Callers have validated every argument; launchers only enqueue work.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include <tuple>
#include <type_traits>
#include <utility>

#include "dqt_device.h"

namespace dqt {

// Kernel launches return the status of that launch itself (hipLaunchKernel),
// never an error some earlier runtime call left behind for hipGetLastError.
template <class K, class T, size_t... I>
hipError_t launch_argv(K k, dim3 grid, dim3 block, hipStream_t s, T& vals, std::index_sequence<I...>) {
  void* argv[] = {static_cast<void*>(&std::get<I>(vals))...};
  return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, argv, 0, s);
}
template <class... P, class... A>
hipError_t launch_kernel(void (*k)(P...), dim3 grid, dim3 block, hipStream_t s, A&&... a) {
  static_assert(sizeof...(P) == sizeof...(A), "argument count");
  std::tuple<std::decay_t<P>...> vals(std::forward<A>(a)...);
  return launch_argv(k, grid, block, s, vals, std::index_sequence_for<P...>{});
}
template <class... P, class... A>
hipError_t launch_kernel_lds(void (*k)(P...), dim3 grid, dim3 block, size_t lds, hipStream_t s, A&&... a) {
  static_assert(sizeof...(P) == sizeof...(A), "argument count");
  std::tuple<std::decay_t<P>...> vals(std::forward<A>(a)...);
  void* argv[sizeof...(P)];
  std::apply([&](auto&... v) {
    int i = 0;
    ((argv[i++] = static_cast<void*>(&v)), ...);
  }, vals);
  return hipLaunchKernel(reinterpret_cast<const void*>(k), grid, block, argv, lds, s);
}
// The first error of a sequence of launches.
struct LaunchStatus {
  hipError_t e = hipSuccess;
  LaunchStatus& operator<<(hipError_t x) {
    if (e == hipSuccess) e = x;
    return *this;
  }
};

// Launch timer (measurement only): while one runs, every GEMM kernel launch
// is bracketed by a pair of events recorded on its stream, one pair per
// launch up to the timer's capacity; launches beyond it are not timed.
// begin gives the pair's slot, or -1 when no timer runs or it is full.
hipError_t launch_timer_begin(hipStream_t s, int* slot);
hipError_t launch_timer_end(int slot, hipStream_t s);
template <class F>
hipError_t timed_launch(hipStream_t s, F&& launch) {
  int slot = -1;
  hipError_t e = launch_timer_begin(s, &slot);
  if (e != hipSuccess) return e;
  e = launch();
  const hipError_t e2 = launch_timer_end(slot, s);
  return e != hipSuccess ? e : e2;
}

// Compute units of the current device, queried on every call (nothing is
// cached across calls or devices).
inline int current_device_cus() {
  int dev = 0, n = 0;
  if (hipGetDevice(&dev) != hipSuccess) return 256;
  if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || n <= 0) return 256;
  return n;
}

struct DxArgs {
  const void* dY;       // [M, d_out]
  const void* Wq;
  void* dX;             // [M, d_in]
  int64_t M, d_in, d_out;
  float alpha;
  bool w_ternary, dy_bf16, dx_bf16;
};

struct DwArgs {
  const void* dY;       // [M, d_out]
  const void* Xq;       // [M, d_in]
  const float* xdq;     // [M]
  float* dW;            // [d_out, d_in]
  float* ws;            // [splits, d_out, d_in] when splits > 1
  int64_t M, d_in, d_out, splits;
  bool act_e4m3, xt_bf16;
};

hipError_t launch_act_quant(const void* X, bool x_bf16, int64_t M, int K, bool e4m3, void* Xq,
                            float* xdq, hipStream_t stream);
// Backward of the RMSNorm feeding a group of linears: dX of the norm's input
// from the sum of up to kMaxNormDy upstream gradients (bf16), and per-block
// partial sums of the gamma gradient, gpart [blocks, K].
constexpr int kMaxNormDy = 4;
hipError_t launch_rmsnorm_backward(int n_dy, const void* const* dY, const void* X, const float* gamma,
                                   const float* rinv, int64_t M, int K, void* dX, float* gpart,
                                   int blocks, hipStream_t stream);
// RMSNorm (fp32, fixed summation order) then the per-token quantisation;
// rinv (nullable) receives each row's 1 / rms.
hipError_t launch_rmsnorm_act_quant(const void* X, bool x_bf16, const float* gamma, float eps, int64_t M,
                                    int K, bool e4m3, void* Xq, float* xdq, float* rinv,
                                    hipStream_t stream);
// up to kMaxBatch inputs with the same M and dtypes in one launch
struct ActIO {
  const void* X;        // [M, K]
  void* Xq;             // [M, K] codes
  float* xdq;           // [M]
  int K;
};
hipError_t launch_act_quant_batch(int n, const ActIO* io, bool x_bf16, int64_t M, bool e4m3,
                                  hipStream_t stream);
// int8 / e4m3 / bf16 matrix-core kernels, batched: up to kMaxBatch linears
// (same dtypes, same token count M) per launch.
constexpr int kMaxBatch = 8;
// The first kSchedBytes of every GEMM workspace are the persistent GEMM's:
// bytes 0-127 hold its tile counters (two 64-byte slots, cleared by a small
// kernel before every launch), bytes 128-143 absorb epilogue stores of
// chunks outside the output.
constexpr size_t kSchedBytes = 256;
struct LinearIO {
  int64_t d_in, d_out;
  float alpha;
  const void* Wq;       // codes
  const void* Xq;       // [M, d_in] quantised input
  const float* xdq;     // [M]
  void* Y;              // [M, d_out]
  const void* dY;       // [M, d_out]
  void* dX;             // [M, d_in]
  float* dW;            // [d_out, d_in]
};
struct BatchCfg {
  int n;
  int64_t M;
  bool w_ternary, act_e4m3, out_bf16;
  bool w_int4;          // 4-bit codes (two's-complement nibbles)
  bool w_int3;          // 3-bit codes (8 weights in 3 bytes)
};
struct BwdPlan {
  int64_t splits;        // dW batch splits when dW runs in a launch of its own
  int64_t splits_dual;   // ... and when it shares one launch with dX
  bool sr_fused;         // unsplit dW: the SR update in its epilogue (else a pass over
  bool sr_fused_dual;    //   dW staged in the workspace); alone / with dX
  int wi, wj;       // dW block tile (64 wi) x (64 wj)
  size_t q_off[kMaxBatch], xt_off[kMaxBatch], part_off[kMaxBatch];
  size_t total;
};
size_t fwd_batch_workspace(int n, const LinearIO* io, int cf, size_t* offs);
size_t fwd_batch_workspace_min(int n, const LinearIO* io, int cf);
// int4 codes [n] -> int8 codes (one byte per weight), n a multiple of 16
hipError_t launch_unpack_int4(const void* src, int8_t* dst, int64_t n, hipStream_t stream);
// int3 codes [n] -> int8 codes, n a multiple of 16
hipError_t launch_unpack_int3(const void* src, int8_t* dst, int64_t n, hipStream_t stream);
hipError_t launch_fwd_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, size_t ws_bytes,
                           hipStream_t stream);
BwdPlan plan_bwd_batch(int n, const LinearIO* io, int64_t M);
hipError_t launch_dx_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                           hipStream_t stream);
hipError_t launch_dw_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                           hipStream_t stream);
// dX and dW of every linear of the batch in one launch (bf16 operands).
hipError_t launch_dxdw_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                             hipStream_t stream);
struct SRTensor;
// dW of every linear of the batch consumed by the SR update of its codes
// (dW is not stored), with dX of every linear in the same launch when
// with_dx (bf16 operands).
hipError_t launch_bwd_sr_batch(const BatchCfg& c, const LinearIO* io, const SRTensor* t, uint64_t seed,
                               uint32_t step, unsigned long long* counters, bool with_dx, uint8_t* ws,
                               const BwdPlan& P, hipStream_t stream);
// fp32-environment kernels
hipError_t launch_dx_f32(const DxArgs& a, hipStream_t stream);
hipError_t launch_dw_f32(const DwArgs& a, hipStream_t stream);
int64_t dw_splits_f32(int64_t d_out, int64_t d_in, int64_t M);
hipError_t launch_split_reduce(const float* ws, int splits, int64_t n, float* out, hipStream_t stream);
// Direct SR update of up to kMaxBatch weight tensors (same code format) in
// one launch.
struct SRTensor {
  uint8_t* wq;          // codes, updated in place
  const float* grad;    // dW
  int64_t nweights;     // multiple of 16
  float c;              // fl32(lr / alpha)
  int qmin, qmax;
  uint32_t tensor_id;
  float alpha;
};
// cf: code format, 0 int8, 1 ternary 2-bit, 2 int4 nibbles, 3 int3 fields
hipError_t launch_sr_update(int cf, int n, const SRTensor* t, uint64_t seed, uint32_t step,
                            unsigned long long* counters, hipStream_t stream);
// One tensor of a device-resident update table (dqt_sr_table_build's
// entries, 64 bytes each).
struct SRTableEntry {
  uint64_t wq;          // codes (device address)
  uint64_t grad;        // dW (device address)
  int64_t nchunks;      // weights / 8
  int64_t tile0;        // first tile (256 chunks) of this tensor in the launch
  float alpha;
  int32_t qmin, qmax;
  uint32_t tensor_id;
  uint32_t reserved[4];
};
static_assert(sizeof(SRTableEntry) == 64, "table entry layout");
// the entry of tensor t whose first tile is tile0, and a tensor's tile count
void sr_table_entry(const SRTensor& t, int64_t tile0, SRTableEntry* e);
int64_t sr_tiles(int64_t nweights);
// Any number of tensors of one code format in one launch; per_tensor
// (nullable) receives each tensor's changed / non-finite counts.
hipError_t launch_sr_update_table(int cf, int n, int64_t tiles, const SRTableEntry* table, float lr,
                                  uint64_t seed, uint32_t step, unsigned long long* counters,
                                  unsigned long long* per_tensor, hipStream_t stream);
// Analysis variants of the update (mode 0 plain SR, 1 nearest, 2 force to
// remain, 3 force to update the bottom `frac` of |delta|).
size_t update_variant_workspace(int n);
hipError_t launch_update_variant(int cf, int n, const SRTensor* t, int mode, float frac,
                                 uint64_t seed, uint32_t step, unsigned long long* counters,
                                 void* ws, hipStream_t stream);
// The literal absmax re-quantisation control (Sec. 5.1); ws: n uint32.
size_t absmax_requant_workspace(int n);
hipError_t launch_absmax_requant(int cf, int n, const SRTensor* t, float lr, float* alpha_out,
                                 unsigned long long* counters, void* ws, hipStream_t stream);
// AdamW with SR (up to kMaxBatch tensors of one code format per launch).
struct AdamTensor {
  uint8_t* wq;          // codes, updated in place
  const float* grad;    // dW
  float* m;             // first moment, updated in place
  float* v;             // second moment, updated in place
  int64_t nweights;     // multiple of 8
  float alpha;
  int qmin, qmax;
  uint32_t tensor_id;
};
struct AdamHyper {
  float lr, beta1, beta2, eps, weight_decay;
};
hipError_t launch_adamw_sr(int cf, int n, const AdamTensor* t, const AdamHyper& hp,
                           uint64_t seed, uint32_t step, unsigned long long* counters,
                           hipStream_t stream);
hipError_t launch_debug_rng(uint64_t seed, uint32_t step, uint32_t tensor_id, uint64_t i0,
                            int64_t n, uint32_t* out, hipStream_t stream);

}  // namespace dqt
