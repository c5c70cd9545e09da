// Internal launcher interface between the C ABI (abi.hip) and the kernels.
// Callers have validated every argument; launchers only enqueue work.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "dqt_device.h"

namespace dqt {

struct FwdArgs {
  const void* Xq;       // [M, d_in] int8 or e4m3
  const float* xdq;     // [M]
  const void* Wq;       // packed ternary or int8 codes
  void* Y;              // [M, d_out]
  int64_t M, d_in, d_out;
  void* ws;             // unpacked weight rows (ternary weights only)
  float alpha;
  bool w_ternary, act_e4m3, y_bf16;
};

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
// int8 / e4m3 / bf16 matrix-core kernels
size_t fwd_workspace_bytes(bool ternary, int64_t d_out, int64_t d_in);
hipError_t launch_fwd_v2(const FwdArgs& a, hipStream_t stream);
hipError_t launch_dx_v2(const DxArgs& a, void* ws_q, hipStream_t stream);
hipError_t launch_dw_v2(const DwArgs& a, void* ws_xt, hipStream_t stream);
void plan_dw_v2(int64_t d_out, int64_t d_in, int64_t M, int* wj, int64_t* splits);
// fp32-environment kernels
hipError_t launch_dx_f32(const DxArgs& a, hipStream_t stream);
hipError_t launch_dw_f32(const DwArgs& a, hipStream_t stream);
int64_t dw_splits_f32(int64_t d_out, int64_t d_in, int64_t M);
hipError_t launch_split_reduce(const float* ws, int splits, int64_t n, float* out, hipStream_t stream);
hipError_t launch_sr_update(bool ternary, uint8_t* wq, const float* grad, int64_t nweights,
                            float c, int qmin, int qmax, uint64_t seed, uint32_t step,
                            uint32_t tensor_id, unsigned long long* counters, hipStream_t stream);
hipError_t launch_debug_rng(uint64_t seed, uint32_t step, uint32_t tensor_id, uint64_t i0,
                            int64_t n, uint32_t* out, hipStream_t stream);

}  // namespace dqt
