// Shared pieces of the MFMA GEMM kernels: accumulator types and epilogues.
#pragma once

#include "dqt_launch.h"

namespace dqt {

enum class Mfma { I8, F8, BF16, F32 };

template <Mfma K> struct AccT { using type = f32x16; };
template <> struct AccT<Mfma::I8> { using type = i32x16; };

// ------------------------------------------------------------- epilogues
// An epilogue maps the accumulator of output (i, j) to the value stored:
//   scale(i)  per-row factor (1 when unused), applied as fl(acc * scale)
//   row(i)    address of output row i; out_bf16 selects the stored dtype.
// The fp32 result is rounded once to bf16 (RNE) when out_bf16 is set.
struct EpiFwd {          // y = fl(fl(acc) * fl(xdq[i] * alpha))
  void* y; int64_t ld; bool bf16; const float* xdq; float alpha;
  static constexpr bool kRowScale = true;
  __device__ float scale(int64_t i) const { return xdq[i] * alpha; }
  // the same factor in two parts: the per-row load, then the multiply
  __device__ float scale_raw(int64_t i) const { return xdq[i]; }
  __device__ float scale_fin(float raw) const { return raw * alpha; }
  __device__ bool out_bf16() const { return bf16; }
  __device__ uint8_t* row(int64_t i, int) const {
    return static_cast<uint8_t*>(y) + i * ld * (bf16 ? 2 : 4);
  }
  __device__ int64_t row_bytes() const { return ld * (bf16 ? 2 : 4); }
  // scalar path used by the fp32-environment kernels
  __device__ void put(int64_t i, int64_t j, float acc) const {
    const float v = acc * scale(i);
    if (bf16) reinterpret_cast<uint16_t*>(y)[i * ld + j] = (uint16_t)f32_to_bf16_bits(v);
    else reinterpret_cast<float*>(y)[i * ld + j] = v;
  }
};
struct EpiScale {        // y = fl(alpha * acc)
  void* y; int64_t ld; bool bf16; float alpha;
  static constexpr bool kRowScale = false;
  __device__ float scale(int64_t) const { return alpha; }
  __device__ float scale_raw(int64_t) const { return 1.0f; }
  __device__ float scale_fin(float) const { return alpha; }
  __device__ bool out_bf16() const { return bf16; }
  __device__ uint8_t* row(int64_t i, int) const {
    return static_cast<uint8_t*>(y) + i * ld * (bf16 ? 2 : 4);
  }
  __device__ int64_t row_bytes() const { return ld * (bf16 ? 2 : 4); }
  __device__ void put(int64_t i, int64_t j, float acc) const {
    const float v = alpha * acc;
    if (bf16) reinterpret_cast<uint16_t*>(y)[i * ld + j] = (uint16_t)f32_to_bf16_bits(v);
    else reinterpret_cast<float*>(y)[i * ld + j] = v;
  }
};
struct EpiPartial {      // fp32 partial sums, one slab per split
  float* y; int64_t ld; int64_t slab;
  static constexpr bool kRowScale = false;
  __device__ float scale(int64_t) const { return 1.0f; }
  __device__ float scale_raw(int64_t) const { return 1.0f; }
  __device__ float scale_fin(float) const { return 1.0f; }
  __device__ bool out_bf16() const { return false; }
  __device__ uint8_t* row(int64_t i, int split) const {
    return reinterpret_cast<uint8_t*>(y + (int64_t)split * slab + i * ld);
  }
  __device__ int64_t row_bytes() const { return ld * 4; }
  __device__ void put(int64_t i, int64_t j, float acc) const {
    y[(int64_t)blockIdx.z * slab + i * ld + j] = acc;
  }
};

}  // namespace dqt
