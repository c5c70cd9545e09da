// Shared pieces of the MFMA GEMM kernels: accumulator types and epilogues.
#pragma once

#include "dqt_launch.h"

namespace dqt {

enum class Mfma { I8, F8, BF16, F32 };

template <Mfma K> struct AccT { using type = f32x16; };
template <> struct AccT<Mfma::I8> { using type = i32x16; };

// ------------------------------------------------------------- epilogues
// (i, j) -> value written.  acc is int32 (I8) or fp32.
struct EpiFwd {          // y = fl(fl(acc) * fl(xdq[i] * alpha))
  void* y; int64_t ld; bool bf16; const float* xdq; float alpha;
  __device__ void put(int64_t i, int64_t j, float acc) const {
    const float f = xdq[i] * alpha;
    const float v = acc * f;
    if (bf16) reinterpret_cast<uint16_t*>(y)[i * ld + j] = (uint16_t)f32_to_bf16_bits(v);
    else reinterpret_cast<float*>(y)[i * ld + j] = v;
  }
};
struct EpiScale {        // y = fl(alpha * acc)
  void* y; int64_t ld; bool bf16; float alpha;
  __device__ void put(int64_t i, int64_t j, float acc) const {
    const float v = alpha * acc;
    if (bf16) reinterpret_cast<uint16_t*>(y)[i * ld + j] = (uint16_t)f32_to_bf16_bits(v);
    else reinterpret_cast<float*>(y)[i * ld + j] = v;
  }
};
struct EpiPartial {      // fp32 partial sums, one slab per split
  float* y; int64_t ld; int64_t slab;
  __device__ void put(int64_t i, int64_t j, float acc) const {
    y[(int64_t)blockIdx.z * slab + i * ld + j] = acc;
  }
};


}  // namespace dqt
