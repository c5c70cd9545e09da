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
  static constexpr bool kTrans = false;
  static constexpr bool kSR = false;
  static constexpr bool kTern = false;
  static constexpr int kCF = 0;
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
  static constexpr bool kTrans = false;
  static constexpr bool kSR = false;
  static constexpr bool kTern = false;
  static constexpr int kCF = 0;
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
  static constexpr bool kTrans = false;
  static constexpr bool kSR = false;
  static constexpr bool kTern = false;
  static constexpr int kCF = 0;
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

// dW consumed where it is formed: each group of 8 consecutive dW entries of
// a row goes through the direct SR update of its 8 codes (Sec. 3.2 Eq. 5)
// and dW itself is never stored.  CF: code format, 0 int8 codes (8 bytes
// per 8 weights), 1 2-bit ternary codes (2 bytes), 2 int4 nibbles (4 bytes).
// TR: the product is formed transposed, dW^T = X~^T dY (rows d_in, columns
// d_out), with the MFMA operands swapped so that each lane still holds four
// consecutive weights of a row of dW; the transposing LDS reads of dY's
// tiles then fall on the wave's two column blocks instead of its four row
// blocks.
template <int CF, bool TR = false>
struct EpiSR {
  uint8_t* wq;          // codes [d_out][d_in], updated in place
  int64_t ldc;          // bytes per code row (d_in / 4, d_in / 2 or d_in)
  int64_t d_in;         // weights per row: the flat index of (n, k) is n d_in + k
  float c, L;           // fl32(lr / alpha); |delta| clamp qmax - qmin + 1
  int qmin, qmax;
  uint32_t k0, k1, step, tid;   // Philox key (seed), step, tensor id
  unsigned long long* counters; // nullable: changed, non-finite (accumulated)
  static constexpr bool kRowScale = false;
  static constexpr bool kTrans = TR;
  static constexpr bool kSR = true;
  static constexpr bool kTern = CF == 1;
  static constexpr int kCF = CF;
  __device__ float scale(int64_t) const { return 1.0f; }
  __device__ float scale_raw(int64_t) const { return 1.0f; }
  __device__ float scale_fin(float) const { return 1.0f; }
  __device__ bool out_bf16() const { return false; }
  __device__ uint8_t* row(int64_t i, int) const { return wq + i * ldc; }
  __device__ int64_t row_bytes() const { return ldc; }
};

}  // namespace dqt
