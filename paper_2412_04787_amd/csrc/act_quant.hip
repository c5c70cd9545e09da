// Per-token 8-bit activation quantisation (Sec. 3.2: inputs and activations
// are quantised to 8 bits following BitNet): absmax per row, then int8 or
// OCP e4m3 codes plus one fp32 dequantisation scale per row.
//
// HBM-bound: reads the row (2 or 4 B/element) and writes 1 B/element.  One
// wave per row; the row is read twice (max, then quantise) and the second
// read is served by the L2/MALL because the wave's row was just streamed.
#include "dqt_launch.h"

namespace dqt {

template <typename TX>
struct RowChunk;  // 16-byte chunk of a row: 8 bf16 or 4 fp32 values

template <>
struct RowChunk<uint16_t> {  // bf16 bits
  static constexpr int kElems = 8;
  __device__ static void load(const uint16_t* p, float (&v)[8]) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = bf16_bits_to_f32(w[i] & 0xFFFFu);
      v[2 * i + 1] = bf16_bits_to_f32(w[i] >> 16);
    }
  }
};
template <>
struct RowChunk<float> {
  static constexpr int kElems = 4;
  __device__ static void load(const float* p, float (&v)[4]) {
    const f32x4 u = *reinterpret_cast<const f32x4*>(p);
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = u[i];
  }
};

template <typename TX, bool E4M3>
__global__ __launch_bounds__(256) void act_quant_kernel(const TX* __restrict__ X, int64_t M, int K,
                                                        uint8_t* __restrict__ Xq,
                                                        float* __restrict__ xdq) {
  using C = RowChunk<TX>;
  constexpr int E = C::kElems;
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = (int64_t)blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
  if (row >= M) return;
  const TX* xr = X + row * (int64_t)K;
  uint8_t* qr = Xq + row * (int64_t)K;
  const int nchunk = K / E;

  float amax = 0.0f;
  for (int c = lane; c < nchunk; c += kWave) {
    float v[E];
    C::load(xr + c * E, v);
#pragma unroll
    for (int i = 0; i < E; ++i) amax = fmaxf(amax, fabsf(v[i]));
  }
  amax = wave_max(amax);
  const float g = fmaxf(amax, 1e-5f);
  const float qscale = E4M3 ? 448.0f : 127.0f;
  const float inv = qscale / g;   // correctly rounded fp32 division
  if (lane == 0) xdq[row] = g / qscale;

  for (int c = lane; c < nchunk; c += kWave) {
    float v[E];
    C::load(xr + c * E, v);
    uint32_t out[E / 4];
#pragma unroll
    for (int w = 0; w < E / 4; ++w) {
      uint32_t word = 0;
#pragma unroll
      for (int i = 0; i < 4; ++i) {
        const float s = v[4 * w + i] * inv;
        uint32_t b;
        if constexpr (E4M3) {
          b = f32_to_e4m3(s);
        } else {
          const float r = fminf(fmaxf(rintf(s), -128.0f), 127.0f);
          b = (uint32_t)(int)r & 0xFFu;
        }
        word |= b << (8 * i);
      }
      out[w] = word;
    }
    if constexpr (E == 8) {
      *reinterpret_cast<uint2*>(qr + c * E) = make_uint2(out[0], out[1]);
    } else {
      *reinterpret_cast<uint32_t*>(qr + c * E) = out[0];
    }
  }
}

hipError_t launch_act_quant(const void* X, bool x_bf16, int64_t M, int K, bool e4m3, void* Xq,
                            float* xdq, hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const int rows_per_block = 4;
  const dim3 grid((unsigned)((M + rows_per_block - 1) / rows_per_block));
  const dim3 block(rows_per_block * kWave);
  uint8_t* q = static_cast<uint8_t*>(Xq);
  if (x_bf16) {
    const uint16_t* x = static_cast<const uint16_t*>(X);
    if (e4m3)
      hipLaunchKernelGGL((act_quant_kernel<uint16_t, true>), grid, block, 0, stream, x, M, K, q, xdq);
    else
      hipLaunchKernelGGL((act_quant_kernel<uint16_t, false>), grid, block, 0, stream, x, M, K, q, xdq);
  } else {
    const float* x = static_cast<const float*>(X);
    if (e4m3)
      hipLaunchKernelGGL((act_quant_kernel<float, true>), grid, block, 0, stream, x, M, K, q, xdq);
    else
      hipLaunchKernelGGL((act_quant_kernel<float, false>), grid, block, 0, stream, x, M, K, q, xdq);
  }
  return hipGetLastError();
}

}  // namespace dqt
