// RMSNorm of each token followed by its 8-bit activation quantisation, in
// one launch (the inputs of a LLaMA block's q/k/v and gate/up linears are
// RMSNorm outputs, and Sec. 3.2 quantises the linears' inputs to 8 bits):
//   s_m  = sum_k fl(x_mk x_mk)                  (fixed fp32 order, below)
//   r_m  = fl(1 / fl(sqrt(fl(fl(s_m / K) + eps))))
//   y_mk = fl(fl(x_mk r_m) gamma_k)
//   g_m  = max(max_k |y_mk|, 1e-5), Xq = quantise(y fl(Q / g_m)), xdq = fl(g_m / Q)
// with Q = 127 (int8, rint and clamp) or 448 (e4m3, saturating RNE).  The
// normalised row y never reaches memory.
//
// One wave per row, 4 rows per block.  Sum order: lane l adds the squares of
// the 8-element chunks l, l + 64, ... (elements in order) into an fp32 sum
// from 0, then a butterfly over lanes (distance 32, 16, ..., 1): every pair
// adds the same two values, so every lane ends with the same total.  Three
// passes over the row (squares; the maximum of |y|; the codes): the first
// reads HBM, the later ones find the row in cache.  HBM traffic per element:
// 2 or 4 bytes read and 1 byte written, plus gamma (read once per pass from
// cache).
#include "dqt_launch.h"

namespace dqt {

namespace {

constexpr int kRows = 4;   // rows (waves) per block

// 8 consecutive elements of a row as fp32 (bf16 rows: one 16-byte load;
// fp32 rows: two)
template <typename TX>
__device__ __forceinline__ void load8(const TX* p, float (&v)[8]) {
  if constexpr (sizeof(TX) == 2) {
    const uint4 u = *reinterpret_cast<const uint4*>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = bf16_bits_to_f32(w[i] & 0xFFFFu);
      v[2 * i + 1] = bf16_bits_to_f32(w[i] >> 16);
    }
  } else {
    const float4 a = *reinterpret_cast<const float4*>(p);
    const float4 b = *reinterpret_cast<const float4*>(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
  }
}

template <typename TX, bool E4M3>
__global__ __launch_bounds__(kRows * kWave) void rmsnorm_quant_kernel(const TX* __restrict__ X,
                                                                    const float* __restrict__ gamma,
                                                                    float eps, int64_t M, int K,
                                                                    uint8_t* __restrict__ Xq,
                                                                    float* __restrict__ xdq,
                                                                    float* __restrict__ rinv) {
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = (int64_t)blockIdx.x * kRows + threadIdx.x / kWave;
  if (row >= M) return;
  const TX* xr = X + row * (int64_t)K;
  uint8_t* qr = Xq + row * (int64_t)K;
  const int nchunk = K / 8;

  // pass 1: the sum of squares in the fixed order
  float s = 0.0f;
  for (int c = lane; c < nchunk; c += kWave) {
    float v[8];
    load8(xr + 8 * c, v);
#pragma unroll
    for (int j = 0; j < 8; ++j) s = s + v[j] * v[j];
  }
#pragma unroll
  for (int d = 32; d > 0; d >>= 1) s = s + __shfl_xor(s, d, kWave);
  const float mean = __fdiv_rn(s, (float)K);
  const float r = __fdiv_rn(1.0f, sqrtf(mean + eps));

  // pass 2: the largest |y|
  float amax = 0.0f;
  for (int c = lane; c < nchunk; c += kWave) {
    float v[8];
    load8(xr + 8 * c, v);
    const float4 g0 = *reinterpret_cast<const float4*>(gamma + 8 * c);
    const float4 g1 = *reinterpret_cast<const float4*>(gamma + 8 * c + 4);
    const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
    for (int j = 0; j < 8; ++j) amax = fmaxf(amax, fabsf((v[j] * r) * g[j]));
  }
  amax = wave_max(amax);
  const float qscale = E4M3 ? 448.0f : 127.0f;
  const float gmax = fmaxf(amax, 1e-5f);
  const float inv = __fdiv_rn(qscale, gmax);
  if (lane == 0) {
    xdq[row] = __fdiv_rn(gmax, qscale);
    if (rinv != nullptr) rinv[row] = r;
  }

  // pass 3: the codes
  for (int c = lane; c < nchunk; c += kWave) {
    float v[8];
    load8(xr + 8 * c, v);
    const float4 g0 = *reinterpret_cast<const float4*>(gamma + 8 * c);
    const float4 g1 = *reinterpret_cast<const float4*>(gamma + 8 * c + 4);
    const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
    float q[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) q[j] = ((v[j] * r) * g[j]) * inv;
    uint32_t w[2];
    if constexpr (E4M3) {
      w[0] = f32x4_to_e4m3x4(q[0], q[1], q[2], q[3]);
      w[1] = f32x4_to_e4m3x4(q[4], q[5], q[6], q[7]);
    } else {
      w[0] = f32x4_to_i8x4(q[0], q[1], q[2], q[3]);
      w[1] = f32x4_to_i8x4(q[4], q[5], q[6], q[7]);
    }
    *reinterpret_cast<uint2*>(qr + 8 * c) = make_uint2(w[0], w[1]);
  }
}

}  // namespace

hipError_t launch_rmsnorm_act_quant(const void* X, bool x_bf16, const float* gamma, float eps, int64_t M,
                                    int K, bool e4m3, void* Xq, float* xdq, float* rinv,
                                    hipStream_t stream) {
  if (M == 0) return hipSuccess;
  const dim3 grid((unsigned)((M + kRows - 1) / kRows)), block(kRows * kWave);
  uint8_t* q = static_cast<uint8_t*>(Xq);
  if (x_bf16) {
    const uint16_t* x = static_cast<const uint16_t*>(X);
    if (e4m3) return launch_kernel(rmsnorm_quant_kernel<uint16_t, true>, grid, block, stream, x, gamma, eps, M, K, q, xdq, rinv);
    return launch_kernel(rmsnorm_quant_kernel<uint16_t, false>, grid, block, stream, x, gamma, eps, M, K, q, xdq, rinv);
  }
  const float* x = static_cast<const float*>(X);
  if (e4m3) return launch_kernel(rmsnorm_quant_kernel<float, true>, grid, block, stream, x, gamma, eps, M, K, q, xdq, rinv);
  return launch_kernel(rmsnorm_quant_kernel<float, false>, grid, block, stream, x, gamma, eps, M, K, q, xdq, rinv);
}

}  // namespace dqt
