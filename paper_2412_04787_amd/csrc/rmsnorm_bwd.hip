// Backward of the RMSNorm that feeds a group of DQT linears, for the model
// step: the linears' dX (the activation quantiser passes the gradient
// through) summed, then the norm's own backward, in one pass pair over the
// rows.  For row m of X [M, K] with r_m from dqt_rmsnorm_act_quant:
//   dn_mk = sum_i dY_i[m, k]                       (fp32, i in order)
//   g_mk  = dn_mk gamma_k
//   c_m   = (sum_k g_mk x_mk) / K
//   dX_mk = r_m g_mk - x_mk r_m^3 c_m              (rounded to bf16)
//   gpart[b, k] = sum over the rows m of block b of dn_mk x_mk r_m
// so dgamma_k = sum_b gpart[b, k] (the caller sums, in a fixed order).
//
// One wave per row, 4 waves per block; block b takes rows 4 b + w,
// 4 b + w + 4 B, ... (B blocks).  Each wave keeps its share of the gamma
// gradient in its own LDS row of K floats (no two lanes touch one slot), and
// the block adds the four rows in order at the end.  HBM traffic per element:
// 2 bytes per dY_i and 2 for x read once (the second pass finds the row in
// cache), 2 bytes of dX written.
#include "dqt_launch.h"

namespace dqt {

namespace {

constexpr int kWaves = 4;

struct DyArgs {
  const uint16_t* p[kMaxNormDy];
};

__device__ __forceinline__ void load8_bf16(const uint16_t* p, float (&v)[8]) {
  const uint4 u = *reinterpret_cast<const uint4*>(p);
  const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
  for (int i = 0; i < 4; ++i) {
    v[2 * i] = bf16_bits_to_f32(w[i] & 0xFFFFu);
    v[2 * i + 1] = bf16_bits_to_f32(w[i] >> 16);
  }
}

template <int NDY>
__global__ __launch_bounds__(kWaves * kWave) void rmsnorm_bwd_kernel(
    DyArgs dy, const uint16_t* __restrict__ X, const float* __restrict__ gamma,
    const float* __restrict__ rinv, int64_t M, int K, uint16_t* __restrict__ dX,
    float* __restrict__ gpart) {
  extern __shared__ float gsh[];              // [kWaves][K]
  const int lane = threadIdx.x & (kWave - 1);
  const int w = threadIdx.x / kWave;
  const int nchunk = K / 8;
  float* mine = gsh + (size_t)w * K;
  for (int k = lane; k < K; k += kWave) mine[k] = 0.0f;
  const float invK = __fdiv_rn(1.0f, (float)K);
  auto dn8 = [&](int64_t off, float (&dn)[8]) {
    load8_bf16(dy.p[0] + off, dn);
#pragma unroll
    for (int i = 1; i < NDY; ++i) {
      float t[8];
      load8_bf16(dy.p[i] + off, t);
#pragma unroll
      for (int j = 0; j < 8; ++j) dn[j] = dn[j] + t[j];
    }
  };
  for (int64_t row = (int64_t)blockIdx.x * kWaves + w; row < M; row += (int64_t)gridDim.x * kWaves) {
    const int64_t base = row * (int64_t)K;
    const float r = rinv[row];
    float dot = 0.0f;
    for (int c = lane; c < nchunk; c += kWave) {
      float dn[8], x[8];
      dn8(base + 8 * c, dn);
      load8_bf16(X + base + 8 * c, x);
      const float4 g0 = *reinterpret_cast<const float4*>(gamma + 8 * c);
      const float4 g1 = *reinterpret_cast<const float4*>(gamma + 8 * c + 4);
      const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
#pragma unroll
      for (int j = 0; j < 8; ++j) dot = dot + (dn[j] * g[j]) * x[j];
    }
#pragma unroll
    for (int d = 32; d > 0; d >>= 1) dot = dot + __shfl_xor(dot, d, kWave);
    const float cr3 = ((dot * invK) * r) * (r * r);
    for (int c = lane; c < nchunk; c += kWave) {
      float dn[8], x[8];
      dn8(base + 8 * c, dn);
      load8_bf16(X + base + 8 * c, x);
      const float4 g0 = *reinterpret_cast<const float4*>(gamma + 8 * c);
      const float4 g1 = *reinterpret_cast<const float4*>(gamma + 8 * c + 4);
      const float g[8] = {g0.x, g0.y, g0.z, g0.w, g1.x, g1.y, g1.z, g1.w};
      uint32_t o[4];
#pragma unroll
      for (int j = 0; j < 8; j += 2) {
        const float a = r * (dn[j] * g[j]) - x[j] * cr3;
        const float b = r * (dn[j + 1] * g[j + 1]) - x[j + 1] * cr3;
        o[j >> 1] = f32_to_bf16_bits(a) | (f32_to_bf16_bits(b) << 16);
      }
      *reinterpret_cast<uint4*>(dX + base + 8 * c) = make_uint4(o[0], o[1], o[2], o[3]);
#pragma unroll
      for (int j = 0; j < 8; ++j) mine[8 * c + j] += (dn[j] * x[j]) * r;
    }
  }
  __syncthreads();
  for (int k = threadIdx.x; k < K; k += kWaves * kWave) {
    float s = gsh[k];
#pragma unroll
    for (int i = 1; i < kWaves; ++i) s = s + gsh[(size_t)i * K + k];
    gpart[(int64_t)blockIdx.x * K + k] = s;
  }
}

}  // namespace

hipError_t launch_rmsnorm_backward(int n_dy, const void* const* dY, const void* X, const float* gamma,
                                   const float* rinv, int64_t M, int K, void* dX, float* gpart,
                                   int blocks, hipStream_t stream) {
  DyArgs a{};
  for (int i = 0; i < n_dy; ++i) a.p[i] = static_cast<const uint16_t*>(dY[i]);
  const size_t lds = (size_t)kWaves * K * sizeof(float);
  const dim3 grid((unsigned)blocks), block(kWaves * kWave);
  const uint16_t* x = static_cast<const uint16_t*>(X);
  uint16_t* dx = static_cast<uint16_t*>(dX);
  switch (n_dy) {
    case 1: return launch_kernel_lds(rmsnorm_bwd_kernel<1>, grid, block, lds, stream, a, x, gamma, rinv, M, K, dx, gpart);
    case 2: return launch_kernel_lds(rmsnorm_bwd_kernel<2>, grid, block, lds, stream, a, x, gamma, rinv, M, K, dx, gpart);
    case 3: return launch_kernel_lds(rmsnorm_bwd_kernel<3>, grid, block, lds, stream, a, x, gamma, rinv, M, K, dx, gpart);
    default: return launch_kernel_lds(rmsnorm_bwd_kernel<4>, grid, block, lds, stream, a, x, gamma, rinv, M, K, dx, gpart);
  }
}

}  // namespace dqt
