// fp32-environment backward products of a DQT linear (Sec. 3.2) on the
// gfx950 fp32 matrix cores (v_mfma_f32_32x32x2_f32):
//   dX[m, k] = alpha sum_n dY[m, n] q[n, k]
//   dW[n, k] = sum_m dY[m, n] X~[m, k],   X~ = value(Xq) * xdq in fp32
// used when the training environment is fp32 (bf16 environments use the
// bf16 kernels).  One kernel template computes C[i, j] = sum_r A(i, r) B(j, r)
// on a 128 x 128 tile with 16 fp32 reduction elements (64 bytes) per row per
// step.  Operand tiles are staged in LDS as [row][64 B] with the reduction
// contiguous (row pitch 80 B, conflict-free ds_read_b128 for 8 rows);
// operands whose reduction index is the source row (q for dX, dY and X~ for
// dW) are transposed in registers on the way in.  Four waves own 64 x 64
// quarters as 2 x 2 MFMA 32x32 blocks.  Lanes 0-31 / 32-63 read the first /
// second 32 bytes of a row's step; A and B use the same lane-to-reduction map.
//
// Also: the fixed-order sum of split-reduction partials used by both dW
// kernels.
#include "gemm_common.h"

namespace dqt {

namespace {

constexpr int BI = 128;
constexpr int BJ = 128;
constexpr int NT = 256;
constexpr int SEG = 64;
constexpr int PITCH = SEG + 16;
constexpr int TILE_BYTES = BI * PITCH;
constexpr int RSTEP = 16;          // fp32 reduction elements per step

using Acc = f32x16;

__device__ __forceinline__ void mma_step(const uint8_t* __restrict__ sA, const uint8_t* __restrict__ sB,
                                         Acc (&acc)[2][2], int lane, int wi, int wj) {
  const int r = lane & 31;
  const int h = lane >> 5;
  i32x4 a[2][2], b[2][2];
#pragma unroll
  for (int t = 0; t < 2; ++t) {
    const uint8_t* pa = sA + (wi * 64 + t * 32 + r) * PITCH + h * 32;
    const uint8_t* pb = sB + (wj * 64 + t * 32 + r) * PITCH + h * 32;
    a[t][0] = *reinterpret_cast<const i32x4*>(pa);
    a[t][1] = *reinterpret_cast<const i32x4*>(pa + 16);
    b[t][0] = *reinterpret_cast<const i32x4*>(pb);
    b[t][1] = *reinterpret_cast<const i32x4*>(pb + 16);
  }
#pragma unroll
  for (int ta = 0; ta < 2; ++ta)
#pragma unroll
    for (int tb = 0; tb < 2; ++tb)
#pragma unroll
      for (int s = 0; s < 8; ++s) {
        const float x = __int_as_float(a[ta][s >> 2][s & 3]);
        const float y = __int_as_float(b[tb][s >> 2][s & 3]);
        acc[ta][tb] = __builtin_amdgcn_mfma_f32_32x32x2f32(x, y, acc[ta][tb], 0, 0, 0);
      }
}

// Row-contiguous fp32 operand (dY for dX): 16-byte chunks, all in or all out.
struct ContigSrc {
  const uint8_t* base;
  int64_t ld;          // bytes between rows
  int64_t rows;
  int64_t red_bytes;
};
struct ContigStager {
  i32x4 v[2];
  __device__ void load(const ContigSrc& s, int64_t row0, int64_t r0, int64_t) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = threadIdx.x + NT * u;
      const int64_t gr = row0 + (c >> 2);
      const int64_t off = r0 * 4 + (c & 3) * 16;
      v[u] = (gr < s.rows && off < s.red_bytes)
                 ? *reinterpret_cast<const i32x4*>(s.base + gr * s.ld + off)
                 : i32x4{0, 0, 0, 0};
    }
  }
  __device__ void store(uint8_t* t) const {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = threadIdx.x + NT * u;
      *reinterpret_cast<i32x4*>(t + (c >> 2) * PITCH + (c & 3) * 16) = v[u];
    }
  }
};

// Transposed sources: the tile row is a column of the source matrix; each
// source yields a pair of adjacent columns (c, c+1) of one source row.
struct DyF32Src {
  const float* p; int64_t ld; int64_t rows; int64_t cols;
  __device__ float2 pairf(int64_t r, int64_t c) const {
    return *reinterpret_cast<const float2*>(p + r * ld + c);
  }
};
template <bool E4M3>
struct XtSrc {
  const uint8_t* p; const float* d; int64_t ld; int64_t rows; int64_t cols;
  __device__ float val(uint32_t code) const {
    return E4M3 ? e4m3_to_f32(code) : (float)(int)(int8_t)code;
  }
  __device__ float2 pairf(int64_t r, int64_t c) const {
    const uint32_t two = *reinterpret_cast<const uint16_t*>(p + r * ld + c);
    const float s = d[r];
    return make_float2(val(two & 0xFFu) * s, val(two >> 8) * s);
  }
};
struct QTernarySrc {
  const uint8_t* p; int64_t ld; int64_t rows; int64_t cols;   // ld = d_in / 4
  __device__ float2 pairf(int64_t r, int64_t c) const {
    const uint32_t cc = (p[r * ld + (c >> 2)] >> (2 * (c & 3))) & 0xFu;
    return make_float2(code_to_f32(cc & 3u), code_to_f32(cc >> 2));
  }
};
struct QInt8Src {
  const int8_t* p; int64_t ld; int64_t rows; int64_t cols;
  __device__ float2 pairf(int64_t r, int64_t c) const {
    const uint32_t two = *reinterpret_cast<const uint16_t*>(p + r * ld + c);
    return make_float2((float)(int)(int8_t)(two & 0xFFu), (float)(int)(int8_t)(two >> 8));
  }
};

// 16 reduction rows x 128 tile rows per step; thread -> tile rows
// (2cp, 2cp+1), reduction rows 4rg .. 4rg+3.
template <class Src>
struct TransF32Stager {
  float2 v[4];
  __device__ void load(const Src& s, int64_t row0, int64_t r0, int64_t r_end) {
    const int cp = threadIdx.x & 63, rg = threadIdx.x >> 6;
    const int64_t c = row0 + 2 * cp;
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      const int64_t rr = r0 + 4 * rg + i;
      v[i] = (rr < r_end && c < s.cols) ? s.pairf(rr, c) : make_float2(0.f, 0.f);
    }
  }
  __device__ void store(uint8_t* t) const {
    const int cp = threadIdx.x & 63, rg = threadIdx.x >> 6;
    *reinterpret_cast<f32x4*>(t + (2 * cp) * PITCH + rg * 16) = f32x4{v[0].x, v[1].x, v[2].x, v[3].x};
    *reinterpret_cast<f32x4*>(t + (2 * cp + 1) * PITCH + rg * 16) = f32x4{v[0].y, v[1].y, v[2].y, v[3].y};
  }
};

template <class SA, class SB, class LA, class LB, class Epi>
__global__ __launch_bounds__(NT) void gemm_f32_kernel(LA la, LB lb, Epi epi, int64_t I, int64_t J,
                                                      int64_t R, int64_t split_len) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[2][2][TILE_BYTES];
  const int64_t r_begin = (int64_t)blockIdx.z * split_len;
  int64_t r_end = r_begin + split_len;
  if (r_end > R) r_end = R;
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wi = wave >> 1, wj = wave & 1;
  const int64_t i0 = (int64_t)blockIdx.y * BI;
  const int64_t j0 = (int64_t)blockIdx.x * BJ;
  Acc acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0.0f;
  const int64_t nsteps = r_end > r_begin ? (r_end - r_begin + RSTEP - 1) / RSTEP : 0;
  SA sa;
  SB sb;
  if (nsteps > 0) {
    sa.load(la, i0, r_begin, r_end);
    sb.load(lb, j0, r_begin, r_end);
    sa.store(smem[0][0]);
    sb.store(smem[0][1]);
  }
  __syncthreads();
  for (int64_t s = 0; s < nsteps; ++s) {
    const int cur = (int)(s & 1);
    const bool more = s + 1 < nsteps;
    if (more) {
      const int64_t rn = r_begin + (s + 1) * RSTEP;
      sa.load(la, i0, rn, r_end);
      sb.load(lb, j0, rn, r_end);
    }
    mma_step(smem[cur][0], smem[cur][1], acc, lane, wi, wj);
    if (more) {
      sa.store(smem[cur ^ 1][0]);
      sb.store(smem[cur ^ 1][1]);
    }
    __syncthreads();
  }
  const int h = lane >> 5;
#pragma unroll
  for (int ta = 0; ta < 2; ++ta)
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const int64_t j = j0 + wj * 64 + tb * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t i = i0 + wi * 64 + ta * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (i < I && j < J) epi.put(i, j, acc[ta][tb][r]);
      }
    }
}

// Fixed-order sum of split partials: out[e] = sum_s ws[s][e], s = 0, 1, ...
__global__ __launch_bounds__(256) void split_reduce_kernel(const float* __restrict__ ws, int splits,
                                                           int64_t n4, float* __restrict__ out) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n4; t += stride) {
    f32x4 s = reinterpret_cast<const f32x4*>(ws)[t];
    for (int k = 1; k < splits; ++k) {
      const f32x4 v = reinterpret_cast<const f32x4*>(ws + (int64_t)k * n4 * 4)[t];
      s[0] = s[0] + v[0];
      s[1] = s[1] + v[1];
      s[2] = s[2] + v[2];
      s[3] = s[3] + v[3];
    }
    reinterpret_cast<f32x4*>(out)[t] = s;
  }
}

dim3 tile_grid(int64_t I, int64_t J, int64_t splits) {
  return dim3((unsigned)((J + BJ - 1) / BJ), (unsigned)((I + BI - 1) / BI), (unsigned)splits);
}

}  // namespace

hipError_t launch_split_reduce(const float* ws, int splits, int64_t n, float* out, hipStream_t stream) {
  const int64_t n4 = n / 4;
  int64_t blocks = (n4 + 255) / 256;
  if (blocks > 256 * 16) blocks = 256 * 16;
  if (blocks < 1) blocks = 1;
  return launch_kernel(split_reduce_kernel, dim3((unsigned)blocks), dim3(256), stream, ws, splits, n4, out);
}

hipError_t launch_dx_f32(const DxArgs& a, hipStream_t stream) {
  const int64_t I = a.M, J = a.d_in, R = a.d_out;
  if (I == 0) return hipSuccess;
  const dim3 grid = tile_grid(I, J, 1), block(NT);
  EpiScale epi{a.dX, J, a.dx_bf16, a.alpha};
  ContigSrc ya{static_cast<const uint8_t*>(a.dY), R * 4, I, R * 4};
  if (a.w_ternary) {
    QTernarySrc qb{static_cast<const uint8_t*>(a.Wq), J / 4, R, J};
    return timed_launch(stream, [&] {
      return launch_kernel(gemm_f32_kernel<ContigStager, TransF32Stager<QTernarySrc>, ContigSrc, QTernarySrc, EpiScale>,
                           grid, block, stream, ya, qb, epi, I, J, R, R);
    });
  } else {
    QInt8Src qb{static_cast<const int8_t*>(a.Wq), J, R, J};
    return timed_launch(stream, [&] {
      return launch_kernel(gemm_f32_kernel<ContigStager, TransF32Stager<QInt8Src>, ContigSrc, QInt8Src, EpiScale>,
                           grid, block, stream, ya, qb, epi, I, J, R, R);
    });
  }
}

int64_t dw_splits_f32(int64_t d_out, int64_t d_in, int64_t M) {
  const int64_t tiles = ((d_out + BI - 1) / BI) * ((d_in + BJ - 1) / BJ);
  int64_t s = (512 + tiles - 1) / tiles;
  const int64_t max_by_len = M / 512;
  if (s > max_by_len) s = max_by_len;
  if (s > 32) s = 32;
  if (s < 1) s = 1;
  return s;
}

hipError_t launch_dw_f32(const DwArgs& a, hipStream_t stream) {
  const int64_t I = a.d_out, J = a.d_in, R = a.M;
  const int64_t splits = dw_splits_f32(I, J, R);
  int64_t len = splits > 1 ? (R + splits - 1) / splits : (R > 0 ? R : 1);
  len = (len + RSTEP - 1) / RSTEP * RSTEP;
  const dim3 grid = tile_grid(I, J, splits), block(NT);
  float* target = splits > 1 ? a.ws : a.dW;
  EpiPartial epi{target, J, I * J};
  DyF32Src ya{static_cast<const float*>(a.dY), I, R, I};
  hipError_t e;
  if (a.act_e4m3) {
    XtSrc<true> xb{static_cast<const uint8_t*>(a.Xq), a.xdq, J, R, J};
    e = timed_launch(stream, [&] {
      return launch_kernel(gemm_f32_kernel<TransF32Stager<DyF32Src>, TransF32Stager<XtSrc<true>>, DyF32Src, XtSrc<true>, EpiPartial>,
                           grid, block, stream, ya, xb, epi, I, J, R, len);
    });
  } else {
    XtSrc<false> xb{static_cast<const uint8_t*>(a.Xq), a.xdq, J, R, J};
    e = timed_launch(stream, [&] {
      return launch_kernel(gemm_f32_kernel<TransF32Stager<DyF32Src>, TransF32Stager<XtSrc<false>>, DyF32Src, XtSrc<false>, EpiPartial>,
                           grid, block, stream, ya, xb, epi, I, J, R, len);
    });
  }
  if (e != hipSuccess || splits == 1) return e;
  return launch_split_reduce(a.ws, (int)splits, I * J, a.dW, stream);
}

}  // namespace dqt
