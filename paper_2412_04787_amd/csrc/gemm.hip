// The three contractions of a DQT linear train step (Sec. 3.2) on gfx950
// matrix cores:
//   forward  Y[m, n]  = sum_k Xq[m, k] q[n, k]    (int8 x int8 -> int32, or
//                                                  e4m3 x ternary -> fp32)
//   dX       dX[m, k] = alpha sum_n dY[m, n] q[n, k]       (bf16 or fp32)
//   dW       dW[n, k] = sum_m dY[m, n] X~[m, k]             (bf16 or fp32)
//
// One kernel template computes C[i, j] = sum_r A(i, r) B(j, r).  A block owns
// a 128 x 128 tile of C and walks the reduction in steps of 64 bytes of
// operand per row (64 int8/e4m3, 32 bf16 or 16 fp32 elements).  Each step
// both operand tiles are staged into LDS as [row][64 B] with the reduction
// contiguous (row pitch 80 B, so 8 consecutive rows of a ds_read_b128 hit
// distinct banks), double-buffered so one barrier per step suffices.  Operands
// whose reduction index is the row index in memory (Q for dX, dY and X~ for
// dW) are transposed in registers on the way in; packed 2-bit codes are
// unpacked and int8/e4m3 activations are dequantised there as well, so the
// MFMA loop only ever sees ready operands.
//
// Four waves of 64 threads each own a 64 x 64 quarter of the tile as 2 x 2
// MFMA 32x32 blocks.  Lane l of a 32x32 block reads row (l mod 32) of A and
// of B; lanes 0-31 take the first 32 bytes of the 64-byte step and lanes
// 32-63 the second.  A and B use the same lane-to-reduction-index map, which
// is all the instruction needs to produce sum_r A(i, r) B(j, r).
#include "dqt_launch.h"

namespace dqt {

constexpr int BI = 128;
constexpr int BJ = 128;
constexpr int NT = 256;
constexpr int SEG = 64;            // bytes of reduction per tile row per step
constexpr int PITCH = SEG + 16;    // LDS row pitch in bytes
constexpr int TILE_BYTES = BI * PITCH;

enum class Mfma { I8, F8, BF16, F32 };

template <Mfma K> struct AccT { using type = f32x16; };
template <> struct AccT<Mfma::I8> { using type = i32x16; };

template <Mfma K> constexpr int elem_bytes() {
  return K == Mfma::BF16 ? 2 : (K == Mfma::F32 ? 4 : 1);
}

// ------------------------------------------------------------- MFMA step
template <Mfma K>
__device__ __forceinline__ void mma_step(const uint8_t* __restrict__ sA,
                                         const uint8_t* __restrict__ sB,
                                         typename AccT<K>::type (&acc)[2][2], int lane, int wi,
                                         int wj) {
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
  for (int ta = 0; ta < 2; ++ta) {
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      if constexpr (K == Mfma::I8) {
        acc[ta][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[ta][0], b[tb][0], acc[ta][tb], 0, 0, 0);
        acc[ta][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(a[ta][1], b[tb][1], acc[ta][tb], 0, 0, 0);
      } else if constexpr (K == Mfma::BF16) {
        acc[ta][tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, a[ta][0]), __builtin_bit_cast(bf16x8, b[tb][0]), acc[ta][tb], 0, 0, 0);
        acc[ta][tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
            __builtin_bit_cast(bf16x8, a[ta][1]), __builtin_bit_cast(bf16x8, b[tb][1]), acc[ta][tb], 0, 0, 0);
      } else if constexpr (K == Mfma::F8) {
        const i32x8 av = {a[ta][0][0], a[ta][0][1], a[ta][0][2], a[ta][0][3],
                          a[ta][1][0], a[ta][1][1], a[ta][1][2], a[ta][1][3]};
        const i32x8 bv = {b[tb][0][0], b[tb][0][1], b[tb][0][2], b[tb][0][3],
                          b[tb][1][0], b[tb][1][1], b[tb][1][2], b[tb][1][3]};
        // both operands e4m3 (format 0), unit E8M0 scales (127 = 2^0)
        acc[ta][tb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, acc[ta][tb], 0, 0, 0,
                                                                      127, 0, 127);
      } else {
#pragma unroll
        for (int s = 0; s < 8; ++s) {
          const float x = __int_as_float(a[ta][s >> 2][s & 3]);
          const float y = __int_as_float(b[tb][s >> 2][s & 3]);
          acc[ta][tb] = __builtin_amdgcn_mfma_f32_32x32x2f32(x, y, acc[ta][tb], 0, 0, 0);
        }
      }
    }
  }
}

// ------------------------------------------------------------- staging
// Row-contiguous operand: row i of the tile starts at base + i * ld bytes and
// the reduction runs along the row.  Every 16-byte chunk is either wholly in
// range or wholly out (the reduction length is a multiple of 16 elements).
struct ContigSrc {
  const uint8_t* base;
  int64_t ld;          // bytes between rows
  int64_t rows;        // valid rows
  int64_t red_bytes;   // valid reduction bytes per row
};
struct ContigStager {
  i32x4 v[2];
  __device__ void load(const ContigSrc& s, int64_t row0, int64_t rb0) {
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int c = threadIdx.x + NT * u;
      const int64_t gr = row0 + (c >> 2);
      const int64_t off = rb0 + (c & 3) * 16;
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

// Packed ternary rows for 1-byte MFMA operands (int8 or e4m3): 64 codes per
// row per step = 16 packed bytes; thread -> (row tid/2, 8 packed bytes).
struct TernarySrc {
  const uint8_t* base;
  int64_t ld;          // packed bytes per row (d_in / 4)
  int64_t rows;
};
template <bool E4M3>
struct TernaryStager {
  uint32_t w[2];
  __device__ void load(const TernarySrc& s, int64_t row0, int64_t k0) {
    const int64_t gr = row0 + (threadIdx.x >> 1);
    const int64_t pb = k0 / 4 + (threadIdx.x & 1) * 8;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      const int64_t off = pb + 4 * u;
      // code 1 (= weight 0) fills out-of-range positions
      w[u] = (gr < s.rows && off < s.ld) ? *reinterpret_cast<const uint32_t*>(s.base + gr * s.ld + off)
                                         : 0x55555555u;
    }
  }
  __device__ void store(uint8_t* t) const {
    uint8_t* dst = t + (threadIdx.x >> 1) * PITCH + (threadIdx.x & 1) * 32;
#pragma unroll
    for (int u = 0; u < 2; ++u) {
      uint32_t o[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const uint32_t sp = spread_codes((w[u] >> (8 * b)) & 0xFFu);
        o[b] = E4M3 ? codes_to_e4m3x4(sp) : codes_to_i8x4(sp);
      }
      *reinterpret_cast<i32x4*>(dst + 16 * u) = i32x4{(int)o[0], (int)o[1], (int)o[2], (int)o[3]};
    }
  }
};

// Transposed sources: the tile row is a COLUMN of the source matrix and the
// reduction runs down the source's rows.  Each source provides pairs of
// adjacent columns (c, c+1) of one source row, as bf16 pairs or fp32 pairs.
struct DyBf16Src {            // dY [M, N] bf16; tile rows = n, reduction = m
  const uint16_t* p; int64_t ld; int64_t rows; int64_t cols;
  __device__ uint32_t pair(int64_t r, int64_t c) const {
    return *reinterpret_cast<const uint32_t*>(p + r * ld + c);
  }
};
struct DyF32Src {
  const float* p; int64_t ld; int64_t rows; int64_t cols;
  __device__ float2 pairf(int64_t r, int64_t c) const {
    return *reinterpret_cast<const float2*>(p + r * ld + c);
  }
};
template <bool E4M3>
struct XtSrc {                // X~ = value(Xq[m, k]) * xdq[m]; tile rows = k, reduction = m
  const uint8_t* p; const float* d; int64_t ld; int64_t rows; int64_t cols;
  __device__ float val(uint32_t code) const {
    return E4M3 ? e4m3_to_f32(code) : (float)(int)(int8_t)code;
  }
  __device__ float2 pairf(int64_t r, int64_t c) const {
    const uint32_t two = *reinterpret_cast<const uint16_t*>(p + r * ld + c);
    const float s = d[r];
    return make_float2(val(two & 0xFFu) * s, val(two >> 8) * s);
  }
  __device__ uint32_t pair(int64_t r, int64_t c) const {
    const float2 f = pairf(r, c);
    return pack_bf16x2(f.x, f.y);
  }
};
struct QTernarySrc {          // q[n, k] packed; tile rows = k, reduction = n
  const uint8_t* p; int64_t ld; int64_t rows; int64_t cols;   // ld = d_in / 4
  __device__ uint32_t codes2(int64_t r, int64_t c) const {
    const uint32_t byte = p[r * ld + (c >> 2)];
    return (byte >> (2 * (c & 3))) & 0xFu;
  }
  __device__ uint32_t pair(int64_t r, int64_t c) const {
    const uint32_t cc = codes2(r, c);
    return code_to_bf16_bits(cc & 3u) | (code_to_bf16_bits(cc >> 2) << 16);
  }
  __device__ float2 pairf(int64_t r, int64_t c) const {
    const uint32_t cc = codes2(r, c);
    return make_float2(code_to_f32(cc & 3u), code_to_f32(cc >> 2));
  }
};
struct QInt8Src {             // q[n, k] int8; tile rows = k, reduction = n
  const int8_t* p; int64_t ld; int64_t rows; int64_t cols;
  __device__ float2 pairf(int64_t r, int64_t c) const {
    const uint32_t two = *reinterpret_cast<const uint16_t*>(p + r * ld + c);
    return make_float2((float)(int)(int8_t)(two & 0xFFu), (float)(int)(int8_t)(two >> 8));
  }
  __device__ uint32_t pair(int64_t r, int64_t c) const {
    const float2 f = pairf(r, c);   // |q| <= 128: exact in bf16, truncation is exact
    return (__float_as_uint(f.x) >> 16) | (__float_as_uint(f.y) & 0xFFFF0000u);
  }
};

// bf16 transposed stager: 32 reduction rows x 128 tile rows per step.
// thread -> tile rows (2cp, 2cp+1), reduction rows 8rg .. 8rg+7.
template <class Src>
struct TransBf16Stager {
  uint32_t v[8];
  __device__ void load(const Src& s, int64_t row0, int64_t r0, int64_t r_end) {
    const int cp = threadIdx.x & 63, rg = threadIdx.x >> 6;
    const int64_t c = row0 + 2 * cp;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
      const int64_t rr = r0 + 8 * rg + i;
      v[i] = (rr < r_end && c < s.cols) ? s.pair(rr, c) : 0u;
    }
  }
  __device__ void store(uint8_t* t) const {
    const int cp = threadIdx.x & 63, rg = threadIdx.x >> 6;
    uint32_t lo[4], hi[4];
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      lo[i] = __builtin_amdgcn_perm(v[2 * i + 1], v[2 * i], 0x05040100u);
      hi[i] = __builtin_amdgcn_perm(v[2 * i + 1], v[2 * i], 0x07060302u);
    }
    *reinterpret_cast<i32x4*>(t + (2 * cp) * PITCH + rg * 16) =
        i32x4{(int)lo[0], (int)lo[1], (int)lo[2], (int)lo[3]};
    *reinterpret_cast<i32x4*>(t + (2 * cp + 1) * PITCH + rg * 16) =
        i32x4{(int)hi[0], (int)hi[1], (int)hi[2], (int)hi[3]};
  }
};

// fp32 transposed stager: 16 reduction rows x 128 tile rows per step.
// thread -> tile rows (2cp, 2cp+1), reduction rows 4rg .. 4rg+3.
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

template <Mfma K, class Epi>
__device__ __forceinline__ void write_tile(const typename AccT<K>::type (&acc)[2][2], const Epi& epi,
                                           int64_t i0, int64_t j0, int64_t I, int64_t J, int lane,
                                           int wi, int wj) {
  const int h = lane >> 5;
#pragma unroll
  for (int ta = 0; ta < 2; ++ta) {
#pragma unroll
    for (int tb = 0; tb < 2; ++tb) {
      const int64_t j = j0 + wj * 64 + tb * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t i = i0 + wi * 64 + ta * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (i < I && j < J) {
          float v;
          if constexpr (K == Mfma::I8) v = (float)acc[ta][tb][r];
          else v = acc[ta][tb][r];
          epi.put(i, j, v);
        }
      }
    }
  }
}

// ------------------------------------------------------------- kernels
// Generic mainloop.  SA/SB stage operand A (tile rows i) and B (tile rows j).
// Reduction range of this block: [r_begin, r_end) in elements.
template <Mfma K, class SA, class SB, class LA, class LB, class Epi>
__device__ __forceinline__ void gemm_body(const LA& la, const LB& lb, const Epi& epi, int64_t I,
                                          int64_t J, int64_t r_begin, int64_t r_end) {
  __shared__ __attribute__((aligned(16))) uint8_t smem[2][2][TILE_BYTES];
  constexpr int RSTEP = SEG / elem_bytes<K>();
  const int lane = threadIdx.x & 63;
  const int wave = threadIdx.x >> 6;
  const int wi = wave >> 1, wj = wave & 1;
  const int64_t i0 = (int64_t)blockIdx.y * BI;
  const int64_t j0 = (int64_t)blockIdx.x * BJ;

  typename AccT<K>::type acc[2][2];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < 2; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0;

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
    mma_step<K>(smem[cur][0], smem[cur][1], acc, lane, wi, wj);
    if (more) {
      sa.store(smem[cur ^ 1][0]);
      sb.store(smem[cur ^ 1][1]);
    }
    __syncthreads();
  }
  write_tile<K>(acc, epi, i0, j0, I, J, lane, wi, wj);
}

// Adapters giving every stager the same load(src, row0, r0, r_end) shape.
template <int EB>
struct ContigA : ContigStager {
  __device__ void load(const ContigSrc& s, int64_t row0, int64_t r0, int64_t) {
    ContigStager::load(s, row0, r0 * EB);
  }
};
template <bool E4M3>
struct TernaryB : TernaryStager<E4M3> {
  __device__ void load(const TernarySrc& s, int64_t row0, int64_t r0, int64_t) {
    TernaryStager<E4M3>::load(s, row0, r0);
  }
};

template <Mfma K, class SA, class SB, class LA, class LB, class Epi>
__global__ __launch_bounds__(NT) void gemm_kernel(LA la, LB lb, Epi epi, int64_t I, int64_t J,
                                                  int64_t R, int64_t split_len) {
  const int64_t rb = (int64_t)blockIdx.z * split_len;
  int64_t re = rb + split_len;
  if (re > R) re = R;
  gemm_body<K, SA, SB>(la, lb, epi, I, J, rb, re);
}

// Fixed-order sum of split partials: dW[e] = sum_s ws[s][e], s = 0, 1, ...
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

// ------------------------------------------------------------- launchers
static dim3 tile_grid(int64_t I, int64_t J, int64_t splits) {
  return dim3((unsigned)((J + BJ - 1) / BJ), (unsigned)((I + BI - 1) / BI), (unsigned)splits);
}

hipError_t launch_fwd(const FwdArgs& a, hipStream_t stream) {
  const int64_t I = a.M, J = a.d_out, R = a.d_in;
  if (I == 0) return hipSuccess;
  const dim3 grid = tile_grid(I, J, 1), block(NT);
  EpiFwd epi{a.Y, J, a.y_bf16, a.xdq, a.alpha};
  ContigSrc xa{static_cast<const uint8_t*>(a.Xq), R, I, R};
  if (a.w_ternary) {
    TernarySrc wb{static_cast<const uint8_t*>(a.Wq), R / 4, J};
    if (a.act_e4m3)
      hipLaunchKernelGGL((gemm_kernel<Mfma::F8, ContigA<1>, TernaryB<true>, ContigSrc, TernarySrc, EpiFwd>),
                         grid, block, 0, stream, xa, wb, epi, I, J, R, R);
    else
      hipLaunchKernelGGL((gemm_kernel<Mfma::I8, ContigA<1>, TernaryB<false>, ContigSrc, TernarySrc, EpiFwd>),
                         grid, block, 0, stream, xa, wb, epi, I, J, R, R);
  } else {
    ContigSrc wb{static_cast<const uint8_t*>(a.Wq), R, J, R};
    hipLaunchKernelGGL((gemm_kernel<Mfma::I8, ContigA<1>, ContigA<1>, ContigSrc, ContigSrc, EpiFwd>),
                       grid, block, 0, stream, xa, wb, epi, I, J, R, R);
  }
  return hipGetLastError();
}

hipError_t launch_dx(const DxArgs& a, hipStream_t stream) {
  // dX[m, k] = alpha sum_n dY[m, n] q[n, k]: I = M, J = d_in, R = d_out.
  const int64_t I = a.M, J = a.d_in, R = a.d_out;
  if (I == 0) return hipSuccess;
  const dim3 grid = tile_grid(I, J, 1), block(NT);
  EpiScale epi{a.dX, J, a.dx_bf16, a.alpha};
  if (a.dy_bf16) {
    ContigSrc ya{static_cast<const uint8_t*>(a.dY), R * 2, I, R * 2};
    if (a.w_ternary) {
      QTernarySrc qb{static_cast<const uint8_t*>(a.Wq), J / 4, R, J};
      hipLaunchKernelGGL((gemm_kernel<Mfma::BF16, ContigA<2>, TransBf16Stager<QTernarySrc>, ContigSrc, QTernarySrc, EpiScale>),
                         grid, block, 0, stream, ya, qb, epi, I, J, R, R);
    } else {
      QInt8Src qb{static_cast<const int8_t*>(a.Wq), J, R, J};
      hipLaunchKernelGGL((gemm_kernel<Mfma::BF16, ContigA<2>, TransBf16Stager<QInt8Src>, ContigSrc, QInt8Src, EpiScale>),
                         grid, block, 0, stream, ya, qb, epi, I, J, R, R);
    }
  } else {
    ContigSrc ya{static_cast<const uint8_t*>(a.dY), R * 4, I, R * 4};
    if (a.w_ternary) {
      QTernarySrc qb{static_cast<const uint8_t*>(a.Wq), J / 4, R, J};
      hipLaunchKernelGGL((gemm_kernel<Mfma::F32, ContigA<4>, TransF32Stager<QTernarySrc>, ContigSrc, QTernarySrc, EpiScale>),
                         grid, block, 0, stream, ya, qb, epi, I, J, R, R);
    } else {
      QInt8Src qb{static_cast<const int8_t*>(a.Wq), J, R, J};
      hipLaunchKernelGGL((gemm_kernel<Mfma::F32, ContigA<4>, TransF32Stager<QInt8Src>, ContigSrc, QInt8Src, EpiScale>),
                         grid, block, 0, stream, ya, qb, epi, I, J, R, R);
    }
  }
  return hipGetLastError();
}

int64_t dw_splits(int64_t d_out, int64_t d_in, int64_t M) {
  // Enough blocks to cover the 256 CUs about twice, each split at least 512
  // tokens long; the split count depends on the shape only.
  const int64_t tiles = ((d_out + BI - 1) / BI) * ((d_in + BJ - 1) / BJ);
  int64_t s = (512 + tiles - 1) / tiles;
  const int64_t max_by_len = M / 512;
  if (s > max_by_len) s = max_by_len;
  if (s > 32) s = 32;
  if (s < 1) s = 1;
  return s;
}

int64_t dw_split_len(int64_t M, int64_t splits, int64_t rstep) {
  int64_t len = (M + splits - 1) / splits;
  len = (len + rstep - 1) / rstep * rstep;
  return len;
}

hipError_t launch_dw(const DwArgs& a, hipStream_t stream) {
  // dW[n, k] = sum_m dY[m, n] X~[m, k]: I = d_out, J = d_in, R = M.
  const int64_t I = a.d_out, J = a.d_in, R = a.M;
  const int64_t splits = a.splits;
  const int rstep = a.xt_bf16 ? SEG / 2 : SEG / 4;
  const int64_t len = splits > 1 ? dw_split_len(R, splits, rstep) : (R > 0 ? R : 1);
  const dim3 grid = tile_grid(I, J, splits), block(NT);
  float* target = splits > 1 ? a.ws : a.dW;
  EpiPartial epi{target, J, I * J};
  if (a.xt_bf16) {
    DyBf16Src ya{static_cast<const uint16_t*>(a.dY), I, R, I};
    if (a.act_e4m3) {
      XtSrc<true> xb{static_cast<const uint8_t*>(a.Xq), a.xdq, J, R, J};
      hipLaunchKernelGGL((gemm_kernel<Mfma::BF16, TransBf16Stager<DyBf16Src>, TransBf16Stager<XtSrc<true>>, DyBf16Src, XtSrc<true>, EpiPartial>),
                         grid, block, 0, stream, ya, xb, epi, I, J, R, len);
    } else {
      XtSrc<false> xb{static_cast<const uint8_t*>(a.Xq), a.xdq, J, R, J};
      hipLaunchKernelGGL((gemm_kernel<Mfma::BF16, TransBf16Stager<DyBf16Src>, TransBf16Stager<XtSrc<false>>, DyBf16Src, XtSrc<false>, EpiPartial>),
                         grid, block, 0, stream, ya, xb, epi, I, J, R, len);
    }
  } else {
    DyF32Src ya{static_cast<const float*>(a.dY), I, R, I};
    if (a.act_e4m3) {
      XtSrc<true> xb{static_cast<const uint8_t*>(a.Xq), a.xdq, J, R, J};
      hipLaunchKernelGGL((gemm_kernel<Mfma::F32, TransF32Stager<DyF32Src>, TransF32Stager<XtSrc<true>>, DyF32Src, XtSrc<true>, EpiPartial>),
                         grid, block, 0, stream, ya, xb, epi, I, J, R, len);
    } else {
      XtSrc<false> xb{static_cast<const uint8_t*>(a.Xq), a.xdq, J, R, J};
      hipLaunchKernelGGL((gemm_kernel<Mfma::F32, TransF32Stager<DyF32Src>, TransF32Stager<XtSrc<false>>, DyF32Src, XtSrc<false>, EpiPartial>),
                         grid, block, 0, stream, ya, xb, epi, I, J, R, len);
    }
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  const int64_t n4 = I * J / 4;
  int64_t blocks = (n4 + 255) / 256;
  if (blocks > 256 * 16) blocks = 256 * 16;
  hipLaunchKernelGGL(split_reduce_kernel, dim3((unsigned)blocks), dim3(256), 0, stream, a.ws,
                     (int)splits, n4, a.dW);
  return hipGetLastError();
}

}  // namespace dqt
