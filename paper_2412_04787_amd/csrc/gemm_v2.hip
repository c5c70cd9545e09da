// MFMA GEMM for the int8 / e4m3 / bf16 contractions of the DQT linear step
// (Sec. 3.2), written for gfx950:
//   C[i, j] = sum_r A(i, r) B(j, r)
// Each operand is either K-contiguous (stored [rows][R], the reduction runs
// along a row) or K-major (stored [R][rows], bf16 only).  Operand tiles move
// global -> LDS by direct-to-LDS DMA (global_load_lds_dwordx4, no VGPR
// staging) into a 4-stage ring, so three steps of loads are in flight while
// the matrix cores work on the fourth.  Fragments come from LDS with
// ds_read_b128 (K-contiguous) or with the transposing ds_read_b64_tr_b16
// (K-major), which hands each lane eight reduction-consecutive bf16 values of
// one row straight from a row-major [R][rows] tile -- the dW = dY^T X~ and
// dX = dY Q products need no register transposes.
//
// Block: 256 threads = 2 x 2 waves; a wave owns 64 x (32 WJ) of C as 2 x WJ
// MFMA 32x32 blocks; the block tile is 128 x (64 WJ).  Step: 64 bytes of
// reduction per tile row (64 int8/e4m3 or 32 bf16 elements).
//
// LDS layouts (per stage, per operand), chosen so that every fragment read is
// free of bank conflicts on 32- and 64-bank LDS:
//   K-contiguous: [rows][64 B]; the 16-byte chunk c of row r sits at
//     position c ^ ((r >> 2) & 3).
//   K-major (bf16): 64-column regions, each [32 reduction rows][128 B]; the
//     32-byte segment s of row k sits at position s ^ (k & 3).
// The DMA writes 64 consecutive 16-byte chunks per wave instruction, so each
// lane loads the global chunk that belongs at its LDS position.
#include "gemm_common.h"

namespace dqt {
namespace v2 {

using lds_u8 = __attribute__((address_space(3))) uint8_t;
typedef short s16x4 __attribute__((ext_vector_type(4)));
using lds_s16x4 = __attribute__((address_space(3))) s16x4;

constexpr int NTH = 256;
constexpr int STAGES = 4;

enum Elem { EI8 = 0, EF8 = 1, EBF16 = 2 };
enum Mode { KC = 0, KM = 1 };

template <int ELEM, int MA, int MB, int WJ>
struct Cfg {
  static constexpr int TRA = 128;              // tile rows of A (I)
  static constexpr int TRB = 64 * WJ;          // tile rows of B (J)
  static constexpr int EB = ELEM == EBF16 ? 2 : 1;
  static constexpr int BK = 64 / EB;           // reduction elements per step
  static constexpr int A_BYTES = TRA * 64;
  static constexpr int B_BYTES = TRB * 64;
  static constexpr int NLA = TRA / 64;         // DMA instructions per thread per stage
  static constexpr int NLB = TRB / 64;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDS = STAGE * STAGES;
  static_assert(ELEM == EBF16 || (MA == KC && MB == KC), "K-major operands are bf16 only");
};

// Global operand: base of element (row 0, reduction 0), row stride in bytes,
// extent of the tile dimension, reduction length (elements).
struct Opnd {
  const uint8_t* p;
  int64_t ld;
  int64_t n;
};

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

// Wait for every outstanding LDS read of this wave; the four fragments are
// tied in and out so that no use of them is scheduled before the wait.
__device__ __forceinline__ void tr_wait4(u32x2& a, u32x2& b, u32x2& c, u32x2& d) {
  asm volatile("s_waitcnt lgkmcnt(0)" : "+v"(a), "+v"(b), "+v"(c), "+v"(d));
}
__device__ __forceinline__ i32x4 join(u32x2 lo, u32x2 hi) {
  return i32x4{(int)lo[0], (int)lo[1], (int)hi[0], (int)hi[1]};
}

__device__ __forceinline__ void dma16(const uint8_t* g, lds_u8* l) {
  __builtin_amdgcn_global_load_lds(g, (__attribute__((address_space(3))) void*)l, 16, 0, 0);
}

template <int N>
__device__ __forceinline__ void wait_vm() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Barrier that keeps the compiler from moving memory accesses across it but
// does not wait for outstanding DMA (the explicit vmcnt waits do that).
__device__ __forceinline__ void block_barrier() {
  __asm__ volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4) | (0 << 8));   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __asm__ volatile("" ::: "memory");
}

// Per-thread DMA plan of one operand: for each of its NL instructions, the
// global address at step 0, the reduction index (relative to the step start)
// that the chunk covers, and the per-step address increment.
template <int MODE, int TR, int EB>
struct Plan {
  static constexpr int NL = TR / 64;
  const uint8_t* g[NL];
  const uint8_t* safe[NL];
  int rk[NL];           // reduction element offset of the chunk within a step
  int64_t inc;          // bytes per step

  __device__ void init(const Opnd& o, int64_t row0, int64_t r_begin) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int q = 0; q < NL; ++q) {
      const int p = q * NTH + tid;                  // physical chunk position
      if constexpr (MODE == KC) {
        const int row = p >> 2;
        const int c = (p & 3) ^ ((row >> 2) & 3);   // logical 16-byte chunk
        int64_t gr = row0 + row;
        if (gr > o.n - 1) gr = o.n - 1;
        g[q] = o.p + gr * o.ld + r_begin * EB + 16 * c;
        safe[q] = o.p + gr * o.ld;
        rk[q] = 16 * c / EB;
      } else {
        const int region = p >> 8;                  // 64-column region
        const int k = (p & 255) >> 3;               // reduction row within the step
        const int pc = p & 7;
        const int seg = (pc >> 1) ^ (k & 3);
        int64_t col = row0 + 64 * region + 16 * seg + 8 * (pc & 1);
        if (col > o.n - 8) col = o.n - 8;
        g[q] = o.p + (r_begin + k) * o.ld + 2 * col;
        safe[q] = o.p + r_begin * o.ld + 2 * col;
        rk[q] = k;
      }
    }
    inc = MODE == KC ? 64 : 32 * o.ld;
  }
};

template <int ELEM, int MA, int MB, int WJ, class Epi>
__global__ __launch_bounds__(NTH) void gemm_v2_kernel(Opnd A, Opnd B, Epi epi, int64_t I,
                                                         int64_t J, int64_t R, int64_t split_len) {
  using C = Cfg<ELEM, MA, MB, WJ>;
  __shared__ __attribute__((aligned(1024))) uint8_t smem_generic[C::LDS];
  lds_u8* smem = (lds_u8*)smem_generic;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wi = wave >> 1, wj = wave & 1;
  const int h = lane >> 5;
  const int64_t i0 = (int64_t)blockIdx.y * C::TRA;
  const int64_t j0 = (int64_t)blockIdx.x * C::TRB;
  const int64_t r_begin = (int64_t)blockIdx.z * split_len;
  int64_t r_end = r_begin + split_len;
  if (r_end > R) r_end = R;
  const int64_t rlen = r_end > r_begin ? r_end - r_begin : 0;
  const int nsteps = (int)((rlen + C::BK - 1) / C::BK);
  const bool tail = (rlen % C::BK) != 0;

  Plan<MA, C::TRA, C::EB> pa;
  Plan<MB, C::TRB, C::EB> pb;
  pa.init(A, i0, r_begin);
  pb.init(B, j0, r_begin);

  auto issue = [&](int s) {
    lds_u8* la = smem + (s % STAGES) * C::STAGE;
    lds_u8* lb = la + C::A_BYTES;
    const bool last = tail && s == nsteps - 1;
    const int64_t rbase = (int64_t)s * C::BK;
#pragma unroll
    for (int q = 0; q < C::NLA; ++q) {
      const uint8_t* g = pa.g[q] + (int64_t)s * pa.inc;
      if (last && rbase + pa.rk[q] >= rlen) g = pa.safe[q];
      dma16(g, la + (q * 4 + wave) * 1024);
    }
#pragma unroll
    for (int q = 0; q < C::NLB; ++q) {
      const uint8_t* g = pb.g[q] + (int64_t)s * pb.inc;
      if (last && rbase + pb.rk[q] >= rlen) g = pb.safe[q];
      dma16(g, lb + (q * 4 + wave) * 1024);
    }
  };
  // zero the chunks this lane loaded past the end of the reduction
  auto zero_tail = [&](int s) {
    lds_u8* la = smem + (s % STAGES) * C::STAGE;
    lds_u8* lb = la + C::A_BYTES;
    const int64_t rbase = (int64_t)s * C::BK;
    const i32x4 z = {0, 0, 0, 0};
#pragma unroll
    for (int q = 0; q < C::NLA; ++q)
      if (rbase + pa.rk[q] >= rlen) *(__attribute__((address_space(3))) i32x4*)(la + (q * NTH + tid) * 16) = z;
#pragma unroll
    for (int q = 0; q < C::NLB; ++q)
      if (rbase + pb.rk[q] >= rlen) *(__attribute__((address_space(3))) i32x4*)(lb + (q * NTH + tid) * 16) = z;
  };

  using AccV = typename AccT<ELEM == EI8 ? Mfma::I8 : Mfma::BF16>::type;
  AccV acc[2][WJ];
#pragma unroll
  for (int a = 0; a < 2; ++a)
#pragma unroll
    for (int b = 0; b < WJ; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0;

  // fragment address parts
  const int frow = lane & 31;
  const int t4 = (lane >> 2) & 3, u4 = lane & 3, ch = (lane >> 4) & 1;

  auto frag_kc = [&](const lds_u8* base, int row, int kk) -> i32x4 {
    const int c = (2 * kk + h) ^ ((row >> 2) & 3);
    return *(const __attribute__((address_space(3))) i32x4*)(base + row * 64 + 16 * c);
  };
  // K-major fragments: two transposing reads give reduction slots 0-3 and
  // 4-7 of the lane's column.  Issued as inline asm: the compiler would
  // otherwise order every such read after all outstanding DMA (vmcnt(0)),
  // serialising the ring; the vmcnt waits and barrier above already order the
  // DMA before these reads, and tr_wait() below orders the reads before use.
  auto frag_km = [&](const lds_u8* base, int col0, int kk, u32x2& lo, u32x2& hi) {
    const int col = col0 + 16 * ch + 4 * u4;
    const int region = col >> 6;
    const int seg = ((col & 63) >> 4) ^ t4;
    const uint32_t a0 = (uint32_t)(uintptr_t)(base + region * 4096 + (16 * kk + 8 * h + t4) * 128 +
                                              32 * seg + 8 * u4);
    asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(lo) : "v"(a0));
    asm volatile("ds_read_b64_tr_b16 %0, %1 offset:512" : "=v"(hi) : "v"(a0));
  };

  const int npre = nsteps < STAGES - 1 ? nsteps : STAGES - 1;
  for (int s = 0; s < npre; ++s) issue(s);

  constexpr int LPS = C::NLA + C::NLB;   // DMA instructions per thread per stage
  for (int it = 0; it < nsteps; ++it) {
    const int ahead = nsteps - 1 - it < STAGES - 2 ? nsteps - 1 - it : STAGES - 2;
    if (ahead >= 2) wait_vm<2 * LPS>();
    else if (ahead == 1) wait_vm<LPS>();
    else wait_vm<0>();
    if (tail && it == nsteps - 1) zero_tail(it);
    block_barrier();
    if (it + STAGES - 1 < nsteps) issue(it + STAGES - 1);

    const lds_u8* la = smem + (it % STAGES) * C::STAGE;
    const lds_u8* lb = la + C::A_BYTES;
    i32x4 fa[2][2], fb[WJ][2];
    u32x2 ta_lo[2][2], ta_hi[2][2], tb_lo[WJ][2], tb_hi[WJ][2];
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        if constexpr (MA == KC) fa[t][kk] = frag_kc(la, wi * 64 + t * 32 + frow, kk);
        else frag_km(la, wi * 64 + t * 32, kk, ta_lo[t][kk], ta_hi[t][kk]);
      }
#pragma unroll
    for (int t = 0; t < WJ; ++t)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        if constexpr (MB == KC) fb[t][kk] = frag_kc(lb, wj * 32 * WJ + t * 32 + frow, kk);
        else frag_km(lb, wj * 32 * WJ + t * 32, kk, tb_lo[t][kk], tb_hi[t][kk]);
      }
    if constexpr (MA == KM) {
      tr_wait4(ta_lo[0][0], ta_hi[0][0], ta_lo[0][1], ta_hi[0][1]);
      tr_wait4(ta_lo[1][0], ta_hi[1][0], ta_lo[1][1], ta_hi[1][1]);
#pragma unroll
      for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) fa[t][kk] = join(ta_lo[t][kk], ta_hi[t][kk]);
    }
    if constexpr (MB == KM) {
#pragma unroll
      for (int t = 0; t < WJ; ++t) tr_wait4(tb_lo[t][0], tb_hi[t][0], tb_lo[t][1], tb_hi[t][1]);
#pragma unroll
      for (int t = 0; t < WJ; ++t)
#pragma unroll
        for (int kk = 0; kk < 2; ++kk) fb[t][kk] = join(tb_lo[t][kk], tb_hi[t][kk]);
    }
#pragma unroll
    for (int ta = 0; ta < 2; ++ta) {
#pragma unroll
      for (int tb = 0; tb < WJ; ++tb) {
        if constexpr (ELEM == EI8) {
          acc[ta][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[ta][0], fb[tb][0], acc[ta][tb], 0, 0, 0);
          acc[ta][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(fa[ta][1], fb[tb][1], acc[ta][tb], 0, 0, 0);
        } else if constexpr (ELEM == EBF16) {
          acc[ta][tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[ta][0]),
                                                                __builtin_bit_cast(bf16x8, fb[tb][0]),
                                                                acc[ta][tb], 0, 0, 0);
          acc[ta][tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, fa[ta][1]),
                                                                __builtin_bit_cast(bf16x8, fb[tb][1]),
                                                                acc[ta][tb], 0, 0, 0);
        } else {
          const i32x8 av = {fa[ta][0][0], fa[ta][0][1], fa[ta][0][2], fa[ta][0][3],
                            fa[ta][1][0], fa[ta][1][1], fa[ta][1][2], fa[ta][1][3]};
          const i32x8 bv = {fb[tb][0][0], fb[tb][0][1], fb[tb][0][2], fb[tb][0][3],
                            fb[tb][1][0], fb[tb][1][1], fb[tb][1][2], fb[tb][1][3]};
          acc[ta][tb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, acc[ta][tb], 0, 0, 0,
                                                                        127, 0, 127);
        }
      }
    }
  }

  // epilogue: lane (j = lane mod 32, h) of block (ta, tb) holds rows
  // 8 (r / 4) + 4 h + (r mod 4), r = 0..15
#pragma unroll
  for (int ta = 0; ta < 2; ++ta) {
#pragma unroll
    for (int tb = 0; tb < WJ; ++tb) {
      const int64_t j = j0 + wj * 32 * WJ + tb * 32 + (lane & 31);
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        const int64_t i = i0 + wi * 64 + ta * 32 + 8 * (r >> 2) + 4 * h + (r & 3);
        if (i < I && j < J) {
          float v;
          if constexpr (ELEM == EI8) v = (float)acc[ta][tb][r];
          else v = acc[ta][tb][r];
          epi.put(i, j, v);
        }
      }
    }
  }
}

}  // namespace v2
}  // namespace dqt

// ------------------------------------------------------------ pre-passes
namespace dqt {
namespace v2 {

// Packed ternary codes -> one operand byte (int8 or e4m3) or one bf16 per
// weight, same [d_out][d_in] row-major order.  Thread -> 16 weights.
template <int OUT>   // 0: int8, 1: e4m3, 2: bf16
__global__ __launch_bounds__(256) void unpack_ternary_kernel(const uint32_t* __restrict__ src,
                                                             int64_t n16, uint8_t* __restrict__ dst) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n16; t += stride) {
    const uint32_t w = src[t];
    if constexpr (OUT < 2) {
      uint32_t o[4];
#pragma unroll
      for (int b = 0; b < 4; ++b) {
        const uint32_t sp = spread_codes((w >> (8 * b)) & 0xFFu);
        o[b] = OUT == 1 ? codes_to_e4m3x4(sp) : codes_to_i8x4(sp);
      }
      reinterpret_cast<uint4*>(dst)[t] = make_uint4(o[0], o[1], o[2], o[3]);
    } else {
      uint32_t o[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const uint32_t c = (w >> (4 * j)) & 0xFu;
        o[j] = code_to_bf16_bits(c & 3u) | (code_to_bf16_bits(c >> 2) << 16);
      }
      uint4* d = reinterpret_cast<uint4*>(dst) + 2 * t;
      d[0] = make_uint4(o[0], o[1], o[2], o[3]);
      d[1] = make_uint4(o[4], o[5], o[6], o[7]);
    }
  }
}

// int8 codes -> bf16 (|q| <= 128 is exact in bf16).  Thread -> 16 weights.
__global__ __launch_bounds__(256) void int8_to_bf16_kernel(const uint4* __restrict__ src, int64_t n16,
                                                           uint4* __restrict__ dst) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n16; t += stride) {
    const uint4 v = src[t];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t two = w[j >> 1] >> (16 * (j & 1));
      const float lo = (float)(int)(int8_t)(two & 0xFFu);
      const float hi = (float)(int)(int8_t)((two >> 8) & 0xFFu);
      o[j] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
    }
    dst[2 * t] = make_uint4(o[0], o[1], o[2], o[3]);
    dst[2 * t + 1] = make_uint4(o[4], o[5], o[6], o[7]);
  }
}

// X~[m, k] = bf16(fl(value(Xq[m, k]) * xdq[m])).  Thread -> 16 elements of one row.
template <bool E4M3>
__global__ __launch_bounds__(256) void dequant_act_kernel(const uint4* __restrict__ xq,
                                                          const float* __restrict__ xdq, int64_t n16,
                                                          int k16, uint4* __restrict__ xt) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n16; t += stride) {
    const float d = xdq[t / k16];
    const uint4 v = xq[t];
    const uint32_t w[4] = {v.x, v.y, v.z, v.w};
    uint32_t o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t two = w[j >> 1] >> (16 * (j & 1));
      float a, b;
      if constexpr (E4M3) {
        a = e4m3_to_f32(two & 0xFFu);
        b = e4m3_to_f32((two >> 8) & 0xFFu);
      } else {
        a = (float)(int)(int8_t)(two & 0xFFu);
        b = (float)(int)(int8_t)((two >> 8) & 0xFFu);
      }
      o[j] = pack_bf16x2(a * d, b * d);
    }
    xt[2 * t] = make_uint4(o[0], o[1], o[2], o[3]);
    xt[2 * t + 1] = make_uint4(o[4], o[5], o[6], o[7]);
  }
}

static dim3 stream_grid(int64_t n) {
  int64_t b = (n + 255) / 256;
  if (b > 256 * 16) b = 256 * 16;
  if (b < 1) b = 1;
  return dim3((unsigned)b);
}

// Tile choice: 128 x 128 (WJ = 2) or 128 x 192 (WJ = 3), whichever needs
// fewer rounds of 256 CUs times tile area -- the matrix-core time when every
// CU runs its blocks back to back.
static int pick_wj(int64_t I, int64_t J, int64_t splits) {
  int best = 2;
  double best_t = 1e300;
  for (int wj = 2; wj <= 3; ++wj) {
    const int64_t trb = 64 * wj;
    const int64_t blocks = ((I + 127) / 128) * ((J + trb - 1) / trb) * splits;
    const double t = (double)((blocks + 255) / 256) * (double)(128 * trb);
    if (t < best_t * 0.999) { best_t = t; best = wj; }
  }
  return best;
}

template <int ELEM, int MA, int MB, class Epi>
static void launch_core(int wj, Opnd A, Opnd B, Epi epi, int64_t I, int64_t J, int64_t R,
                        int64_t splits, int64_t split_len, hipStream_t s) {
  const int64_t trb = 64 * wj;
  const dim3 grid((unsigned)((J + trb - 1) / trb), (unsigned)((I + 127) / 128), (unsigned)splits);
  if (wj == 3)
    hipLaunchKernelGGL((gemm_v2_kernel<ELEM, MA, MB, 3, Epi>), grid, dim3(NTH), 0, s, A, B, epi, I,
                       J, R, split_len);
  else
    hipLaunchKernelGGL((gemm_v2_kernel<ELEM, MA, MB, 2, Epi>), grid, dim3(NTH), 0, s, A, B, epi, I,
                       J, R, split_len);
}

}  // namespace v2

size_t fwd_workspace_bytes(bool ternary, int64_t d_out, int64_t d_in) {
  return ternary ? (size_t)((d_out * d_in + 255) / 256 * 256) : 0;
}

hipError_t launch_fwd_v2(const FwdArgs& a, hipStream_t stream) {
  using namespace v2;
  const int64_t I = a.M, J = a.d_out, R = a.d_in;
  if (I == 0) return hipSuccess;
  const uint8_t* wrows = static_cast<const uint8_t*>(a.Wq);
  if (a.w_ternary) {
    const int64_t n16 = J * R / 16;
    if (a.act_e4m3)
      hipLaunchKernelGGL(unpack_ternary_kernel<1>, stream_grid(n16), dim3(256), 0, stream,
                         static_cast<const uint32_t*>(a.Wq), n16, static_cast<uint8_t*>(a.ws));
    else
      hipLaunchKernelGGL(unpack_ternary_kernel<0>, stream_grid(n16), dim3(256), 0, stream,
                         static_cast<const uint32_t*>(a.Wq), n16, static_cast<uint8_t*>(a.ws));
    wrows = static_cast<const uint8_t*>(a.ws);
  }
  Opnd A{static_cast<const uint8_t*>(a.Xq), R, I};
  Opnd B{wrows, R, J};
  EpiFwd epi{a.Y, J, a.y_bf16, a.xdq, a.alpha};
  const int wj = pick_wj(I, J, 1);
  if (a.act_e4m3)
    launch_core<EF8, KC, KC>(wj, A, B, epi, I, J, R, 1, R, stream);
  else
    launch_core<EI8, KC, KC>(wj, A, B, epi, I, J, R, 1, R, stream);
  return hipGetLastError();
}

hipError_t launch_dx_v2(const DxArgs& a, void* ws_q, hipStream_t stream) {
  using namespace v2;
  // dX[m, k] = alpha sum_n dY[m, n] q[n, k]: I = M, J = d_in, R = d_out
  const int64_t I = a.M, J = a.d_in, R = a.d_out;
  if (I == 0) return hipSuccess;
  const int64_t n16 = R * J / 16;
  if (a.w_ternary)
    hipLaunchKernelGGL(unpack_ternary_kernel<2>, stream_grid(n16), dim3(256), 0, stream,
                       static_cast<const uint32_t*>(a.Wq), n16, static_cast<uint8_t*>(ws_q));
  else
    hipLaunchKernelGGL(int8_to_bf16_kernel, stream_grid(n16), dim3(256), 0, stream,
                       static_cast<const uint4*>(a.Wq), n16, static_cast<uint4*>(ws_q));
  Opnd A{static_cast<const uint8_t*>(a.dY), R * 2, I};
  Opnd B{static_cast<const uint8_t*>(ws_q), J * 2, J};
  EpiScale epi{a.dX, J, a.dx_bf16, a.alpha};
  launch_core<EBF16, KC, KM>(pick_wj(I, J, 1), A, B, epi, I, J, R, 1, R, stream);
  return hipGetLastError();
}

// Split count and tile for dW = dY^T X~ (reduction over M tokens): choose the
// pair that minimises matrix-core rounds plus the fp32 partial traffic.
void plan_dw_v2(int64_t d_out, int64_t d_in, int64_t M, int* wj_out, int64_t* splits_out) {
  double best = 1e300;
  int bw = 2;
  int64_t bs = 1;
  for (int wj = 2; wj <= 3; ++wj) {
    const int64_t trb = 64 * wj;
    const int64_t tiles = ((d_out + 127) / 128) * ((d_in + trb - 1) / trb);
    for (int64_t s = 1; s <= 32; ++s) {
      if (s > 1 && M / s < 256) break;
      const int64_t blocks = tiles * s;
      const double rounds = (double)((blocks + 255) / 256);
      const double steps = (double)((M + s - 1) / s + 31) / 32.0;
      // per-block MFMA time: 2 * 128 * trb * 32 flops per step at ~9.8 TFLOP/s per CU
      const double t_mfma = rounds * steps * (2.0 * 128 * trb * 32) / 9.8e12;
      const double t_part = s > 1 ? (2.0 * s + 1.0) * (double)(d_out * d_in * 4) / 5.0e12 : 0.0;
      const double t = t_mfma + t_part;
      if (t < best * 0.999) { best = t; bw = wj; bs = s; }
    }
  }
  *wj_out = bw;
  *splits_out = bs;
}

hipError_t launch_dw_v2(const DwArgs& a, void* ws_xt, hipStream_t stream) {
  using namespace v2;
  // dW[n, k] = sum_m dY[m, n] X~[m, k]: I = d_out, J = d_in, R = M
  const int64_t I = a.d_out, J = a.d_in, R = a.M;
  int wj;
  int64_t splits;
  plan_dw_v2(I, J, R, &wj, &splits);
  if (R > 0) {
    const int64_t n16 = R * J / 16;
    if (a.act_e4m3)
      hipLaunchKernelGGL(dequant_act_kernel<true>, stream_grid(n16), dim3(256), 0, stream,
                         static_cast<const uint4*>(a.Xq), a.xdq, n16, (int)(J / 16),
                         static_cast<uint4*>(ws_xt));
    else
      hipLaunchKernelGGL(dequant_act_kernel<false>, stream_grid(n16), dim3(256), 0, stream,
                         static_cast<const uint4*>(a.Xq), a.xdq, n16, (int)(J / 16),
                         static_cast<uint4*>(ws_xt));
  }
  int64_t len = splits > 1 ? (R + splits - 1) / splits : (R > 0 ? R : 1);
  len = (len + 31) / 32 * 32;
  float* target = splits > 1 ? a.ws : a.dW;
  Opnd A{static_cast<const uint8_t*>(a.dY), I * 2, I};
  Opnd B{static_cast<const uint8_t*>(ws_xt), J * 2, J};
  EpiPartial epi{target, J, I * J};
  launch_core<EBF16, KM, KM>(wj, A, B, epi, I, J, R, splits, len, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  return launch_split_reduce(a.ws, (int)splits, I * J, a.dW, stream);
}

}  // namespace dqt
