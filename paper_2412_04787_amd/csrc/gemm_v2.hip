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
// Block: 256 threads = 2 x 2 waves; a wave owns (32 WI) x (32 WJ) of C as
// WI x WJ MFMA 32x32 blocks; the block tile is (64 WI) x (64 WJ).  Step: 64 bytes of
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
#include <algorithm>
#include <type_traits>

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

template <int ELEM, int MA, int MB, int WI, int WJ>
struct Cfg {
  static constexpr int TRA = 64 * WI;          // tile rows of A (I)
  static constexpr int TRB = 64 * WJ;          // tile rows of B (J)
  static constexpr int EB = ELEM == EBF16 ? 2 : 1;
  static constexpr int BK = 64 / EB;           // reduction elements per step
  static constexpr int A_BYTES = TRA * 64;
  static constexpr int B_BYTES = TRB * 64;
  static constexpr int NLA = TRA / 64;         // DMA instructions per thread per stage
  static constexpr int NLB = TRB / 64;
  static constexpr int STAGE = A_BYTES + B_BYTES;
  static constexpr int LDS = STAGE * STAGES;
  static_assert(LDS <= 160 * 1024, "LDS budget");
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

// One GEMM problem of a grouped launch, with its tile grid (nbx x nby x
// nbz tiles: column tiles, row tiles, reduction splits) and the index of its
// first tile in the launch.
template <class Epi>
struct Prob {
  Opnd A, B;
  Epi epi;
  int64_t I, J, R, split_len;
  int32_t nbx, nby, nbz, ntiles;
};
constexpr int MAXG = 8;
template <class Epi>
struct Group {
  Prob<Epi> p[MAXG];
  int32_t ng;
};

template <int ELEM, int MA, int MB, int WI, int WJ, class Epi>
__global__ __launch_bounds__(NTH) void gemm_v2_kernel(const Group<Epi> grp) {
  using C = Cfg<ELEM, MA, MB, WI, WJ>;
  __shared__ __attribute__((aligned(1024))) uint8_t smem_generic[C::LDS];
  __shared__ float row_scale[Epi::kRowScale ? C::TRA : 1];
  lds_u8* smem = (lds_u8*)smem_generic;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wi = wave >> 1, wj = wave & 1;
  const int h = lane >> 5;
  // Workgroups are dispatched round-robin over the 8 XCDs (hardware id w
  // runs on XCD w mod 8, each XCD with its own L2), and in order of w within
  // an XCD.  XCD x takes a contiguous 1/8 of every problem's tiles, so that
  // the XCDs get equal work and tiles sharing operand panels share an L2;
  // problems are sorted longest reduction first, so the long tiles start
  // first.  The grid is padded to a multiple of 8 x the largest per-XCD
  // count; padding blocks have no tile and leave at once.
  int g = 0, bx, by, bz;
  {
    const int x = blockIdx.x & 7;
    int k = blockIdx.x >> 3;
    int local = -1;
    for (; g < grp.ng; ++g) {
      const int n = grp.p[g].ntiles;
      const int s0 = (x * n) >> 3, cnt = (((x + 1) * n) >> 3) - s0;
      if (k < cnt) { local = s0 + k; break; }
      k -= cnt;
    }
    if (local < 0) return;
    const int nbx = grp.p[g].nbx, nby = grp.p[g].nby;
    bx = local % nbx;
    by = (local / nbx) % nby;
    bz = local / (nbx * nby);
  }
  const Opnd A = grp.p[g].A;
  const Opnd B = grp.p[g].B;
  const Epi epi = grp.p[g].epi;
  const int64_t I = grp.p[g].I, J = grp.p[g].J, R = grp.p[g].R;
  const int64_t split_len = grp.p[g].split_len;
  const int64_t i0 = (int64_t)by * C::TRA;
  const int64_t j0 = (int64_t)bx * C::TRB;
  const int64_t r_begin = (int64_t)bz * split_len;
  int64_t r_end = r_begin + split_len;
  if (r_end > R) r_end = R;
  const int64_t rlen = r_end > r_begin ? r_end - r_begin : 0;
  const int nsteps = (int)((rlen + C::BK - 1) / C::BK);
  const bool tail = (rlen % C::BK) != 0;

  Plan<MA, C::TRA, C::EB> pa;
  Plan<MB, C::TRB, C::EB> pb;
  pa.init(A, i0, r_begin);
  pb.init(B, j0, r_begin);
  // wave-uniform LDS offset of this wave's DMA chunks (kept in an SGPR)
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  // per-row output scales of this tile: loaded before the first DMA (so the
  // in-order load counter retires them with stage 0) and staged in LDS
  // before the first barrier
  static_assert(C::TRA <= NTH, "one row scale per thread");
  float my_scale = 0.0f;
  if constexpr (Epi::kRowScale) {
    if (tid < C::TRA) {
      int64_t i = i0 + tid;
      if (i > I - 1) i = I - 1;
      my_scale = epi.scale(i);
    }
  }

  // Issue the DMA of stage s (its slot is s mod STAGES).  The per-thread
  // source pointers advance by one step per call, so stages are issued in
  // order 0, 1, 2, ...
  auto issue = [&](int s) {
    lds_u8* la = smem + (s % STAGES) * C::STAGE + wave_u * 1024;
    lds_u8* lb = la + C::A_BYTES;
    const bool last = tail && s == nsteps - 1;
    if (!last) {
#pragma unroll
      for (int q = 0; q < C::NLA; ++q) dma16(pa.g[q] + (int64_t)s * pa.inc, la + q * 4096);
#pragma unroll
      for (int q = 0; q < C::NLB; ++q) dma16(pb.g[q] + (int64_t)s * pb.inc, lb + q * 4096);
    } else {
      const int64_t rbase = (int64_t)s * C::BK;
#pragma unroll
      for (int q = 0; q < C::NLA; ++q)
        dma16(rbase + pa.rk[q] >= rlen ? pa.safe[q] : pa.g[q] + (int64_t)s * pa.inc, la + q * 4096);
#pragma unroll
      for (int q = 0; q < C::NLB; ++q)
        dma16(rbase + pb.rk[q] >= rlen ? pb.safe[q] : pb.g[q] + (int64_t)s * pb.inc, lb + q * 4096);
    }
  };
  // zero the chunks this lane loaded past the end of the reduction (the
  // lane's own DMA for stage s has completed)
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
  AccV acc[WI][WJ];
#pragma unroll
  for (int a = 0; a < WI; ++a)
#pragma unroll
    for (int b = 0; b < WJ; ++b)
#pragma unroll
      for (int r = 0; r < 16; ++r) acc[a][b][r] = 0;

  // fragment address parts
  const int frow = lane & 31;
  const int t4 = (lane >> 2) & 3, u4 = lane & 3, ch = (lane >> 4) & 1;

  // Fragments of one step: fa/fb for K-contiguous operands (ds_read_b128,
  // tracked by the compiler), ka/kb halves for K-major operands (transposing
  // reads issued as inline asm: the compiler would otherwise order every such
  // read after all outstanding DMA, vmcnt(0), serialising the ring; the vmcnt
  // waits and barriers order the DMA before these reads, and frag_wait()
  // orders the reads before use).
  struct Frags {
    i32x4 fa[WI][2], fb[WJ][2];
    u32x2 ka[WI][2][2], kb[WJ][2][2];
  };
  auto read_frags = [&](int s, Frags& F) {
    const lds_u8* la = smem + (s % STAGES) * C::STAGE;
    const lds_u8* lb = la + C::A_BYTES;
#pragma unroll
    for (int t = 0; t < WI; ++t)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        if constexpr (MA == KC) {
          const int row = wi * 32 * WI + t * 32 + frow;
          const int c = (2 * kk + h) ^ ((row >> 2) & 3);
          F.fa[t][kk] = *(const __attribute__((address_space(3))) i32x4*)(la + row * 64 + 16 * c);
        } else {
          const int col = wi * 32 * WI + t * 32 + 16 * ch + 4 * u4;
          const int seg = ((col & 63) >> 4) ^ t4;
          const uint32_t a0 = (uint32_t)(uintptr_t)(la + (col >> 6) * 4096 +
                                                    (16 * kk + 8 * h + t4) * 128 + 32 * seg + 8 * u4);
          asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(F.ka[t][kk][0]) : "v"(a0));
          asm volatile("ds_read_b64_tr_b16 %0, %1 offset:512" : "=v"(F.ka[t][kk][1]) : "v"(a0));
        }
      }
#pragma unroll
    for (int t = 0; t < WJ; ++t)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) {
        if constexpr (MB == KC) {
          const int row = wj * 32 * WJ + t * 32 + frow;
          const int c = (2 * kk + h) ^ ((row >> 2) & 3);
          F.fb[t][kk] = *(const __attribute__((address_space(3))) i32x4*)(lb + row * 64 + 16 * c);
        } else {
          const int col = wj * 32 * WJ + t * 32 + 16 * ch + 4 * u4;
          const int seg = ((col & 63) >> 4) ^ t4;
          const uint32_t a0 = (uint32_t)(uintptr_t)(lb + (col >> 6) * 4096 +
                                                    (16 * kk + 8 * h + t4) * 128 + 32 * seg + 8 * u4);
          asm volatile("ds_read_b64_tr_b16 %0, %1" : "=v"(F.kb[t][kk][0]) : "v"(a0));
          asm volatile("ds_read_b64_tr_b16 %0, %1 offset:512" : "=v"(F.kb[t][kk][1]) : "v"(a0));
        }
      }
  };
  // wait for this wave's outstanding LDS reads; ties the K-major halves so
  // that no use is scheduled before the wait
  auto frag_wait = [&](Frags& F) {
    if constexpr (MA == KM) {
#pragma unroll
      for (int t = 0; t < WI; ++t)
        tr_wait4(F.ka[t][0][0], F.ka[t][0][1], F.ka[t][1][0], F.ka[t][1][1]);
    }
    if constexpr (MB == KM) {
#pragma unroll
      for (int t = 0; t < WJ; ++t)
        tr_wait4(F.kb[t][0][0], F.kb[t][0][1], F.kb[t][1][0], F.kb[t][1][1]);
    }
    if constexpr (MA == KC && MB == KC) __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4) | (0 << 8));
  };
  auto mfma_step = [&](Frags& F) {
    i32x4 fa[WI][2], fb[WJ][2];
#pragma unroll
    for (int t = 0; t < WI; ++t)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) fa[t][kk] = MA == KC ? F.fa[t][kk] : join(F.ka[t][kk][0], F.ka[t][kk][1]);
#pragma unroll
    for (int t = 0; t < WJ; ++t)
#pragma unroll
      for (int kk = 0; kk < 2; ++kk) fb[t][kk] = MB == KC ? F.fb[t][kk] : join(F.kb[t][kk][0], F.kb[t][kk][1]);
#pragma unroll
    for (int ta = 0; ta < WI; ++ta) {
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
          // both operands e4m3 (format 0), unit E8M0 scales (127 = 2^0)
          acc[ta][tb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(av, bv, acc[ta][tb], 0, 0, 0,
                                                                        127, 0, 127);
        }
      }
    }
  };

  // Pipeline.  The ring holds STAGES steps.  Before the loop: DMA of stages
  // 0 .. STAGES-1, then step 0's fragments.  Iteration `it`: wait for stage
  // it+1's DMA, barrier (every wave has its step-it fragments in registers,
  // so slot it mod STAGES is free), DMA stage it+STAGES into that slot, read
  // step it+1's fragments, run step it's MFMAs while those reads land.
  constexpr int LPS = C::NLA + C::NLB;   // DMA instructions per thread per stage
  const int npre = nsteps < STAGES ? nsteps : STAGES;
  for (int s = 0; s < npre; ++s) issue(s);
  auto wait_stages = [&](int pending) {   // allow `pending` later stages in flight
    if (pending >= 3) wait_vm<3 * LPS>();
    else if (pending == 2) wait_vm<2 * LPS>();
    else if (pending == 1) wait_vm<LPS>();
    else wait_vm<0>();
  };
  Frags F0, F1;
  if (nsteps > 0) {
    wait_stages(npre - 1);
    if (tail && nsteps == 1) zero_tail(0);
  }
  if constexpr (Epi::kRowScale) {
    if (tid < C::TRA) row_scale[tid] = my_scale;
  }
  if (nsteps > 0) {
    block_barrier();
    read_frags(0, F0);
    frag_wait(F0);
  }
  auto iteration = [&](int it, Frags& cur, Frags& nxt) {
    if (it + 1 < nsteps) {
      const int issued_last = (it - 1 + STAGES < nsteps - 1) ? it - 1 + STAGES : nsteps - 1;
      wait_stages(issued_last - (it + 1));
      if (tail && it + 1 == nsteps - 1) zero_tail(it + 1);
    }
    block_barrier();
    if (it + STAGES < nsteps) issue(it + STAGES);
    if (it + 1 < nsteps) read_frags(it + 1, nxt);
    mfma_step(cur);
    if (it + 1 < nsteps) frag_wait(nxt);
  };
  int it = 0;
  for (; it + 1 < nsteps; it += 2) {
    iteration(it, F0, F1);
    iteration(it + 1, F1, F0);
  }
  if (it < nsteps) iteration(it, F0, F1);

  // Epilogue.  Lane (j = lane mod 32, h) of MFMA block (ta, tb) holds column
  // j of rows 8 (r / 4) + 4 h + (r mod 4), r = 0..15.  Each wave stages its
  // 32 x (32 WJ) result rows for one ta as fp32 in its own LDS region (the
  // ring is drained first), then writes whole 16-byte chunks of output rows.
  block_barrier();
  constexpr int COLS = 32 * WJ;
  constexpr int PITCHW = COLS + 4;                 // fp32 words per staged row
  lds_u8* stage = smem + wave * (32 * PITCHW * 4);
  const bool obf = epi.out_bf16();
#pragma unroll
  for (int ta = 0; ta < WI; ++ta) {
    const int64_t ibase = i0 + wi * 32 * WI + ta * 32;
    float sc[16];
#pragma unroll
    for (int r = 0; r < 16; ++r)
      sc[r] = Epi::kRowScale ? row_scale[wi * 32 * WI + ta * 32 + 8 * (r >> 2) + 4 * h + (r & 3)]
                             : epi.scale(0);
#pragma unroll
    for (int tb = 0; tb < WJ; ++tb) {
#pragma unroll
      for (int r = 0; r < 16; ++r) {
        float v;
        if constexpr (ELEM == EI8) v = (float)acc[ta][tb][r];
        else v = acc[ta][tb][r];
        v = v * sc[r];
        const int rr = 8 * (r >> 2) + 4 * h + (r & 3);
        *(__attribute__((address_space(3))) float*)(stage + (rr * PITCHW + tb * 32 + (lane & 31)) * 4) = v;
      }
    }
    __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    const int64_t jbase = j0 + wj * COLS;
    // read back whole 16-byte output chunks of rows (8 bf16 or 4 fp32)
    auto store_rows = [&](auto ebytes_tag) {
      constexpr int EBY = decltype(ebytes_tag)::value;
      constexpr int EPC = 16 / EBY;              // elements per chunk
      constexpr int CPR = COLS / EPC;            // chunks per row
#pragma unroll
      for (int c0 = 0; c0 < 32 * CPR; c0 += 64) {
        const int c = c0 + lane;
        const int rr = c / CPR, cc = c % CPR;
        const int64_t i = ibase + rr;
        const int64_t j = jbase + cc * EPC;
        if (i < I && j < J) {
          const lds_u8* src = stage + (rr * PITCHW + cc * EPC) * 4;
          uint8_t* dst = epi.row(i, bz) + j * EBY;
          if constexpr (EBY == 2) {
            const f32x4 a = *(const __attribute__((address_space(3))) f32x4*)src;
            const f32x4 b = *(const __attribute__((address_space(3))) f32x4*)(src + 16);
            *reinterpret_cast<uint4*>(dst) = make_uint4(pack_bf16x2(a[0], a[1]), pack_bf16x2(a[2], a[3]),
                                                        pack_bf16x2(b[0], b[1]), pack_bf16x2(b[2], b[3]));
          } else {
            *reinterpret_cast<f32x4*>(dst) = *(const __attribute__((address_space(3))) f32x4*)src;
          }
        }
      }
    };
    if (obf) store_rows(std::integral_constant<int, 2>{});
    else store_rows(std::integral_constant<int, 4>{});
    __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
  }
}

}  // namespace v2
}  // namespace dqt

// ------------------------------------------------------------ pre-passes
namespace dqt {
namespace v2 {

// Up to MAXG independent element ranges handled by one launch.  Segment s
// owns blocks [b0[s], b0[s+1]); each thread of a block handles one 16-element
// chunk; chunks past n16[s] do nothing.
struct SegTab {
  const void* src[MAXG];
  void* dst[MAXG];
  const float* scale[MAXG];   // per-row scales (activation dequantisation)
  int64_t n16[MAXG];
  int32_t k16[MAXG];          // 16-element chunks per row (activation dequantisation)
  int32_t b0[MAXG + 1];
  int32_t n;
};

__device__ __forceinline__ int seg_of_block(const SegTab& t) {
  int s = 0;
  while (s + 1 < t.n && (int)blockIdx.x >= t.b0[s + 1]) ++s;
  return s;
}

// Packed ternary codes -> one operand byte (int8 or e4m3) or one bf16 per
// weight, same [d_out][d_in] row-major order.
template <int OUT>   // 0: int8, 1: e4m3, 2: bf16
__global__ __launch_bounds__(256) void unpack_ternary_kernel(const SegTab tab) {
  const int s = seg_of_block(tab);
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  if (t >= tab.n16[s]) return;
  const uint32_t w = static_cast<const uint32_t*>(tab.src[s])[t];
  if constexpr (OUT < 2) {
    uint32_t o[4];
#pragma unroll
    for (int b = 0; b < 4; ++b) {
      const uint32_t sp = spread_codes((w >> (8 * b)) & 0xFFu);
      o[b] = OUT == 1 ? codes_to_e4m3x4(sp) : codes_to_i8x4(sp);
    }
    static_cast<uint4*>(tab.dst[s])[t] = make_uint4(o[0], o[1], o[2], o[3]);
  } else {
    uint32_t o[8];
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const uint32_t c = (w >> (4 * j)) & 0xFu;
      o[j] = code_to_bf16_bits(c & 3u) | (code_to_bf16_bits(c >> 2) << 16);
    }
    uint4* d = static_cast<uint4*>(tab.dst[s]) + 2 * t;
    d[0] = make_uint4(o[0], o[1], o[2], o[3]);
    d[1] = make_uint4(o[4], o[5], o[6], o[7]);
  }
}

// int8 codes -> bf16 (|q| <= 128 is exact in bf16).
__global__ __launch_bounds__(256) void int8_to_bf16_kernel(const SegTab tab) {
  const int s = seg_of_block(tab);
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  if (t >= tab.n16[s]) return;
  const uint4 v = static_cast<const uint4*>(tab.src[s])[t];
  const uint32_t w[4] = {v.x, v.y, v.z, v.w};
  uint32_t o[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t two = w[j >> 1] >> (16 * (j & 1));
    const float lo = (float)(int)(int8_t)(two & 0xFFu);
    const float hi = (float)(int)(int8_t)((two >> 8) & 0xFFu);
    o[j] = (__float_as_uint(lo) >> 16) | (__float_as_uint(hi) & 0xFFFF0000u);
  }
  uint4* d = static_cast<uint4*>(tab.dst[s]) + 2 * t;
  d[0] = make_uint4(o[0], o[1], o[2], o[3]);
  d[1] = make_uint4(o[4], o[5], o[6], o[7]);
}

// X~[m, k] = bf16(fl(value(Xq[m, k]) * xdq[m])).
template <bool E4M3>
__global__ __launch_bounds__(256) void dequant_act_kernel(const SegTab tab) {
  const int s = seg_of_block(tab);
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  if (t >= tab.n16[s]) return;
  const float d = tab.scale[s][t / tab.k16[s]];
  const uint4 v = static_cast<const uint4*>(tab.src[s])[t];
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
  uint4* dst = static_cast<uint4*>(tab.dst[s]) + 2 * t;
  dst[0] = make_uint4(o[0], o[1], o[2], o[3]);
  dst[1] = make_uint4(o[4], o[5], o[6], o[7]);
}

// Block tile shapes: (WI, WJ) -> (64 WI) x (64 WJ).
struct Tile {
  int wi, wj;
};
// Relative cost per output element of each tile shape in the operand-delivery
// bound regime the kernel runs in (bytes per flop shrink as the tile grows).
static double tile_cost(Tile t) {
  return 1.0 / (64.0 * t.wi) + 1.0 / (64.0 * t.wj);
}

// Fill in tile grids, sort the problems by reduction steps per tile
// (longest first) and launch one grid over every tile of every problem.
template <int ELEM, int MA, int MB, int WI, int WJ, class Epi>
static void launch_group_t(Group<Epi>& grp, hipStream_t s) {
  using C = Cfg<ELEM, MA, MB, WI, WJ>;
  const int64_t tra = C::TRA, trb = C::TRB;
  int64_t steps[MAXG];
  for (int g = 0; g < grp.ng; ++g) {
    Prob<Epi>& p = grp.p[g];
    p.nbx = (int32_t)((p.J + trb - 1) / trb);
    p.nby = (int32_t)((p.I + tra - 1) / tra);
    p.ntiles = p.nbx * p.nby * p.nbz;
    steps[g] = (std::min(p.split_len, p.R) + C::BK - 1) / C::BK;
  }
  for (int a = 1; a < grp.ng; ++a)          // stable insertion sort, descending
    for (int b = a; b > 0 && steps[b] > steps[b - 1]; --b) {
      std::swap(steps[b], steps[b - 1]);
      std::swap(grp.p[b], grp.p[b - 1]);
    }
  int32_t per_xcd = 0;
  for (int x = 0; x < 8; ++x) {
    int32_t c = 0;
    for (int g = 0; g < grp.ng; ++g) {
      const int32_t n = grp.p[g].ntiles;
      c += ((x + 1) * n >> 3) - (x * n >> 3);
    }
    per_xcd = std::max(per_xcd, c);
  }
  if (per_xcd == 0) return;
  hipLaunchKernelGGL((gemm_v2_kernel<ELEM, MA, MB, WI, WJ, Epi>), dim3((unsigned)(8 * per_xcd)), dim3(NTH),
                     0, s, grp);
}
template <int ELEM, int MA, int MB, class Epi>
static void launch_group(Tile t, Group<Epi>& grp, hipStream_t s) {
  if (t.wi == 4 && t.wj == 4) launch_group_t<ELEM, MA, MB, 4, 4, Epi>(grp, s);
  else if (t.wi == 4 && t.wj == 2) launch_group_t<ELEM, MA, MB, 4, 2, Epi>(grp, s);
  else if (t.wi == 2 && t.wj == 4) launch_group_t<ELEM, MA, MB, 2, 4, Epi>(grp, s);
  else launch_group_t<ELEM, MA, MB, 2, 2, Epi>(grp, s);
}

// Tile shape for a group: the one with the least (rounds of 256 CUs) x
// (tile area) x (cost per element); blocks of the larger tiles run one per CU.
static Tile pick_tile(int n, const int64_t* I, const int64_t* J, const int64_t* splits) {
  static const Tile cands[] = {{2, 2}, {4, 2}, {2, 4}, {4, 4}};
  Tile best = cands[0];
  double best_t = 1e300;
  for (const Tile& t : cands) {
    const int64_t tra = 64 * t.wi, trb = 64 * t.wj;
    int64_t blocks = 0;
    for (int g = 0; g < n; ++g) blocks += ((I[g] + tra - 1) / tra) * ((J[g] + trb - 1) / trb) * splits[g];
    const int per_cu = (t.wi * t.wj <= 4) ? 2 : 1;       // co-resident blocks per CU (LDS)
    const double rounds = (double)((blocks + 256 * per_cu - 1) / (256 * per_cu));
    const double tm = rounds * (double)(tra * trb) * per_cu * tile_cost(t);
    if (tm < best_t * 0.999) { best_t = tm; best = t; }
  }
  return best;
}

static int32_t seal(SegTab& t) {
  int32_t b = 0;
  for (int s = 0; s < t.n; ++s) {
    t.b0[s] = b;
    b += (int32_t)((t.n16[s] + 255) / 256);
  }
  t.b0[t.n] = b;
  return b;
}

}  // namespace v2

using namespace v2;

static size_t align256(size_t n) { return (n + 255) / 256 * 256; }

size_t fwd_batch_workspace(int n, const LinearIO* io, bool ternary, size_t* offs) {
  size_t total = 0;
  for (int l = 0; l < n; ++l) {
    if (offs) offs[l] = total;
    if (ternary) total += align256((size_t)(io[l].d_out * io[l].d_in));
  }
  return total;
}

hipError_t launch_fwd_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, hipStream_t stream) {
  if (c.M == 0 || c.n == 0) return hipSuccess;
  size_t offs[kMaxBatch];
  fwd_batch_workspace(c.n, io, c.w_ternary, offs);
  if (c.w_ternary) {
    SegTab tab{};
    tab.n = c.n;
    for (int l = 0; l < c.n; ++l) {
      tab.src[l] = io[l].Wq;
      tab.dst[l] = ws + offs[l];
      tab.n16[l] = io[l].d_out * io[l].d_in / 16;
    }
    const int32_t blocks = seal(tab);
    if (c.act_e4m3)
      hipLaunchKernelGGL(unpack_ternary_kernel<1>, dim3(blocks), dim3(256), 0, stream, tab);
    else
      hipLaunchKernelGGL(unpack_ternary_kernel<0>, dim3(blocks), dim3(256), 0, stream, tab);
  }
  Group<EpiFwd> grp{};
  grp.ng = c.n;
  int64_t I[kMaxBatch], J[kMaxBatch], S[kMaxBatch];
  for (int l = 0; l < c.n; ++l) {
    Prob<EpiFwd>& p = grp.p[l];
    const uint8_t* rows = c.w_ternary ? ws + offs[l] : static_cast<const uint8_t*>(io[l].Wq);
    p.A = Opnd{static_cast<const uint8_t*>(io[l].Xq), io[l].d_in, c.M};
    p.B = Opnd{rows, io[l].d_in, io[l].d_out};
    p.epi = EpiFwd{io[l].Y, io[l].d_out, c.out_bf16, io[l].xdq, io[l].alpha};
    p.I = c.M;
    p.J = io[l].d_out;
    p.R = io[l].d_in;
    p.split_len = io[l].d_in;
    p.nbz = 1;
    I[l] = p.I; J[l] = p.J; S[l] = 1;
  }
  const Tile tile = pick_tile(c.n, I, J, S);
  if (c.act_e4m3) launch_group<EF8, KC, KC>(tile, grp, stream);
  else launch_group<EI8, KC, KC>(tile, grp, stream);
  return hipGetLastError();
}

// Backward plan for a batch in the bf16 environment: tile width, one split
// count for every dW product of the batch, and the workspace layout
//   per linear: [bf16 weights d_out x d_in][bf16 X~ M x d_in][fp32 partials]
// (partials sized for the larger of this plan's and the fp32 kernels' split).
BwdPlan plan_bwd_batch(int n, const LinearIO* io, int64_t M) {
  BwdPlan P{};
  double best = 1e300;
  static const Tile cands[] = {{2, 2}, {4, 2}, {2, 4}, {4, 4}};
  for (const Tile& t : cands) {
    const int64_t tra = 64 * t.wi, trb = 64 * t.wj;
    const int per_cu = (t.wi * t.wj <= 4) ? 2 : 1;
    for (int64_t s = 1; s <= 32; ++s) {
      if (s > 1 && M / s < 256) break;
      int64_t blocks = 0;
      double part_bytes = 0;
      for (int l = 0; l < n; ++l) {
        blocks += ((io[l].d_out + tra - 1) / tra) * ((io[l].d_in + trb - 1) / trb) * s;
        if (s > 1) part_bytes += (2.0 * s + 1.0) * (double)(io[l].d_out * io[l].d_in * 4);
      }
      const double rounds = (double)((blocks + 256 * per_cu - 1) / (256 * per_cu));
      const double steps = (double)(((M + s - 1) / s + 31) / 32);
      // per step a block moves (tra + trb) * 64 bytes of operands at ~20 B/clk
      // per CU and runs 2 * tra * trb * 32 flops at ~4 Kflop/clk per CU
      const double clk = std::max((double)(tra + trb) * 64.0 / 20.0 * per_cu,
                                  2.0 * tra * trb * 32 / 4096.0 * per_cu);
      const double t_us = rounds * steps * clk / 2400.0 + part_bytes / 5.0e6;
      if (t_us < best * 0.999) { best = t_us; P.wi = t.wi; P.wj = t.wj; P.splits = s; }
    }
  }
  size_t off = 0;
  for (int l = 0; l < n; ++l) {
    const size_t wn = (size_t)(io[l].d_out * io[l].d_in);
    const int64_t s32 = dw_splits_f32(io[l].d_out, io[l].d_in, M);
    const int64_t sp = P.splits > s32 ? P.splits : s32;
    P.q_off[l] = off;
    off += align256(wn * 2);
    P.xt_off[l] = off;
    off += align256((size_t)M * (size_t)io[l].d_in * 2);
    P.part_off[l] = off;
    off += sp > 1 ? align256((size_t)sp * wn * 4) : 0;
  }
  P.total = off;
  return P;
}

hipError_t launch_dx_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                           hipStream_t stream) {
  if (c.M == 0 || c.n == 0) return hipSuccess;
  SegTab tab{};
  tab.n = c.n;
  for (int l = 0; l < c.n; ++l) {
    tab.src[l] = io[l].Wq;
    tab.dst[l] = ws + P.q_off[l];
    tab.n16[l] = io[l].d_out * io[l].d_in / 16;
  }
  const int32_t blocks = seal(tab);
  if (c.w_ternary)
    hipLaunchKernelGGL(unpack_ternary_kernel<2>, dim3(blocks), dim3(256), 0, stream, tab);
  else
    hipLaunchKernelGGL(int8_to_bf16_kernel, dim3(blocks), dim3(256), 0, stream, tab);
  // dX[m, k] = alpha sum_n dY[m, n] q[n, k]: I = M, J = d_in, R = d_out
  Group<EpiScale> grp{};
  grp.ng = c.n;
  int64_t I[kMaxBatch], J[kMaxBatch], S[kMaxBatch];
  for (int l = 0; l < c.n; ++l) {
    Prob<EpiScale>& p = grp.p[l];
    p.A = Opnd{static_cast<const uint8_t*>(io[l].dY), io[l].d_out * 2, c.M};
    p.B = Opnd{ws + P.q_off[l], io[l].d_in * 2, io[l].d_in};
    p.epi = EpiScale{io[l].dX, io[l].d_in, c.out_bf16, io[l].alpha};
    p.I = c.M;
    p.J = io[l].d_in;
    p.R = io[l].d_out;
    p.split_len = io[l].d_out;
    p.nbz = 1;
    I[l] = p.I; J[l] = p.J; S[l] = 1;
  }
  launch_group<EBF16, KC, KM>(pick_tile(c.n, I, J, S), grp, stream);
  return hipGetLastError();
}

hipError_t launch_dw_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                           hipStream_t stream) {
  if (c.n == 0) return hipSuccess;
  // X~ once per distinct quantised input
  int first[kMaxBatch];
  SegTab tab{};
  for (int l = 0; l < c.n; ++l) {
    first[l] = l;
    for (int m = 0; m < l; ++m)
      if (io[m].Xq == io[l].Xq && io[m].d_in == io[l].d_in) { first[l] = first[m]; break; }
    if (first[l] == l && c.M > 0) {
      const int s = tab.n++;
      tab.src[s] = io[l].Xq;
      tab.dst[s] = ws + P.xt_off[l];
      tab.scale[s] = io[l].xdq;
      tab.n16[s] = c.M * io[l].d_in / 16;
      tab.k16[s] = (int32_t)(io[l].d_in / 16);
    }
  }
  if (tab.n > 0) {
    const int32_t blocks = seal(tab);
    if (c.act_e4m3)
      hipLaunchKernelGGL(dequant_act_kernel<true>, dim3(blocks), dim3(256), 0, stream, tab);
    else
      hipLaunchKernelGGL(dequant_act_kernel<false>, dim3(blocks), dim3(256), 0, stream, tab);
  }
  // dW[n, k] = sum_m dY[m, n] X~[m, k]: I = d_out, J = d_in, R = M
  const int64_t splits = P.splits;
  int64_t len = splits > 1 ? (c.M + splits - 1) / splits : (c.M > 0 ? c.M : 1);
  len = (len + 31) / 32 * 32;
  Group<EpiPartial> grp{};
  grp.ng = c.n;
  for (int l = 0; l < c.n; ++l) {
    Prob<EpiPartial>& p = grp.p[l];
    const int64_t I = io[l].d_out, J = io[l].d_in;
    p.A = Opnd{static_cast<const uint8_t*>(io[l].dY), I * 2, I};
    p.B = Opnd{ws + P.xt_off[first[l]], J * 2, J};
    float* target = splits > 1 ? reinterpret_cast<float*>(ws + P.part_off[l]) : io[l].dW;
    p.epi = EpiPartial{target, J, I * J};
    p.I = I;
    p.J = J;
    p.R = c.M;
    p.split_len = len;
    p.nbz = (int32_t)splits;
  }
  launch_group<EBF16, KM, KM>(Tile{P.wi, P.wj}, grp, stream);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess || splits == 1) return e;
  for (int l = 0; l < c.n && e == hipSuccess; ++l)
    e = launch_split_reduce(reinterpret_cast<const float*>(ws + P.part_off[l]), (int)splits,
                            io[l].d_out * io[l].d_in, io[l].dW, stream);
  return e;
}

}  // namespace dqt
