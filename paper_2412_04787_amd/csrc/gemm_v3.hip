// MFMA GEMM for the int8 / e4m3 / bf16 contractions of the DQT linear step
// (Sec. 3.2), written for gfx950:
//   C[i, j] = sum_r A(i, r) B(j, r)
// Each operand is either K-contiguous (stored [rows][R], the reduction runs
// along a row) or K-major (stored [R][rows], bf16 only).
//
// Design (measured on MI355X):
//  * Block tile 256 x 256, 8 waves in a 2 x 4 grid, each wave 128 x 64 as
//    4 x 2 MFMA 32x32 blocks.  Two waves share each SIMD, so one wave's LDS
//    and barrier waits are covered by the other's matrix instructions.  At
//    this tile size a full-rate MFMA loop needs ~32 B/clk/CU of operands.
//  * Operands move global -> LDS with direct-to-LDS DMA
//    (global_load_lds_dwordx4, no VGPR staging) in steps of one 128-byte
//    cache line per tile row (128 int8 / e4m3 or 64 bf16 reduction
//    elements): streaming whole lines delivers ~35 B/clk/CU, half lines only
//    ~21.  Two 64 KB stages: the DMA of step s+1 lands while step s runs.
//  * Persistent grid, one block per CU.  XCD x (workgroups are dispatched
//    round-robin over the 8 XCDs, each with its own L2) owns a contiguous
//    1/8 of every problem's tiles, problems sorted longest reduction first;
//    its blocks take tiles from that list through an atomic counter, so a
//    block that finishes early takes the next one (longest-first list
//    scheduling).  Before a tile's epilogue the
//    block issues the first DMA stage of its next tile, so the load latency
//    hides behind the epilogue.
//  * Fragments come from LDS with ds_read_b128 (K-contiguous) or with the
//    transposing ds_read_b64_tr_b16 (K-major), which hands each lane eight
//    reduction-consecutive bf16 of one row straight from a [R][rows] tile, so
//    dW = dY^T X~ and dX = dY Q need no register transposes.
//
// LDS layouts (per stage, per operand), free of bank conflicts for the
// fragment reads:
//   K-contiguous: [256 rows][128 B]; 16-byte chunk c of row r sits at
//     position c ^ ((r >> 1) & 7).
//   K-major (bf16): four 64-column regions, each [64 reduction rows][128 B];
//     the 32-byte segment s of row k sits at position s ^ (k & 3).
// Each DMA wave instruction fills 1 KB of consecutive LDS positions, so each
// lane loads the global chunk that belongs at its position.
#include <algorithm>
#include <cstdlib>
#include <cstring>
#include <type_traits>

#include "gemm_common.h"
#include "sr_rule.h"

namespace dqt {
namespace v3 {

typedef unsigned int u32x2 __attribute__((ext_vector_type(2)));

#ifndef GEMM_NW
#define GEMM_NW 8
#endif
constexpr int NW = GEMM_NW;           // waves per block: 8 (2 x 4 grid) or 4 (2 x 2)
static_assert(NW == 8 || NW == 4, "8 or 4 waves");
constexpr int NTH = 64 * NW;
constexpr int NTD = NTH;             // threads issuing global -> LDS copies
constexpr int TILE = 256;             // block tile edge (outputs)
constexpr int WI = 4;                 // MFMA 32x32 blocks per wave along rows
constexpr int WJ = NW == 8 ? 2 : 4;   // ... and along columns
constexpr int WGC = TILE / (32 * WJ); // waves per row of the wave grid
// packed ternary codes per tile row per step: one code per reduction element,
// four per byte (32 bytes for an 8-bit step of 128, 16 for a bf16 step of 64)
template <int KB, int EB>
constexpr int pkb() { return KB / EB / 4; }

// Step geometry for KB reduction bytes per tile row per step (128: one cache
// line; 64: half a line, used with more stages in flight).  K-contiguous
// tiles are [256 rows][KB bytes]; K-major (bf16) tiles are KB / 2 reduction
// rows of 256 columns, stored as four 64-column regions.
template <int KB>
struct Geo {
  static_assert(KB == 128 || KB == 64, "step of 64 or 128 bytes");
  static constexpr int OPB = TILE * KB;       // bytes per operand per stage
  static constexpr int NL = OPB / 16 / NTD;   // DMA chunks per DMA thread per operand
  static constexpr int CPR = KB / 16;         // K-contiguous 16-byte chunks per row
  static constexpr int KR = KB / 2;           // K-major rows per step
  static constexpr int NKK = KB / 32;         // MFMA sub-steps per step
  // K-contiguous swizzle: chunk c of row r sits at c ^ swz(r) (conflict-free
  // ds_read_b128 for 8 or 4 chunks per row)
  __device__ static int swz(int r) { return CPR == 8 ? (r >> 1) & 7 : (r >> 2) & 3; }
};


// EF4B: e4m3 A with ternary B as FP4 (E2M1) values formed from the packed
// codes in registers (B must be packed codes)
enum Elem { EI8 = 0, EF8 = 1, EBF16 = 2, EF4B = 3 };
// KCP: K-contiguous packed ternary codes (B only); KF4: K-contiguous FP4
// (E2M1) values, two per byte (B only, with e4m3 A), expanded from the codes
// by a pass into the workspace
enum Mode { KC = 0, KM = 1, KCP = 2, KF4 = 3 };

// bytes per stage: A, then B (bf16 / 8-bit operand, or packed ternary codes)
template <int MB, int KB, int EB>
constexpr int slot_bytes() {
  return Geo<KB>::OPB + (MB == KCP ? TILE * pkb<KB, EB>() : MB == KF4 ? TILE * KB / 2 : Geo<KB>::OPB);
}


// Global operand: base of element (row 0, reduction 0), row stride in bytes,
// extent of the tile dimension.
struct Opnd {
  const uint8_t* p;
  int64_t ld;
  int64_t n;
};

// One GEMM problem of a grouped launch: nbx x nby x nbz tiles (column tiles,
// row tiles, reduction splits).
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
  // tile counters: next[x] is the next tile of XCD x's list to hand out,
  // done[x] counts XCD x's blocks that found the list empty (the last one
  // resets both to zero for the next launch)
  int* sched;
};

typedef short s16x4 __attribute__((ext_vector_type(4)));
// Transposing LDS read: each lane receives four 16-bit values of one column
// from four consecutive rows of a row-major tile (ds_read_b64_tr_b16).
__device__ __forceinline__ u32x2 tr_read(const lds_u8* base, int off) {
  const s16x4 v = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
      (__attribute__((address_space(3))) s16x4*)(base + off));
  return __builtin_bit_cast(u32x2, v);
}
__device__ __forceinline__ i32x4 join(u32x2 lo, u32x2 hi) {
  return i32x4{(int)lo[0], (int)lo[1], (int)hi[0], (int)hi[1]};
}
// 16 packed ternary codes (code q + 1 at bits 2k, 2k+1) -> 16 operand bytes
// in k order, via the byte lookup `lut` (code 0, 1, 2 -> lut bytes 0, 1, 2):
// split the four codes of every byte into four byte planes, transpose the
// 4 x 4 byte matrix, then look each code up.
__device__ __forceinline__ i32x4 expand16(uint32_t x, uint32_t lut) {
  const uint32_t e = x & 0x03030303u, f = (x >> 2) & 0x03030303u;
  const uint32_t g = (x >> 4) & 0x03030303u, h = (x >> 6) & 0x03030303u;
  const uint32_t efl = __builtin_amdgcn_perm(f, e, 0x05010400u), efh = __builtin_amdgcn_perm(f, e, 0x07030602u);
  const uint32_t ghl = __builtin_amdgcn_perm(h, g, 0x05010400u), ghh = __builtin_amdgcn_perm(h, g, 0x07030602u);
  const uint32_t d0 = __builtin_amdgcn_perm(ghl, efl, 0x05040100u), d1 = __builtin_amdgcn_perm(ghl, efl, 0x07060302u);
  const uint32_t d2 = __builtin_amdgcn_perm(ghh, efh, 0x05040100u), d3 = __builtin_amdgcn_perm(ghh, efh, 0x07060302u);
  return i32x4{(int)__builtin_amdgcn_perm(0u, lut, d0), (int)__builtin_amdgcn_perm(0u, lut, d1),
               (int)__builtin_amdgcn_perm(0u, lut, d2), (int)__builtin_amdgcn_perm(0u, lut, d3)};
}
// 16 packed ternary codes (code q + 1 at bits 2k) -> 16 FP4 (E2M1) values,
// value k in nibble k of the 64-bit result (low nibble of each byte first):
// q = -1 -> 0xA (-1.0), 0 -> 0x0, +1 -> 0x2 (+1.0).  Each 8-code half: its
// two bytes to bytes 0 and 2, their nibbles to bytes 0..3, the 2-bit codes
// to nibbles; then nibble = (code bit 1) * 2 + (code == 0) * 0xA.
__device__ __forceinline__ u32x2 expand16_fp4(uint32_t x) {
  auto half = [](uint32_t v) {
    v = (v | (v << 4)) & 0x0F0F0F0Fu;
    const uint32_t u = v | (v << 2);             // codes at nibble bits 0-1 (bits 2-3: junk)
    const uint32_t z = ~u & ~(u >> 1) & 0x11111111u;
    const uint32_t w = z | (z << 2);
    return (u & 0x22222222u) | (w << 1);
  };
  return u32x2{half(__builtin_amdgcn_perm(0u, x, 0x0C010C00u)), half(__builtin_amdgcn_perm(0u, x, 0x0C030C02u))};
}
// Barrier that keeps the compiler from moving memory accesses across it; it
// waits for this wave's LDS accesses but not for outstanding DMA.
__device__ __forceinline__ void block_barrier() {
  __asm__ volatile("" ::: "memory");
  __builtin_amdgcn_s_waitcnt((15) | (3 << 14) | (7 << 4) | (0 << 8));   // lgkmcnt(0)
  __builtin_amdgcn_s_barrier();
  __asm__ volatile("" ::: "memory");
}

// The value x, hidden from the optimiser: per-lane indices derived from it
// are recomputed where they are used instead of being hoisted out of the
// tile loop, where they would hold registers across the main loop.
__device__ __forceinline__ int opaque(int x) {
  __asm__ volatile("" : "+v"(x));
  return x;
}

// Per-thread DMA plan of one operand of one tile: the global address of each
// of its NL chunks at step 0; the reduction offset (elements, within a step)
// the chunks cover, which is the same for all of them; and the distance
// back from a chunk's address to a safe one in the same row (K-contiguous)
// or column (K-major) for loads past the end of the reduction.
template <int MODE, int EB, int KB>
struct Plan {
  using G = Geo<KB>;
  static constexpr int PK = pkb<KB, EB>();
  static constexpr int CH = TILE * PK / 16;   // packed 16-byte chunks per stage
  // packed codes: all threads (32-byte rows), or the first CH threads (16-byte rows)
  static constexpr int NL = MODE == KCP ? (CH >= NTD ? CH / NTD : 1) : MODE == KF4 ? G::NL / 2 : G::NL;
  // K-major: a thread's chunks cover two reduction rows, k and k + KSTEP,
  // when one wave instruction's 8 rows repeat within a region (4 waves)
  static constexpr int KSTEP = MODE == KM && NTD < G::KR * 8 ? NTD / 8 : 0;
  static_assert(KSTEP == 0 || G::KR * 8 == 2 * NTD, "K-major chunks cover at most two reduction rows");
  const uint8_t* g[NL];
  int64_t back;
  int64_t inc;
  int rk;
  // reduction offset of chunk q (elements within the step) and the distance
  // back from it to a safe address
  __device__ int rk_of(int q) const { return rk + (KSTEP && (q & 1) ? KSTEP : 0); }
  __device__ int64_t back_of(int q, int64_t ld) const { return back + (KSTEP && (q & 1) ? KSTEP * ld : 0); }

  __device__ void init(const Opnd& o, int64_t row0, int64_t r_begin, int tid) {
#pragma unroll
    for (int q = 0; q < NL; ++q) {
      const int p = q * NTD + tid;                  // physical 16-byte position
      if constexpr (MODE == KCP) {
        // 32-byte rows: two chunks, swapped on odd groups of 8 rows; 16-byte
        // rows (bf16 steps): one chunk, whose halves the packing arranges
        const int row = PK == 32 ? p >> 1 : p;
        const int c = PK == 32 ? (p & 1) ^ ((row >> 3) & 1) : 0;   // logical 16-byte chunk (64 codes)
        int64_t gr = row0 + row;
        if (gr > o.n - 1) gr = o.n - 1;
        g[q] = o.p + gr * o.ld + r_begin / 4 + 16 * c;
        back = r_begin / 4 + 16 * c;
        rk = 64 * c;
      } else if constexpr (MODE == KF4) {
        // rows of KB / 2 bytes (4 chunks of 32 values), chunk c of row r at
        // position c ^ ((r >> 2) & 3): conflict-free 16-byte reads
        const int row = p >> 2;
        const int c = (p & 3) ^ ((row >> 2) & 3);
        int64_t gr = row0 + row;
        if (gr > o.n - 1) gr = o.n - 1;
        g[q] = o.p + gr * o.ld + r_begin / 2 + 16 * c;
        back = r_begin / 2 + 16 * c;
        rk = 32 * c;
      } else if constexpr (MODE == KC) {
        const int row = p / G::CPR;
        const int c = (p % G::CPR) ^ G::swz(row);   // logical chunk (same for every q)
        int64_t gr = row0 + row;
        if (gr > o.n - 1) gr = o.n - 1;
        g[q] = o.p + gr * o.ld + r_begin * EB + 16 * c;
        back = r_begin * EB + 16 * c;
        rk = 16 * c / EB;
      } else {
        const int region = p / (G::KR * 8);         // 64-column region
        const int k = (p % (G::KR * 8)) >> 3;       // reduction row within the step
        const int pc = p & 7;
        const int seg = (pc >> 1) ^ (k & 3);
        int64_t col = row0 + 64 * region + 16 * seg + 8 * (pc & 1);
        if (col > o.n - 8) col = o.n - 8;
        g[q] = o.p + (r_begin + k) * o.ld + 2 * col;
        if (q == 0) {                               // chunks q > 0: rk_of / back_of
          back = (int64_t)k * o.ld;
          rk = k;
        }
      }
    }
    inc = MODE == KC ? KB : MODE == KCP ? PK : MODE == KF4 ? KB / 2 : G::KR * o.ld;
  }
};

// Tile order within one problem: reduction split bz outermost; within a
// split, bands of kGroupRows tile rows, and within a band column by column
// (problems more than 8 tiles wide; narrower ones stay row-major).  An XCD
// owns a contiguous run of this order, so the 32 tiles its compute units
// hold at once span about 4 tile rows and 8 tile columns, where row-major
// order would span 1-2 rows and 16-32 columns: they share more of their
// operand panels in the XCD's L2 (12 panels per step instead of 18; hidden
// 4096 block: forward -2 %, backward + SR -1.5 %).
#ifndef GEMM_GROUP_ROWS
#define GEMM_GROUP_ROWS 4
#endif
constexpr int kGroupRows = GEMM_GROUP_ROWS;
__host__ __device__ __forceinline__ void tile_coords(int local, int nbx, int nby, int& bx, int& by,
                                                     int& bz) {
  const int per_z = nbx * nby;
  bz = local / per_z;
  const int r = local - bz * per_z;
  const int gr = nbx > 8 ? kGroupRows : 1;
  const int band = r / (gr * nbx);
  const int in = r - band * (gr * nbx);
  const int rows = nby - band * gr < gr ? nby - band * gr : gr;
  by = band * gr + in % rows;
  bx = in / rows;
}

// Tile j of XCD x's list: XCD x owns [x n / 8, (x + 1) n / 8) of every
// problem's n tiles, problems in launch order.  False past the end.
template <class Epi>
__device__ __forceinline__ bool locate(const Group<Epi>& grp, int x, int j, int& g, int& local) {
  for (g = 0; g < grp.ng; ++g) {
    const int n = grp.p[g].ntiles;
    const int s0 = (x * n) >> 3, cnt = (((x + 1) * n) >> 3) - s0;
    if (j < cnt) {
      local = s0 + j;
      return true;
    }
    j -= cnt;
  }
  return false;
}

using lds_f32 = __attribute__((address_space(3))) float;
using lds_u32 = __attribute__((address_space(3))) uint32_t;
using lds_i32 = __attribute__((address_space(3))) int;

// Stage geometry of one instantiation: bytes per stage and stages in flight.
template <int ELEM, int MB, int KB>
struct StageGeo {
  static constexpr int EB = ELEM == EBF16 ? 2 : 1;
  static constexpr int SLOTB = slot_bytes<MB, KB, EB>();
  // as many stages as fit next to the row scales (at most 4)
  static constexpr int NS = 4 * SLOTB + TILE * 4 <= 160 * 1024 ? 4 : 3 * SLOTB + TILE * 4 <= 160 * 1024 ? 3 : 2;
  static constexpr int kBytes = NS * SLOTB;
};

// The persistent grouped GEMM over the tiles of `grp`, with its LDS passed
// in (stages, 256 row factors, a 16-entry code table, the next-tile slot),
// so that two groups can run one after the other in one launch.
template <int ELEM, int MA, int MB, int KB, class Epi>
__device__ __forceinline__ void gemm_v3_body(const Group<Epi>& grp, lds_u8* smem, lds_f32* row_scale,
                                             lds_u32* code_lut, lds_i32* next_tile_p) {
  using G = Geo<KB>;
  static_assert(MB != KCP || KB == 128, "packed codes use 128-byte steps");
  constexpr int EB = ELEM == EBF16 ? 2 : 1;
  constexpr int BK = KB / EB;               // reduction elements per step
  constexpr int OPB = G::OPB;
  constexpr int NL = G::NL;
  constexpr int SLOTB = StageGeo<ELEM, MB, KB>::SLOTB;
  constexpr int PKB = pkb<KB, EB>();
  constexpr int NLB = Plan<MB, EB, KB>::NL;  // DMA chunks per thread for B
  constexpr int NS = StageGeo<ELEM, MB, KB>::NS;
  static_assert(NW * 32 * 128 <= SLOTB, "epilogue staging (32 rows of 128 bytes per wave) fits in one stage");
  constexpr int LPS = NL + NLB;            // DMA instructions per thread per stage (at most)
  // (measured faster for the int8 forward, dX and dW; the e4m3 forward keeps
  // the burst after the barrier)
  constexpr bool kSplitCopies = ELEM != EF8 && ELEM != EF4B;
  static_assert(ELEM != EF4B || MB == KCP || MB == KF4, "FP4 B comes from ternary codes");
  static_assert(MB != KF4 || (ELEM == EF4B && KB == 128), "KF4 holds FP4 B of 128-element steps");
  // bf16 operand from packed codes: two codes (a nibble) -> two bf16 by table
  constexpr bool kLutB = MB == KCP && ELEM == EBF16;

  const int tid = threadIdx.x;
  const int lane = tid & 63;
  const int wave = tid >> 6;
  const int wi = wave / WGC, wj = wave % WGC;
  const int h = lane >> 5;
  const int wave_u = __builtin_amdgcn_readfirstlane(wave);
  // packed B rows of 16 bytes need only the first CH threads' copies
  constexpr int kChB = Plan<MB, EB, KB>::CH;
  const bool b_copies = MB != KCP || kChB >= NTD || wave_u * 64 < kChB;
  const int lps = NL + (b_copies ? NLB : 0);   // this wave's copies per stage
  if constexpr (kLutB) {
    if (tid < 16) {   // entry n: codes (n & 3, n >> 2) -> bf16 (code - 1), low half first
      const uint32_t lo = (uint32_t)((0x00003F800000BF80ull >> (16u * (tid & 3))) & 0xFFFFu);
      const uint32_t hi = (uint32_t)((0x00003F800000BF80ull >> (16u * (tid >> 2))) & 0xFFFFu);
      code_lut[tid] = lo | (hi << 16);
    }
  }
  const int xcd = blockIdx.x & 7;

  // ---- state of the tile being computed
  struct TileState {
    int g;
    int64_t i0, j0, rlen;
    int bz, nsteps;
    bool tail;
  };
  Plan<MA, EB, KB> pa;
  Plan<MB, EB, KB> pb;
  TileState cur;
  float my_scale = 0.0f;

  auto setup = [&](int g, int local, TileState& T) {
    const Prob<Epi>& P = grp.p[g];
    int bx, by, bz;
    tile_coords(local, P.nbx, P.nby, bx, by, bz);
    T.g = g;
    T.i0 = (int64_t)by * TILE;
    T.j0 = (int64_t)bx * TILE;
    T.bz = bz;
    const int64_t r_begin = (int64_t)bz * P.split_len;
    int64_t r_end = r_begin + P.split_len;
    if (r_end > P.R) r_end = P.R;
    T.rlen = r_end > r_begin ? r_end - r_begin : 0;
    T.nsteps = (int)((T.rlen + BK - 1) / BK);
    T.tail = (T.rlen % BK) != 0;
    const int tid_s = opaque(tid);
    pa.init(P.A, T.i0, r_begin, tid_s);
    pb.init(P.B, T.j0, r_begin, tid_s);
    if constexpr (Epi::kRowScale) {
      if (tid < TILE) {
        int64_t i = T.i0 + tid;
        if (i > P.I - 1) i = P.I - 1;
        my_scale = P.epi.scale_raw(i);     // used only in the epilogue
      }
    }
  };

  // DMA of step s of the current plans into stage `slot`.
  auto issue = [&](int s, int slot, const TileState& T) {
    lds_u8* la = smem + slot * SLOTB + wave_u * 1024;
    lds_u8* lb = la + OPB;
    if (!(T.tail && s == T.nsteps - 1)) {
#pragma unroll
      for (int q = 0; q < NL; ++q) dma16(pa.g[q] + (int64_t)s * pa.inc, la + q * (NTD * 16));
      if (b_copies)
#pragma unroll
        for (int q = 0; q < NLB; ++q) dma16(pb.g[q] + (int64_t)s * pb.inc, lb + q * (NTD * 16));
    } else {
      const int64_t rbase = (int64_t)s * BK;
      const Prob<Epi>& P = grp.p[T.g];
#pragma unroll
      for (int q = 0; q < NL; ++q) {
        const bool o = rbase + pa.rk_of(q) >= T.rlen;
        dma16(o ? pa.g[q] - pa.back_of(q, P.A.ld) : pa.g[q] + (int64_t)s * pa.inc, la + q * (NTD * 16));
      }
      if (b_copies)
#pragma unroll
        for (int q = 0; q < NLB; ++q) {
          const bool o = rbase + pb.rk_of(q) >= T.rlen;
          dma16(o ? pb.g[q] - pb.back_of(q, P.B.ld) : pb.g[q] + (int64_t)s * pb.inc, lb + q * (NTD * 16));
        }
    }
  };
  // zero the chunks this thread loaded past the end of the reduction (its
  // own DMA for that stage has completed)
  // (packed B codes past the end need no zeroing: they meet zeroed A)
  auto zero_tail = [&](int s, int slot, const TileState& T) {
    const int dtid = tid;
    lds_u8* la = smem + slot * SLOTB;
    lds_u8* lb = la + OPB;
    const int64_t rbase = (int64_t)s * BK;
    const i32x4 z = {0, 0, 0, 0};
#pragma unroll
    for (int q = 0; q < NL; ++q)
      if (rbase + pa.rk_of(q) >= T.rlen) *(__attribute__((address_space(3))) i32x4*)(la + (q * NTD + dtid) * 16) = z;
    // (packed codes and FP4 values past the end need no zeroing: they meet
    // zeroed A, and neither holds a NaN or an infinity)
    if constexpr (MB != KCP && MB != KF4)
#pragma unroll
      for (int q = 0; q < NL; ++q)
        if (rbase + pb.rk_of(q) >= T.rlen) *(__attribute__((address_space(3))) i32x4*)(lb + (q * NTD + dtid) * 16) = z;
  };

  using AccV = typename AccT<ELEM == EI8 ? Mfma::I8 : Mfma::BF16>::type;
  AccV acc[WI][WJ];

  // fragment address parts
  const int frow = lane & 31;
  const int t4 = (lane >> 2) & 3, u4 = lane & 3, ch = (lane >> 4) & 1;

  // Fragments of one reduction sub-step kk (0..3; 32 bytes of reduction per
  // tile row): K-contiguous ones by ds_read_b128, K-major ones by two
  // transposing reads (inline asm, waited for by frag_wait).
  struct Frags {
    i32x4 fa[WI], fb[WJ];
    u32x2 ka[WI][2], kb[WJ][2];
    uint32_t pb[WJ];          // packed codes (16 per lane), expanded at use
  };
  // pk: bf16 steps from packed codes, this lane's 64 bits of each B row
  // (sub-step kk in bits 16 kk .. 16 kk + 15, read once per step).
  // pq: 8-bit steps from packed codes, this lane's 16-byte half of each B
  // row (64 codes, read once per step; sub-step kk in word kk).  Lane half h
  // then takes reduction elements 64 h .. 64 h + 63 of the step, sub-step kk
  // the 16 from 64 h + 16 kk, and its A chunks follow the same order: chunk
  // 4 h + kk instead of 2 kk + h.  (One 16-byte read per row half is free of
  // bank conflicts; four 4-byte reads of words 2 kk + h, all lanes at one
  // word offset in 32-byte rows, conflicted 4-way and cost the e4m3 forward
  // 9 %.)
  constexpr bool kPq = MB == KCP && !kLutB;
  auto read_frags = [&](const lds_u8* la, const lds_u8* lb, int kk, Frags& F, const u32x2* pk,
                        const i32x4* pq) {
#pragma unroll
    for (int t = 0; t < WI; ++t) {
      if constexpr (MA == KC) {
        const int row = wi * 32 * WI + t * 32 + frow;
        const int c = (kPq ? 4 * h + kk : 2 * kk + h) ^ G::swz(row);
        F.fa[t] = *(const __attribute__((address_space(3))) i32x4*)(la + row * KB + 16 * c);
      } else {
        const int col = wi * 32 * WI + t * 32 + 16 * ch + 4 * u4;
        const int seg = ((col & 63) >> 4) ^ t4;
        const int a0 = (col >> 6) * (G::KR * 128) + (16 * kk + 8 * h + t4) * 128 + 32 * seg + 8 * u4;
        F.ka[t][0] = tr_read(la, a0);
        F.ka[t][1] = tr_read(la, a0 + 512);
      }
    }
#pragma unroll
    for (int t = 0; t < WJ; ++t) {
      if constexpr (kLutB) {
        const uint32_t x16 = (pk[t][kk >> 1] >> (16 * (kk & 1))) & 0xFFFFu;
#pragma unroll
        for (int i = 0; i < 4; ++i) F.fb[t][i] = (int)code_lut[(x16 >> (4 * i)) & 0xFu];
      } else if constexpr (MB == KCP) {
        F.pb[t] = (uint32_t)pq[t][kk];
      } else if constexpr (MB == KF4) {
        // the FP4 operand of sub-step pair m = kk / 2 (read with its even
        // sub-step): lane half h takes the row's 32 values from 64 m + 32 h,
        // which are the elements its e4m3 partner lanes pair them with
        if ((kk & 1) == 0) {
          const int row = wj * 32 * WJ + t * 32 + frow;
          const int c = (kk + h) ^ ((row >> 2) & 3);
          F.fb[t] = *(const __attribute__((address_space(3))) i32x4*)(lb + row * (KB / 2) + 16 * c);
        }
      } else if constexpr (MB == KC) {
        const int row = wj * 32 * WJ + t * 32 + frow;
        const int c = (2 * kk + h) ^ G::swz(row);
        F.fb[t] = *(const __attribute__((address_space(3))) i32x4*)(lb + row * KB + 16 * c);
      } else {
        const int col = wj * 32 * WJ + t * 32 + 16 * ch + 4 * u4;
        const int seg = ((col & 63) >> 4) ^ t4;
        const int a0 = (col >> 6) * (G::KR * 128) + (16 * kk + 8 * h + t4) * 128 + 32 * seg + 8 * u4;
        F.kb[t][0] = tr_read(lb, a0);
        F.kb[t][1] = tr_read(lb, a0 + 512);
      }
    }
  };
  auto opa = [&](const Frags& F, int t) { return MA == KC ? F.fa[t] : join(F.ka[t][0], F.ka[t][1]); };
  auto opb = [&](const Frags& F, int t) {
    if constexpr (kLutB) return F.fb[t];
    else if constexpr (MB == KCP) return expand16(F.pb[t], ELEM == EF8 ? 0x003800B8u : 0x000100FFu);
    else return MB == KC || MB == KF4 ? F.fb[t] : join(F.kb[t][0], F.kb[t][1]);
  };
  // MFMAs of one sub-step (int8 / bf16), or of two sub-steps (e4m3, whose
  // instruction reduces 64 elements: sub-step pairs (0, 1) and (2, 3)).
  auto mfma1 = [&](const Frags& F) {
#pragma unroll
    for (int ta = 0; ta < WI; ++ta)
#pragma unroll
      for (int tb = 0; tb < WJ; ++tb) {
        if constexpr (ELEM == EI8)
          acc[ta][tb] = __builtin_amdgcn_mfma_i32_32x32x32_i8(opb(F, tb), opa(F, ta), acc[ta][tb], 0, 0, 0);
        else if constexpr (Epi::kTrans)   // lanes hold four consecutive rows of one column
          acc[ta][tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, opa(F, ta)),
                                                                __builtin_bit_cast(bf16x8, opb(F, tb)),
                                                                acc[ta][tb], 0, 0, 0);
        else
          acc[ta][tb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(__builtin_bit_cast(bf16x8, opb(F, tb)),
                                                                __builtin_bit_cast(bf16x8, opa(F, ta)),
                                                                acc[ta][tb], 0, 0, 0);
      }
  };
  auto mfma2 = [&](const Frags& F0, const Frags& F1) {
#pragma unroll
    for (int ta = 0; ta < WI; ++ta)
#pragma unroll
      for (int tb = 0; tb < WJ; ++tb) {
        const i32x4 a0 = opa(F0, ta), a1 = opa(F1, ta), b0 = opb(F0, tb), b1 = opb(F1, tb);
        const i32x8 av = {a0[0], a0[1], a0[2], a0[3], a1[0], a1[1], a1[2], a1[3]};
        const i32x8 bv = {b0[0], b0[1], b0[2], b0[3], b1[0], b1[1], b1[2], b1[3]};
        if constexpr (ELEM == EF4B && MB == KF4) {
          // FP4 B from the workspace, already in the instruction's order
          const i32x4 f = F0.fb[tb];
          const i32x8 bv4 = {f[0], f[1], f[2], f[3], 0, 0, 0, 0};
          acc[ta][tb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bv4, av, acc[ta][tb], 4, 0, 0, 127, 0, 127);
        } else if constexpr (ELEM == EF4B) {
          // B as FP4 (format 4: 32 values in the first four registers), A
          // e4m3 (format 0), unit E8M0 scales (127 = 2^0).  With FP4 the
          // first operand's lane half h holds reduction elements 16 h ..
          // 16 h + 15 and 32 + 16 h .. 32 + 16 h + 15 of the instruction
          // (the e4m3 operand: 32 h .. 32 h + 31).  The A chunks cover
          // elements 64 h' + 32 m .. + 31 of the step (m: the sub-step
          // pair), so half h takes the codes of word 2 m + h from both lane
          // halves: one swap of the halves' upper and lower lanes gives
          // them (lanes 0-31 keep their word 2 m and get word 2 m of lanes
          // 32-63, which keep word 2 m + 1 and get that of lanes 0-31).
          const auto sw = __builtin_amdgcn_permlane32_swap(F0.pb[tb], F1.pb[tb], false, false);
          const u32x2 f0 = expand16_fp4(sw[0]), f1 = expand16_fp4(sw[1]);
          const i32x8 bv4 = {(int)f0[0], (int)f0[1], (int)f1[0], (int)f1[1], 0, 0, 0, 0};
          acc[ta][tb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bv4, av, acc[ta][tb], 4, 0, 0, 127, 0, 127);
        } else {
          // both operands e4m3 (format 0), unit E8M0 scales (127 = 2^0)
          acc[ta][tb] = __builtin_amdgcn_mfma_scale_f32_32x32x64_f8f6f4(bv, av, acc[ta][tb], 0, 0, 0, 127, 0, 127);
        }
      }
  };
  auto stage_ptr = [&](int slot) { return smem + slot * SLOTB; };

  // ---- persistent loop over this block's tiles (the counters were cleared
  // by sched_clear_kernel just before this launch)
  lds_i32& next_tile = *next_tile_p;
  int* const next_ctr = grp.sched + xcd;
  if (tid == 0) next_tile = atomicAdd(next_ctr, 1);
  __syncthreads();
  int g0, local0;
  if (!locate(grp, xcd, next_tile, g0, local0)) return;
  setup(g0, local0, cur);
  // Stage of step s of the current tile: (slot0 + s) mod NS.  Before a tile
  // starts, its steps 0 .. NS-2 are in flight.
  int slot0 = 0;
  for (int s = 0; s < NS - 1 && s < cur.nsteps; ++s) issue(s, s, cur);

  // One step from stage `slot`: sub-step kk+1's fragments load while kk's
  // MFMAs run (e4m3: sub-steps are consumed in pairs).
  auto compute = [&](int slot, auto&& mid) {
    const lds_u8* la = stage_ptr(slot);
    const lds_u8* lb = la + OPB;
    // (scheduling barriers keep each group of reads ahead of the MFMAs that
    // precede their use; left alone, the compiler sinks every read next to
    // its first use and exposes the LDS latency)
    u32x2 pk[WJ];
    if constexpr (kLutB) {
#pragma unroll
      for (int t = 0; t < WJ; ++t) {
        // the packing swaps the two 8-byte halves of rows with bit 4 set
        const int row = wj * 32 * WJ + t * 32 + frow;
        pk[t] = *(const __attribute__((address_space(3))) u32x2*)(lb + row * 16 + 8 * (h ^ ((row >> 4) & 1)));
      }
    }
    // (the DMA stores logical 16-byte half c of row r at half c ^ ((r >> 3) & 1))
    i32x4 pq[WJ];
    if constexpr (kPq) {
#pragma unroll
      for (int t = 0; t < WJ; ++t) {
        const int row = wj * 32 * WJ + t * 32 + frow;
        pq[t] = *(const __attribute__((address_space(3))) i32x4*)(lb + row * PKB + 16 * (h ^ ((row >> 3) & 1)));
      }
    }
    Frags F0, F1;
    if constexpr (ELEM != EF8 && ELEM != EF4B) {
      read_frags(la, lb, 0, F0, pk, pq);
      read_frags(la, lb, 1, F1, pk, pq);
      __builtin_amdgcn_sched_barrier(0);
      mfma1(F0);
      __builtin_amdgcn_sched_barrier(0);
      mid();
      __builtin_amdgcn_sched_barrier(0);
      if constexpr (G::NKK == 4) {
        read_frags(la, lb, 2, F0, pk, pq);
        __builtin_amdgcn_sched_barrier(0);
        mfma1(F1);
        __builtin_amdgcn_sched_barrier(0);
        read_frags(la, lb, 3, F1, pk, pq);
        __builtin_amdgcn_sched_barrier(0);
        mfma1(F0);
        __builtin_amdgcn_sched_barrier(0);
      }
      mfma1(F1);
    } else {
      // (e4m3 keeps the compiler's own order: a pair of sub-steps per
      // instruction leaves no registers for a further pair in flight)
      read_frags(la, lb, 0, F0, pk, pq);
      read_frags(la, lb, 1, F1, pk, pq);
      if constexpr (G::NKK == 4) {
        Frags F2, F3;
        read_frags(la, lb, 2, F2, pk, pq);
        mfma2(F0, F1);
        mid();
        read_frags(la, lb, 3, F3, pk, pq);
        mfma2(F2, F3);
      } else {
        mfma2(F0, F1);
        mid();
      }
    }
  };

  // vector stores one thread issues in an epilogue (every chunk is stored;
  // chunks outside the output go to a dummy slot in the workspace)
  constexpr int kStoresBf16 = WI * 32 * (32 * WJ * 2 / 16) / 64;
  constexpr int kStoresF32 = WI * 32 * (32 * WJ * 4 / 16) / 64;
  constexpr int kStoresSR = WI * WJ * 2;      // two 8-weight code chunks per 32 x 32 block
  // the wave's vmcnt counts at most 63 operations in flight (the wave waits
  // at issue beyond that), so "at most 63 newer" is a correct, if
  // conservative, wait when more were issued
  constexpr int kVmMax = 63;
  static_assert(NS * LPS < kVmMax, "vmcnt range");
  uint8_t* const dummy = reinterpret_cast<uint8_t*>(grp.sched) + 128;
  bool first_tile = true;
  int stores_prev = 0;                 // stores per thread of the previous epilogue
  // SR epilogue: changed and non-finite counts of each wave, kept in LDS
  // (the row-scale area, which that epilogue does not use) so that nothing
  // extra stays live in registers across the main loop
  lds_u32* const sr_cnt = (lds_u32*)row_scale;
  if constexpr (Epi::kSR) {
    if (lane == 0) {
      sr_cnt[2 * wave_u] = 0;
      sr_cnt[2 * wave_u + 1] = 0;
    }
  }
  for (;;) {
    int fetched = 0;                   // thread 0: index of the next tile
#pragma unroll
    for (int a = 0; a < WI; ++a)
#pragma unroll
      for (int b = 0; b < WJ; ++b)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[a][b][r] = 0;

    // main loop: step it computes from stage (slot0 + it) mod NS while the
    // next NS - 1 steps load into the other stages.  The first step of a
    // tile waits for every load and store of this thread (the previous
    // epilogue's stores were issued after this tile's first stages).
    for (int it = 0; it < cur.nsteps; ++it) {
      const int slot = (slot0 + it) % NS;
      if (it == 0) {
        // step 0's loads were issued before the previous epilogue's stores
        // (a fixed number per thread), which may stay in flight, as may the
        // tile's later prefetched steps
        const int ahead = (cur.nsteps < NS - 1 ? cur.nsteps : NS - 1) - 1;
        int n = ahead * lps + (first_tile ? 0 : stores_prev);
        if (n > kVmMax) n = kVmMax;
        wait_vm_le<kVmMax>(__builtin_amdgcn_readfirstlane(n));
        first_tile = false;
      } else {
        // copies of steps it + 1 .. it + NS - 2 (those issued) may stay in flight
        const int newer = cur.nsteps - 1 - it < NS - 2 ? cur.nsteps - 1 - it : NS - 2;
        if constexpr (NS == 2) wait_vm<0>();
        else wait_vm_le<(NS - 2) * LPS>(__builtin_amdgcn_readfirstlane(newer * lps));
      }
      if (cur.tail && it == cur.nsteps - 1) zero_tail(it, slot, cur);
      block_barrier();                 // stage `slot` complete; step it - 1's stage is free
      // The two waves of a SIMD take turns: the first half of the waves
      // issues its copies right after the barrier, the other half after its
      // first group of MFMAs, so each SIMD has one wave issuing MFMAs while
      // the other waits for its copies to be taken.
      const bool copy_now = !kSplitCopies || wave_u < NW / 2;
      if (copy_now && it + NS - 1 < cur.nsteps) issue(it + NS - 1, (slot + NS - 1) % NS, cur);
      // fetch the next tile early; its value is needed only at the epilogue
      if (it == 0 && tid == 0) fetched = atomicAdd(next_ctr, 1);
      compute(slot, [&]() {
        if (!copy_now && it + NS - 1 < cur.nsteps) issue(it + NS - 1, (slot + NS - 1) % NS, cur);
      });
    }

    // epilogue parameters of this tile, then the next tile's first stage
    const Prob<Epi>& P = grp.p[cur.g];
    const Epi epi = P.epi;
    const int64_t I = P.I, J = P.J;
    const int64_t i0 = cur.i0, j0 = cur.j0;
    const int bz = cur.bz;
    const int last = (slot0 + cur.nsteps + NS - 1) % NS;   // stage of the last step (staging area)
    if constexpr (Epi::kRowScale) {
      if (tid < TILE) row_scale[tid] = epi.scale_fin(my_scale);
    }
    // SR epilogue: this lane's code chunks, rows sr_r + 16 u of each 32-row
    // block and columns 8 sr_c .. 8 sr_c + 7 of each 32-column block (8
    // weights per chunk: one Philox block, since d_in is a multiple of 8).
    // Loaded here, after the main loop, and waited for before the next
    // tile's copies are issued, so the wait drains nothing else.
    const int sr_r = lane >> 2, sr_c = lane & 3;
    // ternary: both chunks of a 32 x 32 block in one register (u = 0 low
    // half); int8: two words per chunk
    [[maybe_unused]] uint32_t srt[Epi::kSR ? WI : 1][Epi::kSR ? WJ : 1];
    [[maybe_unused]] uint32_t sr8[Epi::kSR && !Epi::kTern ? WI : 1][Epi::kSR && !Epi::kTern ? WJ : 1][2][2];
    auto sr_pos = [&](int ta, int tb, int u, int64_t& n, int64_t& k) {
      if constexpr (Epi::kTrans) {
        // block (ta, tb) of dW^T holds dW rows j0 + .. + 32 tb (d_out) and
        // columns i0 + .. + 32 ta (d_in), laid out as a block of dW
        n = j0 + wj * 32 * WJ + tb * 32 + sr_r + 16 * u;
        k = i0 + wi * 32 * WI + ta * 32 + 8 * sr_c;
        return n < J && k < I;
      } else {
        n = i0 + wi * 32 * WI + ta * 32 + sr_r + 16 * u;
        k = j0 + wj * 32 * WJ + tb * 32 + 8 * sr_c;
        return n < I && k < J;
      }
    };
    if constexpr (Epi::kSR) {
#pragma unroll
      for (int ta = 0; ta < WI; ++ta)
#pragma unroll
        for (int tb = 0; tb < WJ; ++tb)
#pragma unroll
          for (int u = 0; u < 2; ++u) {
            int64_t n, k;
            const bool ok = sr_pos(ta, tb, u, n, k);
            if constexpr (Epi::kTern) {
              const uint8_t* src = ok ? epi.wq + n * epi.ldc + (k >> 2) : dummy;
              const uint32_t v = *reinterpret_cast<const uint16_t*>(src);
              if (u == 0) srt[ta][tb] = v;
              else srt[ta][tb] |= v << 16;
            } else if constexpr (Epi::kCF == CF_I4) {
              const uint8_t* src = ok ? epi.wq + n * epi.ldc + (k >> 1) : dummy;
              sr8[ta][tb][u][0] = *reinterpret_cast<const uint32_t*>(src);
              sr8[ta][tb][u][1] = 0;
            } else if constexpr (Epi::kCF == CF_I3) {
              // three bytes (k / 8 chunks of 3 bytes into the row)
              uint32_t w[4];
              ChunkIO<CF_I3>::load(ok ? epi.wq + n * epi.ldc : dummy, ok ? (k >> 3) : 0, w);
              sr8[ta][tb][u][0] = w[0];
              sr8[ta][tb][u][1] = 0;
            } else {
              const uint8_t* src = ok ? epi.wq + n * epi.ldc + k : dummy;
              const uint2 v = *reinterpret_cast<const uint2*>(src);
              sr8[ta][tb][u][0] = v.x;
              sr8[ta][tb][u][1] = v.y;
            }
          }
    }
    if (tid == 0) next_tile = cur.nsteps > 0 ? fetched : atomicAdd(next_ctr, 1);
    block_barrier();                   // every wave is done with every stage
    int gn, localn;
    const bool more = locate(grp, xcd, next_tile, gn, localn);
    if constexpr (Epi::kSR) wait_vm<0>();   // the codes (nothing else is in flight)
    if (more) {
      const int slotn = (last + 1) % NS;      // the next tile's stages avoid `last`
      setup(gn, localn, cur);
      for (int s = 0; s < NS - 1 && s < cur.nsteps; ++s) issue(s, (slotn + s) % NS, cur);
      slot0 = slotn;
    }

    // The MFMAs take the B fragment as their first operand, so lane
    // (j = lane mod 32, h) of block (ta, tb) holds row 32 ta + j, columns
    // 32 tb + 8 (r / 4) + 4 h + (r mod 4), r = 0..15: four consecutive
    // columns per group of four entries.  Each wave stages 32 rows of 128
    // bytes at a time in its own part of stage `last` (bf16: both column
    // blocks of a pair; fp32: one column block), 16-byte chunk c of row
    // r at chunk c ^ ((r >> 1) & 7), then writes whole 16-byte chunks of
    // output rows.
    const int lane_e = opaque(lane), h_e = lane_e >> 5, j_e = lane_e & 31;
    lds_u8* stage = smem + last * SLOTB + wave * (32 * 128);
    const bool obf = epi.out_bf16();
    const int sw_w = (j_e >> 1) & 7;
    const int rd_row = lane_e >> 3, rd_chunk = lane_e & 7;
    // one row block (32 rows of the wave): its values in LDS, then its rows
    auto epi_block = [&](int ta, auto ebytes_tag) {
      constexpr int EBY = decltype(ebytes_tag)::value;
      const float sc = Epi::kRowScale ? row_scale[wi * 32 * WI + ta * 32 + j_e] : epi.scale(0);
      auto value = [&](int tb, int r) {
        float v;
        if constexpr (ELEM == EI8) v = (float)acc[ta][tb][r];
        else v = acc[ta][tb][r];
        return v * sc;
      };
      // stores the staged 32 x 128 bytes: columns from `col0` (elements)
      // (every lane stores every time, chunks outside the output to a dummy
      // slot, so the number of stores in flight is known)
      auto store_staged = [&](int col0) {
        __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        const int64_t jj = j0 + wj * 32 * WJ + col0 + rd_chunk * (16 / EBY);
        const int rows_left = (int)__builtin_amdgcn_readfirstlane(
            (int)(I - (i0 + wi * 32 * WI + ta * 32) < 32 ? I - (i0 + wi * 32 * WI + ta * 32) : 32));
        uint8_t* const p0 = epi.row(i0 + wi * 32 * WI + ta * 32 + rd_row, bz) + jj * EBY;
        const int64_t rstride = 8 * epi.row_bytes();
        const bool col_ok = jj < J;
#pragma unroll
        for (int u = 0; u < 4; ++u) {
          const int row = rd_row + 8 * u;
          const i32x4 d = *(const __attribute__((address_space(3))) i32x4*)(
              stage + row * 128 + ((rd_chunk ^ ((row >> 1) & 7)) << 4));
          uint8_t* dst = (col_ok && row < rows_left) ? p0 + u * rstride : dummy;
          *reinterpret_cast<i32x4*>(dst) = d;
        }
        __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      };
      if constexpr (EBY == 2) {
#pragma unroll
        for (int tp = 0; tp < WJ / 2; ++tp) {
#pragma unroll
          for (int t2 = 0; t2 < 2; ++t2)
#pragma unroll
            for (int k = 0; k < 4; ++k) {
              const int tb = 2 * tp + t2;
              const u32x2 w = {pack_bf16x2(value(tb, 4 * k), value(tb, 4 * k + 1)),
                               pack_bf16x2(value(tb, 4 * k + 2), value(tb, 4 * k + 3))};
              *(__attribute__((address_space(3))) u32x2*)(
                  stage + j_e * 128 + (((4 * t2 + k) ^ sw_w) << 4) + 8 * h_e) = w;
            }
          store_staged(64 * tp);
        }
      } else {
#pragma unroll
        for (int tb = 0; tb < WJ; ++tb) {
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const f32x4 w = {value(tb, 4 * k), value(tb, 4 * k + 1), value(tb, 4 * k + 2), value(tb, 4 * k + 3)};
            *(__attribute__((address_space(3))) f32x4*)(stage + j_e * 128 + (((2 * k + h_e) ^ sw_w) << 4)) = w;
          }
          store_staged(32 * tb);
        }
      }
    };
    if constexpr (Epi::kSR) {
      // each 32 x 32 block of dW staged in LDS as fp32, then read back as
      // two chunks of 8 consecutive entries of a row per lane, which update
      // their 8 codes; out-of-range chunks count nothing and store their
      // codes to the dummy slot (a fixed number of stores per thread)
      SRArgs sa;
      sa.c = epi.c;
      sa.L = epi.L;
      sa.qmin = epi.qmin;
      sa.qmax = epi.qmax;
      sa.k0 = epi.k0;
      sa.k1 = epi.k1;
      sa.step = epi.step;
      sa.tid = epi.tid;
      uint32_t tc = 0, tn = 0;   // this tile's counts
      // 32 rows x 64 columns (both column blocks of a row block) per wave:
      // two 32 x 128-byte areas, laid out as the fp32 staging above
      static_assert(NW * 32 * 256 <= SLOTB, "SR staging (32 rows of 256 bytes per wave) fits in one stage");
      lds_u8* const st2 = smem + last * SLOTB + wave * (32 * 256);
#pragma unroll
      for (int ta = 0; ta < WI; ++ta) {
#pragma unroll
        for (int tb = 0; tb < WJ; ++tb)
#pragma unroll
          for (int k = 0; k < 4; ++k) {
            const f32x4 w = {(float)acc[ta][tb][4 * k], (float)acc[ta][tb][4 * k + 1],
                             (float)acc[ta][tb][4 * k + 2], (float)acc[ta][tb][4 * k + 3]};
            *(__attribute__((address_space(3))) f32x4*)(st2 + tb * (32 * 128) + j_e * 128 +
                                                          (((2 * k + h_e) ^ sw_w) << 4)) = w;
          }
        __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
        // the row block's 2 WJ chunks from LDS, one at a time (not
        // unrolled: short code, few live registers)
#pragma unroll 1
        for (int cq = 0; cq < 2 * WJ; ++cq) {
          const int tb = cq >> 1, u = cq & 1;
          const int row = sr_r + 16 * u;
          const int sw = (row >> 1) & 7;
          const lds_u8* sb = st2 + tb * (32 * 128) + row * 128;
          f32x4 gv[2];
          gv[0] = *(const __attribute__((address_space(3))) f32x4*)(sb + (((2 * sr_c) ^ sw) << 4));
          gv[1] = *(const __attribute__((address_space(3))) f32x4*)(sb + (((2 * sr_c + 1) ^ sw) << 4));
          int64_t n, k;
          const bool ok = sr_pos(ta, tb, u, n, k);
          uint32_t win[4] = {0u, 0u, 0u, 0u};
          if constexpr (Epi::kTern) {
            uint32_t w2 = srt[ta][0];
#pragma unroll
            for (int t = 1; t < WJ; ++t) w2 = tb == t ? srt[ta][t] : w2;
            win[0] = (w2 >> (16 * u)) & 0xFFFFu;
          } else {
            uint32_t x0 = sr8[ta][0][0][0], x1 = sr8[ta][0][0][1];
#pragma unroll
            for (int t = 0; t < WJ; ++t)
#pragma unroll
              for (int v = 0; v < 2; ++v)
                if (cq == 2 * t + v) {
                  x0 = sr8[ta][t][v][0];
                  x1 = sr8[ta][t][v][1];
                }
            win[0] = x0;
            win[1] = x1;
          }
          uint32_t wout[4];
          uint32_t ch = 0, nf = 0;
          sr_chunk<Epi::kCF, 8>(win, gv, (uint64_t)(n * epi.d_in + k) >> 3, sa, wout, ch, nf);
          if (ok) {
            tc += ch;
            tn += nf;
          }
          if constexpr (Epi::kTern) {
            uint8_t* dst = ok ? epi.wq + n * epi.ldc + (k >> 2) : dummy;
            *reinterpret_cast<uint16_t*>(dst) = (uint16_t)wout[0];
          } else if constexpr (Epi::kCF == CF_I4) {
            uint8_t* dst = ok ? epi.wq + n * epi.ldc + (k >> 1) : dummy;
            *reinterpret_cast<uint32_t*>(dst) = wout[0];
          } else if constexpr (Epi::kCF == CF_I3) {
            // (three single-byte stores: the vmcnt accounting above counts
            // one per chunk, a lower bound, which only makes waits stricter)
            ChunkIO<CF_I3>::store(ok ? epi.wq + n * epi.ldc : dummy, ok ? (k >> 3) : 0, wout);
          } else {
            uint8_t* dst = ok ? epi.wq + n * epi.ldc + k : dummy;
            *reinterpret_cast<uint2*>(dst) = make_uint2(wout[0], wout[1]);
          }
        }
        __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
      }
      tc = wave_sum_u32(tc);
      tn = wave_sum_u32(tn);
      if (lane == 0) {
        sr_cnt[2 * wave_u] += tc;
        sr_cnt[2 * wave_u + 1] += tn;
      }
      stores_prev = kStoresSR;
    } else {
      if (obf) {
#pragma unroll
        for (int ta = 0; ta < WI; ++ta) epi_block(ta, std::integral_constant<int, 2>{});
      } else {
#pragma unroll
        for (int ta = 0; ta < WI; ++ta) epi_block(ta, std::integral_constant<int, 4>{});
      }
      stores_prev = obf ? kStoresBf16 : kStoresF32;
    }
    if (!more) break;
    // a tile without reduction steps has no main-loop barrier before the
    // next epilogue reuses the staging area and the row scales
    if (cur.nsteps == 0) block_barrier();
  }
  if constexpr (Epi::kSR) {
    unsigned long long* const cnt = grp.p[0].epi.counters;
    if (cnt != nullptr && lane == 0) {
      const unsigned long long c = sr_cnt[2 * wave_u], f = sr_cnt[2 * wave_u + 1];
      if (c) atomicAdd(cnt, c);
      if (f) atomicAdd(cnt + 1, f);
    }
  }
}

template <int ELEM, int MA, int MB, int KB, class Epi>
__global__ __launch_bounds__(NTH) void gemm_v3_kernel(const Group<Epi> grp) {
  __shared__ __attribute__((aligned(1024))) uint8_t stages[StageGeo<ELEM, MB, KB>::kBytes];
  __shared__ float row_scale[TILE];
  __shared__ uint32_t code_lut[16];
  __shared__ int next_tile;
  gemm_v3_body<ELEM, MA, MB, KB, Epi>(grp, (lds_u8*)stages, (lds_f32*)row_scale, (lds_u32*)code_lut,
                                       (lds_i32*)&next_tile);
}

// Two groups in one launch: every block takes tiles of the first group until
// its lists are empty, then tiles of the second, so blocks left without a
// tile of the first start on the second at once.
template <int E1, int MA1, int MB1, int KB1, class Epi1, int E2, int MA2, int MB2, int KB2, class Epi2>
__global__ __launch_bounds__(NTH) void gemm_v3_dual_kernel(const Group<Epi1> g1, const Group<Epi2> g2) {
  constexpr int B1 = StageGeo<E1, MB1, KB1>::kBytes, B2 = StageGeo<E2, MB2, KB2>::kBytes;
  __shared__ __attribute__((aligned(1024))) uint8_t stages[B1 > B2 ? B1 : B2];
  __shared__ float row_scale[TILE];
  __shared__ uint32_t code_lut[16];
  __shared__ int next_tile;
  gemm_v3_body<E1, MA1, MB1, KB1, Epi1>(g1, (lds_u8*)stages, (lds_f32*)row_scale, (lds_u32*)code_lut,
                                         (lds_i32*)&next_tile);
  __syncthreads();
  gemm_v3_body<E2, MA2, MB2, KB2, Epi2>(g2, (lds_u8*)stages, (lds_f32*)row_scale, (lds_u32*)code_lut,
                                         (lds_i32*)&next_tile);
}

}  // namespace v3
}  // namespace dqt

// ------------------------------------------------------------ pre-passes
namespace dqt {
namespace v3 {

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

// Packed ternary codes q [d_out][d_in / 4 bytes] -> the B operand of dX in
// packed form: row k (input feature) holds the codes of column k of q in
// steps of 64 output features, 16 bytes per step (ld = 16 ceil(d_out / 64)).
// Within a step, codes n = 64 st + 16 kk + 8 h + e go to 16-bit word kk of
// the 8-byte half h (e at bits 2 e), the halves swapped when bit 4 of k is
// set (the GEMM reads a lane's half with one 8-byte LDS read, free of bank
// conflicts).  Past d_out the code is 1 (zero).
struct TpTab {
  const uint8_t* src[MAXG];
  uint8_t* dst[MAXG];
  int32_t d_out[MAXG], d_in[MAXG];
  int32_t b0[MAXG + 1];
  int32_t n;
};

__global__ __launch_bounds__(256) void pack_codes_t_kernel(const TpTab tab) {
  int s = 0;
  while (s + 1 < tab.n && (int)blockIdx.x >= tab.b0[s + 1]) ++s;
  const int d_out = tab.d_out[s], d_in = tab.d_in[s];
  const int n16 = d_in / 16, nst = (d_out + 63) / 64;
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  if (t >= (int64_t)n16 * nst) return;
  const int j16 = (int)(t % n16), st = (int)(t / n16);   // 16 input features, one step
  const uint8_t* src = tab.src[s] + 4 * j16;
  const int ldw = d_in / 4;
  uint32_t out[16][4];
#pragma unroll
  for (int jj = 0; jj < 16; ++jj)
#pragma unroll
    for (int w = 0; w < 4; ++w) out[jj][w] = 0;
#pragma unroll
  for (int e = 0; e < 64; ++e) {
    const int r = st * 64 + e;
    const uint32_t w = r < d_out ? *reinterpret_cast<const uint32_t*>(src + (int64_t)r * ldw) : 0x55555555u;
    const int kk = e >> 4, hh = (e >> 3) & 1, ee = e & 7;
    const int word = 2 * hh + (kk >> 1);                  // dword of the 16 bytes
    const int shift = 16 * (kk & 1) + 2 * ee;
#pragma unroll
    for (int jj = 0; jj < 16; ++jj) out[jj][word] |= ((w >> (2 * jj)) & 3u) << shift;
  }
  const int ldq = 16 * nst;
  const bool swap = (j16 & 1) != 0;                        // bit 4 of k = 16 j16 + jj
#pragma unroll
  for (int jj = 0; jj < 16; ++jj) {
    const uint4 v = swap ? make_uint4(out[jj][2], out[jj][3], out[jj][0], out[jj][1])
                         : make_uint4(out[jj][0], out[jj][1], out[jj][2], out[jj][3]);
    *reinterpret_cast<uint4*>(tab.dst[s] + (int64_t)(16 * j16 + jj) * ldq + 16 * st) = v;
  }
}

// Packed ternary codes -> one operand byte (int8 or e4m3) per weight, same
// [d_out][d_in] row-major order.
// Four chunks of 16 weights per thread (16 bytes in, 64 out), the last
// thread of a tensor whatever chunks remain.
template <int OUT>
__device__ __forceinline__ uint4 unpack16_ternary(uint32_t w) {
  uint32_t o[4];
#pragma unroll
  for (int b = 0; b < 4; ++b) {
    const uint32_t sp = spread_codes((w >> (8 * b)) & 0xFFu);
    o[b] = OUT == 1 ? codes_to_e4m3x4(sp) : codes_to_i8x4(sp);
  }
  return make_uint4(o[0], o[1], o[2], o[3]);
}
template <int OUT>   // 0: int8, 1: e4m3
__global__ __launch_bounds__(256) void unpack_ternary_kernel(const SegTab tab) {
  const int s = seg_of_block(tab);
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  const int64_t g0 = 4 * t, n16 = tab.n16[s];
  if (g0 >= n16) return;
  uint4* const dst = static_cast<uint4*>(tab.dst[s]);
  if (g0 + 4 <= n16) {
    const uint4 w = static_cast<const uint4*>(tab.src[s])[t];
    dst[g0] = unpack16_ternary<OUT>(w.x);
    dst[g0 + 1] = unpack16_ternary<OUT>(w.y);
    dst[g0 + 2] = unpack16_ternary<OUT>(w.z);
    dst[g0 + 3] = unpack16_ternary<OUT>(w.w);
  } else {
    for (int64_t g = g0; g < n16; ++g) dst[g] = unpack16_ternary<OUT>(static_cast<const uint32_t*>(tab.src[s])[g]);
  }
}

// Packed ternary codes -> FP4 (E2M1) values, two per byte in weight order
// (weight k in the low nibble of byte k / 2 when k is even): the B operand of
// the e4m3 forward.  64 weights per thread (16 bytes in, 32 out: with 16
// weights a thread the pass was held by the few bytes each had in flight);
// n16 a multiple of 4.
__global__ __launch_bounds__(256) void expand_fp4_kernel(const SegTab tab) {
  const int s = seg_of_block(tab);
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  if (t >= tab.n16[s] / 4) return;
  const uint4 w = static_cast<const uint4*>(tab.src[s])[t];
  const u32x2 a = expand16_fp4(w.x), b = expand16_fp4(w.y), c = expand16_fp4(w.z), d = expand16_fp4(w.w);
  uint4* const dst = static_cast<uint4*>(tab.dst[s]) + 2 * t;
  dst[0] = make_uint4(a[0], a[1], b[0], b[1]);
  dst[1] = make_uint4(c[0], c[1], d[0], d[1]);
}

// int4 codes (two's-complement nibbles, weight k at bits 4 (k mod 2) of byte
// k / 2) -> one operand byte per weight (int8, or e4m3, exact for |q| <= 8),
// same order; 16 weights per thread.
template <int OUT>   // 0: int8, 1: e4m3
__global__ __launch_bounds__(256) void unpack_int4_kernel(const SegTab tab) {
  const int s = seg_of_block(tab);
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  if (t >= tab.n16[s]) return;
  const uint2 w2 = static_cast<const uint2*>(tab.src[s])[t];
  const uint32_t w[2] = {w2.x, w2.y};
  uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int q = (int)(w[e >> 3] << (28 - 4 * (e & 7))) >> 28;
    const uint32_t b = OUT == 1 ? f32_to_e4m3((float)q) : ((uint32_t)q & 0xFFu);
    o[e >> 2] |= b << (8 * (e & 3));
  }
  static_cast<uint4*>(tab.dst[s])[t] = make_uint4(o[0], o[1], o[2], o[3]);
}

// 3-bit codes (8 weights in 3 bytes, weight k at bits 3 (k mod 8) of its
// group) -> one operand byte per weight (int8, or e4m3, exact for |q| <= 4),
// same order; 16 weights (6 bytes, read as three 2-byte words) per thread.
template <int OUT>   // 0: int8, 1: e4m3
__global__ __launch_bounds__(256) void unpack_int3_kernel(const SegTab tab) {
  const int s = seg_of_block(tab);
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  if (t >= tab.n16[s]) return;
  const uint16_t* src = static_cast<const uint16_t*>(tab.src[s]) + 3 * t;
  const uint64_t bits = (uint64_t)src[0] | ((uint64_t)src[1] << 16) | ((uint64_t)src[2] << 32);
  uint32_t o[4] = {0u, 0u, 0u, 0u};
#pragma unroll
  for (int e = 0; e < 16; ++e) {
    const int q = (int)((uint32_t)(bits >> (3 * e)) << 29) >> 29;
    const uint32_t b = OUT == 1 ? f32_to_e4m3((float)q) : ((uint32_t)q & 0xFFu);
    o[e >> 2] |= b << (8 * (e & 3));
  }
  static_cast<uint4*>(tab.dst[s])[t] = make_uint4(o[0], o[1], o[2], o[3]);
}

// int8 codes -> bf16 (|q| <= 128 is exact in bf16).
// Weights q [d_out][d_in] (packed ternary codes, or int8) -> the B operand of
// dX with the reduction contiguous: W~T[k][n] = bf16(q[n][k]), rows of d_out
// elements.  One 64 x 64 tile per block, transposed through LDS.
struct TrTab {
  const uint8_t* src[MAXG];
  uint16_t* dst[MAXG];
  int32_t d_out[MAXG], d_in[MAXG];
  int32_t tn[MAXG];           // tiles along n (d_out / 64, rounded up)
  int32_t b0[MAXG + 1];
  int32_t n;
};
template <int CF>
__global__ __launch_bounds__(256) void unpack_t_kernel(const TrTab tab) {
  int s = 0;
  while (s + 1 < tab.n && (int)blockIdx.x >= tab.b0[s + 1]) ++s;
  const int tile = (int)blockIdx.x - tab.b0[s];
  const int n0 = (tile % tab.tn[s]) * 64, k0 = (tile / tab.tn[s]) * 64;
  const int d_out = tab.d_out[s], d_in = tab.d_in[s];
  __shared__ __attribute__((aligned(16))) uint16_t t_lds[64][72];   // [k][n]
  const int t = threadIdx.x;
  {
    // thread t: row n0 + t / 4, reduction elements k0 + 16 (t mod 4) .. + 15
    const int nl = t >> 2, kl = (t & 3) * 16;
    const int n = n0 + nl, k = k0 + kl;
    uint16_t v[16];
    if (n < d_out && k < d_in) {
      if constexpr (CF == CF_T2) {
        const uint32_t w = *reinterpret_cast<const uint32_t*>(tab.src[s] + (int64_t)n * (d_in / 4) + k / 4);
#pragma unroll
        for (int e = 0; e < 16; ++e) v[e] = (uint16_t)code_to_bf16_bits((w >> (2 * e)) & 3u);
      } else if constexpr (CF == CF_I3) {
        // 16 weights: 6 bytes at 3 k / 8 (k a multiple of 16: 2-byte aligned)
        const uint16_t* w3 = reinterpret_cast<const uint16_t*>(tab.src[s] + (int64_t)n * (3 * d_in / 8) + 3 * k / 8);
        const uint64_t bits = (uint64_t)w3[0] | ((uint64_t)w3[1] << 16) | ((uint64_t)w3[2] << 32);
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float f = (float)((int)((uint32_t)(bits >> (3 * e)) << 29) >> 29);
          v[e] = (uint16_t)(__float_as_uint(f) >> 16);   // exact: |q| <= 4
        }
      } else if constexpr (CF == CF_I4) {
        const uint2 w2 = *reinterpret_cast<const uint2*>(tab.src[s] + (int64_t)n * (d_in / 2) + k / 2);
        const uint32_t w[2] = {w2.x, w2.y};
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float f = (float)((int)(w[e >> 3] << (28 - 4 * (e & 7))) >> 28);
          v[e] = (uint16_t)(__float_as_uint(f) >> 16);   // exact: |q| <= 8
        }
      } else {
        const uint4 w4 = *reinterpret_cast<const uint4*>(tab.src[s] + (int64_t)n * d_in + k);
        const uint32_t w[4] = {w4.x, w4.y, w4.z, w4.w};
#pragma unroll
        for (int e = 0; e < 16; ++e) {
          const float f = (float)(int)(int8_t)((w[e >> 2] >> (8 * (e & 3))) & 0xFFu);
          v[e] = (uint16_t)(__float_as_uint(f) >> 16);   // exact: |q| <= 128
        }
      }
    } else {
#pragma unroll
      for (int e = 0; e < 16; ++e) v[e] = 0;
    }
#pragma unroll
    for (int e = 0; e < 16; ++e) t_lds[kl + e][nl] = v[e];
  }
  __syncthreads();
#pragma unroll
  for (int c = t; c < 64 * 8; c += 256) {
    const int kl = c >> 3, ch = c & 7;
    const int k = k0 + kl, n = n0 + ch * 8;
    if (k < d_in && n < d_out)
      *reinterpret_cast<uint4*>(tab.dst[s] + (int64_t)k * d_out + n) =
          *reinterpret_cast<const uint4*>(&t_lds[kl][ch * 8]);
  }
}

// Ternary codes -> W~T as unpack_t_kernel, one block per strip of 64 rows x
// 512 reduction elements: the strip's codes (whole 128-byte lines of each
// row) come into LDS in one pass, eight loads in flight per thread, then its
// eight 64 x 64 tiles are transposed through LDS in turn.  (One block per
// tile read 16 bytes of each row's line and fetched about 4 times the code
// bytes.)
__global__ __launch_bounds__(256) void unpack_t2_strip_kernel(const TrTab tab) {
  int s = 0;
  while (s + 1 < tab.n && (int)blockIdx.x >= tab.b0[s + 1]) ++s;
  const int strip = (int)blockIdx.x - tab.b0[s];
  const int n0 = (strip % tab.tn[s]) * 64, ks0 = (strip / tab.tn[s]) * 512;
  const int d_out = tab.d_out[s], d_in = tab.d_in[s];
  __shared__ uint32_t codes[64][33];                                 // [row][word of 16 codes]
  __shared__ __attribute__((aligned(16))) uint16_t t_lds[64][72];   // [k][n]
  const int t = threadIdx.x;
  {
    // thread t: row n0 + t / 4, words 8 (t mod 4) .. + 7 of the strip
    const int row = t >> 2, n = n0 + row;
    const int wrow = d_in / 16;                       // words of a row
    const uint32_t* src = reinterpret_cast<const uint32_t*>(tab.src[s]) + (int64_t)n * wrow;
    uint32_t w[8];
#pragma unroll
    for (int e = 0; e < 8; ++e) {
      const int kw = ks0 / 16 + 8 * (t & 3) + e;
      w[e] = (n < d_out && kw < wrow) ? src[kw] : 0u;
    }
#pragma unroll
    for (int e = 0; e < 8; ++e) codes[row][8 * (t & 3) + e] = w[e];
  }
  __syncthreads();
  const int nl = t >> 2, kl = (t & 3) * 16;
  for (int j = 0; j < 8; ++j) {
    const int k0 = ks0 + 64 * j;
    if (k0 >= d_in) break;                            // (uniform)
    const uint32_t w = codes[nl][4 * j + (t & 3)];
#pragma unroll
    for (int e = 0; e < 16; ++e) t_lds[kl + e][nl] = (uint16_t)code_to_bf16_bits((w >> (2 * e)) & 3u);
    __syncthreads();
#pragma unroll
    for (int c = t; c < 64 * 8; c += 256) {
      const int kr = c >> 3, ch = c & 7;
      const int k = k0 + kr, n = n0 + ch * 8;
      if (k < d_in && n < d_out)
        *reinterpret_cast<uint4*>(tab.dst[s] + (int64_t)k * d_out + n) =
            *reinterpret_cast<const uint4*>(&t_lds[kr][ch * 8]);
    }
    __syncthreads();
  }
}

// X~T[k, m] = bf16(fl(value(Xq[m, k]) * xdq[m])): the dequantised
// activations transposed (the reduction of dW, over tokens, contiguous).
// One 64 x 64 tile per block, transposed through LDS.
struct DqTab {
  const uint8_t* src[MAXG];   // Xq [M][K]
  uint16_t* dst[MAXG];        // X~T [K][Mp]
  const float* scale[MAXG];   // xdq [M]
  int32_t K[MAXG];
  int32_t tm[MAXG];           // tiles along m
  int32_t b0[MAXG + 1];
  int32_t n;
  int64_t M, Mp;              // tokens, and the row stride of X~T (a multiple of 64)
};
template <bool E4M3>
__global__ __launch_bounds__(256) void dequant_t_kernel(const DqTab tab) {
  int s = 0;
  while (s + 1 < tab.n && (int)blockIdx.x >= tab.b0[s + 1]) ++s;
  const int tile = (int)blockIdx.x - tab.b0[s];
  const int64_t M = tab.M;
  const int K = tab.K[s];
  const int64_t m0 = (int64_t)(tile % tab.tm[s]) * 64;
  const int k0 = (tile / tab.tm[s]) * 64;
  __shared__ __attribute__((aligned(16))) uint16_t t_lds[64][72];   // [k][m]
  const int t = threadIdx.x;
  {
    // thread t: token m0 + t / 4, features k0 + 16 (t mod 4) .. + 15
    const int ml = t >> 2, kl = (t & 3) * 16;
    const int64_t m = m0 + ml;
    const int k = k0 + kl;
    uint32_t o[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (m < M && k < K) {
      const float d = tab.scale[s][m];
      const uint4 v = *reinterpret_cast<const uint4*>(tab.src[s] + m * K + k);
      const uint32_t w[4] = {v.x, v.y, v.z, v.w};
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
    }
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      t_lds[kl + 2 * j][ml] = (uint16_t)(o[j] & 0xFFFFu);
      t_lds[kl + 2 * j + 1][ml] = (uint16_t)(o[j] >> 16);
    }
  }
  __syncthreads();
#pragma unroll
  for (int c = t; c < 64 * 8; c += 256) {
    const int kl = c >> 3, ch = c & 7;
    const int k = k0 + kl;
    const int64_t m = m0 + ch * 8;
    if (k < K && m < M)
      *reinterpret_cast<uint4*>(tab.dst[s] + (int64_t)k * tab.Mp + m) =
          *reinterpret_cast<const uint4*>(&t_lds[kl][ch * 8]);
  }
}

// dW[l] = sum over splits of the fp32 partials of linear l, in split order
// (deterministic), for every linear of a batch in one launch.
struct RedTab {
  const float* src[MAXG];     // [splits][n] partials
  float* dst[MAXG];           // [n]
  int64_t n4[MAXG];           // n / 4
  int32_t b0[MAXG + 1];
  int32_t n, splits;
};
__global__ __launch_bounds__(256) void split_reduce_batch_kernel(const RedTab tab) {
  int s = 0;
  while (s + 1 < tab.n && (int)blockIdx.x >= tab.b0[s + 1]) ++s;
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  const int64_t n4 = tab.n4[s];
  if (t >= n4) return;
  const f32x4* src = reinterpret_cast<const f32x4*>(tab.src[s]);
  f32x4 acc = __builtin_nontemporal_load(src + t);
  for (int k = 1; k < tab.splits; ++k) {
    const f32x4 v = __builtin_nontemporal_load(src + (int64_t)k * n4 + t);
    acc[0] = acc[0] + v[0];
    acc[1] = acc[1] + v[1];
    acc[2] = acc[2] + v[2];
    acc[3] = acc[3] + v[3];
  }
  reinterpret_cast<f32x4*>(tab.dst[s])[t] = acc;
}

// The split-K sum of dW (the same order as split_reduce_batch_kernel, so the
// same dW bits) consumed by the SR update of the codes, 8 weights per
// thread; dW is never stored.
struct RedSRTab {
  const float* src[MAXG];     // [splits][n] partials
  uint8_t* wq[MAXG];          // codes, updated in place
  int64_t n8[MAXG];           // n / 8
  float c[MAXG], L[MAXG];
  int32_t qmin[MAXG], qmax[MAXG];
  uint32_t tid[MAXG];
  int32_t b0[MAXG + 1];
  int32_t n, splits;
  uint32_t k0, k1, step;
  unsigned long long* counters;
};
template <int CF>
__global__ __launch_bounds__(256) void split_reduce_sr_kernel(const RedSRTab tab) {
  int s = 0;
  while (s + 1 < tab.n && (int)blockIdx.x >= tab.b0[s + 1]) ++s;
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[s]) * 256 + threadIdx.x;
  uint32_t ch = 0, nf = 0;
  if (t < tab.n8[s]) {
    const int64_t n4 = 2 * tab.n8[s];
    const f32x4* src = reinterpret_cast<const f32x4*>(tab.src[s]);
    f32x4 gv[2];
    gv[0] = __builtin_nontemporal_load(src + 2 * t);
    gv[1] = __builtin_nontemporal_load(src + 2 * t + 1);
    for (int k = 1; k < tab.splits; ++k) {
#pragma unroll
      for (int e = 0; e < 2; ++e) {
        const f32x4 v = __builtin_nontemporal_load(src + (int64_t)k * n4 + 2 * t + e);
        gv[e][0] = gv[e][0] + v[0];
        gv[e][1] = gv[e][1] + v[1];
        gv[e][2] = gv[e][2] + v[2];
        gv[e][3] = gv[e][3] + v[3];
      }
    }
    SRArgs a;
    a.c = tab.c[s];
    a.L = tab.L[s];
    a.qmin = tab.qmin[s];
    a.qmax = tab.qmax[s];
    a.k0 = tab.k0;
    a.k1 = tab.k1;
    a.step = tab.step;
    a.tid = tab.tid[s];
    uint32_t win[4] = {0u, 0u, 0u, 0u}, wout[4];
    ChunkIO<CF>::load(tab.wq[s], t, win);
    sr_chunk<CF, 8>(win, gv, (uint64_t)t, a, wout, ch, nf);
    ChunkIO<CF>::store(tab.wq[s], t, wout);
  }
  if (tab.counters != nullptr) {
    // one atomic per block (atomics of every wave on one address serialise)
    __shared__ uint32_t red[2][256 / kWave];
    const uint32_t c = wave_sum_u32(ch), f = wave_sum_u32(nf);
    if ((threadIdx.x & (kWave - 1)) == 0) {
      red[0][threadIdx.x / kWave] = c;
      red[1][threadIdx.x / kWave] = f;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long ct = 0, ft = 0;
#pragma unroll
      for (int w = 0; w < 256 / kWave; ++w) {
        ct += red[0][w];
        ft += red[1][w];
      }
      if (ct) atomicAdd(tab.counters, ct);
      if (ft) atomicAdd(tab.counters + 1, ft);
    }
  }
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

// Zeroes the persistent GEMM's tile counters (both 64-byte slots) before
// its launch, so a workspace needs no particular contents.
__global__ __launch_bounds__(64) void sched_clear_kernel(int* sched) {
  if (threadIdx.x < 32) sched[threadIdx.x] = 0;
}

// Tile counts and longest-first order of a group; `slot` picks its 64 bytes
// of tile counters among the workspace's first 128.  Returns the most tiles
// any XCD's list holds.
template <int ELEM, int KB, class Epi>
static int32_t prep_group(Group<Epi>& grp, uint8_t* ws, int slot) {
  grp.sched = reinterpret_cast<int*>(ws + 64 * slot);
  constexpr int64_t BK = KB / (ELEM == EBF16 ? 2 : 1);
  int64_t steps[MAXG];
  for (int g = 0; g < grp.ng; ++g) {
    Prob<Epi>& p = grp.p[g];
    p.nbx = (int32_t)((p.J + TILE - 1) / TILE);
    p.nby = (int32_t)((p.I + TILE - 1) / TILE);
    p.ntiles = p.nbx * p.nby * p.nbz;
    steps[g] = (std::min(p.split_len, p.R) + BK - 1) / BK;
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
  return per_xcd;
}

// Persistent grid over one group: 8 x (blocks per XCD), one block per
// compute unit at most.
template <int ELEM, int MA, int MB, int KB, class Epi>
static hipError_t launch_group(Group<Epi>& grp, uint8_t* ws, hipStream_t s) {
  const int32_t per_xcd = prep_group<ELEM, KB>(grp, ws, 0);
  if (per_xcd == 0) return hipSuccess;
  const int32_t bpx = std::min(per_xcd, std::max(1, current_device_cus() / 8));
  LaunchStatus st;
  st << launch_kernel(sched_clear_kernel, dim3(1), dim3(64), s, reinterpret_cast<int*>(ws));
  st << timed_launch(s, [&] {
    return launch_kernel(gemm_v3_kernel<ELEM, MA, MB, KB, Epi>, dim3((unsigned)(8 * bpx)), dim3(NTH), s, grp);
  });
  return st.e;
}

// Groups g1 then g2 in one launch (tile counters in slots 1 and 0).
template <int E1, int MA1, int MB1, int KB1, class Epi1, int E2, int MA2, int MB2, int KB2, class Epi2>
static hipError_t launch_dual(Group<Epi1>& g1, Group<Epi2>& g2, uint8_t* ws, hipStream_t s) {
  const int32_t p1 = prep_group<E1, KB1>(g1, ws, 1);
  const int32_t p2 = prep_group<E2, KB2>(g2, ws, 0);
  const int32_t per_xcd = std::max(p1, p2);
  if (per_xcd == 0) return hipSuccess;
  const int32_t bpx = std::min(per_xcd, std::max(1, current_device_cus() / 8));
  LaunchStatus st;
  st << launch_kernel(sched_clear_kernel, dim3(1), dim3(64), s, reinterpret_cast<int*>(ws));
  st << timed_launch(s, [&] {
    return launch_kernel(gemm_v3_dual_kernel<E1, MA1, MB1, KB1, Epi1, E2, MA2, MB2, KB2, Epi2>,
                         dim3((unsigned)(8 * bpx)), dim3(NTH), s, g1, g2);
  });
  return st.e;
}

}  // namespace v3

using namespace v3;

// reduction bytes per step of the unpacked 8-bit forward and of the bf16
// backward products (128: full lines, two stages; 64: half lines, four
// stages in flight: 9-11 % slower for the int8 forward on the LLaMA-block
// shapes; the backward's SR epilogue needs a whole 64 KB stage for its
// staging)
#ifndef KB_FWD
#define KB_FWD 128
#endif
#ifndef KB_BWD
#define KB_BWD 128
#endif
// ternary weights against e4m3 activations: B as FP4 values (1) or as e4m3
// bytes (0) in the scaled MFMA
#ifndef FWD_FP4B
#define FWD_FP4B 1
#endif
#ifndef DX_PACKED_B
#define DX_PACKED_B 0
#endif
// dW with the SR update formed transposed (X~^T dY, EpiSR<CF, true>): 1, or
// as dY^T X~ (0)
#ifndef DW_TRANS
#define DW_TRANS 1
#endif
#ifndef UNPACK_T2_STRIP
#define UNPACK_T2_STRIP 1
#endif

static size_t align256(size_t n) { return (n + 255) / 256 * 256; }

hipError_t launch_unpack_int3(const void* src, int8_t* dst, int64_t n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  SegTab tab{};
  tab.n = 1;
  tab.src[0] = src;
  tab.dst[0] = dst;
  tab.n16[0] = n / 16;
  const int32_t blocks = seal(tab);
  return launch_kernel(unpack_int3_kernel<0>, dim3(blocks), dim3(256), stream, tab);
}

hipError_t launch_unpack_int4(const void* src, int8_t* dst, int64_t n, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  SegTab tab{};
  tab.n = 1;
  tab.src[0] = src;
  tab.dst[0] = dst;
  tab.n16[0] = n / 16;
  const int32_t blocks = seal(tab);
  return launch_kernel(unpack_int4_kernel<0>, dim3(blocks), dim3(256), stream, tab);
}

// Ternary weights reach the forward GEMM as packed codes when every d_in of
// the batch is a multiple of 64 (16-byte aligned packed rows); otherwise
// they are first unpacked into the workspace.
static bool fwd_packed(int n, const LinearIO* io) {
  for (int l = 0; l < n; ++l)
    if (io[l].d_in % 64 != 0) return false;
  return true;
}

// Forward workspace: the tile counters, then per linear the operand bytes
// its codes are expanded into (one byte per weight; FP4 uses half).  Ternary
// codes with d_in a multiple of 64 can also run straight from the packed
// codes, expanded in registers, with the counters alone: that form needs
// only fwd_batch_workspace_min, the expanded one (measured faster: the
// expansion in the main loop costs more than a pass and the extra copies)
// is taken whenever the workspace holds it.
size_t fwd_batch_workspace(int n, const LinearIO* io, int cf, size_t* offs) {
  size_t total = kSchedBytes;
  const bool unpack = cf == CF_T2 || cf == CF_I4 || cf == CF_I3;
  for (int l = 0; l < n; ++l) {
    if (offs) offs[l] = total;
    if (unpack) total += align256((size_t)(io[l].d_out * io[l].d_in));
  }
  return total;
}
size_t fwd_batch_workspace_min(int n, const LinearIO* io, int cf) {
  if (cf == CF_T2 && fwd_packed(n, io)) return kSchedBytes;
  return fwd_batch_workspace(n, io, cf, nullptr);
}

hipError_t launch_fwd_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, size_t ws_bytes,
                           hipStream_t stream) {
  if (c.M == 0 || c.n == 0) return hipSuccess;
  LaunchStatus st;
  size_t offs[kMaxBatch];
  const size_t full =
      fwd_batch_workspace(c.n, io, c.w_ternary ? CF_T2 : c.w_int4 ? CF_I4 : c.w_int3 ? CF_I3 : CF_I8, offs);
  const bool aligned = c.w_ternary && fwd_packed(c.n, io);
  // ternary codes straight from the packed form only when the workspace
  // cannot hold their expansion
  const bool packed = aligned && ws_bytes < full;
  // FP4 values of ternary codes in the workspace (e4m3 activations)
  const bool fp4 = aligned && !packed && c.act_e4m3;
  // int8 (or e4m3) copy of the codes in the workspace
  const bool unpacked = (c.w_ternary && !packed && !fp4) || c.w_int4 || c.w_int3;
  if (c.w_int3) {
    SegTab tab{};
    tab.n = c.n;
    for (int l = 0; l < c.n; ++l) {
      tab.src[l] = io[l].Wq;
      tab.dst[l] = ws + offs[l];
      tab.n16[l] = io[l].d_out * io[l].d_in / 16;
    }
    const int32_t blocks = seal(tab);
    if (c.act_e4m3)
      st << launch_kernel(unpack_int3_kernel<1>, dim3(blocks), dim3(256), stream, tab);
    else
      st << launch_kernel(unpack_int3_kernel<0>, dim3(blocks), dim3(256), stream, tab);
  } else if (c.w_int4) {
    SegTab tab{};
    tab.n = c.n;
    for (int l = 0; l < c.n; ++l) {
      tab.src[l] = io[l].Wq;
      tab.dst[l] = ws + offs[l];
      tab.n16[l] = io[l].d_out * io[l].d_in / 16;
    }
    const int32_t blocks = seal(tab);
    if (c.act_e4m3)
      st << launch_kernel(unpack_int4_kernel<1>, dim3(blocks), dim3(256), stream, tab);
    else
      st << launch_kernel(unpack_int4_kernel<0>, dim3(blocks), dim3(256), stream, tab);
  } else if (fp4) {
    SegTab tab{};
    tab.n = c.n;
    for (int l = 0; l < c.n; ++l) {
      tab.src[l] = io[l].Wq;
      tab.dst[l] = ws + offs[l];
      tab.n16[l] = io[l].d_out * io[l].d_in / 16;   // a multiple of 4 (d_in of 64)
    }
    // one thread per 4 chunks
    int32_t blocks = 0;
    for (int l = 0; l < c.n; ++l) {
      tab.b0[l] = blocks;
      blocks += (int32_t)((tab.n16[l] / 4 + 255) / 256);
    }
    tab.b0[c.n] = blocks;
    st << launch_kernel(expand_fp4_kernel, dim3(blocks), dim3(256), stream, tab);
  } else if (c.w_ternary && !packed) {
    SegTab tab{};
    tab.n = c.n;
    for (int l = 0; l < c.n; ++l) {
      tab.src[l] = io[l].Wq;
      tab.dst[l] = ws + offs[l];
      tab.n16[l] = io[l].d_out * io[l].d_in / 16;
    }
    // one thread per 4 chunks
    int32_t blocks = 0;
    for (int l = 0; l < c.n; ++l) {
      tab.b0[l] = blocks;
      blocks += (int32_t)(((tab.n16[l] + 3) / 4 + 255) / 256);
    }
    tab.b0[c.n] = blocks;
    if (c.act_e4m3)
      st << launch_kernel(unpack_ternary_kernel<1>, dim3(blocks), dim3(256), stream, tab);
    else
      st << launch_kernel(unpack_ternary_kernel<0>, dim3(blocks), dim3(256), stream, tab);
  }
  Group<EpiFwd> grp{};
  grp.ng = c.n;
  for (int l = 0; l < c.n; ++l) {
    Prob<EpiFwd>& p = grp.p[l];
    p.A = Opnd{static_cast<const uint8_t*>(io[l].Xq), io[l].d_in, c.M};
    if (packed)
      p.B = Opnd{static_cast<const uint8_t*>(io[l].Wq), io[l].d_in / 4, io[l].d_out};
    else if (fp4)
      p.B = Opnd{ws + offs[l], io[l].d_in / 2, io[l].d_out};
    else if (unpacked)
      p.B = Opnd{ws + offs[l], io[l].d_in, io[l].d_out};
    else
      p.B = Opnd{static_cast<const uint8_t*>(io[l].Wq), io[l].d_in, io[l].d_out};
    p.epi = EpiFwd{io[l].Y, io[l].d_out, c.out_bf16, io[l].xdq, io[l].alpha};
    p.I = c.M;
    p.J = io[l].d_out;
    p.R = io[l].d_in;
    p.split_len = io[l].d_in;
    p.nbz = 1;
  }
  if (packed) {
    if (c.act_e4m3) st << launch_group<FWD_FP4B ? EF4B : EF8, KC, KCP, 128>(grp, ws, stream);
    else st << launch_group<EI8, KC, KCP, 128>(grp, ws, stream);
  } else if (fp4) {
    st << launch_group<EF4B, KC, KF4, 128>(grp, ws, stream);
  } else {
    if (c.act_e4m3) st << launch_group<EF8, KC, KC, KB_FWD>(grp, ws, stream);
    else st << launch_group<EI8, KC, KC, KB_FWD>(grp, ws, stream);
  }
  return st.e;
}

// Backward plan for a batch in the bf16 environment: one split count for
// every dW product of the batch, and the workspace layout
//   per linear: [bf16 weights d_in x d_out][bf16 X~T d_in x Mp][fp32 partials]
// (Mp: M rounded up to a multiple of 64, the row stride of X~T)
// (partials sized for the larger of this plan's and the fp32 kernels' split).
// The split count minimises an estimate of rounds of the persistent grid x
// steps per tile plus the traffic of the partial sums.
static int64_t xt_stride(int64_t M) { return (M + 63) / 64 * 64; }

BwdPlan plan_bwd_batch(int n, const LinearIO* io, int64_t M) {
  BwdPlan P{};
  P.wi = 4;
  P.wj = 4;
  P.splits = 1;
  P.splits_dual = 1;
  const int cus = current_device_cus();
  // a step of a 256 x 256 bf16 tile is ~2048 MFMA cycles at ~2.1 GHz, plus
  // ~2 us of per-tile prologue / epilogue; partials move at ~4 TB/s
  constexpr double kStepUs = 2048.0 / 2100.0, kTileUs = 2.0;
  auto tiles_of = [](int64_t I, int64_t J) { return ((I + TILE - 1) / TILE) * ((J + TILE - 1) / TILE); };
  double dx_us = 0;     // dX work of the whole batch, summed over its tiles
  for (int l = 0; l < n; ++l)
    dx_us += (double)tiles_of(M, io[l].d_in) * ((double)((io[l].d_out + 63) / 64) * kStepUs + kTileUs);
  double best = 1e300, best_dual = 1e300;
  for (int64_t s = 1; s <= 32; ++s) {
    if (s > 1 && M / s < 256) break;
    int64_t tiles = 0;
    double part_bytes = 0;
    for (int l = 0; l < n; ++l) {
      tiles += tiles_of(io[l].d_out, io[l].d_in) * s;
      if (s > 1) part_bytes += (2.0 * s + 1.0) * (double)(io[l].d_out * io[l].d_in * 4);
    }
    const double rounds = (double)((tiles + cus - 1) / cus);
    const double tile_us = (double)(((M + s - 1) / s + 63) / 64) * kStepUs + kTileUs;
    // dW alone: whole rounds of equal tiles
    const double t_us = rounds * tile_us + part_bytes / 4.0e6;
    if (t_us < best * 0.999) { best = t_us; P.splits = s; }
    // dW then dX in one launch: the dW rounds, or the total work spread
    // over every compute unit, whichever is longer
    const double t_dual = std::max(rounds * tile_us, ((double)tiles * tile_us + dx_us) / cus) +
                          part_bytes / 4.0e6;
    if (t_dual < best_dual * 0.999) { best_dual = t_dual; P.splits_dual = s; }
  }
  // The SR update in the dW epilogue saves dW's store and a streaming pass
  // over it, at the price of ~173 vector instructions per 8 weights in the
  // dW tiles.  Measured per call it is the faster form on every LLaMA block
  // (hidden 768, where those tiles are the launch's critical path: 288 us
  // against 300 us staged), so it is the default; DQT_SR_EPILOGUE=staged in
  // the environment stages dW in the workspace and updates it in a pass of
  // its own (same dW bits, same codes), e.g. to test both forms.
  bool fuse = true;
  if (const char* f = getenv("DQT_SR_EPILOGUE")) fuse = strcmp(f, "staged") != 0;
  P.sr_fused = P.splits == 1 && fuse;
  P.sr_fused_dual = P.splits_dual == 1 && fuse;
  const bool stage_dw = (P.splits == 1 && !P.sr_fused) || (P.splits_dual == 1 && !P.sr_fused_dual);
  size_t off = kSchedBytes;
  for (int l = 0; l < n; ++l) {
    const size_t wn = (size_t)(io[l].d_out * io[l].d_in);
    const int64_t s32 = dw_splits_f32(io[l].d_out, io[l].d_in, M);
    const int64_t sp = std::max(std::max(P.splits, P.splits_dual), s32);
    P.q_off[l] = off;
    off += align256(wn * 2);
    P.xt_off[l] = off;
    off += align256((size_t)xt_stride(M) * (size_t)io[l].d_in * 2);
    P.part_off[l] = off;
    off += sp > 1 ? align256((size_t)sp * wn * 4) : stage_dw ? align256(wn * 4) : 0;
  }
  P.total = off;
  return P;
}

// dX[m, k] = alpha sum_n dY[m, n] q[n, k]: I = M, J = d_in, R = d_out.
// Fills the problems of the group and launches the pre-pass that writes its
// B operand into the workspace.
static void prep_dx(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                    hipStream_t stream, Group<EpiScale>& grp, LaunchStatus& st) {
  grp.ng = c.n;
  for (int l = 0; l < c.n; ++l) {
    Prob<EpiScale>& p = grp.p[l];
    p.A = Opnd{static_cast<const uint8_t*>(io[l].dY), io[l].d_out * 2, c.M};
    p.epi = EpiScale{io[l].dX, io[l].d_in, c.out_bf16, io[l].alpha};
    p.I = c.M;
    p.J = io[l].d_in;
    p.R = io[l].d_out;
    p.split_len = io[l].d_out;
    p.nbz = 1;
  }
  if (c.w_ternary && DX_PACKED_B) {
    // codes stay packed: transposed into 16-byte steps, expanded in the GEMM
    // (fewer bytes per step, but the table expansion costs more than the
    // copies it saves in the current main loop)
    TpTab tab{};
    tab.n = c.n;
    int32_t blocks = 0;
    for (int l = 0; l < c.n; ++l) {
      tab.src[l] = static_cast<const uint8_t*>(io[l].Wq);
      tab.dst[l] = ws + P.q_off[l];
      tab.d_out[l] = (int32_t)io[l].d_out;
      tab.d_in[l] = (int32_t)io[l].d_in;
      tab.b0[l] = blocks;
      blocks += (int32_t)(((io[l].d_in / 16) * ((io[l].d_out + 63) / 64) + 255) / 256);
      grp.p[l].B = Opnd{ws + P.q_off[l], 16 * ((io[l].d_out + 63) / 64), io[l].d_in};
    }
    tab.b0[c.n] = blocks;
    st << launch_kernel(pack_codes_t_kernel, dim3((unsigned)blocks), dim3(256), stream, tab);
    return;
  }
  // bf16 weights transposed (reduction contiguous), so both operands are
  // read without the transposing LDS reads
  TrTab tab{};
  tab.n = c.n;
  int32_t blocks = 0;
  for (int l = 0; l < c.n; ++l) {
    tab.src[l] = static_cast<const uint8_t*>(io[l].Wq);
    tab.dst[l] = reinterpret_cast<uint16_t*>(ws + P.q_off[l]);
    tab.d_out[l] = (int32_t)io[l].d_out;
    tab.d_in[l] = (int32_t)io[l].d_in;
    tab.tn[l] = (int32_t)((io[l].d_out + 63) / 64);
    tab.b0[l] = blocks;
    // ternary: strips of 512 reduction elements; else 64 x 64 tiles
    const int kspan = c.w_ternary && UNPACK_T2_STRIP ? 512 : 64;
    blocks += tab.tn[l] * (int32_t)((io[l].d_in + kspan - 1) / kspan);
    grp.p[l].B = Opnd{ws + P.q_off[l], io[l].d_out * 2, io[l].d_in};
  }
  tab.b0[c.n] = blocks;
  if (c.w_ternary && UNPACK_T2_STRIP)
    st << launch_kernel(unpack_t2_strip_kernel, dim3(blocks), dim3(256), stream, tab);
  else if (c.w_ternary)
    st << launch_kernel(unpack_t_kernel<CF_T2>, dim3(blocks), dim3(256), stream, tab);
  else if (c.w_int4)
    st << launch_kernel(unpack_t_kernel<CF_I4>, dim3(blocks), dim3(256), stream, tab);
  else if (c.w_int3)
    st << launch_kernel(unpack_t_kernel<CF_I3>, dim3(blocks), dim3(256), stream, tab);
  else
    st << launch_kernel(unpack_t_kernel<CF_I8>, dim3(blocks), dim3(256), stream, tab);
}

hipError_t launch_dx_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                           hipStream_t stream) {
  if (c.M == 0 || c.n == 0) return hipSuccess;
  Group<EpiScale> grp{};
  LaunchStatus st;
  prep_dx(c, io, ws, P, stream, grp, st);
  if (c.w_ternary && DX_PACKED_B) st << launch_group<EBF16, KC, KCP, 128>(grp, ws, stream);
  else st << launch_group<EBF16, KC, KC, KB_BWD>(grp, ws, stream);
  return st.e;
}

// X~T once per distinct quantised input (the dequantising transpose
// pre-pass); first[l] is the linear whose X~T linear l reads.
static void prep_xt(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                    hipStream_t stream, int* first, LaunchStatus& st) {
  DqTab tab{};
  tab.M = c.M;
  tab.Mp = xt_stride(c.M);
  int32_t blocks = 0;
  for (int l = 0; l < c.n; ++l) {
    first[l] = l;
    for (int m = 0; m < l; ++m)
      if (io[m].Xq == io[l].Xq && io[m].d_in == io[l].d_in) { first[l] = first[m]; break; }
    if (first[l] == l && c.M > 0) {
      const int s = tab.n++;
      tab.src[s] = static_cast<const uint8_t*>(io[l].Xq);
      tab.dst[s] = reinterpret_cast<uint16_t*>(ws + P.xt_off[l]);
      tab.scale[s] = io[l].xdq;
      tab.K[s] = (int32_t)io[l].d_in;
      tab.tm[s] = (int32_t)((c.M + 63) / 64);
      tab.b0[s] = blocks;
      blocks += tab.tm[s] * (int32_t)((io[l].d_in + 63) / 64);
    }
  }
  tab.b0[tab.n] = blocks;
  if (tab.n > 0) {
    if (c.act_e4m3)
      st << launch_kernel(dequant_t_kernel<true>, dim3(blocks), dim3(256), stream, tab);
    else
      st << launch_kernel(dequant_t_kernel<false>, dim3(blocks), dim3(256), stream, tab);
  }
}

// dW[n, k] = sum_m dY[m, n] X~T[k, m]: I = d_out, J = d_in, R = M, split over
// the batch into P.splits parts; make(l) gives linear l's epilogue.
template <class Epi, class MakeEpi>
static void fill_dw(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                    const int* first, Group<Epi>& grp, MakeEpi make) {
  const int64_t splits = P.splits;
  int64_t len = splits > 1 ? (c.M + splits - 1) / splits : (c.M > 0 ? c.M : 1);
  len = (len + 63) / 64 * 64;
  grp.ng = c.n;
  for (int l = 0; l < c.n; ++l) {
    Prob<Epi>& p = grp.p[l];
    const int64_t I = io[l].d_out, J = io[l].d_in;
    p.A = Opnd{static_cast<const uint8_t*>(io[l].dY), I * 2, I};
    p.B = Opnd{ws + P.xt_off[first[l]], xt_stride(c.M) * 2, J};
    p.epi = make(l);
    p.I = I;
    p.J = J;
    p.R = c.M;
    p.split_len = len;
    p.nbz = (int32_t)splits;
  }
}

// dW into dW (one split) or into the workspace partials (several).
static void prep_dw(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                    hipStream_t stream, Group<EpiPartial>& grp, LaunchStatus& st) {
  int first[kMaxBatch];
  prep_xt(c, io, ws, P, stream, first, st);
  fill_dw(c, io, ws, P, first, grp, [&](int l) {
    const int64_t I = io[l].d_out, J = io[l].d_in;
    float* target = P.splits > 1 ? reinterpret_cast<float*>(ws + P.part_off[l]) : io[l].dW;
    return EpiPartial{target, J, I * J};
  });
}

// Sum of the batch-split dW partials into dW.
static hipError_t reduce_dw(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                            hipStream_t stream) {
  if (P.splits == 1) return hipSuccess;
  LaunchStatus st;
  RedTab red{};
  red.n = c.n;
  red.splits = (int32_t)P.splits;
  int32_t blocks = 0;
  for (int l = 0; l < c.n; ++l) {
    red.src[l] = reinterpret_cast<const float*>(ws + P.part_off[l]);
    red.dst[l] = io[l].dW;
    red.n4[l] = io[l].d_out * io[l].d_in / 4;
    red.b0[l] = blocks;
    blocks += (int32_t)((red.n4[l] + 255) / 256);
  }
  red.b0[c.n] = blocks;
  st << launch_kernel(split_reduce_batch_kernel, dim3((unsigned)blocks), dim3(256), stream, red);
  return st.e;
}

hipError_t launch_dw_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                           hipStream_t stream) {
  if (c.n == 0) return hipSuccess;
  Group<EpiPartial> grp{};
  LaunchStatus st;
  prep_dw(c, io, ws, P, stream, grp, st);
  st << launch_group<EBF16, KM, KC, KB_BWD>(grp, ws, stream);
  if (st.e != hipSuccess) return st.e;
  return reduce_dw(c, io, ws, P, stream);
}

// dW and dX of a batch in one persistent launch: dW's tiles first (the
// longer reduction), then dX's, so compute units that draw no dW tile, or
// finish theirs early, go on with dX at once.
hipError_t launch_dxdw_batch(const BatchCfg& c, const LinearIO* io, uint8_t* ws, const BwdPlan& P,
                             hipStream_t stream) {
  if (c.n == 0) return hipSuccess;
  if (c.M == 0 || (c.w_ternary && DX_PACKED_B)) {
    const hipError_t e = launch_dx_batch(c, io, ws, P, stream);
    return e != hipSuccess ? e : launch_dw_batch(c, io, ws, P, stream);
  }
  Group<EpiScale> gx{};
  Group<EpiPartial> gw{};
  BwdPlan Q = P;
  Q.splits = P.splits_dual;
  LaunchStatus st;
  prep_dx(c, io, ws, Q, stream, gx, st);
  prep_dw(c, io, ws, Q, stream, gw, st);
  st << launch_dual<EBF16, KM, KC, KB_BWD, EpiPartial, EBF16, KC, KC, KB_BWD, EpiScale>(gw, gx, ws, stream);
  if (st.e != hipSuccess) return st.e;
  return reduce_dw(c, io, ws, Q, stream);
}

// Partials of a batch-split dW summed and consumed by the SR update.
static hipError_t reduce_sr(const BatchCfg& c, const LinearIO* io, const SRTensor* t, uint64_t seed,
                            uint32_t step, unsigned long long* counters, uint8_t* ws,
                            const BwdPlan& P, hipStream_t stream) {
  LaunchStatus st;
  RedSRTab red{};
  red.n = c.n;
  red.splits = (int32_t)P.splits;
  red.k0 = (uint32_t)seed;
  red.k1 = (uint32_t)(seed >> 32);
  red.step = step;
  red.counters = counters;
  int32_t blocks = 0;
  for (int l = 0; l < c.n; ++l) {
    red.src[l] = reinterpret_cast<const float*>(ws + P.part_off[l]);
    red.wq[l] = t[l].wq;
    red.n8[l] = io[l].d_out * io[l].d_in / 8;
    red.c[l] = t[l].c;
    red.L[l] = (float)(t[l].qmax - t[l].qmin + 1);
    red.qmin[l] = t[l].qmin;
    red.qmax[l] = t[l].qmax;
    red.tid[l] = t[l].tensor_id;
    red.b0[l] = blocks;
    blocks += (int32_t)((red.n8[l] + 255) / 256);
  }
  red.b0[c.n] = blocks;
  if (c.w_ternary)
    st << launch_kernel(split_reduce_sr_kernel<CF_T2>, dim3((unsigned)blocks), dim3(256), stream, red);
  else if (c.w_int4)
    st << launch_kernel(split_reduce_sr_kernel<CF_I4>, dim3((unsigned)blocks), dim3(256), stream, red);
  else if (c.w_int3)
    st << launch_kernel(split_reduce_sr_kernel<CF_I3>, dim3((unsigned)blocks), dim3(256), stream, red);
  else
    st << launch_kernel(split_reduce_sr_kernel<CF_I8>, dim3((unsigned)blocks), dim3(256), stream, red);
  return st.e;
}

// dW of every linear consumed by the SR update of its codes in the GEMM
// epilogue (one split) or in the reduction of the partials (several), with
// dX of every linear in the same launch when with_dx.
template <int CF>
static hipError_t launch_dw_sr_group(const BatchCfg& c, const LinearIO* io, const SRTensor* t, uint64_t seed,
                               uint32_t step, unsigned long long* counters, uint8_t* ws,
                               const BwdPlan& P, const int* first, Group<EpiScale>* gx,
                               hipStream_t stream) {
  constexpr bool TR = DW_TRANS != 0;
  Group<EpiSR<CF, TR>> gw{};
  fill_dw(c, io, ws, P, first, gw, [&](int l) {
    EpiSR<CF, TR> e;
    e.wq = t[l].wq;
    e.ldc = io[l].d_in / 8 * chunk_code_bytes<CF>();
    e.d_in = io[l].d_in;
    e.c = t[l].c;
    e.L = (float)(t[l].qmax - t[l].qmin + 1);
    e.qmin = t[l].qmin;
    e.qmax = t[l].qmax;
    e.k0 = (uint32_t)seed;
    e.k1 = (uint32_t)(seed >> 32);
    e.step = step;
    e.tid = t[l].tensor_id;
    e.counters = counters;
    return e;
  });
  if constexpr (TR) {
    // dW^T = X~^T dY: X~^T [d_in][Mp] (K-contiguous) as the first operand,
    // dY [M][d_out] (K-major) as the second
    for (int l = 0; l < c.n; ++l) {
      Prob<EpiSR<CF, TR>>& p = gw.p[l];
      const int64_t I = io[l].d_in, J = io[l].d_out;
      p.A = Opnd{ws + P.xt_off[first[l]], xt_stride(c.M) * 2, I};
      p.B = Opnd{static_cast<const uint8_t*>(io[l].dY), J * 2, J};
      p.I = I;
      p.J = J;
    }
    if (gx != nullptr)
      return launch_dual<EBF16, KC, KM, KB_BWD, EpiSR<CF, TR>, EBF16, KC, KC, KB_BWD, EpiScale>(gw, *gx, ws, stream);
    return launch_group<EBF16, KC, KM, KB_BWD, EpiSR<CF, TR>>(gw, ws, stream);
  } else {
    if (gx != nullptr)
      return launch_dual<EBF16, KM, KC, KB_BWD, EpiSR<CF>, EBF16, KC, KC, KB_BWD, EpiScale>(gw, *gx, ws, stream);
    return launch_group<EBF16, KM, KC, KB_BWD, EpiSR<CF>>(gw, ws, stream);
  }
}

hipError_t launch_bwd_sr_batch(const BatchCfg& c, const LinearIO* io, const SRTensor* t, uint64_t seed,
                               uint32_t step, unsigned long long* counters, bool with_dx, uint8_t* ws,
                               const BwdPlan& P, hipStream_t stream) {
  if (c.n == 0 || c.M == 0) return hipSuccess;
  if (with_dx && c.w_ternary && DX_PACKED_B) {
    const hipError_t e = launch_dx_batch(c, io, ws, P, stream);
    if (e != hipSuccess) return e;
    with_dx = false;
  }
  BwdPlan Q = P;
  Q.splits = with_dx ? P.splits_dual : P.splits;
  const bool fused = with_dx ? P.sr_fused_dual : P.sr_fused;
  Group<EpiScale> gx{};
  LaunchStatus st;
  if (with_dx) prep_dx(c, io, ws, Q, stream, gx, st);
  int first[kMaxBatch];
  prep_xt(c, io, ws, Q, stream, first, st);
  if (Q.splits == 1 && fused) {
    Group<EpiScale>* const pgx = with_dx ? &gx : nullptr;
    if (c.w_ternary) st << launch_dw_sr_group<CF_T2>(c, io, t, seed, step, counters, ws, Q, first, pgx, stream);
    else if (c.w_int4) st << launch_dw_sr_group<CF_I4>(c, io, t, seed, step, counters, ws, Q, first, pgx, stream);
    else if (c.w_int3) st << launch_dw_sr_group<CF_I3>(c, io, t, seed, step, counters, ws, Q, first, pgx, stream);
    else st << launch_dw_sr_group<CF_I8>(c, io, t, seed, step, counters, ws, Q, first, pgx, stream);
    return st.e;
  }
  Group<EpiPartial> gw{};
  fill_dw(c, io, ws, Q, first, gw, [&](int l) {
    const int64_t I = io[l].d_out, J = io[l].d_in;
    return EpiPartial{reinterpret_cast<float*>(ws + Q.part_off[l]), J, I * J};
  });
  if (with_dx)
    st << launch_dual<EBF16, KM, KC, KB_BWD, EpiPartial, EBF16, KC, KC, KB_BWD, EpiScale>(gw, gx, ws, stream);
  else
    st << launch_group<EBF16, KM, KC, KB_BWD, EpiPartial>(gw, ws, stream);
  if (st.e != hipSuccess) return st.e;
  return reduce_sr(c, io, t, seed, step, counters, ws, Q, stream);
}

}  // namespace dqt
