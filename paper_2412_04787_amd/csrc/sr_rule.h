// The direct stochastic-rounding rule of DQT (Sec. 3.1 Eq. 1, Sec. 3.2
// Eq. 5) on the device, and the Philox4x32-10 counter-based generator that
// feeds it: shared by the streaming update kernel and the dW GEMM's fused
// update epilogue, so both give the same codes for the same gradients.
#pragma once

#include "dqt_launch.h"

namespace dqt {

// a ^ b ^ k in one instruction (k is wave-uniform).
__device__ __forceinline__ uint32_t xor3(uint32_t a, uint32_t b, uint32_t k) {
  uint32_t r;
  asm("v_bitop3_b32 %0, %1, %2, %3 bitop3:0x96" : "=v"(r) : "v"(a), "v"(b), "s"(k));
  return r;
}

// Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11).  The key is
// uniform across the grid, so its schedule stays in scalar registers.
__device__ __forceinline__ uint4 philox10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4(xor3((uint32_t)(p1 >> 32), c.y, k0), (uint32_t)p1,
                   xor3((uint32_t)(p0 >> 32), c.w, k1), (uint32_t)p0);
    k0 += 0x9E3779B9u;
    k1 += 0xBB67AE85u;
  }
  return c;
}

// 16-bit draws for the 8 elements of block `blk` (elements 8*blk .. 8*blk+7)
// from stream s: element j takes word j >> 1, low half for even j.
__device__ __forceinline__ uint4 philox_block(uint64_t blk, uint32_t s, uint32_t step,
                                              uint32_t tid, uint32_t k0, uint32_t k1) {
  return philox10(make_uint4((uint32_t)blk, (uint32_t)(blk >> 32) | (s << 31), step, tid), k0, k1);
}
__device__ __forceinline__ uint32_t half16(uint4 w, int j) {
  const uint32_t word = (j >> 1) == 0 ? w.x : (j >> 1) == 1 ? w.y : (j >> 1) == 2 ? w.z : w.w;
  return (j & 1) ? (word >> 16) : (word & 0xFFFFu);
}

struct SRArgs {
  float c;        // lr / alpha, rounded once to fp32
  float L;        // |delta| clamp: qmax - qmin + 1 (any larger move saturates)
  int qmin, qmax;
  uint32_t k0, k1, step, tid;
};

// One element, the full rule, for a step delta in grid units (x = q +
// delta; an infinite delta saturates).  Returns the new code; sets `tie`
// when the primary 16-bit draw equals the top 16 bits of the threshold (the
// secondary draw decides).  n = trunc(delta); r = delta - n (exact); the
// move to the far side (q + n + sign(r)) happens iff U < T = ceil(|r| 2^32).
__device__ __forceinline__ int sr_one_d(int q, float delta_raw, uint32_t p16, const SRArgs& a,
                                        bool& tie) {
  const float delta = fminf(fmaxf(delta_raw, -a.L), a.L);
  const float n = truncf(delta);
  const float r = delta - n;
  const uint32_t T = (uint32_t)ceilf(fabsf(r) * 4294967296.0f);
  const uint32_t thi = T >> 16;
  tie = (p16 == thi) && (T != 0u);
  const bool move = p16 < thi;
  const int v = q + (int)n + (move ? (r > 0.0f ? 1 : -1) : 0);
  return min(max(v, a.qmin), a.qmax);
}
// The plain update's element: delta = -c g; a non-finite g keeps q.
__device__ __forceinline__ int sr_one(int q, float g, uint32_t p16, const SRArgs& a,
                                      bool& tie, bool& nonfinite) {
  nonfinite = (__float_as_uint(g) & 0x7F800000u) == 0x7F800000u;
  const int v = sr_one_d(q, -(a.c * g), p16, a, tie);
  tie = tie && !nonfinite;
  return nonfinite ? q : v;
}

// Secondary decision for a tie element: move iff S16 < (T & 0xFFFF).
__device__ __forceinline__ int sr_tie_d(int q, float delta_raw, uint32_t s16, const SRArgs& a) {
  const float delta = fminf(fmaxf(delta_raw, -a.L), a.L);
  const float n = truncf(delta);
  const float r = delta - n;
  const uint32_t T = (uint32_t)ceilf(fabsf(r) * 4294967296.0f);
  const bool move = s16 < (T & 0xFFFFu);
  const int v = q + (int)n + (move ? (r > 0.0f ? 1 : -1) : 0);
  return min(max(v, a.qmin), a.qmax);
}
__device__ __forceinline__ int sr_tie(int q, float g, uint32_t s16, const SRArgs& a) {
  return sr_tie_d(q, -(a.c * g), s16, a);
}

// The same rule in fewer instructions, for a finite delta and no tie:
//  * delta = med3(delta, -L, L); n = (int)delta truncates toward zero;
//  * |r| = fract(|delta|) (exact: |delta| - floor(|delta|));
//  * with P = (p16 << 16) | 0xFFFF, p16 < (T >> 16) iff P < T, and
//    p16 == (T >> 16) iff (P - T) mod 2^32 <= 0xFFFF;
//  * F = floor(|r| 2^32) (the conversion truncates) is T or T - 1, and
//    P < F decides as P < T does whenever (P - F) mod 2^32 > 0xFFFF: the two
//    differ only at P = F = T - 1, and P - T = 0xFFFF (T's low half zero, so
//    no draw is below T) is decided P >= T by both.  So the running minimum
//    of P - F flags every element the secondary draw may have to decide.
// `code` is q plus a per-format offset and [lo, hi] the offset range (one
// median-of-three clamps).
__device__ __forceinline__ int sr_fast_d(int code, float delta_raw, uint32_t P, float L, int lo,
                                         int hi, uint32_t& tiemin) {
  const float delta = __builtin_amdgcn_fmed3f(delta_raw, -L, L);
  const int n = (int)delta;
  const float ar = __builtin_amdgcn_fractf(fabsf(delta));
  const uint32_t F = (uint32_t)(ar * 4294967296.0f);
  tiemin = min(tiemin, P - F);
  const int sgn = ((int)__float_as_uint(delta) >> 31) | 1;
  const int v = code + n + (P < F ? sgn : 0);
  int r;
  asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(v), "v"(lo), "v"(hi));
  return r;
}
// The plain update (delta = -c g = nc g).
__device__ __forceinline__ int sr_fast(int code, float g, uint32_t P, float nc, float L, int lo,
                                       int hi, uint32_t& tiemin) {
  return sr_fast_d(code, nc * g, P, L, lo, hi, tiemin);
}

// Code formats of the weights: CF_I8 one byte per weight (two's complement),
// CF_T2 2-bit ternary (code q + 1 at bits 2k of the chunk's first word),
// CF_I4 two's-complement nibbles (weight k at bits 4 (k mod 8) of word k / 8),
// CF_I3 3-bit two's-complement fields, 8 weights in 3 bytes (weight k at
// bits 3 k of the chunk's 24-bit little-endian group).
// A chunk's codes sit in words w[0 .. 3]; `field` is what the fast rule
// moves (q + off, clamped to [qmin + off, qmax + off]).
constexpr int CF_I8 = 0, CF_T2 = 1, CF_I4 = 2, CF_I3 = 3;
// small steps of 4-bit and 3-bit codes in lane arithmetic (1), or each
// weight by the fast rule (0; int8 codes always: their bytes extract in one
// instruction, and the lane form measured 9 % slower for them)
#ifndef SR_INT_SMALL
#define SR_INT_SMALL 1
#endif
// Bytes of codes per chunk of 8 weights.
template <int CF>
constexpr int chunk_code_bytes() { return CF == CF_T2 ? 2 : CF == CF_I3 ? 3 : CF == CF_I4 ? 4 : 8; }
template <int CF>
struct CodeFmt {
  static constexpr int off = CF == CF_T2 ? 1 : 0;
  __device__ static int field(const uint32_t (&w)[4], int j) {
    if constexpr (CF == CF_T2) return (int)((w[0] >> (2 * j)) & 3u);
    else if constexpr (CF == CF_I3) return (int)(w[0] << (29 - 3 * j)) >> 29;
    else if constexpr (CF == CF_I4) return (int)(w[j >> 3] << (28 - 4 * (j & 7))) >> 28;
    else return (int)(int8_t)(w[j >> 2] >> (8 * (j & 3)));
  }
  __device__ static int q_of(const uint32_t (&w)[4], int j) { return field(w, j) - off; }
  // ORs field v of weight j into zeroed words
  __device__ static void put(uint32_t (&w)[4], int j, int v) {
    if constexpr (CF == CF_T2) w[0] |= (uint32_t)v << (2 * j);
    else if constexpr (CF == CF_I3) w[0] |= ((uint32_t)v & 7u) << (3 * j);
    else if constexpr (CF == CF_I4) w[j >> 3] |= ((uint32_t)v & 0xFu) << (4 * (j & 7));
    else w[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
  }
  // replaces field j by v
  __device__ static void set(uint32_t (&w)[4], int j, int v) {
    if constexpr (CF == CF_T2) w[0] = (w[0] & ~(3u << (2 * j))) | ((uint32_t)v << (2 * j));
    else if constexpr (CF == CF_I3) w[0] = (w[0] & ~(7u << (3 * j))) | (((uint32_t)v & 7u) << (3 * j));
    else if constexpr (CF == CF_I4)
      w[j >> 3] = (w[j >> 3] & ~(0xFu << (4 * (j & 7)))) | (((uint32_t)v & 0xFu) << (4 * (j & 7)));
    else w[j >> 2] = (w[j >> 2] & ~(0xFFu << (8 * (j & 3)))) | (((uint32_t)v & 0xFFu) << (8 * (j & 3)));
  }
  // number of weights whose code differs, over a chunk of CW weights
  template <int CW>
  __device__ static uint32_t changed(const uint32_t (&a)[4], const uint32_t (&b)[4]) {
    uint32_t n = 0;
    if constexpr (CF == CF_T2) {
      const uint32_t x = a[0] ^ b[0];
      n = __builtin_popcount((x | (x >> 1)) & 0x55555555u);
    } else if constexpr (CF == CF_I3) {
      const uint32_t x = a[0] ^ b[0];
      n = __builtin_popcount((x | (x >> 1) | (x >> 2)) & 0x00249249u);
    } else if constexpr (CF == CF_I4) {
#pragma unroll
      for (int w = 0; w < (CW + 7) / 8; ++w) {   // (fields past CW weights are zero in both)
        const uint32_t x = a[w] ^ b[w];
        n += __builtin_popcount((x | (x >> 1) | (x >> 2) | (x >> 3)) & 0x11111111u);
      }
    } else {
#pragma unroll
      for (int w = 0; w < CW / 4; ++w) {
        const uint32_t x = a[w] ^ b[w];
        n += __builtin_popcount((((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x) & 0x80808080u);
      }
    }
    return n;
  }
};

// The codes of chunk t (8 consecutive weights, chunk_code_bytes<CF>() bytes
// from byte t * that) of a code array, into / from words w[0 .. 1].  Lanes
// own whole chunks, so no two lanes write one byte.  3-byte chunks are
// moved a byte at a time (their alignment varies).
template <int CF>
struct ChunkIO {
  static constexpr int NB = chunk_code_bytes<CF>();
  __device__ static void load(const uint8_t* wq, int64_t t, uint32_t (&w)[4]) {
    if constexpr (NB == 2) {
      w[0] = reinterpret_cast<const uint16_t*>(wq)[t];
    } else if constexpr (NB == 3) {
      const uint8_t* p = wq + 3 * t;
      w[0] = (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16);
    } else if constexpr (NB == 4) {
      w[0] = reinterpret_cast<const uint32_t*>(wq)[t];
    } else {
      const uint2 v = reinterpret_cast<const uint2*>(wq)[t];
      w[0] = v.x;
      w[1] = v.y;
    }
  }
  __device__ static void store(uint8_t* wq, int64_t t, const uint32_t (&w)[4]) {
    if constexpr (NB == 2) {
      reinterpret_cast<uint16_t*>(wq)[t] = (uint16_t)w[0];
    } else if constexpr (NB == 3) {
      uint8_t* p = wq + 3 * t;
      p[0] = (uint8_t)w[0];
      p[1] = (uint8_t)(w[0] >> 8);
      p[2] = (uint8_t)(w[0] >> 16);
    } else if constexpr (NB == 4) {
      reinterpret_cast<uint32_t*>(wq)[t] = w[0];
    } else {
      reinterpret_cast<uint2*>(wq)[t] = make_uint2(w[0], w[1]);
    }
  }
};

// Ternary codes, a chunk of 8 weights whose steps all satisfy |delta| < 1
// (the usual case: the step sizes of training are a small fraction of a grid
// step), in mask arithmetic.  With n = trunc(delta) = 0 the rule moves q one
// step in the direction of delta iff U < T = ceil(|delta| 2^32).  Let
// h = floor(|delta| 2^16) (exact: |delta| 2^16 = |c 2^16 g| is the rounded
// product scaled by a power of two, and products too small for that to hold
// give h = 0 either way).  A draw with p16 < h moves (U < 2^16 (p16 + 1) <=
// 2^16 h <= T); one with p16 > h does not (U >= 2^16 (h + 1) >= T); p16 = h
// is left to the full rule, which reads the secondary draw.  The moves and
// the signs of delta become bit masks (bit j for weight j), spread to the
// 2-bit fields, and the fields are stepped up (not past code 2) or down (not
// below code 0) by one masked add and one masked subtract.  Returns false,
// with nothing changed, when the chunk holds a step of 1 or more, a
// non-finite gradient, a tie or an invalid code 3: the full rule decides it.
// The moves of a chunk of 8 weights whose steps all satisfy |delta| < 1, as
// bit masks (bit j for weight j): mv, the weights that move one step; up,
// those whose delta is positive.  False when some |delta| >= 1, a gradient
// is not finite or a draw ties (p16 = h).
__device__ __forceinline__ bool small_moves(const f32x4 (&gv)[2], uint4 r, float c, uint32_t& mv,
                                            uint32_t& up) {
  // x = c g 2^16 = -delta 2^16, exact (|c| < 2^100 checked by the caller)
  const float cs = c * 65536.0f;
  float x[8];
#pragma unroll
  for (int j = 0; j < 8; ++j) x[j] = cs * gv[j >> 2][j & 3];
  // largest |x| of the chunk; NaN propagates (IEEE maximum)
  float m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(fabsf(x[0]), fabsf(x[1])), fabsf(x[2]));
  m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(m, fabsf(x[3])), fabsf(x[4]));
  m = __builtin_elementwise_maximum(__builtin_elementwise_maximum(m, fabsf(x[5])), fabsf(x[6]));
  m = __builtin_elementwise_maximum(m, fabsf(x[7]));
  if (!(m < 65536.0f)) return false;
  // bit j of mv: p16 < h (p16 - h < 0, both below 2^16); bit j of up: x < 0
  // (delta > 0); dmin = 0 iff some p16 = h
  uint32_t dmin = 0xFFFFFFFFu;
  mv = 0;
  up = 0;
#pragma unroll
  for (int j = 7; j >= 0; --j) {
    const uint32_t word = (j >> 1) == 0 ? r.x : (j >> 1) == 1 ? r.y : (j >> 1) == 2 ? r.z : r.w;
    const uint32_t p = (j & 1) ? (word >> 16) : (word & 0xFFFFu);
    uint32_t h;
    asm("v_cvt_u32_f32_e64 %0, |%1|" : "=v"(h) : "v"(x[j]));   // floor(|x|), |x| < 2^16
    const uint32_t d = p - h;
    dmin = min(dmin, d);
    mv = __builtin_amdgcn_alignbit(mv, d, 31);
    up = __builtin_amdgcn_alignbit(up, __float_as_uint(x[j]), 31);
  }
  return dmin != 0u;
}

template <class Count>
__device__ __forceinline__ bool sr_chunk_t2_small(uint32_t code, const f32x4 (&gv)[2], uint4 r, float c,
                                                  uint32_t& out, Count& changed) {
  uint32_t mv, up_dir;
  if (!small_moves(gv, r, c, mv, up_dir) || (code & (code >> 1) & 0x5555u) != 0u) return false;
  auto spread = [](uint32_t v) {            // bit j -> bit 2 j (8 bits)
    v = (v | (v << 4)) & 0x0F0Fu;
    v = (v | (v << 2)) & 0x3333u;
    return (v | (v << 1)) & 0x5555u;
  };
  const uint32_t M = spread(mv), U = spread(up_dir);
  const uint32_t up = M & U & ~(code >> 1);                        // not from code 2
  const uint32_t dn = M & ~U & (code | (code >> 1)) & 0x5555u;    // not from code 0
  out = code + up - dn;
  changed += __builtin_popcount(up | dn);
  return true;
}

// The same for two's-complement codes of B = 4 or 3 bits (CF_I4: one word
// of eight nibbles; CF_I3: eight 3-bit fields in the low 24 bits).  Codes
// are offset to u = q + 2^(B-1) (`bias`) and the fields of even and odd
// weights split into two words whose lanes have room above each field (8-
// and 6-bit lanes), so that sums carry no
// further than their own lane: a field is nonzero iff field + (2^(w-1) - 1)
// sets the lane's top bit (w the lane width), u > H iff u + 2^(w-1) - 1 - H
// does, and u < L iff u + 2^(w-1) - L does not.  A moving weight steps up
// unless at qmax, down unless at qmin, by one masked add and one masked
// subtract per lane word.  False (nothing changed) when the moves are not
// all small (small_moves) or a code lies outside [qmin, qmax], which the
// full rule clamps.
template <int CF>
struct SwarFmt;
template <>
struct SwarFmt<CF_I4> {   // lanes of 8 bits; words: even nibbles, odd nibbles
  static constexpr int W = 8, bias = 8;
  static constexpr uint32_t rep = 0x01010101u, off = 0x88888888u, lmask = 0x0F0F0F0Fu;
  __device__ static void split(const uint32_t (&w)[4], uint32_t (&x)[2]) {
    const uint32_t o = w[0] ^ off;
    x[0] = o & lmask;
    x[1] = (o >> 4) & lmask;
  }
  __device__ static uint32_t lanes(uint32_t v, int l) {   // bits l, l + 2, l + 4, l + 6 -> 0, 8, 16, 24
    return (((v >> l) & 0x55u) * 0x41041u) & rep;
  }
  __device__ static void join(const uint32_t (&x)[2], uint32_t (&w)[4]) {
    w[0] = (x[0] | (x[1] << 4)) ^ off;
    w[1] = w[2] = w[3] = 0u;
  }
};
template <>
struct SwarFmt<CF_I3> {   // lanes of 6 bits; words: even fields, odd fields
  static constexpr int W = 6, bias = 4;
  static constexpr uint32_t rep = 0x00041041u, off = 0x00924924u, lmask = 0x001C71C7u;
  __device__ static void split(const uint32_t (&w)[4], uint32_t (&x)[2]) {
    const uint32_t o = w[0] ^ off;
    x[0] = o & lmask;
    x[1] = (o >> 3) & lmask;
  }
  __device__ static uint32_t lanes(uint32_t v, int l) {   // bits l, l + 2, l + 4, l + 6 -> 0, 6, 12, 18
    const uint32_t b = v >> l;
    return (b & 1u) | ((b & 4u) << 4) | ((b & 0x10u) << 8) | ((b & 0x40u) << 12);
  }
  __device__ static void join(const uint32_t (&x)[2], uint32_t (&w)[4]) {
    w[0] = (x[0] | (x[1] << 3)) ^ off;
    w[1] = w[2] = w[3] = 0u;
  }
};

template <int CF, class Count>
__device__ __forceinline__ bool sr_chunk_int_small(const uint32_t (&win)[4], const f32x4 (&gv)[2], uint4 r,
                                                   const SRArgs& a, uint32_t (&wout)[4], Count& changed) {
  using S = SwarFmt<CF>;
  uint32_t mv, up_dir;
  if (!small_moves(gv, r, a.c, mv, up_dir)) return false;
  constexpr uint32_t half = 1u << (S::W - 1);             // a lane's top bit
  constexpr uint32_t top = S::rep * half;
  const uint32_t lo = (uint32_t)(a.qmin + S::bias), hi = (uint32_t)(a.qmax + S::bias);
  uint32_t x[2];
  S::split(win, x);
  uint32_t bad = 0;
#pragma unroll
  for (int l = 0; l < 2; ++l)
    bad |= (x[l] + S::rep * (half - 1u - hi)) | ~(x[l] + S::rep * (half - lo));
  if ((bad & top) != 0u) return false;
  uint32_t moved = 0;
#pragma unroll
  for (int l = 0; l < 2; ++l) {
    const uint32_t m = S::lanes(mv, l), u = S::lanes(up_dir, l);
    const uint32_t not_hi = (((x[l] ^ (S::rep * hi)) + S::rep * (half - 1u)) & top) >> (S::W - 1);
    const uint32_t not_lo = (((x[l] ^ (S::rep * lo)) + S::rep * (half - 1u)) & top) >> (S::W - 1);
    const uint32_t up = m & u & not_hi, dn = m & ~u & not_lo;
    x[l] = x[l] + up - dn;
    moved += __builtin_popcount(up | dn);
  }
  S::join(x, wout);
  changed += moved;
  return true;
}

// The update of one chunk of CW consecutive weights, elements
// 8 blk .. 8 blk + CW - 1 of their tensor (CW / 8 Philox blocks): codes `win`
// (format CF), gradients gv.  Writes the new codes to `wout` and adds the
// changed and non-finite counts.
template <int CF, int CW, class Count>
__device__ __forceinline__ void sr_chunk(const uint32_t (&win)[4], const f32x4 (&gv)[CW / 4], uint64_t blk,
                                         const SRArgs& a, uint32_t (&wout)[4], Count& changed,
                                         Count& nonfin) {
  using F = CodeFmt<CF>;
  constexpr int NG = CW / 4, NB = CW / 8;
  uint4 r[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) r[b] = philox_block(blk + b, 0u, a.step, a.tid, a.k0, a.k1);
  if constexpr (CF == CF_T2 && CW == 8) {
    if (fabsf(a.c) < 0x1p100f) {
      uint32_t o;
      if (sr_chunk_t2_small(win[0], gv, r[0], a.c, o, changed)) {
        wout[0] = o;
        wout[1] = wout[2] = wout[3] = 0u;
        return;
      }
    }
  } else if constexpr (CW == 8 && SR_INT_SMALL && (CF == CF_I4 || CF == CF_I3)) {
    if (fabsf(a.c) < 0x1p100f && sr_chunk_int_small<CF>(win, gv, r[0], a, wout, changed)) return;
  }

  // finite check: a product chain stays finite unless some g is inf/NaN
  // (or a product overflows, which only sends the chunk to the full rule)
  float probe = 0.0f;
#pragma unroll
  for (int u = 0; u < NG; ++u) {
    probe = __builtin_fmaf(gv[u][0], gv[u][1], probe);
    probe = __builtin_fmaf(gv[u][2], gv[u][3], probe);
  }
  uint32_t tiemin = 0xFFFFFFFFu;
  const float nc = -a.c;
#pragma unroll
  for (int w = 0; w < 4; ++w) wout[w] = 0;
#pragma unroll
  for (int j = 0; j < CW; ++j) {
    const float g = gv[j >> 2][j & 3];
    const uint4& rb = r[j >> 3];
    const uint32_t word = ((j >> 1) & 3) == 0 ? rb.x : ((j >> 1) & 3) == 1 ? rb.y : ((j >> 1) & 3) == 2 ? rb.z : rb.w;
    const uint32_t P = (j & 1) ? (word | 0xFFFFu) : ((word << 16) | 0xFFFFu);
    const int v = sr_fast(F::field(win, j), g, P, nc, a.L, a.qmin + F::off, a.qmax + F::off, tiemin);
    F::put(wout, j, v);
  }
  if (tiemin <= 0xFFFFu || !__builtin_isfinite(probe)) {
    // rare (about CW / 65536 per chunk, or a non-finite gradient): full
    // rule, in two passes over the chunk (ties and non-finite entries, then
    // the codes), so no per-element arrays stay live
    uint32_t ties = 0;
#pragma unroll
    for (int j = 0; j < CW; ++j) {
      bool tie, nf;
      (void)sr_one(F::q_of(win, j), gv[j >> 2][j & 3], half16(r[j >> 3], j & 7), a, tie, nf);
      ties |= (tie ? 1u : 0u) << j;
      nonfin += nf ? 1 : 0;
    }
#pragma unroll
    for (int w = 0; w < 4; ++w) wout[w] = 0;
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const uint32_t tb = (ties >> (8 * b)) & 0xFFu;
      const uint4 sb = tb ? philox_block(blk + b, 1u, a.step, a.tid, a.k0, a.k1) : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
      for (int j = 8 * b; j < 8 * b + 8; ++j) {
        bool tie, nf;
        const int v = (tb >> (j & 7)) & 1u
                          ? sr_tie(F::q_of(win, j), gv[j >> 2][j & 3], half16(sb, j & 7), a)
                          : sr_one(F::q_of(win, j), gv[j >> 2][j & 3], half16(r[j >> 3], j & 7), a, tie, nf);
        F::put(wout, j, v + F::off);
      }
    }
  }
  changed += F::template changed<CW>(wout, win);
}

// One chunk of 8 consecutive weights (elements 8 blk .. 8 blk + 7, one
// Philox block) moved by given steps delta[j] in grid units; bit j of `bad`
// keeps code j (counted as non-finite; its delta must be 0).  Codes as in
// sr_chunk.
template <int CF, class Count>
__device__ __forceinline__ void sr_chunk_delta(const uint32_t (&win)[4], const float (&delta)[8], uint32_t bad,
                                               uint64_t blk, const SRArgs& a, uint32_t (&wout)[4],
                                               Count& changed, Count& nonfin) {
  using F = CodeFmt<CF>;
  const uint4 r = philox_block(blk, 0u, a.step, a.tid, a.k0, a.k1);
  uint32_t tiemin = 0xFFFFFFFFu;
#pragma unroll
  for (int w = 0; w < 4; ++w) wout[w] = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t word = (j >> 1) == 0 ? r.x : (j >> 1) == 1 ? r.y : (j >> 1) == 2 ? r.z : r.w;
    const uint32_t P = (j & 1) ? (word | 0xFFFFu) : ((word << 16) | 0xFFFFu);
    const int v = sr_fast_d(F::field(win, j), delta[j], P, a.L, a.qmin + F::off, a.qmax + F::off, tiemin);
    F::put(wout, j, v);
  }
  if (tiemin <= 0xFFFFu) {
    // rare: full rule (a kept element has delta 0, which the rule keeps)
    uint32_t ties = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      bool tie;
      (void)sr_one_d(F::q_of(win, j), delta[j], half16(r, j), a, tie);
      ties |= (tie ? 1u : 0u) << j;
    }
    const uint4 sb = ties ? philox_block(blk, 1u, a.step, a.tid, a.k0, a.k1) : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int w = 0; w < 4; ++w) wout[w] = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      bool tie;
      const int v = (ties >> j) & 1u ? sr_tie_d(F::q_of(win, j), delta[j], half16(sb, j), a)
                                     : sr_one_d(F::q_of(win, j), delta[j], half16(r, j), a, tie);
      F::put(wout, j, v + F::off);
    }
  }
  nonfin += __builtin_popcount(bad);
  changed += F::template changed<8>(wout, win);
}

}  // namespace dqt
