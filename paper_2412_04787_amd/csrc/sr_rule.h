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

// The update of one chunk of CW consecutive weights, elements
// 8 blk .. 8 blk + CW - 1 of their tensor (CW / 8 Philox blocks): codes `win`
// (ternary: 2 CW bits in win[0]; int8: CW / 4 words), gradients gv.  Writes
// the new codes to `wout` and adds the changed and non-finite counts.
template <bool TERNARY, int CW, class Count>
__device__ __forceinline__ void sr_chunk(const uint32_t (&win)[4], const f32x4 (&gv)[CW / 4], uint64_t blk,
                                         const SRArgs& a, uint32_t (&wout)[4], Count& changed,
                                         Count& nonfin) {
  constexpr int NG = CW / 4, NB = CW / 8;
  uint4 r[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) r[b] = philox_block(blk + b, 0u, a.step, a.tid, a.k0, a.k1);

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
    if constexpr (TERNARY) {
      const int code = (int)((win[0] >> (2 * j)) & 3u);
      const int v = sr_fast(code, g, P, nc, a.L, a.qmin + 1, a.qmax + 1, tiemin);
      wout[0] |= (uint32_t)v << (2 * j);
    } else {
      const int code = (int)(int8_t)(win[j >> 2] >> (8 * (j & 3)));
      const int v = sr_fast(code, g, P, nc, a.L, a.qmin, a.qmax, tiemin);
      wout[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
    }
  }
  if (tiemin <= 0xFFFFu || !__builtin_isfinite(probe)) {
    // rare (about CW / 65536 per chunk, or a non-finite gradient): full
    // rule, in two passes over the chunk (ties and non-finite entries, then
    // the codes), so no per-element arrays stay live
    auto q_of = [&](int j) {
      return TERNARY ? (int)((win[0] >> (2 * j)) & 3u) - 1 : (int)(int8_t)(win[j >> 2] >> (8 * (j & 3)));
    };
    uint32_t ties = 0;
#pragma unroll
    for (int j = 0; j < CW; ++j) {
      bool tie, nf;
      (void)sr_one(q_of(j), gv[j >> 2][j & 3], half16(r[j >> 3], j & 7), a, tie, nf);
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
                          ? sr_tie(q_of(j), gv[j >> 2][j & 3], half16(sb, j & 7), a)
                          : sr_one(q_of(j), gv[j >> 2][j & 3], half16(r[j >> 3], j & 7), a, tie, nf);
        if constexpr (TERNARY) wout[0] |= (uint32_t)(v + 1) << (2 * j);
        else wout[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
      }
    }
  }
  // changed codes: count differing 2-bit fields or bytes
  if constexpr (TERNARY) {
    const uint32_t x = wout[0] ^ win[0];
    changed += __builtin_popcount((x | (x >> 1)) & 0x55555555u);
  } else {
#pragma unroll
    for (int w = 0; w < CW / 4; ++w) {
      const uint32_t x = wout[w] ^ win[w];
      changed += __builtin_popcount((((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x) & 0x80808080u);
    }
  }
}

// One chunk of 8 consecutive weights (elements 8 blk .. 8 blk + 7, one
// Philox block) moved by given steps delta[j] in grid units; bit j of `bad`
// keeps code j (counted as non-finite; its delta must be 0).  Codes as in
// sr_chunk.
template <bool TERNARY, class Count>
__device__ __forceinline__ void sr_chunk_delta(const uint32_t (&win)[4], const float (&delta)[8], uint32_t bad,
                                               uint64_t blk, const SRArgs& a, uint32_t (&wout)[4],
                                               Count& changed, Count& nonfin) {
  const uint4 r = philox_block(blk, 0u, a.step, a.tid, a.k0, a.k1);
  auto q_of = [&](int j) {
    return TERNARY ? (int)((win[0] >> (2 * j)) & 3u) - 1 : (int)(int8_t)(win[j >> 2] >> (8 * (j & 3)));
  };
  uint32_t tiemin = 0xFFFFFFFFu;
#pragma unroll
  for (int w = 0; w < 4; ++w) wout[w] = 0;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const uint32_t word = (j >> 1) == 0 ? r.x : (j >> 1) == 1 ? r.y : (j >> 1) == 2 ? r.z : r.w;
    const uint32_t P = (j & 1) ? (word | 0xFFFFu) : ((word << 16) | 0xFFFFu);
    if constexpr (TERNARY) {
      const int code = (int)((win[0] >> (2 * j)) & 3u);
      const int v = sr_fast_d(code, delta[j], P, a.L, a.qmin + 1, a.qmax + 1, tiemin);
      wout[0] |= (uint32_t)v << (2 * j);
    } else {
      const int code = (int)(int8_t)(win[j >> 2] >> (8 * (j & 3)));
      const int v = sr_fast_d(code, delta[j], P, a.L, a.qmin, a.qmax, tiemin);
      wout[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
    }
  }
  if (tiemin <= 0xFFFFu) {
    // rare: full rule (a kept element has delta 0, which the rule keeps)
    uint32_t ties = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      bool tie;
      (void)sr_one_d(q_of(j), delta[j], half16(r, j), a, tie);
      ties |= (tie ? 1u : 0u) << j;
    }
    const uint4 sb = ties ? philox_block(blk, 1u, a.step, a.tid, a.k0, a.k1) : make_uint4(0u, 0u, 0u, 0u);
#pragma unroll
    for (int w = 0; w < 4; ++w) wout[w] = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      bool tie;
      const int v = (ties >> j) & 1u ? sr_tie_d(q_of(j), delta[j], half16(sb, j), a)
                                     : sr_one_d(q_of(j), delta[j], half16(r, j), a, tie);
      if constexpr (TERNARY) wout[0] |= (uint32_t)(v + 1) << (2 * j);
      else wout[j >> 2] |= ((uint32_t)v & 0xFFu) << (8 * (j & 3));
    }
  }
  nonfin += __builtin_popcount(bad);
  if constexpr (TERNARY) {
    const uint32_t x = wout[0] ^ win[0];
    changed += __builtin_popcount((x | (x >> 1)) & 0x55555555u);
  } else {
#pragma unroll
    for (int w = 0; w < 2; ++w) {
      const uint32_t x = wout[w] ^ win[w];
      changed += __builtin_popcount((((x & 0x7F7F7F7Fu) + 0x7F7F7F7Fu) | x) & 0x80808080u);
    }
  }
}

}  // namespace dqt
