// Direct stochastic-rounding update of DQT (Sec. 3.1 Eq. 1, Sec. 3.2 Eq. 5)
// and the Philox4x32-10 counter-based generator that feeds it.
//
// Memory-bound streaming kernel: per weight it reads the packed code and the
// fp32 gradient and writes the code back (4.5 B/weight for 2-bit ternary
// codes, 6 B/weight for int8 codes).  Each lane owns 16 consecutive weights:
// 64 contiguous bytes of gradient, and 4 (ternary) or 16 (int8) whole bytes of
// codes, so no two lanes ever touch the same byte.
#include "dqt_launch.h"

namespace dqt {

// Philox4x32 with 10 rounds (Salmon, Moraes, Dror, Shaw, SC'11).  The key is
// uniform across the grid, so its schedule stays in scalar registers.
__device__ __forceinline__ uint4 philox10(uint4 c, uint32_t k0, uint32_t k1) {
#pragma unroll
  for (int r = 0; r < 10; ++r) {
    const uint64_t p0 = (uint64_t)0xD2511F53u * c.x;
    const uint64_t p1 = (uint64_t)0xCD9E8D57u * c.z;
    c = make_uint4((uint32_t)(p1 >> 32) ^ c.y ^ k0, (uint32_t)p1,
                   (uint32_t)(p0 >> 32) ^ c.w ^ k1, (uint32_t)p0);
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

// One element.  Returns the new code; sets `tie` when the primary 16-bit draw
// equals the top 16 bits of the threshold (the secondary draw decides).
// x = q + delta; n = trunc(delta); r = delta - n (exact); the move to the far
// side (q + n + sign(r)) happens iff U < T = ceil(|r| * 2^32).
__device__ __forceinline__ int sr_one(int q, float g, uint32_t p16, const SRArgs& a,
                                      bool& tie, bool& nonfinite) {
  nonfinite = (__float_as_uint(g) & 0x7F800000u) == 0x7F800000u;
  float delta = -(a.c * g);
  delta = fminf(fmaxf(delta, -a.L), a.L);
  const float n = truncf(delta);
  const float r = delta - n;
  const uint32_t T = (uint32_t)ceilf(fabsf(r) * 4294967296.0f);
  const uint32_t thi = T >> 16;
  tie = !nonfinite && (p16 == thi) && (T != 0u);
  const bool move = p16 < thi;
  int v = q + (int)n + (move ? (r > 0.0f ? 1 : -1) : 0);
  v = min(max(v, a.qmin), a.qmax);
  return nonfinite ? q : v;
}

// Secondary decision for a tie element: move iff S16 < (T & 0xFFFF).
__device__ __forceinline__ int sr_tie(int q, float g, uint32_t s16, const SRArgs& a) {
  float delta = -(a.c * g);
  delta = fminf(fmaxf(delta, -a.L), a.L);
  const float n = truncf(delta);
  const float r = delta - n;
  const uint32_t T = (uint32_t)ceilf(fabsf(r) * 4294967296.0f);
  const bool move = s16 < (T & 0xFFFFu);
  int v = q + (int)n + (move ? (r > 0.0f ? 1 : -1) : 0);
  return min(max(v, a.qmin), a.qmax);
}

constexpr int kMaxSR = kMaxBatch;
// Up to kMaxSR tensors in one launch; tensor s owns blocks [b0[s], b0[s+1]).
struct SRTab {
  uint8_t* wq[kMaxSR];
  const float* grad[kMaxSR];
  int64_t nchunks[kMaxSR];
  float c[kMaxSR], L[kMaxSR];
  int qmin[kMaxSR], qmax[kMaxSR];
  uint32_t tid[kMaxSR];
  int32_t b0[kMaxSR + 1];
  int32_t n;
  uint32_t k0, k1, step;
};

template <bool TERNARY>
__global__ __launch_bounds__(256) void sr_update_kernel(const SRTab tab,
                                                        unsigned long long* __restrict__ counters) {
  int sidx = 0;
  while (sidx + 1 < tab.n && (int)blockIdx.x >= tab.b0[sidx + 1]) ++sidx;
  SRArgs a;
  a.c = tab.c[sidx];
  a.L = tab.L[sidx];
  a.qmin = tab.qmin[sidx];
  a.qmax = tab.qmax[sidx];
  a.k0 = tab.k0;
  a.k1 = tab.k1;
  a.step = tab.step;
  a.tid = tab.tid[sidx];
  uint8_t* __restrict__ wq = tab.wq[sidx];
  const float* __restrict__ grad = tab.grad[sidx];
  unsigned long long changed = 0, nonfin = 0;
  const int64_t t = (int64_t)(blockIdx.x - tab.b0[sidx]) * blockDim.x + threadIdx.x;
  if (t < tab.nchunks[sidx]) {
    const f32x4* gp = reinterpret_cast<const f32x4*>(grad + t * 16);
    f32x4 gv[4];
#pragma unroll
    for (int u = 0; u < 4; ++u) gv[u] = __builtin_nontemporal_load(gp + u);
    int q[16];
    if constexpr (TERNARY) {
      const uint32_t packed = reinterpret_cast<const uint32_t*>(wq)[t];
#pragma unroll
      for (int j = 0; j < 16; ++j) q[j] = (int)((packed >> (2 * j)) & 3u) - 1;
    } else {
      const uint4 packed8 = reinterpret_cast<const uint4*>(wq)[t];
      const uint32_t w4[4] = {packed8.x, packed8.y, packed8.z, packed8.w};
#pragma unroll
      for (int j = 0; j < 16; ++j) q[j] = (int)(int8_t)(w4[j >> 2] >> (8 * (j & 3)));
    }
    const uint64_t blk = (uint64_t)t * 2;
    const uint4 r0 = philox_block(blk, 0u, a.step, a.tid, a.k0, a.k1);
    const uint4 r1 = philox_block(blk + 1, 0u, a.step, a.tid, a.k0, a.k1);
    int nq[16];
    uint32_t ties = 0;
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      const float g = gv[j >> 2][j & 3];
      const uint32_t p16 = half16(j < 8 ? r0 : r1, j & 7);
      bool tie, nf;
      nq[j] = sr_one(q[j], g, p16, a, tie, nf);
      ties |= (tie ? 1u : 0u) << j;
      nonfin += nf ? 1 : 0;
    }
    if (ties) {  // probability ~2^-16 per element: decide with stream 1
      const uint4 s0 = philox_block(blk, 1u, a.step, a.tid, a.k0, a.k1);
      const uint4 s1 = philox_block(blk + 1, 1u, a.step, a.tid, a.k0, a.k1);
#pragma unroll
      for (int j = 0; j < 16; ++j) {
        if (ties & (1u << j)) {
          const float g = gv[j >> 2][j & 3];
          nq[j] = sr_tie(q[j], g, half16(j < 8 ? s0 : s1, j & 7), a);
        }
      }
    }
#pragma unroll
    for (int j = 0; j < 16; ++j) changed += (nq[j] != q[j]) ? 1 : 0;
    if constexpr (TERNARY) {
      uint32_t out = 0;
#pragma unroll
      for (int j = 0; j < 16; ++j) out |= (uint32_t)(nq[j] + 1) << (2 * j);
      reinterpret_cast<uint32_t*>(wq)[t] = out;
    } else {
      uint32_t o[4] = {0, 0, 0, 0};
#pragma unroll
      for (int j = 0; j < 16; ++j) o[j >> 2] |= ((uint32_t)nq[j] & 0xFFu) << (8 * (j & 3));
      reinterpret_cast<uint4*>(wq)[t] = make_uint4(o[0], o[1], o[2], o[3]);
    }
  }
  if (counters != nullptr) {
    changed = wave_sum_u64(changed);
    nonfin = wave_sum_u64(nonfin);
    if ((threadIdx.x & (kWave - 1)) == 0) {
      if (changed) atomicAdd(counters + 0, changed);
      if (nonfin) atomicAdd(counters + 1, nonfin);
    }
  }
}

__global__ __launch_bounds__(256) void debug_rng_kernel(uint32_t* __restrict__ out, uint64_t i0,
                                                        int64_t n, uint32_t k0, uint32_t k1,
                                                        uint32_t step, uint32_t tid) {
  const int64_t stride = (int64_t)gridDim.x * blockDim.x;
  for (int64_t t = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; t < n; t += stride) {
    const uint64_t i = i0 + (uint64_t)t;
    const uint4 p = philox_block(i >> 3, 0u, step, tid, k0, k1);
    const uint4 s = philox_block(i >> 3, 1u, step, tid, k0, k1);
    const int j = (int)(i & 7);
    out[t] = (half16(p, j) << 16) | half16(s, j);
  }
}

hipError_t launch_sr_update(bool ternary, int n, const SRTensor* t, uint64_t seed, uint32_t step,
                            unsigned long long* counters, hipStream_t stream) {
  SRTab tab{};
  tab.n = n;
  tab.k0 = (uint32_t)seed;
  tab.k1 = (uint32_t)(seed >> 32);
  tab.step = step;
  int32_t blocks = 0;
  for (int s = 0; s < n; ++s) {
    tab.wq[s] = t[s].wq;
    tab.grad[s] = t[s].grad;
    tab.nchunks[s] = t[s].nweights / 16;
    tab.c[s] = t[s].c;
    tab.L[s] = (float)(t[s].qmax - t[s].qmin + 1);
    tab.qmin[s] = t[s].qmin;
    tab.qmax[s] = t[s].qmax;
    tab.tid[s] = t[s].tensor_id;
    tab.b0[s] = blocks;
    blocks += (int32_t)((tab.nchunks[s] + 255) / 256);
  }
  tab.b0[n] = blocks;
  if (blocks == 0) return hipSuccess;
  if (ternary)
    hipLaunchKernelGGL(sr_update_kernel<true>, dim3((unsigned)blocks), dim3(256), 0, stream, tab, counters);
  else
    hipLaunchKernelGGL(sr_update_kernel<false>, dim3((unsigned)blocks), dim3(256), 0, stream, tab, counters);
  return hipGetLastError();
}

hipError_t launch_debug_rng(uint64_t seed, uint32_t step, uint32_t tensor_id, uint64_t i0,
                            int64_t n, uint32_t* out, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int threads = 256;
  int64_t blocks = (n + threads - 1) / threads;
  if (blocks > 65536) blocks = 65536;
  hipLaunchKernelGGL(debug_rng_kernel, dim3((unsigned)blocks), dim3(threads), 0, stream, out, i0,
                     n, (uint32_t)seed, (uint32_t)(seed >> 32), step, tensor_id);
  return hipGetLastError();
}

}  // namespace dqt
