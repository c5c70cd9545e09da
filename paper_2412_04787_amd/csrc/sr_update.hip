// Direct stochastic-rounding update of DQT (Sec. 3.1 Eq. 1, Sec. 3.2 Eq. 5)
// and the Philox4x32-10 counter-based generator that feeds it.
//
// Memory-bound streaming kernel: per weight it reads the packed code and the
// fp32 gradient and writes the code back (4.5 B/weight for 2-bit ternary
// codes, 5 B for 4-bit, 6 B for int8).  Each lane owns 8 consecutive weights
// (one Philox block): 32 contiguous bytes of gradient, and 2 (ternary), 4
// (4-bit) or 8 (int8) whole bytes of codes, so no two lanes ever touch the
// same byte.
#include "sr_rule.h"

namespace dqt {

constexpr int kMaxSR = kMaxBatch;
constexpr int kChunksPerTile = 256;   // one chunk of weights per thread
// Up to kMaxSR tensors in one launch; tensor s owns the tiles [b0[s], b0[s+1])
// of 256 chunks each (its last tile may be partial).
struct SRTab {
  uint8_t* wq[kMaxSR];
  const float* grad[kMaxSR];
  int64_t nchunks[kMaxSR];
  float c[kMaxSR], L[kMaxSR];
  int qmin[kMaxSR], qmax[kMaxSR];
  uint32_t tid[kMaxSR];
  int64_t b0[kMaxSR + 1];
  int32_t n;
  uint32_t k0, k1, step;
};

// Code words of CW weights in format CF: 2-bit ternary codes (CW / 4
// bytes, in w[0]), nibbles (CW / 2 bytes) or int8 codes (CW bytes).
template <int CF, int CW>
struct CodeIO {
  static constexpr int NBYTES = CF == CF_T2 ? CW / 4 : CF == CF_I4 ? CW / 2 : CW;
  static constexpr int NWORD = NBYTES >= 4 ? NBYTES / 4 : 1;
  __device__ static void load(const uint8_t* wq, int64_t t, uint32_t (&w)[4]) {
    if constexpr (NBYTES == 2) {
      w[0] = reinterpret_cast<const uint16_t*>(wq)[t];
    } else if constexpr (NBYTES == 4) {
      w[0] = reinterpret_cast<const uint32_t*>(wq)[t];
    } else if constexpr (NBYTES == 8) {
      const uint2 v = reinterpret_cast<const uint2*>(wq)[t];
      w[0] = v.x; w[1] = v.y;
    } else {
      const uint4 v = reinterpret_cast<const uint4*>(wq)[t];
      w[0] = v.x; w[1] = v.y; w[2] = v.z; w[3] = v.w;
    }
  }
  __device__ static void store(uint8_t* wq, int64_t t, const uint32_t (&w)[4]) {
    if constexpr (NBYTES == 2) reinterpret_cast<uint16_t*>(wq)[t] = (uint16_t)w[0];
    else if constexpr (NBYTES == 4) reinterpret_cast<uint32_t*>(wq)[t] = w[0];
    else if constexpr (NBYTES == 8) reinterpret_cast<uint2*>(wq)[t] = make_uint2(w[0], w[1]);
    else reinterpret_cast<uint4*>(wq)[t] = make_uint4(w[0], w[1], w[2], w[3]);
  }
};

// Persistent kernel: block b takes tiles b, b + grid, ...; thread t of a tile
// owns chunk t of CW consecutive weights (4 CW bytes of gradient, CW / 4 or
// CW bytes of codes, so no two lanes touch the same byte).  The change and
// non-finite counts are reduced per block and added with one atomic each.
template <int CF, int CW>
__global__ __launch_bounds__(256) void sr_update_kernel(const SRTab tab,
                                                        unsigned long long* __restrict__ counters) {
  static_assert(CW == 8 || CW == 16, "8 or 16 weights per lane");
  using CIO = CodeIO<CF, CW>;
  constexpr int NG = CW / 4;               // gradient f32x4 per chunk
  constexpr int NB = CW / 8;               // Philox blocks per chunk
  __shared__ unsigned long long red[2][256 / kWave];
  unsigned long long changed = 0, nonfin = 0;
  const int64_t ntiles = tab.b0[tab.n];
  // Software pipeline: the next tile's gradient and codes are requested
  // before the current tile is computed, so loads stay in flight meanwhile.
  int sidx = 0;
  f32x4 ng[NG];
  uint32_t nw[4];
  int64_t nt = 0;
  int ns = 0;
  auto fetch = [&](int64_t tl) {
    while (sidx + 1 < tab.n && tl >= tab.b0[sidx + 1]) ++sidx;   // tiles ascend
    ns = sidx;
    nt = (tl - tab.b0[sidx]) * kChunksPerTile + threadIdx.x;
    if (nt < tab.nchunks[sidx]) {
      const f32x4* gp = reinterpret_cast<const f32x4*>(tab.grad[sidx] + nt * CW);
#pragma unroll
      for (int u = 0; u < NG; ++u) ng[u] = __builtin_nontemporal_load(gp + u);
      CIO::load(tab.wq[sidx], nt, nw);
    }
  };
  int64_t tile = blockIdx.x;
  if (tile < ntiles) fetch(tile);
  for (; tile < ntiles; tile += gridDim.x) {
    const int cs = ns;
    const int64_t t = nt;
    f32x4 gv[NG];
    uint32_t win[4];
#pragma unroll
    for (int u = 0; u < NG; ++u) gv[u] = ng[u];
#pragma unroll
    for (int u = 0; u < CIO::NWORD; ++u) win[u] = nw[u];
    if (tile + gridDim.x < ntiles) fetch(tile + gridDim.x);
    if (t >= tab.nchunks[cs]) continue;
    SRArgs a;
    a.c = tab.c[cs];
    a.L = tab.L[cs];
    a.qmin = tab.qmin[cs];
    a.qmax = tab.qmax[cs];
    a.k0 = tab.k0;
    a.k1 = tab.k1;
    a.step = tab.step;
    a.tid = tab.tid[cs];
    uint8_t* __restrict__ wq = tab.wq[cs];
    uint32_t wout[4];
    sr_chunk<CF, CW>(win, gv, (uint64_t)t * NB, a, wout, changed, nonfin);
    CIO::store(wq, t, wout);
  }
  if (counters != nullptr) {
    changed = wave_sum_u64(changed);
    nonfin = wave_sum_u64(nonfin);
    const int w = threadIdx.x / kWave;
    if ((threadIdx.x & (kWave - 1)) == 0) {
      red[0][w] = changed;
      red[1][w] = nonfin;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long c = 0, f = 0;
#pragma unroll
      for (int i = 0; i < 256 / kWave; ++i) {
        c += red[0][i];
        f += red[1][i];
      }
      if (c) atomicAdd(counters + 0, c);
      if (f) atomicAdd(counters + 1, f);
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

// Blocks of `threads` threads of `fn` resident on the current device at once.
static int occupancy_blocks(const void* fn, int threads) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, 0) != hipSuccess || per_cu <= 0)
    per_cu = 4;
  return cus * per_cu;
}

#ifndef SR_CW
#define SR_CW 8
#endif
constexpr int kCW = SR_CW;   // weights per lane

hipError_t launch_sr_update(int cf, int n, const SRTensor* t, uint64_t seed, uint32_t step,
                            unsigned long long* counters, hipStream_t stream) {
  SRTab tab{};
  tab.n = n;
  tab.k0 = (uint32_t)seed;
  tab.k1 = (uint32_t)(seed >> 32);
  tab.step = step;
  int64_t tiles = 0;
  for (int s = 0; s < n; ++s) {
    tab.wq[s] = t[s].wq;
    tab.grad[s] = t[s].grad;
    tab.nchunks[s] = t[s].nweights / kCW;
    tab.c[s] = t[s].c;
    tab.L[s] = (float)(t[s].qmax - t[s].qmin + 1);
    tab.qmin[s] = t[s].qmin;
    tab.qmax[s] = t[s].qmax;
    tab.tid[s] = t[s].tensor_id;
    tab.b0[s] = tiles;
    tiles += (tab.nchunks[s] + kChunksPerTile - 1) / kChunksPerTile;
  }
  tab.b0[n] = tiles;
  if (tiles == 0) return hipSuccess;
  // as many blocks as fit on the device at once; each loops over tiles
  const int64_t cap = occupancy_blocks(
      cf == CF_T2 ? reinterpret_cast<const void*>(sr_update_kernel<CF_T2, kCW>)
                  : cf == CF_I4 ? reinterpret_cast<const void*>(sr_update_kernel<CF_I4, kCW>)
                                : reinterpret_cast<const void*>(sr_update_kernel<CF_I8, kCW>),
      256);
  const unsigned blocks = (unsigned)(tiles < cap ? tiles : cap);
  if (cf == CF_T2) return launch_kernel(sr_update_kernel<CF_T2, kCW>, dim3(blocks), dim3(256), stream, tab, counters);
  if (cf == CF_I4) return launch_kernel(sr_update_kernel<CF_I4, kCW>, dim3(blocks), dim3(256), stream, tab, counters);
  return launch_kernel(sr_update_kernel<CF_I8, kCW>, dim3(blocks), dim3(256), stream, tab, counters);
}

hipError_t launch_debug_rng(uint64_t seed, uint32_t step, uint32_t tensor_id, uint64_t i0,
                            int64_t n, uint32_t* out, hipStream_t stream) {
  if (n == 0) return hipSuccess;
  const int threads = 256;
  int64_t blocks = (n + threads - 1) / threads;
  if (blocks > 65536) blocks = 65536;
  return launch_kernel(debug_rng_kernel, dim3((unsigned)blocks), dim3(threads), stream, out, i0, n,
                       (uint32_t)seed, (uint32_t)(seed >> 32), step, tensor_id);
}

}  // namespace dqt
