// Analysis variants of the direct update (Sec. 5): rounding q + delta to
// the nearest grid value instead of stochastically (the control that drops
// small updates), and the two interventions on the smallest fraction of a
// step's updates: keep those codes (force to remain), or round them away
// from q (force to update); every other element takes the plain SR update
// of Sec. 3.2 Eq. 5 with the same draws.
//
// The bottom set of a tensor is {key <= tau}: key is the fp32 bit pattern of
// |delta| = |fl(c g)| read as an unsigned integer (monotone in |delta|; a
// non-finite g ranks above every finite one) and tau the k-th smallest key,
// k = floor(frac n).  tau is found exactly on the device by a radix select
// over the keys: bit 31 of a key is always 0 (a non-finite g takes
// 0x7FFFFFFF, which selects the same bottom set as any key above all finite
// ones), so three passes cover bits 30-20, 19-9 and 8-0, each a histogram
// of the keys that match the bits chosen so far, then a scan that picks the
// bin holding the k-th key.  Each pass reads the gradient once (4 B per
// weight).
#include <math.h>

#include <algorithm>

#include "sr_rule.h"

namespace dqt {

namespace {

constexpr int kMaxV = kMaxBatch;
constexpr int kHistBins = 2048;
// A selection block takes 256 threads x `chunks` chunks of 8 weights, chunks
// a multiple of 4 from 4 to 32 chosen by the host for at least ~1024 blocks:
// more weights a block spread its histogram's clearing and flushing (h4096
// block, force-to-update call: 1010 us at 4 chunks, 725 us at 32).
constexpr int kMinChunks = 4, kMaxChunks = 32;

// Radix-select state of one tensor (in the caller's workspace).
struct SelState {
  uint32_t prefix, mask, krem, pad;
  uint32_t hist[kHistBins];
};

struct VarTab {
  uint8_t* wq[kMaxV];
  const float* grad[kMaxV];
  int64_t nweights[kMaxV];
  int64_t b0[kMaxV + 1];         // blocks of 2048 `chunks` chunks (selection passes)
  int32_t chunks;                // chunks of 8 weights per thread (selection passes)
  int64_t t0[kMaxV + 1];         // tiles of 256 chunks (update)
  float c[kMaxV], L[kMaxV];
  int qmin[kMaxV], qmax[kMaxV];
  uint32_t tid[kMaxV];
  uint32_t k[kMaxV];             // bottom-set size; 0: empty
  int32_t n, mode;
  uint32_t k0, k1, step;
};

__device__ __forceinline__ uint32_t delta_key(float g, float c) {
  return __builtin_isfinite(g) ? (__float_as_uint(c * g) & 0x7FFFFFFFu) : 0x7FFFFFFFu;
}

template <int N>
__device__ __forceinline__ int seg_of(const int64_t (&b)[N], int n, int64_t x) {
  int s = 0;
  while (s + 1 < n && x >= b[s + 1]) ++s;
  return s;
}

__global__ __launch_bounds__(256) void sel_init_kernel(const VarTab tab, SelState* __restrict__ st) {
  SelState& S = st[blockIdx.x];
  if (threadIdx.x == 0) {
    S.prefix = 0;
    S.mask = 0;
    S.krem = tab.k[blockIdx.x];
    S.pad = 0;
  }
  for (int i = threadIdx.x; i < kHistBins; i += 256) S.hist[i] = 0;
}

// Histogram of bits [shift, shift + nbits) of the keys that match the bits
// chosen so far.  One block per 2048 chunks of 8 weights of one tensor.
__global__ __launch_bounds__(256) void sel_hist_kernel(const VarTab tab, SelState* __restrict__ st,
                                                       int shift, int nbins) {
  __shared__ uint32_t h[kHistBins];
  const int s = seg_of(tab.b0, tab.n, (int64_t)blockIdx.x);
  for (int i = threadIdx.x; i < nbins; i += 256) h[i] = 0;
  __syncthreads();
  const SelState& S = st[s];
  const uint32_t prefix = S.prefix, mask = S.mask;
  if (tab.k[s] != 0) {
    const int chunks = tab.chunks;
    const int64_t nw = tab.nweights[s];
    const int64_t base = (int64_t)(blockIdx.x - tab.b0[s]) * (2048 * (int64_t)chunks);
    const float c = tab.c[s];
    const f32x4* g4 = reinterpret_cast<const f32x4*>(tab.grad[s]);
    for (int u0 = 0; u0 < chunks; u0 += 4) {
      if (base + (int64_t)u0 * 2048 >= nw) break;          // (block-uniform)
      // four chunks' loads in flight
#pragma unroll
      for (int du = 0; du < 4; ++du) {
        const int64_t e0 = base + ((int64_t)(u0 + du) * 256 + threadIdx.x) * 8;
        if (e0 >= nw) break;
        const f32x4 a = g4[e0 / 4], b = g4[e0 / 4 + 1];
        const float g[8] = {a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3]};
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const uint32_t key = delta_key(g[j], c);
          if ((key & mask) == prefix) atomicAdd(&h[(key >> shift) & (uint32_t)(nbins - 1)], 1u);
        }
      }
    }
  }
  __syncthreads();
  if (tab.k[s] != 0)
    for (int i = threadIdx.x; i < nbins; i += 256)
      if (h[i]) atomicAdd(&st[s].hist[i], h[i]);
}

// The bin holding the krem-th matching key: its bits join the prefix, krem
// drops by the keys of the bins below it; the histogram is cleared.
__global__ __launch_bounds__(256) void sel_pick_kernel(const VarTab tab, SelState* __restrict__ st,
                                                       int shift, int nbins) {
  __shared__ uint32_t part[256];
  __shared__ uint32_t pick_bin, pick_below;
  SelState& S = st[blockIdx.x];
  if (tab.k[blockIdx.x] == 0) return;
  const int per = nbins / 256;                   // 8 or 2 bins per thread
  uint32_t sum = 0;
  for (int i = 0; i < per; ++i) sum += S.hist[threadIdx.x * per + i];
  part[threadIdx.x] = sum;
  if (threadIdx.x == 0) {
    pick_bin = (uint32_t)(nbins - 1);
    pick_below = 0;
  }
  __syncthreads();
  // exclusive prefix of the per-thread sums (Hillis-Steele in LDS)
  for (int off = 1; off < 256; off <<= 1) {
    const uint32_t v = threadIdx.x >= (unsigned)off ? part[threadIdx.x - off] : 0u;
    __syncthreads();
    part[threadIdx.x] += v;
    __syncthreads();
  }
  const uint32_t krem = S.krem;
  const uint32_t incl = part[threadIdx.x], excl = incl - sum;
  if (excl < krem && krem <= incl) {             // exactly one thread
    uint32_t cum = excl;
    for (int i = 0; i < per; ++i) {
      const uint32_t c = S.hist[threadIdx.x * per + i];
      if (cum + c >= krem) {
        pick_bin = (uint32_t)(threadIdx.x * per + i);
        pick_below = cum;
        break;
      }
      cum += c;
    }
  }
  __syncthreads();
  for (int i = threadIdx.x; i < nbins; i += 256) S.hist[i] = 0;
  if (threadIdx.x == 0) {
    S.prefix |= pick_bin << shift;
    S.mask |= (uint32_t)(nbins - 1) << shift;
    S.krem = krem - pick_below;
  }
}

// x = q + delta rounded to the nearest grid value, ties to even.
__device__ __forceinline__ int nearest_code(int q, float g, float c, float L, int qmin, int qmax) {
  const float delta = fminf(fmaxf(-(c * g), -L), L);
  const float n = truncf(delta);
  const float r = delta - n;                     // exact, |r| < 1
  int v = q + (int)n;
  const float ar = fabsf(r);
  const int sgn = r > 0.0f ? 1 : -1;
  if (ar > 0.5f || (ar == 0.5f && ((v + sgn) & 1) == 0)) v += sgn;
  return min(max(v, qmin), qmax);
}

// x = q + delta rounded away from q (ceil for delta > 0, floor for < 0).
__device__ __forceinline__ int away_code(int q, float g, float c, float L, int qmin, int qmax) {
  const float delta = fminf(fmaxf(-(c * g), -L), L);
  const float a = delta > 0.0f ? ceilf(delta) : floorf(delta);
  return min(max(q + (int)a, qmin), qmax);
}

// The update: the plain SR chunk, then the variant's elements replaced.
template <int CF>
__global__ __launch_bounds__(256) void variant_update_kernel(const VarTab tab, const SelState* __restrict__ st,
                                                             unsigned long long* __restrict__ counters) {
  __shared__ unsigned long long red[2][256 / kWave];
  unsigned long long changed = 0, nonfin = 0;
  const int64_t ntiles = tab.t0[tab.n];
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int s = seg_of(tab.t0, tab.n, tile);
    const int64_t t = (tile - tab.t0[s]) * 256 + threadIdx.x;
    if (t >= tab.nweights[s] / 8) continue;
    const f32x4* gp = reinterpret_cast<const f32x4*>(tab.grad[s]) + 2 * t;
    const f32x4 gv[2] = {__builtin_nontemporal_load(gp), __builtin_nontemporal_load(gp + 1)};
    uint32_t win[4] = {0u, 0u, 0u, 0u};
    ChunkIO<CF>::load(tab.wq[s], t, win);
    SRArgs a;
    a.c = tab.c[s];
    a.L = tab.L[s];
    a.qmin = tab.qmin[s];
    a.qmax = tab.qmax[s];
    a.k0 = tab.k0;
    a.k1 = tab.k1;
    a.step = tab.step;
    a.tid = tab.tid[s];
    uint32_t wout[4];
    unsigned long long ch_sr = 0;
    sr_chunk<CF, 8>(win, gv, (uint64_t)t, a, wout, ch_sr, nonfin);
    const bool sel = tab.mode >= 2 && tab.k[s] != 0;
    const uint32_t tau = sel ? st[s].prefix : 0u;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float g = gv[j >> 2][j & 3];
      if (!__builtin_isfinite(g)) continue;      // kept by the SR chunk
      const int q = CodeFmt<CF>::q_of(win, j);
      int v;
      if (tab.mode == 1) v = nearest_code(q, g, a.c, a.L, a.qmin, a.qmax);
      else if (sel && delta_key(g, a.c) <= tau) v = tab.mode == 2 ? q : away_code(q, g, a.c, a.L, a.qmin, a.qmax);
      else continue;
      CodeFmt<CF>::set(wout, j, v + CodeFmt<CF>::off);
    }
    changed += CodeFmt<CF>::template changed<8>(wout, win);
    ChunkIO<CF>::store(tab.wq[s], t, wout);
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

}  // namespace

// ------------------------------------------------------------------------
// The deterministic control of Sec. 5.1 read literally: the updated matrix
// W' = W~ - lr dW is absmax-quantised afresh, with a new per-tensor scale
// alpha' = max|W'| / qmax (Eq. 3-4 with the maximum in place of the mean).
// Two passes over each tensor: the maximum of |W'| (per block, then one
// atomic max on its bit pattern, which orders as the value for |W'| >= 0),
// then the new codes.
namespace {

struct AbsTab {
  uint8_t* wq[kMaxV];
  const float* grad[kMaxV];
  int64_t nweights[kMaxV];
  int64_t t0[kMaxV + 1];         // tiles of 256 chunks
  float alpha[kMaxV], lr;
  int qmin[kMaxV], qmax[kMaxV];
  float* alpha_out;              // [n] device
  uint32_t* wmax;                // [n] device, the max |W'| bits
  int32_t n;
};

// W'_j of a chunk: fl(fl(q alpha) - fl(lr g)), a non-finite g read as 0
template <int CF>
__device__ __forceinline__ void wprime8(const uint32_t (&win)[4], const f32x4 (&gv)[2], float alpha,
                                        float lr, float (&w)[8], uint32_t& nonfin) {
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    const float g = gv[j >> 2][j & 3];
    const bool fin = __builtin_isfinite(g);
    nonfin += fin ? 0u : 1u;
    w[j] = (float)CodeFmt<CF>::q_of(win, j) * alpha - lr * (fin ? g : 0.0f);
  }
}

__global__ __launch_bounds__(64) void absmax_init_kernel(uint32_t* wmax, int n) {
  for (int i = threadIdx.x; i < n; i += 64) wmax[i] = 0u;
}

template <int CF>
__global__ __launch_bounds__(256) void absmax_max_kernel(const AbsTab tab) {
  __shared__ uint32_t red[256 / kWave];
  const int64_t tile = blockIdx.x;
  const int s = seg_of(tab.t0, tab.n, tile);
  const int64_t t = (tile - tab.t0[s]) * 256 + threadIdx.x;
  float m = 0.0f;
  if (t < tab.nweights[s] / 8) {
    const f32x4* gp = reinterpret_cast<const f32x4*>(tab.grad[s]) + 2 * t;
    const f32x4 gv[2] = {gp[0], gp[1]};
    uint32_t win[4] = {0u, 0u, 0u, 0u}, nf = 0;
    ChunkIO<CF>::load(tab.wq[s], t, win);
    float w[8];
    wprime8<CF>(win, gv, tab.alpha[s], tab.lr, w, nf);
#pragma unroll
    for (int j = 0; j < 8; ++j) m = fmaxf(m, fabsf(w[j]));
  }
  m = wave_max(m);
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = __float_as_uint(m);
  __syncthreads();
  if (threadIdx.x == 0) {
    uint32_t b = 0;
#pragma unroll
    for (int i = 0; i < 256 / kWave; ++i) b = max(b, red[i]);
    if (b) atomicMax(tab.wmax + s, b);
  }
}

template <int CF>
__global__ __launch_bounds__(256) void absmax_quant_kernel(const AbsTab tab, unsigned long long* counters) {
  __shared__ uint32_t red[2][256 / kWave];
  const int64_t tile = blockIdx.x;
  const int s = seg_of(tab.t0, tab.n, tile);
  const int64_t t = (tile - tab.t0[s]) * 256 + threadIdx.x;
  const float m = __uint_as_float(tab.wmax[s]);
  const float qp = (float)tab.qmax[s];
  const float sn = m > 0.0f ? __fdiv_rn(qp, m) : 0.0f;
  if (tile == tab.t0[s] && threadIdx.x == 0) tab.alpha_out[s] = m > 0.0f ? __fdiv_rn(m, qp) : tab.alpha[s];
  uint32_t ch = 0, nf = 0;
  if (t < tab.nweights[s] / 8) {
    const f32x4* gp = reinterpret_cast<const f32x4*>(tab.grad[s]) + 2 * t;
    const f32x4 gv[2] = {gp[0], gp[1]};
    uint32_t win[4] = {0u, 0u, 0u, 0u}, wout[4] = {0u, 0u, 0u, 0u};
    ChunkIO<CF>::load(tab.wq[s], t, win);
    float w[8];
    wprime8<CF>(win, gv, tab.alpha[s], tab.lr, w, nf);
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const int v = (int)fminf(fmaxf(rintf(w[j] * sn), (float)tab.qmin[s]), qp);
      CodeFmt<CF>::put(wout, j, v + CodeFmt<CF>::off);
    }
    ch = CodeFmt<CF>::template changed<8>(wout, win);
    ChunkIO<CF>::store(tab.wq[s], t, wout);
  }
  if (counters != nullptr) {
    const uint32_t c = wave_sum_u32(ch), f = wave_sum_u32(nf);
    if ((threadIdx.x & (kWave - 1)) == 0) {
      red[0][threadIdx.x / kWave] = c;
      red[1][threadIdx.x / kWave] = f;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
      unsigned long long ct = 0, ft = 0;
#pragma unroll
      for (int i = 0; i < 256 / kWave; ++i) {
        ct += red[0][i];
        ft += red[1][i];
      }
      if (ct) atomicAdd(counters, ct);
      if (ft) atomicAdd(counters + 1, ft);
    }
  }
}

template <int CF>
hipError_t launch_absmax_cf(const AbsTab& tab, int64_t tiles, unsigned long long* counters,
                            hipStream_t stream) {
  LaunchStatus ls;
  ls << launch_kernel(absmax_init_kernel, dim3(1), dim3(64), stream, tab.wmax, (int)tab.n);
  ls << launch_kernel(absmax_max_kernel<CF>, dim3((unsigned)tiles), dim3(256), stream, tab);
  ls << launch_kernel(absmax_quant_kernel<CF>, dim3((unsigned)tiles), dim3(256), stream, tab, counters);
  return ls.e;
}

}  // namespace

size_t absmax_requant_workspace(int n) { return (size_t)(n > 0 ? n : 0) * 4; }

hipError_t launch_absmax_requant(int cf, int n, const SRTensor* t, float lr, float* alpha_out,
                                 unsigned long long* counters, void* ws, hipStream_t stream) {
  AbsTab tab{};
  tab.n = n;
  tab.lr = lr;
  tab.alpha_out = alpha_out;
  tab.wmax = static_cast<uint32_t*>(ws);
  int64_t tiles = 0;
  for (int s = 0; s < n; ++s) {
    tab.wq[s] = t[s].wq;
    tab.grad[s] = t[s].grad;
    tab.nweights[s] = t[s].nweights;
    tab.alpha[s] = t[s].alpha;
    tab.qmin[s] = t[s].qmin;
    tab.qmax[s] = t[s].qmax;
    tab.t0[s] = tiles;
    tiles += (t[s].nweights / 8 + 255) / 256;
  }
  tab.t0[n] = tiles;
  if (tiles == 0) return hipSuccess;
  if (cf == CF_T2) return launch_absmax_cf<CF_T2>(tab, tiles, counters, stream);
  if (cf == CF_I4) return launch_absmax_cf<CF_I4>(tab, tiles, counters, stream);
  if (cf == CF_I3) return launch_absmax_cf<CF_I3>(tab, tiles, counters, stream);
  return launch_absmax_cf<CF_I8>(tab, tiles, counters, stream);
}

size_t update_variant_workspace(int n) { return (size_t)n * sizeof(SelState); }

hipError_t launch_update_variant(int cf, int n, const SRTensor* t, int mode, float frac,
                                 uint64_t seed, uint32_t step, unsigned long long* counters,
                                 void* ws, hipStream_t stream) {
  VarTab tab{};
  tab.n = n;
  tab.mode = mode;
  tab.k0 = (uint32_t)seed;
  tab.k1 = (uint32_t)(seed >> 32);
  tab.step = step;
  int64_t blocks = 0, tiles = 0;
  bool any_sel = false;
  int64_t total = 0;
  for (int s = 0; s < n; ++s) total += t[s].nweights;
  tab.chunks = (int32_t)std::max<int64_t>(kMinChunks, std::min<int64_t>(kMaxChunks, total / (2048 * 1024) / 4 * 4));
  const int64_t per_block = 2048 * (int64_t)tab.chunks;
  for (int s = 0; s < n; ++s) {
    tab.wq[s] = t[s].wq;
    tab.grad[s] = t[s].grad;
    tab.nweights[s] = t[s].nweights;
    tab.c[s] = t[s].c;
    tab.L[s] = (float)(t[s].qmax - t[s].qmin + 1);
    tab.qmin[s] = t[s].qmin;
    tab.qmax[s] = t[s].qmax;
    tab.tid[s] = t[s].tensor_id;
    const double kk = mode >= 2 ? floor((double)frac * (double)t[s].nweights) : 0.0;
    tab.k[s] = (uint32_t)kk;
    any_sel |= tab.k[s] != 0;
    tab.b0[s] = blocks;
    blocks += (t[s].nweights + per_block - 1) / per_block;
    tab.t0[s] = tiles;
    tiles += (t[s].nweights / 8 + 255) / 256;
  }
  tab.b0[n] = blocks;
  tab.t0[n] = tiles;
  if (tiles == 0) return hipSuccess;
  SelState* st = static_cast<SelState*>(ws);
  LaunchStatus ls;
  if (any_sel) {
    ls << launch_kernel(sel_init_kernel, dim3((unsigned)n), dim3(256), stream, tab, st);
    const int shifts[3] = {20, 9, 0}, bins[3] = {2048, 2048, 512};
    for (int p = 0; p < 3; ++p) {
      ls << launch_kernel(sel_hist_kernel, dim3((unsigned)blocks), dim3(256), stream, tab, st, shifts[p],
                          bins[p]);
      ls << launch_kernel(sel_pick_kernel, dim3((unsigned)n), dim3(256), stream, tab, st, shifts[p], bins[p]);
    }
  }
  const unsigned grid = (unsigned)(tiles < 4096 ? tiles : 4096);
  if (cf == CF_T2)
    ls << launch_kernel(variant_update_kernel<CF_T2>, dim3(grid), dim3(256), stream, tab, st, counters);
  else if (cf == CF_I4)
    ls << launch_kernel(variant_update_kernel<CF_I4>, dim3(grid), dim3(256), stream, tab, st, counters);
  else if (cf == CF_I3)
    ls << launch_kernel(variant_update_kernel<CF_I3>, dim3(grid), dim3(256), stream, tab, st, counters);
  else
    ls << launch_kernel(variant_update_kernel<CF_I8>, dim3(grid), dim3(256), stream, tab, st, counters);
  return ls.e;
}

}  // namespace dqt
