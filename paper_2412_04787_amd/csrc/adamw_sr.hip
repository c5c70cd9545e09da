// AdamW with direct stochastic rounding (Sec. 4.1 trains DQT with AdamW
// modified to round stochastically; the target W' is the AdamW step and the
// update is W^ = SR(W') of Sec. 3.2 Eq. 5, taken in grid units).
//
// Memory-bound streaming kernel: per weight it reads the fp32 gradient and
// the two fp32 moments and the code, and writes the moments and the code
// back (20.5 B/weight with 2-bit ternary codes, 21 B with 4-bit and 22 B
// with int8 codes).  Each
// lane owns 8 consecutive weights (one Philox block), as the plain update.
//
// Per element, in fp32 with round-to-nearest-even after every operation (no
// fused multiply-add; square root and division correctly rounded):
//   m' = b1 m + ob1 g,   v' = b2 v + (ob2 g) g,
//   u = m' / (sqrt(v') k2 + eps),   delta = -(cu u + cd q),
// with the per-call constants b1, b2, ob1 = 1 - b1, ob2 = 1 - b2,
// k2 = 1 / sqrt(1 - b2^t), cu = lr / (alpha (1 - b1^t)) and cd = lr wd formed
// on the host in double and rounded once to fp32.  The code moves by
// Clip(SR(q + delta)) with the plain update's draws.  An element whose
// gradient is non-finite or whose delta is NaN keeps q, m and v and is
// counted as non-finite.
#include <math.h>

#include "sr_rule.h"

namespace dqt {

namespace {

constexpr int kMaxA = kMaxBatch;
constexpr int kAdamChunksPerTile = 256;

struct AdamTab {
  uint8_t* wq[kMaxA];
  const float* grad[kMaxA];
  float* m[kMaxA];
  float* v[kMaxA];
  int64_t nchunks[kMaxA];
  float cu[kMaxA], L[kMaxA];
  int qmin[kMaxA], qmax[kMaxA];
  uint32_t tid[kMaxA];
  int64_t b0[kMaxA + 1];
  int32_t n;
  float b1, ob1, b2, ob2, k2, eps, cd;
  uint32_t k0, k1, step;
};

// Persistent kernel: block b takes tiles b, b + grid, ...; thread t of a tile
// owns chunk t (8 weights).  Counts are reduced per block, one atomic each.
template <int CF>
__global__ __launch_bounds__(256) void adamw_sr_kernel(const AdamTab tab,
                                                       unsigned long long* __restrict__ counters) {
  __shared__ unsigned long long red[2][256 / kWave];
  unsigned long long changed = 0, nonfin = 0;
  const int64_t ntiles = tab.b0[tab.n];
  // Software pipeline: the next tile's gradient, moments and codes are
  // requested before the current tile is computed.
  int sidx = 0, ns = 0;
  int64_t nt = 0;
  f32x4 ng[2], nm[2], nv[2];
  uint32_t nw[4] = {0u, 0u, 0u, 0u};
  auto fetch = [&](int64_t tl) {
    while (sidx + 1 < tab.n && tl >= tab.b0[sidx + 1]) ++sidx;    // tiles ascend
    ns = sidx;
    nt = (tl - tab.b0[sidx]) * kAdamChunksPerTile + threadIdx.x;
    if (nt < tab.nchunks[sidx]) {
      const f32x4* gp = reinterpret_cast<const f32x4*>(tab.grad[sidx]) + 2 * nt;
      const f32x4* mp = reinterpret_cast<const f32x4*>(tab.m[sidx]) + 2 * nt;
      const f32x4* vp = reinterpret_cast<const f32x4*>(tab.v[sidx]) + 2 * nt;
#pragma unroll
      for (int u = 0; u < 2; ++u) {
        ng[u] = __builtin_nontemporal_load(gp + u);
        nm[u] = __builtin_nontemporal_load(mp + u);
        nv[u] = __builtin_nontemporal_load(vp + u);
      }
      ChunkIO<CF>::load(tab.wq[sidx], nt, nw);
    }
  };
  if ((int64_t)blockIdx.x < ntiles) fetch(blockIdx.x);
  for (int64_t tile = blockIdx.x; tile < ntiles; tile += gridDim.x) {
    const int s = ns;
    const int64_t t = nt;
    const f32x4 g4[2] = {ng[0], ng[1]};
    const f32x4 m4[2] = {nm[0], nm[1]};
    const f32x4 v4[2] = {nv[0], nv[1]};
    uint32_t win[4] = {nw[0], nw[1], 0u, 0u};
    if (tile + gridDim.x < ntiles) fetch(tile + gridDim.x);
    if (t >= tab.nchunks[s]) continue;
    f32x4* mp = reinterpret_cast<f32x4*>(tab.m[s]) + 2 * t;
    f32x4* vp = reinterpret_cast<f32x4*>(tab.v[s]) + 2 * t;
    SRArgs a;
    a.c = 0.0f;
    a.L = tab.L[s];
    a.qmin = tab.qmin[s];
    a.qmax = tab.qmax[s];
    a.k0 = tab.k0;
    a.k1 = tab.k1;
    a.step = tab.step;
    a.tid = tab.tid[s];
    const float cu = tab.cu[s];
    float delta[8];
    f32x4 mo[2], vo[2];
    uint32_t bad = 0;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      const float g = g4[j >> 2][j & 3], m = m4[j >> 2][j & 3], v = v4[j >> 2][j & 3];
      const int q = CodeFmt<CF>::q_of(win, j);
      const float m1 = __fadd_rn(__fmul_rn(tab.b1, m), __fmul_rn(tab.ob1, g));
      const float v1 = __fadd_rn(__fmul_rn(tab.b2, v), __fmul_rn(__fmul_rn(tab.ob2, g), g));
      // (sqrtf is the correctly rounded square root in HIP; __fsqrt_rn
      // lowers to the one-ulp hardware approximation)
      const float den = __fadd_rn(__fmul_rn(sqrtf(v1), tab.k2), tab.eps);
      const float u = __fdiv_rn(m1, den);
      const float d = -__fadd_rn(__fmul_rn(cu, u), __fmul_rn(tab.cd, (float)q));
      const bool keep = !__builtin_isfinite(g) || __builtin_isnan(d);
      bad |= (keep ? 1u : 0u) << j;
      delta[j] = keep ? 0.0f : d;
      mo[j >> 2][j & 3] = keep ? m : m1;
      vo[j >> 2][j & 3] = keep ? v : v1;
    }
    uint32_t wout[4];
    sr_chunk_delta<CF>(win, delta, bad, (uint64_t)t, a, wout, changed, nonfin);
    mp[0] = mo[0];
    mp[1] = mo[1];
    vp[0] = vo[0];
    vp[1] = vo[1];
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

int adam_resident_blocks(const void* fn) {
  int dev = 0, cus = 0, per_cu = 0;
  if (hipGetDevice(&dev) != hipSuccess ||
      hipDeviceGetAttribute(&cus, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || cus <= 0)
    cus = 256;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, 256, 0) != hipSuccess || per_cu <= 0)
    per_cu = 4;
  return cus * per_cu;
}

// b^t in double by binary exponentiation (low bit first).
double pow_by_squaring(double b, uint32_t t) {
  double r = 1.0, x = b;
  while (t > 0) {
    if (t & 1u) r = r * x;
    x = x * x;
    t >>= 1;
  }
  return r;
}

}  // namespace

hipError_t launch_adamw_sr(int cf, int n, const AdamTensor* t, const AdamHyper& hp,
                           uint64_t seed, uint32_t step, unsigned long long* counters,
                           hipStream_t stream) {
  AdamTab tab{};
  tab.n = n;
  tab.k0 = (uint32_t)seed;
  tab.k1 = (uint32_t)(seed >> 32);
  tab.step = step;
  const double b1 = (double)hp.beta1, b2 = (double)hp.beta2, lr = (double)hp.lr;
  tab.b1 = hp.beta1;
  tab.b2 = hp.beta2;
  tab.ob1 = (float)(1.0 - b1);
  tab.ob2 = (float)(1.0 - b2);
  tab.k2 = (float)(1.0 / sqrt(1.0 - pow_by_squaring(b2, step)));
  tab.eps = hp.eps;
  tab.cd = (float)(lr * (double)hp.weight_decay);
  const double bc1 = 1.0 - pow_by_squaring(b1, step);
  int64_t tiles = 0;
  for (int s = 0; s < n; ++s) {
    tab.wq[s] = t[s].wq;
    tab.grad[s] = t[s].grad;
    tab.m[s] = t[s].m;
    tab.v[s] = t[s].v;
    tab.nchunks[s] = t[s].nweights / 8;
    tab.cu[s] = (float)(lr / ((double)t[s].alpha * bc1));
    tab.L[s] = (float)(t[s].qmax - t[s].qmin + 1);
    tab.qmin[s] = t[s].qmin;
    tab.qmax[s] = t[s].qmax;
    tab.tid[s] = t[s].tensor_id;
    tab.b0[s] = tiles;
    tiles += (tab.nchunks[s] + kAdamChunksPerTile - 1) / kAdamChunksPerTile;
  }
  tab.b0[n] = tiles;
  if (tiles == 0) return hipSuccess;
  const int64_t cap = adam_resident_blocks(
      cf == CF_T2 ? reinterpret_cast<const void*>(adamw_sr_kernel<CF_T2>)
                  : cf == CF_I4 ? reinterpret_cast<const void*>(adamw_sr_kernel<CF_I4>)
                  : cf == CF_I3 ? reinterpret_cast<const void*>(adamw_sr_kernel<CF_I3>)
                                : reinterpret_cast<const void*>(adamw_sr_kernel<CF_I8>));
  const unsigned blocks = (unsigned)(tiles < cap ? tiles : cap);
  if (cf == CF_T2) return launch_kernel(adamw_sr_kernel<CF_T2>, dim3(blocks), dim3(256), stream, tab, counters);
  if (cf == CF_I4) return launch_kernel(adamw_sr_kernel<CF_I4>, dim3(blocks), dim3(256), stream, tab, counters);
  if (cf == CF_I3) return launch_kernel(adamw_sr_kernel<CF_I3>, dim3(blocks), dim3(256), stream, tab, counters);
  return launch_kernel(adamw_sr_kernel<CF_I8>, dim3(blocks), dim3(256), stream, tab, counters);
}

}  // namespace dqt
