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

constexpr int kChunksPerTile = 256;   // one chunk of 8 weights per thread
constexpr int kCW = 8;                // weights per chunk (one Philox block)
// stages of each wave's load ring (tiles in flight per wave)
#ifndef SR_STAGES
#define SR_STAGES 2
#endif

// One tensor of an update launch: codes, gradient, its chunks of 8 weights
// and the first tile (256 chunks) it owns in the launch's tile order.
struct SRDesc {
  uint8_t* wq;
  const float* grad;
  int64_t nchunks;
  int64_t tile0;
  float c, L;           // fl32(lr / alpha); |delta| clamp qmax - qmin + 1
  int qmin, qmax;
  uint32_t tid;
};

// Tensors passed in the kernel arguments (up to kMaxBatch).
struct SRArgTab {
  static constexpr bool kStrided = true;
  SRDesc d[kMaxBatch];
  int32_t n;
  __device__ SRDesc get(int s) const { return d[s]; }
};
// Tensors described by a table in device memory (any number), built on the
// host by dqt_sr_table_build; the step size is formed per tensor from lr
// and alpha as one correctly rounded fp32 division.
struct SRDevTab {
  static constexpr bool kStrided = false;
  const SRTableEntry* e;
  int32_t n;
  float lr;
  __device__ SRDesc get(int s) const {
    // read through the constant address space: wave-uniform scalar loads,
    // which do not count against the vector memory counter that paces the
    // DMA pipeline
    const auto* ce = reinterpret_cast<const __attribute__((address_space(4))) SRTableEntry*>(
        (const __attribute__((address_space(4))) void*)e);
    const auto& t = ce[s];
    SRDesc d;
    d.wq = reinterpret_cast<uint8_t*>(t.wq);
    d.grad = reinterpret_cast<const float*>(t.grad);
    d.nchunks = t.nchunks;
    d.tile0 = t.tile0;
    d.c = __fdiv_rn(lr, t.alpha);
    d.L = (float)(t.qmax - t.qmin + 1);
    d.qmin = t.qmin;
    d.qmax = t.qmax;
    d.tid = t.tensor_id;
    return d;
  }
};

// Sum of a per-lane count over the block (every thread gets it; the block
// runs this in uniform control flow).  `red` holds one slot per wave.
__device__ __forceinline__ uint32_t block_sum(uint32_t v, uint32_t* red) {
  v = wave_sum_u32(v);
  __syncthreads();                         // earlier readers of `red` are done
  if ((threadIdx.x & (kWave - 1)) == 0) red[threadIdx.x / kWave] = v;
  __syncthreads();
  uint32_t t = 0;
#pragma unroll
  for (int w = 0; w < 256 / kWave; ++w) t += red[w];
  return t;
}

// Persistent streaming kernel.  Thread t of a tile owns chunk t: 32 bytes
// of gradient and whole bytes of codes, so no two lanes write the same byte.
// Loads run SR_STAGES tiles ahead through LDS (below).  Counts are kept per
// lane; the per-tensor counts are summed over the block whenever the tensor
// changes, the totals once at the end.  Measured on the hidden-4096 block
// (ternary, 911 MB per call): loads as per-lane 32-byte pieces into
// registers one tile ahead streamed 4.8 TB/s with no arithmetic at all;
// whole 16-byte-per-lane DMA with the non-temporal hint streams 5.7 TB/s,
// and the full update with the ternary mask path below runs at 5.1 TB/s
// (4.5 TB/s before).
template <int CF, class Tab>
__global__ __launch_bounds__(256) void sr_update_kernel(const Tab tab, int64_t ntiles, uint32_t k0,
                                                        uint32_t k1, uint32_t step,
                                                        unsigned long long* __restrict__ counters,
                                                        unsigned long long* __restrict__ per_tensor) {
  using CIO = ChunkIO<CF>;
  // tiles b, b + G, ... of the launch (few tensors: the front of loads
  // sweeps through memory together), or the contiguous range
  // [b T / G, (b + 1) T / G) (many tensors: a block meets few boundaries)
  const int64_t t_begin = Tab::kStrided ? (int64_t)blockIdx.x : ntiles * blockIdx.x / gridDim.x;
  const int64_t t_end = Tab::kStrided ? ntiles : ntiles * (blockIdx.x + 1) / gridDim.x;
  const int64_t t_inc = Tab::kStrided ? (int64_t)gridDim.x : 1;
  if (t_begin >= t_end) return;
  // tensor of the first tile (binary search over the tensors' first tiles)
  int s0 = 0;
  {
    int lo = 0, hi = tab.n - 1;
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (tab.get(mid).tile0 <= t_begin) lo = mid;
      else hi = mid - 1;
    }
    s0 = lo;
  }
  // Wave w of the block updates chunks 64 w .. 64 w + 63 of each tile.  Its
  // gradients (2 KB) and codes (64 NB bytes) travel global -> LDS by DMA
  // into a private ring of D stages, D tiles ahead, so the bytes in flight
  // do not hold registers; the loads are whole consecutive 16-byte pieces
  // (lane l: bytes 16 l of each KB), each lane then reads its own chunk's
  // 32 bytes back from LDS.  Lanes past the tensor's end load a valid chunk
  // of it (the last one) and skip the update, so every wave issues the same
  // number of loads per tile and the wait counts hold.
  constexpr int D = SR_STAGES;
  constexpr int NB = chunk_code_bytes<CF>();
  constexpr int NCD = (64 * NB + 255) / 256;   // 4-byte DMA loads per lane for the codes
  constexpr int STAGE = 2048 + 256 * NCD;
  constexpr int LPT = 2 + NCD;                 // loads per tile
  constexpr int SPT = 1;   // store instructions per tile counted (at least one; more only waits longer)
  __shared__ __attribute__((aligned(16))) uint8_t ring_raw[4 * D * STAGE];
  const int wv = threadIdx.x >> 6, lane = threadIdx.x & 63;
  lds_u8* ring = reinterpret_cast<lds_u8*>(
      (__attribute__((address_space(3))) void*)(ring_raw)) + wv * D * STAGE;
  SRDesc dn = tab.get(s0);          // tensor of the next tile to load
  int sn = s0;
  auto issue = [&](int d, int64_t tl) {
    while (tl >= dn.tile0 + (dn.nchunks + kChunksPerTile - 1) / kChunksPerTile) dn = tab.get(++sn);
    const int64_t c0 = (tl - dn.tile0) * kChunksPerTile + 64 * wv;
    const int64_t last = dn.nchunks - 1;
    const int64_t ca = min(c0 + (lane >> 1), last), cb = min(c0 + 32 + (lane >> 1), last);
    const uint8_t* g = reinterpret_cast<const uint8_t*>(dn.grad);
    lds_u8* st = ring + d * STAGE;
    dma16_nt(g + ca * 32 + 16 * (lane & 1), st);
    dma16_nt(g + cb * 32 + 16 * (lane & 1), st + 1024);
    const int64_t cbytes = dn.nchunks * NB;   // a multiple of 32 NB bytes
#pragma unroll
    for (int q = 0; q < NCD; ++q)
      dma4(dn.wq + min(c0 * NB + 256 * q + 4 * lane, cbytes - 4), st + 2048 + 256 * q);
  };
  SRDesc dc = tab.get(s0);          // tensor of the tile being updated
  int sc = s0;
  __shared__ uint32_t red[256 / kWave];
  // counts of the current tensor (per lane), and of the tensors before it
  uint32_t ch = 0, nf = 0, ch_done = 0, nf_done = 0;
  // one atomic per block per tensor for the per-tensor counts (tensor
  // changes are block-uniform: all threads work on the same tile)
  auto flush_tensor = [&](int s_) {
    if (per_tensor != nullptr) {
      const uint32_t c = block_sum(ch, red), f = block_sum(nf, red);
      if (threadIdx.x == 0) {
        if (c) atomicAdd(per_tensor + 2 * s_, (unsigned long long)c);
        if (f) atomicAdd(per_tensor + 2 * s_ + 1, (unsigned long long)f);
      }
    }
    ch_done += ch;
    nf_done += nf;
    ch = nf = 0;
  };
  // this block's tiles: t_begin + i t_inc, i < n_t; tile i sits in stage i mod D
  const int64_t n_t = (t_end - t_begin + t_inc - 1) / t_inc;
  uint32_t hist = 0;
  for (int d = 0; d < D && d < n_t; ++d) issue(d, t_begin + d * t_inc);
  int d = 0;
  for (int64_t i = 0; i < n_t; ++i) {
    const int64_t tl = t_begin + i * t_inc;
    // memory operations issued after tile i's loads: the loads of tiles
    // i + 1 .. i + D - 1 that exist, and the stores of the min(i, D) tiles
    // before it (a wave with no chunk of a tile in range stores nothing;
    // `hist` keeps the store counts of the last D tiles, 2 bits each)
    const int64_t later = n_t - 1 - i < D - 1 ? n_t - 1 - i : D - 1;
    int stores = 0;
#pragma unroll
    for (int e = 0; e < D; ++e) stores += (hist >> (2 * e)) & 3u;
    wait_vm_le<(D - 1) * LPT + D * SPT>(__builtin_amdgcn_readfirstlane((int)later * LPT + stores));
    __asm__ volatile("" ::: "memory");
    const lds_u8* st = ring + d * STAGE;
    const f32x4 gv[2] = {*(const __attribute__((address_space(3))) f32x4*)(st + 32 * lane),
                         *(const __attribute__((address_space(3))) f32x4*)(st + 32 * lane + 16)};
    uint32_t win[4] = {0u, 0u, 0u, 0u};
    const lds_u8* cp = st + 2048 + NB * lane;
    if constexpr (NB == 2) {
      win[0] = *(const __attribute__((address_space(3))) uint16_t*)cp;
    } else if constexpr (NB == 3) {
      win[0] = (uint32_t)cp[0] | ((uint32_t)cp[1] << 8) | ((uint32_t)cp[2] << 16);
    } else if constexpr (NB == 4) {
      win[0] = *(const __attribute__((address_space(3))) uint32_t*)cp;
    } else {
      typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));
      const u32x2_t v = *(const __attribute__((address_space(3))) u32x2_t*)cp;
      win[0] = v[0];
      win[1] = v[1];
    }
    // the stage has been read: refill it with tile i + D
    __asm__ volatile("s_waitcnt lgkmcnt(0)" ::: "memory");
    if (i + D < n_t) issue(d, tl + D * t_inc);
    if (tl >= dc.tile0 + (dc.nchunks + kChunksPerTile - 1) / kChunksPerTile) {
      flush_tensor(sc);
      do dc = tab.get(++sc);
      while (tl >= dc.tile0 + (dc.nchunks + kChunksPerTile - 1) / kChunksPerTile);
    }
    const int64_t c0 = (tl - dc.tile0) * kChunksPerTile + 64 * wv;
    const int64_t t = c0 + lane;
    hist = ((hist << 2) | (c0 < dc.nchunks ? (uint32_t)SPT : 0u)) & ((1u << (2 * D)) - 1u);
    if (t < dc.nchunks) {
      SRArgs a;
      a.c = dc.c;
      a.L = dc.L;
      a.qmin = dc.qmin;
      a.qmax = dc.qmax;
      a.k0 = k0;
      a.k1 = k1;
      a.step = step;
      a.tid = dc.tid;
      uint32_t wout[4];
      sr_chunk<CF, kCW>(win, gv, (uint64_t)t, a, wout, ch, nf);
      CIO::store(dc.wq, t, wout);
    }
    d = d + 1 == D ? 0 : d + 1;
  }
  flush_tensor(sc);
  // the launch totals: one atomic per block (atomics from every wave on
  // one address serialise and had held the update far below bandwidth)
  if (counters != nullptr) {
    const uint32_t c = block_sum(ch_done, red), f = block_sum(nf_done, red);
    if (threadIdx.x == 0) {
      if (c) atomicAdd(counters, (unsigned long long)c);
      if (f) atomicAdd(counters + 1, (unsigned long long)f);
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
  int per_cu = 0;
  if (hipOccupancyMaxActiveBlocksPerMultiprocessor(&per_cu, fn, threads, 0) != hipSuccess || per_cu <= 0)
    per_cu = 4;
  return current_device_cus() * per_cu;
}

template <int CF, class Tab>
static hipError_t launch_sr_cf(const Tab& tab, int64_t tiles, uint64_t seed, uint32_t step,
                               unsigned long long* counters, unsigned long long* per_tensor,
                               hipStream_t stream) {
  const auto kern = sr_update_kernel<CF, Tab>;
  const int64_t cap = occupancy_blocks(reinterpret_cast<const void*>(kern), 256);
  const unsigned blocks = (unsigned)(tiles < cap ? tiles : cap);
  return launch_kernel(kern, dim3(blocks), dim3(256), stream, tab, tiles, (uint32_t)seed,
                       (uint32_t)(seed >> 32), step, counters, per_tensor);
}

template <class Tab>
static hipError_t launch_sr(int cf, const Tab& tab, int64_t tiles, uint64_t seed, uint32_t step,
                            unsigned long long* counters, unsigned long long* per_tensor,
                            hipStream_t stream) {
  if (tiles == 0) return hipSuccess;
  if (cf == CF_T2) return launch_sr_cf<CF_T2>(tab, tiles, seed, step, counters, per_tensor, stream);
  if (cf == CF_I4) return launch_sr_cf<CF_I4>(tab, tiles, seed, step, counters, per_tensor, stream);
  if (cf == CF_I3) return launch_sr_cf<CF_I3>(tab, tiles, seed, step, counters, per_tensor, stream);
  return launch_sr_cf<CF_I8>(tab, tiles, seed, step, counters, per_tensor, stream);
}

static int64_t tiles_of(int64_t nweights) {
  return (nweights / kCW + kChunksPerTile - 1) / kChunksPerTile;
}

hipError_t launch_sr_update(int cf, int n, const SRTensor* t, uint64_t seed, uint32_t step,
                            unsigned long long* counters, hipStream_t stream) {
  SRArgTab tab{};
  tab.n = n;
  int64_t tiles = 0;
  for (int s = 0; s < n; ++s) {
    SRDesc& d = tab.d[s];
    d.wq = t[s].wq;
    d.grad = t[s].grad;
    d.nchunks = t[s].nweights / kCW;
    d.tile0 = tiles;
    d.c = t[s].c;
    d.L = (float)(t[s].qmax - t[s].qmin + 1);
    d.qmin = t[s].qmin;
    d.qmax = t[s].qmax;
    d.tid = t[s].tensor_id;
    tiles += tiles_of(t[s].nweights);
  }
  return launch_sr(cf, tab, tiles, seed, step, counters, nullptr, stream);
}

void sr_table_entry(const SRTensor& t, int64_t tile0, SRTableEntry* e) {
  *e = SRTableEntry{};
  e->wq = reinterpret_cast<uint64_t>(t.wq);
  e->grad = reinterpret_cast<uint64_t>(t.grad);
  e->nchunks = t.nweights / kCW;
  e->tile0 = tile0;
  e->alpha = t.alpha;
  e->qmin = t.qmin;
  e->qmax = t.qmax;
  e->tensor_id = t.tensor_id;
}

int64_t sr_tiles(int64_t nweights) { return tiles_of(nweights); }

hipError_t launch_sr_update_table(int cf, int n, int64_t total_weights_tiles, const SRTableEntry* table,
                                  float lr, uint64_t seed, uint32_t step, unsigned long long* counters,
                                  unsigned long long* per_tensor, hipStream_t stream) {
  SRDevTab tab{table, n, lr};
  return launch_sr(cf, tab, total_weights_tiles, seed, step, counters, per_tensor, stream);
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
