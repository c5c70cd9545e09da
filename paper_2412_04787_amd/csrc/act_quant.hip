// Per-token 8-bit activation quantisation (Sec. 3.2: inputs and activations
// are quantised to 8 bits following BitNet): absmax per row, then int8 or
// OCP e4m3 codes plus one fp32 dequantisation scale per row.
//
// HBM-bound: reads the row (2 or 4 B/element) once and writes 1 B/element.
// One wave per row.  Rows of up to 64 x 24 16-byte chunks are held in
// registers between the absmax and the quantisation (the row is read from
// memory once); longer rows are read twice, the second time from cache.
// Up to kMaxBatch inputs (same M and dtypes) are quantised by one launch.
#include "dqt_launch.h"

namespace dqt {

namespace {

typedef int i32x4v __attribute__((ext_vector_type(4)));

template <typename TX>
struct RowChunk;  // 16-byte chunk of a row: 8 bf16 or 4 fp32 values

template <>
struct RowChunk<uint16_t> {  // bf16 bits
  static constexpr int kElems = 8;
  __device__ static void decode(i32x4v u, float (&v)[8]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) {
      v[2 * i] = bf16_bits_to_f32((uint32_t)u[i] & 0xFFFFu);
      v[2 * i + 1] = bf16_bits_to_f32((uint32_t)u[i] >> 16);
    }
  }
};
template <>
struct RowChunk<float> {
  static constexpr int kElems = 4;
  __device__ static void decode(i32x4v u, float (&v)[4]) {
#pragma unroll
    for (int i = 0; i < 4; ++i) v[i] = __int_as_float(u[i]);
  }
};

struct ActTab {
  const void* X[kMaxBatch];
  uint8_t* Xq[kMaxBatch];
  float* xdq[kMaxBatch];
  int32_t K[kMaxBatch];
  int32_t nch[kMaxBatch];      // 16-lane kernel: chunks per lane of each input
  int32_t b0[kMaxBatch + 1];   // first block of each input
  int32_t n;
  int64_t M;
};

constexpr int kRowsPerBlock = 4;

__device__ __forceinline__ int seg_of(const ActTab& t) {
  int s = 0;
  while (s + 1 < t.n && (int)blockIdx.x >= t.b0[s + 1]) ++s;
  return s;
}

template <bool E4M3, int E>
__device__ __forceinline__ void quantise_store(const float (&v)[E], float inv, uint8_t* dst) {
  uint32_t out[E / 4];
#pragma unroll
  for (int w = 0; w < E / 4; ++w) {
    if constexpr (E4M3) {
      out[w] = f32x4_to_e4m3x4(v[4 * w] * inv, v[4 * w + 1] * inv, v[4 * w + 2] * inv, v[4 * w + 3] * inv);
    } else {
      out[w] = f32x4_to_i8x4(v[4 * w] * inv, v[4 * w + 1] * inv, v[4 * w + 2] * inv, v[4 * w + 3] * inv);
    }
  }
  if constexpr (E == 8) {
    *reinterpret_cast<uint2*>(dst) = make_uint2(out[0], out[1]);
  } else {
    *reinterpret_cast<uint32_t*>(dst) = out[0];
  }
}

// NCH > 0: the lane's chunks lane, lane + 64, ... (at most NCH of them) stay
// in registers.  NCH == 0: two passes over the row.
template <typename TX, bool E4M3, int NCH>
__global__ __launch_bounds__(256) void act_quant_kernel(const ActTab tab) {
  using C = RowChunk<TX>;
  constexpr int E = C::kElems;
  const int s = seg_of(tab);
  const int lane = threadIdx.x & (kWave - 1);
  const int64_t row = (int64_t)(blockIdx.x - tab.b0[s]) * kRowsPerBlock + (threadIdx.x / kWave);
  if (row >= tab.M) return;
  const int K = tab.K[s];
  const TX* xr = static_cast<const TX*>(tab.X[s]) + row * (int64_t)K;
  uint8_t* qr = tab.Xq[s] + row * (int64_t)K;
  const int nchunk = K / E;
  const float qscale = E4M3 ? 448.0f : 127.0f;

  float amax = 0.0f;
  if constexpr (NCH > 0) {
    i32x4v raw[NCH];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int idx = lane + kWave * c;
      raw[c] = __builtin_nontemporal_load(reinterpret_cast<const i32x4v*>(xr + (idx < nchunk ? idx : nchunk - 1) * E));
    }
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      float v[E];
      C::decode(raw[c], v);
      float m = 0.0f;
#pragma unroll
      for (int i = 0; i < E; ++i) m = fmaxf(m, fabsf(v[i]));
      amax = lane + kWave * c < nchunk ? fmaxf(amax, m) : amax;
    }
    amax = wave_max(amax);
    const float g = fmaxf(amax, 1e-5f);
    const float inv = qscale / g;   // correctly rounded fp32 division
    if (lane == 0) tab.xdq[s][row] = g / qscale;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
      const int idx = lane + kWave * c;
      if (idx < nchunk) {
        float v[E];
        C::decode(raw[c], v);
        quantise_store<E4M3, E>(v, inv, qr + idx * E);
      }
    }
  } else {
    for (int c = lane; c < nchunk; c += kWave) {
      float v[E];
      C::decode(*reinterpret_cast<const i32x4v*>(xr + c * E), v);
#pragma unroll
      for (int i = 0; i < E; ++i) amax = fmaxf(amax, fabsf(v[i]));
    }
    amax = wave_max(amax);
    const float g = fmaxf(amax, 1e-5f);
    const float inv = qscale / g;
    if (lane == 0) tab.xdq[s][row] = g / qscale;
    for (int c = lane; c < nchunk; c += kWave) {
      float v[E];
      C::decode(*reinterpret_cast<const i32x4v*>(xr + c * E), v);
      quantise_store<E4M3, E>(v, inv, qr + c * E);
    }
  }
}

// Rows of up to 16 x 16 chunks: 16 lanes per row, 4 rows per wave, 16 rows
// per block.  A row's chunks are lane, lane + 16, ... (each load instruction
// reads 256 contiguous bytes of 4 rows) and stay in registers; the row max
// is formed by rotations within the 16-lane DPP row, without LDS.
__device__ __forceinline__ float row16_max(float v) {
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x128, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x124, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x122, 0xF, 0xF, false)));
  v = fmaxf(v, __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(v), 0x121, 0xF, 0xF, false)));
  return v;
}
constexpr int kRows16 = 16;   // rows per block of the 16-lane kernel

template <typename TX, bool E4M3, int NCH>
__device__ __forceinline__ void act_quant16_rows(const ActTab& tab, int s) {
  using C = RowChunk<TX>;
  constexpr int E = C::kElems;
  const int lane = threadIdx.x & (kWave - 1);
  const int l16 = lane & 15;
  const int64_t row = (int64_t)(blockIdx.x - tab.b0[s]) * kRows16 + (threadIdx.x >> 4);
  const bool valid = row < tab.M;
  const int K = tab.K[s];
  const TX* xr = static_cast<const TX*>(tab.X[s]) + (valid ? row : 0) * (int64_t)K;
  uint8_t* qr = tab.Xq[s] + row * (int64_t)K;
  const int nchunk = K / E;
  const float qscale = E4M3 ? 448.0f : 127.0f;
  // every lane loads all NCH chunks (past the row end it reloads the last
  // one), so the loads issue back to back; those chunks do not count
  i32x4v raw[NCH];
  float amax = 0.0f;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int idx = l16 + 16 * c;
    raw[c] = __builtin_nontemporal_load(reinterpret_cast<const i32x4v*>(xr + (idx < nchunk ? idx : nchunk - 1) * E));
  }
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    float v[E];
    C::decode(raw[c], v);
    float m = 0.0f;
#pragma unroll
    for (int i = 0; i < E; ++i) m = fmaxf(m, fabsf(v[i]));
    amax = l16 + 16 * c < nchunk ? fmaxf(amax, m) : amax;
  }
  amax = row16_max(amax);
  const float g = fmaxf(amax, 1e-5f);
  const float inv = qscale / g;   // correctly rounded fp32 division
  if (valid && l16 == 0) tab.xdq[s][row] = g / qscale;
#pragma unroll
  for (int c = 0; c < NCH; ++c) {
    const int idx = l16 + 16 * c;
    if (valid && idx < nchunk) {
      float v[E];
      C::decode(raw[c], v);
      quantise_store<E4M3, E>(v, inv, qr + idx * E);
    }
  }
}

// Inputs of any row length up to 256 chunks in one launch: each block runs
// the variant of its input (a uniform branch), 16 rows per block.
template <typename TX, bool E4M3>
__global__ __launch_bounds__(256) void act_quant16_kernel(const ActTab tab) {
  const int s = seg_of(tab);
  switch (tab.nch[s]) {
    case 1: act_quant16_rows<TX, E4M3, 1>(tab, s); break;
    case 2: act_quant16_rows<TX, E4M3, 2>(tab, s); break;
    case 4: act_quant16_rows<TX, E4M3, 4>(tab, s); break;
    case 8: act_quant16_rows<TX, E4M3, 8>(tab, s); break;
    default: act_quant16_rows<TX, E4M3, 16>(tab, s); break;
  }
}

template <typename TX, bool E4M3>
hipError_t launch16_t(const ActTab& tab, int32_t blocks, hipStream_t stream) {
  return launch_kernel(act_quant16_kernel<TX, E4M3>, dim3((unsigned)blocks), dim3(256), stream, tab);
}

template <typename TX, bool E4M3>
hipError_t launch_t(const ActTab& tab, int nch, int32_t blocks, hipStream_t stream) {
  const dim3 grid((unsigned)blocks), block(kRowsPerBlock * kWave);
  switch (nch) {
    case 1: return launch_kernel(act_quant_kernel<TX, E4M3, 1>, grid, block, stream, tab);
    case 2: return launch_kernel(act_quant_kernel<TX, E4M3, 2>, grid, block, stream, tab);
    case 4: return launch_kernel(act_quant_kernel<TX, E4M3, 4>, grid, block, stream, tab);
    case 8: return launch_kernel(act_quant_kernel<TX, E4M3, 8>, grid, block, stream, tab);
    case 16: return launch_kernel(act_quant_kernel<TX, E4M3, 16>, grid, block, stream, tab);
    case 24: return launch_kernel(act_quant_kernel<TX, E4M3, 24>, grid, block, stream, tab);
    default: return launch_kernel(act_quant_kernel<TX, E4M3, 0>, grid, block, stream, tab);
  }
}

}  // namespace

// Kernel variant of a row of `chunks` 16-byte chunks: 16 lanes per row with
// NCH chunks per lane (code 16 + NCH), or a whole wave per row with NCH
// chunks per lane (code 64 + NCH; NCH 0: two passes over the row).
static int act_variant(int chunks) {
  if (chunks <= 16 * 16) {
    const int per = (chunks + 15) / 16;
    for (int c : {1, 2, 4, 8, 16})
      if (per <= c) return 16 + c;
  }
  const int per = (chunks + kWave - 1) / kWave;
  for (int c : {1, 2, 4, 8, 16, 24})
    if (per <= c) return 64 + c;
  return 64;
}

hipError_t launch_act_quant_batch(int n, const ActIO* io, bool x_bf16, int64_t M, bool e4m3,
                                  hipStream_t stream) {
  if (M == 0 || n == 0) return hipSuccess;
  const int E = x_bf16 ? 8 : 4;
  // one launch for every input of at most 256 chunks per row (16 lanes per
  // row, the chunk count per lane chosen per input), one per variant of the
  // whole-wave kernel for longer rows
  bool done[kMaxBatch] = {};
  LaunchStatus st;
  for (int s0 = 0; s0 < n; ++s0) {
    if (done[s0]) continue;
    const int var = act_variant(io[s0].K / E);
    const bool v16 = var < 64;
    ActTab tab{};
    tab.M = M;
    const int rows_per_block = v16 ? kRows16 : kRowsPerBlock;
    int32_t blocks = 0;
    for (int s = s0; s < n; ++s) {
      const int vs = act_variant(io[s].K / E);
      if (done[s] || (v16 ? vs >= 64 : vs != var)) continue;
      done[s] = true;
      const int t = tab.n++;
      tab.X[t] = io[s].X;
      tab.Xq[t] = static_cast<uint8_t*>(io[s].Xq);
      tab.xdq[t] = io[s].xdq;
      tab.K[t] = io[s].K;
      tab.nch[t] = v16 ? vs - 16 : 0;
      tab.b0[t] = blocks;
      blocks += (int32_t)((M + rows_per_block - 1) / rows_per_block);
    }
    tab.b0[tab.n] = blocks;
    if (v16) {
      if (x_bf16) {
        if (e4m3) st << launch16_t<uint16_t, true>(tab, blocks, stream);
        else st << launch16_t<uint16_t, false>(tab, blocks, stream);
      } else {
        if (e4m3) st << launch16_t<float, true>(tab, blocks, stream);
        else st << launch16_t<float, false>(tab, blocks, stream);
      }
    } else {
      const int nch = var - 64;
      if (x_bf16) {
        if (e4m3) st << launch_t<uint16_t, true>(tab, nch, blocks, stream);
        else st << launch_t<uint16_t, false>(tab, nch, blocks, stream);
      } else {
        if (e4m3) st << launch_t<float, true>(tab, nch, blocks, stream);
        else st << launch_t<float, false>(tab, nch, blocks, stream);
      }
    }
  }
  return st.e;
}

hipError_t launch_act_quant(const void* X, bool x_bf16, int64_t M, int K, bool e4m3, void* Xq,
                            float* xdq, hipStream_t stream) {
  const ActIO io{X, Xq, xdq, K};
  return launch_act_quant_batch(1, &io, x_bf16, M, e4m3, stream);
}

}  // namespace dqt
