// C ABI of libdqt: argument checking and dispatch to the gfx950 kernels.
// Every check runs before anything is enqueued; see include/dqt.h for the
// contract of each entry point.
#include <math.h>
#include <string.h>

#include "../../include/dqt.h"
#include "dqt_launch.h"

namespace {

constexpr int32_t kVersion = 1 * 10000 + 0 * 100 + 0;
// |acc| <= 128 * 128 * d_in must stay below 2^31 for the int32 forward.
constexpr int64_t kMaxDin = 65536;

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15u) == 0; }

dqt_status check_weight(const dqt_weight* w) {
  if (w == nullptr) return DQT_ERR_NULL;
  if (w->d_in < 16 || w->d_out < 16 || (w->d_in % 16) != 0 || (w->d_out % 16) != 0)
    return DQT_ERR_SHAPE;
  if (w->d_in > kMaxDin) return DQT_ERR_SHAPE;
  if (w->reserved != 0) return DQT_ERR_RANGE;
  if (w->wfmt == DQT_TERNARY2) {
    if (w->qmin != -1 || w->qmax != 1) return DQT_ERR_RANGE;
  } else if (w->wfmt == DQT_I8) {
    if (w->qmin < -128 || w->qmax > 127 || w->qmin >= w->qmax) return DQT_ERR_RANGE;
  } else {
    return DQT_ERR_DTYPE;
  }
  if (!(isfinite(w->alpha) && w->alpha > 0.0f)) return DQT_ERR_RANGE;
  return DQT_OK;
}

bool is_float_type(int32_t t) { return t == DQT_F32 || t == DQT_BF16; }

dqt_status from_hip(hipError_t e) { return e == hipSuccess ? DQT_OK : DQT_ERR_HIP; }

}  // namespace

extern "C" {

const char* dqt_status_string(int32_t status) {
  switch (status) {
    case DQT_OK: return "DQT_OK";
    case DQT_ERR_NULL: return "DQT_ERR_NULL: a required pointer is NULL";
    case DQT_ERR_SHAPE: return "DQT_ERR_SHAPE: a dimension is out of range or not a multiple of 16";
    case DQT_ERR_ALIGN: return "DQT_ERR_ALIGN: a pointer is not 16-byte aligned";
    case DQT_ERR_DTYPE: return "DQT_ERR_DTYPE: a dtype is not allowed in that position";
    case DQT_ERR_RANGE: return "DQT_ERR_RANGE: qmin/qmax/alpha/lr out of range";
    case DQT_ERR_WORKSPACE: return "DQT_ERR_WORKSPACE: workspace missing or too small";
    case DQT_ERR_UNSUPPORTED: return "DQT_ERR_UNSUPPORTED: combination not implemented";
    case DQT_ERR_HIP: return "DQT_ERR_HIP: the HIP runtime reported an error";
    default: return "unknown dqt_status";
  }
}

int32_t dqt_version(void) { return kVersion; }

dqt_status dqt_act_quant(const void* X, int32_t x_t, int64_t M, int32_t K, int32_t act_q,
                         void* Xq, float* xdq, void* stream) {
  if (M < 0 || K < 16 || (K % 16) != 0) return DQT_ERR_SHAPE;
  if (!is_float_type(x_t) || (act_q != DQT_I8 && act_q != DQT_FP8E4M3)) return DQT_ERR_DTYPE;
  if (M == 0) return DQT_OK;
  if (X == nullptr || Xq == nullptr || xdq == nullptr) return DQT_ERR_NULL;
  if (!aligned16(X) || !aligned16(Xq) || !aligned16(xdq)) return DQT_ERR_ALIGN;
  return from_hip(dqt::launch_act_quant(X, x_t == DQT_BF16, M, K, act_q == DQT_FP8E4M3, Xq, xdq,
                                        static_cast<hipStream_t>(stream)));
}

size_t dqt_linear_fwd_workspace(const dqt_weight* w) {
  if (check_weight(w) != DQT_OK) return 0;
  return dqt::fwd_workspace_bytes(w->wfmt == DQT_TERNARY2, w->d_out, w->d_in);
}

dqt_status dqt_linear_fwd(const dqt_weight* w, const void* Wq, const void* X, int32_t x_t,
                          int64_t M, int32_t act_q, void* Xq, float* xdq, void* Y, int32_t y_t,
                          void* ws, size_t ws_bytes, void* stream) {
  dqt_status st = check_weight(w);
  if (st != DQT_OK) return st;
  if (M < 0) return DQT_ERR_SHAPE;
  if (act_q != DQT_I8 && act_q != DQT_FP8E4M3) return DQT_ERR_DTYPE;
  if (!is_float_type(y_t)) return DQT_ERR_DTYPE;
  if (X != nullptr && !is_float_type(x_t)) return DQT_ERR_DTYPE;
  if (act_q == DQT_FP8E4M3 && w->wfmt != DQT_TERNARY2) return DQT_ERR_UNSUPPORTED;
  if (M == 0) return DQT_OK;
  if (Wq == nullptr || Xq == nullptr || xdq == nullptr || Y == nullptr) return DQT_ERR_NULL;
  if (!aligned16(Wq) || !aligned16(Xq) || !aligned16(xdq) || !aligned16(Y) ||
      (X != nullptr && !aligned16(X)))
    return DQT_ERR_ALIGN;
  const size_t need = dqt_linear_fwd_workspace(w);
  if (need > 0 && (ws == nullptr || ws_bytes < need)) return DQT_ERR_WORKSPACE;
  if (need > 0 && !aligned16(ws)) return DQT_ERR_ALIGN;
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (X != nullptr) {
    st = from_hip(dqt::launch_act_quant(X, x_t == DQT_BF16, M, w->d_in, act_q == DQT_FP8E4M3, Xq,
                                        xdq, s));
    if (st != DQT_OK) return st;
  }
  dqt::FwdArgs a;
  a.Xq = Xq;
  a.xdq = xdq;
  a.Wq = Wq;
  a.Y = Y;
  a.M = M;
  a.d_in = w->d_in;
  a.d_out = w->d_out;
  a.ws = ws;
  a.alpha = w->alpha;
  a.w_ternary = w->wfmt == DQT_TERNARY2;
  a.act_e4m3 = act_q == DQT_FP8E4M3;
  a.y_bf16 = y_t == DQT_BF16;
  return from_hip(dqt::launch_fwd_v2(a, s));
}

// Backward workspace layout (each region 256-byte aligned):
//   [fp32 split partials: splits * d_out * d_in]   (when splits > 1)
//   [bf16 weights: d_out * d_in]                   (bf16-environment dX)
//   [bf16 X~: M * d_in]                            (bf16-environment dW)
struct BwdLayout {
  int64_t splits;
  size_t part, q, xt, total;
};
static size_t align256(size_t n) { return (n + 255) / 256 * 256; }
static BwdLayout bwd_layout(const dqt_weight* w, int64_t M) {
  BwdLayout L;
  int wj;
  int64_t s_v2;
  dqt::plan_dw_v2(w->d_out, w->d_in, M, &wj, &s_v2);
  const int64_t s_f32 = dqt::dw_splits_f32(w->d_out, w->d_in, M);
  L.splits = s_v2 > s_f32 ? s_v2 : s_f32;
  const size_t wn = (size_t)w->d_out * (size_t)w->d_in;
  L.part = L.splits > 1 ? align256((size_t)L.splits * wn * sizeof(float)) : 0;
  L.q = align256(wn * 2);
  L.xt = align256((size_t)M * (size_t)w->d_in * 2);
  L.total = L.part + L.q + L.xt;
  return L;
}

size_t dqt_linear_bwd_workspace(const dqt_weight* w, int64_t M) {
  if (check_weight(w) != DQT_OK || M < 0) return 0;
  return bwd_layout(w, M).total;
}

dqt_status dqt_linear_bwd(const dqt_weight* w, const void* Wq, const void* Xq, int32_t act_q,
                          const float* xdq, const void* dY, int32_t dy_t, int64_t M,
                          int32_t xt_t, void* dX, int32_t dx_t, float* dW, void* ws,
                          size_t ws_bytes, void* stream) {
  dqt_status st = check_weight(w);
  if (st != DQT_OK) return st;
  if (M < 0) return DQT_ERR_SHAPE;
  if (act_q != DQT_I8 && act_q != DQT_FP8E4M3) return DQT_ERR_DTYPE;
  if (!is_float_type(dy_t) || !is_float_type(xt_t)) return DQT_ERR_DTYPE;
  if (dX != nullptr && !is_float_type(dx_t)) return DQT_ERR_DTYPE;
  if (dW != nullptr && dy_t != xt_t) return DQT_ERR_UNSUPPORTED;
  if (dX == nullptr && dW == nullptr) return DQT_OK;
  const BwdLayout L = bwd_layout(w, M);
  if (ws == nullptr || ws_bytes < L.total) return DQT_ERR_WORKSPACE;
  if (!aligned16(ws)) return DQT_ERR_ALIGN;
  uint8_t* wsb = static_cast<uint8_t*>(ws);
  if (dW != nullptr) {
    if (!aligned16(dW)) return DQT_ERR_ALIGN;
    if (M > 0 && (Xq == nullptr || xdq == nullptr)) return DQT_ERR_NULL;
  }
  if (M > 0) {
    if (dY == nullptr) return DQT_ERR_NULL;
    if (!aligned16(dY)) return DQT_ERR_ALIGN;
    if (Xq != nullptr && !aligned16(Xq)) return DQT_ERR_ALIGN;
    if (xdq != nullptr && !aligned16(xdq)) return DQT_ERR_ALIGN;
  }
  if (dX != nullptr) {
    if (M > 0 && Wq == nullptr) return DQT_ERR_NULL;
    if (!aligned16(dX) || (Wq != nullptr && !aligned16(Wq))) return DQT_ERR_ALIGN;
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  if (dX != nullptr && M > 0) {
    dqt::DxArgs a;
    a.dY = dY;
    a.Wq = Wq;
    a.dX = dX;
    a.M = M;
    a.d_in = w->d_in;
    a.d_out = w->d_out;
    a.alpha = w->alpha;
    a.w_ternary = w->wfmt == DQT_TERNARY2;
    a.dy_bf16 = dy_t == DQT_BF16;
    a.dx_bf16 = dx_t == DQT_BF16;
    st = from_hip(a.dy_bf16 ? dqt::launch_dx_v2(a, wsb + L.part, s) : dqt::launch_dx_f32(a, s));
    if (st != DQT_OK) return st;
  }
  if (dW != nullptr) {
    dqt::DwArgs a;
    a.dY = dY;
    a.Xq = Xq;
    a.xdq = xdq;
    a.dW = dW;
    a.ws = reinterpret_cast<float*>(wsb);
    a.M = M;
    a.d_in = w->d_in;
    a.d_out = w->d_out;
    a.splits = L.splits;
    a.act_e4m3 = act_q == DQT_FP8E4M3;
    a.xt_bf16 = xt_t == DQT_BF16;
    st = from_hip(a.xt_bf16 ? dqt::launch_dw_v2(a, wsb + L.part + L.q, s) : dqt::launch_dw_f32(a, s));
  }
  return st;
}

dqt_status dqt_sr_update(const dqt_weight* w, void* Wq, const float* dW, float lr, uint64_t seed,
                         uint32_t step, unsigned long long* counters, void* stream) {
  dqt_status st = check_weight(w);
  if (st != DQT_OK) return st;
  if (Wq == nullptr || dW == nullptr) return DQT_ERR_NULL;
  if (!aligned16(Wq) || !aligned16(dW)) return DQT_ERR_ALIGN;
  if (counters != nullptr && (reinterpret_cast<uintptr_t>(counters) & 7u) != 0) return DQT_ERR_ALIGN;
  if (!(isfinite(lr) && lr >= 0.0f)) return DQT_ERR_RANGE;
  const float c = lr / w->alpha;  // one correctly rounded fp32 division
  if (!isfinite(c)) return DQT_ERR_RANGE;
  const int64_t n = (int64_t)w->d_out * (int64_t)w->d_in;
  return from_hip(dqt::launch_sr_update(w->wfmt == DQT_TERNARY2, static_cast<uint8_t*>(Wq), dW, n,
                                        c, w->qmin, w->qmax, seed, step, w->tensor_id, counters,
                                        static_cast<hipStream_t>(stream)));
}

dqt_status dqt_debug_rng(uint64_t seed, uint32_t step, uint32_t tensor_id, uint64_t i0, int64_t n,
                         uint32_t* out, void* stream) {
  if (n < 0) return DQT_ERR_SHAPE;
  if (n == 0) return DQT_OK;
  if (out == nullptr) return DQT_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(out) & 3u) != 0) return DQT_ERR_ALIGN;
  return from_hip(dqt::launch_debug_rng(seed, step, tensor_id, i0, n, out,
                                        static_cast<hipStream_t>(stream)));
}

dqt_status dqt_absmean_init(const float* W0, int64_t n, int32_t qmin, int32_t qmax, int8_t* q,
                            float* alpha) {
  if (W0 == nullptr || q == nullptr || alpha == nullptr) return DQT_ERR_NULL;
  if (n <= 0) return DQT_ERR_SHAPE;
  if (qmin < -128 || qmax > 127 || qmin >= qmax || qmax <= 0) return DQT_ERR_RANGE;
  double sum = 0.0;
  for (int64_t i = 0; i < n; ++i) sum += fabs((double)W0[i]);
  const double am = sum / (double)n;
  if (!(am > 0.0) || !isfinite(am)) return DQT_ERR_RANGE;
  const double s = (double)qmax / am;
  for (int64_t i = 0; i < n; ++i) {
    double v = nearbyint((double)W0[i] * s);   // default rounding: half to even
    v = v < qmin ? qmin : (v > qmax ? qmax : v);
    q[i] = (int8_t)v;
  }
  *alpha = (float)(am / (double)qmax);
  return DQT_OK;
}

dqt_status dqt_pack_ternary(const int8_t* q, int64_t rows, int64_t cols, uint8_t* packed) {
  if (q == nullptr || packed == nullptr) return DQT_ERR_NULL;
  if (rows < 0 || cols < 0 || (cols % 4) != 0) return DQT_ERR_SHAPE;
  const int64_t pc = cols / 4;
  for (int64_t r = 0; r < rows; ++r) {
    for (int64_t b = 0; b < pc; ++b) {
      uint32_t byte = 0;
      for (int j = 0; j < 4; ++j) {
        const int v = q[r * cols + 4 * b + j];
        if (v < -1 || v > 1) return DQT_ERR_RANGE;
        byte |= (uint32_t)(v + 1) << (2 * j);
      }
      packed[r * pc + b] = (uint8_t)byte;
    }
  }
  return DQT_OK;
}

dqt_status dqt_unpack_ternary(const uint8_t* packed, int64_t rows, int64_t cols, int8_t* q) {
  if (q == nullptr || packed == nullptr) return DQT_ERR_NULL;
  if (rows < 0 || cols < 0 || (cols % 4) != 0) return DQT_ERR_SHAPE;
  const int64_t pc = cols / 4;
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t b = 0; b < pc; ++b)
      for (int j = 0; j < 4; ++j)
        q[r * cols + 4 * b + j] = (int8_t)((int)((packed[r * pc + b] >> (2 * j)) & 3u) - 1);
  return DQT_OK;
}

}  // extern "C"
