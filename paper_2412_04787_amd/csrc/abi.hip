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
  } else if (w->wfmt == DQT_INT4) {
    if (w->qmin < -8 || w->qmax > 7 || w->qmin >= w->qmax) return DQT_ERR_RANGE;
  } else if (w->wfmt == DQT_INT3) {
    if (w->qmin < -4 || w->qmax > 3 || w->qmin >= w->qmax) return DQT_ERR_RANGE;
  } else {
    return DQT_ERR_DTYPE;
  }
  if (!(isfinite(w->alpha) && w->alpha > 0.0f)) return DQT_ERR_RANGE;
  return DQT_OK;
}

// code format of the update kernels: 0 int8, 1 ternary 2-bit, 2 int4 nibbles
int code_format(int32_t wfmt) {
  return wfmt == DQT_TERNARY2 ? 1 : wfmt == DQT_INT4 ? 2 : wfmt == DQT_INT3 ? 3 : 0;
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
  if (M < 0 || M > (int64_t(1) << 28) || K < 16 || (K % 16) != 0) return DQT_ERR_SHAPE;
  if (!is_float_type(x_t) || (act_q != DQT_I8 && act_q != DQT_FP8E4M3)) return DQT_ERR_DTYPE;
  if (M == 0) return DQT_OK;
  if (X == nullptr || Xq == nullptr || xdq == nullptr) return DQT_ERR_NULL;
  if (!aligned16(X) || !aligned16(Xq) || !aligned16(xdq)) return DQT_ERR_ALIGN;
  return from_hip(dqt::launch_act_quant(X, x_t == DQT_BF16, M, K, act_q == DQT_FP8E4M3, Xq, xdq,
                                        static_cast<hipStream_t>(stream)));
}

dqt_status dqt_rmsnorm_act_quant(const void* X, int32_t x_t, const float* gamma, float eps,
                                 int64_t M, int32_t K, int32_t act_q, void* Xq, float* xdq,
                                 float* rinv, void* stream) {
  if (M < 0 || M > (int64_t(1) << 28) || K < 16 || (K % 16) != 0) return DQT_ERR_SHAPE;
  if (!is_float_type(x_t) || (act_q != DQT_I8 && act_q != DQT_FP8E4M3)) return DQT_ERR_DTYPE;
  if (!(isfinite(eps) && eps > 0.0f)) return DQT_ERR_RANGE;
  if (M == 0) return DQT_OK;
  if (X == nullptr || gamma == nullptr || Xq == nullptr || xdq == nullptr) return DQT_ERR_NULL;
  if (!aligned16(X) || !aligned16(gamma) || !aligned16(Xq) || !aligned16(xdq)) return DQT_ERR_ALIGN;
  if (rinv != nullptr && (reinterpret_cast<uintptr_t>(rinv) & 3u) != 0) return DQT_ERR_ALIGN;
  return from_hip(dqt::launch_rmsnorm_act_quant(X, x_t == DQT_BF16, gamma, eps, M, K, act_q == DQT_FP8E4M3,
                                                Xq, xdq, rinv, static_cast<hipStream_t>(stream)));
}

dqt_status dqt_rmsnorm_backward(int32_t n_dy, const void* const* dY, const void* X, int32_t x_t,
                                const float* gamma, const float* rinv, int64_t M, int32_t K,
                                void* dX, float* gpart, int32_t blocks, void* stream) {
  if (n_dy < 1 || n_dy > dqt::kMaxNormDy) return DQT_ERR_SHAPE;
  if (M < 0 || M > (int64_t(1) << 28) || K < 16 || (K % 16) != 0 || K > 8192) return DQT_ERR_SHAPE;
  if (blocks < 1 || blocks > 65536) return DQT_ERR_SHAPE;
  if (x_t != DQT_BF16) return DQT_ERR_DTYPE;
  if (dY == nullptr || X == nullptr || gamma == nullptr || rinv == nullptr || dX == nullptr ||
      gpart == nullptr)
    return DQT_ERR_NULL;
  for (int i = 0; i < n_dy; ++i) {
    if (dY[i] == nullptr) return DQT_ERR_NULL;
    if (!aligned16(dY[i])) return DQT_ERR_ALIGN;
  }
  if (!aligned16(X) || !aligned16(gamma) || !aligned16(dX) || !aligned16(gpart)) return DQT_ERR_ALIGN;
  if ((reinterpret_cast<uintptr_t>(rinv) & 3u) != 0) return DQT_ERR_ALIGN;
  return from_hip(dqt::launch_rmsnorm_backward(n_dy, dY, X, gamma, rinv, M, K, dX, gpart, blocks,
                                               static_cast<hipStream_t>(stream)));
}

dqt_status dqt_act_quant_batch(int32_t n, const dqt_act_io* io, int32_t x_t, int64_t M,
                               int32_t act_q, void* stream) {
  if (n < 0 || n > DQT_MAX_BATCH) return DQT_ERR_SHAPE;
  if (n > 0 && io == nullptr) return DQT_ERR_NULL;
  if (M < 0 || M > (int64_t(1) << 28)) return DQT_ERR_SHAPE;
  if (!is_float_type(x_t) || (act_q != DQT_I8 && act_q != DQT_FP8E4M3)) return DQT_ERR_DTYPE;
  dqt::ActIO a[dqt::kMaxBatch];
  for (int s = 0; s < n; ++s) {
    if (io[s].K < 16 || (io[s].K % 16) != 0 || io[s].reserved != 0) return DQT_ERR_SHAPE;
    if (M > 0 && (io[s].X == nullptr || io[s].Xq == nullptr || io[s].xdq == nullptr)) return DQT_ERR_NULL;
    if (!aligned16(io[s].X) || !aligned16(io[s].Xq) || !aligned16(io[s].xdq)) return DQT_ERR_ALIGN;
    a[s] = dqt::ActIO{io[s].X, io[s].Xq, io[s].xdq, io[s].K};
  }
  if (M == 0 || n == 0) return DQT_OK;
  return from_hip(dqt::launch_act_quant_batch(n, a, x_t == DQT_BF16, M, act_q == DQT_FP8E4M3,
                                              static_cast<hipStream_t>(stream)));
}

// ----------------------------------------------------------------- batches

namespace {

// Checks shared by every batch call; fills the launcher's view of the batch.
dqt_status check_batch(int32_t n, const dqt_linear_io* io, dqt::LinearIO* L, int32_t* wfmt) {
  if (n < 1 || n > DQT_MAX_BATCH) return DQT_ERR_SHAPE;
  if (io == nullptr) return DQT_ERR_NULL;
  for (int l = 0; l < n; ++l) {
    const dqt_status st = check_weight(io[l].w);
    if (st != DQT_OK) return st;
    if (l == 0) *wfmt = io[l].w->wfmt;
    else if (io[l].w->wfmt != *wfmt) return DQT_ERR_UNSUPPORTED;
    L[l] = dqt::LinearIO{};
    L[l].d_in = io[l].w->d_in;
    L[l].d_out = io[l].w->d_out;
    L[l].alpha = io[l].w->alpha;
    L[l].Wq = io[l].Wq;
    L[l].Xq = io[l].Xq;
    L[l].xdq = io[l].xdq;
    L[l].Y = io[l].Y;
    L[l].dY = io[l].dY;
    L[l].dX = io[l].dX;
    L[l].dW = io[l].dW;
  }
  return DQT_OK;
}

}  // namespace

namespace {

// The smallest workspace a forward batch accepts (the packed form of ternary
// codes needs only the counters); 0 for a batch the checks refuse.
size_t fwd_batch_workspace_least(int32_t n, const dqt_linear_io* io) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  if (check_batch(n, io, L, &wfmt) != DQT_OK) return 0;
  return dqt::fwd_batch_workspace_min(n, L, code_format(wfmt));
}

}  // namespace

size_t dqt_linear_fwd_batch_workspace(int32_t n, const dqt_linear_io* io) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  if (check_batch(n, io, L, &wfmt) != DQT_OK) return 0;
  return dqt::fwd_batch_workspace(n, L, code_format(wfmt), nullptr);
}

dqt_status dqt_linear_fwd_batch(int32_t n, const dqt_linear_io* io, int64_t M, int32_t act_q,
                                int32_t y_t, void* ws, size_t ws_bytes, void* stream) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  dqt_status st = check_batch(n, io, L, &wfmt);
  if (st != DQT_OK) return st;
  if (M < 0) return DQT_ERR_SHAPE;
  if (act_q != DQT_I8 && act_q != DQT_FP8E4M3) return DQT_ERR_DTYPE;
  if (!is_float_type(y_t)) return DQT_ERR_DTYPE;
  // e4m3 operands hold the weights exactly only for |q| <= 16 (ternary, 4-bit)
  if (act_q == DQT_FP8E4M3 && wfmt == DQT_I8) return DQT_ERR_UNSUPPORTED;
  if (M == 0) return DQT_OK;
  for (int l = 0; l < n; ++l) {
    if (io[l].Wq == nullptr || io[l].Xq == nullptr || io[l].xdq == nullptr || io[l].Y == nullptr)
      return DQT_ERR_NULL;
    if (!aligned16(io[l].Wq) || !aligned16(io[l].Xq) || !aligned16(io[l].xdq) || !aligned16(io[l].Y))
      return DQT_ERR_ALIGN;
  }
  const size_t need = dqt::fwd_batch_workspace_min(n, L, code_format(wfmt));
  if (need > 0 && (ws == nullptr || ws_bytes < need)) return DQT_ERR_WORKSPACE;
  if (need > 0 && !aligned16(ws)) return DQT_ERR_ALIGN;
  dqt::BatchCfg c{n, M, wfmt == DQT_TERNARY2, act_q == DQT_FP8E4M3, y_t == DQT_BF16};
  c.w_int4 = wfmt == DQT_INT4;
  c.w_int3 = wfmt == DQT_INT3;
  return from_hip(dqt::launch_fwd_batch(c, L, static_cast<uint8_t*>(ws), ws == nullptr ? 0 : ws_bytes,
                                        static_cast<hipStream_t>(stream)));
}

size_t dqt_linear_bwd_batch_workspace(int32_t n, const dqt_linear_io* io, int64_t M) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  if (check_batch(n, io, L, &wfmt) != DQT_OK || M < 0) return 0;
  return dqt::plan_bwd_batch(n, L, M).total;
}

dqt_status dqt_linear_bwd_batch(int32_t n, const dqt_linear_io* io, int64_t M, int32_t act_q,
                                int32_t dy_t, int32_t xt_t, int32_t dx_t, void* ws,
                                size_t ws_bytes, void* stream) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  dqt_status st = check_batch(n, io, L, &wfmt);
  if (st != DQT_OK) return st;
  if (M < 0) return DQT_ERR_SHAPE;
  if (act_q != DQT_I8 && act_q != DQT_FP8E4M3) return DQT_ERR_DTYPE;
  if (!is_float_type(dy_t) || !is_float_type(xt_t) || !is_float_type(dx_t)) return DQT_ERR_DTYPE;
  bool any_dx = false, any_dw = false;
  for (int l = 0; l < n; ++l) {
    any_dx |= io[l].dX != nullptr;
    any_dw |= io[l].dW != nullptr;
  }
  if (any_dw && dy_t != xt_t) return DQT_ERR_UNSUPPORTED;
  if (!any_dx && !any_dw) return DQT_OK;
  const dqt::BwdPlan P = dqt::plan_bwd_batch(n, L, M);
  if (ws == nullptr || ws_bytes < P.total) return DQT_ERR_WORKSPACE;
  if (!aligned16(ws)) return DQT_ERR_ALIGN;
  for (int l = 0; l < n; ++l) {
    if (io[l].dW != nullptr) {
      if (!aligned16(io[l].dW)) return DQT_ERR_ALIGN;
      if (M > 0 && (io[l].Xq == nullptr || io[l].xdq == nullptr)) return DQT_ERR_NULL;
    }
    if ((io[l].dX != nullptr || io[l].dW != nullptr) && M > 0) {
      if (io[l].dY == nullptr) return DQT_ERR_NULL;
      if (!aligned16(io[l].dY)) return DQT_ERR_ALIGN;
    }
    if (io[l].Xq != nullptr && !aligned16(io[l].Xq)) return DQT_ERR_ALIGN;
    if (io[l].xdq != nullptr && !aligned16(io[l].xdq)) return DQT_ERR_ALIGN;
    if (io[l].dX != nullptr) {
      if (M > 0 && io[l].Wq == nullptr) return DQT_ERR_NULL;
      if (!aligned16(io[l].dX) || (io[l].Wq != nullptr && !aligned16(io[l].Wq))) return DQT_ERR_ALIGN;
    }
  }
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* wsb = static_cast<uint8_t*>(ws);
  dqt::LinearIO sub[DQT_MAX_BATCH];
  // every linear wants both gradients on the bf16 matrix-core path: one
  // launch holds the tiles of both products
  bool both = M > 0 && dy_t == DQT_BF16 && xt_t == DQT_BF16;
  for (int l = 0; l < n; ++l) both &= io[l].dX != nullptr && io[l].dW != nullptr;
  if (both) {
    dqt::BatchCfg c{n, M, wfmt == DQT_TERNARY2, act_q == DQT_FP8E4M3, dx_t == DQT_BF16};
    c.w_int4 = wfmt == DQT_INT4;
    c.w_int3 = wfmt == DQT_INT3;
    return from_hip(dqt::launch_dxdw_batch(c, L, wsb, P, s));
  }
  // dX for the linears that want it
  int nx = 0;
  dqt::BwdPlan Px = P;
  for (int l = 0; l < n; ++l)
    if (io[l].dX != nullptr) {
      Px.q_off[nx] = P.q_off[l];
      sub[nx++] = L[l];
    }
  if (nx > 0 && M > 0) {
    if (dy_t == DQT_BF16) {
      dqt::BatchCfg c{nx, M, wfmt == DQT_TERNARY2, act_q == DQT_FP8E4M3, dx_t == DQT_BF16};
      c.w_int4 = wfmt == DQT_INT4;
      c.w_int3 = wfmt == DQT_INT3;
      st = from_hip(dqt::launch_dx_batch(c, sub, wsb, Px, s));
    } else {
      for (int l = 0; l < nx && st == DQT_OK; ++l) {
        dqt::DxArgs a;
        a.dY = sub[l].dY;
        a.Wq = sub[l].Wq;
        if (wfmt == DQT_INT4 || wfmt == DQT_INT3) {
          // packed codes -> one int8 code per weight, in the weight area of the workspace
          int8_t* q8 = reinterpret_cast<int8_t*>(wsb + Px.q_off[l]);
          const int64_t nwt = sub[l].d_out * sub[l].d_in;
          st = from_hip(wfmt == DQT_INT4 ? dqt::launch_unpack_int4(sub[l].Wq, q8, nwt, s)
                                         : dqt::launch_unpack_int3(sub[l].Wq, q8, nwt, s));
          if (st != DQT_OK) break;
          a.Wq = q8;
        }
        a.dX = sub[l].dX;
        a.M = M;
        a.d_in = sub[l].d_in;
        a.d_out = sub[l].d_out;
        a.alpha = sub[l].alpha;
        a.w_ternary = wfmt == DQT_TERNARY2;
        a.dy_bf16 = false;
        a.dx_bf16 = dx_t == DQT_BF16;
        st = from_hip(dqt::launch_dx_f32(a, s));
      }
    }
    if (st != DQT_OK) return st;
  }
  // dW for the linears that want it
  int nw = 0;
  dqt::BwdPlan Pw = P;
  for (int l = 0; l < n; ++l)
    if (io[l].dW != nullptr) {
      Pw.xt_off[nw] = P.xt_off[l];
      Pw.part_off[nw] = P.part_off[l];
      sub[nw++] = L[l];
    }
  if (nw > 0) {
    if (xt_t == DQT_BF16) {
      dqt::BatchCfg c{nw, M, wfmt == DQT_TERNARY2, act_q == DQT_FP8E4M3, false};
      c.w_int4 = wfmt == DQT_INT4;
      c.w_int3 = wfmt == DQT_INT3;
      st = from_hip(dqt::launch_dw_batch(c, sub, wsb, Pw, s));
    } else {
      for (int l = 0; l < nw && st == DQT_OK; ++l) {
        dqt::DwArgs a;
        a.dY = sub[l].dY;
        a.Xq = sub[l].Xq;
        a.xdq = sub[l].xdq;
        a.dW = sub[l].dW;
        a.ws = reinterpret_cast<float*>(wsb + Pw.part_off[l]);
        a.M = M;
        a.d_in = sub[l].d_in;
        a.d_out = sub[l].d_out;
        a.splits = 0;
        a.act_e4m3 = act_q == DQT_FP8E4M3;
        a.xt_bf16 = false;
        st = from_hip(dqt::launch_dw_f32(a, s));
      }
    }
  }
  return st;
}

dqt_status dqt_linear_bwd_sr_batch(int32_t n, const dqt_linear_io* io, int64_t M, int32_t act_q,
                                   int32_t dy_t, int32_t xt_t, int32_t dx_t, float lr,
                                   uint64_t seed, uint32_t step, unsigned long long* counters,
                                   void* ws, size_t ws_bytes, void* stream) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  dqt_status st = check_batch(n, io, L, &wfmt);
  if (st != DQT_OK) return st;
  if (M < 0) return DQT_ERR_SHAPE;
  if (act_q != DQT_I8 && act_q != DQT_FP8E4M3) return DQT_ERR_DTYPE;
  if (!is_float_type(dy_t) || !is_float_type(xt_t) || !is_float_type(dx_t)) return DQT_ERR_DTYPE;
  if (dy_t != DQT_BF16 || xt_t != DQT_BF16) return DQT_ERR_UNSUPPORTED;
  if (counters != nullptr && (reinterpret_cast<uintptr_t>(counters) & 7u) != 0) return DQT_ERR_ALIGN;
  if (!(isfinite(lr) && lr >= 0.0f)) return DQT_ERR_RANGE;
  dqt::SRTensor t[DQT_MAX_BATCH];
  int nx = 0;
  for (int l = 0; l < n; ++l) {
    if (io[l].dW != nullptr) return DQT_ERR_UNSUPPORTED;
    if (io[l].Wq == nullptr) return DQT_ERR_NULL;
    if (!aligned16(io[l].Wq)) return DQT_ERR_ALIGN;
    if (M > 0) {
      if (io[l].Xq == nullptr || io[l].xdq == nullptr || io[l].dY == nullptr) return DQT_ERR_NULL;
      if (!aligned16(io[l].Xq) || !aligned16(io[l].xdq) || !aligned16(io[l].dY)) return DQT_ERR_ALIGN;
    }
    if (io[l].dX != nullptr) {
      if (!aligned16(io[l].dX)) return DQT_ERR_ALIGN;
      ++nx;
    }
    const float c = lr / io[l].w->alpha;   // one correctly rounded fp32 division
    if (!isfinite(c)) return DQT_ERR_RANGE;
    t[l].wq = static_cast<uint8_t*>(io[l].Wq);
    t[l].grad = nullptr;
    t[l].nweights = (int64_t)io[l].w->d_out * (int64_t)io[l].w->d_in;
    t[l].c = c;
    t[l].qmin = io[l].w->qmin;
    t[l].qmax = io[l].w->qmax;
    t[l].tensor_id = io[l].w->tensor_id;
  }
  const dqt::BwdPlan P = dqt::plan_bwd_batch(n, L, M);
  if (ws == nullptr || ws_bytes < P.total) return DQT_ERR_WORKSPACE;
  if (!aligned16(ws)) return DQT_ERR_ALIGN;
  if (M == 0) return DQT_OK;
  hipStream_t s = static_cast<hipStream_t>(stream);
  uint8_t* wsb = static_cast<uint8_t*>(ws);
  dqt::BatchCfg c{n, M, wfmt == DQT_TERNARY2, act_q == DQT_FP8E4M3, dx_t == DQT_BF16};
  c.w_int4 = wfmt == DQT_INT4;
  c.w_int3 = wfmt == DQT_INT3;
  if (nx > 0 && nx < n) {
    // dX of the linears that want it first (it reads the codes before the
    // update), then dW and the update of every linear
    dqt::LinearIO sub[DQT_MAX_BATCH];
    dqt::BwdPlan Px = P;
    int k = 0;
    for (int l = 0; l < n; ++l)
      if (io[l].dX != nullptr) {
        Px.q_off[k] = P.q_off[l];
        sub[k++] = L[l];
      }
    dqt::BatchCfg cx{nx, M, c.w_ternary, c.act_e4m3, c.out_bf16};
    cx.w_int4 = wfmt == DQT_INT4;
    cx.w_int3 = wfmt == DQT_INT3;
    st = from_hip(dqt::launch_dx_batch(cx, sub, wsb, Px, s));
    if (st != DQT_OK) return st;
  }
  return from_hip(dqt::launch_bwd_sr_batch(c, L, t, seed, step, counters, nx == n, wsb, P, s));
}

size_t dqt_update_variant_workspace(int32_t n) {
  if (n < 0 || n > DQT_MAX_BATCH) return 0;
  return dqt::update_variant_workspace(n);
}

dqt_status dqt_update_variant_batch(int32_t n, const dqt_linear_io* io, float lr, uint64_t seed,
                                    uint32_t step, int32_t mode, float frac,
                                    unsigned long long* counters, void* ws, size_t ws_bytes,
                                    void* stream) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  dqt_status st = check_batch(n, io, L, &wfmt);
  if (st != DQT_OK) return st;
  if (mode < DQT_UPD_SR || mode > DQT_UPD_FORCE_CHANGE) return DQT_ERR_RANGE;
  if (counters != nullptr && (reinterpret_cast<uintptr_t>(counters) & 7u) != 0) return DQT_ERR_ALIGN;
  if (!(isfinite(lr) && lr >= 0.0f)) return DQT_ERR_RANGE;
  const bool force = mode == DQT_UPD_FORCE_REMAIN || mode == DQT_UPD_FORCE_CHANGE;
  if (force && !(frac >= 0.0f && frac <= 1.0f)) return DQT_ERR_RANGE;
  dqt::SRTensor t[DQT_MAX_BATCH];
  for (int l = 0; l < n; ++l) {
    if (io[l].Wq == nullptr || io[l].dW == nullptr) return DQT_ERR_NULL;
    if (!aligned16(io[l].Wq) || !aligned16(io[l].dW)) return DQT_ERR_ALIGN;
    const float c = lr / io[l].w->alpha;
    if (!isfinite(c)) return DQT_ERR_RANGE;
    t[l].wq = static_cast<uint8_t*>(io[l].Wq);
    t[l].grad = io[l].dW;
    t[l].nweights = (int64_t)io[l].w->d_out * (int64_t)io[l].w->d_in;
    if (force && t[l].nweights >= (int64_t(1) << 32)) return DQT_ERR_SHAPE;
    t[l].c = c;
    t[l].qmin = io[l].w->qmin;
    t[l].qmax = io[l].w->qmax;
    t[l].tensor_id = io[l].w->tensor_id;
  }
  if (force) {
    if (ws == nullptr || ws_bytes < dqt::update_variant_workspace(n)) return DQT_ERR_WORKSPACE;
    if (!aligned16(ws)) return DQT_ERR_ALIGN;
  }
  return from_hip(dqt::launch_update_variant(code_format(wfmt), n, t, mode, frac, seed, step,
                                             counters, ws, static_cast<hipStream_t>(stream)));
}

size_t dqt_absmax_requant_workspace(int32_t n) {
  if (n < 1 || n > DQT_MAX_BATCH) return 0;
  return dqt::absmax_requant_workspace(n);
}

dqt_status dqt_absmax_requant_batch(int32_t n, const dqt_linear_io* io, float lr, float* alpha_out,
                                    unsigned long long* counters, void* ws, size_t ws_bytes,
                                    void* stream) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  dqt_status st = check_batch(n, io, L, &wfmt);
  if (st != DQT_OK) return st;
  if (alpha_out == nullptr) return DQT_ERR_NULL;
  if ((reinterpret_cast<uintptr_t>(alpha_out) & 3u) != 0) return DQT_ERR_ALIGN;
  if (counters != nullptr && (reinterpret_cast<uintptr_t>(counters) & 7u) != 0) return DQT_ERR_ALIGN;
  if (!(isfinite(lr) && lr >= 0.0f)) return DQT_ERR_RANGE;
  if (ws == nullptr || ws_bytes < dqt::absmax_requant_workspace(n)) return DQT_ERR_WORKSPACE;
  if ((reinterpret_cast<uintptr_t>(ws) & 3u) != 0) return DQT_ERR_ALIGN;
  dqt::SRTensor t[DQT_MAX_BATCH];
  for (int l = 0; l < n; ++l) {
    if (io[l].Wq == nullptr || io[l].dW == nullptr) return DQT_ERR_NULL;
    if (!aligned16(io[l].Wq) || !aligned16(io[l].dW)) return DQT_ERR_ALIGN;
    t[l].wq = static_cast<uint8_t*>(io[l].Wq);
    t[l].grad = io[l].dW;
    t[l].nweights = (int64_t)io[l].w->d_out * (int64_t)io[l].w->d_in;
    t[l].c = 0.0f;
    t[l].qmin = io[l].w->qmin;
    t[l].qmax = io[l].w->qmax;
    t[l].tensor_id = io[l].w->tensor_id;
    t[l].alpha = io[l].w->alpha;
  }
  return from_hip(dqt::launch_absmax_requant(code_format(wfmt), n, t, lr, alpha_out, counters, ws,
                                             static_cast<hipStream_t>(stream)));
}

dqt_status dqt_adamw_sr_update_batch(int32_t n, const dqt_linear_io* io, float* const* m,
                                     float* const* v, const dqt_adamw* hp, uint64_t seed,
                                     uint32_t step, unsigned long long* counters, void* stream) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  dqt_status st = check_batch(n, io, L, &wfmt);
  if (st != DQT_OK) return st;
  if (hp == nullptr || (n > 0 && (m == nullptr || v == nullptr))) return DQT_ERR_NULL;
  if (counters != nullptr && (reinterpret_cast<uintptr_t>(counters) & 7u) != 0) return DQT_ERR_ALIGN;
  if (!(isfinite(hp->lr) && hp->lr >= 0.0f)) return DQT_ERR_RANGE;
  if (!(hp->beta1 >= 0.0f && hp->beta1 < 1.0f && hp->beta2 >= 0.0f && hp->beta2 < 1.0f))
    return DQT_ERR_RANGE;
  if (!(isfinite(hp->eps) && hp->eps > 0.0f)) return DQT_ERR_RANGE;
  if (!(isfinite(hp->weight_decay) && hp->weight_decay >= 0.0f)) return DQT_ERR_RANGE;
  if (step == 0) return DQT_ERR_RANGE;
  dqt::AdamTensor t[DQT_MAX_BATCH];
  for (int l = 0; l < n; ++l) {
    if (io[l].Wq == nullptr || io[l].dW == nullptr || m[l] == nullptr || v[l] == nullptr)
      return DQT_ERR_NULL;
    if (!aligned16(io[l].Wq) || !aligned16(io[l].dW) || !aligned16(m[l]) || !aligned16(v[l]))
      return DQT_ERR_ALIGN;
    // the bias-corrected step in grid units must be finite
    double b1t = 1.0, x = (double)hp->beta1;
    for (uint32_t e = step; e > 0; e >>= 1) {
      if (e & 1u) b1t *= x;
      x *= x;
    }
    const double cu = (double)hp->lr / ((double)io[l].w->alpha * (1.0 - b1t));
    if (!isfinite((float)cu)) return DQT_ERR_RANGE;
    t[l].wq = static_cast<uint8_t*>(io[l].Wq);
    t[l].grad = io[l].dW;
    t[l].m = m[l];
    t[l].v = v[l];
    t[l].nweights = (int64_t)io[l].w->d_out * (int64_t)io[l].w->d_in;
    t[l].alpha = io[l].w->alpha;
    t[l].qmin = io[l].w->qmin;
    t[l].qmax = io[l].w->qmax;
    t[l].tensor_id = io[l].w->tensor_id;
  }
  const dqt::AdamHyper h{hp->lr, hp->beta1, hp->beta2, hp->eps, hp->weight_decay};
  return from_hip(dqt::launch_adamw_sr(code_format(wfmt), n, t, h, seed, step, counters,
                                       static_cast<hipStream_t>(stream)));
}

dqt_status dqt_adamw_sr_update(const dqt_weight* w, void* Wq, const float* dW, float* m, float* v,
                               const dqt_adamw* hp, uint64_t seed, uint32_t step,
                               unsigned long long* counters, void* stream) {
  dqt_linear_io io{};
  io.w = w;
  io.Wq = Wq;
  io.dW = const_cast<float*>(dW);
  return dqt_adamw_sr_update_batch(1, &io, &m, &v, hp, seed, step, counters, stream);
}

dqt_status dqt_sr_update_batch(int32_t n, const dqt_linear_io* io, float lr, uint64_t seed,
                               uint32_t step, unsigned long long* counters, void* stream) {
  dqt::LinearIO L[DQT_MAX_BATCH];
  int32_t wfmt;
  dqt_status st = check_batch(n, io, L, &wfmt);
  if (st != DQT_OK) return st;
  if (counters != nullptr && (reinterpret_cast<uintptr_t>(counters) & 7u) != 0) return DQT_ERR_ALIGN;
  if (!(isfinite(lr) && lr >= 0.0f)) return DQT_ERR_RANGE;
  dqt::SRTensor t[DQT_MAX_BATCH];
  for (int l = 0; l < n; ++l) {
    if (io[l].Wq == nullptr || io[l].dW == nullptr) return DQT_ERR_NULL;
    if (!aligned16(io[l].Wq) || !aligned16(io[l].dW)) return DQT_ERR_ALIGN;
    const float c = lr / io[l].w->alpha;   // one correctly rounded fp32 division
    if (!isfinite(c)) return DQT_ERR_RANGE;
    t[l].wq = static_cast<uint8_t*>(io[l].Wq);
    t[l].grad = io[l].dW;
    t[l].nweights = (int64_t)io[l].w->d_out * (int64_t)io[l].w->d_in;
    t[l].c = c;
    t[l].qmin = io[l].w->qmin;
    t[l].qmax = io[l].w->qmax;
    t[l].tensor_id = io[l].w->tensor_id;
  }
  return from_hip(dqt::launch_sr_update(code_format(wfmt), n, t, seed, step, counters,
                                        static_cast<hipStream_t>(stream)));
}

// ---------------------------------------------------------- update tables

namespace {

// Checks of one update-table batch (any n, one code format).  Returns the
// launch's tile count in *tiles; writes the table entries when `out` is
// given.
dqt_status check_table(int32_t n, const dqt_linear_io* io, float lr, int32_t* wfmt, int64_t* tiles,
                       dqt::SRTableEntry* out) {
  if (n < 1) return DQT_ERR_SHAPE;
  if (io == nullptr) return DQT_ERR_NULL;
  if (!(isfinite(lr) && lr >= 0.0f)) return DQT_ERR_RANGE;
  *tiles = 0;
  for (int l = 0; l < n; ++l) {
    const dqt_status st = check_weight(io[l].w);
    if (st != DQT_OK) return st;
    if (l == 0) *wfmt = io[l].w->wfmt;
    else if (io[l].w->wfmt != *wfmt) return DQT_ERR_UNSUPPORTED;
    if (io[l].Wq == nullptr || io[l].dW == nullptr) return DQT_ERR_NULL;
    if (!aligned16(io[l].Wq) || !aligned16(io[l].dW)) return DQT_ERR_ALIGN;
    if (!isfinite(lr / io[l].w->alpha)) return DQT_ERR_RANGE;   // the step in grid units
    dqt::SRTensor t;
    t.wq = static_cast<uint8_t*>(io[l].Wq);
    t.grad = io[l].dW;
    t.nweights = (int64_t)io[l].w->d_out * (int64_t)io[l].w->d_in;
    t.c = 0.0f;
    t.qmin = io[l].w->qmin;
    t.qmax = io[l].w->qmax;
    t.tensor_id = io[l].w->tensor_id;
    t.alpha = io[l].w->alpha;
    if (out != nullptr) dqt::sr_table_entry(t, *tiles, &out[l]);
    *tiles += dqt::sr_tiles(t.nweights);
  }
  return DQT_OK;
}

}  // namespace

size_t dqt_sr_table_bytes(int32_t n) {
  return n < 1 ? 0 : (size_t)n * sizeof(dqt::SRTableEntry);
}

dqt_status dqt_sr_table_build(int32_t n, const dqt_linear_io* io, void* table, size_t table_bytes) {
  if (n < 1) return DQT_ERR_SHAPE;
  if (table == nullptr) return DQT_ERR_NULL;
  if (table_bytes < dqt_sr_table_bytes(n)) return DQT_ERR_WORKSPACE;
  int32_t wfmt;
  int64_t tiles;
  return check_table(n, io, 0.0f, &wfmt, &tiles, static_cast<dqt::SRTableEntry*>(table));
}

dqt_status dqt_sr_update_table(int32_t n, const dqt_linear_io* io, const void* table, float lr,
                               uint64_t seed, uint32_t step, unsigned long long* counters,
                               unsigned long long* per_tensor, void* stream) {
  int32_t wfmt;
  int64_t tiles;
  const dqt_status st = check_table(n, io, lr, &wfmt, &tiles, nullptr);
  if (st != DQT_OK) return st;
  if (table == nullptr) return DQT_ERR_NULL;
  if (!aligned16(table)) return DQT_ERR_ALIGN;
  if (counters != nullptr && (reinterpret_cast<uintptr_t>(counters) & 7u) != 0) return DQT_ERR_ALIGN;
  if (per_tensor != nullptr && (reinterpret_cast<uintptr_t>(per_tensor) & 7u) != 0) return DQT_ERR_ALIGN;
  return from_hip(dqt::launch_sr_update_table(code_format(wfmt), n, tiles,
                                              static_cast<const dqt::SRTableEntry*>(table), lr, seed,
                                              step, counters, per_tensor,
                                              static_cast<hipStream_t>(stream)));
}

// ---------------------------------------------------------- single linears

size_t dqt_linear_fwd_workspace(const dqt_weight* w) {
  dqt_linear_io io{};
  io.w = w;
  return dqt_linear_fwd_batch_workspace(1, &io);
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
  if (act_q == DQT_FP8E4M3 && w->wfmt == DQT_I8) return DQT_ERR_UNSUPPORTED;
  if (M == 0) return DQT_OK;
  if (Wq == nullptr || Xq == nullptr || xdq == nullptr || Y == nullptr) return DQT_ERR_NULL;
  if (!aligned16(Wq) || !aligned16(Xq) || !aligned16(xdq) || !aligned16(Y) ||
      (X != nullptr && !aligned16(X)))
    return DQT_ERR_ALIGN;
  dqt_linear_io io{};
  io.w = w;
  io.Wq = const_cast<void*>(Wq);
  io.Xq = Xq;
  io.xdq = xdq;
  io.Y = Y;
  // refused before the quantisation is launched
  const size_t need = fwd_batch_workspace_least(1, &io);
  if (need > 0 && (ws == nullptr || ws_bytes < need)) return DQT_ERR_WORKSPACE;
  if (need > 0 && !aligned16(ws)) return DQT_ERR_ALIGN;
  if (X != nullptr) {
    st = from_hip(dqt::launch_act_quant(X, x_t == DQT_BF16, M, w->d_in, act_q == DQT_FP8E4M3, Xq,
                                        xdq, static_cast<hipStream_t>(stream)));
    if (st != DQT_OK) return st;
  }
  return dqt_linear_fwd_batch(1, &io, M, act_q, y_t, ws, ws_bytes, stream);
}

size_t dqt_linear_bwd_workspace(const dqt_weight* w, int64_t M) {
  dqt_linear_io io{};
  io.w = w;
  return dqt_linear_bwd_batch_workspace(1, &io, M);
}

dqt_status dqt_linear_bwd(const dqt_weight* w, const void* Wq, const void* Xq, int32_t act_q,
                          const float* xdq, const void* dY, int32_t dy_t, int64_t M,
                          int32_t xt_t, void* dX, int32_t dx_t, float* dW, void* ws,
                          size_t ws_bytes, void* stream) {
  dqt_linear_io io{};
  io.w = w;
  io.Wq = const_cast<void*>(Wq);
  io.Xq = Xq;
  io.xdq = xdq;
  io.dY = dY;
  io.dX = dX;
  io.dW = dW;
  if (dX == nullptr && !is_float_type(dx_t)) dx_t = DQT_F32;   // unused
  return dqt_linear_bwd_batch(1, &io, M, act_q, dy_t, xt_t, dx_t, ws, ws_bytes, stream);
}

dqt_status dqt_sr_update(const dqt_weight* w, void* Wq, const float* dW, float lr, uint64_t seed,
                         uint32_t step, unsigned long long* counters, void* stream) {
  dqt_linear_io io{};
  io.w = w;
  io.Wq = Wq;
  io.dW = const_cast<float*>(dW);
  return dqt_sr_update_batch(1, &io, lr, seed, step, counters, stream);
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

dqt_status dqt_pack_int4(const int8_t* q, int64_t rows, int64_t cols, uint8_t* packed) {
  if (q == nullptr || packed == nullptr) return DQT_ERR_NULL;
  if (rows < 0 || cols < 0 || (cols % 2) != 0) return DQT_ERR_SHAPE;
  const int64_t pc = cols / 2;
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t b = 0; b < pc; ++b) {
      const int lo = q[r * cols + 2 * b], hi = q[r * cols + 2 * b + 1];
      if (lo < -8 || lo > 7 || hi < -8 || hi > 7) return DQT_ERR_RANGE;
      packed[r * pc + b] = (uint8_t)(((uint32_t)lo & 0xFu) | (((uint32_t)hi & 0xFu) << 4));
    }
  return DQT_OK;
}

dqt_status dqt_unpack_int4(const uint8_t* packed, int64_t rows, int64_t cols, int8_t* q) {
  if (q == nullptr || packed == nullptr) return DQT_ERR_NULL;
  if (rows < 0 || cols < 0 || (cols % 2) != 0) return DQT_ERR_SHAPE;
  const int64_t pc = cols / 2;
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t b = 0; b < pc; ++b)
      for (int j = 0; j < 2; ++j) {
        const int v = (packed[r * pc + b] >> (4 * j)) & 0xF;
        q[r * cols + 2 * b + j] = (int8_t)(v >= 8 ? v - 16 : v);
      }
  return DQT_OK;
}

dqt_status dqt_pack_int3(const int8_t* q, int64_t rows, int64_t cols, uint8_t* packed) {
  if (q == nullptr || packed == nullptr) return DQT_ERR_NULL;
  if (rows < 0 || cols < 0 || (cols % 8) != 0) return DQT_ERR_SHAPE;
  const int64_t groups = cols / 8;
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t g = 0; g < groups; ++g) {
      uint32_t bits = 0;
      for (int j = 0; j < 8; ++j) {
        const int v = q[r * cols + 8 * g + j];
        if (v < -4 || v > 3) return DQT_ERR_RANGE;
        bits |= ((uint32_t)v & 7u) << (3 * j);
      }
      uint8_t* p = packed + r * (3 * groups) + 3 * g;
      p[0] = (uint8_t)bits;
      p[1] = (uint8_t)(bits >> 8);
      p[2] = (uint8_t)(bits >> 16);
    }
  return DQT_OK;
}

dqt_status dqt_unpack_int3(const uint8_t* packed, int64_t rows, int64_t cols, int8_t* q) {
  if (q == nullptr || packed == nullptr) return DQT_ERR_NULL;
  if (rows < 0 || cols < 0 || (cols % 8) != 0) return DQT_ERR_SHAPE;
  const int64_t groups = cols / 8;
  for (int64_t r = 0; r < rows; ++r)
    for (int64_t g = 0; g < groups; ++g) {
      const uint8_t* p = packed + r * (3 * groups) + 3 * g;
      const uint32_t bits = (uint32_t)p[0] | ((uint32_t)p[1] << 8) | ((uint32_t)p[2] << 16);
      for (int j = 0; j < 8; ++j) {
        const int v = (int)((bits >> (3 * j)) & 7u);
        q[r * cols + 8 * g + j] = (int8_t)(v >= 4 ? v - 8 : v);
      }
    }
  return DQT_OK;
}

}  // extern "C"
