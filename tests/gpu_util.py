"""Helpers for the GPU parity tests: moving seeded numpy inputs to the device
and running the library's entry points on them.  Inputs go to both sides
unchanged; the oracle sees exactly the values the GPU sees."""
from __future__ import annotations

import sys

import numpy as np
import torch

from oracle import dqt_oracle as O
from paper_2412_04787_amd import dqt

DEV = "cuda:0"


def log(msg: str):
    print(msg, flush=True)
    sys.stdout.flush()


def to_dev(x: np.ndarray, dtype: str):
    """fp32 numpy -> device tensor in dtype ('f32' or 'bf16'), plus the fp32
    numpy values the device tensor holds."""
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    if dtype == "bf16":
        t = t.to(torch.bfloat16)
    t = t.to(DEV)
    return t, t.float().cpu().numpy()


def act_code(kind: str) -> int:
    return dqt.DQT_I8 if kind == "i8" else dqt.DQT_FP8E4M3


def float_code(kind: str) -> int:
    return dqt.DQT_BF16 if kind == "bf16" else dqt.DQT_F32


def torch_float(kind: str):
    return torch.bfloat16 if kind == "bf16" else torch.float32


def weight_codes_dev(q: np.ndarray, wfmt: str):
    """int8 codes -> device buffer in the library's weight layout."""
    if wfmt == "ternary":
        packed = O.pack_ternary(q)
        return torch.from_numpy(packed).to(DEV)
    if wfmt == "i4":
        return torch.from_numpy(O.pack_int4(q)).to(DEV)
    if wfmt == "i3":
        return torch.from_numpy(O.pack_int3(q)).to(DEV)
    return torch.from_numpy(np.ascontiguousarray(q, dtype=np.int8)).to(DEV)


def weight_codes_host(buf, wfmt: str, d_in: int) -> np.ndarray:
    a = buf.cpu().numpy()
    if wfmt == "ternary":
        return O.unpack_ternary(a, d_in)
    if wfmt == "i4":
        return O.unpack_int4(a.reshape(-1, d_in // 2), d_in)
    if wfmt == "i3":
        return O.unpack_int3(a.reshape(-1, 3 * d_in // 8), d_in)
    return a.astype(np.int8)


def make_weight(d_out, d_in, wfmt, qmin, qmax, alpha, tensor_id=0):
    code = {"ternary": dqt.DQT_TERNARY2, "i4": dqt.DQT_INT4, "i3": dqt.DQT_INT3}.get(wfmt, dqt.DQT_I8)
    return dqt.weight(d_out, d_in, code, qmin, qmax, float(alpha), tensor_id)


def run_fwd(w, Wq, X_dev, act: str, y_out: str):
    M, K = X_dev.shape
    Xq = torch.empty((M, K), dtype=torch.int8 if act == "i8" else torch.uint8, device=DEV)
    xdq = torch.empty((max(M, 1),), dtype=torch.float32, device=DEV)
    Y = torch.empty((M, w.d_out), dtype=torch_float(y_out), device=DEV)
    ws = dqt.workspace(dqt.dqt_linear_fwd_workspace(w))
    dqt.dqt_linear_fwd(w, Wq, X_dev, M, act_code(act), Xq, xdq, Y, ws)
    return Xq, xdq, Y


def run_bwd(w, Wq, Xq, act: str, xdq, dY_dev, xt: str, dx_out: str | None = "f32",
            want_dw: bool = True):
    M = dY_dev.shape[0]
    dX = None if dx_out is None else torch.empty((M, w.d_in), dtype=torch_float(dx_out), device=DEV)
    dW = torch.empty((w.d_out, w.d_in), dtype=torch.float32, device=DEV) if want_dw else None
    ws = dqt.workspace(dqt.dqt_linear_bwd_workspace(w, M))
    dqt.dqt_linear_bwd(w, Wq, Xq, act_code(act), xdq, dY_dev, M, float_code(xt), dX, dW, ws)
    return dX, dW


def gemm_close(got, ref64, absbound, rel=1e-3, bf16_out=False):
    """Componentwise |got - ref| <= rel * sum|terms| (+ 1 bf16 ulp of ref when
    the output is bf16) and normwise ||got - ref|| <= rel * ||ref||."""
    got = np.asarray(got, dtype=np.float64)
    ref = np.asarray(ref64, dtype=np.float64)
    tol = rel * np.asarray(absbound, dtype=np.float64)
    if bf16_out:
        tol = tol + np.abs(ref) * 2.0 ** -8
    err = np.abs(got - ref)
    bad = err > tol + 1e-30
    nrm = np.linalg.norm(got - ref) <= rel * np.linalg.norm(ref) + 1e-30 + (
        np.linalg.norm(ref) * 2.0 ** -8 if bf16_out else 0.0)
    return (not bad.any()) and bool(nrm), int(bad.sum()), float(err.max(initial=0.0))
