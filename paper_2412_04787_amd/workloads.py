"""Synthetic workloads for the DQT linear train step: shapes and seeded draws.

This module only draws random numbers and describes shapes.  It holds none of
the method's arithmetic (no quantisation, no scale computation, no rounding),
so the HIP path and the CPU oracle can both take their inputs from it.

Every draw comes from numpy's PCG64 seeded with
``SeedSequence([seed, workload_id, stream])``, where ``stream`` names the
tensor being drawn; drawing one tensor never shifts another's values.

The paper trains LLaMA-structured models on Wikipedia / FineWeb (Sec. 4.1);
those corpora are not used here.  The draws below stand in for them with the
shapes of LLaMA-block linears and simple value distributions:
  * initial real-valued weights W0 ~ N(0, 0.02)   (std 0.02)
  * activations X ~ N(0, 1)
  * upstream gradients dY ~ N(0, 0.01)            (std 1e-2)
"""

from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass(frozen=True)
class Linear:
    name: str
    d_in: int
    d_out: int
    input: str          # linears with the same input name share one X


@dataclass(frozen=True)
class Workload:
    name: str
    wid: int
    M: int                      # tokens
    linears: tuple
    wfmt: str                   # "ternary" (2-bit), "i3" (3-bit), "i4" (4-bit) packed, or "i8"
    qmin: int
    qmax: int
    init: str                   # "uniform": q ~ U{-1,0,1}, scale from W0
                                # "absmean": Eq. 2-4 applied to W0
    act: str                    # activation code type: "i8" or "e4m3"
    x_dtype: str                # dtype X arrives in: "f32" or "bf16"
    dy_dtype: str               # dtype dY arrives in
    xt: str                     # environment dtype of X~ in the dW product
    y_out: str                  # forward output dtype
    dx_out: str                 # dX dtype
    lr: float
    x_std: float = 1.0
    dy_std: float = 1e-2
    w0_std: float = 0.02
    seed: int = 0
    sr_step: int = 1
    notes: str = field(default="", compare=False)

    @property
    def inputs(self):
        seen = []
        for lin in self.linears:
            if lin.input not in seen:
                seen.append(lin.input)
        return seen

    def input_width(self, name: str) -> int:
        for lin in self.linears:
            if lin.input == name:
                return lin.d_in
        raise KeyError(name)

    @property
    def n_weights(self) -> int:
        return sum(l.d_in * l.d_out for l in self.linears)

    @property
    def train_flops(self) -> int:
        """fwd + dX + dW: three dense contractions of 2*M*d_in*d_out each."""
        return sum(6 * self.M * l.d_in * l.d_out for l in self.linears)


def _llama_linears(h: int, ffn: int):
    return (
        Linear("q", h, h, "attn_in"),
        Linear("k", h, h, "attn_in"),
        Linear("v", h, h, "attn_in"),
        Linear("o", h, h, "attn_out"),
        Linear("gate", h, ffn, "mlp_in"),
        Linear("up", h, ffn, "mlp_in"),
        Linear("down", ffn, h, "mlp_hidden"),
    )


WORKLOADS = {
    # One 256x256 ternary linear, 512 tokens, fp32 environment.
    "single_256": Workload(
        name="single_256", wid=0, M=512,
        linears=(Linear("lin", 256, 256, "x"),),
        wfmt="ternary", qmin=-1, qmax=1, init="uniform", act="i8",
        x_dtype="f32", dy_dtype="f32", xt="f32", y_out="f32", dx_out="f32",
        lr=1e-3),
    # The seven linears of a LLaMA block at hidden 768 / FFN 2048,
    # 8 x 1024 = 8192 tokens, ternary weights, bf16 environment.
    "llama_h768": Workload(
        name="llama_h768", wid=1, M=8192, linears=_llama_linears(768, 2048),
        wfmt="ternary", qmin=-1, qmax=1, init="absmean", act="i8",
        x_dtype="bf16", dy_dtype="bf16", xt="bf16", y_out="bf16", dx_out="bf16",
        lr=3e-4),
    # Hidden 2048 / FFN 5632, 16384 tokens, 8-bit weights on -127..127.
    "llama_h2048": Workload(
        name="llama_h2048", wid=2, M=16384, linears=_llama_linears(2048, 5632),
        wfmt="i8", qmin=-127, qmax=127, init="absmean", act="i8",
        x_dtype="bf16", dy_dtype="bf16", xt="bf16", y_out="bf16", dx_out="bf16",
        lr=3e-4),
    # Hidden 4096 / FFN 11008, 8192 tokens, ternary weights, e4m3 activations.
    "llama_h4096": Workload(
        name="llama_h4096", wid=3, M=8192, linears=_llama_linears(4096, 11008),
        wfmt="ternary", qmin=-1, qmax=1, init="absmean", act="e4m3",
        x_dtype="bf16", dy_dtype="bf16", xt="bf16", y_out="bf16", dx_out="bf16",
        lr=1e-4),
    # The hidden-2048 block with 4-bit weights (the n = 4 grid of Eq. 3,
    # -8..7, packed two per byte).
    "llama_h2048_int4": Workload(
        name="llama_h2048_int4", wid=5, M=16384, linears=_llama_linears(2048, 5632),
        wfmt="i4", qmin=-8, qmax=7, init="absmean", act="i8",
        x_dtype="bf16", dy_dtype="bf16", xt="bf16", y_out="bf16", dx_out="bf16",
        lr=3e-4),
    # The hidden-2048 block with 3-bit weights (the n = 3 grid of Eq. 3,
    # -4..3, 8 weights in 3 bytes).
    "llama_h2048_int3": Workload(
        name="llama_h2048_int3", wid=6, M=16384, linears=_llama_linears(2048, 5632),
        wfmt="i3", qmin=-4, qmax=3, init="absmean", act="i8",
        x_dtype="bf16", dy_dtype="bf16", xt="bf16", y_out="bf16", dx_out="bf16",
        lr=3e-4),
}

# Stream ids: which tensor a draw belongs to.
_S_W0, _S_QDRAW, _S_X, _S_DY = 1, 2, 3, 4


def rng_for(seed: int, wid: int, *stream: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(np.random.SeedSequence([seed, wid, *stream])))


def draw_normal(shape, std: float, seed: int, wid: int, *stream: int) -> np.ndarray:
    """fp32 normal draws N(0, std) for one tensor."""
    g = rng_for(seed, wid, *stream)
    return (g.standard_normal(size=shape, dtype=np.float32) * np.float32(std)).astype(np.float32)


def draw_ternary(shape, seed: int, wid: int, *stream: int) -> np.ndarray:
    """int8 draws uniform on {-1, 0, 1}."""
    g = rng_for(seed, wid, *stream)
    return (g.integers(0, 3, size=shape, dtype=np.int64) - 1).astype(np.int8)


def draw_int(shape, lo: int, hi: int, seed: int, wid: int, *stream: int) -> np.ndarray:
    """int8 draws uniform on lo..hi inclusive."""
    g = rng_for(seed, wid, *stream)
    return g.integers(lo, hi + 1, size=shape, dtype=np.int64).astype(np.int8)


def weight_draws(wl: Workload, li: int):
    """Raw draws for linear li: W0 [d_out, d_in] fp32, and (init == 'uniform'
    only) a uniform ternary draw q [d_out, d_in]."""
    lin = wl.linears[li]
    W0 = draw_normal((lin.d_out, lin.d_in), wl.w0_std, wl.seed, wl.wid, _S_W0, li)
    q = None
    if wl.init == "uniform":
        q = draw_ternary((lin.d_out, lin.d_in), wl.seed, wl.wid, _S_QDRAW, li)
    return W0, q


def input_draw(wl: Workload, input_name: str, M: int | None = None) -> np.ndarray:
    """X [M, d_in] fp32 draws for one distinct layer input."""
    M = wl.M if M is None else M
    ii = wl.inputs.index(input_name)
    return draw_normal((M, wl.input_width(input_name)), wl.x_std, wl.seed, wl.wid, _S_X, ii)


def grad_draw(wl: Workload, li: int, M: int | None = None) -> np.ndarray:
    """dY [M, d_out] fp32 draws for linear li."""
    M = wl.M if M is None else M
    lin = wl.linears[li]
    return draw_normal((M, lin.d_out), wl.dy_std, wl.seed, wl.wid, _S_DY, li)
