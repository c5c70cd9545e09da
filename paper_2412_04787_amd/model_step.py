"""Train step of a LLaMA-shaped model whose block linears are DQT layers.

Sec. 4.1 trains LLaMA-structured models (RMSNorm, rotary position
embeddings, SwiGLU feed-forward) in which every weight matrix of the blocks
is a DQT layer: low-bit codes with a fixed per-tensor scale, 8-bit
activations in the forward (Sec. 3.2), and the stochastic-rounding update of
Eq. 5 applied to the codes directly, with no high-precision copy.  This
module runs that step on one GPU.

What runs where:
  * The seven linears of each block (q, k, v, o, gate, up, down) run in this
    library's kernels through its C ABI.  Linears that share an input form
    one group: its input is quantised once (the block norms and the
    quantisation are one fused launch, dqt_rmsnorm_act_quant), its forward is
    one batched call, and its backward is one call (dqt_linear_bwd_sr_batch)
    that forms dX and applies Eq. 5 to the codes in the dW product's
    epilogue, so dW never reaches memory.  A layer's codes are not read again
    in the step once its backward has run, so updating them there is the
    step's update.
  * The rest is the environment the linears are trained in, in PyTorch:
    token embedding and LM head (dense bf16 compute, fp32 master weights
    trained by AdamW, as BitNet-style models keep them), causal attention
    (PyTorch's flash kernels), the rotary embedding, SiLU, the residual adds,
    the backward of the norms and the loss.

Initialisation (untimed): codes by Eq. 2-4 for the ternary grid from
W0 ~ N(0, 0.02) (alpha = mean |W0|, q = Clip(Round(W0 / alpha), -1, 1));
embedding and head N(0, 0.02); norm weights 1.
"""

from __future__ import annotations

import math
from dataclasses import dataclass

from . import dqt


@dataclass(frozen=True)
class ModelConfig:
    name: str
    layers: int
    hidden: int
    heads: int
    ffn: int
    vocab: int
    batch: int
    seq: int
    lr: float
    eps: float = 1e-6
    rope_base: float = 10000.0
    seed: int = 0

    @property
    def tokens(self) -> int:
        return self.batch * self.seq

    def linears(self):
        """(group name, [(linear name, d_in, d_out)]) of one block; linears in
        one group share their input."""
        h, f = self.hidden, self.ffn
        return [("attn_in", [("q", h, h), ("k", h, h), ("v", h, h)]),
                ("attn_out", [("o", h, h)]),
                ("mlp_in", [("gate", h, f), ("up", h, f)]),
                ("mlp_hidden", [("down", f, h)])]

    @property
    def dqt_weights(self) -> int:
        return self.layers * sum(di * do for _, g in self.linears() for _, di, do in g)

    def step_flops(self) -> dict:
        """Algorithmic flops of one train step (forward + backward)."""
        T = self.tokens
        lin = 6 * T * self.dqt_weights
        head = 6 * T * self.vocab * self.hidden
        # causal attention: Q K^T and P V over the lower triangle, backward twice the forward
        attn = 3 * 2 * self.batch * self.seq * self.seq * self.hidden * self.layers
        return {"dqt_linears": lin, "lm_head": head, "attention": attn,
                "total": lin + head + attn}


MODELS = {
    # 24 layers, hidden 2048, 16 heads, FFN 5632, vocab 32000; 8 x 2048 tokens
    "llama24_h2048": ModelConfig(name="llama24_h2048", layers=24, hidden=2048, heads=16,
                                 ffn=5632, vocab=32000, batch=8, seq=2048, lr=3e-4),
    # a small model of the same structure, for tests
    "tiny": ModelConfig(name="tiny", layers=2, hidden=256, heads=4, ffn=512, vocab=1000,
                        batch=2, seq=128, lr=3e-4),
}


# blocks of the norm backward (each one sums the gamma gradient of its rows)
MS_NORM_BLOCKS = 1024


def _pack_ternary_dev(q):
    """int8 codes {-1, 0, 1} [d_out, d_in] -> packed bytes [d_out, d_in / 4]:
    code q + 1 of weight k at bits 2 (k mod 4) of byte k / 4."""
    torch = dqt._torch()
    c = (q + 1).to(torch.uint8).view(q.shape[0], -1, 4)
    return (c[..., 0] | (c[..., 1] << 2) | (c[..., 2] << 4) | (c[..., 3] << 6)).contiguous()


class _Group:
    """The DQT linears of one block that share an input."""

    def __init__(self, model, layer: int, gname: str, lins):
        torch = dqt._torch()
        self.model = model
        self.layer = layer
        self.gname = gname
        self.d_in = lins[0][1]
        self.d_outs = [do for _, _, do in lins]
        self.weights, self.codes = [], []
        dev = model.dev
        for name, d_in, d_out in lins:
            tid = model.next_tensor_id()
            g = torch.Generator(device=dev)
            g.manual_seed(model.cfg.seed * 1_000_003 + tid)
            W0 = torch.randn((d_out, d_in), generator=g, device=dev, dtype=torch.float32) * 0.02
            alpha = float(W0.double().abs().mean())          # Eq. 2: AbsMean of W0
            q = torch.clamp(torch.round(W0 / alpha), -1, 1).to(torch.int8)   # Eq. 3-4, Q_p = 1
            del W0
            self.codes.append(_pack_ternary_dev(q))
            self.weights.append(dqt.weight(d_out, d_in, dqt.DQT_TERNARY2, -1, 1, alpha, tid))


class _DQTGroupFn:
    """Autograd function of one group: x (or RMSNorm(x) * gamma) is quantised
    to int8 per token and fed to the group's linears; the backward returns
    dX (the quantiser passes the gradient through, and the norm's backward is
    taken here) and updates the codes by Eq. 5."""

    _cls = None

    @classmethod
    def get(cls):
        if cls._cls is not None:
            return cls._cls
        torch = dqt._torch()

        class Fn(torch.autograd.Function):
            @staticmethod
            def forward(ctx, x, gamma, grp):
                m = grp.model
                T = x.shape[0]
                Xq = torch.empty(x.shape, dtype=torch.int8, device=x.device)
                xdq = torch.empty((T,), dtype=torch.float32, device=x.device)
                rinv = None
                if gamma is None:
                    dqt.dqt_act_quant(x, dqt.DQT_I8, Xq, xdq)
                else:
                    rinv = torch.empty((T,), dtype=torch.float32, device=x.device)
                    dqt.dqt_rmsnorm_act_quant(x, gamma, m.cfg.eps, dqt.DQT_I8, Xq, xdq, rinv)
                Ys = [torch.empty((T, d_out), dtype=torch.bfloat16, device=x.device)
                      for d_out in grp.d_outs]
                io = dqt.linear_io([dict(w=w, Wq=c, Xq=Xq, xdq=xdq, Y=Y)
                                    for w, c, Y in zip(grp.weights, grp.codes, Ys)])
                dqt.dqt_linear_fwd_batch(io, T, dqt.DQT_I8, dqt.DQT_BF16,
                                         m.workspace(dqt.dqt_linear_fwd_batch_workspace(io)))
                ctx.grp = grp
                ctx.has_gamma = gamma is not None
                if gamma is None:
                    ctx.save_for_backward(Xq, xdq)
                else:
                    ctx.save_for_backward(Xq, xdq, x, gamma, rinv)
                return tuple(Ys)

            @staticmethod
            def backward(ctx, *dYs):
                grp = ctx.grp
                m = grp.model
                saved = ctx.saved_tensors
                Xq, xdq = saved[0], saved[1]
                T = Xq.shape[0]
                dXs = [torch.empty((T, grp.d_in), dtype=torch.bfloat16, device=Xq.device)
                       for _ in grp.d_outs]
                ents = []
                for w, c, dY, dX, d_out in zip(grp.weights, grp.codes, dYs, dXs, grp.d_outs):
                    if dY is None:
                        dY = torch.zeros((T, d_out), dtype=torch.bfloat16, device=Xq.device)
                    ents.append(dict(w=w, Wq=c, Xq=Xq, xdq=xdq, dY=dY.contiguous(), dX=dX))
                io = dqt.linear_io(ents)
                dqt.dqt_linear_bwd_sr_batch(io, T, dqt.DQT_I8, dqt.DQT_BF16, dqt.DQT_BF16,
                                            dqt.DQT_BF16, m.cfg.lr, m.cfg.seed, m.step_no,
                                            m.counters,
                                            m.workspace(dqt.dqt_linear_bwd_batch_workspace(io, T)))
                if not ctx.has_gamma:
                    if len(dXs) == 1:
                        return dXs[0], None, None
                    dn = dXs[0].float()
                    for d in dXs[1:]:
                        dn += d.float()
                    return dn.to(torch.bfloat16), None, None
                # the norm's backward (y = x r gamma, r = (mean(x^2) + eps)^(-1/2))
                # on the sum of the linears' dX, in one kernel; the gamma
                # gradient from its per-block partial sums
                x, gamma, rinv = saved[2], saved[3], saved[4]
                dx = torch.empty_like(x)
                gpart = torch.empty((MS_NORM_BLOCKS, x.shape[1]), dtype=torch.float32,
                                    device=x.device)
                dqt.dqt_rmsnorm_backward(dXs, x, gamma, rinv, dx, gpart)
                return dx, gpart.sum(0), None

        cls._cls = Fn
        return Fn


class DQTModel:
    """Parameters and train step of a LLaMA-shaped model with DQT linears."""

    def __init__(self, cfg: ModelConfig, device="cuda:0"):
        torch = dqt._torch()
        dqt.load()
        self.cfg = cfg
        self.dev = device
        self._tid = 0
        self.step_no = 0
        self._ws = None
        self.counters = torch.zeros((2,), dtype=torch.int64, device=device)
        g = torch.Generator(device=device)
        g.manual_seed(cfg.seed)
        H, V = cfg.hidden, cfg.vocab
        P = torch.nn.Parameter
        self.emb = P(torch.randn((V, H), generator=g, device=device) * 0.02)
        self.head = P(torch.randn((V, H), generator=g, device=device) * 0.02)
        self.final_norm = P(torch.ones((H,), device=device))
        self.norms = []
        self.groups = []
        for layer in range(cfg.layers):
            self.norms.append((P(torch.ones((H,), device=device)), P(torch.ones((H,), device=device))))
            self.groups.append({gname: _Group(self, layer, gname, lins)
                                for gname, lins in cfg.linears()})
        dense = [self.emb, self.head, self.final_norm] + [p for n in self.norms for p in n]
        self.opt = torch.optim.AdamW(dense, lr=cfg.lr, betas=(0.9, 0.95), weight_decay=0.1)
        hd = H // cfg.heads
        inv = 1.0 / (cfg.rope_base ** (torch.arange(0, hd, 2, device=device, dtype=torch.float32) / hd))
        ang = torch.arange(cfg.seq, device=device, dtype=torch.float32)[:, None] * inv[None, :]
        self.cos = torch.cos(ang).to(torch.bfloat16)[None, None]   # [1, 1, S, hd/2]
        self.sin = torch.sin(ang).to(torch.bfloat16)[None, None]

    def next_tensor_id(self) -> int:
        t = self._tid
        self._tid += 1
        return t

    def workspace(self, nbytes: int):
        """One device workspace for every call (calls on one stream run in
        order); grown when a call needs more."""
        if nbytes == 0:
            return None
        if self._ws is None or self._ws.numel() * 4 < nbytes:
            self._ws = dqt.workspace(nbytes, self.dev)
        return self._ws

    def _rope(self, x):
        # x [B, nh, S, hd]: rotate the two halves of each head
        h = x.shape[-1] // 2
        x1, x2 = x[..., :h], x[..., h:]
        c, s = self.cos, self.sin
        return self._cat((x1 * c - x2 * s, x1 * s + x2 * c))

    @staticmethod
    def _cat(parts):
        return dqt._torch().cat(parts, dim=-1)

    def loss(self, tokens, targets):
        """Forward of one batch: mean next-token cross-entropy (fp32)."""
        torch = dqt._torch()
        F = torch.nn.functional
        from torch.nn.attention import SDPBackend, sdpa_kernel
        cfg = self.cfg
        B, S, H, nh = cfg.batch, cfg.seq, cfg.hidden, cfg.heads
        hd = H // nh
        fn = _DQTGroupFn.get()
        h = F.embedding(tokens.reshape(-1), self.emb.to(torch.bfloat16))     # [T, H] bf16
        for layer in range(cfg.layers):
            grp = self.groups[layer]
            n_attn, n_mlp = self.norms[layer]
            q, k, v = fn.apply(h, n_attn, grp["attn_in"])
            q, k, v = (t.view(B, S, nh, hd).transpose(1, 2) for t in (q, k, v))
            q, k = self._rope(q), self._rope(k)
            # flash / memory-efficient kernels only (no fallback to the math path)
            with sdpa_kernel([SDPBackend.FLASH_ATTENTION, SDPBackend.EFFICIENT_ATTENTION]):
                a = F.scaled_dot_product_attention(q, k, v, is_causal=True)
            a = a.transpose(1, 2).reshape(B * S, H)
            (o,) = fn.apply(a, None, grp["attn_out"])
            h = h + o
            gt, up = fn.apply(h, n_mlp, grp["mlp_in"])
            (d,) = fn.apply(F.silu(gt) * up, None, grp["mlp_hidden"])
            h = h + d
        hn = F.rms_norm(h.float(), (H,), weight=self.final_norm, eps=cfg.eps).to(torch.bfloat16)
        logits = hn @ self.head.to(torch.bfloat16).t()
        return F.cross_entropy(logits.float(), targets.reshape(-1))

    def train_step(self, tokens, targets):
        """One step: forward, backward (the DQT codes are updated by Eq. 5
        inside it, keyed by this step's number), AdamW on the dense
        parameters.  Returns the loss tensor (not synchronised)."""
        self.step_no += 1
        self.opt.zero_grad(set_to_none=True)
        loss = self.loss(tokens, targets)
        loss.backward()
        self.opt.step()
        return loss.detach()


def synthetic_batch(cfg: ModelConfig, step: int, device="cuda:0"):
    """Uniform-random token ids [batch, seq] and the next-token targets."""
    torch = dqt._torch()
    g = torch.Generator(device=device)
    g.manual_seed(cfg.seed * 7919 + step)
    ids = torch.randint(0, cfg.vocab, (cfg.batch, cfg.seq + 1), generator=g, device=device)
    return ids[:, :-1].contiguous(), ids[:, 1:].contiguous()


def initial_loss_expected(cfg: ModelConfig) -> float:
    """Uniform targets: the loss of a near-uniform predictor is ln(vocab)."""
    return math.log(cfg.vocab)
