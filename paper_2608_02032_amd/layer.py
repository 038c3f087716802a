"""A trainable DART layer on top of libdart (the MQAR smoke training of the
paper's App. D.1: two-layer models, chunk size 16, state size N in {16, 64}).

Every step of the DART path -- the width-4 convolution with SiLU, the step
sizes, the chunked scan with its chunk memories, state-memory attention with
the gated residual, the gated RMSNorm -- runs forward and backward in the
library's HIP kernels through the torch.autograd.Function wrappers below;
PyTorch supplies the plain GEMMs around them (input and output projections,
embeddings, the LM head), the optimiser and device memory.  The residual-
stream RMSNorm and the D skip are elementwise torch ops.

Storage is float32 (the library's fp32 path); the gradients the library
returns are float32 as well.
"""
from __future__ import annotations

import math

import torch
import torch.nn as nn
import torch.nn.functional as F

from . import dart


# --------------------------------------------------------------------------- #
# autograd wrappers: forward and backward both in libdart
# --------------------------------------------------------------------------- #

class _ConvSiLU(torch.autograd.Function):
    @staticmethod
    def forward(ctx, x, w, b):
        out, _ = dart.conv1d_silu(x, w, b)
        ctx.save_for_backward(x, w, b)
        return out

    @staticmethod
    def backward(ctx, dout):
        x, w, b = ctx.saved_tensors
        g = dart.conv1d_silu_bwd(x, w, dout.contiguous(), bias=b)
        return g["din"], g["dweight"], g["dbias"]


class _DtSoftplus(torch.autograd.Function):
    @staticmethod
    def forward(ctx, raw, bias):
        ctx.save_for_backward(raw, bias)
        return dart.dt_softplus(raw, bias)

    @staticmethod
    def backward(ctx, ddt):
        raw, bias = ctx.saved_tensors
        draw, dbias = dart.dt_softplus_bwd(raw, ddt.contiguous(), bias=bias)
        return draw, dbias


class _Scan(torch.autograd.Function):
    """(x, dt, A, B, C) -> (y_ssd, memories): Sec. 2 recurrence, Sec. 3 chunk
    memories; the backward takes the memories' gradient from SMA."""

    @staticmethod
    def forward(ctx, x, dt, A, Bm, Cm, chunk):
        y, mem, _ = dart.ssd_chunk_scan(x, dt, A, Bm, Cm, chunk, h_last=False)
        ctx.chunk = chunk
        ctx.save_for_backward(x, dt, A, Bm, Cm)
        return y, mem

    @staticmethod
    def backward(ctx, dy, dmem):
        x, dt, A, Bm, Cm = ctx.saved_tensors
        if dy is None:
            dy = torch.zeros_like(x)
        g = dart.ssd_bwd(x, dt, A, Bm, Cm, ctx.chunk, dy.contiguous(),
                         dmem=None if dmem is None else dmem.contiguous())
        return g["dx"], g["ddt"], g["dA"], g["dB"], g["dC"], None


class _Sma(torch.autograd.Function):
    """(q, e, C, memories, gate pre-activation, y_ssd) -> y = y_ssd + SiLU(z) R:
    Sec. 3 and App. B.1; the backward recomputes the scores (App. C)."""

    @staticmethod
    def forward(ctx, q, e, Cm, mem, z, y_ssd, chunk):
        y, lse = dart.sma_fwd(q, e, Cm, mem, z, y_ssd, chunk)
        ctx.chunk = chunk
        ctx.save_for_backward(q, e, Cm, mem, z, lse)
        return y

    @staticmethod
    def backward(ctx, dy):
        q, e, Cm, mem, z, lse = ctx.saved_tensors
        dy = dy.contiguous()
        g = dart.sma_bwd(q, e, Cm, mem, z, lse, dy, ctx.chunk)
        return g["dq"], g["de"], g["dC"], g["dmem"], g["dz"], dy, None


class _GatedNorm(torch.autograd.Function):
    @staticmethod
    def forward(ctx, y, z, w):
        ctx.save_for_backward(y, z, w)
        return dart.gated_rmsnorm(y, z, w)

    @staticmethod
    def backward(ctx, dout):
        y, z, w = ctx.saved_tensors
        g = dart.gated_rmsnorm_bwd(y, z, dout.contiguous(), weight=w)
        return g["dy"], g["dz"], g["dweight"]


# --------------------------------------------------------------------------- #
# the block and a small language model
# --------------------------------------------------------------------------- #

def _rmsnorm(u, w, eps=1e-6):
    return u * torch.rsqrt(u.pow(2).mean(-1, keepdim=True) + eps) * w


class DartBlock(nn.Module):
    """Mamba-2 block with DART's state-memory attention branch (Sec. 3):
    in_proj -> [gate z | x, B, C (conv1d + SiLU) | dt | Q | E | SMA gate]
    -> scan (memories kept) -> SMA + SiLU-gated residual -> + D x
    -> gated RMSNorm with z -> out_proj, around a pre-norm residual."""

    def __init__(self, d_model, d_state=16, headdim=64, expand=2, chunk=16, ngroups=1):
        super().__init__()
        d_inner = expand * d_model
        if d_inner % headdim:
            raise ValueError("expand * d_model must be a multiple of headdim")
        self.H = d_inner // headdim
        self.P, self.N, self.G, self.S = headdim, d_state, ngroups, chunk
        self.d_inner = d_inner
        self.conv_dim = d_inner + 2 * ngroups * d_state
        widths = [d_inner, self.conv_dim, self.H, ngroups * d_state, ngroups * headdim, self.H]
        self.splits = widths
        self.norm_w = nn.Parameter(torch.ones(d_model))
        self.in_proj = nn.Linear(d_model, sum(widths), bias=False)
        with torch.no_grad():
            # the SMA gate projection W_G starts at zero (Sec. 3)
            self.in_proj.weight[-self.H:].zero_()
        self.conv_w = nn.Parameter(torch.randn(self.conv_dim, 4) / 2.0)
        self.conv_b = nn.Parameter(torch.zeros(self.conv_dim))
        dt0 = torch.exp(torch.empty(self.H).uniform_(math.log(1e-3), math.log(1e-1)))
        self.dt_bias = nn.Parameter(dt0 + torch.log(-torch.expm1(-dt0)))  # softplus^-1
        self.A_log = nn.Parameter(torch.log(torch.empty(self.H).uniform_(1.0, 16.0)))
        self.D = nn.Parameter(torch.ones(self.H))
        self.out_norm_w = nn.Parameter(torch.ones(d_inner))
        self.out_proj = nn.Linear(d_inner, d_model, bias=False)

    def forward(self, u):
        B_, L, _ = u.shape
        H, P, N, G = self.H, self.P, self.N, self.G
        proj = self.in_proj(_rmsnorm(u, self.norm_w))
        z, xbc, dtr, q, e, g = torch.split(proj, self.splits, dim=-1)
        xbc = _ConvSiLU.apply(xbc.contiguous(), self.conv_w, self.conv_b)
        x, Bm, Cm = torch.split(xbc, [self.d_inner, G * N, G * N], dim=-1)
        x = x.reshape(B_, L, H, P).contiguous()
        Bm = Bm.reshape(B_, L, G, N).contiguous()
        Cm = Cm.reshape(B_, L, G, N).contiguous()
        dt = _DtSoftplus.apply(dtr.contiguous(), self.dt_bias)
        A = -torch.exp(self.A_log)
        y_ssd, mem = _Scan.apply(x, dt, A, Bm, Cm, self.S)
        y = _Sma.apply(q.reshape(B_, L, G, N).contiguous(), e.reshape(B_, L, G, P).contiguous(),
                       Cm, mem, g.contiguous(), y_ssd, self.S)
        y = y + self.D.view(1, 1, H, 1) * x
        y = _GatedNorm.apply(y.reshape(B_, L, self.d_inner), z.contiguous(), self.out_norm_w)
        return u + self.out_proj(y)


class DartLM(nn.Module):
    """Embedding -> DART blocks -> RMSNorm -> LM head (untied, App. D.1)."""

    def __init__(self, vocab, d_model=64, n_layers=2, d_state=16, chunk=16, headdim=64, expand=2):
        super().__init__()
        self.emb = nn.Embedding(vocab, d_model)
        self.blocks = nn.ModuleList(
            [DartBlock(d_model, d_state, headdim, expand, chunk) for _ in range(n_layers)])
        self.norm_w = nn.Parameter(torch.ones(d_model))
        self.head = nn.Linear(d_model, vocab, bias=False)

    def forward(self, tokens):
        u = self.emb(tokens)
        for blk in self.blocks:
            u = blk(u)
        return self.head(_rmsnorm(u, self.norm_w))


def train_mqar(steps, L=256, R=None, batch=64, d_model=64, d_state=16, chunk=16, lr=1e-3,
               seed=0, vocab=None, log_every=0, device="cuda"):
    """Train DartLM on MQAR batches drawn fresh each step (R pairs, default the
    first curriculum stage L/16) with AdamW, gradient clipping at 1.0 and a
    linear learning-rate decay.  Returns the per-step losses and the query
    accuracy of each step's batch (before the update)."""
    import numpy as np

    from . import mqar
    vocab = vocab or mqar.MqarVocab()
    R = R or L // 16
    torch.manual_seed(seed)
    rng = np.random.default_rng(seed)
    model = DartLM(vocab.size, d_model, 2, d_state, chunk).to(device)
    opt = torch.optim.AdamW(model.parameters(), lr=lr, weight_decay=0.1, betas=(0.9, 0.95))
    sched = torch.optim.lr_scheduler.LambdaLR(opt, lambda s: 1.0 - s / max(steps, 1))
    losses, accs = [], []
    for step in range(steps):
        tok, lab = mqar.mqar_batch(rng, batch, L, R, vocab)
        tok = torch.from_numpy(tok).to(device)
        lab = torch.from_numpy(lab).to(device)
        logits = model(tok)
        loss = F.cross_entropy(logits.view(-1, vocab.size), lab.view(-1), ignore_index=mqar.IGNORE)
        with torch.no_grad():
            m = lab != mqar.IGNORE
            acc = (logits.argmax(-1)[m] == lab[m]).float().mean()
        opt.zero_grad(set_to_none=True)
        loss.backward()
        torch.nn.utils.clip_grad_norm_(model.parameters(), 1.0)
        opt.step()
        sched.step()
        losses.append(float(loss.detach()))
        accs.append(float(acc))
        if log_every and (step % log_every == 0 or step == steps - 1):
            print("step %4d loss %.4f acc %.3f" % (step, losses[-1], accs[-1]), flush=True)
    return losses, accs
