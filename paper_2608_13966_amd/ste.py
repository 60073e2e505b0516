"""Training through the reconstruction: a linear layer whose forward pass uses
QUASAR's reconstruction r of latent weights W, with the straight-through
estimator (Sec. 3.2: the gradient is evaluated at r and applied to W), and
whose optimiser step is the fused AdamW + reconstruction of libquasar.so.

The forward/backward products are ordinary torch matmuls (the model around
the path); the optimiser update and the reconstruction run in the HIP kernels
behind ``quasar_adamw_reconstruct``.
"""
from __future__ import annotations

import math

import torch

from . import quasar as Q


class _STELinear(torch.autograd.Function):
    """y = x r^T; dL/dx = dL/dy r; dL/dW := dL/dr = dL/dy^T x (straight through)."""

    @staticmethod
    def forward(ctx, x, weight, r):
        ctx.save_for_backward(x, r)
        return x @ r.to(x.dtype).t()

    @staticmethod
    def backward(ctx, gy):
        x, r = ctx.saved_tensors
        gx = gy @ r.to(gy.dtype)
        gw = gy.reshape(-1, gy.shape[-1]).t() @ x.reshape(-1, x.shape[-1])
        return gx, gw.to(torch.float32), None


class QuasarLinear(torch.nn.Module):
    """Linear layer (no bias) with fp32 latent weights trained by AdamW and
    quantised by QUASAR at every step.

    ``weight`` is the latent W (a Parameter, so autograd delivers its
    gradient); ``m`` and ``v`` are AdamW's moments; ``r`` (bf16) is the
    reconstruction the forward pass uses; ``codes``/``scales``/``zeros`` are
    the deployable form of r.  Call :meth:`step` after ``backward()``.
    """

    def __init__(self, in_features: int, out_features: int, *, fmt="int", bits=4, group=128,
                 clips=(1.0, 0.95, 0.9, 0.85, 0.8, 0.75, 0.7, 0.65), lr=1e-3, betas=(0.9, 0.999), eps=1e-8,
                 weight_decay=0.0, weighting="h", device="cuda", generator=None):
        super().__init__()
        if fmt == "nvfp4":
            raise ValueError("QuasarLinear supports the INT formats (NVFP4 needs the tensor amax state)")
        w = torch.empty(out_features, in_features, device=device, dtype=torch.float32)
        torch.nn.init.kaiming_uniform_(w, a=math.sqrt(5), generator=generator)
        self.weight = torch.nn.Parameter(w)
        self.register_buffer("m", torch.zeros_like(w))
        self.register_buffer("v", torch.zeros_like(w))
        self.cfg = dict(fmt=fmt, bits=bits, group=group, clips=tuple(clips), weighting=weighting)
        self.hp = dict(lr=lr, beta1=betas[0], beta2=betas[1], eps=eps, weight_decay=weight_decay)
        self.t = 0
        # initial reconstruction: no saliency yet (v = 0), so every group keeps
        # the min-max RTN dequantiser of the first clip (Standard QAT)
        out = Q.reconstruct(self.weight.data, self.v.clone(), None, want_diag=True, **self.cfg)
        self.register_buffer("r", out["r"].to(torch.bfloat16))
        self._out = None
        self.codes, self.scales, self.zeros = out["codes"], out["scales"], out["zeros"]

    def forward(self, x):
        return _STELinear.apply(x, self.weight, self.r)

    @torch.no_grad()
    def step(self):
        """One fused AdamW step on the latent weights from their gradient,
        then the reconstruction of the result into ``r`` (in place)."""
        g = self.weight.grad
        if g is None:
            raise RuntimeError("no gradient: call backward() first")
        self.t += 1
        if self._out is None:
            d = Q.Descriptor(*self.weight.shape, w_dtype=Q.F32, g_dtype=Q.F32, **self.cfg)
            self._out = Q.alloc_outputs(d, self.weight.data, want_r=False, want_diag=True, has_amax=True)
            self._out["r"] = self.r
        Q.adamw_reconstruct(self.weight.data, self.m, self.v, g.contiguous(), step=self.t, out=self._out,
                            r_dtype="bf16", **self.cfg, **self.hp)
        self.codes, self.scales, self.zeros = self._out["codes"], self._out["scales"], self._out["zeros"]
        self.weight.grad = None
