"""Pseudo-quantised linear module for SPHQuant's layer-wise fine-tuning (Sec. 3.3; App. A steps
6-10), on the library's device kernels.

The trainable parameters are the angle logits ``phi`` of the codebook (Eq. 9-10) and one radius
parameter ``rho`` per 8-D weight vector (r = softplus(rho)); the signs and direction indices stay
fixed after initialisation. Every forward rebuilds the codebook (``sph_angular_codebook``) and the
fake-quantised weight (``sph_fake_quant_forward``); the backward runs the straight-through
gradients (``sph_fake_quant_backward``, ``sph_angular_codebook_backward``). Only the product of the
activations with the rebuilt weight is a plain library GEMM (torch.matmul). ``finalize`` returns
the discrete codes and fp16 codebook of App. A step 10, ready for ``pack`` and the decode path.
"""
from __future__ import annotations

import numpy as np

from . import sph as B


def _torch():
    import torch
    return torch


class _AngularCodebook:
    """autograd Function: phi [2^D][7] -> codebook [2^D][8] (Eq. 9-10)."""

    @staticmethod
    def build():
        torch = _torch()

        class Fn(torch.autograd.Function):
            @staticmethod
            def forward(ctx, phi, dir_bits, eps):
                ctx.save_for_backward(phi)
                ctx.dir_bits, ctx.eps = dir_bits, eps
                return B.angular_codebook(dir_bits, phi.detach(), eps)

            @staticmethod
            def backward(ctx, grad_c):
                (phi,) = ctx.saved_tensors
                return B.angular_codebook_backward(ctx.dir_bits, phi.detach(), grad_c, ctx.eps), None, None

        return Fn


class _FakeQuant:
    """autograd Function: (rho, codebook) -> W^ with straight-through gradients."""

    @staticmethod
    def build():
        torch = _torch()

        class Fn(torch.autograd.Function):
            @staticmethod
            def forward(ctx, rho, codebook, mod):
                w, r_hat = B.fake_quant_forward(mod.dir_bits, mod.radius_bits, rho.detach(), mod.signs,
                                                mod.dir_idx, codebook.detach())
                ctx.save_for_backward(rho, codebook, r_hat)
                ctx.mod = mod
                return w

            @staticmethod
            def backward(ctx, grad_w):
                rho, codebook, r_hat = ctx.saved_tensors
                m = ctx.mod
                g_rho, g_cb = B.fake_quant_backward(m.dir_bits, m.radius_bits, rho.detach(), m.signs,
                                                    m.dir_idx, codebook.detach(), r_hat, grad_w,
                                                    m.perm, m.offsets, workspace=m._bwd_ws)
                return g_rho, g_cb, None

        return Fn


_FNS = {}


def _fn(name):
    if name not in _FNS:
        _FNS[name] = {"angular": _AngularCodebook, "fq": _FakeQuant}[name].build()
    return _FNS[name]


def make_module(w, dir_bits: int, radius_bits: int, init_codebook=None, kmeans_uniforms=None,
                kmeans_iters: int = 20, eps: float = B.ANGLE_EPS, bias=None):
    """A pseudo-quantised linear layer y = x W^T (+ bias) initialised from a dense device fp32
    matrix ``w`` [n][k] (App. A steps 5-7): the codebook is ``init_codebook`` (device fp16 bits
    [2^D][8]), refined by radius-weighted spherical k-means when ``kmeans_uniforms`` (device fp64
    draws) is given; signs and directions come from the device encoder; rho from Eq. 6's radius;
    phi from the inverse of Eq. 9-10."""
    torch = _torch()

    class SphFakeQuantLinear(torch.nn.Module):
        def __init__(self):
            super().__init__()
            self.dir_bits, self.radius_bits, self.eps = dir_bits, radius_bits, eps
            n, k = w.shape
            self.n, self.k = n, k
            cb16 = init_codebook
            if kmeans_uniforms is not None:
                cb16, _obj, _idx = B.kmeans_codebook(dir_bits, radius_bits, w, kmeans_uniforms, init_codebook,
                                                     kmeans_iters)
            codes = B.encode(dir_bits, radius_bits, w, cb16)
            cb32 = cb16.view(torch.float16).float()
            self.register_buffer("signs", codes["signs"])
            self.register_buffer("dir_idx", codes["dir"])
            perm, off = B.direction_groups(dir_bits, codes["dir"].cpu().numpy().view(np.uint16))
            self.register_buffer("perm", torch.from_numpy(perm).to(w.device))
            self.register_buffer("offsets", torch.from_numpy(off).to(w.device))
            self.phi = torch.nn.Parameter(B.angular_logits(dir_bits, cb32, eps))
            self.rho = torch.nn.Parameter(B.fake_quant_init_rho(dir_bits, radius_bits, w, codes["dir"], cb32))
            self.bias = None if bias is None else torch.nn.Parameter(bias.detach().clone().float())
            nb = ctypes_size(dir_bits)
            self._bwd_ws = torch.empty(nb, dtype=torch.uint8, device=w.device)

        def codebook(self):
            return _fn("angular").apply(self.phi, self.dir_bits, self.eps)

        def weight(self):
            return _fn("fq").apply(self.rho, self.codebook(), self)

        def forward(self, x):
            y = torch.matmul(x, self.weight().t())
            return y if self.bias is None else y + self.bias

        @torch.no_grad()
        def finalize(self):
            """App. A step 10: the discrete codes (host numpy, as ``pack`` takes them) and the fp16
            codebook, and the fp32 weight they decode to up to the fp16 rounding of the codebook."""
            c = self.codebook()
            w_hat, _r, cq = B.fake_quant_forward(self.dir_bits, self.radius_bits, self.rho, self.signs,
                                                 self.dir_idx, c, want_codes=True)
            codes = B.codes_to_host({"signs": self.signs, "dir": self.dir_idx, **cq})
            cb16 = c.half().cpu().numpy().view(np.uint16)
            return codes, cb16, w_hat

    return SphFakeQuantLinear()


def ctypes_size(dir_bits: int) -> int:
    import ctypes
    nb = ctypes.c_size_t(0)
    B._check(B.load_library().sph_fake_quant_backward_workspace_bytes(dir_bits, ctypes.byref(nb)),
             "sph_fake_quant_backward_workspace_bytes")
    return nb.value
