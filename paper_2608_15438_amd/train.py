"""Encoder training with the selective similarity loss L_sim (Sec. 3.2.2,
Eq. similarityconfig and the mask of Eq. 8), untimed.  On the GPU the
pairwise input distances run on the library's fp32 matrix-core kernel
(nr_pair_sqdist) and the loss, mask and latent gradient in one fused pass
over the pairs (nr_lsim_grad); the encoder's own layers are torch Linear
modules.  lsim_loss below is the same loss in PyTorch (CPU checks).

For a mini-batch of B rows x (scaled as the encoder sees them) and their
latents l, with rho = sqrt(L_dim / E_dim):
  S_emb(i, j) = ||x_i - x_j||,  S_lat(i, j) = ||l_i - l_j||,
  Mask(i, j) = [i != j and (S_emb <= tau_emb or S_lat <= gamma rho tau_emb)],
  L_sim = sum(Mask * (S_lat - gamma rho S_emb)^2) / sum(Mask).
tau_emb is either fixed or, per batch, a quantile of the off-diagonal S_emb
(the paper's mask keeps roughly the most similar 0.5 % of the pairs).
"""
from __future__ import annotations

import math
from dataclasses import replace
from typing import Callable, Optional

import numpy as np
import torch

from .index_build import Encoder


def pairwise_dist(a: torch.Tensor) -> torch.Tensor:
    """||a_i - a_j|| for all pairs, from |a|^2 - 2 a.a' + |a'|^2 (one GEMM),
    clamped at 0; the diagonal is set to 0 and kept out of the square root,
    and a 1e-20 floor under it keeps the derivative finite for coinciding
    points (their distance gradient is then 0, not 0 * inf)."""
    n2 = (a * a).sum(1)
    d2 = (n2[:, None] - 2.0 * (a @ a.T) + n2[None, :]).clamp_min(0.0)
    eye = torch.eye(a.shape[0], dtype=torch.bool, device=a.device)
    d2 = torch.where(eye, torch.ones_like(d2), d2)
    return torch.where(eye, torch.zeros_like(d2), torch.sqrt(d2 + 1e-20))


def lsim_loss(x: torch.Tensor, lat: torch.Tensor, gamma: float, tau_emb: Optional[float] = None,
              quantile: float = 0.005):
    """(L_sim, tau_emb used, mask fraction) of one batch."""
    B, E = x.shape
    L = lat.shape[1]
    rho = math.sqrt(L / E)
    with torch.no_grad():
        s_emb = pairwise_dist(x)
        off = ~torch.eye(B, dtype=torch.bool, device=x.device)
        if tau_emb is None:
            tau_emb = float(torch.quantile(s_emb[off].float()[: 1 << 24], quantile))
    s_lat = pairwise_dist(lat)
    mask = off & ((s_emb <= tau_emb) | (s_lat.detach() <= gamma * rho * tau_emb))
    m = mask.to(lat.dtype)
    n = m.sum()
    loss = (m * (s_lat - gamma * rho * s_emb) ** 2).sum() / n.clamp_min(1.0)
    return loss, tau_emb, float(n) / (B * (B - 1))


class _LsimGpu(torch.autograd.Function):
    """L_sim of one batch from the fused kernel's (numerator, count) and
    latent gradient; backward hands that gradient on (the mask held fixed)."""

    @staticmethod
    def forward(ctx, lat, num_cnt, grad):
        cnt = num_cnt[1].clamp_min(1.0)
        ctx.save_for_backward(grad, cnt)
        return (num_cnt[0] / cnt).to(lat.dtype)

    @staticmethod
    def backward(ctx, g):
        grad, cnt = ctx.saved_tensors
        return (grad * (g / cnt)).to(grad.dtype), None, None


def lsim_loss_gpu(x: torch.Tensor, lat: torch.Tensor, gamma: float,
                  tau_emb: Optional[float] = None, quantile: float = 0.005):
    """(L_sim, tau_emb used, mask fraction) of one batch on the library's
    kernels; tau_emb defaults to the quantile of the off-diagonal input
    distances (taken on their squares, the same order)."""
    from . import neuroute as NR
    B, E = x.shape
    L = lat.shape[1]
    gr = gamma * math.sqrt(L / E)
    d2 = NR.nr_pair_sqdist(x.float().contiguous())
    if tau_emb is None:
        off = ~torch.eye(B, dtype=torch.bool, device=x.device)
        tau_emb = math.sqrt(float(torch.quantile(d2[off][: 1 << 24], quantile)))
    num_cnt, grad = NR.nr_lsim_grad(d2, lat.detach().float().contiguous(), gr, tau_emb)
    loss = _LsimGpu.apply(lat, num_cnt, grad)
    return loss, tau_emb, float(num_cnt[1]) / (B * (B - 1))


class _Mlp(torch.nn.Module):
    """The encoder as trainable fp32 layers (ReLU between layers, the input
    scaled as at query time)."""

    def __init__(self, enc: Encoder, device):
        super().__init__()
        self.scale = enc.input_scale
        self.lin = torch.nn.ModuleList()
        for W, b in zip(enc.weights, enc.biases):
            l = torch.nn.Linear(W.shape[1], W.shape[0])
            with torch.no_grad():
                l.weight.copy_(torch.as_tensor(np.asarray(W)))
                l.bias.copy_(torch.as_tensor(np.asarray(b)))
            self.lin.append(l)
        self.to(device)

    def forward(self, x):
        h = x * self.scale
        for i, l in enumerate(self.lin):
            h = l(h)
            if i + 1 < len(self.lin):
                h = torch.relu(h)
        return h

    def encoder(self, like: Encoder) -> Encoder:
        return replace(like, weights=[l.weight.detach().float().cpu().numpy() for l in self.lin],
                       biases=[l.bias.detach().float().cpu().numpy() for l in self.lin])


def train_encoder(enc: Encoder, rows_fn: Callable, n: int, steps: int, batch: int = 4096,
                  lr: float = 2e-4, gamma: float = 0.6, tau_emb: Optional[float] = None,
                  quantile: float = 0.005, seed: int = 0, device="cuda", log=None) -> Encoder:
    """Adam on L_sim over seeded batches of rows drawn from [0, n) (the
    encoder has no BatchNorm; its biases and weights are trained)."""
    dev = torch.device(device)
    net = _Mlp(enc, dev)
    opt = torch.optim.Adam(net.parameters(), lr=lr)
    g = torch.Generator(device="cpu").manual_seed(seed)
    for it in range(steps):
        ids = torch.randint(0, n, (batch,), generator=g)
        x = torch.as_tensor(rows_fn(ids.to(dev))).to(dev).float()
        xs = x * enc.input_scale
        lat = net(x)
        fn = lsim_loss_gpu if dev.type == "cuda" else lsim_loss
        loss, tau, frac = fn(xs, lat, gamma, tau_emb, quantile)
        opt.zero_grad(set_to_none=True)
        loss.backward()
        opt.step()
        if log and (it % max(1, steps // 10) == 0 or it == steps - 1):
            log(f"train step {it}: L_sim {float(loss.detach()):.5f}, tau_emb {tau:.4f}, "
                f"mask {frac:.4%}")
    return net.encoder(enc)
