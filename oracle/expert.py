"""Tenant-private action expert (config 4): forward, loss and weight
gradients in fp64 -- oracle (test infrastructure only).

Sec. 5.2 treats the action head as the tenant-private action module next to
the resident base model (for GR00T- / pi0.5-style models a transformer
"action expert" reading the VLM's features); App. A.3 feeds each tenant's
decode with the shared features of its own requests.  Reading used here (the
paper gives no layer definition): per sample, the expert embeds its
``chunk`` noisy action tokens (``W_in``), runs ``L`` blocks of
[RMSNorm -> self-attention over the sample's action tokens -> RMSNorm ->
cross-attention whose keys / values are projected from *that sample's*
valid backbone rows -> RMSNorm -> GELU MLP], each with a residual, then a
final RMSNorm and ``W_out``; no biases.  Loss: the tenant's mean squared
error against its targets; gradients for every expert weight and norm gain.
The backbone is frozen: nothing flows back into the shared features.

``rnd=True`` rounds to bf16 exactly where the GPU stores a GEMM
operand in bf16 (forward: every GEMM input activation; backward: every
incoming gradient before it meets a GEMM), computing everything else in
fp64.  Attention's matrix products take bf16 operands too: q, k and v are
stored in bf16 by their projections, the probabilities are rounded before
they meet v (unnormalised, relative to the row maximum; the row sum that
normalises the output stays unrounded), and in the backward the incoming
output gradient is rounded before it meets v and the probabilities, the
recomputed (normalised) probabilities before they meet it, and the score
gradient before it meets q and k; the row term sum(dO * O) uses the
unrounded values.  That is the GPU's precision contract.  It does not make the two
agree to fp32 rounding: a value that lands near a bf16 rounding boundary
can round the other way on the GPU, which moves it by one bf16 step, and
the change propagates.  fp32-sized perturbations before every rounding point
move this mode's predictions and gradients by 1e-3 (2 layers) to 5e-3
(6 layers) relative L2, so the stage-wise bar against this mode is 1e-2
relative L2 (about twice that floor).  With ``rnd=False`` the whole expert
is plain fp64 (pinned against finite differences); the GPU is compared with
that mode too, at a bar derived from the distance between the two modes.

Flow-matching objective (the GR00T / pi0.5-style training of such experts):
per sample a flow time tau in (0, 1) and noise eps of the action chunk's
shape are given; the expert's input is the point x = tau eps + (1 - tau) A
on the straight path from the clean actions A to the noise, its regression
target is that path's velocity dx/dtau = eps - A, and every action token's
embedding receives W_time phi(tau), with phi(tau) the sinusoidal features
sin(1000 tau w_j), cos(1000 tau w_j), w_j = 10000^(-j / (D/2)), j < D/2.

Implemented with torch float64 CPU tensors and autograd for the chain rule
(a library primitive; the custom ``Linear`` only decides rounding points).
"""
from __future__ import annotations

from typing import Dict, List, Sequence

import numpy as np
import torch

from .backbone import bf16_to_f64


def _round_bf16(t: torch.Tensor) -> torch.Tensor:
    """Round fp64 values to the nearest bf16 (ties to even), returned in fp64."""
    f = t.to(torch.float32)
    u = f.view(torch.int32).to(torch.int64) & 0xFFFFFFFF
    lsb = (u >> 16) & 1
    r = ((u + 0x7FFF + lsb) >> 16) << 16
    r = torch.where(r >= 2 ** 31, r - 2 ** 32, r).to(torch.int32)
    return r.view(torch.float32).to(torch.float64)


class _Linear(torch.autograd.Function):
    """y = x W^T with the GPU's rounding points: x is already bf16-valued; the
    incoming gradient is rounded to bf16 before both backward products."""

    @staticmethod
    def forward(ctx, x, W, rnd):
        ctx.save_for_backward(x, W)
        ctx.rnd = rnd
        return x @ W.T

    @staticmethod
    def backward(ctx, dy):
        x, W = ctx.saved_tensors
        if ctx.rnd:
            dy = _round_bf16(dy)
        return dy @ W, dy.T @ x, None


def linear(x, W, rnd: bool):
    return _Linear.apply(x, W, rnd)


class _RoundST(torch.autograd.Function):
    """Forward: round to bf16 (a stored GEMM operand); backward: identity."""

    @staticmethod
    def forward(ctx, t):
        return _round_bf16(t)

    @staticmethod
    def backward(ctx, g):
        return g


def _q(t, rnd):
    return _RoundST.apply(t) if rnd else t


def _rms(x, g, eps):
    return x / torch.sqrt(torch.mean(x * x, dim=-1, keepdim=True) + eps) * g


def _gelu(u):
    c = np.sqrt(2.0 / np.pi)
    return 0.5 * u * (1.0 + torch.tanh(c * (u + 0.044715 * u ** 3)))


class _AttnRnd(torch.autograd.Function):
    """One head of softmax(q k^T * scale) v with the GPU's bf16 operands of
    every product (q, k, v already bf16-valued); see the module docstring."""

    @staticmethod
    def forward(ctx, q, k, v, scale):
        s = (q @ k.T) * scale
        m = torch.max(s, dim=-1, keepdim=True).values
        pu = torch.exp(s - m)
        lsum = torch.sum(pu, dim=-1, keepdim=True)
        o = (_round_bf16(pu) @ v) / lsum
        ctx.save_for_backward(q, k, v, o, m + torch.log(lsum))
        ctx.scale = scale
        return o

    @staticmethod
    def backward(ctx, do):
        q, k, v, o, lse = ctx.saved_tensors
        p = torch.exp((q @ k.T) * ctx.scale - lse)
        dor = _round_bf16(do)
        drow = torch.sum(do * o, dim=-1, keepdim=True)
        ds = p * (dor @ v.T - drow)
        dv = _round_bf16(p).T @ dor
        dsr = _round_bf16(ds)
        return (dsr @ k) * ctx.scale, (dsr.T @ q) * ctx.scale, dv, None


def _attn(q, k, v, heads, rnd=False):
    """Bidirectional multi-head attention: q [Lq, d], k/v [Lk, d]; with rnd the
    GPU's bf16 operands of the attention products (q, k, v rounded by the
    caller)."""
    Lq, d = q.shape
    hd = d // heads
    out = []
    for h in range(heads):
        sl = slice(h * hd, (h + 1) * hd)
        if rnd:
            out.append(_AttnRnd.apply(q[:, sl], k[:, sl], v[:, sl], 1.0 / np.sqrt(hd)))
            continue
        s = (q[:, sl] @ k[:, sl].T) / np.sqrt(hd)
        out.append(torch.softmax(s, dim=-1) @ v[:, sl])
    return torch.cat(out, dim=1)


def time_features(tau: float, dim: int) -> np.ndarray:
    """phi(tau) [dim]: sin(1000 tau w_j) for j < dim/2, then cos(1000 tau w_j),
    w_j = 10000^(-j / (dim/2))."""
    half = dim // 2
    w = 10000.0 ** (-np.arange(half, dtype=np.float64) / half)
    ang = 1000.0 * float(tau) * w
    return np.concatenate([np.sin(ang), np.cos(ang)])


def flow_inputs(tau: float, noise: np.ndarray, actions: np.ndarray):
    """(x, v): the point tau * noise + (1 - tau) * actions of the straight path
    and its velocity d x / d tau = noise - actions."""
    e = np.asarray(noise, np.float64)
    a = np.asarray(actions, np.float64)
    return float(tau) * e + (1.0 - float(tau)) * a, e - a


def expert_params(w: dict) -> Dict[str, torch.Tensor]:
    """fp64 leaf tensors (requires_grad) from an expert weight dict of bf16
    bit arrays: w_in [d][a], w_out [a][d], gf [d], and per layer
    wqkv_s [3d][d], wo_s [d][d], wq_c [d][d], wkv_c [2d][dp], wo_c [d][d],
    w_up [f][d], w_down [d][f], g1, g2, g3 [d]."""
    P = {}
    for k in ("w_in", "w_out", "gf", "w_time"):
        if k in w:
            P[k] = torch.tensor(bf16_to_f64(w[k]), requires_grad=True)
    for l, lw in enumerate(w["layers"]):
        for k, v in lw.items():
            P[f"{l}.{k}"] = torch.tensor(bf16_to_f64(v), requires_grad=True)
    return P


def expert_forward(P, n_layers: int, heads: int, eps: float, u: Sequence[np.ndarray],
                   z: Sequence[np.ndarray], rnd: bool, taus: Sequence[float] = None) -> List[torch.Tensor]:
    """Predictions [chunk, a] of every sample.  ``u[i]``: its input action
    tokens [chunk, a]; ``z[i]``: its valid backbone rows [len_i, dp] (bf16 bits
    or floats); ``taus[i]`` (flow matching): its flow time, whose features
    phi(tau) projected by ``w_time`` are added to every token's embedding."""
    preds = []
    for i, (ui, zi) in enumerate(zip(u, z)):
        zt = torch.tensor(bf16_to_f64(zi) if zi.dtype == np.uint16 else np.asarray(zi, np.float64))
        x = linear(_q(torch.tensor(np.asarray(ui, np.float64)), rnd), P["w_in"], rnd)
        if taus is not None:
            phi = np.tile(time_features(taus[i], P["w_time"].shape[1]), (np.asarray(ui).shape[0], 1))
            x = x + linear(_q(torch.tensor(phi), rnd), P["w_time"], rnd)
        for l in range(n_layers):
            g = lambda k: P[f"{l}.{k}"]  # noqa: E731
            d = x.shape[1]
            h = _q(_rms(x, g("g1"), eps), rnd)
            qkv = _q(linear(h, g("wqkv_s"), rnd), rnd)
            a = _attn(qkv[:, :d], qkv[:, d:2 * d], qkv[:, 2 * d:], heads, rnd)
            x = x + linear(_q(a, rnd), g("wo_s"), rnd)
            h = _q(_rms(x, g("g2"), eps), rnd)
            q = _q(linear(h, g("wq_c"), rnd), rnd)
            kv = _q(linear(zt, g("wkv_c"), rnd), rnd)
            a = _attn(q, kv[:, :d], kv[:, d:], heads, rnd)
            x = x + linear(_q(a, rnd), g("wo_c"), rnd)
            h = _q(_rms(x, g("g3"), eps), rnd)
            m = _q(_gelu(linear(h, g("w_up"), rnd)), rnd)
            x = x + linear(m, g("w_down"), rnd)
        y = _q(_rms(x, P["gf"], eps), rnd)
        preds.append(linear(y, P["w_out"], rnd))
    return preds


def expert_step(w: dict, n_layers: int, heads: int, eps: float, u, z, targets, rnd: bool = False,
                flow_t=None) -> Dict:
    """Forward, the tenant's MSE loss and the gradient of every parameter.

    ``targets``: [n, chunk, a].  With ``flow_t`` ([n] flow times), ``u`` is
    the noise and ``targets`` the clean actions: the expert reads
    ``flow_inputs`` and regresses the path velocity (flow matching).
    Returns {"pred": [n, chunk, a] fp64, "loss": float, "grads": {name: fp64
    array}} with names as in ``expert_params``."""
    P = expert_params(w)
    if flow_t is not None:
        pairs = [flow_inputs(flow_t[i], u[i], targets[i]) for i in range(len(u))]
        u = [x for x, _ in pairs]
        targets = np.stack([v for _, v in pairs])
    preds = expert_forward(P, n_layers, heads, eps, u, z, rnd, None if flow_t is None else list(flow_t))
    Y = torch.stack(preds)
    T = torch.tensor(np.asarray(targets, np.float64)).reshape(Y.shape)
    loss = torch.mean((Y - T) ** 2)
    loss.backward()
    return {"pred": Y.detach().numpy(), "loss": float(loss.detach()),
            "grads": {k: v.grad.numpy().copy() for k, v in P.items()}}
