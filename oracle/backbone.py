"""Frozen shared-backbone forward, one sample at a time, in fp64 -- oracle
(test infrastructure only).

Sec. 4.3 / App. A.3: the shared frozen prefix ("base model", VLM) encodes
the canonical batch once (``encode``); Sec. 5.2: group execution runs one
shared base-model forward over the concatenated tenant inputs.  Since the
samples of a batch do not interact in that forward, the result for each
sample is the forward of that sample alone -- which is what this module
computes.  The paper gives no layer-level definition; the readings used
are a pre-RMSNorm transformer block with bidirectional attention over the
sample's own valid tokens, no positional term (inputs are pre-embedded),
RMSNorm ``x / sqrt(mean(x^2) + eps) * g``, tanh-form GELU, a GELU MLP
``W_down gelu(W_up h)`` or a GeGLU MLP ``W_down (gelu(W_gate h) * W_up h)``,
no biases, and a final RMSNorm whose output is the shared feature.

Backbone variants (the VLM families the paper's tenants build on): a causal
mask inside each sample; rotary position embedding of q and k (rotate-half
form, frequencies theta^(-2i/hd)) with positions counted from 0 inside every
sample; fewer key/value heads than query heads (query head h reads key/value
head h // (H / Hkv)).  Each sample still runs alone, so positions restart per
sample by construction.

All arithmetic is fp64 on the exactly widened bf16 inputs and weights.
"""
from __future__ import annotations

from typing import Callable, List, Sequence

import numpy as np


def bf16_to_f64(bits: np.ndarray) -> np.ndarray:
    """Widen bf16 bit patterns (uint16) exactly to fp64."""
    u = np.asarray(bits, dtype=np.uint16).astype(np.uint32) << np.uint32(16)
    return u.view(np.float32).astype(np.float64)


def rms_norm(x: np.ndarray, g: np.ndarray, eps: float) -> np.ndarray:
    """Row-wise RMSNorm: x / sqrt(mean(x^2) + eps) * g."""
    ms = np.mean(x * x, axis=-1, keepdims=True)
    return x / np.sqrt(ms + eps) * g


def gelu(u: np.ndarray) -> np.ndarray:
    """tanh-form GELU: 0.5 u (1 + tanh(sqrt(2/pi) (u + 0.044715 u^3)))."""
    c = np.sqrt(2.0 / np.pi)
    return 0.5 * u * (1.0 + np.tanh(c * (u + 0.044715 * u ** 3)))


def gelu_grad(u: np.ndarray) -> np.ndarray:
    """d/du of the tanh-form GELU, in closed form."""
    c = np.sqrt(2.0 / np.pi)
    inner = c * (u + 0.044715 * u ** 3)
    t = np.tanh(inner)
    return 0.5 * (1.0 + t) + 0.5 * u * (1.0 - t * t) * c * (1.0 + 3 * 0.044715 * u * u)


def softmax_rows(s: np.ndarray) -> np.ndarray:
    m = np.max(s, axis=-1, keepdims=True)
    e = np.exp(s - m)
    return e / np.sum(e, axis=-1, keepdims=True)


def attention(q: np.ndarray, k: np.ndarray, v: np.ndarray, heads: int, kv_heads: int = 0,
              causal: bool = False) -> np.ndarray:
    """Multi-head attention over one sample's rows (bidirectional, or causal:
    row j attends to rows 0..j).

    q: [len, heads*hd]; k, v: [len, kv_heads*hd], head h in columns
    [h*hd, (h+1)*hd); query head h reads key/value head h // (heads/kv_heads).
    """
    L, d = q.shape
    hd = d // heads
    kvh = kv_heads or heads
    group = heads // kvh
    out = np.empty_like(q)
    scale = 1.0 / np.sqrt(hd)
    for h in range(heads):
        sl = slice(h * hd, (h + 1) * hd)
        kl = slice((h // group) * hd, (h // group + 1) * hd)
        s = (q[:, sl] @ k[:, kl].T) * scale
        if causal:
            s = np.where(np.tril(np.ones((L, L), dtype=bool)), s, -np.inf)
        out[:, sl] = softmax_rows(s) @ v[:, kl]
    return out


def rope(x: np.ndarray, heads: int, theta: float, positions: np.ndarray) -> np.ndarray:
    """Rotary embedding of every head of x [len, heads*hd]: for i < hd/2 the
    pair (x_i, x_{i+hd/2}) of the row at position p is rotated by the angle
    p * theta^(-2i/hd)."""
    L, w = x.shape
    hd = w // heads
    half = hd // 2
    i = np.arange(half, dtype=np.float64)
    ang = np.asarray(positions, np.float64)[:, None] * theta ** (-2.0 * i / hd)[None, :]
    c, s = np.cos(ang), np.sin(ang)
    out = np.empty_like(x)
    for h in range(heads):
        a = x[:, h * hd: h * hd + half]
        b = x[:, h * hd + half: (h + 1) * hd]
        out[:, h * hd: h * hd + half] = a * c - b * s
        out[:, h * hd + half: (h + 1) * hd] = b * c + a * s
    return out


class LayerF64:
    """fp64 copy of one backbone layer's weights ([out][in] layout)."""

    def __init__(self, w: dict, glu: bool):
        self.wqkv = bf16_to_f64(w["wqkv"])
        self.wo = bf16_to_f64(w["wo"])
        self.w_up = bf16_to_f64(w["w_up"])
        self.w_gate = bf16_to_f64(w["w_gate"]) if glu else None
        self.w_down = bf16_to_f64(w["w_down"])
        self.g1 = bf16_to_f64(w["g1"])
        self.g2 = bf16_to_f64(w["g2"])


def layer_forward(x: np.ndarray, lw: LayerF64, heads: int, eps: float, kv_heads: int = 0, causal: bool = False,
                  rope_theta: float = 0.0) -> np.ndarray:
    """One pre-RMSNorm block on one sample's rows x [len, d]."""
    L, d = x.shape
    hd = d // heads
    kvw = (kv_heads or heads) * hd
    h = rms_norm(x, lw.g1, eps)
    qkv = h @ lw.wqkv.T
    q, k, v = qkv[:, :d], qkv[:, d:d + kvw], qkv[:, d + kvw:d + 2 * kvw]
    if rope_theta > 0:
        pos = np.arange(L)
        q = rope(q, heads, rope_theta, pos)
        k = rope(k, kv_heads or heads, rope_theta, pos)
    a = attention(q, k, v, heads, kv_heads, causal)
    x = x + a @ lw.wo.T
    h = rms_norm(x, lw.g2, eps)
    if lw.w_gate is None:
        m = gelu(h @ lw.w_up.T)
    else:
        m = gelu(h @ lw.w_gate.T) * (h @ lw.w_up.T)
    return x + m @ lw.w_down.T


def backbone_forward(samples: Sequence[np.ndarray], layer_weights: Callable[[int], dict],
                     n_layers: int, heads: int, glu: bool, eps: float,
                     gf_bits: np.ndarray, kv_heads: int = 0, causal: bool = False,
                     rope_theta: float = 0.0) -> List[np.ndarray]:
    """Final hidden states z [len_i, d] (fp64) of each sample, each run alone.

    ``samples[i]`` holds the sample's valid rows only (bf16 bits or floats).
    ``layer_weights(l)`` returns layer l's bf16 weight dict; layers are
    visited outermost so each layer is widened to fp64 once, but no row of
    one sample ever meets a row of another.
    """
    xs = [bf16_to_f64(s) if s.dtype == np.uint16 else np.asarray(s, np.float64) for s in samples]
    for l in range(n_layers):
        lw = LayerF64(layer_weights(l), glu)
        xs = [layer_forward(x, lw, heads, eps, kv_heads, causal, rope_theta) for x in xs]
        del lw
    gf = bf16_to_f64(gf_bits)
    return [rms_norm(x, gf, eps) for x in xs]


def pool(z: np.ndarray) -> np.ndarray:
    """Shared feature handed to a tenant's MLP head: mean over the sample's
    valid rows of the final hidden state."""
    return z.mean(axis=0)
