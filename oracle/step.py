"""Isolated-execution reference of the whole group-batched step -- oracle
(test infrastructure only).

Sec. 5.2 defines the grouped step against serial execution: the same
per-tenant results, with the repeated base-model forward removed.  The
reference therefore runs every sample through the backbone alone and every
tenant's head over its own samples alone (``isolated``), and, as a second
and independently arranged formulation used only to pin the first, runs
one packed batch with an explicit block-diagonal attention mask
(``packed_block_diagonal``).
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence, Tuple

import numpy as np

from . import backbone as bb
from . import heads as hd


def _sample_rows(wl, r: int, s: int) -> np.ndarray:
    req = wl.requests[r]
    return req.embeds[s, : int(req.lengths[s])]


def isolated(wl, samples: Optional[Sequence[Tuple[int, int]]] = None,
             heads: bool = True) -> Dict:
    """Per-sample hidden states and pooled features, per-tenant head results.

    ``samples``: (request, sample) pairs to run; default all.  Head results
    need every sample of a tenant, so they are computed only for tenants
    whose samples are all included.
    Returns {"hidden": {(r,s): z}, "pooled": {(r,s): p},
             "tenants": {g: tenant_step result}}.
    """
    spec = wl.spec
    b = spec.backbone
    if samples is None:
        samples = [(r, s) for r, req in enumerate(wl.requests) for s in range(req.n)]
    samples = list(samples)
    xs = [_sample_rows(wl, r, s) for r, s in samples]
    if wl.layers:
        getw = lambda l: wl.layers[l]  # noqa: E731
    else:
        import workloads
        getw = lambda l: workloads.layer_weights(spec, l)  # noqa: E731
    zs = bb.backbone_forward(xs, getw, b.layers, b.heads, b.glu, b.eps, wl.gf, b.kv_heads, b.causal,
                             b.rope_theta)
    hidden = dict(zip(samples, zs))
    pooled = {k: bb.pool(z) for k, z in hidden.items()}
    out = {"hidden": hidden, "pooled": pooled, "tenants": {}}
    if heads:
        have = set(samples)
        for g in range(spec.G):
            rows = [(r, s) for r, req in enumerate(wl.requests) if req.tenant == g for s in range(req.n)]
            if not rows or any(k not in have for k in rows):
                continue
            P = np.stack([pooled[k] for k in rows])
            out["tenants"][g] = tenant_from_pooled(wl, g, P)
    return out


def tenant_from_pooled(wl, g: int, P: np.ndarray) -> Dict:
    """Head forward, loss and grads of tenant g given its pooled rows in
    arrival order (used stage-wise with features produced elsewhere)."""
    import workloads
    tgt = workloads.tenant_targets(wl, g)
    return hd.tenant_step(np.asarray(P, np.float64), wl.heads[g], tgt)


def packed_block_diagonal(wl, align: int = 1) -> List[np.ndarray]:
    """Second formulation: one physical batch of all samples (rows in
    arrival order, each sample padded to a multiple of ``align`` with zero
    rows) run through the backbone with a block-diagonal key mask; returns
    the valid rows of each sample.  Used only to pin ``isolated``."""
    spec = wl.spec
    b = spec.backbone
    lens, blocks = [], []
    for req in wl.requests:
        for s in range(req.n):
            L = int(req.lengths[s])
            Lp = -(-L // align) * align
            x = np.zeros((Lp, b.d))
            x[:L] = bb.bf16_to_f64(req.embeds[s, :L])
            lens.append(L)
            blocks.append(x)
    seg = np.concatenate([np.full(x.shape[0], i) for i, x in enumerate(blocks)])
    pos = np.concatenate([np.arange(x.shape[0]) for x in blocks])
    valid_key = pos < np.array(lens)[seg]
    mask = (seg[:, None] == seg[None, :]) & valid_key[None, :]
    if b.causal:
        mask &= pos[None, :] <= pos[:, None]
    x = np.concatenate(blocks)
    d, H = b.d, b.heads
    hdim = d // H
    Hkv = b.kv_heads or H
    kvw = Hkv * hdim
    for l in range(b.layers):
        lw = bb.LayerF64(wl.layers[l], b.glu)
        h = bb.rms_norm(x, lw.g1, b.eps)
        qkv = h @ lw.wqkv.T
        q, k, v = qkv[:, :d], qkv[:, d:d + kvw], qkv[:, d + kvw:d + 2 * kvw]
        if b.rope_theta > 0:  # positions within each sample (the physical row index would be wrong)
            q = bb.rope(q, H, b.rope_theta, pos)
            k = bb.rope(k, Hkv, b.rope_theta, pos)
        a = np.empty((x.shape[0], d))
        for hh in range(H):
            sl = slice(hh * hdim, (hh + 1) * hdim)
            kl = slice((hh // (H // Hkv)) * hdim, (hh // (H // Hkv) + 1) * hdim)
            s = (q[:, sl] @ k[:, kl].T) / np.sqrt(hdim)
            s = np.where(mask, s, -np.inf)
            a[:, sl] = bb.softmax_rows(s) @ v[:, kl]
        x = x + a @ lw.wo.T
        h = bb.rms_norm(x, lw.g2, b.eps)
        m = bb.gelu(h @ lw.w_up.T) if lw.w_gate is None else bb.gelu(h @ lw.w_gate.T) * (h @ lw.w_up.T)
        x = x + m @ lw.w_down.T
    z = bb.rms_norm(x, bb.bf16_to_f64(wl.gf), b.eps)
    out, off = [], 0
    for L, blk in zip(lens, blocks):
        out.append(z[off: off + L])
        off += blk.shape[0]
    return out
