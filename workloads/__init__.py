"""Seeded synthetic inputs for the group-batched step.

This module only *draws inputs*: tenant schemas, per-sample token counts,
bf16 token embeddings, backbone and head weights, and regression targets.
It holds none of the method's arithmetic, so both the fp64 oracle and the
GPU path may read from it without sharing any compute code.

Every tensor has its own numpy ``PCG64`` stream, keyed by
``SeedSequence([seed, config_id, stream])``; a tensor's values therefore do
not depend on which other tensors were drawn or in which order, so the
oracle can regenerate a single layer and the generator can fill tensors
from several threads.

The five workload shapes stand in for the paper's LIBERO / CALVIN tenant
batches on StarVLA- and OpenPI-style models (Sec. 5.2); no dataset item or
model weight is reproduced.  bf16 values are carried as ``uint16`` bit
patterns (round-to-nearest-even from fp32 draws).
"""
from __future__ import annotations

import concurrent.futures as _cf
import dataclasses
import os
from typing import List, Optional, Sequence, Tuple

import numpy as np

__all__ = [
    "BackboneSpec", "TenantSpec", "WorkloadSpec", "Request", "Workload",
    "config_spec", "make_workload", "f32_to_bf16_bits", "bf16_bits_to_f32",
    "zipf_counts", "CONFIG_IDS",
]

CONFIG_IDS = (1, 2, 3, 4, 5)

# --------------------------------------------------------------------------
# bf16 bit-pattern helpers (input preparation only)
# --------------------------------------------------------------------------


def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round fp32 values to bf16, nearest-even, returned as uint16 bits."""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    lsb = (u >> np.uint32(16)) & np.uint32(1)
    return ((u + np.uint32(0x7FFF) + lsb) >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    """Exact widening of bf16 bit patterns to fp32."""
    return (np.asarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


# --------------------------------------------------------------------------
# specs
# --------------------------------------------------------------------------


@dataclasses.dataclass(frozen=True)
class BackboneSpec:
    layers: int
    d: int
    heads: int
    ffn: int
    glu: bool          # GeGLU MLP (gate and up projections) instead of GELU MLP
    eps: float = 1e-6  # RMSNorm epsilon
    kv_heads: int = 0  # key/value heads (0: one per query head; 1: multi-query; else grouped)
    causal: bool = False      # causal mask inside each sample instead of bidirectional
    rope_theta: float = 0.0   # > 0: rotary embedding of q and k, positions restart in every sample

    @property
    def head_dim(self) -> int:
        return self.d // self.heads

    @property
    def n_kv(self) -> int:
        return self.kv_heads or self.heads

    @property
    def qkv_rows(self) -> int:
        return (self.heads + 2 * self.n_kv) * self.head_dim


@dataclasses.dataclass(frozen=True)
class TenantSpec:
    n_samples: int
    img_tokens: int            # fixed image-patch tokens per sample
    text_lo: int               # text length drawn uniform on [text_lo, text_hi]
    text_hi: int
    max_len: int               # canonical padded length of this tenant's request rows
    head_dims: Tuple[int, ...]  # MLP head widths, input first, output (= action_dim*chunk) last
    action_dim: int
    chunk: int
    schema_sig: int = 0x4A4E5056_4C414631  # shared-prefix interface signature
    # action expert instead of an MLP head: (layers, d, heads, ffn); None = MLP head
    expert: Optional[Tuple[int, int, int, int]] = None


@dataclasses.dataclass(frozen=True)
class WorkloadSpec:
    config_id: int
    backbone: BackboneSpec
    tenants: Tuple[TenantSpec, ...]
    seed: int = 0
    name: str = ""
    # action-expert tenants trained with the flow-matching objective: width of
    # the sinusoidal flow-time features (0 = plain regression on the inputs)
    flow_time_dim: int = 0

    @property
    def G(self) -> int:
        return len(self.tenants)


@dataclasses.dataclass
class Request:
    """One tenant's request: ``n`` samples padded to ``max_len`` rows of width d."""
    tenant: int
    lengths: np.ndarray   # int32 [n], valid token count per sample
    embeds: np.ndarray    # uint16 (bf16 bits) [n, max_len, d]; rows >= length are filler
    first: int = 0        # index of this request's first sample within its tenant's submission

    @property
    def n(self) -> int:
        return int(self.lengths.shape[0])

    @property
    def max_len(self) -> int:
        return int(self.embeds.shape[1])


@dataclasses.dataclass
class Workload:
    spec: WorkloadSpec
    requests: List[Request]
    # backbone weights, bf16 bits, [out][in] layout; per layer a dict
    #   wqkv [(H + 2 Hkv) hd, d] (rows: q then k then v, head-major inside each),
    #   wo [d, d], w_up [f, d], w_gate [f, d] (GeGLU only), w_down [d, f],
    #   g1 [d], g2 [d]; plus final-norm gain gf [d]
    layers: List[dict]
    gf: np.ndarray
    # per tenant: list of (W fp32 [out, in], b fp32 [out]); GELU between layers
    heads: List[List[Tuple[np.ndarray, np.ndarray]]]
    # per tenant: fp32 [n_g, chunk, action_dim], rows in that tenant's submission order
    targets: List[np.ndarray]
    # per tenant (action-expert tenants only, else None): expert weights, noisy actions
    experts: List[Optional[dict]] = dataclasses.field(default_factory=list)
    noisy: List[Optional[np.ndarray]] = dataclasses.field(default_factory=list)
    # flow matching (flow_time_dim > 0): per tenant flow times [n] fp32; ``noisy``
    # then holds the noise, ``targets`` the clean actions, and each expert dict
    # a ``w_time`` [d][flow_time_dim]
    flow_t: List[Optional[np.ndarray]] = dataclasses.field(default_factory=list)


# --------------------------------------------------------------------------
# the five workloads
# --------------------------------------------------------------------------

_BB_SMALL = BackboneSpec(layers=2, d=128, heads=4, ffn=512, glu=False)
_BB_BASE = BackboneSpec(layers=12, d=768, heads=12, ffn=3072, glu=False)
_BB_2B = BackboneSpec(layers=18, d=2048, heads=8, ffn=16384, glu=True)
# Backbone variants on the 2B shapes: one key/value head and rotary positions
# over a bidirectional prefix (a Gemma-style prefix encoder), and grouped
# key/value heads with causal attention and rotary positions (a Qwen-style
# decoder used as the prefix encoder).
_BB_2B_MQA = BackboneSpec(layers=18, d=2048, heads=8, ffn=16384, glu=True, kv_heads=1, rope_theta=10000.0)
_BB_2B_GQA = BackboneSpec(layers=18, d=2048, heads=16, ffn=16384, glu=True, kv_heads=2, causal=True,
                          rope_theta=1000000.0)

# Config 3's eight tenants cover every action_dim in {7,14,32} and chunk in {1,10,50}.
_CFG3_SCHEMAS = ((7, 1), (7, 10), (7, 50), (14, 1), (14, 10), (14, 50), (32, 10), (32, 50))
_CFG25_SCHEMAS = ((7, 1), (7, 8), (14, 4), (32, 10))
# config 4's per-tenant action expert: 6 blocks, width 1024, 8 heads, MLP 4096
_EXPERT_300M = (6, 1024, 8, 4096)


def _rng(seed: int, cfg: int, stream: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence([seed, cfg, stream]))


# stream ids
_S_META = 1
_S_LEN = 10_000          # + request index
_S_EMB = 20_000          # + request index
_S_LAYER = 100_000       # + 16*layer + tensor index
_S_HEAD = 500_000        # + 16*tenant + layer
_S_TGT = 600_000         # + tenant
_S_EXP = 700_000         # + 64*tenant + tensor index
_S_NOISE = 900_000       # + tenant
_S_FLOW = 950_000        # + tenant: flow times
_S_TIME = 970_000        # + tenant: flow-time projection


def zipf_counts(total: int, n_ranks: int, s: float) -> List[int]:
    """Per-rank sample counts for a Zipf(s) split of ``total`` samples.

    Floors of ``total * w_k`` with ``w_k ~ k^-s``; the remainder goes to the
    largest fractional parts (ties to the lower rank); every rank gets >= 1.
    """
    w = np.array([k ** (-s) for k in range(1, n_ranks + 1)], dtype=np.float64)
    w /= w.sum()
    exact = total * w
    base = np.floor(exact).astype(np.int64)
    base = np.maximum(base, 1)
    rem = total - int(base.sum())
    frac = exact - np.floor(exact)
    order = sorted(range(n_ranks), key=lambda k: (-frac[k], k))
    i = 0
    while rem > 0:
        base[order[i % n_ranks]] += 1
        rem -= 1
        i += 1
    while rem < 0:  # only if the >=1 floor overshot: take from the largest ranks
        k = int(np.argmax(base))
        base[k] -= 1
        rem += 1
    return [int(c) for c in base]


def config_spec(cfg: int, seed: int = 0) -> WorkloadSpec:
    """Shapes of the five synthetic workloads (tenant metadata drawn from ``seed``)."""
    if cfg == 1:
        t = (
            TenantSpec(8, 16, 4, 16, 32, (128, 256, 7), 7, 1),
            TenantSpec(8, 16, 4, 16, 32, (128, 256, 56), 14, 4),
        )
        return WorkloadSpec(1, _BB_SMALL, t, seed, "tiny: 2 tenants x 8, 2-layer d128")
    if cfg == 2:
        t = tuple(TenantSpec(32, 196, 8, 48, 244, (768, 1024, a * c), a, c) for a, c in _CFG25_SCHEMAS)
        return WorkloadSpec(2, _BB_BASE, t, seed, "4 tenants x 32, 12-layer d768")
    if cfg == 3:
        t = tuple(TenantSpec(32, 256, 16, 64, 320, (2048, 1024, 1024, a * c), a, c) for a, c in _CFG3_SCHEMAS)
        return WorkloadSpec(3, _BB_2B, t, seed, "8 tenants x 32, 18-layer d2048 GeGLU (2B-shaped)")
    if cfg == 4:
        rng = _rng(seed, 4, _S_META)
        t = []
        for _ in range(16):
            cams = int(rng.integers(1, 4))
            n = int(rng.integers(4, 33))
            a = int(rng.choice([7, 14, 32]))
            t.append(TenantSpec(n, 256 * cams, 16, 96, 256 * cams + 96, (768, 1024, a * 50), a, 50,
                                expert=_EXPERT_300M))
        return WorkloadSpec(4, _BB_BASE, tuple(t), seed, "16 heterogeneous tenants, camera counts 1-3")
    if cfg == 5:
        rng = _rng(seed, 5, _S_META)
        counts = zipf_counts(512, 32, 1.2)
        perm = rng.permutation(32)
        per_tenant = [0] * 32
        for rank, tnt in enumerate(perm):
            per_tenant[int(tnt)] = counts[rank]
        t = []
        for g in range(32):
            cams = int(rng.integers(1, 4))
            a, c = _CFG25_SCHEMAS[int(rng.integers(0, 4))]
            t.append(TenantSpec(per_tenant[g], 256 * cams, 16, 64, 256 * cams + 64, (768, 1024, a * c), a, c))
        return WorkloadSpec(5, _BB_BASE, tuple(t), seed, "32 tenants, Zipf(1.2) counts totalling 512")
    if cfg in (6, 7):
        t = tuple(TenantSpec(32, 256, 16, 64, 320, (2048, 1024, 1024, a * c), a, c) for a, c in _CFG3_SCHEMAS)
        if cfg == 6:
            return WorkloadSpec(6, _BB_2B_MQA, t, seed, "8 tenants x 32, 2B-shaped, 1 KV head, RoPE, bidirectional")
        return WorkloadSpec(7, _BB_2B_GQA, t, seed, "8 tenants x 32, 2B-shaped, 16 heads / 2 KV heads, causal, RoPE")
    if cfg == 8:
        # the 16 heterogeneous tenants of config 4 (same draws), their experts
        # trained with the flow-matching objective
        return dataclasses.replace(config_spec(4, seed), flow_time_dim=1024,
                                   name="16 heterogeneous tenants, flow-matching action experts")
    raise ValueError(f"unknown config {cfg}")


# --------------------------------------------------------------------------
# drawing
# --------------------------------------------------------------------------


def _normal_bf16(rng: np.random.Generator, shape, std: float) -> np.ndarray:
    x = rng.standard_normal(shape, dtype=np.float32)
    if std != 1.0:
        x *= np.float32(std)
    return f32_to_bf16_bits(x)


def layer_weights(spec: WorkloadSpec, layer: int) -> dict:
    """bf16 weights of one backbone layer, ~N(0, 0.02); norm gains are 1."""
    bb = spec.backbone
    d, f = bb.d, bb.ffn

    def w(idx, shape):
        return _normal_bf16(_rng(spec.seed, spec.config_id, _S_LAYER + 16 * layer + idx), shape, 0.02)

    out = {
        "wqkv": w(0, (bb.qkv_rows, d)),
        "wo": w(1, (d, d)),
        "w_up": w(2, (f, d)),
        "w_down": w(4, (d, f)),
        "g1": f32_to_bf16_bits(np.ones(d, np.float32)),
        "g2": f32_to_bf16_bits(np.ones(d, np.float32)),
    }
    if bb.glu:
        out["w_gate"] = w(3, (f, d))
    return out


def draw_lengths(spec: WorkloadSpec, tenant: int) -> np.ndarray:
    t = spec.tenants[tenant]
    rng = _rng(spec.seed, spec.config_id, _S_LEN + tenant)
    txt = rng.integers(t.text_lo, t.text_hi + 1, size=t.n_samples)
    return (t.img_tokens + txt).astype(np.int32)


def draw_embeds(spec: WorkloadSpec, tenant: int) -> np.ndarray:
    """bf16 [n, max_len, d] ~N(0,1); rows past a sample's length are filler
    drawn from the same law, so any leak of padding into results shows."""
    t = spec.tenants[tenant]
    rng = _rng(spec.seed, spec.config_id, _S_EMB + tenant)
    return _normal_bf16(rng, (t.n_samples, t.max_len, spec.backbone.d), 1.0)


def head_weights(spec: WorkloadSpec, tenant: int) -> List[Tuple[np.ndarray, np.ndarray]]:
    """fp32 head layers: W ~ N(0, 1/in), b ~ N(0, 0.02)."""
    t = spec.tenants[tenant]
    out = []
    for k in range(len(t.head_dims) - 1):
        fin, fout = t.head_dims[k], t.head_dims[k + 1]
        rng = _rng(spec.seed, spec.config_id, _S_HEAD + 16 * tenant + k)
        W = (rng.standard_normal((fout, fin), dtype=np.float32) * np.float32(1.0 / np.sqrt(fin))).astype(np.float32)
        b = (rng.standard_normal(fout, dtype=np.float32) * np.float32(0.02)).astype(np.float32)
        out.append((W, b))
    return out


def expert_weights(spec: WorkloadSpec, tenant: int) -> dict:
    """bf16 action-expert weights ~N(0, 0.02), norm gains 1, [out][in] layout:
    w_in [d][a], w_out [a][d], gf [d]; per layer wqkv_s [3d][d], wo_s [d][d],
    wq_c [d][d], wkv_c [2d][dp] (keys then values, projected from the
    backbone's width dp), wo_c [d][d], w_up [f][d], w_down [d][f], g1..g3 [d]."""
    t = spec.tenants[tenant]
    L, d, _, f = t.expert
    dp, a = spec.backbone.d, t.action_dim
    k = [0]

    def w(shape):
        k[0] += 1
        rng = _rng(spec.seed, spec.config_id, _S_EXP + 64 * tenant + k[0])
        return _normal_bf16(rng, shape, 0.02)

    ones = f32_to_bf16_bits(np.ones(d, np.float32))
    out = {"w_in": w((d, a)), "w_out": w((a, d)), "gf": ones.copy(), "layers": []}
    for _ in range(L):
        out["layers"].append({"wqkv_s": w((3 * d, d)), "wo_s": w((d, d)), "wq_c": w((d, d)),
                              "wkv_c": w((2 * d, dp)), "wo_c": w((d, d)), "w_up": w((f, d)),
                              "w_down": w((d, f)), "g1": ones.copy(), "g2": ones.copy(), "g3": ones.copy()})
    return out


def draw_noisy_actions(spec: WorkloadSpec, tenant: int) -> np.ndarray:
    """fp32 [n, chunk, action_dim] ~N(0,1): the expert's input action tokens."""
    t = spec.tenants[tenant]
    rng = _rng(spec.seed, spec.config_id, _S_NOISE + tenant)
    return rng.standard_normal((t.n_samples, t.chunk, t.action_dim), dtype=np.float32)


def draw_flow_times(spec: WorkloadSpec, tenant: int) -> np.ndarray:
    """fp32 [n]: flow times 0.001 + 0.999 * Beta(1.5, 1), one per sample."""
    t = spec.tenants[tenant]
    rng = _rng(spec.seed, spec.config_id, _S_FLOW + tenant)
    return (0.001 + 0.999 * rng.beta(1.5, 1.0, size=t.n_samples)).astype(np.float32)


def time_weights(spec: WorkloadSpec, tenant: int) -> np.ndarray:
    """bf16 [d][flow_time_dim] ~N(0, 0.02): the flow-time projection."""
    d = spec.tenants[tenant].expert[1]
    return _normal_bf16(_rng(spec.seed, spec.config_id, _S_TIME + tenant), (d, spec.flow_time_dim), 0.02)


def draw_targets(spec: WorkloadSpec, tenant: int) -> np.ndarray:
    t = spec.tenants[tenant]
    rng = _rng(spec.seed, spec.config_id, _S_TGT + tenant)
    return rng.standard_normal((t.n_samples, t.chunk, t.action_dim), dtype=np.float32)


def _threads() -> int:
    return max(1, min(16, os.cpu_count() or 1))


def make_workload(spec_or_cfg, seed: int = 0, with_weights: bool = True,
                  request_split: Optional[Sequence[int]] = None,
                  request_order: Optional[Sequence[int]] = None) -> Workload:
    """Draw every input of a workload.

    By default each tenant submits one request.  ``request_split[g] = k``
    cuts tenant g's samples into k contiguous requests; ``request_order``
    permutes the resulting request list (arrival order), e.g. to interleave
    tenants.
    """
    spec = spec_or_cfg if isinstance(spec_or_cfg, WorkloadSpec) else config_spec(int(spec_or_cfg), seed)
    G = spec.G
    with _cf.ThreadPoolExecutor(_threads()) as ex:
        lens = [draw_lengths(spec, g) for g in range(G)]
        emb_f = [ex.submit(draw_embeds, spec, g) for g in range(G)]
        lay_f = [ex.submit(layer_weights, spec, l) for l in range(spec.backbone.layers)] if with_weights else []
        embeds = [f.result() for f in emb_f]
        layers = [f.result() for f in lay_f]
    requests: List[Request] = []
    for g in range(G):
        k = 1 if request_split is None else int(request_split[g])
        cuts = np.linspace(0, spec.tenants[g].n_samples, k + 1).round().astype(int)
        for a, b in zip(cuts[:-1], cuts[1:]):
            if b > a:
                requests.append(Request(g, lens[g][a:b].copy(), embeds[g][a:b], int(a)))
    if request_order is not None:
        requests = [requests[i] for i in request_order]
    gf = f32_to_bf16_bits(np.ones(spec.backbone.d, np.float32))
    heads = [head_weights(spec, g) if spec.tenants[g].expert is None else None for g in range(G)]
    targets = [draw_targets(spec, g) for g in range(G)]
    experts = [expert_weights(spec, g) if spec.tenants[g].expert is not None else None for g in range(G)]
    noisy = [draw_noisy_actions(spec, g) if spec.tenants[g].expert is not None else None for g in range(G)]
    flow = spec.flow_time_dim > 0
    flow_t = [draw_flow_times(spec, g) if flow and spec.tenants[g].expert is not None else None for g in range(G)]
    if flow:
        for g in range(G):
            if experts[g] is not None:
                experts[g]["w_time"] = time_weights(spec, g)
    return Workload(spec, requests, layers, gf, heads, targets, experts, noisy, flow_t)


def tenant_rows(wl: Workload, tenant: int) -> List[Tuple[int, int]]:
    """(request index, sample index) pairs of a tenant, in arrival order."""
    out = []
    for r, req in enumerate(wl.requests):
        if req.tenant == tenant:
            out.extend((r, s) for s in range(req.n))
    return out


def tenant_rows_of(wl: Workload, tenant: int, arr: np.ndarray) -> np.ndarray:
    """Rows of a per-tenant array (submission order) in arrival order."""
    idx = []
    for req in wl.requests:
        if req.tenant == tenant:
            idx.extend(range(req.first, req.first + req.n))
    return arr[np.array(idx, dtype=np.int64)]


def tenant_targets(wl: Workload, tenant: int) -> np.ndarray:
    """Targets of ``tenant`` in the order its samples arrive in ``wl.requests``."""
    idx = []
    for req in wl.requests:
        if req.tenant == tenant:
            idx.extend(range(req.first, req.first + req.n))
    return wl.targets[tenant][np.array(idx, dtype=np.int64)]
