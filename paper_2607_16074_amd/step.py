"""The group-batched step as four library calls, with caller-owned buffers.

``GroupStep`` holds the device copies of the frozen backbone and of every
tenant's head, allocates the buffers a given group of requests needs once
(``prepare``), and then runs

    jn_pack_group -> jn_backbone_forward -> jn_tenant_heads_fwd_bwd -> jn_unpack

(``jn_tenant_experts_fwd_bwd`` in place of the heads call when the group's
tenants carry action experts)

on one stream (``run``) with no allocation and no host synchronisation.
``InferStep`` is the inference-side counterpart: one physical batch made
resident by ``jn_infer_plan_create`` (pack, shared encode, split, forward-only
decode), launched eagerly or replayed as a captured HIP graph.
``isolated_runs`` builds one such step per tenant over the same device
weights: the serial-execution comparator of grouped execution, using the
same kernels and the same tile rule.
"""
from __future__ import annotations

from typing import Dict, List, Optional, Sequence

import numpy as np

from . import (EXPERT_LAYER_FIELDS, AdamWTenant, Backbone, Context, Expert, ExpertIO, Head, HeadIO, InferPlan,
               Request, Tenant, jn_adamw_workspace_size, jn_infer_workspace_size, jn_backbone_forward, jn_backbone_workspace_size, jn_experts_workspace_size,
               jn_heads_workspace_size, jn_pack_group, jn_pack_plan, jn_pack_tenant_sizes, jn_tenant_adamw_step,
               jn_tenant_experts_fwd_bwd, jn_tenant_heads_fwd_bwd, jn_unpack)


def _dev_bf16(bits: np.ndarray, device):
    import torch
    t = torch.from_numpy(np.ascontiguousarray(bits).view(np.int16))
    return t.to(device, non_blocking=False).view(torch.bfloat16)


def _dev_f32(a: np.ndarray, device):
    import torch
    return torch.from_numpy(np.ascontiguousarray(a, dtype=np.float32)).to(device)


class Model:
    """Device weights: frozen backbone + per-tenant heads or action experts."""

    def __init__(self, backbone: Backbone, heads: List[Optional[Head]], tenant_meta: List[dict], prefix_sig: int,
                 experts: Optional[List[Optional[Expert]]] = None):
        self.backbone = backbone
        self.heads = heads
        self.experts = experts or [None] * len(heads)
        self.tenant_meta = tenant_meta  # action_dim, chunk per tenant
        self.prefix_sig = prefix_sig

    @classmethod
    def from_arrays(cls, layers: List[dict], gf: np.ndarray, n_heads: int, eps: float,
                    heads: List[Optional[list]], tenant_meta: List[dict], prefix_sig: int, device="cuda",
                    experts: Optional[List[Optional[dict]]] = None, n_kv_heads: int = 0, causal: bool = False,
                    rope_theta: float = 0.0):
        """``layers``: per layer dict of bf16 bit arrays; ``heads``: per tenant
        list of (W fp32 [out,in], b fp32 [out]) or None; ``experts``: per
        tenant None or a dict of bf16 bit arrays (w_in, w_out, gf, layers)
        with ``tenant_meta[g]["expert_heads"]`` attention heads."""
        dl = [{k: _dev_bf16(v, device) for k, v in L.items()} for L in layers]
        bb = Backbone(dl, _dev_bf16(gf, device), n_heads, eps, n_kv_heads, causal, rope_theta)
        hs, xs = [], []
        for g, layers_g in enumerate(heads):
            if layers_g is None:
                hs.append(None)
            else:
                W = [_dev_f32(w, device) for w, _ in layers_g]
                b = [_dev_f32(x, device) for _, x in layers_g]
                hs.append(Head(W, b, tenant_meta[g]["action_dim"], tenant_meta[g]["chunk"]))
            e = experts[g] if experts is not None else None
            if e is None:
                xs.append(None)
            else:
                xl = [{k: _dev_bf16(v, device) for k, v in L.items()} for L in e["layers"]]
                xs.append(Expert(_dev_bf16(e["w_in"], device), _dev_bf16(e["w_out"], device),
                                 _dev_bf16(e["gf"], device), xl, tenant_meta[g]["expert_heads"],
                                 tenant_meta[g]["chunk"], bb.d, eps,
                                 _dev_bf16(e["w_time"], device) if "w_time" in e else None))
        return cls(bb, hs, tenant_meta, prefix_sig, xs)


class GroupStep:
    """One group of requests over a subset of tenants, buffers allocated once."""

    def __init__(self, model: Model, requests: Sequence[Request], targets: Dict[int, np.ndarray],
                 tenants: Sequence[int], align: int = 1, ctx: Optional[Context] = None, device="cuda",
                 noisy: Optional[Dict[int, np.ndarray]] = None, flow_t: Optional[Dict[int, np.ndarray]] = None):
        import torch
        self.model = model
        self.ctx = ctx or Context()
        self.tenants = list(tenants)              # global tenant ids, table order
        slot = {g: k for k, g in enumerate(self.tenants)}
        # requests re-labelled to table slots
        self.requests = [Request(slot[r.tenant], r.embeds, r.lengths, r.max_len) for r in requests]
        self.align = align
        d = model.backbone.d
        self.table = [Tenant(model.prefix_sig, d) for _ in self.tenants]
        sz = jn_pack_plan(self.requests, self.table, d, align)
        self.N, self.T = sz.N, sz.T
        self.maps = torch.empty(int(sz.map_bytes), dtype=torch.uint8, device=device)
        self.tokens = torch.empty((self.T, d), dtype=torch.bfloat16, device=device)
        self.hidden = torch.empty((self.T, d), dtype=torch.bfloat16, device=device)
        self.bb_ws = torch.empty(jn_backbone_workspace_size(model.backbone, self.T), dtype=torch.uint8, device=device)
        self.experts = [model.experts[g] for g in self.tenants]
        self.use_experts = self.experts[0] is not None
        if any((x is not None) != self.use_experts for x in self.experts):
            raise ValueError("a group mixes expert tenants with MLP-head tenants")
        self.heads = [model.heads[g] for g in self.tenants]
        self.pooled = torch.empty((self.N, d), dtype=torch.float32, device=device)
        self.out_hidden = [torch.empty((r.n, r.max_len, d), dtype=torch.bfloat16, device=device) for r in self.requests]
        # pack once to size the tenant-stage workspace from a real packed batch
        self.packed = jn_pack_group(self.ctx, self.requests, self.table, d, align, self.maps, self.tokens)
        self.ios = []
        if self.use_experts:
            n_s, rows = jn_pack_tenant_sizes(self.requests, self.table, d, align)
            for k, g in enumerate(self.tenants):
                e = model.experts[g]
                w_in, w_out, gf, xl = e.w_in, e.w_out, e.gf, e.layers
                f32 = lambda t: torch.empty(t.shape, dtype=torch.float32, device=device)  # noqa: E731
                shape = (int(n_s[k]), e.struct.chunk, e.struct.action_dim)
                self.ios.append(ExpertIO(int(n_s[k]), int(rows[k]), _dev_f32(noisy[g], device).reshape(shape),
                                         _dev_f32(targets[g], device).reshape(shape),
                                         torch.empty(shape, dtype=torch.float32, device=device),
                                         torch.empty(1, dtype=torch.float32, device=device),
                                         f32(w_in), f32(w_out), f32(gf),
                                         [{k2: f32(L[k2]) for k2 in EXPERT_LAYER_FIELDS} for L in xl],
                                         _dev_f32(flow_t[g], device) if e.w_time is not None else None,
                                         f32(e.w_time) if e.w_time is not None else None))
            self.hd_ws = torch.empty(jn_experts_workspace_size(self.packed, self.experts, self.ios), dtype=torch.uint8,
                                     device=device)
        else:
            for k, g in enumerate(self.tenants):
                h = model.heads[g]
                n_g = int(sum(r.n for r in self.requests if r.tenant == k))
                tgt = _dev_f32(targets[g], device)
                acts = torch.empty((n_g, int(h.dims[-1])), dtype=torch.float32, device=device)
                loss = torch.empty(1, dtype=torch.float32, device=device)
                dW = [torch.empty_like(w) for w in h.W]
                db = [torch.empty_like(x) for x in h.b]
                self.ios.append(HeadIO(tgt, acts, loss, dW, db))
            self.hd_ws = torch.empty(jn_heads_workspace_size(self.packed, self.heads), dtype=torch.uint8,
                                     device=device)
        self.valid_tokens = int(sum(int(r.lengths.sum()) for r in self.requests))

    # the four calls -------------------------------------------------------
    def pack(self):
        d = self.model.backbone.d
        self.packed = jn_pack_group(self.ctx, self.requests, self.table, d, self.align, self.maps, self.tokens)

    def backbone(self):
        jn_backbone_forward(self.ctx, self.model.backbone, self.packed, self.hidden, self.bb_ws)

    def heads_fwd_bwd(self):
        if self.use_experts:
            jn_tenant_experts_fwd_bwd(self.ctx, self.packed, self.hidden, self.experts, self.ios, self.hd_ws)
        else:
            jn_tenant_heads_fwd_bwd(self.ctx, self.packed, self.hidden, self.heads, self.ios, self.hd_ws,
                                    self.pooled)

    def unpack(self):
        d = self.model.backbone.d
        jn_unpack(self.ctx, self.packed, self.requests, self.hidden, d * 2, self.out_hidden)

    def run(self):
        self.pack()
        self.backbone()
        self.heads_fwd_bwd()
        self.unpack()


class InferStep:
    """A resident decode-only step over one group of requests on a stream of
    its own (graph capture needs a non-null stream): ``launch`` enqueues the
    kernels, ``capture`` records one launch into a HIP graph, ``replay``
    launches that graph.  ``actions[k]`` is tenant ``tenants[k]``'s output,
    rows in its arrival order."""

    def __init__(self, model: Model, requests: Sequence[Request], tenants: Sequence[int], align: int = 1,
                 device="cuda", stream=None):
        import torch
        self.model = model
        self.stream = stream if stream is not None else torch.cuda.Stream(device=device)
        self.ctx = Context(self.stream)
        self.tenants = list(tenants)
        slot = {g: k for k, g in enumerate(self.tenants)}
        self.requests = [Request(slot[r.tenant], r.embeds, r.lengths, r.max_len) for r in requests]
        d = model.backbone.d
        self.table = [Tenant(model.prefix_sig, d) for _ in self.tenants]
        self.heads = [model.heads[g] for g in self.tenants]
        if any(h is None for h in self.heads):
            raise ValueError("InferStep serves MLP-head tenants")
        self.actions = [torch.empty((int(sum(r.n for r in self.requests if r.tenant == k)), int(h.dims[-1])),
                                    dtype=torch.float32, device=device) for k, h in enumerate(self.heads)]
        nbytes = jn_infer_workspace_size(self.requests, self.table, d, align, model.backbone, self.heads)
        self.ws = torch.empty(nbytes, dtype=torch.uint8, device=device)
        torch.cuda.synchronize()
        self.plan = InferPlan(self.ctx, self.requests, self.table, d, align, model.backbone, self.heads,
                              self.actions, self.ws)

    def launch(self):
        self.plan.launch()

    def capture(self):
        self.plan.capture()

    def replay(self):
        self.plan.replay()

    def synchronize(self):
        self.stream.synchronize()


class TenantOptimizer:
    """Per-tenant AdamW over the tenants of one ``GroupStep``: after the
    group's tenant stage, ``step()`` updates every tenant's own parameters
    from its own gradients in one launch and advances only those tenants'
    versions.  MLP heads are updated in place (fp32); an action expert keeps
    fp32 master weights here and its bf16 weights receive the rounded update.
    Moments start at zero."""

    def __init__(self, group: "GroupStep", lr: float = 1e-4, betas=(0.9, 0.999), eps: float = 1e-8,
                 weight_decay: float = 0.0):
        import torch
        self.group = group
        self.hyper = dict(lr=lr, beta1=betas[0], beta2=betas[1], eps=eps, weight_decay=weight_decay)
        self.versions = {g: 0 for g in group.tenants}
        self.sets = []   # per tenant: (params, grads, bf16 copies or None)
        for k, g in enumerate(group.tenants):
            if group.use_experts:
                e, io = group.experts[k], group.ios[k]
                pairs = [(e.w_in, io.dw_in), (e.w_out, io.dw_out), (e.gf, io.dgf)]
                if e.w_time is not None:
                    pairs.append((e.w_time, io.dw_time))
                for L, Lg in zip(e.layers, io.layers):
                    pairs += [(L[n], Lg[n]) for n in EXPERT_LAYER_FIELDS]
                masters = [w.float().contiguous() for w, _ in pairs]
                self.sets.append((masters, [gr for _, gr in pairs], [w for w, _ in pairs]))
            else:
                h, io = group.heads[k], group.ios[k]
                self.sets.append((list(h.W) + list(h.b), list(io.dW) + list(io.db), None))
        self.m = [[torch.zeros_like(p) for p in ps] for ps, _, _ in self.sets]
        self.v = [[torch.zeros_like(p) for p in ps] for ps, _, _ in self.sets]
        self.ws = torch.empty(jn_adamw_workspace_size(self._tenants(1)), dtype=torch.uint8, device=group.tokens.device)

    def _tenants(self, bump: int):
        out = []
        for k, g in enumerate(self.group.tenants):
            ps, gs, b16 = self.sets[k]
            out.append(AdamWTenant(ps, gs, self.m[k], self.v[k], self.versions[g] + bump, bf16_out=b16, **self.hyper))
        return out

    def step(self):
        ten = self._tenants(1)
        jn_tenant_adamw_step(self.group.ctx, ten, self.ws)
        for g in self.group.tenants:
            self.versions[g] += 1


def isolated_runs(model: Model, requests: Sequence[Request], targets: Dict[int, np.ndarray],
                  tenants: Sequence[int], align: int = 1, ctx: Optional[Context] = None, device="cuda",
                  noisy: Optional[Dict[int, np.ndarray]] = None, flow_t: Optional[Dict[int, np.ndarray]] = None):
    """One ``GroupStep`` per tenant (its own requests only), sharing the weights."""
    ctx = ctx or Context()
    out = []
    for g in tenants:
        reqs = [r for r in requests if r.tenant == g]
        out.append(GroupStep(model, reqs, targets, [g], align, ctx, device, noisy, flow_t))
    return out


def from_workload(wl, device="cuda", with_noisy: bool = False):
    """Device model, requests and targets from a workload description.

    ``wl`` needs: ``spec`` (backbone: layers/d/heads/eps; tenants: action_dim,
    chunk, schema_sig), ``layers``, ``gf``, ``heads``, ``targets`` and
    ``requests`` (tenant, lengths, embeds bf16 bits, first); for action-expert
    tenants also ``experts`` and ``noisy``.  ``with_noisy`` adds a fourth
    result: every expert tenant's noisy action tokens in arrival order.
    """
    spec = wl.spec
    meta = [{"action_dim": t.action_dim, "chunk": t.chunk,
             "expert_heads": t.expert[2] if t.expert is not None else 0} for t in spec.tenants]
    b = spec.backbone
    model = Model.from_arrays(wl.layers, wl.gf, b.heads, b.eps, wl.heads, meta, spec.tenants[0].schema_sig, device,
                              getattr(wl, "experts", None), b.kv_heads, b.causal, b.rope_theta)
    reqs = [Request(r.tenant, _dev_bf16(r.embeds, device), r.lengths) for r in wl.requests]
    targets, noisy = {}, {}
    for g in range(spec.G):
        idx = np.array([k for r in wl.requests if r.tenant == g for k in range(r.first, r.first + r.n)],
                       dtype=np.int64)
        t = np.asarray(wl.targets[g], np.float32)[idx]
        if spec.tenants[g].expert is None:
            targets[g] = t.reshape(len(idx), -1)
        else:
            targets[g] = t
            noisy[g] = np.asarray(wl.noisy[g], np.float32)[idx]
    if with_noisy:
        return model, reqs, targets, noisy
    return model, reqs, targets


def flow_times(wl) -> Optional[Dict[int, np.ndarray]]:
    """Flow times of every flow-matching expert tenant in arrival order, or
    None when the workload trains its experts by plain regression."""
    ft = getattr(wl, "flow_t", None)
    if not ft or all(x is None for x in ft):
        return None
    out = {}
    for g, x in enumerate(ft):
        if x is not None:
            idx = [i for r in wl.requests if r.tenant == g for i in range(r.first, r.first + r.n)]
            out[g] = np.asarray(x, np.float32)[np.array(idx, dtype=np.int64)]
    return out
