"""MI355X (gfx950) group-batched step of JoyNexus multi-tenant group batching.

Thin Python binding of ``libjoynexus.so`` (C ABI in ``include/joynexus.h``):
the functions below carry the C names and only marshal arguments -- every
step of the path runs in the library's HIP kernels.  PyTorch supplies device
memory and streams.  Importing this package fails if the library is not
built; there is no fallback implementation.
"""
from __future__ import annotations

import ctypes as C
from typing import List, Optional, Sequence

import numpy as np

from . import _abi
from ._abi import (EXPERT_LAYER_FIELDS, JN_OK, STATUS_NAMES, jn_adamw_tenant, jn_backbone, jn_expert, jn_expert_io,
                   jn_expert_layer, jn_expert_layer_grads, jn_head, jn_head_io, jn_layer, jn_pack_opts,
                   jn_pack_sizes, jn_packed, jn_request, jn_tenant)

_lib = _abi.load()

__all__ = [
    "JNError", "Context", "Request", "Tenant", "Backbone", "Head", "HeadIO",
    "jn_pack_plan", "jn_pack_maps_host", "jn_pack_group", "jn_backbone_workspace_size",
    "jn_backbone_forward", "jn_heads_workspace_size", "jn_tenant_heads_fwd_bwd", "jn_tenant_heads_fwd_bwd_noalloc",
    "HEADS_SCRATCH_BYTES", "jn_unpack",
    "Expert", "ExpertIO", "jn_pack_tenant_sizes", "jn_experts_workspace_size", "jn_tenant_experts_fwd_bwd",
    "AdamWTenant", "jn_adamw_workspace_size", "jn_tenant_adamw_step",
    "Collector", "InferPlan", "jn_infer_workspace_size",
    "lib_path",
]


def lib_path() -> str:
    return _abi.LIB_PATH


class JNError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {msg}")
        self.status = status


def _check(st: int, ctx: "Context" = None, what: str = ""):
    if st != JN_OK:
        msg = _lib.jn_last_error(ctx.handle).decode() if ctx is not None else what
        raise JNError(st, msg or what)


def _ptr(t) -> int:
    """Device pointer of a torch tensor (or an int)."""
    if t is None:
        return None
    return t if isinstance(t, int) else t.data_ptr()


class Context:
    """A library context bound to a HIP stream (default: torch's current stream)."""

    def __init__(self, stream=None):
        import torch
        if stream is None:
            stream = torch.cuda.current_stream()
        self.stream = stream
        h = C.c_void_p()
        _check(_lib.jn_ctx_create(C.byref(h), C.c_void_p(stream.cuda_stream)), what="jn_ctx_create")
        self.handle = h

    def set_trace(self, enable: bool):
        """Bracket every kernel this context launches with timing events."""
        _check(_lib.jn_ctx_set_trace(self.handle, 1 if enable else 0), self)

    def set_option(self, option: int, value: int):
        """jn_ctx_set_option: e.g. ``_abi.JN_OPT_EXPERT_TRANSPOSES``."""
        _check(_lib.jn_ctx_set_option(self.handle, int(option), int(value)), self)

    def trace_read(self, cap: int = 1 << 16) -> list:
        """[(op name, M, N, K, ms)] of the traced launches, in launch order."""
        buf = (_abi.jn_trace_entry * cap)()
        n = C.c_int32()
        _check(_lib.jn_ctx_trace_read(self.handle, buf, cap, C.byref(n)), self)
        return [(_abi.OPS.get(e.op, str(e.op)), e.M, e.N, e.K, e.ms) for e in buf[: n.value]]

    def close(self):
        if self.handle:
            _lib.jn_ctx_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


# ---------------------------------------------------------------- marshal ---

class Request:
    """A tenant request: ``embeds`` device bf16 [n, max_len, d], host lengths."""

    def __init__(self, tenant: int, embeds, lengths, max_len: int = None):
        self.tenant = int(tenant)
        self.embeds = embeds
        self.lengths = np.ascontiguousarray(lengths, dtype=np.int32)
        self.n = int(self.lengths.shape[0])
        self.max_len = int(max_len) if max_len is not None else int(embeds.shape[1])


class Tenant:
    def __init__(self, prefix_sig: int, d_model: int):
        self.prefix_sig = int(prefix_sig)
        self.d_model = int(d_model)


def _requests(reqs: Sequence[Request]):
    arr = (jn_request * len(reqs))()
    keep = []
    for i, r in enumerate(reqs):
        lens = r.lengths
        keep.append(lens)
        arr[i].tenant = r.tenant
        arr[i].n_samples = r.n
        arr[i].max_len = r.max_len
        arr[i].embeds = _ptr(r.embeds) if r.embeds is not None else None
        arr[i].lengths = lens.ctypes.data_as(C.POINTER(C.c_int32))
    return arr, keep


def _tenants(ten: Sequence[Tenant]):
    arr = (jn_tenant * len(ten))()
    for i, t in enumerate(ten):
        arr[i].prefix_sig = t.prefix_sig
        arr[i].d_model = t.d_model
    return arr


def _opts(d: int, align: int):
    o = jn_pack_opts()
    o.d_model = d
    o.align = align
    return o


# ---------------------------------------------------------------- pack ------

def jn_pack_plan(reqs: Sequence[Request], tenants: Sequence[Tenant], d: int, align: int = 1) -> jn_pack_sizes:
    ra, keep = _requests(reqs)
    ta = _tenants(tenants)
    out = jn_pack_sizes()
    o = _opts(d, align)
    _check(_lib.jn_pack_plan(ra, len(reqs), ta, len(tenants), C.byref(o), C.byref(out)), what="jn_pack_plan")
    return out


def jn_pack_maps_host(reqs: Sequence[Request], tenants: Sequence[Tenant], d: int, align: int = 1) -> dict:
    """Index maps computed on the host by the library (numpy int32 arrays)."""
    sz = jn_pack_plan(reqs, tenants, d, align)
    buf = np.zeros(int(sz.map_bytes), dtype=np.uint8)
    ra, keep = _requests(reqs)
    ta = _tenants(tenants)
    out = jn_packed()
    o = _opts(d, align)
    _check(_lib.jn_pack_maps_host(ra, len(reqs), ta, len(tenants), C.byref(o),
                                  buf.ctypes.data_as(C.c_void_p), buf.nbytes, C.byref(out)), what="jn_pack_maps_host")
    base = buf.ctypes.data
    res = {"N": out.N, "T": out.T, "max_seqlen": out.max_seqlen, "req_sig": out.req_sig}
    for name in jn_packed.MAP_FIELDS:
        off = C.cast(getattr(out, name), C.c_void_p).value - base
        res[name] = buf[off: off + 4 * out.map_len(name)].view(np.int32).copy()
    return res


class Packed:
    """A packed batch: the C struct plus the tensors it points into."""

    def __init__(self, struct: jn_packed, maps, tokens):
        self.struct = struct
        self.maps = maps
        self.tokens = tokens

    def __getattr__(self, k):
        return getattr(self.struct, k)

    def map_tensor(self, name: str):
        """View of one device index map as an int32 tensor."""
        import torch
        off = C.cast(getattr(self.struct, name), C.c_void_p).value - self.maps.data_ptr()
        n = self.struct.map_len(name)
        return self.maps[off: off + 4 * n].view(torch.int32)


def jn_pack_group(ctx: Context, reqs: Sequence[Request], tenants: Sequence[Tenant], d: int, align: int,
                  maps, tokens) -> Packed:
    ra, keep = _requests(reqs)
    ta = _tenants(tenants)
    out = jn_packed()
    o = _opts(d, align)
    _check(_lib.jn_pack_group(ctx.handle, ra, len(reqs), ta, len(tenants), C.byref(o), _ptr(maps),
                              maps.numel() * maps.element_size(), _ptr(tokens),
                              tokens.numel() * tokens.element_size(), C.byref(out)), ctx)
    return Packed(out, maps, tokens)


# ------------------------------------------------------------ backbone ------

class Backbone:
    """Device weights of the frozen backbone (lists of torch bf16 tensors)."""

    def __init__(self, layers: List[dict], gf, n_heads: int, eps: float, n_kv_heads: int = 0, causal: bool = False,
                 rope_theta: float = 0.0):
        self.layers = layers
        self.gf = gf
        self.n_heads = int(n_heads)
        self.n_kv_heads = int(n_kv_heads)
        self.causal = bool(causal)
        self.rope_theta = float(rope_theta)
        self.eps = float(eps)
        self.d = int(gf.shape[0])
        self.ffn = int(layers[0]["w_up"].shape[0])
        arr = (jn_layer * len(layers))()
        for i, L in enumerate(layers):
            arr[i].wqkv = _ptr(L["wqkv"])
            arr[i].wo = _ptr(L["wo"])
            arr[i].w_up = _ptr(L["w_up"])
            arr[i].w_gate = _ptr(L.get("w_gate"))
            arr[i].w_down = _ptr(L["w_down"])
            arr[i].g1 = _ptr(L["g1"])
            arr[i].g2 = _ptr(L["g2"])
        self._arr = arr
        s = jn_backbone()
        s.n_layers = len(layers)
        s.d = self.d
        s.n_heads = self.n_heads
        s.ffn = self.ffn
        s.eps = self.eps
        s.n_kv_heads = self.n_kv_heads
        s.causal = 1 if self.causal else 0
        s.rope_theta = self.rope_theta
        s.layers = C.cast(arr, C.POINTER(jn_layer))
        s.gf = _ptr(gf)
        self.struct = s


def jn_backbone_workspace_size(bb: Backbone, T: int) -> int:
    n = C.c_size_t()
    _check(_lib.jn_backbone_workspace_size(C.byref(bb.struct), T, C.byref(n)), what="jn_backbone_workspace_size")
    return int(n.value)


def jn_backbone_forward(ctx: Context, bb: Backbone, packed: Packed, hidden, ws):
    _check(_lib.jn_backbone_forward(ctx.handle, C.byref(bb.struct), C.byref(packed.struct), _ptr(hidden),
                                    _ptr(ws), ws.numel() * ws.element_size()), ctx)


# --------------------------------------------------------------- heads ------

class Head:
    """A tenant's MLP head: lists of device fp32 W [out, in] and b [out]."""

    def __init__(self, W: list, b: list, action_dim: int, chunk: int):
        self.W, self.b = W, b
        self.dims = np.array([int(W[0].shape[1])] + [int(w.shape[0]) for w in W], dtype=np.int32)
        s = jn_head()
        s.n_layers = len(W)
        s.action_dim = int(action_dim)
        s.chunk = int(chunk)
        self._W = (C.c_void_p * len(W))(*[_ptr(w) for w in W])
        self._b = (C.c_void_p * len(b))(*[_ptr(x) for x in b])
        s.dims = self.dims.ctypes.data_as(C.POINTER(C.c_int32))
        s.W = C.cast(self._W, C.POINTER(C.c_void_p))
        s.b = C.cast(self._b, C.POINTER(C.c_void_p))
        self.struct = s


class HeadIO:
    """A tenant's targets and outputs (device fp32 tensors)."""

    def __init__(self, targets, actions, loss, dW: list, db: list):
        self.targets, self.actions, self.loss, self.dW, self.db = targets, actions, loss, dW, db
        s = jn_head_io()
        s.targets = _ptr(targets)
        s.actions = _ptr(actions)
        s.loss = _ptr(loss)
        self._dW = (C.c_void_p * len(dW))(*[_ptr(w) for w in dW])
        self._db = (C.c_void_p * len(db))(*[_ptr(x) for x in db])
        s.dW = C.cast(self._dW, C.POINTER(C.c_void_p))
        s.db = C.cast(self._db, C.POINTER(C.c_void_p))
        self.struct = s


def _head_arrays(heads: Sequence[Head], ios: Sequence[HeadIO] = None):
    ha = (jn_head * len(heads))(*[h.struct for h in heads])
    ia = (jn_head_io * len(ios))(*[x.struct for x in ios]) if ios is not None else None
    return ha, ia


def jn_heads_workspace_size(packed: Packed, heads: Sequence[Head]) -> int:
    ha, _ = _head_arrays(heads)
    n = C.c_size_t()
    _check(_lib.jn_heads_workspace_size(C.byref(packed.struct), ha, len(heads), C.byref(n)),
           what="jn_heads_workspace_size")
    return int(n.value)


def jn_tenant_heads_fwd_bwd(ctx: Context, packed: Packed, hidden, heads: Sequence[Head], ios: Sequence[HeadIO],
                            ws, pooled=None):
    ha, ia = _head_arrays(heads, ios)
    _check(_lib.jn_tenant_heads_fwd_bwd(ctx.handle, C.byref(packed.struct), _ptr(hidden), ha, ia, len(heads),
                                        _ptr(ws), ws.numel() * ws.element_size(), _ptr(pooled)), ctx)


# Size of the library-owned workspace of the allocation-free heads call
# (JN_HEADS_SCRATCH_BYTES in joynexus.h).
HEADS_SCRATCH_BYTES = 64 << 20


def jn_tenant_heads_fwd_bwd_noalloc(ctx: Context, packed: Packed, hidden, heads: Sequence[Head],
                                    ios: Sequence[HeadIO], pooled=None):
    """The heads call on the library's own per-GPU scratch array (no
    workspace argument; allocates nothing)."""
    ha, ia = _head_arrays(heads, ios)
    _check(_lib.jn_tenant_heads_fwd_bwd_noalloc(ctx.handle, C.byref(packed.struct), _ptr(hidden), ha, ia,
                                                len(heads), _ptr(pooled)), ctx)


# ------------------------------------------------------- action expert ------

def jn_pack_tenant_sizes(reqs: Sequence[Request], tenants: Sequence[Tenant], d: int, align: int = 1):
    """(samples [G] int32, prefix rows [G] int64) of every tenant in the group."""
    ra, keep = _requests(reqs)
    ta = _tenants(tenants)
    G = len(tenants)
    n = np.zeros(G, np.int32)
    r = np.zeros(G, np.int64)
    _check(_lib.jn_pack_tenant_sizes(ra, len(reqs), ta, G, C.byref(_opts(d, align)),
                                     n.ctypes.data_as(C.POINTER(C.c_int32)),
                                     r.ctypes.data_as(C.POINTER(C.c_int64))), what="jn_pack_tenant_sizes")
    return n, r


class Expert:
    """A tenant's action expert: device bf16 tensors w_in [d, a], w_out [a, d],
    gf [d] and per layer a dict with the keys of ``EXPERT_LAYER_FIELDS``."""

    def __init__(self, w_in, w_out, gf, layers: List[dict], n_heads: int, chunk: int, d_prefix: int, eps: float,
                 w_time=None):
        self.w_in, self.w_out, self.gf, self.layers, self.w_time = w_in, w_out, gf, layers, w_time
        s = jn_expert()
        s.n_layers = len(layers)
        s.d = int(w_in.shape[0])
        s.n_heads = int(n_heads)
        s.ffn = int(layers[0]["w_up"].shape[0])
        s.action_dim = int(w_in.shape[1])
        s.chunk = int(chunk)
        s.d_prefix = int(d_prefix)
        s.eps = float(eps)
        s.w_in, s.w_out, s.gf = _ptr(w_in), _ptr(w_out), _ptr(gf)
        if w_time is not None:  # flow matching: [d, d_time] flow-time projection
            s.w_time = _ptr(w_time)
            s.d_time = int(w_time.shape[1])
        self._layers = (jn_expert_layer * len(layers))(
            *[jn_expert_layer(*[_ptr(lw[k]) for k in EXPERT_LAYER_FIELDS]) for lw in layers])
        s.layers = C.cast(self._layers, C.POINTER(jn_expert_layer))
        self.struct = s


class ExpertIO:
    """A tenant's expert inputs and outputs (device fp32 tensors): noisy /
    targets / pred [n, chunk, a], loss [1], dw_in, dw_out, dgf and per layer
    a dict of gradients keyed as ``EXPERT_LAYER_FIELDS``."""

    def __init__(self, n_samples: int, prefix_rows: int, noisy, targets, pred, loss, dw_in, dw_out, dgf,
                 layers: List[dict], flow_t=None, dw_time=None):
        self.noisy, self.targets, self.pred, self.loss = noisy, targets, pred, loss
        self.dw_in, self.dw_out, self.dgf, self.layers = dw_in, dw_out, dgf, layers
        self.flow_t, self.dw_time = flow_t, dw_time
        s = jn_expert_io()
        s.n_samples = int(n_samples)
        s.prefix_rows = int(prefix_rows)
        s.noisy, s.targets, s.pred, s.loss = _ptr(noisy), _ptr(targets), _ptr(pred), _ptr(loss)
        s.dw_in, s.dw_out, s.dgf = _ptr(dw_in), _ptr(dw_out), _ptr(dgf)
        s.flow_t, s.dw_time = _ptr(flow_t), _ptr(dw_time)
        self._layers = (jn_expert_layer_grads * len(layers))(
            *[jn_expert_layer_grads(*[_ptr(lg[k]) for k in EXPERT_LAYER_FIELDS]) for lg in layers])
        s.layers = C.cast(self._layers, C.POINTER(jn_expert_layer_grads))
        self.struct = s


def _expert_arrays(ex: Sequence[Expert], ios: Sequence[ExpertIO]):
    ea = (jn_expert * len(ex))(*[e.struct for e in ex])
    ia = (jn_expert_io * len(ios))(*[x.struct for x in ios])
    return ea, ia


def jn_experts_workspace_size(packed: Packed, ex: Sequence[Expert], ios: Sequence[ExpertIO]) -> int:
    ea, ia = _expert_arrays(ex, ios)
    n = C.c_size_t()
    _check(_lib.jn_experts_workspace_size(C.byref(packed.struct), ea, ia, len(ex), C.byref(n)),
           what="jn_experts_workspace_size")
    return int(n.value)


def jn_tenant_experts_fwd_bwd(ctx: Context, packed: Packed, hidden, ex: Sequence[Expert], ios: Sequence[ExpertIO],
                              ws):
    ea, ia = _expert_arrays(ex, ios)
    _check(_lib.jn_tenant_experts_fwd_bwd(ctx.handle, C.byref(packed.struct), _ptr(hidden), ea, ia, len(ex),
                                          _ptr(ws), ws.numel() * ws.element_size()), ctx)


# ---------------------------------------------------- tenant optimizer ------

class AdamWTenant:
    """One tenant's AdamW step: lists of device fp32 tensors (params, grads,
    first and second moments), optional bf16 copies (None entries allowed),
    hyperparameters and the 1-based index of this step."""

    def __init__(self, params: list, grads: list, m: list, v: list, step: int, lr: float, beta1: float = 0.9,
                 beta2: float = 0.999, eps: float = 1e-8, weight_decay: float = 0.0, bf16_out: Optional[list] = None):
        self.tensors = (params, grads, m, v, bf16_out)
        n = len(params)
        import torch
        if not (len(grads) == len(m) == len(v) == n) or (bf16_out is not None and len(bf16_out) != n):
            raise ValueError("params, grads, m, v (and bf16_out) must have one entry per tensor")
        for i in range(n):
            for name, t in (("params", params[i]), ("grads", grads[i]), ("m", m[i]), ("v", v[i])):
                if t.dtype != torch.float32 or not t.is_contiguous() or t.numel() != params[i].numel():
                    raise TypeError(f"{name}[{i}] must be a contiguous float32 tensor of {params[i].numel()} elements")
            if bf16_out is not None and bf16_out[i] is not None:
                b = bf16_out[i]
                if b.dtype != torch.bfloat16 or not b.is_contiguous() or b.numel() != params[i].numel():
                    raise TypeError(f"bf16_out[{i}] must be a contiguous bfloat16 tensor of {params[i].numel()} elements")
        s = jn_adamw_tenant()
        s.lr, s.beta1, s.beta2, s.eps, s.weight_decay = float(lr), float(beta1), float(beta2), float(eps), float(weight_decay)
        s.n_tensors = n
        s.step = int(step)
        mk = lambda xs: (C.c_void_p * max(n, 1))(*[_ptr(x) for x in xs])  # noqa: E731
        self._p, self._g, self._m, self._v = mk(params), mk(grads), mk(m), mk(v)
        self._n = (C.c_int64 * max(n, 1))(*[int(x.numel()) for x in params])
        s.params = C.cast(self._p, C.POINTER(C.c_void_p))
        s.grads = C.cast(self._g, C.POINTER(C.c_void_p))
        s.m = C.cast(self._m, C.POINTER(C.c_void_p))
        s.v = C.cast(self._v, C.POINTER(C.c_void_p))
        s.numel = C.cast(self._n, C.POINTER(C.c_int64))
        if bf16_out is not None:
            self._b = (C.c_void_p * max(n, 1))(*[_ptr(x) if x is not None else None for x in bf16_out])
            s.bf16_out = C.cast(self._b, C.POINTER(C.c_void_p))
        self.struct = s


def jn_adamw_workspace_size(tenants: Sequence[AdamWTenant]) -> int:
    arr = (jn_adamw_tenant * len(tenants))(*[t.struct for t in tenants])
    n = C.c_size_t()
    _check(_lib.jn_adamw_workspace_size(arr, len(tenants), C.byref(n)), what="jn_adamw_workspace_size")
    return int(n.value)


def jn_tenant_adamw_step(ctx: Context, tenants: Sequence[AdamWTenant], ws):
    arr = (jn_adamw_tenant * len(tenants))(*[t.struct for t in tenants])
    _check(_lib.jn_tenant_adamw_step(ctx.handle, arr, len(tenants), _ptr(ws), ws.numel() * ws.element_size()), ctx)


# -------------------------------------------------------------- unpack ------

def jn_unpack(ctx: Context, packed: Packed, reqs: Sequence[Request], rows, row_bytes: int, outs: Sequence):
    ra, keep = _requests(reqs)
    oa = (C.c_void_p * len(outs))(*[_ptr(o) for o in outs])
    _check(_lib.jn_unpack(ctx.handle, C.byref(packed.struct), ra, len(reqs), _ptr(rows), int(row_bytes), oa), ctx)


# ------------------------------------------------ inference-side batching ---

class Collector:
    """The inference queue's FIFO-compatible-prefix collector (host only):
    ``jn_collector_create / submit / poll / status``."""

    def __init__(self, max_batch_samples: int, timeout_us: int):
        h = C.c_void_p()
        _check(_lib.jn_collector_create(C.byref(h), int(max_batch_samples), int(timeout_us)),
               what="jn_collector_create")
        self.handle = h

    def submit(self, request_id: int, prefix_sig: int, d_model: int, n_samples: int, arrival_us: int):
        _check(_lib.jn_collector_submit(self.handle, int(request_id), int(prefix_sig), int(d_model), int(n_samples),
                                        int(arrival_us)), what="jn_collector_submit")

    def poll(self, now_us: int, cap: int = 4096) -> list:
        """Request ids of the batch ready at ``now_us`` (empty if none)."""
        ids = (C.c_int64 * max(cap, 1))()
        n = C.c_int32()
        _check(_lib.jn_collector_poll(self.handle, int(now_us), ids, int(cap), C.byref(n)), what="jn_collector_poll")
        return list(ids[: n.value])

    def status(self):
        """(queued requests, time the current prefix becomes ready or -1)."""
        n, t = C.c_int32(), C.c_int64()
        _check(_lib.jn_collector_status(self.handle, C.byref(n), C.byref(t)), what="jn_collector_status")
        return int(n.value), int(t.value)

    def close(self):
        if self.handle:
            _lib.jn_collector_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass


def jn_infer_workspace_size(reqs: Sequence[Request], tenants: Sequence[Tenant], d: int, align: int, bb: Backbone,
                            heads: Sequence[Head]) -> int:
    ra, keep = _requests(reqs)
    ha, _ = _head_arrays(heads)
    o = _opts(d, align)
    n = C.c_size_t()
    _check(_lib.jn_infer_workspace_size(ra, len(reqs), _tenants(tenants), len(tenants), C.byref(o),
                                        C.byref(bb.struct), ha, C.byref(n)), what="jn_infer_workspace_size")
    return int(n.value)


class InferPlan:
    """``jn_infer_plan_*``: a resident decode-only step over one physical batch
    (device buffers stay referenced here for the plan's lifetime)."""

    def __init__(self, ctx: Context, reqs: Sequence[Request], tenants: Sequence[Tenant], d: int, align: int,
                 bb: Backbone, heads: Sequence[Head], actions: Sequence, ws):
        ra, keep = _requests(reqs)
        ha, _ = _head_arrays(heads)
        o = _opts(d, align)
        acts = (C.c_void_p * len(actions))(*[_ptr(a) for a in actions])
        h = C.c_void_p()
        _check(_lib.jn_infer_plan_create(ctx.handle, ra, len(reqs), _tenants(tenants), len(tenants), C.byref(o),
                                         C.byref(bb.struct), ha, acts, _ptr(ws), ws.numel() * ws.element_size(),
                                         C.byref(h)), ctx)
        self.handle = h
        self.ctx = ctx
        self._keep = (reqs, bb, heads, actions, ws)

    def packed(self):
        """(jn_packed struct, hidden device pointer) of the plan's batch."""
        s = jn_packed()
        hid = C.c_void_p()
        _check(_lib.jn_infer_plan_packed(self.handle, C.byref(s), C.byref(hid)), what="jn_infer_plan_packed")
        return s, hid.value

    def launch(self):
        _check(_lib.jn_infer_plan_launch(self.ctx.handle, self.handle), self.ctx)

    def capture(self):
        _check(_lib.jn_infer_plan_capture(self.ctx.handle, self.handle), self.ctx)

    def replay(self):
        _check(_lib.jn_infer_plan_replay(self.ctx.handle, self.handle), self.ctx)

    def close(self):
        if self.handle:
            _lib.jn_infer_plan_destroy(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass
