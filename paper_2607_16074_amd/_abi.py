"""ctypes mirror of ``include/joynexus.h`` (argument marshalling only).

Every function of the C ABI is exposed under its own name; device buffers
are passed as raw pointers (``tensor.data_ptr()``), host arrays as ctypes
arrays.  Nothing here computes any part of the step.
"""
from __future__ import annotations

import ctypes as C
import os

_HERE = os.path.dirname(os.path.abspath(__file__))
# the in-tree build; JN_LIB_PATH selects another build of the same sources
LIB_PATH = os.environ.get("JN_LIB_PATH") or os.path.join(_HERE, "libjoynexus.so")

JN_OK, JN_EINVAL, JN_EINCOMPAT, JN_ESHAPE, JN_ENOSPACE, JN_EHIP, JN_EUNSUPPORTED = range(7)
JN_OPT_EXPERT_TRANSPOSES = 1  # jn_ctx_set_option: expert gradient GEMMs on materialised transposes
STATUS_NAMES = {0: "JN_OK", 1: "JN_EINVAL", 2: "JN_EINCOMPAT", 3: "JN_ESHAPE", 4: "JN_ENOSPACE",
                5: "JN_EHIP", 6: "JN_EUNSUPPORTED"}

EXPORTS = (
    "jn_ctx_create", "jn_ctx_destroy", "jn_ctx_set_stream", "jn_last_error", "jn_ctx_set_trace",
    "jn_ctx_trace_read", "jn_ctx_set_option",
    "jn_pack_plan", "jn_pack_maps_host", "jn_pack_group",
    "jn_backbone_workspace_size", "jn_backbone_forward",
    "jn_heads_workspace_size", "jn_tenant_heads_fwd_bwd", "jn_tenant_heads_fwd_bwd_noalloc",
    "jn_pack_tenant_sizes", "jn_experts_workspace_size", "jn_tenant_experts_fwd_bwd",
    "jn_adamw_workspace_size", "jn_tenant_adamw_step",
    "jn_unpack",
    "jn_collector_create", "jn_collector_destroy", "jn_collector_submit", "jn_collector_poll",
    "jn_collector_status",
    "jn_infer_workspace_size", "jn_infer_plan_create", "jn_infer_plan_packed", "jn_infer_plan_launch",
    "jn_infer_plan_capture", "jn_infer_plan_replay", "jn_infer_plan_destroy",
)


OPS = {1: "pack", 2: "rmsnorm", 3: "gemm_qkv", 4: "attention", 5: "gemm_o", 6: "gemm_up", 7: "gemm_down",
       8: "pool", 9: "head_fwd", 10: "loss", 11: "head_bwd", 12: "unpack", 13: "expert_gemm",
       14: "expert_attention", 15: "expert_other", 16: "optimizer", 17: "rope"}


class jn_trace_entry(C.Structure):
    _fields_ = [("op", C.c_int32), ("M", C.c_int32), ("N", C.c_int32), ("K", C.c_int32), ("ms", C.c_float),
                ("reserved", C.c_int32)]


class jn_request(C.Structure):
    _fields_ = [("tenant", C.c_int32), ("n_samples", C.c_int32), ("max_len", C.c_int32),
                ("reserved", C.c_int32), ("embeds", C.c_void_p), ("lengths", C.POINTER(C.c_int32))]


class jn_tenant(C.Structure):
    _fields_ = [("prefix_sig", C.c_uint64), ("d_model", C.c_int32), ("reserved", C.c_int32)]


class jn_pack_opts(C.Structure):
    _fields_ = [("d_model", C.c_int32), ("align", C.c_int32)]


class jn_pack_sizes(C.Structure):
    _fields_ = [("N", C.c_int32), ("T", C.c_int32), ("max_seqlen", C.c_int32), ("reserved", C.c_int32),
                ("map_bytes", C.c_int64), ("token_bytes", C.c_int64)]


_I32P = C.POINTER(C.c_int32)


class jn_packed(C.Structure):
    _fields_ = [("R", C.c_int32), ("G", C.c_int32), ("N", C.c_int32), ("T", C.c_int32), ("d", C.c_int32),
                ("max_seqlen", C.c_int32), ("align", C.c_int32), ("req_sig", C.c_int32),
                ("max_tenant_n", C.c_int32),
                ("tokens", C.c_void_p),
                ("seqlens", _I32P), ("cu_seqlens", _I32P), ("sample_request", _I32P), ("sample_local", _I32P),
                ("sample_tenant", _I32P), ("tenant_sample_off", _I32P), ("tenant_perm", _I32P),
                ("sample_tenant_rank", _I32P), ("token_sample", _I32P), ("token_pos", _I32P),
                ("req_table", C.c_void_p)]

    MAP_FIELDS = ("seqlens", "cu_seqlens", "sample_request", "sample_local", "sample_tenant",
                  "tenant_sample_off", "tenant_perm", "sample_tenant_rank", "token_sample", "token_pos")

    def map_len(self, name: str) -> int:
        return {"cu_seqlens": self.N + 1, "tenant_sample_off": self.G + 1,
                "token_sample": self.T, "token_pos": self.T}.get(name, self.N)


class jn_layer(C.Structure):
    _fields_ = [("wqkv", C.c_void_p), ("wo", C.c_void_p), ("w_up", C.c_void_p), ("w_gate", C.c_void_p),
                ("w_down", C.c_void_p), ("g1", C.c_void_p), ("g2", C.c_void_p)]


class jn_backbone(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d", C.c_int32), ("n_heads", C.c_int32), ("ffn", C.c_int32),
                ("eps", C.c_float), ("n_kv_heads", C.c_int32), ("layers", C.POINTER(jn_layer)), ("gf", C.c_void_p),
                ("causal", C.c_int32), ("rope_theta", C.c_float)]


class jn_head(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("action_dim", C.c_int32), ("chunk", C.c_int32), ("reserved", C.c_int32),
                ("dims", _I32P), ("W", C.POINTER(C.c_void_p)), ("b", C.POINTER(C.c_void_p))]


class jn_head_io(C.Structure):
    _fields_ = [("targets", C.c_void_p), ("actions", C.c_void_p), ("loss", C.c_void_p),
                ("dW", C.POINTER(C.c_void_p)), ("db", C.POINTER(C.c_void_p))]


EXPERT_LAYER_FIELDS = ("wqkv_s", "wo_s", "wq_c", "wkv_c", "wo_c", "w_up", "w_down", "g1", "g2", "g3")


class jn_expert_layer(C.Structure):
    _fields_ = [(k, C.c_void_p) for k in EXPERT_LAYER_FIELDS]


class jn_expert(C.Structure):
    _fields_ = [("n_layers", C.c_int32), ("d", C.c_int32), ("n_heads", C.c_int32), ("ffn", C.c_int32),
                ("action_dim", C.c_int32), ("chunk", C.c_int32), ("d_prefix", C.c_int32), ("eps", C.c_float),
                ("w_in", C.c_void_p), ("w_out", C.c_void_p), ("gf", C.c_void_p),
                ("layers", C.POINTER(jn_expert_layer)), ("w_time", C.c_void_p), ("d_time", C.c_int32),
                ("reserved", C.c_int32)]


class jn_expert_layer_grads(C.Structure):
    _fields_ = [(k, C.c_void_p) for k in EXPERT_LAYER_FIELDS]


class jn_expert_io(C.Structure):
    _fields_ = [("n_samples", C.c_int32), ("reserved", C.c_int32), ("prefix_rows", C.c_int64),
                ("noisy", C.c_void_p), ("targets", C.c_void_p), ("pred", C.c_void_p), ("loss", C.c_void_p),
                ("dw_in", C.c_void_p), ("dw_out", C.c_void_p), ("dgf", C.c_void_p),
                ("layers", C.POINTER(jn_expert_layer_grads)), ("flow_t", C.c_void_p), ("dw_time", C.c_void_p)]


class jn_adamw_tenant(C.Structure):
    _fields_ = [("lr", C.c_float), ("beta1", C.c_float), ("beta2", C.c_float), ("eps", C.c_float),
                ("weight_decay", C.c_float), ("n_tensors", C.c_int32), ("step", C.c_int64),
                ("params", C.POINTER(C.c_void_p)), ("grads", C.POINTER(C.c_void_p)), ("m", C.POINTER(C.c_void_p)),
                ("v", C.POINTER(C.c_void_p)), ("numel", C.POINTER(C.c_int64)), ("bf16_out", C.POINTER(C.c_void_p))]


_lib = None


def load(path: str = LIB_PATH) -> C.CDLL:
    """Load the built library and declare its prototypes (raises if missing)."""
    global _lib
    if _lib is not None:
        return _lib
    if not os.path.exists(path):
        raise ImportError(f"{path} is not built; run __graft_entry__.build() (hipcc --offload-arch=gfx950)")
    lib = C.CDLL(path)
    P, V = C.POINTER, C.c_void_p
    sig = {
        "jn_ctx_create": (C.c_int, [P(V), V]),
        "jn_ctx_destroy": (None, [V]),
        "jn_ctx_set_stream": (C.c_int, [V, V]),
        "jn_last_error": (C.c_char_p, [V]),
        "jn_ctx_set_trace": (C.c_int, [V, C.c_int32]),
        "jn_ctx_set_option": (C.c_int, [V, C.c_int32, C.c_int32]),
        "jn_ctx_trace_read": (C.c_int, [V, P(jn_trace_entry), C.c_int32, P(C.c_int32)]),
        "jn_pack_plan": (C.c_int, [P(jn_request), C.c_int32, P(jn_tenant), C.c_int32, P(jn_pack_opts),
                                   P(jn_pack_sizes)]),
        "jn_pack_maps_host": (C.c_int, [P(jn_request), C.c_int32, P(jn_tenant), C.c_int32, P(jn_pack_opts),
                                        V, C.c_size_t, P(jn_packed)]),
        "jn_pack_group": (C.c_int, [V, P(jn_request), C.c_int32, P(jn_tenant), C.c_int32, P(jn_pack_opts),
                                    V, C.c_size_t, V, C.c_size_t, P(jn_packed)]),
        "jn_backbone_workspace_size": (C.c_int, [P(jn_backbone), C.c_int32, P(C.c_size_t)]),
        "jn_backbone_forward": (C.c_int, [V, P(jn_backbone), P(jn_packed), V, V, C.c_size_t]),
        "jn_heads_workspace_size": (C.c_int, [P(jn_packed), P(jn_head), C.c_int32, P(C.c_size_t)]),
        "jn_tenant_heads_fwd_bwd": (C.c_int, [V, P(jn_packed), V, P(jn_head), P(jn_head_io), C.c_int32, V,
                                              C.c_size_t, V]),
        "jn_tenant_heads_fwd_bwd_noalloc": (C.c_int, [V, P(jn_packed), V, P(jn_head), P(jn_head_io), C.c_int32,
                                                      V]),
        "jn_pack_tenant_sizes": (C.c_int, [P(jn_request), C.c_int32, P(jn_tenant), C.c_int32, P(jn_pack_opts),
                                           P(C.c_int32), P(C.c_int64)]),
        "jn_experts_workspace_size": (C.c_int, [P(jn_packed), P(jn_expert), P(jn_expert_io), C.c_int32,
                                                P(C.c_size_t)]),
        "jn_tenant_experts_fwd_bwd": (C.c_int, [V, P(jn_packed), V, P(jn_expert), P(jn_expert_io), C.c_int32, V,
                                                C.c_size_t]),
        "jn_adamw_workspace_size": (C.c_int, [P(jn_adamw_tenant), C.c_int32, P(C.c_size_t)]),
        "jn_tenant_adamw_step": (C.c_int, [V, P(jn_adamw_tenant), C.c_int32, V, C.c_size_t]),
        "jn_unpack": (C.c_int, [V, P(jn_packed), P(jn_request), C.c_int32, V, C.c_size_t, P(V)]),
        "jn_collector_create": (C.c_int, [P(V), C.c_int32, C.c_int64]),
        "jn_collector_destroy": (None, [V]),
        "jn_collector_submit": (C.c_int, [V, C.c_int64, C.c_uint64, C.c_int32, C.c_int32, C.c_int64]),
        "jn_collector_poll": (C.c_int, [V, C.c_int64, P(C.c_int64), C.c_int32, P(C.c_int32)]),
        "jn_collector_status": (C.c_int, [V, P(C.c_int32), P(C.c_int64)]),
        "jn_infer_workspace_size": (C.c_int, [P(jn_request), C.c_int32, P(jn_tenant), C.c_int32, P(jn_pack_opts),
                                              P(jn_backbone), P(jn_head), P(C.c_size_t)]),
        "jn_infer_plan_create": (C.c_int, [V, P(jn_request), C.c_int32, P(jn_tenant), C.c_int32, P(jn_pack_opts),
                                           P(jn_backbone), P(jn_head), P(V), V, C.c_size_t, P(V)]),
        "jn_infer_plan_packed": (C.c_int, [V, P(jn_packed), P(V)]),
        "jn_infer_plan_launch": (C.c_int, [V, V]),
        "jn_infer_plan_capture": (C.c_int, [V, V]),
        "jn_infer_plan_replay": (C.c_int, [V, V]),
        "jn_infer_plan_destroy": (None, [V]),
    }
    for name, (res, args) in sig.items():
        f = getattr(lib, name)
        f.restype = res
        f.argtypes = args
    _lib = lib
    return lib
