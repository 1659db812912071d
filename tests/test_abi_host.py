"""CPU checks of the C ABI library: it loads, exports every declared entry
point, its ctypes mirror matches the C struct layout, and the host-side pack
plan equals the oracle's plan bit for bit (App. A.3: slices recorded by
canonicalize-and-pad), including edge cases and error statuses."""
import ctypes as C
import os
import re
import subprocess

import numpy as np
import pytest

from oracle import plan as oplan

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "joynexus.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:jn_status|void|const char\*)\s+(jn_\w+)\(", text, re.M)))


def test_library_exports_every_declared_symbol(lib):
    names = declared_functions()
    assert len(names) >= 12
    so = C.CDLL(lib.lib_path())
    for n in names:
        assert hasattr(so, n), n
    from paper_2607_16074_amd import _abi
    assert set(names) == set(_abi.EXPORTS)


def test_noalloc_scratch_size_matches_header(lib):
    text = open(HEADER).read()
    m = re.search(r"#define JN_HEADS_SCRATCH_BYTES \((\d+)u << (\d+)\)", text)
    assert m and int(m.group(1)) << int(m.group(2)) == lib.HEADS_SCRATCH_BYTES


def test_struct_layout_matches_c(tmp_path, lib):
    """sizeof / offsetof from the C compiler against the ctypes mirror."""
    from paper_2607_16074_amd import _abi
    structs = {"jn_request": _abi.jn_request, "jn_tenant": _abi.jn_tenant, "jn_pack_opts": _abi.jn_pack_opts,
               "jn_pack_sizes": _abi.jn_pack_sizes, "jn_packed": _abi.jn_packed, "jn_layer": _abi.jn_layer,
               "jn_backbone": _abi.jn_backbone, "jn_head": _abi.jn_head, "jn_head_io": _abi.jn_head_io,
               "jn_expert_layer": _abi.jn_expert_layer, "jn_expert": _abi.jn_expert,
               "jn_expert_layer_grads": _abi.jn_expert_layer_grads, "jn_expert_io": _abi.jn_expert_io,
               "jn_trace_entry": _abi.jn_trace_entry, "jn_adamw_tenant": _abi.jn_adamw_tenant}
    lines = ['#include <stdio.h>', '#include <stddef.h>', '#include "joynexus.h"', "int main(void){"]
    for name, cls in structs.items():
        lines.append(f'printf("{name} %zu\\n", sizeof({name}));')
        for f, _ in cls._fields_:
            lines.append(f'printf("{name}.{f} %zu\\n", offsetof({name}, {f}));')
    lines.append("return 0;}")
    src = tmp_path / "layout.c"
    src.write_text("\n".join(lines))
    exe = tmp_path / "layout"
    subprocess.run(["gcc", "-I", os.path.join(ROOT, "include"), str(src), "-o", str(exe)], check=True)
    out = subprocess.run([str(exe)], capture_output=True, text=True, check=True).stdout.split("\n")
    got = dict(l.split() for l in out if l.strip())
    for name, cls in structs.items():
        assert int(got[name]) == C.sizeof(cls), name
        for f, _ in cls._fields_:
            assert int(got[f"{name}.{f}"]) == getattr(cls, f).offset, f"{name}.{f}"


# ------------------------------------------------------------- host plan ---

def _reqs(lib, tenants, lengths, max_lens):
    return [lib.Request(t, 4096, np.array(l, np.int32), m) for t, l, m in zip(tenants, lengths, max_lens)]


CASES = [
    # (request tenants, lengths per request, max_len per request, G, align)
    ([0], [[1]], [1], 1, 1),                                       # smallest possible batch
    ([0, 1], [[5, 9, 1], [12, 3]], [12, 12], 2, 1),
    ([1, 0, 1, 0], [[3, 4], [7], [1, 1, 1], [8, 2]], [8, 7, 4, 8], 2, 16),  # interleaved tenants
    ([2, 0, 1], [[64, 63, 65], [1], [128]], [65, 1, 128], 3, 64),     # lengths at/around align
    ([0, 0, 0], [[10], [20], [30]], [10, 20, 30], 1, 4),              # one tenant, several requests
]


@pytest.mark.parametrize("case", range(len(CASES)))
def test_host_plan_bit_exact(lib, case):
    tn, lens, mls, G, align = CASES[case]
    d = 128
    got = lib.jn_pack_maps_host(_reqs(lib, tn, lens, mls), [lib.Tenant(7, d)] * G, d, align)
    ref = oplan.pack_plan(tn, lens, mls, G, align)
    assert got["N"] == ref["N"] and got["T"] == ref["T"]
    for k in ("seqlens", "cu_seqlens", "sample_request", "sample_local", "sample_tenant", "tenant_sample_off",
              "tenant_perm", "sample_tenant_rank", "token_sample", "token_pos"):
        assert got[k].dtype == np.int32 and np.array_equal(got[k], ref[k]), k
    sz = lib.jn_pack_plan(_reqs(lib, tn, lens, mls), [lib.Tenant(7, d)] * G, d, align)
    assert sz.token_bytes == ref["T"] * d * 2 and sz.max_seqlen == max(max(l) for l in lens)


def test_host_plan_random_bit_exact(lib):
    rng = np.random.default_rng(7)
    for trial in range(20):
        G = int(rng.integers(1, 6))
        R = int(rng.integers(G, 3 * G + 1))
        tn = list(rng.permutation(np.concatenate([np.arange(G), rng.integers(0, G, R - G)])))
        mls = [int(rng.integers(1, 300)) for _ in range(R)]
        lens = [list(rng.integers(1, m + 1, size=int(rng.integers(1, 9)))) for m in mls]
        align = int(rng.choice([1, 2, 8, 16, 64, 128]))
        got = lib.jn_pack_maps_host(_reqs(lib, tn, lens, mls), [lib.Tenant(1, 256)] * G, 256, align)
        ref = oplan.pack_plan(tn, lens, mls, G, align)
        for k in ("cu_seqlens", "tenant_perm", "sample_tenant_rank", "token_sample", "token_pos",
                  "tenant_sample_off", "sample_request", "sample_local"):
            assert np.array_equal(got[k], ref[k]), (trial, k)


def test_host_plan_errors(lib):
    d = 64
    T = lambda g=1: [lib.Tenant(7, d)] * g  # noqa: E731
    bad = [
        (_reqs(lib, [0], [[0]], [4]), T(), lib._abi.JN_ESHAPE),          # empty sample
        (_reqs(lib, [0], [[5]], [4]), T(), lib._abi.JN_ESHAPE),          # longer than max_len
        (_reqs(lib, [0], [[2]], [4]), T(2), lib._abi.JN_ESHAPE),         # tenant 1 has nothing
        (_reqs(lib, [3], [[2]], [4]), T(2), lib._abi.JN_ESHAPE),         # tenant outside the table
        (_reqs(lib, [0, 1], [[2], [2]], [4, 4]), [lib.Tenant(7, d), lib.Tenant(8, d)], lib._abi.JN_EINCOMPAT),
        (_reqs(lib, [0, 1], [[2], [2]], [4, 4]), [lib.Tenant(7, d), lib.Tenant(7, 2 * d)], lib._abi.JN_EINCOMPAT),
    ]
    for reqs, ten, code in bad:
        with pytest.raises(lib.JNError) as e:
            lib.jn_pack_plan(reqs, ten, d, 1)
        assert e.value.status == code
    with pytest.raises(lib.JNError) as e:
        lib.jn_pack_plan(_reqs(lib, [0], [[2]], [4]), T(), d, 0)
    assert e.value.status == lib._abi.JN_EINVAL
    # a batch whose packed rows overflow 32-bit row indices (lengths only; nothing is read)
    big = 1 << 30
    with pytest.raises(lib.JNError) as e:
        lib.jn_pack_plan(_reqs(lib, [0], [[big, big]], [big]), T(), d, 1)
    assert e.value.status == lib._abi.JN_ESHAPE


def test_request_signature_tells_splits_apart(lib):
    """The batch records the shape of the request list it was packed from, so
    that an unpack given another split of the same samples (same total, other
    per-request counts or canonical lengths) can be refused on the host."""
    d = 64
    T = [lib.Tenant(7, d)] * 2
    a = lib.jn_pack_maps_host(_reqs(lib, [0, 0, 1], [[3, 4], [5], [2, 2]], [8, 8, 4]), T, d, 1)
    b = lib.jn_pack_maps_host(_reqs(lib, [0, 0, 1], [[3, 4], [5], [2, 2]], [8, 8, 4]), T, d, 16)
    c = lib.jn_pack_maps_host(_reqs(lib, [0, 0, 1], [[3], [4, 5], [2, 2]], [8, 8, 4]), T, d, 1)
    e = lib.jn_pack_maps_host(_reqs(lib, [0, 0, 1], [[3, 4], [5], [2, 2]], [8, 9, 4]), T, d, 1)
    f = lib.jn_pack_maps_host(_reqs(lib, [0, 0, 1], [[1, 1], [1], [1, 1]], [8, 8, 4]), T, d, 1)
    assert a["N"] == c["N"] == e["N"]
    assert a["req_sig"] == b["req_sig"] == f["req_sig"]   # lengths and alignment do not enter
    assert len({a["req_sig"], c["req_sig"], e["req_sig"]}) == 3


# ------------------------------------------------------ expert validation ---

def test_pack_tenant_sizes_match_plan(lib):
    rng = np.random.default_rng(11)
    for trial in range(10):
        G = int(rng.integers(1, 5))
        R = int(rng.integers(G, 2 * G + 2))
        tn = list(rng.permutation(np.concatenate([np.arange(G), rng.integers(0, G, R - G)])))
        mls = [int(rng.integers(1, 200)) for _ in range(R)]
        lens = [list(rng.integers(1, m + 1, size=int(rng.integers(1, 6)))) for m in mls]
        align = int(rng.choice([1, 16, 64]))
        n, rows = lib.jn_pack_tenant_sizes(_reqs(lib, tn, lens, mls), [lib.Tenant(1, 128)] * G, 128, align)
        for g in range(G):
            mine = [l for t, ls in zip(tn, lens) if t == g for l in ls]
            assert n[g] == len(mine) and rows[g] == sum(mine), (trial, g)


def _host_packed(lib, tn, lens, mls, G, d):
    """A jn_packed whose maps live in host memory (enough for size queries)."""
    import ctypes as C
    sz = lib.jn_pack_plan(_reqs(lib, tn, lens, mls), [lib.Tenant(1, d)] * G, d, 1)
    buf = np.zeros(int(sz.map_bytes), dtype=np.uint8)
    ra, keep = lib._requests(_reqs(lib, tn, lens, mls))
    out = lib._abi.jn_packed()
    st = lib._lib.jn_pack_maps_host(ra, len(tn), lib._tenants([lib.Tenant(1, d)] * G), G,
                                    C.byref(lib._opts(d, 1)), buf.ctypes.data_as(C.c_void_p), buf.nbytes,
                                    C.byref(out))
    assert st == 0
    return lib.Packed(out, buf, None), buf, keep


def _fake_expert(lib, d=256, H=4, f=512, L=1, a=7, chunk=10, dp=128):
    import torch
    e = lambda *s: torch.zeros(s, dtype=torch.bfloat16)  # noqa: E731
    layers = [{"wqkv_s": e(3 * d, d), "wo_s": e(d, d), "wq_c": e(d, d), "wkv_c": e(2 * d, dp), "wo_c": e(d, d),
               "w_up": e(f, d), "w_down": e(d, f), "g1": e(d), "g2": e(d), "g3": e(d)} for _ in range(L)]
    return lib.Expert(e(d, a), e(a, d), e(d), layers, H, chunk, dp, 1e-6)


def _fake_io(lib, n, rows, d=256, f=512, L=1, a=7, chunk=10, dp=128):
    import torch
    z = lambda *s: torch.zeros(s, dtype=torch.float32)  # noqa: E731
    layers = [{"wqkv_s": z(3 * d, d), "wo_s": z(d, d), "wq_c": z(d, d), "wkv_c": z(2 * d, dp), "wo_c": z(d, d),
               "w_up": z(f, d), "w_down": z(d, f), "g1": z(d), "g2": z(d), "g3": z(d)} for _ in range(L)]
    return lib.ExpertIO(n, rows, z(n, chunk, a), z(n, chunk, a), z(n, chunk, a), z(1), z(d, a), z(a, d), z(d),
                        layers)


def test_experts_workspace_validation(lib):
    """Shape contract of jn_tenant_experts_fwd_bwd, checked on the host."""
    E = lib._abi
    tn, lens, mls = [0, 1], [[5, 9, 1], [12, 3]], [12, 12]
    p, buf, keep = _host_packed(lib, tn, lens, mls, 2, 128)
    ex = [_fake_expert(lib), _fake_expert(lib, a=32)]
    ios = [_fake_io(lib, 3, 15), _fake_io(lib, 2, 15, a=32)]
    n0 = lib.jn_experts_workspace_size(p, ex, ios)
    assert n0 > 0
    bad = [
        (lambda: ([ex[0]], [ios[0]]), E.JN_EINVAL),                                   # G differs from the batch
        (lambda: (ex, [_fake_io(lib, 2, 15), ios[1]]), E.JN_ESHAPE),                  # sample count
        (lambda: (ex, [_fake_io(lib, 3, 2), ios[1]]), E.JN_ESHAPE),                   # prefix rows < samples
        (lambda: ([_fake_expert(lib, chunk=65), _fake_expert(lib, a=32, chunk=65)],
                  [_fake_io(lib, 3, 15, chunk=65), _fake_io(lib, 2, 15, a=32, chunk=65)]), E.JN_EUNSUPPORTED),
        (lambda: ([_fake_expert(lib, H=8), _fake_expert(lib, H=8, a=32)], ios), E.JN_EUNSUPPORTED),  # hd 32
        (lambda: ([_fake_expert(lib, a=33), ex[1]], [_fake_io(lib, 3, 15, a=33), ios[1]]), E.JN_EUNSUPPORTED),
        (lambda: ([_fake_expert(lib, dp=256), _fake_expert(lib, a=32, dp=256)], ios), E.JN_EINCOMPAT),
        (lambda: ([ex[0], _fake_expert(lib, f=1024, a=32)], ios), E.JN_EUNSUPPORTED),  # shapes differ
        (lambda: (ex, [_fake_io(lib, 3, 1000), ios[1]]), E.JN_ESHAPE),                 # prefix beyond the batch
    ]
    for make, code in bad:
        exs, iss = make()
        with pytest.raises(lib.JNError) as e:
            lib.jn_experts_workspace_size(p, exs, iss)
        assert e.value.status == code, (code, e.value)
    # null weight and unaligned gradient pointers
    ex_null = _fake_expert(lib)
    ex_null._layers[0].wo_c = None
    with pytest.raises(lib.JNError) as e:
        lib.jn_experts_workspace_size(p, [ex_null, ex[1]], ios)
    assert e.value.status == E.JN_EINVAL
    io_un = _fake_io(lib, 3, 15)
    io_un._layers[0].w_up = io_un._layers[0].w_up + 4
    with pytest.raises(lib.JNError) as e:
        lib.jn_experts_workspace_size(p, ex, [io_un, ios[1]])
    assert e.value.status == E.JN_EINVAL


def test_adamw_validation(lib):
    import torch
    z = lambda n: torch.zeros(n, dtype=torch.float32)  # noqa: E731
    good = lambda **kw: lib.AdamWTenant([z(8)], [z(8)], [z(8)], [z(8)], **{"step": 1, "lr": 1e-3, **kw})  # noqa: E731
    assert lib.jn_adamw_workspace_size([good(), good(step=3)]) > 0
    E = lib._abi
    for kw in ({"step": 0}, {"beta1": 1.0}, {"beta2": -0.1}, {"eps": 0.0}, {"lr": -1.0}):
        with pytest.raises(lib.JNError) as e:
            lib.jn_adamw_workspace_size([good(**kw)])
        assert e.value.status == E.JN_EINVAL, kw
    # an unaligned parameter pointer
    t = good()
    t._p[0] = t._p[0] + 4
    with pytest.raises(lib.JNError) as e:
        lib.jn_adamw_workspace_size([t])
    assert e.value.status == E.JN_EINVAL
