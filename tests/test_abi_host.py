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


def test_struct_layout_matches_c(tmp_path, lib):
    """sizeof / offsetof from the C compiler against the ctypes mirror."""
    from paper_2607_16074_amd import _abi
    structs = {"jn_request": _abi.jn_request, "jn_tenant": _abi.jn_tenant, "jn_pack_opts": _abi.jn_pack_opts,
               "jn_pack_sizes": _abi.jn_pack_sizes, "jn_packed": _abi.jn_packed, "jn_layer": _abi.jn_layer,
               "jn_backbone": _abi.jn_backbone, "jn_head": _abi.jn_head, "jn_head_io": _abi.jn_head_io}
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
