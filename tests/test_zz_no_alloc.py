"""The allocation-free heads call (jn_tenant_heads_fwd_bwd_noalloc) against
the workspace-taking call it mirrors, through the C ABI.

Two calls in a row on one GPU share the library's scratch array: the first
on the 4-tenant 12-layer d768 group (128 samples), the second on the tiny
2-tenant group (16 samples), so the second runs over what the first left in
the array.  Both must equal the workspace call bit for bit (same kernels, same
reduction orders).  A problem larger than the array is refused before
anything is enqueued.
"""
import sys

import numpy as np
import pytest

import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def jn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_16074_amd as lib
    return lib


def _fresh_ios(jn, st):
    ios = []
    for io in st.ios:
        ios.append(jn.HeadIO(io.targets, torch.full_like(io.actions, 7.0), torch.full_like(io.loss, 7.0),
                             [torch.full_like(w, 7.0) for w in io.dW], [torch.full_like(b, 7.0) for b in io.db]))
    return ios


def _same(a, b):
    return a.shape == b.shape and torch.equal(a, b)


def _check_against_workspace_call(jn, st):
    st.run()
    ios = _fresh_ios(jn, st)
    pooled = torch.full_like(st.pooled, 7.0)
    jn.jn_tenant_heads_fwd_bwd_noalloc(st.ctx, st.packed, st.hidden, st.heads, ios, pooled)
    torch.cuda.synchronize()
    assert _same(pooled, st.pooled)
    for k, (a, b) in enumerate(zip(ios, st.ios)):
        assert _same(a.actions, b.actions), k
        assert _same(a.loss, b.loss), k
        for x, y in zip(a.dW + a.db, b.dW + b.db):
            assert _same(x, y), k


def test_noalloc_heads_equal_workspace_call_twice(jn):
    from paper_2607_16074_amd import step as jstep
    for cfg in (2, 1):   # the second call is the smaller one
        wl = W.make_workload(cfg)
        model, reqs, targets = jstep.from_workload(wl)
        st = jstep.GroupStep(model, reqs, targets, list(range(wl.spec.G)))
        need = jn.jn_heads_workspace_size(st.packed, st.heads)
        _say(f"no-alloc heads, config {cfg}: N={st.N}, workspace {need} B of {jn.HEADS_SCRATCH_BYTES}")
        assert need <= jn.HEADS_SCRATCH_BYTES
        _check_against_workspace_call(jn, st)


def test_noalloc_heads_refuse_oversize(jn):
    """A group whose head workspace exceeds the array: JN_ENOSPACE, nothing
    written."""
    from paper_2607_16074_amd import step as jstep
    n = 33000   # pooled features alone: 33000 x 512 x 4 B > 64 MiB
    ten = (W.TenantSpec(n, 0, 1, 1, 1, (512, 64, 6), 3, 2),)
    spec = W.WorkloadSpec(96, W.BackboneSpec(1, 512, 4, 256, False), ten, 0, "oversize heads")
    wl = W.make_workload(spec)
    model, reqs, targets = jstep.from_workload(wl)
    st = jstep.GroupStep(model, reqs, targets, [0])
    need = jn.jn_heads_workspace_size(st.packed, st.heads)
    _say(f"no-alloc heads, oversize: N={st.N}, workspace {need} B")
    assert need > jn.HEADS_SCRATCH_BYTES
    ios = _fresh_ios(jn, st)
    torch.cuda.synchronize()
    with pytest.raises(jn.JNError) as e:
        jn.jn_tenant_heads_fwd_bwd_noalloc(st.ctx, st.packed, st.hidden, st.heads, ios, None)
    assert e.value.status == jn._abi.JN_ENOSPACE
    torch.cuda.synchronize()
    assert bool((ios[0].actions == 7.0).all()) and bool((ios[0].loss == 7.0).all())
