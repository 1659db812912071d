"""GPU parity of the per-tenant AdamW step against the fp64 oracle.

The C ABI carries the hyperparameters as fp32, so the oracle is given the
same fp32-rounded values (e.g. beta2 = 0.999f, whose 1 - beta2 differs from
0.001 by 5e-5 relative).

Bars (fp32 arithmetic of a few operations per element): parameters within
4e-7 relative plus 2e-6 * lr absolute, moments within 1e-6 relative plus
1e-7 * max|g| absolute; bf16 copies bit-exact against rounding the GPU's own
fp32 result (the rounding decision taken in the kernel's precision).
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


def check(p_gpu, m_gpu, v_gpu, ref, lr, gmax):
    p, m, v = ref
    assert np.all(np.abs(p_gpu - p) <= 4e-7 * np.abs(p) + 2e-6 * lr), float(np.max(np.abs(p_gpu - p)))
    assert np.all(np.abs(m_gpu - m) <= 1e-6 * np.abs(m) + 1e-7 * gmax)
    assert np.all(np.abs(v_gpu - v) <= 1e-6 * np.abs(v) + 1e-7 * gmax * gmax)


def test_adamw_three_tenants_several_steps(jn):
    """Mixed tensor sizes (tails of 1..3 elements, several blocks), per-tenant
    hyperparameters and versions, bf16 copies on one tenant, three steps."""
    from oracle import optim
    rng = np.random.default_rng(0)
    sizes = [[1, 5, 4099], [70001, 16], [3, 8192]]
    hyper = [dict(lr=1e-3, beta1=0.9, beta2=0.999, eps=1e-8, weight_decay=0.0),
             dict(lr=3e-4, beta1=0.8, beta2=0.99, eps=1e-6, weight_decay=0.1),
             dict(lr=1e-2, beta1=0.95, beta2=0.9, eps=1e-7, weight_decay=0.01)]
    start = [1, 5, 2]
    dev = "cuda"
    host = [[dict(p=rng.standard_normal(n).astype(np.float32), m=np.zeros(n, np.float32), v=np.zeros(n, np.float32))
             for n in sz] for sz in sizes]
    P = [[torch.from_numpy(t["p"].copy()).to(dev) for t in ten] for ten in host]
    M = [[torch.zeros(len(t["p"]), device=dev) for t in ten] for ten in host]
    V = [[torch.zeros(len(t["p"]), device=dev) for t in ten] for ten in host]
    B = [None, None, [torch.zeros(len(t["p"]), dtype=torch.bfloat16, device=dev) for t in host[2]]]
    ctx = jn.Context()
    for it in range(3):
        grads = [[(rng.standard_normal(len(t["p"])) * 10.0 ** rng.integers(-3, 2)).astype(np.float32)
                  for t in ten] for ten in host]
        Gd = [[torch.from_numpy(g).to(dev) for g in gs] for gs in grads]
        ts = [jn.AdamWTenant(P[k], Gd[k], M[k], V[k], start[k] + it, bf16_out=B[k], **hyper[k]) for k in range(3)]
        ws = torch.empty(jn.jn_adamw_workspace_size(ts), dtype=torch.uint8, device=dev)
        _say(f"adamw step {it}")
        jn.jn_tenant_adamw_step(ctx, ts, ws)
        torch.cuda.synchronize()
        for k in range(3):
            h32 = {n: float(np.float32(x)) for n, x in hyper[k].items()}
            for j, t in enumerate(host[k]):
                ref = optim.adamw_step(t["p"], grads[k][j], t["m"], t["v"], start[k] + it, **h32)
                pg, mg, vg = P[k][j].cpu().numpy(), M[k][j].cpu().numpy(), V[k][j].cpu().numpy()
                check(pg, mg, vg, ref, hyper[k]["lr"], float(np.max(np.abs(grads[k][j]))))
                if B[k] is not None:
                    bits = B[k][j].view(torch.int16).cpu().numpy().view(np.uint16)
                    assert np.array_equal(bits, W.f32_to_bf16_bits(pg))
                # continue from the GPU's state (what the next step reads)
                t["p"], t["m"], t["v"] = pg, mg, vg


def test_adamw_after_group_step_heads(jn):
    """The tiny two-tenant workload: heads fwd/bwd, then one optimizer step per
    tenant from its own gradients; versions advance only for the group."""
    from oracle import optim
    from paper_2607_16074_amd import step as jstep
    wl = W.make_workload(1)
    model, reqs, targets = jstep.from_workload(wl)
    st = jstep.GroupStep(model, [r for r in reqs if r.tenant == 1], targets, [1])   # tenant 1 alone
    st.run()
    before = [t.cpu().numpy().copy() for t in list(st.heads[0].W) + list(st.heads[0].b)]
    grads = [t.cpu().numpy().copy() for t in list(st.ios[0].dW) + list(st.ios[0].db)]
    opt = jstep.TenantOptimizer(st, lr=1e-3, weight_decay=0.01)
    opt.step()
    torch.cuda.synchronize()
    assert opt.versions == {1: 1}
    after = [t.cpu().numpy() for t in list(st.heads[0].W) + list(st.heads[0].b)]
    f = lambda x: float(np.float32(x))  # noqa: E731  (the hyperparameters travel as fp32)
    for p0, g, p1 in zip(before, grads, after):
        ref = optim.adamw_step(p0, g, np.zeros_like(p0), np.zeros_like(p0), 1, f(1e-3), f(0.9), f(0.999), f(1e-8),
                               f(0.01))
        assert np.all(np.abs(p1 - ref[0]) <= 4e-7 * np.abs(ref[0]) + 2e-6 * 1e-3)


def test_adamw_errors_enqueue_nothing(jn):
    ctx = jn.Context()
    p = torch.ones(64, device="cuda")
    g, m, v = torch.ones_like(p), torch.zeros_like(p), torch.zeros_like(p)
    ws = torch.empty(4096, dtype=torch.uint8, device="cuda")
    for kw in ({"step": 0}, {"beta1": 1.5}):
        t = jn.AdamWTenant([p], [g], [m], [v], **{"step": 1, "lr": 1e-3, **kw})
        with pytest.raises(jn.JNError):
            jn.jn_tenant_adamw_step(ctx, [t], ws)
    with pytest.raises(jn.JNError):
        jn.jn_tenant_adamw_step(ctx, [jn.AdamWTenant([p], [g], [m], [v], step=1, lr=1e-3)], ws[:16])
    torch.cuda.synchronize()
    assert torch.equal(p, torch.ones_like(p)) and torch.equal(m, torch.zeros_like(m))
