"""GPU tests of the resident inference plan (jn_infer_plan_*) and of the
collector feeding it (App. A.3 inference queue).

* The decode-only step equals the training path's forward bitwise: the same
  pack, backbone, pool and head-forward kernels on the same rows.
* Actions against the fp64 oracle (isolated per-sample backbone, per-tenant
  head): within 2e-2 max-relative per tenant, end to end through the bf16
  backbone (the training path's head stage is pinned stage-wise at 1e-3).
* A captured HIP graph replays to the eager result bitwise, replay after
  replay, with eager work and new observations in the same input buffers in
  between.
* Batches formed by the collector give every request the actions it gets in
  one large group (results do not depend on batch composition).
* Error statuses enqueue nothing.
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


def maxrel(g, o):
    return float(np.max(np.abs(np.asarray(g, np.float64) - o)) / max(np.max(np.abs(o)), 1e-30))


def test_infer_equals_training_forward_and_oracle(jn):
    from paper_2607_16074_amd import step as jstep
    import oracle
    wl = W.make_workload(1)
    _say("infer vs training forward: config 1")
    model, reqs, targets = jstep.from_workload(wl)
    G = wl.spec.G
    tr = jstep.GroupStep(model, reqs, targets, list(range(G)))
    tr.run()
    inf = jstep.InferStep(model, reqs, list(range(G)))
    inf.launch()
    inf.synchronize()
    torch.cuda.synchronize()
    ref = oracle.step.isolated(wl)
    for k in range(G):
        a = inf.actions[k].cpu().numpy()
        assert np.array_equal(a, tr.ios[k].actions.cpu().numpy()), k
        o = np.asarray(ref["tenants"][k]["actions"], np.float64)
        assert maxrel(a, o) < 2e-2, (k, maxrel(a, o))


def test_graph_replay_matches_eager(jn):
    from paper_2607_16074_amd import step as jstep
    wl = W.make_workload(2)
    _say("graph replay: config-2 model, 4 tenants x 2 samples")
    model, reqs, _ = jstep.from_workload(wl)
    sub = [jn.Request(r.tenant, r.embeds[:2].clone(), r.lengths[:2]) for r in reqs]
    inf = jstep.InferStep(model, sub, list(range(wl.spec.G)))
    inf.launch()
    inf.synchronize()
    eager0 = [a.clone() for a in inf.actions]
    for a in inf.actions:
        a.fill_(float("nan"))
    torch.cuda.synchronize()
    inf.capture()
    gen = torch.Generator(device="cuda").manual_seed(3)
    for rep in range(3):
        if rep > 0:  # new observations in the same input buffers
            for r in sub:
                r.embeds.copy_(torch.randn(r.embeds.shape, device="cuda", generator=gen).to(torch.bfloat16))
        torch.cuda.synchronize()
        inf.replay()
        inf.synchronize()
        replayed = [a.clone() for a in inf.actions]
        # unrelated eager work between replays
        x = torch.randn(512, 512, device="cuda")
        (x @ x).sum().item()
        inf.launch()
        inf.synchronize()
        eager = [a.clone() for a in inf.actions]
        for k in range(len(sub)):
            assert torch.equal(replayed[k], eager[k]), (rep, k)
        if rep == 0:
            for k in range(len(sub)):
                assert torch.equal(eager[k], eager0[k])
        else:
            assert not torch.equal(eager[0], eager0[0])


def test_collector_batches_match_one_group(jn):
    from paper_2607_16074_amd import step as jstep
    wl = W.make_workload(1)
    _say("collector-formed batches: config 1 split into single-sample requests")
    model, reqs, _ = jstep.from_workload(wl)
    # one request per sample, arrival interleaved across the two tenants
    singles = []
    for s in range(8):
        for r in reqs:
            singles.append(jn.Request(r.tenant, r.embeds[s:s + 1].clone(), r.lengths[s:s + 1]))
    full = jstep.InferStep(model, singles, [0, 1])
    full.launch()
    full.synchronize()
    # tenant-order row of each single request in the full group
    row_of = {}
    cnt = [0, 0]
    for i, q in enumerate(singles):
        row_of[i] = (q.tenant, cnt[q.tenant])
        cnt[q.tenant] += 1
    col = jn.Collector(max_batch_samples=5, timeout_us=50)
    for i, q in enumerate(singles):
        col.submit(i, model.prefix_sig, model.backbone.d, 1, 10 * i)
    batches = []
    while True:
        ids = col.poll(10 ** 9)
        if not ids:
            break
        batches.append(ids)
    assert sum(len(b) for b in batches) == len(singles)
    assert [len(b) for b in batches] == [5, 5, 5, 1]
    for ids in batches:
        tens = sorted({singles[i].tenant for i in ids})
        st = jstep.InferStep(model, [singles[i] for i in ids], tens)
        st.launch()
        st.synchronize()
        seen = {g: 0 for g in tens}
        for i in ids:
            g = singles[i].tenant
            k = tens.index(g)
            got = st.actions[k][seen[g]].cpu()
            seen[g] += 1
            tg, row = row_of[i]
            assert torch.equal(got, full.actions[tg][row].cpu()), (ids, i)


def test_errors_enqueue_nothing(jn):
    from paper_2607_16074_amd import step as jstep
    wl = W.make_workload(1)
    _say("infer plan error statuses")
    model, reqs, _ = jstep.from_workload(wl)
    inf = jstep.InferStep(model, reqs, [0, 1])
    with pytest.raises(jn.JNError) as e:
        inf.replay()                      # nothing captured yet
    assert "EINVAL" in str(e.value)
    # a context on the null stream cannot capture
    nullctx = jn.Context(torch.cuda.default_stream())
    with pytest.raises(jn.JNError) as e:
        jn.InferPlan(nullctx, inf.requests, inf.table, model.backbone.d, 1, model.backbone, inf.heads,
                     inf.actions, inf.ws).capture()
    assert "EUNSUPPORTED" in str(e.value)
    # undersized workspace: nothing written
    for a in inf.actions:
        a.fill_(7.0)
    torch.cuda.synchronize()
    small = torch.empty(inf.ws.numel() - 256, dtype=torch.uint8, device="cuda")
    with pytest.raises(jn.JNError) as e:
        jn.InferPlan(inf.ctx, inf.requests, inf.table, model.backbone.d, 1, model.backbone, inf.heads,
                     inf.actions, small)
    assert "ENOSPACE" in str(e.value)
    torch.cuda.synchronize()
    assert all(bool((a == 7.0).all()) for a in inf.actions)
