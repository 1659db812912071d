"""GPU parity of the group-batched step against the fp64 oracle.

Bars: index maps and packed / unpacked rows bit-exact; bf16 outputs (hidden
states, pooled features) within 2e-2 max-relative per sample
(max|gpu - oracle| / max|oracle| over that sample); head outputs, losses and
weight gradients within 1e-3 relative L2 per tensor, checked stage-wise (the
oracle's fp64 head takes the GPU's pooled features).  Grouped execution
must equal isolated per-tenant execution, and padding / arrival order must
not change any sample's result -- bitwise, since every output element is
reduced in an order that does not depend on batch composition.
"""
import dataclasses
import sys

import numpy as np
import pytest

import workloads as W

torch = pytest.importorskip("torch")
pytestmark = pytest.mark.gpu

BF16_TOL = 2e-2
GRAD_TOL = 1e-3


def _say(msg):
    print(msg, flush=True)
    sys.stdout.flush()


@pytest.fixture(scope="module")
def jn():
    if not torch.cuda.is_available():
        pytest.skip("no GPU")
    import paper_2607_16074_amd as lib
    return lib


def run_group(wl, align=1, tenants=None):
    from paper_2607_16074_amd import step as jstep
    model, reqs, targets = jstep.from_workload(wl)
    G = wl.spec.G
    st = jstep.GroupStep(model, reqs, targets, list(range(G)) if tenants is None else tenants, align)
    st.run()
    torch.cuda.synchronize()
    return st


def tenant_order_keys(wl):
    """(request, sample) keys in tenant order (stable by arrival)."""
    return [(r, s) for g in range(wl.spec.G) for r, q in enumerate(wl.requests) if q.tenant == g for s in range(q.n)]


def maxrel(g, o):
    return float(np.max(np.abs(np.asarray(g, np.float64) - o)) / max(np.max(np.abs(o)), 1e-30))


def rel_l2(g, o):
    o = np.asarray(o, np.float64)
    return float(np.linalg.norm(np.asarray(g, np.float64) - o) / max(np.linalg.norm(o), 1e-30))


def bf16_np(t):
    return W.bf16_bits_to_f32(t.contiguous().view(torch.int16).cpu().numpy().view(np.uint16))


def check_heads_stagewise(wl, st):
    import oracle
    pooled = st.pooled.cpu().numpy().astype(np.float64)
    off = 0
    worst = 0.0
    for k, g in enumerate(st.tenants):
        n = sum(q.n for q in wl.requests if q.tenant == g)
        ref = oracle.step.tenant_from_pooled(wl, g, pooled[off: off + n])
        off += n
        io = st.ios[k]
        acts = io.actions.cpu().numpy()
        assert rel_l2(acts, ref["actions"]) < GRAD_TOL, ("actions", g)
        loss = float(io.loss.cpu())
        assert abs(loss - ref["loss"]) <= GRAD_TOL * abs(ref["loss"]), ("loss", g, loss, ref["loss"])
        for layer, (dW, db) in enumerate(ref["grads"]):
            e1 = rel_l2(io.dW[layer].cpu().numpy(), dW)
            e2 = rel_l2(io.db[layer].cpu().numpy(), db)
            worst = max(worst, e1, e2)
            assert e1 < GRAD_TOL and e2 < GRAD_TOL, (g, layer, e1, e2)
    return worst


def check_golden(wl, st, margin, pooled=True):
    """Every tenant of a full-size workload against the stored fp64 oracle
    values (tests/golden/backbone_golden.py): per chosen sample, its stored
    hidden rows, every row's projections and (MLP-head groups) its pooled
    feature, each within the per-sample max-relative bar."""
    import backbone_golden as BG
    gold = BG.load(wl.spec.config_id)
    hid = bf16_np(st.hidden)
    cu = st.packed.map_tensor("cu_seqlens").cpu().numpy()
    res = BG.compare(wl, gold, hid, cu, st.pooled.cpu().numpy() if pooled else None)
    assert res["tenants"] == wl.spec.G
    _say(f"  stored oracle: {res['samples']} samples of {res['tenants']} tenants: rows {res['rows']:.3e} "
         f"projections {res['proj']:.3e} pooled {res['pooled']:.3e}")
    margin(f"cfg{wl.spec.config_id} hidden+pooled, {res['samples']} samples / all {res['tenants']} tenants, max-rel",
           res["worst"], BF16_TOL)
    for g, e in sorted(res["per_tenant"].items()):
        assert e < BF16_TOL, ("tenant", g, e)
    return res


# ------------------------------------------------------------------ pack ---

def _small_spec(d=128, ns=(3, 5, 2), lo=1, hi=40, max_len=48, layers=1, heads=4, ffn=256, glu=False):
    ten = tuple(W.TenantSpec(n, 0, lo, hi, max_len, (d, 64, 6), 3, 2) for n in ns)
    return W.WorkloadSpec(90, W.BackboneSpec(layers, d, heads, ffn, glu), ten, 0, "small")


@pytest.mark.parametrize("align", [1, 16, 64])
def test_pack_unpack_bit_exact(jn, align):
    from oracle import plan as oplan
    from paper_2607_16074_amd import step as jstep
    spec = _small_spec()
    wl = W.make_workload(spec, request_split=(2, 3, 1), request_order=[3, 0, 5, 1, 4, 2])
    _say(f"pack/unpack align={align}")
    st = run_group(wl, align)
    ref = oplan.pack_plan([q.tenant for q in wl.requests], [q.lengths for q in wl.requests],
                          [q.max_len for q in wl.requests], spec.G, align)
    for name in ("seqlens", "cu_seqlens", "sample_request", "sample_local", "sample_tenant", "tenant_sample_off",
                 "tenant_perm", "sample_tenant_rank", "token_sample", "token_pos"):
        got = st.packed.map_tensor(name).cpu().numpy()
        assert np.array_equal(got, ref[name]), name
    tok = st.tokens.view(torch.int16).cpu().numpy().view(np.uint16)
    assert np.array_equal(tok, oplan.pack_tokens(ref, [q.embeds for q in wl.requests]))
    # unpack of the packed tokens restores every valid row and zeroes padding
    outs = [torch.full((q.n, q.max_len, spec.backbone.d), 7, dtype=torch.int16, device="cuda")
            for q in wl.requests]
    jn.jn_unpack(st.ctx, st.packed, st.requests, st.tokens, spec.backbone.d * 2, outs)
    torch.cuda.synchronize()
    for q, o in zip(wl.requests, outs):
        o = o.cpu().numpy().view(np.uint16)
        for s in range(q.n):
            L = q.lengths[s]
            assert np.array_equal(o[s, :L], q.embeds[s, :L])
            assert not o[s, L:].any()
    # a row width that is not a multiple of 16 bytes (4-byte lanes)
    rows = torch.arange(st.T * 3, dtype=torch.int32, device="cuda").view(st.T, 3)
    outs = [torch.full((q.n, q.max_len, 3), -5, dtype=torch.int32, device="cuda") for q in wl.requests]
    jn.jn_unpack(st.ctx, st.packed, st.requests, rows, 12, outs)
    torch.cuda.synchronize()
    back = oplan.unpack_tokens(ref, rows.cpu().numpy(), [(q.n, q.max_len, 3) for q in wl.requests])
    for o, b in zip(outs, back):
        assert np.array_equal(o.cpu().numpy(), b)


def test_pack_config_workloads(jn):
    """Bit-exact packing of the tiny and the 4-tenant configurations."""
    from oracle import plan as oplan
    for cfg in (1, 2):
        wl = W.make_workload(cfg, with_weights=False)
        wl.layers = [W.layer_weights(W.config_spec(cfg), 0)]  # one layer is enough to build the step
        _say(f"pack config {cfg}")
        from paper_2607_16074_amd import step as jstep
        model, reqs, targets = jstep.from_workload(wl)
        st = jstep.GroupStep(model, reqs, targets, list(range(wl.spec.G)))
        torch.cuda.synchronize()
        ref = oplan.pack_plan([q.tenant for q in wl.requests], [q.lengths for q in wl.requests],
                              [q.max_len for q in wl.requests], wl.spec.G, 1)
        tok = st.tokens.view(torch.int16).cpu().numpy().view(np.uint16)
        assert np.array_equal(tok, oplan.pack_tokens(ref, [q.embeds for q in wl.requests]))
        for name in ("cu_seqlens", "tenant_perm", "token_sample", "token_pos"):
            assert np.array_equal(st.packed.map_tensor(name).cpu().numpy(), ref[name]), (cfg, name)


# -------------------------------------------------------------- backbone ---

def _check_backbone(wl, st, keys=None):
    import oracle
    iso = oracle.step.isolated(wl, samples=keys, heads=False)
    hid = bf16_np(st.hidden)
    cu = st.packed.map_tensor("cu_seqlens").cpu().numpy()
    flat = [(r, s) for r, q in enumerate(wl.requests) for s in range(q.n)]
    worst = 0.0
    for i, key in enumerate(flat):
        if key not in iso["hidden"]:
            continue
        z = iso["hidden"][key]
        g = hid[cu[i]: cu[i] + z.shape[0]]
        e = maxrel(g, z)
        worst = max(worst, e)
        assert e < BF16_TOL, (key, e)
        # alignment rows of the hidden output are zero
        assert not hid[cu[i] + z.shape[0]: cu[i + 1]].any()
    return worst


@pytest.mark.parametrize("variant", ["norm_only", "attention_only", "full", "full_glu"])
def test_backbone_variants(jn, variant):
    """Isolate the pieces: zeroing W_o and W_down leaves the final norm of the
    input; zeroing W_down leaves the attention branch; then everything."""
    spec = _small_spec(layers=2, glu=variant == "full_glu", ns=(4, 3), hi=150, max_len=160)
    wl = W.make_workload(spec, request_split=(2, 1))
    for L in wl.layers:
        if variant == "norm_only":
            L["wo"][:] = 0
        if variant in ("norm_only", "attention_only"):
            L["w_down"][:] = 0
        # larger weights than the workload default so every branch matters
        for k in ("wqkv", "wo", "w_up", "w_down", "w_gate"):
            if k in L and L[k].any():
                L[k][:] = W.f32_to_bf16_bits(W.bf16_bits_to_f32(L[k]) * 4.0)
    _say(f"backbone variant {variant}")
    st = run_group(wl, align=16)
    worst = _check_backbone(wl, st)
    _say(f"  worst hidden max-rel {worst:.3e}")


@pytest.mark.parametrize("hd", [32, 64, 128, 256])
def test_attention_head_dims(jn, hd):
    """Every head width of the attention kernel, ragged lengths (1 .. 300)."""
    d = 512
    spec = _small_spec(d=d, heads=d // hd, ns=(5, 4), lo=1, hi=300, max_len=300, layers=1, ffn=256)
    wl = W.make_workload(spec, request_split=(2, 2), request_order=[2, 0, 3, 1])
    wl.requests[0].lengths[0] = 1       # a one-token sample
    wl.requests[1].lengths[-1] = 300    # a full-length sample
    for L in wl.layers:
        L["w_down"][:] = 0
        L["wqkv"][:] = W.f32_to_bf16_bits(W.bf16_bits_to_f32(L["wqkv"]) * 3.0)
    _say(f"attention hd={hd}")
    st = run_group(wl, align=1)
    worst = _check_backbone(wl, st)
    _say(f"  worst hidden max-rel {worst:.3e}")


# ------------------------------------------------------------ end to end ---

def test_config1_end_to_end(jn, margin):
    import oracle
    wl = W.make_workload(1)
    _say("config 1")
    st = run_group(wl)
    worst = _check_backbone(wl, st)
    ref = oracle.step.isolated(wl)
    pooled = st.pooled.cpu().numpy()
    for k, key in enumerate(tenant_order_keys(wl)):
        assert maxrel(pooled[k], ref["pooled"][key]) < BF16_TOL
    gw = check_heads_stagewise(wl, st)
    # end-to-end head gradients (informational bound, bf16 backbone)
    for k, g in enumerate(st.tenants):
        for layer, (dW, db) in enumerate(ref["tenants"][g]["grads"]):
            assert rel_l2(st.ios[k].dW[layer].cpu().numpy(), dW) < BF16_TOL
    margin("cfg1 hidden, all samples, max-rel", worst, BF16_TOL)
    margin("cfg1 head stage, rel-L2", gw, GRAD_TOL)
    _say(f"  hidden {worst:.3e}  head grads (stage-wise) {gw:.3e}")


@pytest.mark.parametrize("cfg", [2, 5])
def test_config_sampled_end_to_end(jn, cfg, margin):
    """Full-size 12-layer d768 configurations: every tenant against the
    stored oracle values (config 2: first and last sample of each of the 4
    tenants; config 5: one sample of each of the 32 tenants), the oracle run
    here on sampled samples (first and last of every fourth tenant, all rows
    elementwise), and every tenant's head stage."""
    wl = W.make_workload(cfg)
    _say(f"config {cfg}: N={sum(q.n for q in wl.requests)}")
    st = run_group(wl)
    check_golden(wl, st, margin)
    keys = []
    for r, q in enumerate(wl.requests):
        if r % 4 == 0:
            keys += [(r, 0), (r, q.n - 1)] if q.n > 1 else [(r, 0)]
    keys = keys[:8]
    worst = _check_backbone(wl, st, keys)
    gw = check_heads_stagewise(wl, st)
    margin(f"cfg{cfg} hidden, {len(keys)} samples all rows, max-rel", worst, BF16_TOL)
    margin(f"cfg{cfg} head stage (actions, dW, db), all tenants, rel-L2", gw, GRAD_TOL)
    _say(f"  hidden {worst:.3e} on {len(keys)} samples, head grads {gw:.3e}")


def test_config3_sampled_end_to_end(jn, margin):
    """The 2B-shaped configuration (18-layer d2048 GeGLU, 8 tenants x 32) in
    the launch configuration the benchmark times: one sample of every tenant
    against the stored oracle values (including the batch's last sample,
    whose rows run in the GEMMs' row-split tail); the oracle run here on the
    first sample of the first tenant and the last sample of the last tenant
    (all rows elementwise, each ~6 s of fp64 work); head stage of all eight
    tenants."""
    wl = W.make_workload(3)
    _say(f"config 3: N={sum(q.n for q in wl.requests)}")
    st = run_group(wl)
    check_golden(wl, st, margin)
    keys = [(0, 0), (len(wl.requests) - 1, wl.requests[-1].n - 1)]
    worst = _check_backbone(wl, st, keys)
    gw = check_heads_stagewise(wl, st)
    margin("cfg3 hidden, 2 samples all rows, max-rel", worst, BF16_TOL)
    margin("cfg3 head stage (actions, dW, db), all 8 tenants, rel-L2", gw, GRAD_TOL)
    _say(f"  hidden {worst:.3e} on {len(keys)} samples, head grads {gw:.3e}")


def test_split_k_short_batch_2b(jn):
    """A one-sample batch on the 2B-shaped backbone: the O projection (K=2048)
    and the down projection (K=16384) have too few tiles for the GPU and run
    split over K (2 and 4 ranges, fp32 partials added in range order).  The
    hidden rows match the oracle's isolated run of that sample, the head
    stage matches stage-wise, and two runs are bitwise equal."""
    import oracle
    from paper_2607_16074_amd import Request
    from paper_2607_16074_amd import step as jstep
    import paper_2607_16074_amd._abi as abi  # noqa: F401
    wl = W.make_workload(3)
    model, reqs, targets = jstep.from_workload(wl)
    one = [Request(reqs[0].tenant, reqs[0].embeds[:1], reqs[0].lengths[:1])]
    g0 = reqs[0].tenant
    _say(f"split-K: one sample of tenant {g0}, {int(one[0].lengths[0])} rows, 18-layer d2048")
    st = jstep.GroupStep(model, one, {g0: targets[g0][:1]}, [g0])
    st.run()
    torch.cuda.synchronize()
    h1 = st.hidden.clone()
    st.run()
    torch.cuda.synchronize()
    assert torch.equal(h1, st.hidden)
    ref = oracle.step.isolated(wl, samples=[(0, 0)], heads=False)
    z = ref["hidden"][(0, 0)]
    e = maxrel(bf16_np(st.hidden)[: z.shape[0]], z)
    _say(f"  hidden max-rel {e:.3e}")
    assert e < BF16_TOL
    pooled = st.pooled.cpu().numpy().astype(np.float64)
    tres = oracle.heads.tenant_step(pooled, wl.heads[g0], np.asarray(targets[g0][:1], np.float64))
    assert rel_l2(st.ios[0].actions.cpu().numpy(), tres["actions"]) < GRAD_TOL


def test_ragged_weight_widths_on_the_large_tile(jn):
    """The 256x256 GEMM tile with weight widths that are not multiples of 256
    (QKV 1152, O and down 384, so their last column tile is half outside):
    ~77K tokens make the tile planner choose that tile for these projections,
    so its load clamps and the staged epilogues' column bounds run on partial
    tiles.  Oracle on the first, a middle and the last sample."""
    ten = tuple(W.TenantSpec(130, 256, 16, 64, 320, (384, 64, 6), 3, 2) for _ in range(2))
    spec = W.WorkloadSpec(94, W.BackboneSpec(2, 384, 6, 1408, True), ten, 0, "ragged widths")
    wl = W.make_workload(spec)
    T = int(sum(int(q.lengths.sum()) for q in wl.requests))
    _say(f"ragged widths: d=384 ffn=1408 GeGLU, {T} tokens")
    st = run_group(wl)
    last = len(wl.requests) - 1
    keys = [(0, 0), (0, wl.requests[0].n // 2), (last, wl.requests[last].n - 1)]
    worst = _check_backbone(wl, st, keys)
    _say(f"  worst hidden max-rel {worst:.3e}")


def test_single_sample_of_length_one(jn):
    """The smallest batch: one tenant, one request, one sample of one token,
    padded to a canonical length of 4 (degenerate attention: softmax over one
    key; pooling over one row)."""
    import oracle
    ten = (W.TenantSpec(1, 0, 1, 1, 4, (128, 64, 6), 3, 2),)
    spec = W.WorkloadSpec(92, W.BackboneSpec(2, 128, 4, 256, False), ten, 0, "single")
    wl = W.make_workload(spec)
    assert wl.requests[0].lengths.tolist() == [1]
    _say("single sample, length 1")
    st = run_group(wl, align=16)
    _check_backbone(wl, st)
    ref = oracle.step.isolated(wl)
    assert maxrel(st.pooled.cpu().numpy()[0], ref["pooled"][(0, 0)]) < BF16_TOL
    check_heads_stagewise(wl, st)


def test_grouped_equals_isolated_bitwise(jn):
    """The defining invariant (Sec. 5.2): grouping changes no tenant's result."""
    _grouped_equals_isolated(W.make_workload(2))


def test_grouped_equals_isolated_bitwise_geglu(jn):
    """The same invariant across GEMM loops and tile shapes: a GeGLU backbone
    where the 2-sample tenant's rows (first in the packed batch) go through
    the 256x256 ring loop in the grouped run (~18K tokens) and through 128x128
    tiles of the interleaved loop in its own run (~600 tokens).  ffn = 1920
    keeps every launch of both runs unsplit over K (a K split adds fp32
    partials in another order, the one documented exception)."""
    ten = (W.TenantSpec(2, 256, 16, 64, 320, (512, 64, 6), 3, 2), W.TenantSpec(60, 256, 16, 64, 320, (512, 64, 6), 3, 2))
    spec = W.WorkloadSpec(95, W.BackboneSpec(2, 512, 4, 1920, True), ten, 0, "geglu bitwise")
    _say("grouped == isolated, GeGLU backbone, 2 + 60 samples")
    _grouped_equals_isolated(W.make_workload(spec))


def test_head_k_split_ragged(jn):
    """Head GEMMs whose contraction is split into K ranges with ragged ends
    (K = 512, 600, 1030: ranges of 256, 320 and 288 columns, the last one
    short) and a tenant of 40 samples (two row tiles): stage-wise against the
    oracle at the head bar, and grouped == isolated bitwise (the split depends
    on K only)."""
    ten = (W.TenantSpec(3, 0, 1, 30, 40, (512, 600, 1030, 6), 3, 2),
           W.TenantSpec(40, 0, 1, 30, 40, (512, 1030, 6), 3, 2),
           W.TenantSpec(5, 0, 1, 30, 40, (512, 64, 6), 3, 2))
    spec = W.WorkloadSpec(96, W.BackboneSpec(1, 512, 4, 256, False), ten, 0, "head k split")
    wl = W.make_workload(spec)
    _say("heads with ragged K ranges: 3 + 40 + 5 samples")
    st = run_group(wl)
    check_heads_stagewise(wl, st)
    _grouped_equals_isolated(wl)


def _grouped_equals_isolated(wl):
    from paper_2607_16074_amd import step as jstep
    model, reqs, targets = jstep.from_workload(wl)
    grouped = jstep.GroupStep(model, reqs, targets, list(range(wl.spec.G)))
    grouped.run()
    iso = jstep.isolated_runs(model, reqs, targets, list(range(wl.spec.G)), ctx=grouped.ctx)
    for s in iso:
        s.run()
    torch.cuda.synchronize()
    off = 0
    for g, s in enumerate(iso):
        n = s.N
        assert torch.equal(grouped.pooled[off: off + n], s.pooled), g
        assert torch.equal(grouped.ios[g].loss, s.ios[0].loss)
        for a, b in zip(grouped.ios[g].dW + grouped.ios[g].db, s.ios[0].dW + s.ios[0].db):
            assert torch.equal(a, b), g
        off += n
    # unpacked hidden states per request are identical too
    for r, q in enumerate(wl.requests):
        assert torch.equal(grouped.out_hidden[r], iso[q.tenant].out_hidden[0]), r


def test_padding_and_order_invariance_bitwise(jn):
    wl = W.make_workload(1, request_split=(2, 2))
    a = run_group(wl, align=1)
    b = run_group(wl, align=64)
    wlp = W.make_workload(1, request_split=(2, 2), request_order=[3, 1, 0, 2])
    c = run_group(wlp, align=16)
    # alignment padding: everything bitwise equal
    assert torch.equal(a.pooled, b.pooled)
    for g in range(2):
        assert torch.equal(a.ios[g].loss, b.ios[g].loss)
        assert all(torch.equal(x, y) for x, y in zip(a.ios[g].dW, b.ios[g].dW))
    for r in range(4):
        assert torch.equal(a.out_hidden[r], b.out_hidden[r])
    # arrival order: each sample's rows bitwise equal; a tenant's loss and
    # gradients sum its rows in the new order (fp32 rounding only)
    perm = [3, 1, 0, 2]
    for new_r, old_r in enumerate(perm):
        assert torch.equal(c.out_hidden[new_r], a.out_hidden[old_r])
    ka = {key: k for k, key in enumerate(tenant_order_keys(wl))}
    for k, (r, s) in enumerate(tenant_order_keys(wlp)):
        assert torch.equal(c.pooled[k], a.pooled[ka[(perm[r], s)]])
    for g in range(2):
        assert abs(float(c.ios[g].loss) - float(a.ios[g].loss)) <= 1e-5 * abs(float(a.ios[g].loss))
        for x, y in zip(a.ios[g].dW, c.ios[g].dW):
            assert rel_l2(y.cpu().numpy(), x.cpu().numpy().astype(np.float64)) < 1e-5


def test_determinism(jn):
    wl = W.make_workload(1)
    st = run_group(wl)
    h1 = st.hidden.clone()
    g1 = [x.clone() for x in st.ios[1].dW]
    st.run()
    torch.cuda.synchronize()
    assert torch.equal(h1, st.hidden)
    assert all(torch.equal(a, b) for a, b in zip(g1, st.ios[1].dW))


def test_errors_enqueue_nothing(jn):
    """A non-OK status leaves every output untouched."""
    from paper_2607_16074_amd import step as jstep
    wl = W.make_workload(1)
    st = run_group(wl)
    before = st.hidden.clone()
    small = torch.empty(16, dtype=torch.uint8, device="cuda")
    with pytest.raises(jn.JNError) as e:
        jn.jn_backbone_forward(st.ctx, st.model.backbone, st.packed, st.hidden, small)
    assert e.value.status == jn._abi.JN_ENOSPACE
    with pytest.raises(jn.JNError) as e:
        jn.jn_tenant_heads_fwd_bwd(st.ctx, st.packed, st.hidden, st.heads[:1], st.ios[:1], st.hd_ws)
    assert e.value.status == jn._abi.JN_EINVAL

    # unpack with the same samples split differently over the requests: the
    # packed sample positions would index past a request's buffer
    from paper_2607_16074_amd import Request
    resplit = [Request(0, st.requests[0].embeds[:5], st.requests[0].lengths[:5]),
               Request(1, torch.cat([st.requests[0].embeds[5:], st.requests[1].embeds]),
                       np.concatenate([st.requests[0].lengths[5:], st.requests[1].lengths]),
                       st.requests[1].max_len)]
    outs = [torch.full((len(q.lengths), q.max_len, st.model.backbone.d), 3, dtype=torch.int16, device="cuda")
            for q in resplit]
    before_out = [o.clone() for o in outs]
    with pytest.raises(jn.JNError) as e:
        jn.jn_unpack(st.ctx, st.packed, resplit, st.hidden, st.model.backbone.d * 2, outs)
    assert e.value.status == jn._abi.JN_ESHAPE

    class _Wide:  # the same layers described with a width beyond the kernels' range
        struct = jn._abi.jn_backbone.from_buffer_copy(st.model.backbone.struct)
    _Wide.struct.d, _Wide.struct.n_heads = 4224, 33
    with pytest.raises(jn.JNError) as e:
        jn.jn_backbone_forward(st.ctx, _Wide, st.packed, st.hidden, small)
    assert e.value.status == jn._abi.JN_EUNSUPPORTED
    torch.cuda.synchronize()
    assert torch.equal(before, st.hidden)
    assert all(torch.equal(a, b) for a, b in zip(outs, before_out))
