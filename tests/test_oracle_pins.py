"""Pins of the fp64 oracle against facts outside the oracle itself.

Each test ties an oracle function to a closed form, an identity, a special
case that reduces to a library routine (scipy / torch float64 on the CPU),
brute force on tiny inputs, finite differences, or an invariant the paper
fixes for group batching (Sec. 5.2: grouped execution only removes repeated
base-model work; App. A.3: features are split back by the recorded slices,
nothing is averaged across tenants).
"""
import dataclasses

import numpy as np
import pytest
import scipy.special
import torch
import torch.nn.functional as F

import oracle
import workloads as W
from oracle import backbone as bb
from oracle import heads as hd
from oracle import plan as pl
from oracle import step as st

RTOL_F64 = 1e-12


def tiny_spec(glu=False, layers=2, d=16, heads=2, ffn=32, ns=(3, 2), lens=(5, 9), max_len=12, seed=0):
    bbs = W.BackboneSpec(layers=layers, d=d, heads=heads, ffn=ffn, glu=glu)
    ten = []
    for g, n in enumerate(ns):
        a, c = (3, 2) if g % 2 == 0 else (2, 1)
        ten.append(W.TenantSpec(n, lens[0] - 1, 1, lens[1] - lens[0] + 1, max_len, (d, 8, a * c), a, c))
    return W.WorkloadSpec(99, bbs, tuple(ten), seed, "tiny")


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


# ---------------------------------------------------------------- elementwise pieces

def test_bf16_widening_known_bits():
    bits = np.array([0x0000, 0x3F80, 0xC000, 0x3F81, 0x4049, 0x0001], dtype=np.uint16)
    want = [0.0, 1.0, -2.0, 1.0078125, 3.140625, 2.0 ** -133]
    assert bb.bf16_to_f64(bits).tolist() == want


def test_rmsnorm_constant_row_and_scale_invariance():
    d, eps = 64, 1e-6
    for c in (-3.0, 0.5, 7.0):
        x = np.full((1, d), c)
        g = np.linspace(0.5, 2.0, d)
        np.testing.assert_allclose(bb.rms_norm(x, g, eps)[0], c / np.sqrt(c * c + eps) * g, rtol=1e-15)
    rng = np.random.default_rng(1)
    x = rng.standard_normal((5, d))
    y = bb.rms_norm(x, np.ones(d), 0.0)
    np.testing.assert_allclose(np.mean(y * y, axis=1), 1.0, rtol=1e-13)
    np.testing.assert_allclose(bb.rms_norm(1e3 * x, np.ones(d), 0.0), y, rtol=1e-12)
    # torch's own RMSNorm
    t = F.rms_norm(torch.from_numpy(x), (d,), torch.from_numpy(np.full(d, 1.5)), eps=1e-6).numpy()
    np.testing.assert_allclose(bb.rms_norm(x, np.full(d, 1.5), 1e-6), t, rtol=1e-12)


def test_gelu_identities_and_library():
    u = np.linspace(-8, 8, 2001)
    # tanh form satisfies gelu(u) - gelu(-u) == u exactly (odd part is u/2)
    np.testing.assert_allclose(bb.gelu(u) - bb.gelu(-u), u, atol=1e-14)
    assert bb.gelu(np.array([0.0]))[0] == 0.0
    # close to the exact GELU u * Phi(u); the tanh form's error stays below 1e-3
    exact = u * scipy.special.ndtr(u)
    assert np.max(np.abs(bb.gelu(u) - exact)) < 1e-3
    # torch's tanh-approximate GELU
    t = F.gelu(torch.from_numpy(u), approximate="tanh").numpy()
    np.testing.assert_allclose(bb.gelu(u), t, rtol=1e-12, atol=1e-15)


def test_gelu_grad_finite_difference():
    u = np.linspace(-6, 6, 1201)
    h = 1e-5
    fd = (bb.gelu(u + h) - bb.gelu(u - h)) / (2 * h)
    np.testing.assert_allclose(bb.gelu_grad(u), fd, atol=1e-9)
    assert bb.gelu_grad(np.array([0.0]))[0] == 0.5


def test_softmax_rows():
    rng = np.random.default_rng(2)
    s = rng.standard_normal((4, 9)) * 5
    p = bb.softmax_rows(s)
    np.testing.assert_allclose(p.sum(axis=1), 1.0, rtol=1e-15)
    np.testing.assert_allclose(bb.softmax_rows(s + 123.0), p, rtol=1e-12)
    assert bb.softmax_rows(np.array([[42.0]]))[0, 0] == 1.0
    np.testing.assert_allclose(p, scipy.special.softmax(s, axis=1), rtol=1e-13)


# ---------------------------------------------------------------- attention

@pytest.mark.parametrize("L,d,H", [(1, 8, 2), (5, 16, 2), (13, 32, 4)])
def test_attention_against_torch_sdpa(L, d, H):
    rng = np.random.default_rng(L)
    q, k, v = (rng.standard_normal((L, d)) for _ in range(3))
    hdim = d // H
    tq, tk, tv = (torch.from_numpy(a).reshape(L, H, hdim).transpose(0, 1).contiguous() for a in (q, k, v))
    ref = F.scaled_dot_product_attention(tq, tk, tv).transpose(0, 1).reshape(L, d).numpy()
    np.testing.assert_allclose(bb.attention(q, k, v, H), ref, rtol=1e-11, atol=1e-13)


def test_attention_special_cases():
    rng = np.random.default_rng(3)
    L, d, H = 7, 12, 3
    q, k, v = (rng.standard_normal((L, d)) for _ in range(3))
    # zero queries: every row is the mean of the sample's values
    out = bb.attention(np.zeros((L, d)), k, v, H)
    np.testing.assert_allclose(out, np.broadcast_to(v.mean(axis=0), (L, d)), rtol=1e-13)
    # one row: output equals v
    np.testing.assert_allclose(bb.attention(q[:1], k[:1], v[:1], H), v[:1], rtol=1e-15)
    # no positions: permuting the rows permutes the outputs
    p = rng.permutation(L)
    np.testing.assert_allclose(bb.attention(q[p], k[p], v[p], H), bb.attention(q, k, v, H)[p], rtol=1e-12)
    # a dominant key selects its value row, per head
    k2 = k.copy()
    big = np.zeros(d)
    big[: d // H] = 1.0
    qq = np.tile(big * 60, (L, 1))
    k2[4] = big * 60
    out = bb.attention(qq, k2, v, H)
    np.testing.assert_allclose(out[:, : d // H], np.broadcast_to(v[4, : d // H], (L, d // H)), rtol=1e-9)


# ---------------------------------------------------------------- layer / backbone

def _torch_layer(x, lw, H, eps):
    """Same block composed from torch float64 library routines."""
    t = lambda a: torch.from_numpy(np.ascontiguousarray(a))  # noqa: E731
    x = t(x)
    d = x.shape[1]
    h = F.rms_norm(x, (d,), t(lw.g1), eps=eps)
    qkv = F.linear(h, t(lw.wqkv))
    L = x.shape[0]
    q, k, v = (qkv[:, i * d:(i + 1) * d].reshape(L, H, d // H).transpose(0, 1) for i in range(3))
    a = F.scaled_dot_product_attention(q, k, v).transpose(0, 1).reshape(L, d)
    x = x + F.linear(a, t(lw.wo))
    h = F.rms_norm(x, (d,), t(lw.g2), eps=eps)
    if lw.w_gate is None:
        m = F.gelu(F.linear(h, t(lw.w_up)), approximate="tanh")
    else:
        m = F.gelu(F.linear(h, t(lw.w_gate)), approximate="tanh") * F.linear(h, t(lw.w_up))
    return (x + F.linear(m, t(lw.w_down))).numpy()


@pytest.mark.parametrize("glu", [False, True])
def test_layer_against_torch_float64(glu):
    spec = tiny_spec(glu=glu, d=32, heads=4, ffn=48)
    w = W.layer_weights(spec, 0)
    rng = np.random.default_rng(5)
    w["g1"] = W.f32_to_bf16_bits(rng.uniform(0.5, 1.5, 32).astype(np.float32))
    w["g2"] = W.f32_to_bf16_bits(rng.uniform(0.5, 1.5, 32).astype(np.float32))
    # larger weights than the workload's so every term matters
    for key in ("wqkv", "wo", "w_up", "w_down") + (("w_gate",) if glu else ()):
        w[key] = W.f32_to_bf16_bits(rng.standard_normal(w[key].shape).astype(np.float32) * 0.3)
    lw = bb.LayerF64(w, glu)
    x = rng.standard_normal((9, 32))
    np.testing.assert_allclose(bb.layer_forward(x, lw, 4, 1e-6), _torch_layer(x, lw, 4, 1e-6), rtol=1e-10, atol=1e-11)


def test_layer_residual_only_when_outputs_zero():
    spec = tiny_spec()
    w = W.layer_weights(spec, 0)
    w["wo"] = np.zeros_like(w["wo"])
    w["w_down"] = np.zeros_like(w["w_down"])
    lw = bb.LayerF64(w, False)
    x = np.random.default_rng(6).standard_normal((4, 16))
    assert np.array_equal(bb.layer_forward(x, lw, 2, 1e-6), x)


def test_backbone_zero_blocks_is_final_norm_of_input():
    spec = tiny_spec(layers=3)
    wl = W.make_workload(spec)
    for lw in wl.layers:
        lw["wo"][:] = 0
        lw["w_down"][:] = 0
    x = wl.requests[0].embeds[1, : wl.requests[0].lengths[1]]
    z = bb.backbone_forward([x], lambda l: wl.layers[l], 3, 2, False, 1e-6, wl.gf)[0]
    x64 = bb.bf16_to_f64(x)
    want = x64 / np.sqrt(np.mean(x64 ** 2, axis=1, keepdims=True) + 1e-6)
    np.testing.assert_allclose(z, want, rtol=1e-14)


# ---------------------------------------------------------------- grouped == isolated

@pytest.mark.parametrize("glu,align", [(False, 1), (True, 4), (False, 16)])
def test_packed_block_diagonal_equals_isolated(glu, align):
    wl = W.make_workload(tiny_spec(glu=glu), request_split=(2, 1))
    iso = st.isolated(wl, heads=False)
    packed = st.packed_block_diagonal(wl, align=align)
    keys = [(r, s) for r, req in enumerate(wl.requests) for s in range(req.n)]
    assert len(keys) == len(packed)
    for key, zp in zip(keys, packed):
        assert rel(zp, iso["hidden"][key]) < RTOL_F64


def test_padding_invariance():
    spec = tiny_spec(max_len=12)
    wl = W.make_workload(spec)
    base = st.isolated(wl)
    # wider canonical padding with garbage filler
    spec2 = dataclasses.replace(spec, tenants=tuple(dataclasses.replace(t, max_len=20) for t in spec.tenants))
    wl2 = W.make_workload(spec2)
    for r, (a, b) in enumerate(zip(wl.requests, wl2.requests)):
        b.embeds[:] = W.f32_to_bf16_bits(np.full(b.embeds.shape, 1e4, np.float32))
        b.embeds[:, :12] = a.embeds
        assert np.array_equal(a.lengths, b.lengths)
    other = st.isolated(wl2)
    for k in base["hidden"]:
        assert np.array_equal(base["hidden"][k], other["hidden"][k])
    for g in base["tenants"]:
        assert base["tenants"][g]["loss"] == other["tenants"][g]["loss"]


def test_request_permutation_invariance():
    spec = tiny_spec(ns=(4, 3))
    wl = W.make_workload(spec, request_split=(2, 2))
    wlp = W.make_workload(spec, request_split=(2, 2), request_order=[3, 0, 2, 1])
    a, b = st.isolated(wl), st.isolated(wlp)
    for g in a["tenants"]:
        ta, tb = a["tenants"][g], b["tenants"][g]
        assert abs(ta["loss"] - tb["loss"]) <= 1e-12 * abs(ta["loss"])
        for (dwa, dba), (dwb, dbb) in zip(ta["grads"], tb["grads"]):
            assert rel(dwb, dwa) < 1e-12 and rel(dbb, dba) < 1e-12


def test_tenant_isolation():
    spec = tiny_spec(ns=(3, 3))
    wl = W.make_workload(spec)
    a = st.isolated(wl)
    wl.requests[0].embeds[:] = W.f32_to_bf16_bits(np.random.default_rng(9).standard_normal(
        wl.requests[0].embeds.shape).astype(np.float32))
    wl.targets[0] = wl.targets[0] + 1.0
    b = st.isolated(wl)
    ta, tb = a["tenants"][1], b["tenants"][1]
    assert ta["loss"] == tb["loss"]
    for (x, y), (u, v) in zip(ta["grads"], tb["grads"]):
        assert np.array_equal(x, u) and np.array_equal(y, v)
    assert a["tenants"][0]["loss"] != b["tenants"][0]["loss"]


# ---------------------------------------------------------------- heads

def _tiny_head(rng, dims=(6, 5, 4, 3)):
    return [(rng.standard_normal((o, i)), rng.standard_normal(o)) for i, o in zip(dims[:-1], dims[1:])]


def test_head_grads_central_differences():
    rng = np.random.default_rng(11)
    layers = _tiny_head(rng)
    P = rng.standard_normal((4, 6))
    tgt = rng.standard_normal((4, 3))
    res = hd.tenant_step(P, layers, tgt)
    h = 1e-6
    for k, (Wk, bk) in enumerate(layers):
        for arr, g in ((Wk, res["grads"][k][0]), (bk, res["grads"][k][1])):
            fd = np.zeros_like(arr)
            for idx in np.ndindex(arr.shape):
                old = arr[idx]
                arr[idx] = old + h
                lp = hd.tenant_step(P, layers, tgt)["loss"]
                arr[idx] = old - h
                lm = hd.tenant_step(P, layers, tgt)["loss"]
                arr[idx] = old
                fd[idx] = (lp - lm) / (2 * h)
            assert np.max(np.abs(fd - g)) <= 1e-7 * max(1.0, np.max(np.abs(g)))


def test_head_against_torch_autograd():
    rng = np.random.default_rng(12)
    layers = _tiny_head(rng, (8, 7, 5))
    P = rng.standard_normal((6, 8))
    tgt = rng.standard_normal((6, 5))
    res = hd.tenant_step(P, layers, tgt)
    tl = [(torch.tensor(Wk, requires_grad=True), torch.tensor(bk, requires_grad=True)) for Wk, bk in layers]
    x = torch.from_numpy(P)
    for k, (Wk, bk) in enumerate(tl):
        x = F.linear(x, Wk, bk)
        if k + 1 < len(tl):
            x = F.gelu(x, approximate="tanh")
    loss = F.mse_loss(x, torch.from_numpy(tgt))
    loss.backward()
    assert abs(loss.item() - res["loss"]) < 1e-13
    np.testing.assert_allclose(res["actions"], x.detach().numpy(), rtol=1e-13)
    for (Wk, bk), (gw, gb) in zip(tl, res["grads"]):
        np.testing.assert_allclose(gw, Wk.grad.numpy(), rtol=1e-11, atol=1e-15)
        np.testing.assert_allclose(gb, bk.grad.numpy(), rtol=1e-11, atol=1e-15)


def test_head_closed_forms():
    rng = np.random.default_rng(13)
    layers = [(np.zeros((5, 4)), np.zeros(5)), (np.zeros((3, 5)), np.array([1.0, -2.0, 0.5]))]
    P = rng.standard_normal((7, 4))
    Z, X, Y = hd.head_forward(P, layers)
    assert np.array_equal(Y, np.broadcast_to([1.0, -2.0, 0.5], (7, 3)))
    # loss of an exact prediction is 0, of a unit offset is 1
    assert hd.mse_loss(Y, Y.copy())[0] == 0.0
    assert hd.mse_loss(Y, Y - 1.0)[0] == 1.0
    # a single linear layer: dW = (2/n) (Y - t)^T P, db = column sums
    Wl, bl = rng.standard_normal((3, 4)), rng.standard_normal(3)
    tgt = rng.standard_normal((7, 3))
    res = hd.tenant_step(P, [(Wl, bl)], tgt)
    E = P @ Wl.T + bl - tgt
    np.testing.assert_allclose(res["grads"][0][0], 2 * E.T @ P / E.size, rtol=1e-13)
    np.testing.assert_allclose(res["grads"][0][1], 2 * E.sum(axis=0) / E.size, rtol=1e-13)


# ---------------------------------------------------------------- plan

def _meta(wl):
    return ([r.tenant for r in wl.requests], [r.lengths.tolist() for r in wl.requests],
            [r.max_len for r in wl.requests])


@pytest.mark.parametrize("align", [1, 4, 16, 64])
def test_plan_roundtrip_and_structure(align):
    spec = tiny_spec(ns=(4, 3))
    wl = W.make_workload(spec, request_split=(2, 2), request_order=[1, 3, 0, 2])
    t, lens, ml = _meta(wl)
    p = pl.pack_plan(t, lens, ml, spec.G, align)
    flat = [L for ls in lens for L in ls]
    assert p["N"] == len(flat)
    steps = np.diff(p["cu_seqlens"])
    assert np.array_equal(steps, -(-np.array(flat) // align) * align)
    assert np.array_equal(p["tenant_perm"], np.argsort(p["sample_tenant"], kind="stable"))
    assert np.array_equal(p["sample_tenant_rank"][p["tenant_perm"]], np.arange(p["N"]))
    assert np.array_equal(np.diff(p["tenant_sample_off"]), np.bincount(p["sample_tenant"], minlength=spec.G))
    seen = {(int(i), int(j)) for i, j in zip(p["token_sample"], p["token_pos"]) if i >= 0}
    assert seen == {(i, j) for i, L in enumerate(flat) for j in range(L)}
    tok = pl.pack_tokens(p, [r.embeds for r in wl.requests])
    back = pl.unpack_tokens(p, tok, [r.embeds.shape for r in wl.requests])
    for r, req in enumerate(wl.requests):
        for s in range(req.n):
            L = req.lengths[s]
            assert np.array_equal(back[r][s, :L], req.embeds[s, :L])
            assert not back[r][s, L:].any()
    assert not tok[p["token_sample"] < 0].any()


def test_plan_errors():
    with pytest.raises(pl.PlanError):
        pl.pack_plan([0], [[0]], [4], 1)
    with pytest.raises(pl.PlanError):
        pl.pack_plan([0], [[5]], [4], 1)
    with pytest.raises(pl.PlanError):
        pl.pack_plan([0], [[2]], [4], 2)       # tenant 1 has no samples
    with pytest.raises(pl.PlanError):
        pl.pack_plan([2], [[2]], [4], 2)       # tenant outside the table
    with pytest.raises(pl.Incompatible):
        pl.pack_plan([0, 1], [[2], [3]], [4, 4], 2, tenant_sig=[1, 2])
    with pytest.raises(pl.Incompatible):
        pl.pack_plan([0, 1], [[2], [3]], [4, 4], 2, tenant_d=[8, 16], d=8)


def test_zipf_counts():
    c = W.zipf_counts(512, 32, 1.2)
    assert sum(c) == 512 and min(c) >= 1
    assert all(a >= b for a, b in zip(c, c[1:]))
    w = np.array([k ** -1.2 for k in range(1, 33)])
    assert np.max(np.abs(np.array(c) - 512 * w / w.sum())) < 1.0


def test_config_shapes():
    """Workload recipes follow the stated shapes (ranges of lengths, counts)."""
    for cfg, (G, N, lo, hi) in {1: (2, 16, 20, 32), 2: (4, 128, 204, 244), 3: (8, 256, 272, 320),
                                  5: (32, 512, 272, 832)}.items():
        spec = W.config_spec(cfg)
        assert spec.G == G and sum(t.n_samples for t in spec.tenants) == N
        for g in range(G):
            L = W.draw_lengths(spec, g)
            assert L.min() >= lo and L.max() <= hi and L.max() <= spec.tenants[g].max_len
