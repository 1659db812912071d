"""Pins of the oracle's backbone variants (causal mask, rotary positions that
restart in every sample, grouped / multi-query key-value heads) against
independent formulations, library routines and invariants."""
import numpy as np
import pytest
import torch
import torch.nn.functional as F

import workloads as W
from oracle import backbone as bb
from oracle import step as st

RTOL = 1e-12


def rel(a, b):
    a = np.asarray(a, np.float64)
    b = np.asarray(b, np.float64)
    return float(np.max(np.abs(a - b)) / max(np.max(np.abs(b)), 1e-300))


def variant_spec(kv=2, causal=True, theta=10000.0, heads=4, d=32, glu=False, ns=(3, 2), lens=(4, 11), max_len=12):
    bbs = W.BackboneSpec(layers=2, d=d, heads=heads, ffn=48, glu=glu, kv_heads=kv, causal=causal, rope_theta=theta)
    ten = []
    for g, n in enumerate(ns):
        a, c = (3, 2) if g % 2 == 0 else (2, 1)
        ten.append(W.TenantSpec(n, lens[0] - 1, 1, lens[1] - lens[0] + 1, max_len, (d, 8, a * c), a, c))
    return W.WorkloadSpec(98, bbs, tuple(ten), 0, "variant")


def test_rope_equals_complex_rotation():
    """Each pair (x_i, x_{i+hd/2}) is the complex number x_i + j x_{i+hd/2}
    multiplied by exp(j p theta^(-2i/hd))."""
    rng = np.random.default_rng(0)
    H, hd, L, theta = 3, 8, 7, 500.0
    x = rng.standard_normal((L, H * hd))
    pos = rng.integers(0, 1000, L)
    got = bb.rope(x, H, theta, pos)
    for h in range(H):
        z = x[:, h * hd: h * hd + hd // 2] + 1j * x[:, h * hd + hd // 2: (h + 1) * hd]
        w = np.exp(1j * pos[:, None] * theta ** (-np.arange(hd // 2) * 2.0 / hd)[None, :])
        r = z * w
        assert rel(got[:, h * hd: h * hd + hd // 2], r.real) < RTOL
        assert rel(got[:, h * hd + hd // 2: (h + 1) * hd], r.imag) < RTOL
    # position 0 is the identity; rotations keep every pair's norm
    assert np.array_equal(bb.rope(x, H, theta, np.zeros(L, int)), x)
    a, b = got[:, :hd // 2], got[:, hd // 2:hd]
    assert rel(a * a + b * b, x[:, :hd // 2] ** 2 + x[:, hd // 2:hd] ** 2) < RTOL


def test_rope_scores_depend_on_relative_position():
    """q(m) . k(n) after rotation depends on m - n only: shifting every
    position by a constant leaves the attention output unchanged."""
    rng = np.random.default_rng(1)
    H, hd, L = 2, 16, 9
    q, k, v = (rng.standard_normal((L, H * hd)) for _ in range(3))
    pos = np.arange(L)
    out0 = bb.attention(bb.rope(q, H, 1e4, pos), bb.rope(k, H, 1e4, pos), v, H)
    out1 = bb.attention(bb.rope(q, H, 1e4, pos + 123), bb.rope(k, H, 1e4, pos + 123), v, H)
    assert rel(out1, out0) < 1e-10
    # and it is not position-blind
    out2 = bb.attention(bb.rope(q, H, 1e4, pos[::-1]), bb.rope(k, H, 1e4, pos), v, H)
    assert rel(out2, out0) > 1e-3


@pytest.mark.parametrize("kv", [1, 2, 4])
@pytest.mark.parametrize("causal", [False, True])
def test_attention_matches_torch_sdpa(kv, causal):
    rng = np.random.default_rng(2)
    H, hd, L = 4, 8, 10
    q = rng.standard_normal((L, H * hd))
    k, v = rng.standard_normal((L, kv * hd)), rng.standard_normal((L, kv * hd))
    got = bb.attention(q, k, v, H, kv, causal)
    tq = torch.from_numpy(q).view(L, H, hd).transpose(0, 1)[None]
    tk = torch.from_numpy(k).view(L, kv, hd).transpose(0, 1)[None]
    tv = torch.from_numpy(v).view(L, kv, hd).transpose(0, 1)[None]
    ref = F.scaled_dot_product_attention(tq, tk, tv, is_causal=causal, enable_gqa=True)
    ref = ref[0].transpose(0, 1).reshape(L, H * hd).numpy()
    assert rel(got, ref) < RTOL


def test_causal_first_row_and_prefix_invariance():
    rng = np.random.default_rng(3)
    spec = variant_spec()
    lw = bb.LayerF64(W.layer_weights(spec, 0), False)
    x = rng.standard_normal((11, spec.backbone.d))
    H, kv, th = spec.backbone.heads, spec.backbone.kv_heads, spec.backbone.rope_theta
    y = bb.layer_forward(x, lw, H, 1e-6, kv, True, th)
    # rows 0..5 do not see rows 6..10
    x2 = x.copy()
    x2[6:] = rng.standard_normal((5, spec.backbone.d)) * 10
    y2 = bb.layer_forward(x2, lw, H, 1e-6, kv, True, th)
    assert np.array_equal(y2[:6], y[:6])
    assert rel(y2[6:], y[6:]) > 1e-3
    # row 0 attends to itself only: attention output = its own value rows
    q = rng.standard_normal((5, H * 8))
    kk, vv = rng.standard_normal((5, kv * 8)), rng.standard_normal((5, kv * 8))
    a = bb.attention(q, kk, vv, H, kv, True)
    for h in range(H):
        g = h // (H // kv)
        assert rel(a[0, h * 8:(h + 1) * 8], vv[0, g * 8:(g + 1) * 8]) < RTOL


@pytest.mark.parametrize("kv", [1, 2])
def test_gqa_equals_mha_with_repeated_kv_weights(kv):
    """Grouped key/value heads equal multi-head attention whose key and value
    projections repeat each group's rows for every query head of the group."""
    rng = np.random.default_rng(4)
    H, hd, d = 4, 8, 32
    spec = variant_spec(kv=kv, d=d, heads=H)
    w = W.layer_weights(spec, 0)
    lw = bb.LayerF64(w, False)
    lw_mha = bb.LayerF64(w, False)
    q_rows = lw.wqkv[:d]
    k_rows = lw.wqkv[d:d + kv * hd]
    v_rows = lw.wqkv[d + kv * hd:]
    rep = lambda m: np.concatenate([m[(h // (H // kv)) * hd:(h // (H // kv) + 1) * hd] for h in range(H)])  # noqa: E731
    lw_mha.wqkv = np.concatenate([q_rows, rep(k_rows), rep(v_rows)])
    x = rng.standard_normal((9, d))
    for causal, th in ((False, 0.0), (True, 1e4)):
        y = bb.layer_forward(x, lw, H, 1e-6, kv, causal, th)
        y_mha = bb.layer_forward(x, lw_mha, H, 1e-6, 0, causal, th)
        assert rel(y, y_mha) < RTOL


@pytest.mark.parametrize("variant", [dict(kv=2, causal=True, theta=1e4), dict(kv=1, causal=False, theta=1e4),
                                     dict(kv=4, causal=True, theta=0.0)])
@pytest.mark.parametrize("align", [1, 4])
def test_grouped_equals_isolated_with_variants(variant, align):
    """The packed formulation (block-diagonal, causal where asked, positions
    counted inside each sample) equals per-sample runs."""
    spec = variant_spec(**variant)
    wl = W.make_workload(spec, request_split=(2, 1))
    iso = st.isolated(wl, heads=False)
    packed = st.packed_block_diagonal(wl, align)
    keys = [(r, s) for r, q in enumerate(wl.requests) for s in range(q.n)]
    for key, z in zip(keys, packed):
        assert rel(z, iso["hidden"][key]) < RTOL, key
