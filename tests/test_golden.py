"""The stored full-size oracle values (tests/golden/backbone_golden.py):
they are what the oracle computes, and the comparison that the GPU tests run
on them catches a wrong row anywhere in a sample, a wrong pooled feature and
values that belong to other inputs."""
import numpy as np
import pytest

import workloads as W

BG = pytest.importorskip("backbone_golden")


@pytest.fixture(scope="module")
def cfg2():
    import oracle
    wl = W.make_workload(2)
    gold = BG.load(2)
    keys = [tuple(int(v) for v in k) for k in gold["keys"]]
    assert keys == BG.chosen_samples(wl)
    res = oracle.step.isolated(wl, samples=keys, heads=False)
    # a stand-in for the device output: the oracle's own rows for the chosen
    # samples (every other row zero), packed in arrival order
    lens = [int(L) for q in wl.requests for L in q.lengths]
    cu = np.concatenate([[0], np.cumsum(lens)])
    hidden = np.zeros((cu[-1], wl.spec.backbone.d))
    flat = [(r, s) for r, q in enumerate(wl.requests) for s in range(q.n)]
    order = [(r, s) for g in range(wl.spec.G) for r, q in enumerate(wl.requests) if q.tenant == g for s in range(q.n)]
    pooled = np.zeros((len(order), wl.spec.backbone.d))
    for i, k in enumerate(flat):
        if k in res["hidden"]:
            hidden[cu[i]: cu[i + 1]] = res["hidden"][k]
            pooled[order.index(k)] = res["pooled"][k]
    return wl, gold, hidden, cu, pooled


def test_every_tenant_has_stored_samples():
    for cfg in (2, 3, 4, 5, 6, 7):
        spec = W.config_spec(cfg)
        gold = BG.load(cfg)
        assert gold["keys"].shape[0] >= spec.G, cfg
        assert gold["rows"].shape[1:] == (BG.N_ROWS, spec.backbone.d)
        assert gold["proj_off"][-1] == gold["proj"].shape[0] == int(gold["lengths"].sum())
        np.testing.assert_allclose(np.linalg.norm(gold["dirs"], axis=1), 1.0, rtol=1e-12)


def test_stored_values_are_the_oracle(cfg2):
    wl, gold, hidden, cu, pooled = cfg2
    res = BG.compare(wl, gold, hidden, cu, pooled)
    assert res["tenants"] == 4 and res["samples"] == 8
    assert res["worst"] < 1e-6   # fp32 storage of fp64 values


def test_planted_errors_are_caught(cfg2):
    wl, gold, hidden, cu, pooled = cfg2
    keys = [tuple(int(v) for v in k) for k in gold["keys"]]
    flat = [(r, s) for r, q in enumerate(wl.requests) for s in range(q.n)]
    i = flat.index(keys[3])
    stored = set(int(j) for j in gold["row_idx"][3])
    j = next(j for j in range(1, 200) if j not in stored)   # a row that is not stored in full
    scale = float(gold["maxabs"][3])
    bad = hidden.copy()
    bad[cu[i] + j] += 0.05 * scale * np.sign(np.random.default_rng(0).standard_normal(bad.shape[1]))
    res = BG.compare(wl, gold, bad, cu, pooled)
    assert res["per_tenant"][wl.requests[keys[3][0]].tenant] > 2e-2
    bad = hidden.copy()
    bad[cu[i] + j], bad[cu[i] + j + 1] = hidden[cu[i] + j + 1], hidden[cu[i] + j]   # two rows swapped
    assert BG.compare(wl, gold, bad, cu, pooled)["worst"] > 2e-2
    badp = pooled.copy()
    badp[31, 100:140] *= 1.1   # tenant-order row 31: the last sample of tenant 0
    assert BG.compare(wl, gold, hidden, cu, badp)["pooled"] > 2e-2


def test_other_inputs_are_refused(cfg2):
    import copy
    wl, gold, hidden, cu, pooled = cfg2
    other = copy.copy(wl)
    other.layers = list(wl.layers)
    other.layers[3] = dict(wl.layers[3], wo=wl.layers[3]["wo"].copy())
    other.layers[3]["wo"][0, 0] ^= 1   # one bit of one weight
    with pytest.raises(AssertionError, match="other inputs"):
        BG.compare(other, gold, hidden, cu, pooled)
