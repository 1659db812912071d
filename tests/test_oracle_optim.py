"""Pins of the AdamW oracle (per-tenant optimizer step)."""
import numpy as np
import torch

from oracle import optim


def test_matches_torch_adamw_float64_over_several_steps():
    rng = np.random.default_rng(0)
    shapes = [(7, 5), (13,), (3, 4, 2)]
    hyper = dict(lr=3e-3, beta1=0.85, beta2=0.97, eps=1e-7, weight_decay=0.05)
    ps = [rng.standard_normal(s) for s in shapes]
    tp = [torch.tensor(p.copy(), requires_grad=True) for p in ps]
    opt = torch.optim.AdamW(tp, lr=hyper["lr"], betas=(hyper["beta1"], hyper["beta2"]), eps=hyper["eps"],
                            weight_decay=hyper["weight_decay"])
    ms = [np.zeros(s) for s in shapes]
    vs = [np.zeros(s) for s in shapes]
    for step in range(1, 6):
        gs = [rng.standard_normal(s) for s in shapes]
        for t, g in zip(tp, gs):
            t.grad = torch.tensor(g)
        opt.step()
        out = optim.tenant_step(list(zip(ps, gs, ms, vs)), hyper, step)
        ps = [o[0] for o in out]
        ms = [o[1] for o in out]
        vs = [o[2] for o in out]
        for p, t in zip(ps, tp):
            assert np.allclose(p, t.detach().numpy(), rtol=1e-13, atol=1e-15)


def test_first_step_closed_form():
    # with zero moments the first update is p(1 - lr wd) - lr g / (|g| + eps)
    rng = np.random.default_rng(1)
    p, g = rng.standard_normal(50), rng.standard_normal(50)
    lr, wd, eps = 1e-2, 0.1, 1e-8
    q, m, v = optim.adamw_step(p, g, np.zeros(50), np.zeros(50), 1, lr, 0.9, 0.999, eps, wd)
    assert np.allclose(q, p * (1 - lr * wd) - lr * g / (np.abs(g) + eps), rtol=1e-12, atol=1e-15)
    assert np.allclose(m, 0.1 * g) and np.allclose(v, 0.001 * g * g)


def test_zero_gradient_only_decays():
    p = np.linspace(-2, 2, 9)
    q, m, v = optim.adamw_step(p, np.zeros(9), np.zeros(9), np.zeros(9), 3, 0.5, 0.9, 0.999, 1e-8, 0.2)
    assert np.array_equal(m, np.zeros(9)) and np.array_equal(v, np.zeros(9))
    assert np.allclose(q, p * (1 - 0.5 * 0.2), rtol=1e-15)
