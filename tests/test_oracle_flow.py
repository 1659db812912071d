"""Pins of the flow-matching objective of the action-expert oracle: the path
and its velocity, the flow-time features, the gradient of the time projection
by central differences, and reductions to the plain regression step."""
import numpy as np
import torch

import workloads as W
from oracle import expert as ex

from test_oracle_expert import inputs, tiny_expert


def with_time(w, rng, d=16, dt=8, scale=0.3):
    w = dict(w)
    w["w_time"] = W.f32_to_bf16_bits((rng.standard_normal((d, dt)) * scale).astype(np.float32))
    return w


def test_velocity_is_path_derivative():
    rng = np.random.default_rng(0)
    e, a = rng.standard_normal((5, 3)), rng.standard_normal((5, 3))
    for tau in (0.0, 0.3, 0.999):
        x, v = ex.flow_inputs(tau, e, a)
        h = 1e-6
        xp, _ = ex.flow_inputs(tau + h, e, a)
        xm, _ = ex.flow_inputs(tau - h, e, a)
        assert np.allclose((xp - xm) / (2 * h), v, rtol=0, atol=1e-8)
    assert np.array_equal(ex.flow_inputs(0.0, e, a)[0], a)   # tau = 0: the clean actions
    assert np.array_equal(ex.flow_inputs(1.0, e, a)[0], e)   # tau = 1: the noise


def test_time_features_complex_form():
    for tau in (0.0, 0.01, 0.5, 0.999):
        dim = 16
        phi = ex.time_features(tau, dim)
        z = np.exp(1j * 1000.0 * tau * np.power(10000.0, -np.arange(dim // 2) / (dim // 2)))
        assert np.allclose(phi[: dim // 2], z.imag, atol=1e-12) and np.allclose(phi[dim // 2:], z.real, atol=1e-12)
    assert np.array_equal(ex.time_features(0.0, 8), np.array([0, 0, 0, 0, 1, 1, 1, 1], np.float64))


def test_flow_grads_central_differences():
    rng = np.random.default_rng(5)
    w = with_time(tiny_expert(rng), rng)
    u, z, t = inputs(rng)
    taus = [0.2, 0.85]
    res = ex.expert_step(w, 2, 2, 1e-6, u, z, t, rnd=False, flow_t=taus)
    P = ex.expert_params(w)
    pairs = [ex.flow_inputs(taus[i], u[i], t[i]) for i in range(len(u))]
    xin = [x for x, _ in pairs]
    vel = torch.tensor(np.stack([v for _, v in pairs]))
    h = 1e-6
    for name in ("w_time", "w_in", "0.wq_c", "1.g3", "w_out"):
        base = P[name].detach().numpy()
        for idx in [tuple(rng.integers(0, s) for s in base.shape) for _ in range(3)]:
            def loss_at(delta):
                Q = {k: v.detach().clone() for k, v in P.items()}
                Q[name][idx] += delta
                with torch.no_grad():
                    Y = torch.stack(ex.expert_forward(Q, 2, 2, 1e-6, xin, z, False, taus))
                    return float(torch.mean((Y - vel) ** 2))
            fd = (loss_at(h) - loss_at(-h)) / (2 * h)
            g = res["grads"][name][idx]
            assert abs(fd - g) <= 1e-6 * max(1.0, abs(g)) + 1e-9, (name, idx, fd, g)


def test_reductions():
    rng = np.random.default_rng(6)
    w = with_time(tiny_expert(rng), rng)
    u, z, t = inputs(rng)
    taus = [0.4, 0.7]
    # zero time projection: the plain step on the path points against the velocities
    wz = dict(w)
    wz["w_time"] = np.zeros_like(w["w_time"])
    fl = ex.expert_step(wz, 2, 2, 1e-6, u, z, t, flow_t=taus)
    pairs = [ex.flow_inputs(taus[i], u[i], t[i]) for i in range(2)]
    plain = ex.expert_step({k: v for k, v in w.items() if k != "w_time"}, 2, 2, 1e-6, [x for x, _ in pairs], z,
                           np.stack([v for _, v in pairs]))
    assert abs(fl["loss"] - plain["loss"]) <= 1e-12 * abs(plain["loss"])
    assert np.allclose(fl["pred"], plain["pred"], rtol=1e-12, atol=1e-14)
    # zero output projection: zero prediction, loss = mean squared velocity
    w0 = dict(w)
    w0["w_out"] = np.zeros_like(w["w_out"])
    r0 = ex.expert_step(w0, 2, 2, 1e-6, u, z, t, flow_t=taus)
    v = np.stack([v for _, v in pairs])
    assert not r0["pred"].any()
    assert abs(r0["loss"] - float(np.mean(v * v))) <= 1e-12
    # the time projection matters when it is not zero
    assert abs(ex.expert_step(w, 2, 2, 1e-6, u, z, t, flow_t=taus)["loss"] - fl["loss"]) > 1e-6
