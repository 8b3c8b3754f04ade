"""Pins for the oracle's Adam (no GPU): closed forms and torch.optim.Adam."""
import numpy as np
import torch

from oracle import optim


def test_first_step_is_a_scaled_sign():
    # t = 1: m_hat = g, v_hat = g^2, so the step is lr * g / (|g| + eps)
    g = np.array([0.3, -2.0, 1e-3, 0.0, -5e-9])
    w, m, v = optim.adam(np.zeros(5), g, np.zeros(5), np.zeros(5), 1, 0.01)
    np.testing.assert_allclose(w, -0.01 * g / (np.abs(g) + 1e-8), rtol=1e-12, atol=0)
    np.testing.assert_allclose(m, 0.1 * g, rtol=1e-15)
    np.testing.assert_allclose(v, 0.001 * g * g, rtol=1e-12)


def test_constant_gradient_keeps_the_step():
    # with g fixed, the bias corrections make m_hat = g and v_hat = g^2 at every t
    g = np.array([0.5, -0.25, 4.0])
    w, m, v = np.zeros(3), np.zeros(3), np.zeros(3)
    for t in range(1, 40):
        w_new, m, v = optim.adam(w, g, m, v, t, 0.1)
        np.testing.assert_allclose(w - w_new, 0.1 * g / (np.abs(g) + 1e-8), rtol=1e-9)
        w = w_new


def test_matches_torch_adam():
    g_rng = np.random.Generator(np.random.PCG64(5))
    w0 = g_rng.normal(size=50)
    p = torch.nn.Parameter(torch.tensor(w0, dtype=torch.float64))
    opt = torch.optim.Adam([p], lr=0.01)
    w, m, v = w0.copy(), np.zeros(50), np.zeros(50)
    for t in range(1, 25):
        g = g_rng.normal(size=50) * (0.1 if t % 3 else 3.0)
        p.grad = torch.tensor(g, dtype=torch.float64)
        opt.step()
        w, m, v = optim.adam(w, g, m, v, t, 0.01)
        np.testing.assert_allclose(w, p.detach().numpy(), rtol=1e-12, atol=1e-15)
