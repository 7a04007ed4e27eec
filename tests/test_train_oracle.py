"""Pins for the training-time DMS attention oracle (continuous decisions,
Sec. 3.1 Eq. 1 and Fig. 1b): binary decisions reduce to the inference mask,
fractional decisions equal key duplication under plain softmax attention,
gradients match finite differences, and the Gumbel-sigmoid matches its
logistic / two-Gumbel definitions."""
import math

import numpy as np
import pytest
import torch

import oracle
from oracle import dense_dms_attention


def _rand(seed, B, T, H, g, d):
    rng = np.random.default_rng(seed)
    return (rng.normal(size=(B, T, H * g, d)), rng.normal(size=(B, T, H, d)),
            rng.normal(size=(B, T, H, d)), rng)


@pytest.mark.parametrize("w", [1, 3, 7])
def test_binary_decisions_equal_inference_mask(w):
    q, k, v, rng = _rand(w, 2, 20, 2, 3, 8)
    a = (rng.uniform(size=(2, 20, 2)) < 0.5).astype(np.float64)
    O, _ = oracle.train_attention(q, k, v, a, w, 3)
    for b in range(2):
        ref = dense_dms_attention(q[b], k[b], v[b], a[b].astype(np.uint8), w, 3)
        assert np.allclose(O[b], ref, atol=1e-12)


def test_fractional_decision_equals_key_duplication():
    """alpha_j = 1 - 1/m_j outside the window weights key j by 1/m_j: the same
    as plain softmax attention where, scaling every weight by M = 6, key j
    appears 6 / m_j times and window keys 6 times."""
    T, d, w = 16, 8, 4
    q, k, v, rng = _rand(11, 1, T, 1, 1, d)
    m = rng.choice([1, 2, 3], size=T)
    a = (1.0 - 1.0 / m).reshape(1, T, 1)
    O, _ = oracle.train_attention(q, k, v, a, w, 1)
    for t in range(T):
        reps = [6 if j > t - w else 6 // m[j] for j in range(t + 1)]
        kk = np.repeat(k[0, : t + 1, 0], reps, axis=0)
        vv = np.repeat(v[0, : t + 1, 0], reps, axis=0)
        ref = torch.nn.functional.scaled_dot_product_attention(
            torch.tensor(q[0, t:t + 1, 0])[None], torch.tensor(kk)[None], torch.tensor(vv)[None])[0, 0]
        assert np.allclose(O[0, t, 0], ref.numpy(), atol=1e-12), t


def test_window_covering_history_is_causal():
    q, k, v, rng = _rand(5, 1, 12, 2, 2, 8)
    a = rng.uniform(size=(1, 12, 2))
    O, _ = oracle.train_attention(q, k, v, a, 12, 2)
    kk = np.repeat(k, 2, axis=2)
    vv = np.repeat(v, 2, axis=2)
    ref = torch.nn.functional.scaled_dot_product_attention(
        torch.tensor(q).transpose(1, 2), torch.tensor(kk).transpose(1, 2),
        torch.tensor(vv).transpose(1, 2), is_causal=True).transpose(1, 2)
    assert np.allclose(O, ref.numpy(), atol=1e-12)


def test_lse_is_log_of_the_normaliser():
    q, k, v, rng = _rand(6, 1, 10, 1, 2, 4)
    a = rng.uniform(size=(1, 10, 1))
    w = 3
    _, L = oracle.train_attention(q, k, v, a, w, 2)
    scale = 0.5
    for qh in range(2):
        for t in range(10):
            z = 0.0
            for j in range(t + 1):
                wt = 1.0 if j > t - w else 1.0 - a[0, j, 0]
                z += wt * math.exp(float(q[0, t, qh] @ k[0, j, 0]) * scale)
            assert abs(L[0, qh, t] - math.log(z)) < 1e-12


@pytest.mark.parametrize("seed", [0, 1])
def test_gradients_match_finite_differences(seed):
    B, T, H, g, d, w = 1, 9, 2, 2, 4, 3
    q, k, v, rng = _rand(20 + seed, B, T, H, g, d)
    a = rng.uniform(0.05, 0.95, size=(B, T, H))
    dout = rng.normal(size=(B, T, H * g, d))
    dq, dk, dv, da = oracle.train_attention_grads(q, k, v, a, dout, w, g)
    f = lambda qq, kk, vv, aa: float((oracle.train_attention(qq, kk, vv, aa, w, g)[0] * dout).sum())
    eps = 1e-6
    for arr, grad, which in ((q, dq, 0), (k, dk, 1), (v, dv, 2), (a, da, 3)):
        for _ in range(6):
            idx = tuple(int(rng.integers(s)) for s in arr.shape)
            args = [q, k, v, a]
            p, m = [x.copy() for x in args], [x.copy() for x in args]
            p[which][idx] += eps
            m[which][idx] -= eps
            fd = (f(*p) - f(*m)) / (2 * eps)
            assert abs(fd - grad[idx]) < 1e-6 * max(1.0, abs(fd)), (which, idx, fd, grad[idx])
    # keys inside every query's window get no decision gradient: the last w
    assert np.all(da[:, T - w:, :] == 0)


def _grad_at_hard_decisions_ok():
    """At alpha_j in {0, 1} (the ends of its range) the decision gradient is
    the one-sided derivative of the forward definition: second-order one-sided
    differences of the output, stepping into [0, 1]."""
    B, T, H, g, d, w = 1, 10, 1, 2, 4, 2
    q, k, v, rng = _rand(31, B, T, H, g, d)
    a = (rng.uniform(size=(B, T, H)) < 0.5).astype(np.float64)
    dout = rng.normal(size=(B, T, H * g, d))
    _, _, _, da = oracle.train_attention_grads(q, k, v, a, dout, w, g)
    if not np.isfinite(da).all():
        return False
    f = lambda aa: float((oracle.train_attention(q, k, v, aa, w, g)[0] * dout).sum())
    h = 1e-4
    for j in range(T - w):
        step = -h if a[0, j, 0] == 1.0 else h
        a1, a2 = a.copy(), a.copy()
        a1[0, j, 0] += step
        a2[0, j, 0] += 2 * step
        fd = (-3 * f(a) + 4 * f(a1) - f(a2)) / (2 * step)
        if abs(fd - da[0, j, 0]) > 1e-6 * max(1.0, abs(fd)):
            return False
    return True


def test_gradient_at_hard_decisions_is_the_one_sided_derivative():
    assert _grad_at_hard_decisions_ok()


def test_logistic_noise_inverts_the_logistic_cdf():
    u = (np.arange(1, 2000) + 0.5) / 2001
    L = oracle.logistic_noise(u)
    assert np.allclose(1.0 / (1.0 + np.exp(-L)), u, atol=1e-14)


def test_logistic_noise_is_a_difference_of_gumbels():
    rng = np.random.default_rng(3)
    n = 200000
    g1 = -np.log(-np.log(rng.uniform(size=n)))
    g2 = -np.log(-np.log(rng.uniform(size=n)))
    x = np.sort(g1 - g2)
    ecdf = (np.arange(n) + 0.5) / n
    ks = np.abs(ecdf - 1.0 / (1.0 + np.exp(-x))).max()
    assert ks < 1.36 / math.sqrt(n) * 1.5        # Kolmogorov-Smirnov, well inside 5%


def test_gumbel_sigmoid_limits_and_gradient():
    rng = np.random.default_rng(4)
    x = rng.normal(0, 3, 500)
    u = rng.uniform(0.001, 0.999, 500)
    z = x + np.log(u / (1 - u))
    hard = oracle.gumbel_sigmoid(x, u, 1e-4)
    keep = np.abs(z) > 1e-2
    assert np.array_equal(hard[keep] > 0.5, z[keep] > 0)
    assert np.allclose(hard[keep], (z[keep] > 0).astype(float), atol=1e-12)
    tau = 0.7
    a = oracle.gumbel_sigmoid(x, u, tau)
    eps = 1e-6
    fd = (oracle.gumbel_sigmoid(x + eps, u, tau) - oracle.gumbel_sigmoid(x - eps, u, tau)) / (2 * eps)
    assert np.allclose(oracle.gumbel_sigmoid_grad(a, np.ones_like(a), tau), fd, atol=1e-8)


# ----------------------------------------------------------------------------
# planted mistakes
# ----------------------------------------------------------------------------

def _pins_pass():
    try:
        test_binary_decisions_equal_inference_mask(3)
        test_fractional_decision_equals_key_duplication()
        test_window_covering_history_is_causal()
        test_lse_is_log_of_the_normaliser()
        test_logistic_noise_inverts_the_logistic_cdf()
        test_gumbel_sigmoid_limits_and_gradient()
    except AssertionError:
        return False
    return True


def test_pins_pass_unmodified():
    assert _pins_pass()


@pytest.mark.parametrize("mutant", ["inclusive_window", "log_alpha", "no_scale", "tau_times",
                                    "noise_sign", "weights_alpha"])
def test_planted_mistake_is_caught(monkeypatch, mutant):
    mod = oracle.train_oracle
    orig_attn = mod._torch_attention
    if mutant == "inclusive_window":
        monkeypatch.setattr(mod, "_torch_attention", lambda q, k, v, a, w, g, s: orig_attn(q, k, v, a, w + 1, g, s))
    elif mutant == "log_alpha":
        def bad(q, k, v, a, w, g, s):
            return orig_attn(q, k, v, 1.0 - a, w, g, s)
        monkeypatch.setattr(mod, "_torch_attention", bad)
    elif mutant == "no_scale":
        monkeypatch.setattr(mod, "_torch_attention", lambda q, k, v, a, w, g, s: orig_attn(q, k, v, a, w, g, 1.0))
    elif mutant == "tau_times":
        monkeypatch.setattr(mod, "gumbel_sigmoid", lambda x, u, tau: 1.0 / (1.0 + np.exp(
            -(np.asarray(x, np.float64) + mod.logistic_noise(u)) * tau)))
    elif mutant == "weights_alpha":
        orig_w = mod._torch_attention_weights
        monkeypatch.setattr(mod, "_torch_attention_weights",
                            lambda q, k, v, a, w, g, s: orig_w(q, k, v, 1.0 - a, w, g, s))
        assert not _grad_at_hard_decisions_ok()
        return
    elif mutant == "noise_sign":
        monkeypatch.setattr(mod, "logistic_noise", lambda u: np.log1p(-np.asarray(u, np.float64)) - np.log(u))
    for name in ("gumbel_sigmoid", "logistic_noise", "train_attention"):
        monkeypatch.setattr(oracle, name, getattr(mod, name))
    assert not _pins_pass()
