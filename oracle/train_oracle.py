"""CPU oracle for training-time DMS attention.  TEST INFRASTRUCTURE ONLY.

Only the tests, the smoke check and the benchmark's CPU-baseline leg may use
this module; the GPU library never calls it and shares no code with it.

What it computes (paper: "Inference-Time Hyper-Scaling with KV Cache
Compression", arxiv 2506.05345):

* Sec. 3.1 (Eq. 1): during retrofitting each token t of each KV head gets a
  continuous decision alpha_t in [0, 1] drawn from a Gumbel-sigmoid with
  logit h_t w^T + b and a low temperature tau.  Here the Gumbel-sigmoid is
  the binary-Concrete form: alpha = sigmoid((x + L) / tau) with logistic
  noise L = log(u) - log(1 - u), u ~ U(0, 1) (the difference of two
  independent Gumbel(0, 1) variables is logistic); u is an input.
* Sec. 3.1 and Fig. 1b: the decisions build the additive mask M_alpha --
  -inf above the diagonal, 0 for the w most recent positions (delayed
  eviction), log(1 - alpha_j) elsewhere -- added to the scaled scores of
  every query head that reads the KV head; outputs are softmax attention.
* Gradients of the attention output with respect to q, k, v and alpha, and
  of alpha with respect to its logit, come from automatic differentiation
  of these plain float64 definitions (torch on the CPU).  For alpha the
  attention is written with the mask as weights (1 - alpha_j), the same
  function, so that at alpha_j = 1 the gradient is the finite derivative
  from below rather than 0 * inf.
"""
from __future__ import annotations

import math

import numpy as np

__all__ = ["logistic_noise", "gumbel_sigmoid", "gumbel_sigmoid_grad", "train_attention",
           "train_attention_grads"]


def logistic_noise(u):
    """L = log(u) - log(1 - u): a Logistic(0, 1) draw from u ~ U(0, 1)."""
    u = np.asarray(u, np.float64)
    return np.log(u) - np.log1p(-u)


def gumbel_sigmoid(logits, u, tau):
    """alpha = sigmoid((logit + L(u)) / tau)."""
    z = (np.asarray(logits, np.float64) + logistic_noise(u)) / tau
    with np.errstate(over="ignore"):
        return 1.0 / (1.0 + np.exp(-z))


def gumbel_sigmoid_grad(alpha, dalpha, tau):
    """d loss / d logit = d loss / d alpha * alpha (1 - alpha) / tau."""
    a = np.asarray(alpha, np.float64)
    return np.asarray(dalpha, np.float64) * a * (1.0 - a) / tau


def _torch_attention(q, k, v, alpha, w, group, scale):
    """q [B, T, Hq, d], k / v [B, T, Hkv, d], alpha [B, T, Hkv] (torch float64)."""
    import torch
    B, T, Hq, d = q.shape
    Hkv = Hq // group
    t = torch.arange(T)[:, None]
    j = torch.arange(T)[None, :]
    causal = j > t
    window = j > t - w
    outs = []
    for h in range(Hkv):
        a = alpha[:, :, h]                                     # [B, T]
        outside = torch.log1p(-a)[:, None, :].expand(B, T, T)  # bias log(1 - alpha_j)
        bias = torch.where(window, torch.zeros_like(outside), outside)
        bias = torch.where(causal, torch.full_like(bias, -math.inf), bias)
        for qh in range(h * group, (h + 1) * group):
            s = torch.einsum("btd,bjd->btj", q[:, :, qh], k[:, :, h]) * scale + bias
            m = s.max(dim=-1, keepdim=True).values
            p = torch.exp(s - m)
            den = p.sum(dim=-1, keepdim=True)
            o = torch.einsum("btj,bjd->btd", p, v[:, :, h]) / den
            lse = (m + torch.log(den))[..., 0]
            outs.append((qh, o, lse))
    outs.sort(key=lambda x: x[0])
    O = torch.stack([o for _, o, _ in outs], dim=2)            # [B, T, Hq, d]
    LSE = torch.stack([l for _, _, l in outs], dim=1)          # [B, Hq, T]
    return O, LSE


def train_attention(q, k, v, alpha, w, group, scale=None):
    """DMS attention with continuous decisions: returns (O [B, T, Hq, d],
    LSE [B, Hq, T], natural log of each softmax denominator at its max)."""
    import torch
    q = torch.as_tensor(np.asarray(q, np.float64))
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    O, L = _torch_attention(q, torch.as_tensor(np.asarray(k, np.float64)),
                            torch.as_tensor(np.asarray(v, np.float64)),
                            torch.as_tensor(np.asarray(alpha, np.float64)), w, group, scale)
    return O.numpy(), L.numpy()


def _torch_attention_weights(q, k, v, alpha, w, group, scale):
    """The same attention with the mask applied as weights: softmax with the
    additive bias log(1 - alpha_j) equals exp(score) * (1 - alpha_j)
    renormalised.  Automatic differentiation of this form gives the finite
    one-sided derivative at alpha_j = 1 (where d log(1 - alpha) / d alpha is
    infinite and the additive form yields 0 * inf)."""
    import torch
    B, T, Hq, d = q.shape
    Hkv = Hq // group
    t = torch.arange(T)[:, None]
    j = torch.arange(T)[None, :]
    causal = j > t
    window = j > t - w
    outs = []
    for h in range(Hkv):
        a = alpha[:, :, h]
        keep = (1.0 - a)[:, None, :].expand(B, T, T)
        mult = torch.where(window, torch.ones_like(keep), keep)
        mult = torch.where(causal, torch.zeros_like(mult), mult)
        for qh in range(h * group, (h + 1) * group):
            s = torch.einsum("btd,bjd->btj", q[:, :, qh], k[:, :, h]) * scale
            s = torch.where(causal, torch.full_like(s, -math.inf), s)
            m = s.max(dim=-1, keepdim=True).values.detach()
            p = torch.exp(s - m) * mult
            o = torch.einsum("btj,bjd->btd", p, v[:, :, h]) / p.sum(dim=-1, keepdim=True)
            outs.append((qh, o))
    outs.sort(key=lambda x: x[0])
    return torch.stack([o for _, o in outs], dim=2)


def train_attention_grads(q, k, v, alpha, dout, w, group, scale=None):
    """(dq, dk, dv, dalpha) of sum(O * dout) by autograd of the definition
    (weights form; at alpha_j = 1 dalpha_j is the derivative from below)."""
    import torch
    q = torch.tensor(np.asarray(q, np.float64), requires_grad=True)
    k = torch.tensor(np.asarray(k, np.float64), requires_grad=True)
    v = torch.tensor(np.asarray(v, np.float64), requires_grad=True)
    a = torch.tensor(np.asarray(alpha, np.float64), requires_grad=True)
    if scale is None:
        scale = 1.0 / math.sqrt(q.shape[-1])
    O = _torch_attention_weights(q, k, v, a, w, group, scale)
    (O * torch.as_tensor(np.asarray(dout, np.float64))).sum().backward()
    return q.grad.numpy(), k.grad.numpy(), v.grad.numpy(), a.grad.numpy()
