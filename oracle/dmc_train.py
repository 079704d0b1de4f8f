"""Float64 CPU oracle of DMC's training-time forward and backward.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the HIP library and
imports nothing from it.

What it computes (Nawrot et al., "Dynamic Memory Compression", ICML 2024):

* Sec. 3.2, gradient estimation: the discrete decision is relaxed to
  alpha_t ~ Gumbel-sigmoid(k_t[0] - c, tau), i.e.
  alpha_t = sigmoid((k_t[0] - c + g_t) / tau) with g_t logistic noise (the
  difference of two Gumbel samples).  The noise is an input: the caller draws
  it.
* Sec. 3.1: importance omega_t = sigmoid(q_t[0]) of the query head that
  supplies it (the group's first head for grouped-query attention, or 1 for
  uniform weighting), floored at 2**-100 as at inference.
* Sec. 3.2, partial accumulations: with continuous alpha the key/value state
  of position j follows z_i = alpha_i z_{i-1} + omega_i,
  k~_i = (alpha_i k~_{i-1} z_{i-1} + k_i omega_i) / z_i (same for v).  With
  window grouping (Sec. 3.3) it is evaluated for every position j over its
  last w tokens only, started afresh (z = omega, state = the token) at the
  window's first token.  Keys enter with element 0 set to zero (it is never
  part of a score).
* Sec. 3.2, intermediate compression steps, and the masking appendix: query i
  attends to every unrolled state j <= i with the additive mask
  log(1 - alpha_{j+1}) for j < i and 0 for j = i (-inf above the diagonal),
  added to the scores q_i[1:d] . k~_j[1:d] / sqrt(d).  log(1 - alpha_{j+1})
  is evaluated as log-sigmoid(-x_{j+1}) of the Gumbel-sigmoid logit x.

The forward is written as the recurrence itself, position by position (the
window loop in the paper's order), vectorised only across independent
(batch, kv-head) units.  The backward is torch autograd of that forward in
float64 -- the gradient by definition; the pins check it against central
finite differences.

Readings (listed in the design notes as well): the training path always uses
a finite window w >= 1 (the paper trains with w = 12); alpha_0 enters neither
a state nor the mask; omega comes from the group's first query head or is 1.
"""
from __future__ import annotations

import math

import torch

OMEGA_FLOOR = 2.0 ** -100


def relaxed_decisions(k0, noise, c, tau):
    """Gumbel-sigmoid relaxation (Sec. 3.2): logit x = (k0 - c + g) / tau and
    alpha = sigmoid(x)."""
    x = (k0 - c + noise) / tau
    return torch.sigmoid(x), x


def importance(q0, omega_src="lead"):
    """omega from the first query neuron of the supplying head [..., n]."""
    if omega_src == "uniform":
        return torch.ones_like(q0)
    assert omega_src == "lead", omega_src
    return torch.clamp_min(torch.sigmoid(q0), OMEGA_FLOOR)


def unrolled_states(kh, v, alpha, omega, window):
    """States of every position (Sec. 3.2 partial accumulation over a window
    of the last `window` tokens, Sec. 3.3).  kh, v: [U, n, d]; alpha, omega:
    [U, n].  Returns K~, V~ [U, n, d] and z [U, n]."""
    U, n, d = kh.shape
    Ks, Vs, zs = [], [], []
    for j in range(n):
        a = max(0, j - window + 1)
        z = omega[:, a]
        K, V = kh[:, a], v[:, a]
        for i in range(a + 1, j + 1):
            zn = alpha[:, i] * z + omega[:, i]
            K = (alpha[:, i, None] * K * z[:, None] + kh[:, i] * omega[:, i, None]) / zn[:, None]
            V = (alpha[:, i, None] * V * z[:, None] + v[:, i] * omega[:, i, None]) / zn[:, None]
            z = zn
        Ks.append(K)
        Vs.append(V)
        zs.append(z)
    return torch.stack(Ks, 1), torch.stack(Vs, 1), torch.stack(zs, 1)


def attention_mask(x):
    """Additive mask of the masking appendix for logits x [U, n]: entry
    (i, j) is 0 on the diagonal, log(1 - alpha_{j+1}) = log-sigmoid(-x_{j+1})
    below it and -inf above it.  Returns [U, n, n]."""
    U, n = x.shape
    col = torch.zeros((U, n), dtype=x.dtype)
    col[:, : n - 1] = torch.nn.functional.logsigmoid(-x[:, 1:])
    M = col[:, None, :].expand(U, n, n).clone()
    i = torch.arange(n)[:, None]
    j = torch.arange(n)[None, :]
    M = torch.where((j == i)[None], torch.zeros((), dtype=x.dtype), M)
    M = torch.where((j > i)[None], torch.full((), -math.inf, dtype=x.dtype), M)
    return M


def train_forward(q, k, v, noise, c=5.0, tau=0.1, window=12, omega_src="lead"):
    """Training-time DMC attention of one layer.

    q: [B, n, Hq, d]; k, v: [B, n, Hkv, d]; noise: [B, n, Hkv] logistic noise.
    Returns out [B, n, Hq, d] and alpha [B, n, Hkv] (float64 tensors, in the
    autograd graph of the inputs).
    """
    assert window >= 1
    B, n, Hq, d = q.shape
    Hkv = k.shape[2]
    G = Hq // Hkv
    U = B * Hkv
    ku = k.permute(0, 2, 1, 3).reshape(U, n, d)
    vu = v.permute(0, 2, 1, 3).reshape(U, n, d)
    qu = q.reshape(B, n, Hkv, G, d).permute(0, 2, 3, 1, 4).reshape(U, G, n, d)
    nu = noise.permute(0, 2, 1).reshape(U, n)
    alpha, x = relaxed_decisions(ku[:, :, 0], nu, c, tau)
    omega = importance(qu[:, 0, :, 0], omega_src)
    kh = torch.cat([torch.zeros_like(ku[:, :, :1]), ku[:, :, 1:]], dim=2)   # k[0] <- 0
    K, V, _ = unrolled_states(kh, vu, alpha, omega, window)
    qz = torch.cat([torch.zeros_like(qu[..., :1]), qu[..., 1:]], dim=3)       # q[0] <- 0
    s = qz @ K[:, None].transpose(2, 3) / math.sqrt(d)                        # [U, G, n, n]
    p = torch.softmax(s + attention_mask(x)[:, None], dim=-1)
    out = p @ V[:, None]                                                      # [U, G, n, d]
    out = out.reshape(B, Hkv, G, n, d).permute(0, 3, 1, 2, 4).reshape(B, n, Hq, d)
    return out, alpha.reshape(B, Hkv, n).permute(0, 2, 1)


def train_backward(q, k, v, noise, dout, dalpha=None, c=5.0, tau=0.1, window=12,
                   omega_src="lead"):
    """Gradients (dq, dk, dv) of sum(out * dout) + sum(alpha * dalpha) by
    autograd of train_forward, in float64."""
    q, k, v = (torch.as_tensor(t, dtype=torch.float64).clone().requires_grad_(True)
               for t in (q, k, v))
    noise = torch.as_tensor(noise, dtype=torch.float64)
    out, alpha = train_forward(q, k, v, noise, c, tau, window, omega_src)
    loss = (out * torch.as_tensor(dout, dtype=torch.float64)).sum()
    if dalpha is not None:
        loss = loss + (alpha * torch.as_tensor(dalpha, dtype=torch.float64)).sum()
    dq, dk, dv = torch.autograd.grad(loss, (q, k, v))
    return dq, dk, dv
