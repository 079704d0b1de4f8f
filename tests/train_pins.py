"""Pins that tie the float64 training oracle (oracle/dmc_train.py) to what
the paper and mathematics fix.

Each check takes the training-oracle module (so the mutation test can hand
in a broken copy).  None re-types an oracle formula: they use the paper's
printed mask table and Gumbel-sigmoid value, the discrete limit (which must
reproduce the pinned inference oracle's prompt attention), plain causal
attention through torch's scaled_dot_product_attention, the closed
product form of the partial accumulation, and central finite differences of
the forward for the backward.
"""
from __future__ import annotations

import math

import numpy as np
import torch

import oracle

from tests.oracle_pins import _golden


def _t(x):
    return torch.as_tensor(np.asarray(x), dtype=torch.float64)


def _inputs(rng, B, n, Hkv, G, d):
    q = rng.standard_normal((B, n, Hkv * G, d))
    k = rng.standard_normal((B, n, Hkv, d))
    v = rng.standard_normal((B, n, Hkv, d))
    return q, k, v


def check_mask_table(T):
    """The additive-mask table of Sec. 3.2: row i has log(1 - alpha_1),
    ..., log(1 - alpha_i) in columns 0..i-1, 0 on the diagonal and -inf
    to its right."""
    rng = np.random.default_rng(1)
    n = 6
    alpha = rng.uniform(0.05, 0.95, size=n)
    x = np.log(alpha / (1 - alpha))                       # logits of alpha
    M = T.attention_mask(_t(x)[None])[0].numpy()
    for i in range(n):
        for j in range(n):
            if j > i:
                assert M[i, j] == -math.inf, (i, j)
            elif j == i:
                assert M[i, j] == 0.0, (i, j)
            else:
                assert abs(M[i, j] - math.log(1 - alpha[j + 1])) < 1e-12, (i, j)


def check_gumbel_sigmoid_start(T):
    """Sec. 4: c = 5 makes alpha = 0.0067 at the start of training (k[0] = 0,
    no noise, tau = 1); the noise enters with the logit, and tau divides it."""
    g = _golden("sigmoid_c5.json")
    a, x = T.relaxed_decisions(_t(0.0), _t(0.0), g["c"], 1.0)
    assert round(float(a), g["decimals"]) == g["printed_value"]
    a2, _ = T.relaxed_decisions(_t(0.0), _t(5.0), 5.0, 1.0)
    assert abs(float(a2) - 0.5) < 1e-15                    # noise cancels the bias
    a3, x3 = T.relaxed_decisions(_t(1.0), _t(0.0), 0.0, 0.25)
    assert abs(float(x3) - 4.0) < 1e-15 and abs(float(a3) - 1 / (1 + math.exp(-4))) < 1e-15


def check_states_product_form(T):
    """Closed form of the partial accumulation: over a window starting at a,
    state j = sum_t c_tj k_t / sum_t c_tj with c_tj = omega_t prod_{r=t+1..j}
    alpha_r (the first token's own alpha never enters)."""
    rng = np.random.default_rng(2)
    U, n, d = 2, 11, 3
    kh = rng.standard_normal((U, n, d))
    v = rng.standard_normal((U, n, d))
    alpha = rng.uniform(0, 1, size=(U, n))
    omega = rng.uniform(0.1, 1, size=(U, n))
    for w in (1, 2, 4, n):
        K, V, z = (x.numpy() for x in T.unrolled_states(_t(kh), _t(v), _t(alpha), _t(omega), w))
        for u in range(U):
            for j in range(n):
                a = max(0, j - w + 1)
                c = np.array([omega[u, t] * np.prod(alpha[u, t + 1:j + 1]) for t in range(a, j + 1)])
                assert abs(z[u, j] - c.sum()) < 1e-12
                np.testing.assert_allclose(K[u, j], c @ kh[u, a:j + 1] / c.sum(), atol=1e-12)
                np.testing.assert_allclose(V[u, j], c @ v[u, a:j + 1] / c.sum(), atol=1e-12)


def check_discrete_limit_is_inference(T):
    """With decisions driven to exactly 0 or 1 (tau tiny, logits away from
    0) the training forward is the inference-time prompt attention of the
    pinned oracle (windowed, and unwindowed for a window as long as the
    sequence)."""
    rng = np.random.default_rng(3)
    B, n, Hkv, G, d = 2, 20, 2, 2, 6
    for w in (3, 12, n):
        q, k, v = _inputs(rng, B, n, Hkv, G, d)
        acc = rng.uniform(size=(B, n, Hkv)) < 0.6
        k[..., 0] = np.where(acc, 1.0, -1.0) * rng.uniform(0.5, 2.0, size=(B, n, Hkv))
        noise = np.zeros((B, n, Hkv))
        out, alpha = T.train_forward(_t(q), _t(k), _t(v), _t(noise), c=0.0, tau=1e-4, window=w)
        assert set(np.unique(alpha.numpy()[:, 1:])) <= {0.0, 1.0}
        orc = oracle.DMCOracle(1, B, Hkv * G, Hkv, d, n, window=0 if w == n else w)
        ref, _ = orc.prefill_attend(0, q, k, v)
        np.testing.assert_allclose(out.numpy(), ref, atol=1e-10, rtol=1e-10)


def check_all_append_is_causal(T):
    """alpha = 0 everywhere: every state is its own token and the mask is
    causal, so the forward is causal softmax attention over dims 1..d-1 with
    scale 1/sqrt(d) (torch's scaled_dot_product_attention)."""
    rng = np.random.default_rng(4)
    B, n, Hkv, G, d = 1, 13, 2, 2, 8
    q, k, v = _inputs(rng, B, n, Hkv, G, d)
    k[..., 0] = -50.0
    out, _ = T.train_forward(_t(q), _t(k), _t(v), _t(np.zeros((B, n, Hkv))), c=0.0, tau=0.01,
                             window=5)
    qh = _t(q[..., 1:]).permute(0, 2, 1, 3)                          # [B, Hq, n, d-1]
    kh = _t(np.repeat(k[..., 1:], G, axis=2)).permute(0, 2, 1, 3)
    vh = _t(np.repeat(v, G, axis=2)).permute(0, 2, 1, 3)
    ref = torch.nn.functional.scaled_dot_product_attention(qh, kh, vh, is_causal=True,
                                                           scale=1 / math.sqrt(d))
    np.testing.assert_allclose(out.numpy(), ref.permute(0, 2, 1, 3).numpy(), atol=1e-12)


def check_backward_finite_differences(T):
    """The backward against central differences of the forward (dq, dk, dv,
    including the decision and importance neurons and the dalpha path)."""
    rng = np.random.default_rng(5)
    B, n, Hkv, G, d = 1, 6, 1, 2, 4
    q, k, v = _inputs(rng, B, n, Hkv, G, d)
    noise = rng.logistic(size=(B, n, Hkv))
    dout = rng.standard_normal((B, n, Hkv * G, d))
    dal = rng.standard_normal((B, n, Hkv))
    c, tau, w = 0.3, 0.7, 3
    dq, dk, dv = T.train_backward(q, k, v, noise, dout, dal, c=c, tau=tau, window=w)

    def f(qq, kk, vv):
        out, alpha = T.train_forward(_t(qq), _t(kk), _t(vv), _t(noise), c=c, tau=tau, window=w)
        return float((out.numpy() * dout).sum() + (alpha.numpy() * dal).sum())

    h = 1e-6
    for name, x, g in (("q", q, dq), ("k", k, dk), ("v", v, dv)):
        g = g.numpy()
        for idx in np.ndindex(x.shape):
            xp, xm = x.copy(), x.copy()
            xp[idx] += h
            xm[idx] -= h
            args_p = [q, k, v]
            args_m = [q, k, v]
            pos = "qkv".index(name)
            args_p[pos], args_m[pos] = xp, xm
            fd = (f(*args_p) - f(*args_m)) / (2 * h)
            assert abs(fd - g[idx]) < 1e-6 * max(1.0, abs(fd)), (name, idx, fd, g[idx])


def check_uniform_weighting(T):
    """Uniform weighting: omega = 1, so the query neuron gets no gradient and
    with alpha = 1 throughout a window the state is the window's plain mean."""
    rng = np.random.default_rng(6)
    B, n, Hkv, G, d = 1, 9, 1, 1, 5
    q, k, v = _inputs(rng, B, n, Hkv, G, d)
    k[..., 0] = 60.0
    noise = np.zeros((B, n, Hkv))
    dout = rng.standard_normal((B, n, Hkv * G, d))
    dq, _, _ = T.train_backward(q, k, v, noise, dout, c=0.0, tau=1.0, window=4,
                                omega_src="uniform")
    assert np.all(dq.numpy()[..., 0] == 0.0)
    kh = _t(k[0, :, 0].copy())
    kh[:, 0] = 0.0
    alpha = torch.ones((1, n), dtype=torch.float64)
    K, V, z = T.unrolled_states(kh[None], _t(v[0, :, 0])[None], alpha, T.importance(
        _t(q[0, :, 0, 0])[None], "uniform"), 4)
    for j in range(n):
        a = max(0, j - 3)
        np.testing.assert_allclose(K[0, j].numpy(), kh[a:j + 1].numpy().mean(axis=0), atol=1e-12)
        assert abs(float(z[0, j]) - (j - a + 1)) < 1e-12


ALL_CHECKS = [check_mask_table, check_gumbel_sigmoid_start, check_states_product_form,
              check_discrete_limit_is_inference, check_all_append_is_causal,
              check_backward_finite_differences, check_uniform_weighting]
