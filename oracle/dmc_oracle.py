"""Float64 CPU oracle for the DMC decode hot path.

TEST INFRASTRUCTURE ONLY.  Nothing on the product path may import, call or
execute this module: only the test-suite, the smoke check and the CPU-baseline
leg of the benchmark use it.  It shares no code with the HIP library and
imports nothing from it.

What it computes (Nawrot et al., "Dynamic Memory Compression: Retrofitting
LLMs for Accelerated Inference", ICML 2024):

* Sec. 3.1 (Inference), the equation that re-uses the first key and query
  neurons: alpha_t = round(sigmoid(k_t[0])), omega_t = sigmoid(q_t[0]).
* Algorithm 1 (single-head KV cache update with DMC): after extracting
  alpha/omega, k_t[0] and q_t[0] are set to zero; alpha_t = 1 accumulates
  (z_t = z_{t-1} + omega_t, last slot <- (K_l z_{t-1} + k_t omega_t) / z_t,
  same for V), alpha_t = 0 appends (z_t = omega_t, push k_t and v_t).
* Sec. 3.1, last paragraph: attention is the ordinary softmax attention of
  Sec. 2.1 (scores q.k / sqrt(d_h)) over the compressed per-head sequences;
  every layer and head is updated independently.

The update is an iteration, so the oracle runs the algorithm itself, token
by token, in the paper's order.  It is vectorised only across independent
(batch, kv-head) units, which the paper states are independent; nothing is
blocked, fused or reordered within a unit.

Readings where the paper is silent or ambiguous (each is listed in the
design notes of the repository):

1. Decision: round(sigmoid(x)) is evaluated exactly as (x > 0) -- sigmoid is
   strictly increasing with sigmoid(0) = 1/2, and the tie rounds half to even,
   i.e. to 0.  Computing sigmoid first would collapse tiny |x| to 1/2.
2. Bias c (training uses sigmoid(k[0] - c), Sec. 3.2 and Sec. 4): a
   configuration value, default 0 (Algorithm 1 as printed): alpha = (k0 > c).
3. First token of every unit: Algorithm 1 needs a last slot to accumulate
   into; the partial-accumulation equation (Sec. 3.2) starts with z_0 = omega_0
   and k_0 = k_0, so with an empty cache the token is appended (alpha_0 := 0).
4. The query at step t attends to the cache *after* the step-t update
   (Algorithm 1 returns the updated K, V; the training mask has a zero
   diagonal).
5. Scale 1/sqrt(d_h) with the full head dimension (the masking appendix
   writes q[1:d_h].k[1:d_h]/sqrt(d_h)).  Stored keys have element 0 = 0 and
   the query's element 0 is zeroed before the scores; v is never zeroed.
6. Grouped-query attention: alpha comes from the kv head's own key; omega
   comes from the first query head of the group ("lead"), or optionally the
   mean of the group's sigmoid(q[0]) ("group_mean").  The paper combines DMC
   with GQA but does not say which query head supplies omega.
7. omega is floored at 2**-100 so that z never becomes 0 (sigmoid underflows
   only for q[0] below about -69, which synthetic inputs never reach).
8. Prefill (the prompt phase) equals n sequential updates without attention;
   prompt-phase attention is each token's update followed by its attention
   (reading 4 at every prompt position).
9. Variants of the appendix ablations: uniform weighting (omega = 1) and
   DMC-HardC (decision and importance of kv head 0 of a batch row shared by
   all heads of the layer; the paper does not name the head).
10. Window grouping (Sec. 3.3), when a window w is set: every step's
   partial accumulation runs over the last w tokens only, restarted at the
   window's first token, so a slot is the omega-weighted mean of the last
   min(w, length) tokens of its segment; the unit caches those raw tokens.

Parity pins (see tests/oracle_pins.py): the worked decision example of
Sec. 3.2, sigmoid(-5) = 0.0067 (Sec. 4), all-append = vanilla attention via
torch's scaled_dot_product_attention, all-accumulate closed form, fixed
memory pooling = avg_pool1d (Appendix, DMC ablations), brute force against
the unrolled-state + additive-mask formulation of Sec. 3.2, exact-arithmetic
decisions, permutation equivariance.  bf16 rounding drift of the device
cache beyond the stated tolerance is parity unpinned (the paper prints no
numeric compressed cache).
"""
from __future__ import annotations

import math

import numpy as np

OMEGA_FLOOR = 2.0 ** -100


# ----------------------------------------------------------------------------
# Sec. 3.1: decision and importance scores
# ----------------------------------------------------------------------------

def sigmoid(x):
    """Logistic function 1 / (1 + exp(-x)) in float64."""
    x = np.asarray(x, dtype=np.float64)
    return 1.0 / (1.0 + np.exp(-x))


def decision(k0, c=0.0):
    """alpha = round(sigmoid(k0 - c)), evaluated exactly (reading 1, 2).

    sigmoid(k0 - c) > 1/2 exactly when k0 > c; at k0 == c the value 1/2
    rounds half to even, to 0.  Inputs are widened to float64, in which the
    comparison of a bf16/fp32 value with an fp32 bias is exact.
    """
    k0 = np.asarray(k0, dtype=np.float64)
    return (k0 > np.float64(np.float32(c))).astype(np.int64)


def importance(q0_group, omega_src="lead"):
    """omega from the first query neuron(s) of a kv head's query group.

    q0_group: [..., G] values q[h, 0] of the G query heads sharing the kv head.
    'lead' takes the first head of the group, 'group_mean' the mean of the
    heads' sigmoids (reading 6); both floored at 2**-100 (reading 7).
    'uniform' is the uniform-weighting ablation of the appendix: every token
    of a segment weighs 1, so a slot is the plain mean of its segment.
    """
    q0_group = np.asarray(q0_group, dtype=np.float64)
    if omega_src == "lead":
        w = sigmoid(q0_group[..., 0])
    elif omega_src == "group_mean":
        w = sigmoid(q0_group).mean(axis=-1)
    elif omega_src == "uniform":
        return np.ones(q0_group.shape[:-1])
    else:
        raise ValueError(omega_src)
    return np.maximum(w, OMEGA_FLOOR)


# ----------------------------------------------------------------------------
# Algorithm 1 state for the units of one layer
# ----------------------------------------------------------------------------

class LayerCache:
    """Compressed caches of U independent (batch, kv-head) units of one layer.

    K, V: [U, cap, d] float64 slots (only the first l[u] are meaningful),
    l: [U] slot counts, z: [U] running importance sum of the open (last)
    slot -- the only z Algorithm 1 ever reads again.

    window > 0 selects the window-grouping approximation (Sec. 3.3): the
    partial accumulation of every step is evaluated over the last `window`
    tokens only, restarted at the window's first token; the unit keeps those
    tokens (k with element 0 zeroed, v, omega, alpha) to do so.
    """

    def __init__(self, units, head_dim, cap, window=0):
        self.U, self.d, self.cap = int(units), int(head_dim), int(cap)
        self.K = np.zeros((self.U, self.cap, self.d))
        self.V = np.zeros((self.U, self.cap, self.d))
        self.l = np.zeros(self.U, dtype=np.int64)
        self.z = np.zeros(self.U)
        self.window = int(window)
        if self.window:
            w = self.window
            self.wk = np.zeros((self.U, w, self.d))
            self.wv = np.zeros((self.U, w, self.d))
            self.ww = np.zeros((self.U, w))
            self.wa = np.zeros((self.U, w), dtype=np.int64)
            self.wn = np.zeros(self.U, dtype=np.int64)   # tokens seen by the unit

    def load(self, K, V, lengths, z):
        """Install an existing compressed cache (dense [U, >=max l, d])."""
        assert not self.window, "a windowed cache needs its token window; it is not imported"
        lengths = np.asarray(lengths, dtype=np.int64)
        assert lengths.shape == (self.U,) and lengths.max(initial=0) <= self.cap
        self.K[:] = 0.0
        self.V[:] = 0.0
        for u in range(self.U):
            n = lengths[u]
            self.K[u, :n] = np.asarray(K[u, :n], dtype=np.float64)
            self.V[u, :n] = np.asarray(V[u, :n], dtype=np.float64)
        self.l[:] = lengths
        self.z[:] = np.asarray(z, dtype=np.float64)

    # -- Algorithm 1 --------------------------------------------------------
    def update(self, k, v, q0_group, active=None, c=0.0, omega_src="lead", logits=None):
        """One step of Algorithm 1 for every active unit.

        k, v: [U, d] new key/value; q0_group: [U, G] first query neuron of the
        group's query heads; logits: [U] decision neurons (default k[:, 0],
        the unit's own key).  Returns alpha [U] and the slot index [U] each
        token went to (-1 for inactive units).
        """
        k = np.array(k, dtype=np.float64)           # private copies: inputs stay const
        v = np.array(v, dtype=np.float64)
        active = np.ones(self.U, bool) if active is None else np.asarray(active, bool)

        # Algorithm 1, the decision and the importance; reading 3: an empty cache appends
        alpha = decision(k[:, 0] if logits is None else logits, c) * (self.l > 0)
        omega = importance(q0_group, omega_src)
        # the decision neuron is cleared from the key: k_t[0] <- 0 (q_t[0] is zeroed
        # where scores are formed)
        k[:, 0] = 0.0

        acc = np.nonzero(active & (alpha == 1))[0]
        app = np.nonzero(active & (alpha == 0))[0]
        assert np.all(self.l[app] < self.cap), "oracle cache capacity exceeded"
        if self.window:
            self._windowed(k, v, alpha, omega, acc, app)
            return alpha, np.where(active, self.l - 1, -1)

        # alpha = 1: omega-weighted running mean into the last slot l-1, z grows by omega
        if acc.size:
            last = self.l[acc] - 1
            z_prev = self.z[acc]
            z_t = z_prev + omega[acc]
            self.K[acc, last] = (self.K[acc, last] * z_prev[:, None]
                                 + k[acc] * omega[acc, None]) / z_t[:, None]
            self.V[acc, last] = (self.V[acc, last] * z_prev[:, None]
                                 + v[acc] * omega[acc, None]) / z_t[:, None]
            self.z[acc] = z_t
        # alpha = 0: append a slot, z restarts at omega
        if app.size:
            pos = self.l[app]
            self.z[app] = omega[app]
            self.K[app, pos] = k[app]
            self.V[app, pos] = v[app]
            self.l[app] = pos + 1

        slot = np.where(active, self.l - 1, -1)
        return alpha, slot

    def _windowed(self, k, v, alpha, omega, acc, app):
        """Window grouping (Sec. 3.3): push the token into the unit's window,
        then evaluate the partial-accumulation recurrence of Sec. 3.2 over the
        window, started afresh at its first token (z = omega, state = k):
        z_j = alpha_j z_{j-1} + omega_j, state_j = (alpha_j state_{j-1} z_{j-1}
        + k_j omega_j) / z_j.  The result is the open slot (a new one when the
        token appends)."""
        w = self.window
        for u in np.concatenate([acc, app]):
            pos = self.wn[u] % w
            self.wk[u, pos], self.wv[u, pos] = k[u], v[u]
            self.ww[u, pos], self.wa[u, pos] = omega[u], alpha[u]
            self.wn[u] += 1
            m = min(self.wn[u], w)
            order = [(self.wn[u] - m + i) % w for i in range(m)]
            z = self.ww[u, order[0]]
            kt, vt = self.wk[u, order[0]].copy(), self.wv[u, order[0]].copy()
            for i in order[1:]:
                a, om = self.wa[u, i], self.ww[u, i]
                zn = a * z + om
                kt = (a * kt * z + self.wk[u, i] * om) / zn
                vt = (a * vt * z + self.wv[u, i] * om) / zn
                z = zn
            if alpha[u] == 0:
                self.l[u] += 1
            self.K[u, self.l[u] - 1], self.V[u, self.l[u] - 1] = kt, vt
            self.z[u] = z

    # -- Sec. 2.1 attention over the compressed sequence ---------------------
    def attend(self, u, q_heads):
        """Softmax attention of the query heads q_heads [G, d] of unit u."""
        q = np.array(q_heads, dtype=np.float64)
        q[:, 0] = 0.0                                  # Algorithm 1: q_t[0] leaves the score
        n = self.l[u]
        K, V = self.K[u, :n], self.V[u, :n]
        s = (q @ K.T) / math.sqrt(self.d)              # [G, n]
        s = s - s.max(axis=1, keepdims=True)
        p = np.exp(s)
        return (p @ V) / p.sum(axis=1, keepdims=True)


class DMCOracle:
    """All layers of a DMC cache: batch B, Hq query heads, Hkv kv heads.

    Unit u = b * Hkv + g holds the compressed sequence of kv head g of
    sequence b; query heads g*G .. g*G+G-1 attend to it (G = Hq / Hkv).
    """

    def __init__(self, num_layers, batch, num_q_heads, num_kv_heads, head_dim,
                 max_slots, decision_bias=0.0, omega_src="lead", decision_src="per_head",
                 window=0):
        assert num_q_heads % num_kv_heads == 0
        assert decision_src in ("per_head", "shared_layer")
        self.L, self.B = int(num_layers), int(batch)
        self.Hq, self.Hkv, self.d = int(num_q_heads), int(num_kv_heads), int(head_dim)
        self.G = self.Hq // self.Hkv
        self.c, self.omega_src = float(np.float32(decision_bias)), omega_src
        self.decision_src = decision_src
        self.layers = [LayerCache(self.B * self.Hkv, self.d, max_slots, window)
                       for _ in range(self.L)]

    def _q0_groups(self, q0):
        """[B, Hq] first query neurons -> [B*Hkv, G]."""
        return np.asarray(q0, dtype=np.float64).reshape(self.B * self.Hkv, self.G)

    def _decision_inputs(self, k0, q0):
        """Decision logits [U] and query-neuron groups [U, G] of one step.

        k0: [B, Hkv] first key neurons, q0: [B, Hq] first query neurons.
        'shared_layer' (DMC-HardC, appendix ablations: decision and
        importance shared by the heads of a layer) takes both from kv head 0
        of the batch row for every head of the row (reading: the paper does
        not name the head).
        """
        k0 = np.asarray(k0, dtype=np.float64)
        q0g = self._q0_groups(q0).reshape(self.B, self.Hkv, self.G)
        if self.decision_src == "shared_layer":
            k0 = np.repeat(k0[:, :1], self.Hkv, axis=1)
            q0g = np.repeat(q0g[:, :1], self.Hkv, axis=1)
        U = self.B * self.Hkv
        return k0.reshape(U), q0g.reshape(U, self.G)

    def decode_step(self, layer, q, k, v):
        """One auto-regressive step of one layer: update, then attend.

        q: [B, Hq, d]; k, v: [B, Hkv, d].  Returns out [B, Hq, d] (float64)
        and slot_index [B, Hkv] (the slot each new token went to).
        """
        lc = self.layers[layer]
        q = np.asarray(q, dtype=np.float64)
        U = self.B * self.Hkv
        logits, q0g = self._decision_inputs(np.asarray(k)[:, :, 0], q[:, :, 0])
        _, slot = lc.update(np.asarray(k).reshape(U, self.d),
                            np.asarray(v).reshape(U, self.d),
                            q0g, c=self.c, omega_src=self.omega_src, logits=logits)
        out = np.empty((self.B, self.Hq, self.d))
        qg = q.reshape(U, self.G, self.d)
        for u in range(U):
            b, g = divmod(u, self.Hkv)
            out[b, g * self.G:(g + 1) * self.G] = lc.attend(u, qg[u])
        return out, slot.reshape(self.B, self.Hkv)

    def prefill(self, layer, k, v, q0, prompt_lens=None):
        """Prompt phase of one layer: n sequential updates, no attention.

        k, v: [B, n, Hkv, d]; q0: [B, n, Hq] first query neurons.  The layer's
        cache must be empty.  Tokens t >= prompt_lens[b] are ignored.
        Returns slot_index [B, Hkv, n] (-1 for ignored tokens).
        """
        lc = self.layers[layer]
        assert not lc.l.any(), "prefill expects an empty layer cache"
        k = np.asarray(k, dtype=np.float64)
        v = np.asarray(v, dtype=np.float64)
        q0 = np.asarray(q0, dtype=np.float64)
        B, n = k.shape[:2]
        lens = np.full(B, n) if prompt_lens is None else np.asarray(prompt_lens)
        U = self.B * self.Hkv
        slots = np.full((U, n), -1, dtype=np.int64)
        for t in range(n):
            active = np.repeat(t < lens, self.Hkv)
            logits, q0g = self._decision_inputs(k[:, t, :, 0], q0[:, t])
            _, slot = lc.update(k[:, t].reshape(U, self.d), v[:, t].reshape(U, self.d),
                                q0g, active=active, c=self.c, omega_src=self.omega_src,
                                logits=logits)
            slots[:, t] = slot
        return slots.reshape(self.B, self.Hkv, n)

    def prefill_attend(self, layer, q, k, v, prompt_lens=None):
        """Prompt phase with attention: for every prompt token in order, the
        Algorithm 1 update and then the attention of its query heads over the
        updated cache -- the inference semantics of Sec. 3.1 applied to each
        prompt position (equivalently the training-time view of Sec. 3.2 with
        discrete decisions).

        q: [B, n, Hq, d]; k, v: [B, n, Hkv, d].  The layer's cache must be
        empty.  Returns out [B, n, Hq, d] (zeros for tokens past a row's
        prompt length) and slot_index [B, Hkv, n].
        """
        lc = self.layers[layer]
        assert not lc.l.any(), "prefill expects an empty layer cache"
        q = np.asarray(q, dtype=np.float64)
        k = np.asarray(k, dtype=np.float64)
        v = np.asarray(v, dtype=np.float64)
        B, n = k.shape[:2]
        lens = np.full(B, n) if prompt_lens is None else np.asarray(prompt_lens)
        U = self.B * self.Hkv
        out = np.zeros((self.B, n, self.Hq, self.d))
        slots = np.full((U, n), -1, dtype=np.int64)
        for t in range(n):
            active = np.repeat(lens > t, self.Hkv)
            logits, q0g = self._decision_inputs(k[:, t, :, 0], q[:, t, :, 0])
            _, slot = lc.update(k[:, t].reshape(U, self.d), v[:, t].reshape(U, self.d),
                                q0g, active=active, c=self.c, omega_src=self.omega_src,
                                logits=logits)
            slots[:, t] = slot
            qg = q[:, t].reshape(U, self.G, self.d)
            for u in np.nonzero(active)[0]:
                b, g = divmod(u, self.Hkv)
                out[b, t, g * self.G:(g + 1) * self.G] = lc.attend(u, qg[u])
        return out, slots.reshape(self.B, self.Hkv, n)

    def export(self, layer):
        """Dense copy of one layer: K, V [B, Hkv, cap, d], lengths, z [B, Hkv]."""
        lc = self.layers[layer]
        sh = (self.B, self.Hkv)
        return (lc.K.reshape(sh + lc.K.shape[1:]).copy(),
                lc.V.reshape(sh + lc.V.shape[1:]).copy(),
                lc.l.reshape(sh).copy(), lc.z.reshape(sh).copy())

    def load(self, layer, K, V, lengths, z):
        """Install a dense cache K, V [B, Hkv, >=max l, d], lengths, z [B, Hkv]."""
        U = self.B * self.Hkv
        K = np.asarray(K)
        self.layers[layer].load(K.reshape((U,) + K.shape[2:]),
                                np.asarray(V).reshape((U,) + K.shape[2:]),
                                np.asarray(lengths).reshape(U),
                                np.asarray(z).reshape(U))


# ----------------------------------------------------------------------------
# Per-unit helpers used by sampled parity checks at full size
# ----------------------------------------------------------------------------

class UnitOracle:
    """A single (layer, batch, kv-head) unit: Algorithm 1 plus attention.

    Used where only a sample of units can be followed on the CPU.  It runs
    the same LayerCache code with U = 1.
    """

    def __init__(self, head_dim, cap, decision_bias=0.0, omega_src="lead"):
        self.lc = LayerCache(1, head_dim, cap)
        self.c, self.omega_src = float(np.float32(decision_bias)), omega_src

    def load(self, K, V, length, z):
        self.lc.load(np.asarray(K)[None], np.asarray(V)[None], [length], [z])

    def step(self, q_group, k, v):
        """q_group [G, d], k, v [d] -> (out [G, d], slot index)."""
        q_group = np.asarray(q_group, dtype=np.float64)
        _, slot = self.lc.update(np.asarray(k)[None], np.asarray(v)[None],
                                 q_group[None, :, 0], c=self.c,
                                 omega_src=self.omega_src)
        return self.lc.attend(0, q_group), int(slot[0])

    @property
    def length(self):
        return int(self.lc.l[0])

    @property
    def z(self):
        return float(self.lc.z[0])

    def slots(self):
        n = self.length
        return self.lc.K[0, :n].copy(), self.lc.V[0, :n].copy()
