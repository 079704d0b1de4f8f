"""Pins that tie the float64 oracle to what the paper and mathematics fix.

Each check takes the oracle *module* (so the mutation test can hand in a
deliberately broken copy) and raises AssertionError on a mismatch.  None of
them re-types an oracle formula: they use printed values of the paper,
closed forms, library routines (torch's scaled_dot_product_attention and
avg_pool1d), exact decimal arithmetic, and a second, independent
formulation of DMC attention (unrolled intermediate states with the additive
mask of Sec. 3.2).
"""
from __future__ import annotations

import decimal
import itertools
import json
import math
import os

import numpy as np

GOLDEN = os.path.join(os.path.dirname(os.path.abspath(__file__)), "golden")


def _golden(name):
    with open(os.path.join(GOLDEN, name)) as f:
        return json.load(f)


def _close(a, b, tol=1e-11, what=""):
    a, b = np.asarray(a, dtype=np.float64), np.asarray(b, dtype=np.float64)
    assert a.shape == b.shape, (what, a.shape, b.shape)
    err = np.max(np.abs(a - b), initial=0.0)
    assert err <= tol * max(1.0, np.max(np.abs(b), initial=0.0)), f"{what}: max err {err}"


def _run_single_unit(O, k, v, q, c=0.0, omega_src="lead"):
    """Decode a whole sequence through a 1-layer, batch-1, 1-kv-head oracle.

    k, v: [n, d]; q: [n, G, d].  Returns outputs [n, G, d], slots [n], oracle.
    """
    n, d = k.shape
    G = q.shape[1]
    orc = O.DMCOracle(1, 1, G, 1, d, max_slots=n, decision_bias=c, omega_src=omega_src)
    outs, slots = [], []
    for t in range(n):
        o, s = orc.decode_step(0, q[t][None], k[t][None, None], v[t][None, None])
        outs.append(o[0])
        slots.append(int(s[0, 0]))
    return np.array(outs), np.array(slots), orc


# ----------------------------------------------------------------------------
# An independent formulation: unrolled states + additive mask (Sec. 3.2)
# ----------------------------------------------------------------------------

def unrolled_attention(k, v, omega, alpha, q):
    """Outputs of every query under the training-time view of Sec. 3.2.

    The partial-accumulation recurrence (Sec. 3.2) keeps every intermediate
    state (z_0 = omega_0, k~_0 = k_0; z_i = z_{i-1} alpha_i + omega_i,
    k~_i = (alpha_i k~_{i-1} z_{i-1} + k_i omega_i) / z_i, same for v).
    Query i attends to state j < i with additive mask log(1 - alpha_{j+1})
    and to its own state with mask 0; future states are masked.  alpha_0 is
    unused.  k has its element 0 already zeroed; q is [n, G, d].
    """
    n, d = k.shape
    kt, vt = np.zeros_like(k), np.zeros_like(v)
    z = np.zeros(n)
    for i in range(n):
        if i == 0:
            z[0], kt[0], vt[0] = omega[0], k[0], v[0]
        else:
            z[i] = z[i - 1] * alpha[i] + omega[i]
            kt[i] = (alpha[i] * kt[i - 1] * z[i - 1] + k[i] * omega[i]) / z[i]
            vt[i] = (alpha[i] * vt[i - 1] * z[i - 1] + v[i] * omega[i]) / z[i]
    out = np.zeros((n,) + q.shape[1:])
    for i in range(n):
        mask = np.full(n, -np.inf)
        mask[i] = 0.0
        for j in range(i):
            mask[j] = 0.0 if alpha[j + 1] == 0 else -np.inf   # log(1 - alpha)
        qq = q[i].copy()
        qq[:, 0] = 0.0
        s = qq @ kt.T / math.sqrt(d) + mask[None, :]
        p = np.exp(s - s.max(axis=1, keepdims=True))
        out[i] = (p @ vt) / p.sum(axis=1, keepdims=True)
    return out


def _logits_for(alpha, rng):
    """k[0] values realising the given decisions at bias 0."""
    mag = rng.uniform(0.5, 3.0, size=len(alpha))
    return np.where(np.asarray(alpha) == 1, mag, -mag)


# ----------------------------------------------------------------------------
# Checks
# ----------------------------------------------------------------------------

def check_worked_example(O):
    """Sec. 3.2 example alpha_{1:5} = (1,1,0,1,0): slot map, l, query-5 view."""
    ex = _golden("worked_example.json")
    rng = np.random.default_rng(5)
    d = 6
    alpha = [1] + ex["alpha_1_to_5"]             # token 0 would accumulate if allowed
    n = len(alpha)
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    q = rng.standard_normal((n, 1, d))
    k[:, 0] = _logits_for(alpha, rng)
    outs, slots, orc = _run_single_unit(O, k, v, q)
    assert slots.tolist() == ex["token_to_slot"], slots
    assert int(orc.layers[0].l[0]) == ex["num_slots"]
    # query 5 sees exactly the final states of the three segments
    kh = k.copy()
    kh[:, 0] = 0.0
    omega = 1.0 / (1.0 + np.exp(-q[:, 0, 0]))
    vis = ex["query5_visible_unrolled_states"]
    eff_alpha = np.array([0] + ex["alpha_1_to_5"])
    ref = unrolled_attention(kh, v, omega, eff_alpha, q)
    _close(outs[5], ref[5], what="worked example query 5")
    # the same query restricted by hand to the visible states
    kt = np.zeros_like(kh)
    vt = np.zeros_like(v)
    z = 0.0
    for i in range(n):
        if i == 0 or eff_alpha[i] == 0:
            z, kt[i], vt[i] = omega[i], kh[i], v[i]
        else:
            zn = z + omega[i]
            kt[i] = (kt[i - 1] * z + kh[i] * omega[i]) / zn
            vt[i] = (vt[i - 1] * z + v[i] * omega[i]) / zn
            z = zn
    qq = q[5, 0].copy()
    qq[0] = 0.0
    s = np.array([qq @ kt[j] for j in vis]) / math.sqrt(d)
    p = np.exp(s - s.max())
    _close(outs[5, 0], (p[:, None] * vt[vis]).sum(0) / p.sum(), what="query 5 visible set")


def check_sigmoid_c5(O):
    """Sec. 4: c = 5 gives alpha = 0.0067 (sigmoid(-5) to four decimals)."""
    ex = _golden("sigmoid_c5.json")
    val = float(O.sigmoid(0.0 - ex["c"]))
    assert round(val, ex["decimals"]) == ex["printed_value"], val
    # importance score is the same logistic function of q[0]
    assert abs(float(O.importance(np.array([[-ex["c"]]]))[0]) - val) < 1e-15


def _exact_round_sigmoid(x, c):
    """round-half-even(sigmoid(x - c)) in 400-digit decimal arithmetic."""
    with decimal.localcontext() as ctx:
        ctx.prec = 400
        t = decimal.Decimal(float(x)) - decimal.Decimal(float(c))
        s = decimal.Decimal(1) / (decimal.Decimal(1) + (-t).exp())
        half = decimal.Decimal(1) / 2
        return 1 if s > half else 0        # s == 1/2 rounds to the even value 0


def check_exact_decisions(O):
    """Decisions equal the exactly rounded sigmoid, including tiny inputs."""
    f32 = np.float32
    tiny = [0.0, -0.0, 1e-45, -1e-45, 1.4e-45, 1e-38, -1e-38, 6e-8, -6e-8,
            1e-30, 0.5, -0.5, 3.0, -3.0]
    for c in (0.0, 5.0, -1.5):
        vals = [c + t for t in tiny] + [float(np.nextafter(f32(c), f32(np.inf))),
                                          float(np.nextafter(f32(c), f32(-np.inf))), c]
        vals = [float(f32(x)) for x in vals]
        got = O.decision(np.array(vals), c)
        want = [_exact_round_sigmoid(x, c) for x in vals]
        assert list(map(int, got)) == want, (c, vals, got, want)


def check_all_append_vanilla(O):
    """All-append decisions reproduce vanilla attention (Sec. 2.1-2.2)."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(7)
    n, d, G = 23, 8, 2
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    q = rng.standard_normal((n, G, d))
    k[:, 0] = -np.abs(k[:, 0]) - 0.1             # never accumulate
    outs, slots, orc = _run_single_unit(O, k, v, q)
    assert slots.tolist() == list(range(n))
    for t in range(n):
        qt = torch.from_numpy(q[t][:, None, 1:])                 # [G, 1, d-1]
        kt = torch.from_numpy(k[None, :t + 1, 1:]).expand(G, -1, -1)
        vt = torch.from_numpy(v[None, :t + 1]).expand(G, -1, -1)
        ref = F.scaled_dot_product_attention(qt, kt, vt, scale=1.0 / math.sqrt(d))
        _close(outs[t], ref[:, 0].numpy(), what=f"vanilla t={t}")
    # a loaded cache whose keys keep element 0: q[0] must still not count
    lc = O.LayerCache(1, d, n)
    K = rng.standard_normal((1, n, d))
    V = rng.standard_normal((1, n, d))
    lc.load(K, V, [n], [1.0])
    qq = rng.standard_normal((G, d))
    ref = F.scaled_dot_product_attention(
        torch.from_numpy(qq[:, None, 1:]), torch.from_numpy(K[:, :, 1:]).expand(G, -1, -1),
        torch.from_numpy(V).expand(G, -1, -1), scale=1.0 / math.sqrt(d))
    _close(lc.attend(0, qq), ref[:, 0].numpy(), what="loaded cache")


def check_all_accumulate(O):
    """All-accumulate: one slot = omega-weighted mean; output = that value."""
    rng = np.random.default_rng(11)
    n, d = 17, 5
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    q = rng.standard_normal((n, 1, d))
    k[:, 0] = np.abs(k[:, 0]) + 0.1
    outs, slots, orc = _run_single_unit(O, k, v, q)
    assert slots.tolist() == [0] * n
    w = 1.0 / (1.0 + np.exp(-q[:, 0, 0]))
    kh = k.copy()
    kh[:, 0] = 0.0
    for t in range(n):
        _close(outs[t, 0], np.average(v[:t + 1], axis=0, weights=w[:t + 1]),
               what=f"accumulate out t={t}")
    K, V, lens, z = orc.export(0)
    assert lens[0, 0] == 1
    _close(K[0, 0, 0], np.average(kh, axis=0, weights=w), what="accumulated key")
    _close(V[0, 0, 0], np.average(v, axis=0, weights=w), what="accumulated value")
    _close(z[0, 0], w.sum(), what="z")


def check_segments(O):
    """Random decisions: slot count, slot indices and segment closed form."""
    rng = np.random.default_rng(13)
    for trial in range(6):
        n, d = int(rng.integers(1, 40)), 4
        alpha = rng.integers(0, 2, size=n)
        k = rng.standard_normal((n, d))
        v = rng.standard_normal((n, d))
        q = rng.standard_normal((n, 1, d))
        k[:, 0] = _logits_for(alpha, rng)
        _, slots, orc = _run_single_unit(O, k, v, q)
        eff = alpha.copy()
        eff[0] = 0
        starts = np.nonzero(eff == 0)[0]
        assert int(orc.layers[0].l[0]) == 1 + int((alpha[1:] == 0).sum())
        assert slots.tolist() == (np.cumsum(1 - eff) - 1).tolist()
        K, V, lens, z = orc.export(0)
        w = 1.0 / (1.0 + np.exp(-q[:, 0, 0]))
        kh = k.copy()
        kh[:, 0] = 0.0
        bounds = list(starts) + [n]
        for s in range(len(starts)):
            a, b = bounds[s], bounds[s + 1]
            _close(K[0, 0, s], np.average(kh[a:b], axis=0, weights=w[a:b]), what="seg K")
            _close(V[0, 0, s], np.average(v[a:b], axis=0, weights=w[a:b]), what="seg V")
        _close(z[0, 0], w[starts[-1]:].sum(), what="z of the open segment")


def check_avg_pool(O):
    """Fixed memory pooling (DMC ablations): periodic appends, constant omega
    reduce to avg_pool1d with kernel = stride = CR."""
    import torch
    import torch.nn.functional as F
    rng = np.random.default_rng(17)
    cr, m, d = 4, 6, 8
    n = cr * m
    alpha = np.array([0 if t % cr == 0 else 1 for t in range(n)])
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    q = rng.standard_normal((n, 1, d))
    q[:, 0, 0] = 0.3                              # constant omega
    k[:, 0] = _logits_for(alpha, rng)
    _, _, orc = _run_single_unit(O, k, v, q)
    K, V, lens, _ = orc.export(0)
    assert lens[0, 0] == m
    kh = k.copy()
    kh[:, 0] = 0.0
    pk = F.avg_pool1d(torch.from_numpy(kh.T[None]), cr, cr)[0].T.numpy()
    pv = F.avg_pool1d(torch.from_numpy(v.T[None]), cr, cr)[0].T.numpy()
    _close(K[0, 0, :m], pk, what="pooled K")
    _close(V[0, 0, :m], pv, what="pooled V")


def check_bruteforce_unrolled(O):
    """Every decision pattern for n <= 8 (d in {4, 8}) against the unrolled
    states with the additive mask (Sec. 3.2), run as a batch of units."""
    rng = np.random.default_rng(19)
    for n, d, G in ((8, 4, 1), (6, 8, 2)):
        pats = np.array(list(itertools.product((0, 1), repeat=n - 1)))
        P = len(pats)
        alpha = np.concatenate([np.zeros((P, 1), int), pats], axis=1)      # [P, n]
        k = rng.standard_normal((P, n, d))
        v = rng.standard_normal((P, n, d))
        q = rng.standard_normal((P, n, G, d))
        k[:, :, 0] = np.where(alpha == 1, 1.0, -1.0) * rng.uniform(0.5, 2, (P, n))
        k[:, 0, 0] = rng.uniform(0.5, 2, P)          # token 0 must append anyway
        orc = O.DMCOracle(1, P, G, 1, d, max_slots=n)
        outs = np.zeros((P, n, G, d))
        for t in range(n):
            o, _ = orc.decode_step(0, q[:, t], k[:, t][:, None], v[:, t][:, None])
            outs[:, t] = o
        kh = k.copy()
        kh[:, :, 0] = 0.0
        for p in range(P):
            omega = 1.0 / (1.0 + np.exp(-q[p, :, 0, 0]))
            ref = unrolled_attention(kh[p], v[p], omega, alpha[p], q[p])
            _close(outs[p], ref, tol=1e-10, what=f"pattern {pats[p]}")


def check_gqa_omega(O):
    """GQA: alpha from the kv head, omega from the lead query head (or the
    group mean); each query head of the group attends to the shared cache."""
    rng = np.random.default_rng(23)
    n, d, G = 9, 4, 4
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    q = rng.standard_normal((n, G, d))
    k[:, 0] = np.abs(k[:, 0]) + 0.1                        # all accumulate
    for src in ("lead", "group_mean"):
        outs, _, _ = _run_single_unit(O, k, v, q, omega_src=src)
        sig = 1.0 / (1.0 + np.exp(-q[:, :, 0]))
        w = sig[:, 0] if src == "lead" else sig.mean(axis=1)
        for t in range(n):
            want = np.average(v[:t + 1], axis=0, weights=w[:t + 1])
            for h in range(G):
                _close(outs[t, h], want, what=f"{src} head {h}")


def check_permutation(O):
    """Independent units: permuting batch rows / kv heads permutes results."""
    rng = np.random.default_rng(29)
    B, Hkv, G, d, n = 3, 2, 2, 4, 7
    Hq = Hkv * G
    q = rng.standard_normal((n, B, Hq, d))
    k = rng.standard_normal((n, B, Hkv, d))
    v = rng.standard_normal((n, B, Hkv, d))
    pb, pg = np.array([2, 0, 1]), np.array([1, 0])
    ph = np.concatenate([np.arange(g * G, (g + 1) * G) for g in pg])
    o1 = O.DMCOracle(1, B, Hq, Hkv, d, max_slots=n)
    o2 = O.DMCOracle(1, B, Hq, Hkv, d, max_slots=n)
    for t in range(n):
        a, sa = o1.decode_step(0, q[t], k[t], v[t])
        b, sb = o2.decode_step(0, q[t][pb][:, ph], k[t][pb][:, pg], v[t][pb][:, pg])
        _close(b, a[pb][:, ph], tol=0.0, what="permuted outputs")
        assert (sb == sa[pb][:, pg]).all()


def check_prefill_matches_decode(O):
    """The prompt phase equals sequential updates, ragged prompts included."""
    rng = np.random.default_rng(31)
    B, Hq, Hkv, d, n = 3, 4, 2, 4, 11
    G = Hq // Hkv
    k = rng.standard_normal((B, n, Hkv, d))
    v = rng.standard_normal((B, n, Hkv, d))
    q0 = rng.standard_normal((B, n, Hq))
    lens = np.array([11, 0, 5])
    a = O.DMCOracle(1, B, Hq, Hkv, d, max_slots=n)
    slots = a.prefill(0, k, v, q0, prompt_lens=lens)
    for b in range(B):
        for g in range(Hkv):
            qq = np.zeros((n, G, d))
            qq[:, :, 0] = q0[b, :, g * G:(g + 1) * G]
            _, s1, ob = _run_single_unit(O, k[b, :lens[b], g], v[b, :lens[b], g], qq[:lens[b]])
            assert slots[b, g, :lens[b]].tolist() == s1.tolist()
            assert (slots[b, g, lens[b]:] == -1).all()
            K1, V1, l1, z1 = ob.export(0)
            K2, V2, l2, z2 = a.export(0)
            assert l1[0, 0] == l2[b, g]
            _close(K2[b, g, :l2[b, g]], K1[0, 0, :l1[0, 0]], tol=0.0, what="prefill K")
            _close(V2[b, g, :l2[b, g]], V1[0, 0, :l1[0, 0]], tol=0.0, what="prefill V")


def check_prefill_attend(O):
    """Prompt-phase attention equals token-by-token decode steps and the
    unrolled states with the additive mask of Sec. 3.2, per unit; ragged
    prompt lengths leave zero outputs past each row's end."""
    rng = np.random.default_rng(37)
    B, Hkv, G, d, n = 3, 2, 2, 4, 9
    Hq = Hkv * G
    q = rng.standard_normal((B, n, Hq, d))
    k = rng.standard_normal((B, n, Hkv, d))
    v = rng.standard_normal((B, n, Hkv, d))
    lens = np.array([9, 4, 0])
    orc = O.DMCOracle(1, B, Hq, Hkv, d, max_slots=n)
    out, slots = orc.prefill_attend(0, q, k, v, prompt_lens=lens)
    for b in range(B):
        assert (out[b, lens[b]:] == 0).all()
        for g in range(Hkv):
            m = lens[b]
            if m == 0:
                assert (slots[b, g] == -1).all()
                continue
            kk = k[b, :m, g].copy()
            alpha = (kk[:, 0] > 0).astype(int)
            alpha[0] = 0
            kk[:, 0] = 0.0
            omega = 1.0 / (1.0 + np.exp(-q[b, :m, g * G, 0]))
            ref = unrolled_attention(kk, v[b, :m, g], omega, alpha, q[b, :m, g * G:(g + 1) * G])
            _close(out[b, :m, g * G:(g + 1) * G], ref, tol=1e-10, what=f"prefill attend {(b, g)}")
            assert slots[b, g, :m].tolist() == (np.cumsum(1 - alpha) - 1).tolist()


def check_uniform_weighting(O):
    """Uniform weighting (appendix ablations): every slot is the plain
    arithmetic mean of its segment (np.mean), z of the open slot is the
    segment's token count, and attention is softmax over those means."""
    rng = np.random.default_rng(41)
    n, d, G = 37, 6, 2
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    q = rng.standard_normal((n, G, d)) * 3.0          # varied q[0]: learned omega would differ
    orc = O.DMCOracle(1, 1, G, 1, d, max_slots=n, omega_src="uniform")
    outs = []
    for t in range(n):
        o, _ = orc.decode_step(0, q[t][None], k[t][None, None], v[t][None, None])
        outs.append(o[0])
    alpha = (k[:, 0] > 0).astype(int)
    alpha[0] = 0
    starts = list(np.nonzero(alpha == 0)[0]) + [n]
    kh = k.copy()
    kh[:, 0] = 0.0
    Km = np.array([kh[a:b].mean(axis=0) for a, b in zip(starts[:-1], starts[1:])])
    Vm = np.array([v[a:b].mean(axis=0) for a, b in zip(starts[:-1], starts[1:])])
    K, V, l, z = orc.export(0)
    L = int(l[0, 0])
    assert L == len(starts) - 1
    _close(K[0, 0, :L], Km, what="uniform slots K")
    _close(V[0, 0, :L], Vm, what="uniform slots V")
    assert abs(z[0, 0] - (starts[-1] - starts[-2])) < 1e-12
    qq = q[-1].copy()
    qq[:, 0] = 0.0
    sc = qq @ Km.T / math.sqrt(d)
    p = np.exp(sc - sc.max(axis=1, keepdims=True))
    _close(outs[-1], (p @ Vm) / p.sum(axis=1, keepdims=True), what="uniform attention")


def check_shared_layer_decisions(O):
    """DMC-HardC (decision and importance shared by a layer's heads, taken
    from kv head 0 of the row) equals per-head DMC run on inputs whose every
    head carries head 0's decision and importance neurons; all heads of a row
    then have equal lengths.  Both omega sources, prefill and decode."""
    rng = np.random.default_rng(43)
    B, Hkv, G, d, n = 2, 3, 2, 8, 24
    Hq = Hkv * G
    for src in ("lead", "group_mean"):
        k = rng.standard_normal((B, n, Hkv, d))
        v = rng.standard_normal((B, n, Hkv, d))
        q = rng.standard_normal((B, n, Hq, d))
        k2, q2 = k.copy(), q.copy()
        for g in range(Hkv):
            k2[:, :, g, 0] = k[:, :, 0, 0]
            q2[:, :, g * G:(g + 1) * G, 0] = q[:, :, 0:G, 0]
        hard = O.DMCOracle(1, B, Hq, Hkv, d, max_slots=2 * n, omega_src=src,
                           decision_src="shared_layer")
        ref = O.DMCOracle(1, B, Hq, Hkv, d, max_slots=2 * n, omega_src=src)
        half = n // 2
        s1 = hard.prefill(0, k[:, :half], v[:, :half], q[:, :half, :, 0])
        s2 = ref.prefill(0, k2[:, :half], v[:, :half], q2[:, :half, :, 0])
        assert (s1 == s2).all()
        for t in range(half, n):
            o1, i1 = hard.decode_step(0, q[:, t], k[:, t], v[:, t])
            o2, i2 = ref.decode_step(0, q2[:, t], k2[:, t], v[:, t])
            assert (i1 == i2).all()
            _close(o1, o2, tol=0.0, what=f"shared-layer decode {src}")
        l = hard.export(0)[2]
        assert (l == l[:, :1]).all(), l


def _run_window(O, k, v, q, w):
    n, d = k.shape
    G = q.shape[1]
    orc = O.DMCOracle(1, 1, G, 1, d, max_slots=n, window=w)
    outs, slots = [], []
    for t in range(n):
        o, s_ = orc.decode_step(0, q[t][None], k[t][None, None], v[t][None, None])
        outs.append(o[0])
        slots.append(int(s_[0, 0]))
    return np.array(outs), np.array(slots), orc


def check_window_segments(O):
    """Window grouping (Sec. 3.3): every slot is the omega-weighted mean
    (np.average) of the last min(w, length) tokens of its segment; z is the
    omega sum of the open segment's last min(w, length) tokens; slot indices
    are the segment indices.  w = 1 keeps each segment's last token."""
    rng = np.random.default_rng(47)
    n, d = 40, 6
    for w in (1, 3, 12):
        k = rng.standard_normal((n, d))
        v = rng.standard_normal((n, d))
        q = rng.standard_normal((n, 1, d))
        k[:, 0] = _logits_for(rng.uniform(size=n) < 0.8, rng)   # long runs of accumulation
        outs, slots, orc = _run_window(O, k, v, q, w)
        alpha = (k[:, 0] > 0).astype(int)
        alpha[0] = 0
        assert slots.tolist() == (np.cumsum(1 - alpha) - 1).tolist()
        starts = list(np.nonzero(alpha == 0)[0]) + [n]
        omega = 1.0 / (1.0 + np.exp(-q[:, 0, 0]))
        kh = k.copy()
        kh[:, 0] = 0.0
        K, V, l, z = orc.export(0)
        assert int(l[0, 0]) == len(starts) - 1
        for j, (a, b) in enumerate(zip(starts[:-1], starts[1:])):
            lo = max(a, b - w)
            _close(K[0, 0, j], np.average(kh[lo:b], axis=0, weights=omega[lo:b]), what=f"w{w} K{j}")
            _close(V[0, 0, j], np.average(v[lo:b], axis=0, weights=omega[lo:b]), what=f"w{w} V{j}")
            if w == 1:
                _close(K[0, 0, j], kh[b - 1], what="w1 last token")
        a, b = starts[-2], starts[-1]
        assert abs(z[0, 0] - omega[max(a, b - w):b].sum()) < 1e-12


def check_window_wide_is_exact(O):
    """A window at least as long as the sequence changes nothing."""
    rng = np.random.default_rng(53)
    n, d, G = 30, 8, 2
    k = rng.standard_normal((n, d))
    v = rng.standard_normal((n, d))
    q = rng.standard_normal((n, G, d))
    o1, s1, _ = _run_window(O, k, v, q, n)
    o2, s2, _ = _run_single_unit(O, k, v, q)
    assert (s1 == s2).all()
    _close(o1, o2, tol=1e-12, what="wide window")


def windowed_unrolled_attention(k, v, omega, alpha, q, w):
    """Training-time view with window grouping (Sec. 3.2 + Sec. 3.3): the
    state of position j is the partial-accumulation recurrence over
    positions max(0, j-w+1) .. j, started afresh at the first of them; query
    i sees its own state and each state j < i with alpha_{j+1} = 0."""
    n, d = k.shape
    kt, vt = np.zeros_like(k), np.zeros_like(v)
    for j in range(n):
        j0 = max(0, j - w + 1)
        z, ks, vs = omega[j0], k[j0].copy(), v[j0].copy()
        for i in range(j0 + 1, j + 1):
            zn = alpha[i] * z + omega[i]
            ks = (alpha[i] * ks * z + k[i] * omega[i]) / zn
            vs = (alpha[i] * vs * z + v[i] * omega[i]) / zn
            z = zn
        kt[j], vt[j] = ks, vs
    out = np.zeros((n,) + q.shape[1:])
    for i in range(n):
        vis = [j for j in range(i) if alpha[j + 1] == 0] + [i]
        qq = q[i].copy()
        qq[:, 0] = 0.0
        s = qq @ kt[vis].T / math.sqrt(d)
        p = np.exp(s - s.max(axis=1, keepdims=True))
        out[i] = (p @ vt[vis]) / p.sum(axis=1, keepdims=True)
    return out


def check_window_bruteforce(O):
    """Every decision pattern of a short sequence, windows 2 and 3: decode
    outputs equal the windowed unrolled-state formulation."""
    rng = np.random.default_rng(59)
    n, d = 7, 4
    for w in (2, 3):
        for bits in itertools.product([0, 1], repeat=n - 1):
            alpha = np.array((0,) + bits)
            k = rng.standard_normal((n, d))
            v = rng.standard_normal((n, d))
            q = rng.standard_normal((n, 1, d))
            k[:, 0] = _logits_for(alpha, rng)
            outs, _, _ = _run_window(O, k, v, q, w)
            kh = k.copy()
            kh[:, 0] = 0.0
            omega = 1.0 / (1.0 + np.exp(-q[:, 0, 0]))
            ref = windowed_unrolled_attention(kh, v, omega, alpha, q, w)
            _close(outs, ref, tol=1e-10, what=f"window {w} pattern {bits}")


ALL_CHECKS = [check_worked_example, check_sigmoid_c5, check_exact_decisions,
              check_all_append_vanilla, check_all_accumulate, check_segments,
              check_avg_pool, check_bruteforce_unrolled, check_gqa_omega,
              check_permutation, check_prefill_matches_decode, check_prefill_attend,
              check_uniform_weighting, check_shared_layer_decisions, check_window_segments,
              check_window_wide_is_exact, check_window_bruteforce]
