"""Plant plausible mistakes in a copy of the oracle and require that at least
one pin catches each of them (CPU only; the real oracle is never modified)."""
import importlib.util
import os
import sys

import pytest

from tests import oracle_pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "dmc_oracle.py")

MUTATIONS = {
    "sigmoid_sign": ("1.0 / (1.0 + np.exp(-x))", "1.0 / (1.0 + np.exp(x))"),
    "tie_rounds_up": ("return (k0 > np.float64", "return (k0 >= np.float64"),
    "no_bias": ("(k0 > np.float64(np.float32(c)))", "(k0 > 0.0)"),
    "first_token_may_accumulate": ("else logits, c) * (self.l > 0)", "else logits, c)"),
    "key_not_zeroed": ("        k[:, 0] = 0.0\n", "        pass\n"),
    "query_not_zeroed": ("        q[:, 0] = 0.0                                  # Algorithm 1: q_t[0] leaves the score",
                         "        pass"),
    "z_drops_omega": ("z_t = z_prev + omega[acc]", "z_t = z_prev + 0.5"),
    "merge_drops_old_weight": ("(self.K[acc, last] * z_prev[:, None]", "(self.K[acc, last]"),
    "value_uses_key": ("+ v[acc] * omega[acc, None]) / z_t[:, None]",
                       "+ k[acc] * omega[acc, None]) / z_t[:, None]"),
    "append_keeps_z": ("self.z[app] = omega[app]", "self.z[app] = self.z[app] + omega[app]"),
    "append_overwrites_last": ("pos = self.l[app]\n", "pos = np.maximum(self.l[app] - 1, 0)\n"),
    "wrong_scale": ("/ math.sqrt(self.d)", "/ math.sqrt(self.d - 1)"),
    "softmax_wrong_axis": ("p.sum(axis=1, keepdims=True)", "p.sum(axis=0, keepdims=True)"),
    "omega_last_head": ("w = sigmoid(q0_group[..., 0])", "w = sigmoid(q0_group[..., -1])"),
    "alpha_inverted": ("acc = np.nonzero(active & (alpha == 1))[0]",
                       "acc = np.nonzero(active & (alpha == 0) & (self.l > 0))[0]"),
    "slot_index_off_by_one": ("slot = np.where(active, self.l - 1, -1)",
                              "slot = np.where(active, self.l, -1)"),
    "prefill_ignores_lens": ("active = np.repeat(t < lens, self.Hkv)",
                             "active = np.repeat(t < n, self.Hkv)"),
    "prefill_attend_ignores_lens": ("active = np.repeat(lens > t, self.Hkv)",
                                    "active = np.repeat(n > t, self.Hkv)"),
    "uniform_weight_is_learned": ("        return np.ones(q0_group.shape[:-1])\n",
                                  "        w = sigmoid(q0_group[..., 0])\n"),
    "shared_decision_own_head": ("            k0 = np.repeat(k0[:, :1], self.Hkv, axis=1)\n", ""),
    "shared_importance_own_group": ("            q0g = np.repeat(q0g[:, :1], self.Hkv, axis=1)\n", ""),
    "window_never_resets": ("                a, om = self.wa[u, i], self.ww[u, i]",
                            "                a, om = 1, self.ww[u, i]"),
    "window_one_short": ("            m = min(self.wn[u], w)", "            m = min(self.wn[u], max(w - 1, 1))"),
}


def _mutant(name, old, new):
    with open(SRC) as f:
        text = f.read()
    assert text.count(old) == 1, f"mutation {name}: anchor not unique/absent"
    spec = importlib.util.spec_from_loader(f"oracle_mutant_{name}", loader=None)
    mod = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = mod
    exec(compile(text.replace(old, new), f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_mutation_is_caught(name):
    mod = _mutant(name, *MUTATIONS[name])
    caught = []
    for check in oracle_pins.ALL_CHECKS:
        try:
            check(mod)
        except Exception as e:  # AssertionError or a crash both count
            caught.append((check.__name__, type(e).__name__))
    assert caught, f"no pin catches mutation {name}"
