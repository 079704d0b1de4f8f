"""The float64 training oracle against its pins, and planted mistakes in a
copy of it that the pins must catch (CPU only)."""
import importlib.util
import os
import sys

import pytest

import oracle.dmc_train as T
from tests import train_pins

SRC = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))),
                   "oracle", "dmc_train.py")

MUTATIONS = {
    "noise_sign": ("x = (k0 - c + noise) / tau", "x = (k0 - c - noise) / tau"),
    "tau_multiplies": ("x = (k0 - c + noise) / tau", "x = (k0 - c + noise) * tau"),
    "mask_own_alpha": ("col[:, : n - 1] = torch.nn.functional.logsigmoid(-x[:, 1:])",
                       "col[:, : n - 1] = torch.nn.functional.logsigmoid(-x[:, :-1])"),
    "diagonal_masked": ("M = torch.where((j == i)[None], torch.zeros((), dtype=x.dtype), M)",
                        "M = M"),
    "window_one_long": ("a = max(0, j - window + 1)", "a = max(0, j - window)"),
    "window_start_uses_alpha": ("        z = omega[:, a]\n", "        z = omega[:, a] * alpha[:, a]\n"),
    "z_drops_omega": ("zn = alpha[:, i] * z + omega[:, i]", "zn = alpha[:, i] * z + 0.5"),
    # both zeroings dropped (either one alone keeps element 0 out of every score)
    "first_neurons_scored": [
        ("kh = torch.cat([torch.zeros_like(ku[:, :, :1]), ku[:, :, 1:]], dim=2)   # k[0] <- 0",
         "kh = ku"),
        ("qz = torch.cat([torch.zeros_like(qu[..., :1]), qu[..., 1:]], dim=3)       # q[0] <- 0",
         "qz = qu")],
    "omega_last_head": ("omega = importance(qu[:, 0, :, 0], omega_src)",
                        "omega = importance(qu[:, -1, :, 0], omega_src)"),
    "scale_d_minus_1": ("/ math.sqrt(d)                        # [U, G, n, n]",
                        "/ math.sqrt(d - 1)                    # [U, G, n, n]"),
}


@pytest.mark.parametrize("check", train_pins.ALL_CHECKS, ids=lambda f: f.__name__)
def test_train_pin(check):
    check(T)


def _mutant(name, edits):
    with open(SRC) as f:
        text = f.read()
    for old, new in (edits if isinstance(edits, list) else [edits]):
        assert text.count(old) == 1, f"mutation {name}: anchor not unique/absent"
        text = text.replace(old, new)
    spec = importlib.util.spec_from_loader(f"train_mutant_{name}", loader=None)
    mod = importlib.util.module_from_spec(spec)
    sys.modules[spec.name] = mod
    exec(compile(text, f"<mutant {name}>", "exec"), mod.__dict__)
    return mod


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_train_mutation_is_caught(name):
    mod = _mutant(name, MUTATIONS[name])
    caught = []
    for check in train_pins.ALL_CHECKS:
        try:
            check(mod)
        except Exception as e:  # AssertionError or a crash both count
            caught.append((check.__name__, type(e).__name__))
    assert caught, f"no pin catches mutation {name}"
