"""GPU: seeded random configurations through prompt attention, the
compacted cache and decode, against the float64 oracle, through the C ABI.

The fixed-grid tests pin chosen boundaries.  Here every case draws its
shape, query group, head dimension, page size, dtype, prompt lengths,
per-head compression ratios, decision bias, importance source, decision
source, window and forced split independently, so that combinations the
grids skip are exercised too: pages of 8 or 16 slots under grouped queries,
ragged tails in every block and chunk loop, stream-K ranges cut inside
units, empty and one-token prompts next to long ones."""
import numpy as np
import pytest

from tests.gpu_helpers import Pair, log, random_step
from workloads import decision_logits

pytestmark = pytest.mark.gpu

CASES = 256


def _draw(seed):
    rng = np.random.default_rng(9000 + seed)
    c = {
        "dtype": "fp32" if rng.random() < 0.2 else "bf16",
        "d": int(rng.choice([64, 128])),
        "G": int(rng.choice([1, 2, 4, 8])),
        "Hkv": int(rng.integers(1, 4)),
        "B": int(rng.integers(1, 4)),
        "page": int(rng.choice([8, 16, 32, 32, 64])),
        "n": int(rng.integers(1, 261)),
        "bias": float(rng.choice([0.0, 0.0, 1.5])),
        "omega": str(rng.choice(["lead", "lead", "group_mean", "uniform"])),
        "decision": "shared_layer" if rng.random() < 0.15 else "per_head",
        "window": int(rng.choice([0, 0, 0, 3, 12])),
        "split": int(rng.choice([0, 0, 7, 23])),
    }
    # prompt lengths: the full prompt, a random cut, and the edge lengths 0 and 1
    lens = rng.integers(0, c["n"] + 1, size=c["B"])
    lens[0] = c["n"]
    if c["B"] > 2:
        lens[2] = int(rng.choice([0, 1]))
    c["lens"] = [int(x) for x in lens]
    c["crs"] = [float(x) for x in rng.choice([1.0, 1.5, 3.0, 8.0, 1e9], size=c["Hkv"])]
    return rng, c


@pytest.mark.parametrize("seed", range(CASES))
def test_random_configuration(torch_cuda, seed):
    import torch
    rng, c = _draw(seed)
    log(f"case random seed={seed} {c}")
    B, n, Hkv, G, d, dtype = c["B"], c["n"], c["Hkv"], c["G"], c["d"], c["dtype"]
    steps = 4
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, page_size=c["page"], max_slots=n + steps + 8,
              bias=c["bias"], omega_src=c["omega"], split_tile=c["split"], max_prompt_len=n,
              decision_src=c["decision"], window=c["window"])
    dt = torch.float32 if dtype == "fp32" else torch.bfloat16
    k = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    v = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    q = rng.standard_normal((B, n, Hkv * G, d), dtype=np.float32)
    k[..., 0] = decision_logits(rng.uniform(size=(B, n, Hkv)), np.asarray(c["crs"])[None, None],
                                c["bias"])
    k, v, q = (torch.from_numpy(x).to(dt).cuda() for x in (k, v, q))
    err = pr.prefill_attend(0, k, v, q, prompt_lens=c["lens"])
    pr.compare_cache(0)
    for _ in range(steps):
        err = max(err, pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.asarray(c["crs"]),
                                                  dtype, "cuda", c["bias"])))
    pr.compare_cache(0)
    pr.ok()
    log(f"  lengths {pr.gpu.lengths(0).cpu().numpy().tolist()}, max abs err {err:.3e}")
