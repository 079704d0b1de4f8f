"""Variants of the appendix ablations on the GPU against the float64 oracle:
uniform weighting (omega = 1), DMC-HardC (decision and importance shared by
the heads of a layer, from kv head 0 of each batch row) and the padded
per-unit layout of DMC-C (one page as large as the slot capacity)."""
import numpy as np
import pytest

from tests.gpu_helpers import Pair, log, random_step
from workloads import decision_logits

pytestmark = pytest.mark.gpu


def _prompt(rng, B, n, Hkv, G, d, crs, dtype):
    import torch
    k = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    v = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    q = rng.standard_normal((B, n, Hkv * G, d), dtype=np.float32)
    k[..., 0] = decision_logits(rng.uniform(size=(B, n, Hkv)), np.asarray(crs)[None, None])
    dt = torch.float32 if dtype == "fp32" else torch.bfloat16
    return tuple(torch.from_numpy(x).to(dt).cuda() for x in (k, v, q))


def _run(pr, rng, B, Hkv, G, d, crs, dtype, n, steps, lens=None):
    k, v, q = _prompt(rng, B, n, Hkv, G, d, crs, dtype)
    err = pr.prefill_attend(0, k, v, q, prompt_lens=lens)
    pr.compare_cache(0)
    for _ in range(steps):
        err = max(err, pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.array(crs), dtype,
                                                 "cuda")))
    pr.compare_cache(0)
    pr.ok()
    return err


@pytest.mark.parametrize("dtype,d,G", [("bf16", 128, 1), ("bf16", 128, 8), ("fp32", 64, 2)])
def test_uniform_weighting(torch_cuda, dtype, d, G):
    log(f"case uniform omega dtype={dtype} d={d} G={G}")
    B, Hkv, n = 3, 2, 150
    rng = np.random.default_rng(200 + d + G)
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, max_slots=n + 40, max_prompt_len=n, omega_src="uniform")
    err = _run(pr, rng, B, Hkv, G, d, [2.0, 9.0], dtype, n, 30, lens=[n, 70, 1])
    log(f"  max abs err {err:.3e}")


@pytest.mark.parametrize("dtype,d,G,omega", [("bf16", 128, 1, "lead"), ("bf16", 128, 8, "lead"),
                                             ("bf16", 64, 4, "group_mean"), ("fp32", 128, 2, "lead")])
def test_shared_layer_decisions(torch_cuda, dtype, d, G, omega):
    """DMC-HardC: every head of a row follows kv head 0, so per-row lengths
    are equal across heads (bit-exact against the oracle as well)."""
    log(f"case shared-layer dtype={dtype} d={d} G={G} omega={omega}")
    B, Hkv, n = 2, 4, 130
    rng = np.random.default_rng(300 + d + G)
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, max_slots=n + 40, max_prompt_len=n, omega_src=omega,
              decision_src="shared_layer")
    err = _run(pr, rng, B, Hkv, G, d, [3.0, 1.0, 12.0, 2.0], dtype, n, 30)
    lens = pr.gpu.lengths(0).cpu().numpy()
    assert (lens == lens[:, :1]).all(), lens
    log(f"  lengths {lens[:, 0].tolist()}, max abs err {err:.3e}")


@pytest.mark.parametrize("dtype,G,page", [("bf16", 1, 256), ("bf16", 4, 512), ("fp32", 2, 1024)])
def test_padded_unit_layout(torch_cuda, dtype, G, page):
    """DMC-C storage: one page per unit as large as its slot capacity (a
    padded [B, H, capacity, d] tensor), prompt with attention then decode."""
    log(f"case padded layout dtype={dtype} G={G} page={page}")
    B, Hkv, d, n = 2, 3, 128, 200
    rng = np.random.default_rng(400 + G + page)
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, page_size=page, max_slots=page, max_prompt_len=n)
    err = _run(pr, rng, B, Hkv, G, d, [1.5, 4.0, 30.0], dtype, n, 24)
    assert pr.gpu.pages_used() == B * Hkv
    log(f"  max abs err {err:.3e}")
