"""GPU: layers with more units than the decode kernel's full slot-space table
holds in LDS (grouped table entries, every g-th unit's offset), through the
C ABI: Llama-2-7B heads at batch 512 (16,384 units, vector-ALU decode) and
Llama-2-70B grouped-query heads at batch 1024 (8,192 units, matrix-core
decode).  Ragged imported caches, then decode steps; every unit's slot index
and length against the oracle's decision rule, and the outputs, slots and z
of >= 64 sampled units against per-unit oracles (units are independent).  A
forced split cuts units into many pieces, so ranges start inside groups."""
import numpy as np
import pytest

import oracle
from tests.gpu_helpers import assert_close, f64, log, random_step

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("B,Hq,Hkv,split", [(512, 32, 32, 0), (512, 32, 32, 23), (1024, 64, 8, 0)])
def test_grouped_slot_space_table(torch_cuda, B, Hq, Hkv, split):
    import torch
    import paper_2403_09636_amd as P
    d, G, steps, dense = 128, Hq // Hkv, 3, 72
    U = B * Hkv
    log(f"case grouped table B={B} Hq={Hq} Hkv={Hkv} ({U} units) split={split}")
    rng = np.random.default_rng(U + split)
    lens_np = rng.integers(0, dense + 1, size=(B, Hkv)).astype(np.int32)
    lens_np[rng.random((B, Hkv)) < 0.05] = 0            # some empty units
    K = torch.randn((B, Hkv, dense, d), generator=torch.Generator().manual_seed(U)).to(torch.bfloat16).cuda()
    V = torch.randn((B, Hkv, dense, d), generator=torch.Generator().manual_seed(U + 1)).to(torch.bfloat16).cuda()
    K[..., 0] = 0
    z_np = (rng.random((B, Hkv)) + 0.5).astype(np.float32)
    cfg = P.make_config(1, B, Hq, Hkv, d, "bf16", 32, dense + steps + 1, split_tile=split)
    cache = P.DMCCache(cfg, device="cuda")
    cache.import_(0, K, V, torch.from_numpy(lens_np).cuda(), torch.from_numpy(z_np).cuda())
    units = sorted({(int(b), int(g)) for b, g in zip(rng.integers(B, size=64), rng.integers(Hkv, size=64))}
                   | {(0, 0), (B - 1, Hkv - 1)})
    orcs = {}
    for b, g in units:
        o = oracle.DMCOracle(1, 1, G, 1, d, dense + steps + 1)
        n = int(lens_np[b, g])
        o.load(0, f64(K[b, g, :n])[None, None], f64(V[b, g, :n])[None, None], np.array([[n]]),
               np.array([[float(z_np[b, g])]]))
        orcs[(b, g)] = o
    del K, V
    lens = lens_np.astype(np.int64)
    worst = 0.0
    for s in range(steps):
        q, k, v = random_step(rng, B, Hq, Hkv, d, np.full(Hkv, 3.0), "bf16", "cuda")
        si = torch.empty((B, Hkv), dtype=torch.int32, device="cuda")
        out = cache.decode_step(0, q, k, v, slot_index=si)
        alpha = oracle.decision(f64(k[:, :, 0]), 0.0) * (lens > 0)
        want = np.where(alpha == 1, lens - 1, lens)
        assert (si.cpu().numpy() == want).all(), f"step {s}: slot indices"
        lens = lens + (1 - alpha)
        for (b, g), o in orcs.items():
            ref, _ = o.decode_step(0, f64(q[b, g * G:(g + 1) * G])[None], f64(k[b, g])[None, None],
                                   f64(v[b, g])[None, None])
            worst = max(worst, assert_close(f64(out[b, g * G:(g + 1) * G]), ref[0], "bf16",
                                            f"step {s} unit {(b, g)} output"))
    assert (cache.lengths(0).cpu().numpy() == lens).all(), "lengths"
    Kx, Vx, zx = cache.export(0, dense_slots=dense + steps)
    for (b, g), o in orcs.items():
        Kr, Vr, lr, zr = o.export(0)
        n = int(lr[0, 0])
        assert_close(f64(Kx[b, g, :n]), Kr[0, 0, :n], "bf16", f"unit {(b, g)} keys")
        assert_close(f64(Vx[b, g, :n]), Vr[0, 0, :n], "bf16", f"unit {(b, g)} values")
        if n:
            assert abs(float(zx[b, g]) - zr[0, 0]) <= 1e-4 * max(1.0, abs(zr[0, 0])), "z"
    cache.check()
    log(f"  {len(orcs)} sampled units, max abs err {worst:.3e}")
