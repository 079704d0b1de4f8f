"""GPU: the allocation-free decode entry point (dmc_decode_step_static), whose
split-K records live in the library's static device scratch, against
dmc_decode_step on identical caches, through the C ABI.

Two calls in a row share the scratch: the first on a larger cache, the second
on a smaller one (fewer units, so it reads only what it wrote itself, over
what the first call left).  Units are cut into several pieces (split_tile)
so that partial records and the per-unit record table are really used.
Results must be bit-identical (same kernels, same record layout) and the
slot indices equal; a cache whose records exceed the scratch is refused."""
import numpy as np
import pytest

from tests.gpu_helpers import log, random_step

pytestmark = pytest.mark.gpu


def _pair(P, torch, B, Hkv, G, d, dense, split, seed):
    rng = np.random.default_rng(seed)
    lens = torch.from_numpy(rng.integers(dense // 3, dense + 1, size=(B, Hkv)).astype(np.int32)).cuda()
    K = torch.randn((B, Hkv, dense, d), generator=torch.Generator().manual_seed(seed)).to(torch.bfloat16).cuda()
    V = torch.randn((B, Hkv, dense, d), generator=torch.Generator().manual_seed(seed + 1)).to(torch.bfloat16).cuda()
    K[..., 0] = 0
    z = torch.rand((B, Hkv)).cuda() + 0.5
    cfg = P.make_config(1, B, Hkv * G, Hkv, d, "bf16", 32, dense + 8, split_tile=split)
    ref, sta = P.DMCCache(cfg, device="cuda"), P.DMCCache(cfg, device="cuda")
    for c in (ref, sta):
        c.import_(0, K, V, lens, z)
    return ref, sta, rng


def _step_both(torch, ref, sta, rng, B, Hkv, G, d, what):
    q, k, v = random_step(rng, B, Hkv * G, Hkv, d, np.full(Hkv, 3.0), "bf16", "cuda")
    out_r = torch.empty((B, Hkv * G, d), dtype=torch.bfloat16, device="cuda")
    out_s = torch.full_like(out_r, 7.0)
    si_r = torch.empty((B, Hkv), dtype=torch.int32, device="cuda")
    si_s = torch.full_like(si_r, -9)
    ref.decode_step(0, q, k, v, out=out_r, slot_index=si_r)
    sta.decode_step_static(0, q, k, v, out_s, slot_index=si_s)
    torch.cuda.synchronize()
    assert torch.equal(si_r, si_s), f"{what}: slot indices"
    assert torch.equal(out_r, out_s), f"{what}: outputs differ (max abs " \
        f"{(out_r.float() - out_s.float()).abs().max().item():.3e})"
    assert torch.isfinite(out_s.float()).all()


@pytest.mark.parametrize("G", [1, 8])
def test_static_decode_matches_decode_step(torch_cuda, G):
    import torch
    import paper_2403_09636_amd as P
    d = 128
    # first call: 16 x 4 units of up to 300 slots cut into 48-slot pieces
    log(f"case static decode G={G}: call 1 (B=16, Hkv=4, split 48)")
    ref, sta, rng = _pair(P, torch, 16, 4, G, d, 300, 48, 70 + G)
    _step_both(torch, ref, sta, rng, 16, 4, G, d, "call 1")
    # second call, smaller input: 3 x 2 units, other lengths, other pieces
    log(f"case static decode G={G}: call 2 (B=3, Hkv=2, split 20)")
    ref2, sta2, rng2 = _pair(P, torch, 3, 2, G, d, 90, 20, 90 + G)
    _step_both(torch, ref2, sta2, rng2, 3, 2, G, d, "call 2")
    # the first caches again, one more step each: the scratch now holds call 2's records
    log(f"case static decode G={G}: call 3 (first caches again)")
    _step_both(torch, ref, sta, rng, 16, 4, G, d, "call 3")
    for c in (ref, sta, ref2, sta2):
        c.check()
    assert torch.equal(ref.lengths(0), sta.lengths(0))
    assert torch.equal(ref2.lengths(0), sta2.lengths(0))


def test_static_decode_refuses_records_beyond_scratch(torch_cuda):
    import torch
    import paper_2403_09636_amd as P
    log("case static decode over the scratch limit")
    # split_tile 1 over 16 units x 1024 slots: 16384 ranges of 8 x 132 fp32 > 64 MiB
    cfg = P.make_config(1, 2, 64, 8, 128, "bf16", 32, 1024, num_pages=64, split_tile=1)
    cache = P.DMCCache(cfg, device="cuda")
    q = torch.zeros((2, 64, 128), dtype=torch.bfloat16, device="cuda")
    k = torch.zeros((2, 8, 128), dtype=torch.bfloat16, device="cuda")
    out = torch.empty_like(q)
    with pytest.raises(P.DMCError) as e:
        cache.decode_step_static(0, q, k, k.clone(), out)
    assert e.value.status == P.binding.DMC_ERR_UNSUPPORTED
    assert "static" in str(e.value)
    cache.decode_step(0, q, k, k.clone(), out=out)      # the workspace entry point still serves it
    cache.check()
