"""GPU: dmc_decode_step captured in a HIP graph and replayed.

Every decode call of a layer uses the same device buffers (the step's last
kernel copies the post-step lengths back), so a graph of one step -- the
usual serving graph, one step per layer per token -- replays correctly, and
so does one of two steps.  Each replay must equal the same number of eager
steps on a second cache with the same inputs, bit for bit, with eager work
and synchronisations between replays.
"""
import numpy as np
import pytest

from tests.gpu_helpers import f64, log, random_step

pytestmark = pytest.mark.gpu


@pytest.mark.parametrize("nsteps", [1, 2])
@pytest.mark.parametrize("G", [1, 8])
def test_decode_graph_replay(torch_cuda, G, nsteps):
    import torch
    import paper_2403_09636_amd as P
    log(f"case graph replay G={G} steps per graph={nsteps}")
    B, Hkv, d, dense = 4, 4, 128, 100
    Hq = Hkv * G
    rng = np.random.default_rng(300 + G)
    lens = torch.from_numpy(rng.integers(60, dense + 1, size=(B, Hkv)).astype(np.int32)).cuda()
    K = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    V = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    K[..., 0] = 0
    z = torch.rand((B, Hkv)).cuda() + 0.5
    cfg = P.make_config(1, B, Hq, Hkv, d, "bf16", 32, dense + 16)
    eager, graphed, warm = (P.DMCCache(cfg, device="cuda") for _ in range(3))
    for c in (eager, graphed, warm):
        c.import_(0, K, V, lens, z)
    crs = np.full(Hkv, 2.0)
    steps = [random_step(rng, B, Hq, Hkv, d, crs, "bf16", "cuda") for _ in range(nsteps)]
    warm.decode_step(0, *steps[0])             # code objects loaded before the capture
    torch.cuda.synchronize()

    outs = [torch.empty((B, Hq, d), dtype=torch.bfloat16, device="cuda") for _ in range(nsteps)]
    slots = [torch.empty((B, Hkv), dtype=torch.int32, device="cuda") for _ in range(nsteps)]
    graph = torch.cuda.CUDAGraph()
    with torch.cuda.graph(graph):
        for i in range(nsteps):
            graphed.decode_step(0, *steps[i], out=outs[i], slot_index=slots[i])

    for rep in range(3):
        graph.replay()
        torch.cuda.synchronize()
        _ = (torch.randn(1000, device="cuda") * 2).sum().item()   # eager work between replays
        for i in range(nsteps):
            ref_out = torch.empty_like(outs[i])
            ref_slot = torch.empty_like(slots[i])
            eager.decode_step(0, *steps[i], out=ref_out, slot_index=ref_slot)
            torch.cuda.synchronize()
            assert torch.equal(slots[i], ref_slot), f"replay {rep} step {i}: slot indices"
            assert torch.equal(outs[i], ref_out), f"replay {rep} step {i}: outputs"
    assert torch.equal(graphed.lengths(0), eager.lengths(0))
    ng = int(graphed.lengths(0).max())
    Kg, Vg, zg = graphed.export(0, dense_slots=ng)
    Ke, Ve, ze = eager.export(0, dense_slots=ng)
    assert torch.equal(Kg, Ke) and torch.equal(Vg, Ve) and torch.equal(zg, ze)
    assert np.isfinite(f64(outs[-1])).all()
    graphed.check()
    eager.check()
