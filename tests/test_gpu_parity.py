"""GPU parity: the HIP path (through the C ABI) against the float64 oracle.

Small and ragged shapes that finish in seconds on the CPU side but span
several pages, split-K tiles and 64-token prefill chunks, plus the edge
cases of the method (empty cache, first token, all-append, all-accumulate,
one slot, page and tile boundaries, ragged and empty prompts).
"""
import numpy as np
import pytest

from tests.gpu_helpers import Pair, f64, log, random_step
from workloads import WORKLOADS, decision_logits, decode_inputs_np

pytestmark = pytest.mark.gpu




def test_tiny_workload_full(torch_cuda):
    """1 layer, batch 1, 4 heads (CR 1, 2, 4, 8), d64, fp32, 256 steps from
    an empty cache: every output, slot index, length, slot and z."""
    w = WORKLOADS["tiny"]
    log(f"case tiny: {w.notes}")
    pr = Pair(1, w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, "fp32",
              max_slots=w.max_slots)
    worst = 0.0
    for step in range(w.decode_steps):
        q, k, v = (t.cuda() for t in decode_inputs_np(w, step, 0))
        worst = max(worst, pr.decode(0, q, k, v))
        if step % 64 == 63:
            pr.compare_cache(0)
    pr.compare_cache(0)
    pr.ok()
    lens = pr.gpu.lengths(0).cpu().numpy()[0]
    log(f"tiny: final lengths {lens.tolist()} max abs err {worst:.2e}")
    assert lens[0] == w.decode_steps            # CR 1 head appends every token


VARIANTS = [
    # dtype, d, G, page, tile, omega, bias
    ("bf16", 128, 1, 32, 0, "lead", 0.0),
    ("bf16", 128, 1, 32, 8, "lead", 0.0),
    ("bf16", 64, 2, 16, 24, "lead", 0.0),
    ("bf16", 128, 4, 8, 40, "group_mean", 0.0),
    ("bf16", 128, 8, 32, 32, "lead", 0.7),
    ("fp32", 128, 1, 32, 16, "lead", 0.0),
    ("fp32", 64, 4, 32, 0, "group_mean", -0.5),
    ("fp32", 128, 8, 64, 64, "lead", 0.0),
    ("fp32", 64, 1, 256, 7, "lead", 0.0),
    # grouped-query caches on matrix cores (bf16, G >= 4, 32-slot pages)
    ("bf16", 128, 4, 32, 0, "lead", 0.0),
    ("bf16", 64, 8, 32, 0, "group_mean", 0.0),
    ("bf16", 64, 4, 32, 16, "lead", -0.3),
    ("bf16", 128, 8, 32, 5, "group_mean", 0.0),
    # one slot per range: units split into up to 75 pieces (> 64 records in the combine)
    ("fp32", 64, 1, 32, 1, "lead", 0.0),
]


@pytest.mark.parametrize("dtype,d,G,page,tile,omega,bias", VARIANTS)
def test_decode_variants(torch_cuda, dtype, d, G, page, tile, omega, bias):
    """2 layers, ragged CR per head (1..16), 75 steps: crosses pages and
    split tiles; all outputs and the exported caches."""
    log(f"case variants dtype={dtype} d={d} G={G} page={page} tile={tile} omega={omega} c={bias}")
    B, Hkv, L, steps = 3, 3, 2, 75
    rng = np.random.default_rng(100 + d + G + page + tile)
    pr = Pair(L, B, Hkv * G, Hkv, d, dtype, page_size=page, max_slots=steps, bias=bias,
              omega_src=omega, split_tile=tile)
    crs = [np.array([1.0, 3.0, 16.0]), np.array([2.0, 1.0, 1.5])]
    for step in range(steps):
        for layer in range(L):
            q, k, v = random_step(rng, B, Hkv * G, Hkv, d, crs[layer], dtype, "cuda", bias)
            pr.decode(layer, q, k, v)
    for layer in range(L):
        pr.compare_cache(layer)
    pr.ok()


def test_all_accumulate_single_slot(torch_cuda):
    """Every token after the first accumulates: one slot per unit, output =
    omega-weighted mean of the values (checked against the oracle)."""
    log("case all-accumulate")
    rng = np.random.default_rng(7)
    pr = Pair(1, 2, 4, 2, 128, "fp32", max_slots=4, split_tile=8)
    for step in range(60):
        q, k, v = random_step(rng, 2, 4, 2, 128, np.array([1e9, 1e9]), "fp32", "cuda")
        k[:, :, 0] = 3.0 + step
        pr.decode(0, q, k, v)
    assert (pr.gpu.lengths(0).cpu().numpy() == 1).all()
    pr.compare_cache(0)
    pr.ok()


def test_split_tile_independence(torch_cuda):
    """The same inputs with tiny split tiles and with one tile per unit give
    the same slot indices and outputs within fp32 rounding; repeated runs
    are bitwise identical (no race between the update and the readers)."""
    import torch
    log("case split-tile independence")
    outs = {}
    for tile in (8, 1000, 8):
        rng = np.random.default_rng(42)
        pr = Pair(1, 2, 2, 2, 128, "fp32", max_slots=300, split_tile=tile)
        res = []
        for step in range(300):
            q, k, v = random_step(rng, 2, 2, 2, 128, np.array([1.0, 4.0]), "fp32", "cuda")
            out = torch.empty_like(q)
            pr.gpu.decode_step(0, q, k, v, out=out)
            res.append(out.cpu())
        pr.ok()
        outs.setdefault(tile, []).append(torch.stack(res))
    a, b = outs[8]
    assert torch.equal(a, b), "two identical runs differ"
    assert torch.allclose(a, outs[1000][0], atol=2e-6, rtol=2e-6)


@pytest.mark.parametrize("dtype,d,G", [("bf16", 128, 1), ("fp32", 64, 2), ("bf16", 128, 8)])
def test_prefill_then_decode(torch_cuda, dtype, d, G):
    """Prefill with ragged prompt lengths (0, 1, 31, 32, 33, 64, 65, n) and
    per-head CR, then decode: slot indices, lengths, slots, z, outputs."""
    import torch
    log(f"case prefill dtype={dtype} d={d} G={G}")
    n, Hkv = 200, 2
    lens = [0, 1, 31, 32, 33, 64, 65, n]
    B = len(lens)
    rng = np.random.default_rng(11 + d + G)
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, max_slots=n + 40, max_prompt_len=n, split_tile=64)
    k = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    v = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    q0 = rng.standard_normal((B, n, Hkv * G), dtype=np.float32)
    k[..., 0] = decision_logits(rng.uniform(size=(B, n, Hkv)), np.array([3.0, 100.0])[None, None])
    dt = torch.float32 if dtype == "fp32" else torch.bfloat16
    kt, vt, qt = (torch.from_numpy(x).to(dt).cuda() for x in (k, v, q0))
    pr.prefill(0, kt, vt, qt, prompt_lens=lens)
    pr.compare_cache(0)
    for step in range(40):
        q, kk, vv = random_step(rng, B, Hkv * G, Hkv, d, np.array([3.0, 100.0]), dtype, "cuda")
        pr.decode(0, q, kk, vv)
    pr.compare_cache(0)
    pr.ok()


def test_prefill_strided_full_q(torch_cuda):
    """Prefill reads k, v through arbitrary (B, n, H) strides and q from a
    full [B, n, Hq, d] tensor; a prompt that never appends after token 0
    forms one segment spanning many 64-token chunks."""
    import torch
    log("case prefill strided")
    B, n, Hkv, G, d = 2, 300, 2, 2, 128
    rng = np.random.default_rng(5)
    pr = Pair(1, B, Hkv * G, Hkv, d, "bf16", max_slots=n + 8)
    big = torch.randn((B, Hkv, n, d), generator=torch.Generator().manual_seed(1)).to(torch.bfloat16)
    big[..., 0] = torch.from_numpy(decision_logits(rng.uniform(size=(B, Hkv, n)),
                                                   np.array([1e9, 2.0])[None, :, None])
                                   ).to(torch.bfloat16)
    k = big.cuda().permute(0, 2, 1, 3)                   # [B, n, Hkv, d], non-contiguous
    v = torch.randn((n, B, Hkv, d)).to(torch.bfloat16).cuda().permute(1, 0, 2, 3)
    q = torch.randn((B, n, Hkv * G, d)).to(torch.bfloat16).cuda()
    slot = torch.empty((B, Hkv, n), dtype=torch.int32, device="cuda")
    pr.gpu.prefill(0, k, v, q, slot_index=slot)
    s_ref = pr.orc.prefill(0, f64(k), f64(v), f64(q[..., 0]))
    assert (slot.cpu().numpy() == s_ref).all()
    assert pr.gpu.lengths(0).cpu().numpy()[:, 0].tolist() == [1, 1]
    pr.compare_cache(0)
    pr.ok()


def test_empty_prompt_then_decode(torch_cuda):
    import torch
    log("case empty prompt")
    pr = Pair(1, 2, 2, 2, 64, "bf16", max_slots=40)
    z = torch.empty((2, 0, 2, 64), dtype=torch.bfloat16, device="cuda")
    pr.gpu.prefill(0, z, z, torch.empty((2, 0, 2), dtype=torch.bfloat16, device="cuda"), n=0)
    assert (pr.gpu.lengths(0).cpu().numpy() == 0).all()
    rng = np.random.default_rng(3)
    for _ in range(40):
        pr.decode(0, *random_step(rng, 2, 2, 2, 64, np.array([2.0, 5.0]), "bf16", "cuda"))
    pr.compare_cache(0)
    pr.ok()


@pytest.mark.parametrize("G,d", [(1, 128), (4, 128), (8, 64)])
def test_import_export_roundtrip(torch_cuda, G, d):
    """Importing a dense cache and exporting it is the identity on the
    valid slots (bit-exact) and zero elsewhere; then decode on top of it.
    G >= 4 exercises the transposed value pages of matrix-core caches."""
    import torch
    log(f"case import/export G={G} d={d}")
    B, Hkv, dense = 3, 2, 70
    lens = np.array([[0, 1], [31, 32], [33, 70]], dtype=np.int32)
    pr = Pair(1, B, Hkv * G, Hkv, d, "bf16", max_slots=80, split_tile=32)
    K = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    V = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    z = torch.rand((B, Hkv)).cuda() * 3 + 0.1
    lt = torch.from_numpy(lens).cuda()
    pr.gpu.import_(0, K, V, lt, z)
    pr.orc.load(0, f64(K), f64(V), lens, f64(z))
    K2, V2, z2 = pr.gpu.export(0, dense_slots=dense)
    mask = torch.arange(dense, device="cuda")[None, None, :] < lt[:, :, None]
    assert torch.equal(K2[mask], K[mask]) and torch.equal(V2[mask], V[mask])
    assert (K2[~mask] == 0).all() and (V2[~mask] == 0).all()
    assert torch.equal(z2[lt > 0], z[lt > 0])
    rng = np.random.default_rng(9)
    for _ in range(10):
        pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.array([1.5, 3.0]), "bf16", "cuda"))
    pr.compare_cache(0)
    pr.ok()


@pytest.mark.parametrize("G", [1, 8])
def test_decode_many_pieces_per_unit(torch_cuda, G):
    """About 100 slots per wave of the full decode grid (512 units of 260-560
    slots), so most units are cut into four or five pieces whose partial
    records the combine merges.  Every unit's output, slot index, length and
    slots are checked over several steps.  G = 1 runs the vector-ALU kernel,
    G = 8 the matrix-core kernel."""
    import torch
    B, Hkv, d = (16, 32, 64) if G == 1 else (64, 8, 64)
    log(f"case many pieces per unit G={G} units={B * Hkv}")
    rng = np.random.default_rng(77 + G)
    lens = rng.integers(260, 560, size=(B, Hkv)).astype(np.int32)
    lens[0, 0], lens[-1, -1] = 1, 0                     # a one-slot and an empty unit
    dense, steps = int(lens.max()), 4
    pr = Pair(1, B, Hkv * G, Hkv, d, "bf16", max_slots=dense + steps)
    K = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    V = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    K[..., 0] = 0                                        # stored keys have element 0 cleared
    z = torch.rand((B, Hkv)).cuda() * 3 + 0.1
    pr.gpu.import_(0, K, V, torch.from_numpy(lens).cuda(), z)
    pr.orc.load(0, f64(K), f64(V), lens, f64(z))
    cr = rng.choice([1.0, 2.0, 4.0], size=Hkv)
    for _ in range(steps):
        pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, cr, "bf16", "cuda"))
    pr.compare_cache(0)
    pr.ok()


def test_pool_exhaustion_sets_flag(torch_cuda):
    """A pool too small for the appends: the device flag reports
    DMC_ERR_CAPACITY, every page is used, nothing is written out of bounds
    (the page pool is the last thing the export can see)."""
    import paper_2403_09636_amd as P
    log("case pool exhaustion")
    rng = np.random.default_rng(1)
    pr = Pair(1, 2, 2, 2, 64, "bf16", page_size=8, max_slots=64, num_pages=5)
    for _ in range(24):
        q, k, v = random_step(rng, 2, 2, 2, 64, np.array([1.0, 1.0]), "bf16", "cuda")
        pr.gpu.decode_step(0, q, k, v)
    assert pr.gpu.status() == P.binding.DMC_ERR_CAPACITY
    assert pr.gpu.pages_used() == 5
    lens = pr.gpu.lengths(0).cpu().numpy()
    assert lens.sum() <= 5 * 8 and lens.max() <= 24
    pr.gpu.reset()
    assert pr.gpu.status() == 0 and pr.gpu.pages_used() == 0


def test_slot_capacity_sets_flag(torch_cuda):
    import paper_2403_09636_amd as P
    log("case slot capacity")
    rng = np.random.default_rng(2)
    pr = Pair(1, 1, 1, 1, 128, "fp32", max_slots=10)
    for _ in range(12):
        pr.gpu.decode_step(0, *random_step(rng, 1, 1, 1, 128, np.array([1.0]), "fp32", "cuda"))
    assert pr.gpu.status() == P.binding.DMC_ERR_CAPACITY
    assert pr.gpu.lengths(0).cpu().numpy()[0, 0] == 10


def test_bad_import_length_sets_flag(torch_cuda):
    import torch
    import paper_2403_09636_amd as P
    log("case bad import length")
    pr = Pair(1, 1, 2, 2, 64, "bf16", max_slots=16)
    K = torch.zeros((1, 2, 8, 64), dtype=torch.bfloat16, device="cuda")
    pr.gpu.import_(0, K, K, torch.tensor([[3, 9]], dtype=torch.int32, device="cuda"),
                   torch.ones((1, 2), device="cuda"))
    assert pr.gpu.status() == P.binding.DMC_ERR_INVALID_ARG
    assert pr.gpu.lengths(0).cpu().numpy().tolist() == [[3, 0]]


def test_prompt_token_stride_bound(torch_cuda):
    """Up to 64 consecutive prompt tokens are addressed from one base with
    32-bit offsets: a k or v token stride of 32 MiB or more is refused before
    anything is enqueued, one just below is accepted."""
    import torch
    import paper_2403_09636_amd as P
    log("case prompt token stride bound")
    pr = Pair(1, 1, 1, 1, 64, "bf16", max_slots=8, num_pages=8, max_prompt_len=2)
    big = 1 << 24                      # elements: 32 MiB of bf16
    buf = torch.zeros(big + 64, dtype=torch.bfloat16, device="cuda")
    q = torch.zeros((1, 2, 1, 64), dtype=torch.bfloat16, device="cuda")
    for stride, ok in ((big, False), (big - 64, True)):
        k = torch.as_strided(buf, (1, 2, 1, 64), (2 * big, stride, 64, 1))
        v = torch.zeros((1, 2, 1, 64), dtype=torch.bfloat16, device="cuda")
        for kk, vv in ((k, v), (v, k)):
            if ok:
                pr.gpu.prefill(0, kk, vv, q)
            else:
                with pytest.raises(P.DMCError) as e:
                    pr.gpu.prefill(0, kk, vv, q)
                assert e.value.status == P.binding.DMC_ERR_UNSUPPORTED
    pr.ok()
    assert pr.gpu.lengths(0).cpu().numpy().tolist() == [[2]]   # k[0] = 0: both tokens append


@pytest.mark.parametrize("d,jitter", [(128, 4), (128, 0), (64, 3)])
def test_whole_unit_partition(torch_cuda, d, jitter):
    """The matrix-core decode gives every wave whole units when unit lengths are
    near-uniform (here 2048 units of 100 +- jitter slots: two per wave at d = 128,
    one at d = 64), so no unit is split and every output is written by its owner
    directly.  Every unit's output, slot index, length, slots and z against the
    oracle over three steps, with appends crossing page boundaries."""
    import torch
    log(f"case whole-unit partition d={d} jitter={jitter}")
    B, Hkv, G, steps = 256, 8, 8, 3
    rng = np.random.default_rng(91 + d + jitter)
    lens = (100 + rng.integers(-jitter, jitter + 1, size=(B, Hkv))).astype(np.int32)
    dense = int(lens.max())
    pr = Pair(1, B, Hkv * G, Hkv, d, "bf16", max_slots=dense + steps)
    K = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    V = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    K[..., 0] = 0
    z = torch.rand((B, Hkv)).cuda() * 3 + 0.1
    pr.gpu.import_(0, K, V, torch.from_numpy(lens).cuda(), z)
    pr.orc.load(0, f64(K), f64(V), lens, f64(z))
    err = 0.0
    for _ in range(steps):
        err = max(err, pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.full(Hkv, 2.0), "bf16",
                                                 "cuda")))
    pr.compare_cache(0)
    pr.ok()
    log(f"  max abs err {err:.3e}")


def test_largest_matrix_core_unit_table(torch_cuda):
    """Grouped-query bf16 caches decode on matrix cores with a 128 KB chunk ring
    in LDS at d = 128; the largest slot-space table of one entry per unit
    (8175 units; here 8168) fills the rest of the compute unit's LDS.  Imported
    caches of 40-70 slots (two or three pages per unit), three steps, every
    unit against the oracle."""
    import torch
    log("case largest matrix-core unit table")
    B, Hkv, G, d, steps = 1021, 8, 8, 128, 3
    rng = np.random.default_rng(78)
    lens = rng.integers(40, 71, size=(B, Hkv)).astype(np.int32)
    dense = int(lens.max())
    pr = Pair(1, B, Hkv * G, Hkv, d, "bf16", max_slots=dense + steps)
    K = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    V = torch.randn((B, Hkv, dense, d)).to(torch.bfloat16).cuda()
    K[..., 0] = 0
    z = torch.rand((B, Hkv)).cuda() * 3 + 0.1
    pr.gpu.import_(0, K, V, torch.from_numpy(lens).cuda(), z)
    pr.orc.load(0, f64(K), f64(V), lens, f64(z))
    for _ in range(steps):
        pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.full(Hkv, 2.0), "bf16", "cuda"))
    pr.compare_cache(0)
    pr.ok()


def test_largest_unit_table(torch_cuda):
    """batch * kv heads near the decode kernel's LDS slot-table limit (64 KB):
    16000 units of one query head each, a few steps from empty, against the
    oracle on a sample of units (slot indices of all units bit-exact)."""
    import torch
    import oracle
    import paper_2403_09636_amd as P
    log("case largest unit table")
    B, H, d, steps = 1000, 16, 64, 3
    cfg = P.make_config(1, B, H, H, d, "bf16", 32, 8)
    cache = P.DMCCache(cfg, device="cuda")
    orc = oracle.DMCOracle(1, B, H, H, d, 8)
    rng = np.random.default_rng(77)
    for _ in range(steps):
        q, k, v = random_step(rng, B, H, H, d, np.full(H, 2.0), "bf16", "cuda")
        si = torch.empty((B, H), dtype=torch.int32, device="cuda")
        out = cache.decode_step(0, q, k, v, slot_index=si)
        ref, ref_si = orc.decode_step(0, f64(q), f64(k), f64(v))
        assert (si.cpu().numpy() == ref_si).all()
        err = np.abs(f64(out) - ref)
        assert (err <= 2e-2 + 1e-2 * np.abs(ref)).all(), err.max()
    cache.check()
