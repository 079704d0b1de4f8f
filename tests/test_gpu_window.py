"""Window grouping (Sec. 3.3) on the GPU against the float64 oracle: every
step's partial accumulation over the last w tokens of the open segment, so
a slot is the omega-weighted mean of its segment's last min(w, length)
tokens.  Decode from an empty cache, prompt compaction, prompt attention and
decode after both, through the C ABI."""
import numpy as np
import pytest

from tests.gpu_helpers import Pair, log, random_step
from workloads import decision_logits

pytestmark = pytest.mark.gpu

# per-head compression: always append, moderate, longer than a 12-token
# window, and a single segment for the whole run
CRS = [1.0, 4.0, 20.0, 1e9]


def _prompt(rng, B, n, Hkv, G, d, crs, dtype):
    import torch
    k = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    v = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    q = rng.standard_normal((B, n, Hkv * G, d), dtype=np.float32)
    k[..., 0] = decision_logits(rng.uniform(size=(B, n, Hkv)), np.asarray(crs)[None, None])
    dt = torch.float32 if dtype == "fp32" else torch.bfloat16
    return tuple(torch.from_numpy(x).to(dt).cuda() for x in (k, v, q))


@pytest.mark.parametrize("dtype,d,G,w,split", [
    ("fp32", 64, 1, 1, 0), ("fp32", 128, 2, 3, 7), ("bf16", 128, 1, 12, 0), ("bf16", 128, 1, 12, 9),
    ("bf16", 64, 2, 5, 0), ("bf16", 128, 8, 12, 0), ("bf16", 128, 4, 64, 13), ("bf16", 64, 8, 2, 0),
])
def test_window_decode_from_empty(torch_cuda, dtype, d, G, w, split):
    """Decode steps from an empty cache; the windows of the long segments
    slide many times; forced split ranges cut units into several pieces."""
    log(f"case window decode dtype={dtype} d={d} G={G} w={w} split={split}")
    B, Hkv, steps = 2, 4, 90
    rng = np.random.default_rng(500 + d + G + w + split)
    page = 32 if G >= 4 else 16   # bf16 G >= 4 with 32-slot pages decodes on matrix cores
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, page_size=page, max_slots=steps + 8, split_tile=split,
              window=w)
    err = 0.0
    for _ in range(steps):
        err = max(err, pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.array(CRS), dtype,
                                                 "cuda")))
    pr.compare_cache(0)
    pr.ok()
    log(f"  lengths {pr.gpu.lengths(0).cpu().numpy().tolist()}, max abs err {err:.3e}")


@pytest.mark.parametrize("dtype,d,G,w,page", [
    ("bf16", 128, 1, 12, 32), ("bf16", 128, 8, 12, 32), ("bf16", 64, 4, 7, 16),
    ("fp32", 128, 1, 12, 32), ("fp32", 64, 2, 1, 8), ("bf16", 128, 2, 64, 64),
])
def test_window_prefill_then_decode(torch_cuda, dtype, d, G, w, page):
    """Prompt compaction with ragged lengths (0, 1, across 64-token chunks),
    then decode continuing each unit's window from the prompt's tail."""
    log(f"case window prefill dtype={dtype} d={d} G={G} w={w} page={page}")
    B, Hkv, n = 5, 4, 230
    lens = [n, 0, 1, 65, 140]
    rng = np.random.default_rng(600 + d + G + w + page)
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, page_size=page, max_slots=n + 40, max_prompt_len=n,
              window=w)
    k, v, q = _prompt(rng, B, n, Hkv, G, d, CRS, dtype)
    pr.prefill(0, k, v, q[..., 0].contiguous(), prompt_lens=lens)
    pr.compare_cache(0)
    err = 0.0
    for _ in range(30):
        err = max(err, pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.array(CRS), dtype,
                                                 "cuda")))
    pr.compare_cache(0)
    pr.ok()
    log(f"  max abs err {err:.3e}")


@pytest.mark.parametrize("dtype,G,w", [("bf16", 4, 64), ("bf16", 8, 1), ("fp32", 1, 5)])
def test_window_prefill_long_segments(torch_cuda, dtype, G, w):
    """An 8300-token prompt whose segments run to hundreds of tokens: one
    compaction work item then covers more than 64 start-mask words (4096
    tokens), and most of its rows lie outside every window and are not read.
    One unit keeps a single segment, so the open segment's token ring is
    filled from the prompt's last tokens."""
    log(f"case window prefill long segments dtype={dtype} G={G} w={w}")
    B, Hkv, d, n = 1, 2, 128, 8300
    crs = [150.0, 1e9]
    rng = np.random.default_rng(900 + G + w)
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, page_size=32, max_slots=n + 16, max_prompt_len=n,
              window=w)
    k, v, q = _prompt(rng, B, n, Hkv, G, d, crs, dtype)
    pr.prefill(0, k, v, q[..., 0].contiguous())
    pr.compare_cache(0)
    err = 0.0
    for _ in range(6):
        err = max(err, pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.array(crs), dtype,
                                                 "cuda")))
    pr.compare_cache(0)
    pr.ok()
    log(f"  lengths {pr.gpu.lengths(0).cpu().numpy().tolist()}, max abs err {err:.3e}")


@pytest.mark.parametrize("dtype,d,G,w,page", [
    ("bf16", 128, 1, 12, 32), ("bf16", 128, 2, 12, 32), ("bf16", 128, 4, 12, 32),
    ("bf16", 128, 8, 12, 32), ("bf16", 64, 1, 3, 16), ("bf16", 128, 1, 40, 8),
    ("fp32", 128, 1, 12, 32), ("fp32", 64, 4, 5, 16), ("fp32", 64, 8, 1, 32),
])
def test_window_prompt_attend(torch_cuda, dtype, d, G, w, page):
    """Prompt attention with windowed open states (each query sees the
    closed segments' windowed means and the mean of its own segment's last
    min(w, .) tokens), ragged lengths, then decode."""
    log(f"case window prompt dtype={dtype} d={d} G={G} w={w} page={page}")
    B, Hkv, n = 6, 4, 200
    lens = [0, 1, 33, 64, 129, n]
    rng = np.random.default_rng(700 + d + 10 * G + w + page)
    pr = Pair(1, B, Hkv * G, Hkv, d, dtype, page_size=page, max_slots=n + 24, max_prompt_len=n,
              window=w)
    k, v, q = _prompt(rng, B, n, Hkv, G, d, CRS, dtype)
    err = pr.prefill_attend(0, k, v, q, prompt_lens=lens)
    pr.compare_cache(0)
    for _ in range(12):
        err = max(err, pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.array(CRS), dtype,
                                                 "cuda")))
    pr.compare_cache(0)
    pr.ok()
    log(f"  max abs err {err:.3e}")


def test_window_wide_equals_exact(torch_cuda):
    """A window longer than any segment gives the exact Algorithm 1 cache:
    the windowed GPU path matches the unwindowed oracle."""
    import oracle
    log("case window wider than every segment")
    B, Hkv, G, d, n = 2, 2, 2, 128, 60
    rng = np.random.default_rng(811)
    pr = Pair(1, B, Hkv * G, Hkv, d, "fp32", max_slots=n + 20, max_prompt_len=n, window=64)
    pr.orc = oracle.DMCOracle(1, B, Hkv * G, Hkv, d, n + 20)   # exact, no window
    k, v, q = _prompt(rng, B, n, Hkv, G, d, [3.0, 1e9], "fp32")
    pr.prefill_attend(0, k, v, q)
    for _ in range(3):
        pr.decode(0, *random_step(rng, B, Hkv * G, Hkv, d, np.array([3.0, 1e9]), "fp32", "cuda"))
    pr.compare_cache(0)
    pr.ok()


def test_window_import_unsupported(torch_cuda):
    """A windowed cache cannot be imported from slots (its raw tokens are
    unknown): the call fails before any launch."""
    import torch
    import paper_2403_09636_amd as P
    log("case window import refused")
    cfg = P.make_config(1, 1, 2, 2, 64, max_slots_per_seq=64, window=12)
    cache = P.DMCCache(cfg)
    K = torch.zeros((1, 2, 8, 64), dtype=torch.bfloat16, device="cuda")
    lens = torch.full((1, 2), 4, dtype=torch.int32, device="cuda")
    z = torch.ones((1, 2), dtype=torch.float32, device="cuda")
    with pytest.raises(P.DMCError) as e:
        cache.import_(0, K, K.clone(), lens, z)
    assert e.value.status == P.binding.DMC_ERR_UNSUPPORTED
    cache.check()


def test_window_prompt_sampled_7b_layer(torch_cuda):
    """Llama-2-7B layer shape (B=2, n=4096, 32 heads, d=128, CR per head in
    {1, 2, 4, 8}) with w = 12, in the bench's launch configuration: every
    output row of 4 sampled units against a per-unit windowed oracle, then 4
    decode steps with those units' outputs checked."""
    import torch
    import oracle
    import paper_2403_09636_amd as P
    import workloads as W
    from tests.gpu_helpers import assert_close, f64
    log("case window prompt 7b layer sampled")
    w = W.scaled(W.WORKLOADS["llama7b_layer"], batch=2)
    k, v, q = W.prompt_full_torch(w, 0, "cuda")
    n = w.prompt_len
    cfg = P.make_config(1, w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype,
                        w.page_size, n + 8, max_prompt_len=n, window=12)
    cache = P.DMCCache(cfg, device="cuda")
    out = cache.prefill_attend(0, k, v, q)
    steps = [W.decode_inputs_torch(w, s, 0, "cuda") for s in range(4)]
    outs = [cache.decode_step(0, *x) for x in steps]
    torch.cuda.synchronize()
    cache.check()
    units = [(0, 0), (1, 31), (0, 17), (1, 6)]
    for b, g in units:
        orc = oracle.DMCOracle(1, 1, 1, 1, w.head_dim, max_slots=n + 8, window=12)
        o_ref, _ = orc.prefill_attend(0, f64(q[b:b + 1, :, g:g + 1]), f64(k[b:b + 1, :, g:g + 1]),
                                      f64(v[b:b + 1, :, g:g + 1]))
        err = assert_close(f64(out[b, :, g]), o_ref[0, :, 0], "bf16", f"prompt unit {(b, g)}")
        for (qs, ks, vs), o in zip(steps, outs):
            o_ref, _ = orc.decode_step(0, f64(qs[b:b + 1, g:g + 1]), f64(ks[b:b + 1, g:g + 1]),
                                       f64(vs[b:b + 1, g:g + 1]))
            err = max(err, assert_close(f64(o[b, g]), o_ref[0, 0], "bf16", f"decode unit {(b, g)}"))
        log(f"  unit {(b, g)} max abs err {err:.3e}")
