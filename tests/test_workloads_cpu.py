"""The seeded input recipes and the benchmark's byte accounting (CPU)."""
import math

import numpy as np
import pytest

import workloads as W


def test_decision_logits_append_rate():
    """k[0] = Logistic + log(CR - 1) appends (k[0] <= 0) with probability 1/CR."""
    u = np.random.default_rng(0).uniform(size=400_000)
    for cr in (1.0, 1.5, 2.0, 4.0, 8.0, 16.0, 32.0):
        rate = float((W.decision_logits(u, cr) <= 0).mean())
        assert abs(rate - 1.0 / cr) < 4 * math.sqrt((1 / cr) * (1 - 1 / cr) / u.size) + 1e-12, cr
    # the bias shifts the threshold: compare against c instead of 0
    assert ((W.decision_logits(u, 4.0, bias=2.5) <= 2.5).mean() - 0.25) < 0.01


def test_llama7b_stack_calibrated_to_global_4x():
    w = W.WORKLOADS["llama7b_stack"]
    lens = W.precompressed_lengths(w)
    assert lens.shape == (32, 32)
    assert lens.sum() * 4 == lens.size * w.prompt_len            # global CR exactly 4
    assert lens.min() >= w.prompt_len // 16 and lens.max() <= w.prompt_len
    crs = w.prompt_len / lens
    assert 1.0 <= crs.min() and crs.max() <= 16.0
    assert np.allclose(W.effective_crs(w), crs)


def test_llama13b_skew_shape():
    w = W.WORKLOADS["llama13b_skew"]
    crs = W.head_crs(w)
    assert np.isclose((crs == 1.0).mean(), 0.1)
    rest = crs[crs != 1.0]
    assert rest.min() >= 16.0 and rest.max() <= 32.0
    lens = W.precompressed_lengths(w)
    global_cr = lens.size * w.prompt_len / lens.sum()
    assert 6.5 < global_cr < 8.0


def test_prompt_recipe_statistics():
    w = W.scaled(W.WORKLOADS["llama7b_layer"], batch=2, prompt_len=2048)
    k, v, q0 = W.prompt_np(w, 0)
    assert k.shape == (2, 2048, 32, 128) and q0.shape == (2, 2048, 32)
    crs = W.head_crs(w)[0]
    app = (k[..., 0].float().numpy() <= 0).mean(axis=(0, 1))
    assert np.allclose(app, 1.0 / crs, atol=0.05)
    vv = v.float().numpy()
    assert abs(vv.mean()) < 0.01 and abs(vv.std() - 1.0) < 0.01


def test_seeds_are_distinct_and_stable():
    w = W.WORKLOADS["tiny"]
    a = W.decode_inputs_np(w, 3, 0)[0]
    b = W.decode_inputs_np(w, 3, 0)[0]
    c = W.decode_inputs_np(w, 4, 0)[0]
    assert (a == b).all() and not (a == c).all()
    assert len({W.seed_for(w, s, l) for s in range(50) for l in range(80)}) == 4000


def test_pool_pages_cover_prefill_lengths():
    """The pool sized for a prefilled cache holds the realised lengths."""
    w = W.scaled(W.WORKLOADS["llama70b_gqa"], num_layers=1, batch=4)
    rng = np.random.default_rng(1)
    crs = W.head_crs(w)[0]
    n = w.prompt_len
    need = 0
    for _ in range(4):
        app = rng.uniform(size=(w.batch, n, w.num_kv_heads)) < 1.0 / crs
        app[:, 0] = True
        lens = app.sum(axis=1) + w.decode_steps
        need = max(need, int(np.ceil(lens / w.page_size).sum()))
    assert need <= W.pool_pages(w, w.decode_steps)


def test_sample_units_include_extremes():
    w = W.WORKLOADS["llama7b_stack"]
    units = W.sample_units(w, 64)
    lens = W.precompressed_lengths(w)[0]
    assert (0, 0, int(np.argmax(lens))) in units and (0, 0, int(np.argmin(lens))) in units
    assert len(set(units)) == len(units) >= 64


def test_algorithmic_bytes_formula():
    import bench
    w = W.scaled(W.WORKLOADS["llama70b_gqa"], batch=1, num_kv_heads=2, num_q_heads=16)
    before = np.array([[0, 31]])
    after = np.array([[1, 32]])
    d, s, G, P = w.head_dim, w.elem_bytes, w.group, w.page_size
    per_unit = [2 * d * s * lb + 2 * d * s + (2 * G + 2) * d * s + 16 + 4 * -(-la // P)
                for lb, la in zip(before[0], after[0])]
    assert bench.algorithmic_bytes(before, after, w, P) == sum(per_unit)


@pytest.mark.parametrize("n", [1, 3])
def test_bench_refuses_more_than_one_gpu(n):
    import subprocess
    import sys
    res = subprocess.run([sys.executable, "bench.py", "--gpus", str(n + 1)], capture_output=True,
                         text=True, cwd=__import__("os").path.dirname(__import__("os").path.dirname(
                             __import__("os").path.abspath(__file__))))
    assert res.returncode == 2 and "one GPU" in res.stderr


def test_bench_window_bookkeeping():
    """The benchmark's host-side window accounting (open-segment lengths
    after a prompt, prompt tokens a windowed compaction reads) against a
    per-unit loop over the segments."""
    import bench
    rng = np.random.default_rng(0)
    for _ in range(20):
        B, n, H = 2, 50, 3
        k0 = rng.standard_normal((B, n, H)) + rng.uniform(-1, 2)
        w = int(rng.integers(1, 15))
        ref_sl = np.zeros((B, H), int)
        ref_reads = 0
        for b in range(B):
            for h in range(H):
                starts = [0] + [t for t in range(1, n) if not k0[b, t, h] > 0]
                ends = starts[1:] + [n]
                ref_sl[b, h] = ends[-1] - starts[-1]
                ref_reads += sum(min(w, e - s) for s, e in zip(starts, ends))
        assert (bench.segment_lengths_after_prompt(k0, n) == ref_sl).all()
        assert bench.windowed_prompt_reads(k0, w) == ref_reads


def test_cpu_baseline_worker_counts_unit_steps():
    """The oracle-timing worker runs whole units (four decode steps each) on
    the workload's lengths and reports the time spent inside the steps."""
    import bench
    w = W.scaled(W.WORKLOADS["llama7b_stack"], num_layers=2, num_kv_heads=2, num_q_heads=2)
    lens = np.full((2, 2), 40)
    steps, spent, units = bench._oracle_unit_steps((3, 0.05, 2, 2, w.head_dim, w.group, lens,
                                                    w.prompt_len))
    assert units >= 1 and steps == 4 * units and spent > 0
