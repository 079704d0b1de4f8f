"""Seeded synthetic inputs for the DMC decode path.

This module produces *inputs* only: activations, decision logits and
pre-compressed caches with the shapes and statistics of the paper's Llama 2
throughput workloads (Sec. 5.2: 2K-token prompts, bf16, largest batch that
fits; Fig. "cr_heatmap": compression ratios differ per layer and head).  It
holds none of the method's arithmetic.  Both the HIP path and the oracle
consume the tensors it returns; the oracle receives them widened to float64.

Decision logits: the paper's training relaxation draws
alpha ~ Gumbel-sigmoid(k[0] - c, tau) (Sec. 3.2); the difference of two
Gumbel variables is logistic, so k[0] = Logistic(0, 1) + log(CR - 1) makes
the rounded decision append with probability exactly 1 / CR, i.i.d. over
time (the paper finds alpha flat over positions, appendix "Compression
analysis").  CR = 1 uses k[0] = -(1 + |Logistic|) (always append).
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field

import numpy as np

# ----------------------------------------------------------------------------
# Workload shapes
# ----------------------------------------------------------------------------


@dataclass(frozen=True)
class Workload:
    name: str
    index: int                 # seed namespace
    num_layers: int
    batch: int
    num_q_heads: int
    num_kv_heads: int
    head_dim: int
    dtype: str                 # "fp32" | "bf16"
    prompt_len: int            # context length (prefilled or pre-compressed)
    decode_steps: int
    cache_kind: str            # "empty" | "prefill" | "precompressed"
    cr_kind: str               # per-(layer, kv-head) CR recipe
    page_size: int = 32
    notes: str = field(default="", compare=False)

    @property
    def group(self):
        return self.num_q_heads // self.num_kv_heads

    @property
    def units_per_layer(self):
        return self.batch * self.num_kv_heads

    @property
    def max_slots(self):
        return self.prompt_len + self.decode_steps

    @property
    def elem_bytes(self):
        return 4 if self.dtype == "fp32" else 2


WORKLOADS = {
    "tiny": Workload("tiny", 1, 1, 1, 4, 4, 64, "fp32", 0, 256, "empty", "tiny_1248",
                     notes="1 layer, batch 1, 4 heads, d64, fp32, empty prompt, "
                           "256 decode steps, CR per head (1, 2, 4, 8)"),
    "llama7b_layer": Workload("llama7b_layer", 2, 1, 16, 32, 32, 128, "bf16", 4096, 128,
                              "prefill", "uniform_1248",
                              notes="one Llama-2-7B attention layer, batch 16, 4096-token "
                                    "prompt compressed by prefill at CR drawn from "
                                    "{1,2,4,8} per head, then 128 decode steps"),
    "llama7b_stack": Workload("llama7b_stack", 3, 32, 64, 32, 32, 128, "bf16", 4096, 64,
                              "precompressed", "loguniform_1_16_global4",
                              notes="Llama-2-7B decode stack, 32 layers x 32 heads, batch "
                                    "64, 4096-token context pre-compressed at global 4x "
                                    "(per layer/head CR log-uniform in [1, 16], "
                                    "calibrated), 64 decode steps"),
    "llama13b_skew": Workload("llama13b_skew", 4, 40, 128, 40, 40, 128, "bf16", 8192, 32,
                              "precompressed", "skew_10pct_cr1_rest_16_32",
                              notes="Llama-2-13B shape, batch 128, 8192 context, 10% of "
                                    "heads at CR 1 and the rest log-uniform in [16, 32]"),
    "llama70b_gqa": Workload("llama70b_gqa", 5, 80, 256, 64, 8, 128, "bf16", 4096, 64,
                             "prefill", "const_2",
                             notes="Llama-2-70B GQA shape, 64 query / 8 kv heads, batch "
                                   "256, 4096-token prompts compressed by prefill at CR 2 "
                                   "per kv head, 64 decode steps"),
    "llama7b_train": Workload("llama7b_train", 6, 1, 4, 32, 32, 128, "bf16", 4096, 0, "train",
                              "uniform_1248",
                              notes="one Llama-2-7B attention layer in continued pre-training: "
                                    "4 sequences of 4096 tokens (the paper's sequence length), "
                                    "c = 5, tau = 0.1, w = 12, per-head target CR from "
                                    "{1,2,4,8}"),
}

# Training hyperparameters of the paper (Sec. 4): Gumbel-sigmoid constant c,
# temperature tau and window w.
TRAIN_C, TRAIN_TAU, TRAIN_WINDOW = 5.0, 0.1, 12


def scaled(w: Workload, **kw) -> Workload:
    """A copy of a workload with some fields replaced (smaller test cases)."""
    d = dict(w.__dict__)
    d.update(kw)
    return Workload(**d)


# ----------------------------------------------------------------------------
# Seeds
# ----------------------------------------------------------------------------

PROMPT_STREAM = 0


def seed_for(w: Workload, stream: int, layer: int) -> int:
    """Seed of one (stream, layer) pair: stream 0 is the prompt or cache,
    stream 1 + s the inputs of decode step s."""
    return ((1000 * w.index + stream) * 1000 + layer) & 0x7FFFFFFFFFFF


def np_rng(w: Workload, stream: int, layer: int) -> np.random.Generator:
    return np.random.Generator(np.random.PCG64(seed_for(w, stream, layer)))


# ----------------------------------------------------------------------------
# Per-(layer, kv-head) compression ratios
# ----------------------------------------------------------------------------

def head_crs(w: Workload) -> np.ndarray:
    """[L, Hkv] target compression ratio of every (layer, kv head)."""
    rng = np.random.Generator(np.random.PCG64(1000 * w.index + 999))
    L, H = w.num_layers, w.num_kv_heads
    if w.cr_kind == "tiny_1248":
        return np.tile(np.array([1.0, 2.0, 4.0, 8.0])[:H], (L, 1))
    if w.cr_kind == "uniform_1248":
        return rng.choice(np.array([1.0, 2.0, 4.0, 8.0]), size=(L, H))
    if w.cr_kind == "const_2":
        return np.full((L, H), 2.0)
    if w.cr_kind == "loguniform_1_16_global4":
        return np.exp(rng.uniform(0.0, math.log(16.0), size=(L, H)))
    if w.cr_kind == "skew_10pct_cr1_rest_16_32":
        cr = np.exp(rng.uniform(math.log(16.0), math.log(32.0), size=(L, H)))
        flat = cr.reshape(-1)
        flat[rng.choice(flat.size, size=int(round(0.1 * flat.size)), replace=False)] = 1.0
        return cr
    raise ValueError(w.cr_kind)


def precompressed_lengths(w: Workload) -> np.ndarray:
    """[L, Hkv] slot counts of a pre-compressed cache (same for every batch row).

    log-uniform[1, 16]: lengths round(s * n / CR) clamped to [n/16, n], with the
    scale s found by bisection so the global ratio (total tokens over total
    slots) is exactly 4; the residual of rounding is spread one slot at a time.
    The skewed recipe uses round(n / CR) directly.
    """
    n = w.prompt_len
    cr = head_crs(w)
    if w.cr_kind == "skew_10pct_cr1_rest_16_32":
        return np.clip(np.round(n / cr), 1, n).astype(np.int64)
    if w.cr_kind != "loguniform_1_16_global4":
        raise ValueError(w.cr_kind)
    target = cr.size * n // 4
    lo_len, hi_len = n // 16, n

    def lengths(s):
        return np.clip(np.round(s * n / cr), lo_len, hi_len).astype(np.int64)

    lo, hi = 0.0, 16.0
    for _ in range(200):
        mid = 0.5 * (lo + hi)
        if lengths(mid).sum() < target:
            lo = mid
        else:
            hi = mid
    lens = lengths(hi)
    flat = lens.reshape(-1)
    order = np.argsort(-flat, kind="stable")
    i = 0
    while flat.sum() != target:          # spread the rounding residual
        j = order[i % flat.size]
        step = 1 if flat.sum() < target else -1
        if lo_len <= flat[j] + step <= hi_len:
            flat[j] += step
        i += 1
    return lens


def pool_pages(w: Workload, steps: int) -> int:
    """Pages a cache for this workload needs after `steps` decode steps.

    Pre-compressed caches: exact.  Prefilled caches: the expected slot count
    1 + (n - 1) / CR of every (layer, kv head) plus six standard deviations of
    the binomial append count, capped at n, plus one slot per decode step.
    """
    n, P = w.prompt_len, w.page_size
    if w.cache_kind == "precompressed":
        return int(w.batch * np.ceil((precompressed_lengths(w) + steps) / P).sum())
    cr = head_crs(w)
    pa = 1.0 / cr
    expect = 1 + (n - 1) * pa + 6.0 * np.sqrt(n * pa * (1 - pa))
    slots = np.minimum(np.ceil(expect), n) + steps
    return int(w.batch * np.ceil(slots / P).sum())


def effective_crs(w: Workload) -> np.ndarray:
    """[L, Hkv] CR that drives decode-step decisions."""
    if w.cache_kind == "precompressed":
        return w.prompt_len / precompressed_lengths(w).astype(np.float64)
    return head_crs(w)


# ----------------------------------------------------------------------------
# Decision logits and activations
# ----------------------------------------------------------------------------

def decision_logits(u: np.ndarray, cr: np.ndarray, bias: float = 0.0) -> np.ndarray:
    """k[0] values whose rounded sigmoid (bias c) appends with probability 1/cr.

    u ~ U(0, 1) i.i.d.; logit(u) is Logistic(0, 1).
    """
    u = np.clip(np.asarray(u, dtype=np.float64), 1e-12, 1 - 1e-12)
    lam = np.log(u) - np.log1p(-u)
    cr = np.broadcast_to(np.asarray(cr, dtype=np.float64), lam.shape)
    with np.errstate(divide="ignore"):
        shifted = lam + np.log(np.maximum(cr - 1.0, 0.0))
    return np.where(cr > 1.0, shifted, -(1.0 + np.abs(lam))) + bias


def _np_cast(x: np.ndarray, dtype: str):
    """fp32 numpy array -> torch tensor of the workload dtype (RNE cast)."""
    import torch
    t = torch.from_numpy(np.ascontiguousarray(x, dtype=np.float32))
    return t if dtype == "fp32" else t.to(torch.bfloat16)


def decode_inputs_np(w: Workload, step: int, layer: int, bias: float = 0.0):
    """q [B, Hq, d], k, v [B, Hkv, d] of one decode step as CPU torch tensors.

    N(0, 1) activations; k[..., 0] replaced by decision logits at the
    (layer, head) CR; q[..., 0] stays N(0, 1) so omega = sigmoid(N(0, 1)).
    """
    rng = np_rng(w, 1 + step, layer)
    B, Hq, Hkv, d = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim
    q = rng.standard_normal((B, Hq, d), dtype=np.float32)
    k = rng.standard_normal((B, Hkv, d), dtype=np.float32)
    v = rng.standard_normal((B, Hkv, d), dtype=np.float32)
    cr = effective_crs(w)[layer]
    k[:, :, 0] = decision_logits(rng.uniform(size=(B, Hkv)), cr[None, :], bias)
    return _np_cast(q, w.dtype), _np_cast(k, w.dtype), _np_cast(v, w.dtype)


def prompt_np(w: Workload, layer: int, bias: float = 0.0, n: int | None = None):
    """Prompt-phase inputs of one layer as CPU torch tensors.

    k, v [B, n, Hkv, d]; q0 [B, n, Hq] (the prompt compactor reads only the
    first query neuron, so only that slice is materialised).
    """
    rng = np_rng(w, PROMPT_STREAM, layer)
    n = w.prompt_len if n is None else n
    B, Hq, Hkv, d = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim
    k = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    v = rng.standard_normal((B, n, Hkv, d), dtype=np.float32)
    q0 = rng.standard_normal((B, n, Hq), dtype=np.float32)
    cr = effective_crs(w)[layer]
    k[..., 0] = decision_logits(rng.uniform(size=(B, n, Hkv)), cr[None, None, :], bias)
    return _np_cast(k, w.dtype), _np_cast(v, w.dtype), _np_cast(q0, w.dtype)


# ----------------------------------------------------------------------------
# Device-side generation for the full-size workloads (torch RNG)
# ----------------------------------------------------------------------------

def _torch_dtype(w: Workload):
    import torch
    return torch.float32 if w.dtype == "fp32" else torch.bfloat16


def _gen(w: Workload, stream: int, layer: int, device):
    import torch
    g = torch.Generator(device=device)
    g.manual_seed(seed_for(w, stream, layer))
    return g


def _torch_logits(u, cr_row, bias):
    """Torch twin of decision_logits for device tensors (cr_row per kv head)."""
    import torch
    u = u.clamp(1e-7, 1 - 1e-7)
    lam = torch.log(u) - torch.log1p(-u)
    cr = torch.as_tensor(cr_row, dtype=torch.float32, device=u.device)
    cr = cr.expand_as(lam)
    shifted = lam + torch.log(torch.clamp(cr - 1.0, min=1e-30))
    return torch.where(cr > 1.0, shifted, -(1.0 + lam.abs())) + bias


def decode_inputs_torch(w: Workload, step: int, layer: int, device, bias: float = 0.0):
    """Device twin of decode_inputs_np (different stream, same statistics)."""
    import torch
    g = _gen(w, 1 + step, layer, device)
    B, Hq, Hkv, d = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim
    q = torch.randn((B, Hq, d), generator=g, device=device)
    k = torch.randn((B, Hkv, d), generator=g, device=device)
    v = torch.randn((B, Hkv, d), generator=g, device=device)
    u = torch.rand((B, Hkv), generator=g, device=device)
    k[:, :, 0] = _torch_logits(u, effective_crs(w)[layer][None, :], bias)
    dt = _torch_dtype(w)
    return q.to(dt), k.to(dt), v.to(dt)


def _randn_rows(shape, g, device, dt):
    """N(0, 1) of dtype dt, generated one leading row at a time (bounded fp32 temporaries)."""
    import torch
    out = torch.empty(shape, dtype=dt, device=device)
    for i in range(shape[0]):
        out[i] = torch.randn(shape[1:], generator=g, device=device)
    return out


def prompt_torch(w: Workload, layer: int, device, bias: float = 0.0, n: int | None = None):
    """Device twin of prompt_np: k, v [B, n, Hkv, d], q0 [B, n, Hq]."""
    import torch
    g = _gen(w, PROMPT_STREAM, layer, device)
    n = w.prompt_len if n is None else n
    B, Hq, Hkv, d = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim
    dt = _torch_dtype(w)
    k = _randn_rows((B, n, Hkv, d), g, device, dt)
    v = _randn_rows((B, n, Hkv, d), g, device, dt)
    q0 = torch.randn((B, n, Hq), generator=g, device=device).to(dt)
    u = torch.rand((B, n, Hkv), generator=g, device=device)
    k[..., 0] = _torch_logits(u, effective_crs(w)[layer][None, None, :], bias).to(dt)
    return k, v, q0


def prompt_full_torch(w: Workload, layer: int, device, bias: float = 0.0, n: int | None = None):
    """Prompt inputs with whole query rows (for prompt-phase attention):
    k, v [B, n, Hkv, d] and q [B, n, Hq, d], all N(0, 1), k[..., 0] from the
    decision logits of each (layer, kv head)."""
    g = _gen(w, PROMPT_STREAM, layer, device)
    import torch
    n = w.prompt_len if n is None else n
    B, Hq, Hkv, d = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim
    dt = _torch_dtype(w)
    k = _randn_rows((B, n, Hkv, d), g, device, dt)
    v = _randn_rows((B, n, Hkv, d), g, device, dt)
    q = _randn_rows((B, n, Hq, d), g, device, dt)
    u = torch.rand((B, n, Hkv), generator=g, device=device)
    k[..., 0] = _torch_logits(u, effective_crs(w)[layer][None, None, :], bias).to(dt)
    return k, v, q


def precompressed_torch(w: Workload, layer: int, device):
    """A pre-compressed cache for one layer (inputs to the cache import).

    K, V dense [B, Hkv, Lmax, d] with N(0, 1) slots (K element 0 = 0, as DMC
    stores keys), lengths [B, Hkv] int32 and z [B, Hkv] = CR / 2 (the expected
    importance sum of a CR-token segment at mean omega 1/2).
    """
    import torch
    lens_np = precompressed_lengths(w)[layer]                  # [Hkv]
    B, Hkv, d = w.batch, w.num_kv_heads, w.head_dim
    lmax = int(lens_np.max())
    g = _gen(w, PROMPT_STREAM, layer, device)
    dt = _torch_dtype(w)
    K = _randn_rows((B, Hkv, lmax, d), g, device, dt)
    V = _randn_rows((B, Hkv, lmax, d), g, device, dt)
    K[..., 0] = 0
    lengths = torch.as_tensor(lens_np, dtype=torch.int32, device=device).repeat(B, 1)
    crs = w.prompt_len / lens_np.astype(np.float64)
    z = torch.as_tensor(0.5 * crs, dtype=torch.float32, device=device).repeat(B, 1)
    return K, V, lengths.contiguous(), z.contiguous()


def sample_units(w: Workload, count: int, seed: int = 12345):
    """A seeded sample of (layer, b, g) units, always including the unit with
    the longest and the shortest cache of layer 0 when the cache is ragged."""
    rng = np.random.Generator(np.random.PCG64(seed))
    L, B, H = w.num_layers, w.batch, w.num_kv_heads
    total = L * B * H
    pick = rng.choice(total, size=min(count, total), replace=False)
    units = [(int(i // (B * H)), int((i // H) % B), int(i % H)) for i in pick]
    if w.cache_kind == "precompressed":
        lens = precompressed_lengths(w)[0]
        for g in (int(np.argmax(lens)), int(np.argmin(lens))):
            if (0, 0, g) not in units:
                units.append((0, 0, g))
    return sorted(units)


def train_inputs_torch(w: Workload, layer: int, device, c: float = TRAIN_C):
    """Training-step inputs of one layer on the device: q [B, n, Hq, d], k, v
    [B, n, Hkv, d] ~ N(0, 1) in the workload dtype, k[..., 0] = c + log(CR - 1)
    + N(0, 0.3) per kv head (c - 3 for CR 1), so that with the logistic
    noise [B, n, Hkv] (fp32, the Gumbel-sigmoid's draws) a decision
    accumulates with probability about 1 - 1/CR; dout ~ N(0, 1) is the
    incoming gradient."""
    import torch
    g = _gen(w, PROMPT_STREAM, layer, device)
    n = w.prompt_len
    B, Hq, Hkv, d = w.batch, w.num_q_heads, w.num_kv_heads, w.head_dim
    dt = _torch_dtype(w)
    q = _randn_rows((B, n, Hq, d), g, device, dt)
    k = _randn_rows((B, n, Hkv, d), g, device, dt)
    v = _randn_rows((B, n, Hkv, d), g, device, dt)
    dout = _randn_rows((B, n, Hq, d), g, device, dt)
    cr = torch.as_tensor(head_crs(w)[layer], dtype=torch.float32, device=device)
    k0 = torch.where(cr > 1, c + torch.log(torch.clamp(cr - 1, min=1e-30)), torch.full_like(cr, c - 3))
    jitter = 0.3 * torch.randn((B, n, Hkv), generator=g, device=device)
    k[..., 0] = (k0[None, None, :] + jitter).to(dt)
    u = torch.rand((B, n, Hkv), generator=g, device=device).clamp(1e-7, 1 - 1e-7)
    noise = (torch.log(u) - torch.log1p(-u)).contiguous()
    return q, k, v, noise, dout
