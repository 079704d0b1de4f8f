"""Shared drivers for the GPU parity tests: run the HIP path through the C
ABI and the float64 oracle on the same seeded inputs, compare."""
from __future__ import annotations

import math
import sys

import numpy as np

import oracle
from workloads import decision_logits

TOL = {"fp32": (1e-5, 1e-5), "bf16": (2e-2, 1e-2)}   # (atol, rtol)


def log(msg):
    print(msg, flush=True)
    sys.stdout.flush()


def f64(t):
    """torch tensor (any dtype, any device) -> float64 numpy."""
    import torch
    return t.detach().to("cpu", torch.float32).numpy().astype(np.float64)


def assert_close(got, want, dtype, what):
    atol, rtol = TOL[dtype]
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    assert got.shape == want.shape, (what, got.shape, want.shape)
    err = np.abs(got - want)
    bad = err > atol + rtol * np.abs(want)
    if bad.any():
        i = np.unravel_index(np.argmax(err - (atol + rtol * np.abs(want))), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; worst at {i}: "
                             f"got {got[i]!r} want {want[i]!r}; max abs err {err.max():.3e}")
    return float(err.max(initial=0.0))


def torch_dtype(dtype):
    import torch
    return torch.float32 if dtype == "fp32" else torch.bfloat16


def random_step(rng, B, Hq, Hkv, d, cr, dtype, device, bias=0.0):
    """q, k, v of one decode step on `device` (k[0] from decision logits)."""
    import torch
    q = rng.standard_normal((B, Hq, d), dtype=np.float32)
    k = rng.standard_normal((B, Hkv, d), dtype=np.float32)
    v = rng.standard_normal((B, Hkv, d), dtype=np.float32)
    k[:, :, 0] = decision_logits(rng.uniform(size=(B, Hkv)), np.asarray(cr)[None, :], bias)
    dt = torch_dtype(dtype)
    return tuple(torch.from_numpy(x).to(dt).to(device) for x in (q, k, v))


class Pair:
    """A DMCCache on the GPU and a DMCOracle fed the same inputs."""

    def __init__(self, L, B, Hq, Hkv, d, dtype="bf16", page_size=32, max_slots=512,
                 num_pages=None, bias=0.0, omega_src="lead", split_tile=0, max_prompt_len=0,
                 decision_src="per_head", window=0):
        import paper_2403_09636_amd as P
        self.cfg = P.make_config(L, B, Hq, Hkv, d, dtype, page_size, max_slots, num_pages, bias,
                                 omega_src, split_tile, max_prompt_len, decision_src, window)
        self.gpu = P.DMCCache(self.cfg, device="cuda")
        self.orc = oracle.DMCOracle(L, B, Hq, Hkv, d, max_slots, decision_bias=bias,
                                    omega_src=omega_src, decision_src=decision_src,
                                    window=window)
        self.dtype, self.B, self.Hq, self.Hkv, self.d = dtype, B, Hq, Hkv, d

    def decode(self, layer, q, k, v, check_out=True):
        import torch
        out = torch.empty_like(q)
        slot = torch.empty((self.B, self.Hkv), dtype=torch.int32, device=q.device)
        self.gpu.decode_step(layer, q, k, v, out=out, slot_index=slot)
        o_ref, s_ref = self.orc.decode_step(layer, f64(q), f64(k), f64(v))
        got_slot = slot.cpu().numpy()
        assert (got_slot == s_ref).all(), f"slot index mismatch:\n{got_slot}\n{s_ref}"
        err = assert_close(f64(out), o_ref, self.dtype, "decode output") if check_out else 0.0
        return err

    def prefill(self, layer, k, v, q0, prompt_lens=None):
        import torch
        B, n = k.shape[:2]
        slot = torch.full((B, self.Hkv, n), -7, dtype=torch.int32, device=k.device)
        lens_t = None if prompt_lens is None else torch.as_tensor(
            prompt_lens, dtype=torch.int32, device=k.device)
        self.gpu.prefill(layer, k, v, q0, prompt_lens=lens_t, slot_index=slot)
        s_ref = self.orc.prefill(layer, f64(k), f64(v), f64(q0), prompt_lens=prompt_lens)
        got = slot.cpu().numpy()
        assert (got == s_ref).all(), "prefill slot index mismatch"

    def prefill_attend(self, layer, k, v, q, prompt_lens=None, out=None):
        """Prompt attention on both sides: slot indices bit-exact, outputs
        (zeros past each row's prompt length) within tolerance."""
        import torch
        B, n = k.shape[:2]
        slot = torch.full((B, self.Hkv, n), -7, dtype=torch.int32, device=k.device)
        lens_t = None if prompt_lens is None else torch.as_tensor(
            prompt_lens, dtype=torch.int32, device=k.device)
        out = self.gpu.prefill_attend(layer, k, v, q, out=out, prompt_lens=lens_t, slot_index=slot)
        o_ref, s_ref = self.orc.prefill_attend(layer, f64(q), f64(k), f64(v),
                                               prompt_lens=prompt_lens)
        got = slot.cpu().numpy()
        assert (got == s_ref).all(), "prompt slot index mismatch"
        return assert_close(f64(out), o_ref, self.dtype, "prompt attention output")

    def compare_cache(self, layer):
        """Lengths bit-exact; slots and z within tolerance."""
        K_ref, V_ref, l_ref, z_ref = self.orc.export(layer)
        lens = self.gpu.lengths(layer).cpu().numpy()
        assert (lens == l_ref).all(), f"lengths mismatch:\n{lens}\n{l_ref}"
        dense = int(max(1, l_ref.max()))
        K, V, z = self.gpu.export(layer, dense_slots=dense)
        K, V, z = f64(K), f64(V), f64(z)
        mask = np.arange(dense)[None, None, :] < l_ref[:, :, None]
        assert_close(K[mask], K_ref[:, :, :dense][mask], self.dtype, "cache keys")
        assert_close(V[mask], V_ref[:, :, :dense][mask], self.dtype, "cache values")
        assert (K[~mask] == 0).all() and (V[~mask] == 0).all(), "export padding not zero"
        has = l_ref > 0
        # z is fp32 in both precisions; its tolerance follows the slot dtype's rtol
        zt = 1e-5 if self.dtype == "fp32" else 1e-4
        assert np.allclose(z[has], z_ref[has], rtol=zt, atol=zt), "z mismatch"

    def ok(self):
        self.gpu.check()


def expected_lengths_after(orc_lengths, k0, bias):
    """Slot counts after one step from the oracle's decision rule."""
    a = oracle.decision(k0, bias) * (orc_lengths > 0)
    return orc_lengths + (1 - a)


def scale_for(d):
    return 1.0 / math.sqrt(d)
