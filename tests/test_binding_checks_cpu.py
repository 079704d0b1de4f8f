"""The binding's argument checks, on CPU tensors (no GPU): every tensor
property the C ABI cannot see -- dtype, shape against the configuration,
contiguity or a contiguous last dimension where the header requires it,
16-byte alignment, overlap of outputs with inputs, and the device -- is
rejected with DMCError before any library call.  Each case breaks exactly
one property; the all-valid case on the CPU fails only on the device."""
import pytest
import torch

import paper_2403_09636_amd as P
from paper_2403_09636_amd import binding as Bd

DEV = torch.device("cuda", 0)
B, HQ, HKV, D = 2, 8, 2, 64


def _cfg(dtype="bf16"):
    return P.make_config(1, B, HQ, HKV, D, dtype, page_size=32, max_slots_per_seq=128)


def _misaligned(shape, dtype=torch.bfloat16):
    base = torch.zeros(int(torch.tensor(shape).prod()) + 8, dtype=dtype)
    return base[1:1 + int(torch.tensor(shape).prod())].view(shape)


def _raises(fn, msg):
    with pytest.raises(P.DMCError) as e:
        fn()
    assert msg in str(e.value), str(e.value)


def _decode_args():
    bf = torch.bfloat16
    return dict(q=torch.zeros(B, HQ, D, dtype=bf), k=torch.zeros(B, HKV, D, dtype=bf),
                v=torch.zeros(B, HKV, D, dtype=bf), out=torch.zeros(B, HQ, D, dtype=bf),
                slot_index=torch.zeros(B, HKV, dtype=torch.int32))


@pytest.mark.parametrize("name,bad,msg", [
    ("q", torch.zeros(B, HQ, D, dtype=torch.float32), "dtype"),
    ("q", torch.zeros(B, HKV, D, dtype=torch.bfloat16), "shape"),     # kv-shaped query
    ("k", torch.zeros(B, HQ, D, dtype=torch.bfloat16), "shape"),
    ("v", torch.zeros(B, HKV, D + 8, dtype=torch.bfloat16), "shape"),
    ("out", torch.zeros(B, D, HQ, dtype=torch.bfloat16).transpose(1, 2), "contiguous"),
    ("q", _misaligned((B, HQ, D)), "aligned"),
    ("slot_index", torch.zeros(B, HKV, dtype=torch.int64), "dtype"),
    ("slot_index", torch.zeros(B, HQ, dtype=torch.int32), "shape"),
])
def test_decode_rejections(name, bad, msg):
    a = _decode_args()
    a[name] = bad
    _raises(lambda: Bd.check_decode_args(_cfg(), DEV, **a), msg)


def test_decode_fp32_cache_rejects_bf16():
    _raises(lambda: Bd.check_decode_args(_cfg("fp32"), DEV, **_decode_args()), "dtype")


def test_decode_out_overlapping_q():
    a = _decode_args()
    a["out"] = a["q"]
    _raises(lambda: Bd.check_decode_args(_cfg(), DEV, **a), "overlaps")


def test_decode_valid_cpu_tensors_fail_on_device():
    _raises(lambda: Bd.check_decode_args(_cfg(), DEV, **_decode_args()), "is on cpu")


def _prefill_args(n=40):
    bf = torch.bfloat16
    return dict(k=torch.zeros(B, n, HKV, D, dtype=bf), v=torch.zeros(B, n, HKV, D, dtype=bf),
                q=torch.zeros(B, n, HQ, dtype=bf), n=n,
                prompt_lens=torch.zeros(B, dtype=torch.int32),
                slot_index=torch.zeros(B, HKV, n, dtype=torch.int32))


@pytest.mark.parametrize("name,bad,msg", [
    ("k", torch.zeros(B, 40, HKV, D, dtype=torch.float32), "dtype"),
    ("k", torch.zeros(B, 40, HQ, D, dtype=torch.bfloat16), "shape"),
    ("v", torch.zeros(B, 30, HKV, D, dtype=torch.bfloat16), "fewer than n"),
    ("k", torch.zeros(B, 40, HKV, D + 8, dtype=torch.bfloat16), "shape"),
    ("k", torch.zeros(B, 40, HKV, D, 2, dtype=torch.bfloat16)[..., 0], "last dimension"),
    ("v", torch.zeros(B, 41, HKV, D, dtype=torch.bfloat16)[:, :40].reshape(B, 40, HKV, D), None),
    ("k", torch.zeros(B, 40, HKV * D + 4, dtype=torch.bfloat16)[..., :HKV * D].unflatten(2, (HKV, D)),
     "multiples of 8"),
    ("q", torch.zeros(B, 40, HKV, dtype=torch.bfloat16), "shape"),
    ("q", torch.zeros(B, 40, HQ, dtype=torch.float32), "dtype"),
    ("prompt_lens", torch.zeros(B + 1, dtype=torch.int32), "shape"),
    ("prompt_lens", torch.zeros(B, dtype=torch.int64), "dtype"),
    ("slot_index", torch.zeros(B, HKV, 39, dtype=torch.int32), "shape"),
])
def test_prefill_rejections(name, bad, msg):
    a = _prefill_args()
    a[name] = bad
    if msg is None:      # a valid variant (a contiguous copy): fails only on the device
        msg = "is on cpu"
    _raises(lambda: Bd.check_prefill_args(_cfg(), DEV, **a), msg)


def test_prefill_prompt_too_long():
    a = _prefill_args(n=129)
    _raises(lambda: Bd.check_prefill_args(_cfg(), DEV, **a), "prompt length")


def test_prefill_attend_needs_full_query_and_out():
    a = _prefill_args()
    bf = torch.bfloat16
    # prompt attention reads every query element: a [B, n, Hq] tensor of q[..., 0] is refused
    _raises(lambda: Bd.check_prefill_args(_cfg(), DEV, **a, full_q=True,
                                          out=torch.zeros(B, 40, HQ, D, dtype=bf)), "shape")
    a["q"] = torch.zeros(B, 40, HQ, D, dtype=bf)
    _raises(lambda: Bd.check_prefill_args(_cfg(), DEV, **a, full_q=True,
                                          out=torch.zeros(B, 40, HKV, D, dtype=bf)), "shape")
    _raises(lambda: Bd.check_prefill_args(_cfg(), DEV, **a, full_q=True, out=a["q"]), "overlaps")
    _raises(lambda: Bd.check_prefill_args(_cfg(), DEV, **a, full_q=True,
                                          out=_misaligned((B, 40, HQ, D))), "aligned")
    _raises(lambda: Bd.check_prefill_args(_cfg(), DEV, **a, full_q=True,
                                          out=torch.zeros(B, 40, HQ, D, dtype=bf)), "is on cpu")


@pytest.mark.parametrize("name,msg", [
    ("K_dtype", "dtype"), ("V_shape", "shape"), ("lengths_dtype", "dtype"),
    ("z_dtype", "dtype"), ("K_noncontig", "contiguous"), ("valid", "is on cpu"),
])
def test_import_rejections(name, msg):
    bf = torch.bfloat16
    K = torch.zeros(B, HKV, 16, D, dtype=bf)
    V = torch.zeros(B, HKV, 16, D, dtype=bf)
    lens = torch.zeros(B, HKV, dtype=torch.int32)
    z = torch.zeros(B, HKV, dtype=torch.float32)
    if name == "K_dtype":
        K = K.float()
    elif name == "V_shape":
        V = torch.zeros(B, HKV, 15, D, dtype=bf)
    elif name == "lengths_dtype":
        lens = lens.long()
    elif name == "z_dtype":
        z = z.to(bf)
    elif name == "K_noncontig":
        K = torch.zeros(B, 16, HKV, D, dtype=bf).transpose(1, 2)
    _raises(lambda: Bd.check_import_args(_cfg(), DEV, K, V, lens, z), msg)


@pytest.mark.parametrize("name,msg", [
    ("noise_dtype", "dtype"), ("k_shape", "shape"), ("out_dtype", "dtype"),
    ("dq_shape", "shape"), ("valid", "is on cpu"),
])
def test_train_rejections(name, msg):
    cfg = P.make_train_config(1, 20, HQ, HKV, D, "bf16")
    bf = torch.bfloat16
    q = torch.zeros(1, 20, HQ, D, dtype=bf)
    k = torch.zeros(1, 20, HKV, D, dtype=bf)
    v = torch.zeros(1, 20, HKV, D, dtype=bf)
    noise = torch.zeros(1, 20, HKV, dtype=torch.float32)
    out = torch.zeros(1, 20, HQ, D, dtype=bf)
    dq = torch.zeros(1, 20, HQ, D, dtype=bf)
    if name == "noise_dtype":
        noise = noise.to(bf)
    elif name == "k_shape":
        k = torch.zeros(1, 20, HQ, D, dtype=bf)
    elif name == "out_dtype":
        out = out.float()
    elif name == "dq_shape":
        dq = torch.zeros(1, 20, HKV, D, dtype=bf)
    _raises(lambda: Bd.check_train_args(cfg, DEV, q, k, v, noise,
                                        (("out", out, "q"), ("dq", dq, "q"))), msg)
