"""Training-time DMC attention (Sec. 3.2, 3.3, masking appendix) on the GPU
against the float64 training oracle (autograd backward), through the C ABI:
forward outputs and relaxed decisions, then dq, dk, dv."""
import numpy as np
import pytest

import oracle.dmc_train as T
from tests.gpu_helpers import TOL, f64, log, torch_dtype

pytestmark = pytest.mark.gpu


def _inputs(rng, B, n, Hkv, G, d, crs, c):
    """q, k, v ~ N(0, 1); k[0] = c + log(CR - 1) per kv head, so that with
    the logistic noise P(alpha > 1/2) = 1 - 1/CR (CR = 1: c - 3)."""
    q = rng.standard_normal((B, n, Hkv * G, d)).astype(np.float32)
    k = rng.standard_normal((B, n, Hkv, d)).astype(np.float32)
    v = rng.standard_normal((B, n, Hkv, d)).astype(np.float32)
    crs = np.asarray(crs, dtype=np.float64)
    k0 = np.where(crs > 1, c + np.log(np.maximum(crs - 1, 1e-12)), c - 3.0)
    k[..., 0] = k0[None, None, :].astype(np.float32) + 0.3 * rng.standard_normal((B, n, Hkv)).astype(np.float32)
    noise = rng.logistic(size=(B, n, Hkv)).astype(np.float32)
    dout = rng.standard_normal((B, n, Hkv * G, d)).astype(np.float32)
    dalpha = (0.5 * rng.standard_normal((B, n, Hkv))).astype(np.float32)
    return q, k, v, noise, dout, dalpha


def _grad_close(got, want, dtype, what):
    """Gradients: elementwise |got - want| <= atol * scale + rtol * |want|,
    with scale = max(1, max|want|) taken over the slice being checked.  The
    decision and importance neurons (element 0 of every key and query row)
    get their gradient through alpha and omega (dk[..., 0] = dx / tau is an
    order of magnitude above the other entries at tau = 0.1), so element 0
    and elements 1.. are checked separately, each against its own scale --
    a dropped term in either part cannot hide behind the other's magnitude.
    Returns the worst error over scale of each part."""
    got, want = np.asarray(got, np.float64), np.asarray(want, np.float64)
    parts = ((f"{what}[..., 0]", got[..., :1], want[..., :1]),
             (f"{what}[..., 1:]", got[..., 1:], want[..., 1:]))
    return tuple(_close_scaled(g, w, dtype, name) for name, g, w in parts)


def _close_scaled(got, want, dtype, what):
    atol, rtol = TOL[dtype]
    scale = max(1.0, float(np.abs(want).max(initial=0.0)))
    err = np.abs(got - want)
    bad = err > atol * scale + rtol * np.abs(want)
    worst = float(err.max(initial=0.0)) / scale
    if bad.any():
        i = np.unravel_index(np.argmax(err - rtol * np.abs(want)), err.shape)
        raise AssertionError(f"{what}: {bad.sum()} of {bad.size} outside tolerance; worst at {i}: "
                             f"got {got[i]!r} want {want[i]!r}; max err / scale {worst:.3e} "
                             f"(scale {scale:.3g})")
    return worst


CASES = [
    # dtype, d, G, B, Hkv, n, window, c, tau, crs, omega, dalpha
    ("fp32", 64, 1, 2, 2, 70, 12, 5.0, 0.1, [2.0, 8.0], "lead", False),
    ("fp32", 128, 2, 1, 2, 100, 3, 1.0, 1.0, [1.0, 4.0], "lead", True),
    ("fp32", 64, 8, 1, 1, 40, 1, 0.0, 0.5, [3.0], "lead", True),
    ("fp32", 64, 4, 1, 2, 90, 64, 5.0, 0.3, [20.0, 2.0], "lead", False),
    ("fp32", 128, 1, 1, 2, 33, 12, 5.0, 0.1, [4.0, 4.0], "uniform", True),
    ("fp32", 64, 2, 2, 1, 1, 12, 5.0, 0.1, [4.0], "lead", True),
    ("bf16", 128, 1, 2, 2, 100, 12, 5.0, 0.1, [2.0, 6.0], "lead", True),
    ("bf16", 128, 8, 1, 2, 64, 12, 5.0, 0.5, [4.0, 1.0], "lead", False),
    ("bf16", 64, 2, 1, 2, 80, 5, 2.0, 1.0, [3.0, 10.0], "lead", True),
    # several 128-token tiles and 32-row blocks, ragged tail
    ("bf16", 128, 1, 1, 2, 300, 12, 5.0, 0.1, [1.0, 8.0], "lead", True),
    ("bf16", 64, 4, 1, 2, 201, 12, 5.0, 0.1, [2.0, 4.0], "uniform", False),
    ("bf16", 128, 2, 2, 1, 161, 64, 5.0, 0.2, [16.0], "lead", True),
    # every width class of the matrix-core states pass (w = 1, 17, 18, 40)
    ("bf16", 64, 1, 1, 2, 90, 1, 5.0, 0.1, [3.0, 1.0], "lead", True),
    ("bf16", 128, 1, 1, 1, 70, 17, 3.0, 0.2, [6.0], "lead", False),
    ("bf16", 128, 4, 1, 2, 120, 18, 5.0, 0.1, [8.0, 2.0], "uniform", True),
    ("bf16", 64, 1, 1, 1, 150, 40, 5.0, 0.3, [30.0], "lead", True),
    # degenerate and block-boundary lengths on the matrix-core kernels
    ("bf16", 128, 1, 1, 2, 1, 12, 5.0, 0.1, [2.0, 4.0], "lead", True),
    ("bf16", 128, 4, 2, 1, 2, 12, 5.0, 0.1, [3.0], "uniform", False),
    ("bf16", 64, 2, 1, 2, 33, 3, 5.0, 0.1, [2.0, 8.0], "lead", True),
]


@pytest.mark.parametrize("case", CASES, ids=lambda c: "-".join(str(x) for x in c[:7]))
def test_train_forward_backward(torch_cuda, case):
    import torch
    import paper_2403_09636_amd as P
    dtype, d, G, B, Hkv, n, w, c, tau, crs, omega, use_dalpha = case
    log(f"case train {case}")
    rng = np.random.default_rng(900 + d + 10 * G + n + w)
    q, k, v, noise, dout, dalpha = _inputs(rng, B, n, Hkv, G, d, crs, c)
    dt = torch_dtype(dtype)
    qt, kt, vt, dot = (torch.from_numpy(x).to(dt).cuda() for x in (q, k, v, dout))
    nt = torch.from_numpy(noise).cuda()
    dat = torch.from_numpy(dalpha).cuda() if use_dalpha else None
    cfg = P.make_train_config(B, n, Hkv * G, Hkv, d, dtype, decision_bias=c, temperature=tau,
                              window=w, omega_src=omega)
    tr = P.DMCTrainer(cfg)
    alpha = torch.empty((B, n, Hkv), dtype=torch.float32, device="cuda")
    out = tr.forward(qt, kt, vt, nt, alpha=alpha)
    dq, dk, dv = tr.backward(qt, kt, vt, nt, out, dot, dalpha=dat)
    torch.cuda.synchronize()

    qo, ko, vo, do = (torch.from_numpy(f64(x)) for x in (qt, kt, vt, dot))
    no = torch.from_numpy(noise.astype(np.float64))
    o_ref, a_ref = T.train_forward(qo, ko, vo, no, c, tau, w, omega)
    rq, rk, rv = T.train_backward(qo, ko, vo, no, do, dalpha.astype(np.float64) if use_dalpha else None,
                                  c, tau, w, omega)
    atol, rtol = TOL[dtype]
    a_err = np.abs(alpha.cpu().numpy() - a_ref.detach().numpy()).max()
    assert a_err < 1e-5, f"alpha error {a_err}"
    o_err = np.abs(f64(out) - o_ref.detach().numpy())
    assert (o_err <= atol + rtol * np.abs(o_ref.detach().numpy())).all(), f"output max err {o_err.max()}"
    errs = [_grad_close(f64(x), r.numpy(), dtype, name)
            for x, r, name in ((dq, rq, "dq"), (dk, rk, "dk"))]
    ev = _close_scaled(f64(dv), rv.numpy(), dtype, "dv")
    log(f"  out {o_err.max():.2e}  dq[0] {errs[0][0]:.2e} dq[1:] {errs[0][1]:.2e}  "
        f"dk[0] {errs[1][0]:.2e} dk[1:] {errs[1][1]:.2e}  dv {ev:.2e} (of each part's scale)")


def test_train_full_size_sampled(torch_cuda):
    """The bench's training workload (one Llama-2-7B layer: 4 x 4096 tokens,
    32 heads, d = 128, bf16, c = 5, tau = 0.1, w = 12) in its launch
    configuration; one (batch row, head) unit checked in full against the
    oracle -- forward rows, relaxed decisions and dq, dk, dv of that unit
    (units are independent, so its slice of the inputs fixes them)."""
    import torch
    import paper_2403_09636_amd as P
    import workloads as W
    w = W.WORKLOADS["llama7b_train"]
    log("case train full size sampled")
    q, k, v, noise, dout = W.train_inputs_torch(w, 0, "cuda")
    B, n = w.batch, w.prompt_len
    cfg = P.make_train_config(B, n, w.num_q_heads, w.num_kv_heads, w.head_dim, w.dtype,
                              W.TRAIN_C, W.TRAIN_TAU, W.TRAIN_WINDOW)
    tr = P.DMCTrainer(cfg)
    alpha = torch.empty((B, n, w.num_kv_heads), dtype=torch.float32, device="cuda")
    out = tr.forward(q, k, v, noise, alpha=alpha)
    dq, dk, dv = tr.backward(q, k, v, noise, out, dout)
    torch.cuda.synchronize()
    b, g = 2, 19
    sl = (slice(b, b + 1), slice(None), slice(g, g + 1))
    qo, ko, vo, do = (torch.from_numpy(f64(x[sl])) for x in (q, k, v, dout))
    no = torch.from_numpy(f64(noise[sl]))
    o_ref, a_ref = T.train_forward(qo, ko, vo, no, W.TRAIN_C, W.TRAIN_TAU, W.TRAIN_WINDOW)
    rq, rk, rv = T.train_backward(qo, ko, vo, no, do, None, W.TRAIN_C, W.TRAIN_TAU, W.TRAIN_WINDOW)
    a_err = np.abs(f64(alpha[sl]) - a_ref.detach().numpy()).max()
    assert a_err < 1e-5, f"alpha error {a_err}"
    o_err = np.abs(f64(out[sl]) - o_ref.detach().numpy())
    assert (o_err <= 2e-2 + 1e-2 * np.abs(o_ref.detach().numpy())).all(), o_err.max()
    errs = [_grad_close(f64(x[sl]), r.numpy(), "bf16", name)
            for x, r, name in ((dq, rq, "dq"), (dk, rk, "dk"))]
    ev = _close_scaled(f64(dv[sl]), rv.numpy(), "bf16", "dv")
    log(f"  unit {(b, g)}: out {o_err.max():.2e}  dq[0] {errs[0][0]:.2e} dq[1:] {errs[0][1]:.2e}  "
        f"dk[0] {errs[1][0]:.2e} dk[1:] {errs[1][1]:.2e}  dv {ev:.2e}")
