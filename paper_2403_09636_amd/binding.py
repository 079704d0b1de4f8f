"""ctypes binding of libdmc.so (the gfx950 DMC decode-path library).

Argument marshalling only: every step of the path runs in the library's HIP
kernels.  PyTorch supplies device memory and the current HIP stream.  If the
library is missing or fails to load, importing this module raises -- there
is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from ctypes import POINTER, c_char_p, c_float, c_int32, c_int64, c_size_t, c_void_p

HERE = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(HERE, "libdmc.so")

DMC_OK, DMC_ERR_INVALID_ARG, DMC_ERR_UNSUPPORTED, DMC_ERR_CAPACITY, DMC_ERR_HIP = range(5)
DMC_BF16, DMC_FP32 = 0, 1
DMC_OMEGA_LEAD_QHEAD, DMC_OMEGA_GROUP_MEAN, DMC_OMEGA_UNIFORM = 0, 1, 2
DMC_DECISION_PER_HEAD, DMC_DECISION_SHARED_LAYER = 0, 1
OMEGA_SRC = {"lead": DMC_OMEGA_LEAD_QHEAD, "group_mean": DMC_OMEGA_GROUP_MEAN,
             "uniform": DMC_OMEGA_UNIFORM}
DECISION_SRC = {"per_head": DMC_DECISION_PER_HEAD, "shared_layer": DMC_DECISION_SHARED_LAYER}
STATUS_NAMES = {0: "DMC_OK", 1: "DMC_ERR_INVALID_ARG", 2: "DMC_ERR_UNSUPPORTED",
                3: "DMC_ERR_CAPACITY", 4: "DMC_ERR_HIP"}

#: Every entry point declared in include/dmc.h.
EXPORTS = ("dmc_cache_workspace_bytes", "dmc_cache_alloc", "dmc_cache_free", "dmc_cache_reset",
           "dmc_prefill_compress", "dmc_prefill_attend", "dmc_decode_step", "dmc_decode_step_static",
           "dmc_cache_lengths", "dmc_cache_export",
           "dmc_cache_import", "dmc_cache_check", "dmc_cache_pages_used", "dmc_last_error",
           "dmc_train_workspace_bytes", "dmc_train_forward", "dmc_train_backward")


class CacheConfig(ctypes.Structure):
    """Mirror of dmc_cache_config."""
    _fields_ = [("num_layers", c_int32), ("batch", c_int32), ("num_q_heads", c_int32),
                ("num_kv_heads", c_int32), ("head_dim", c_int32), ("dtype", c_int32),
                ("page_size", c_int32), ("max_slots_per_seq", c_int32), ("num_pages", c_int64),
                ("decision_bias", c_float), ("omega_src", c_int32), ("split_tile", c_int32),
                ("max_prompt_len", c_int32), ("decision_src", c_int32), ("window", c_int32)]


class TrainConfig(ctypes.Structure):
    """Mirror of dmc_train_config."""
    _fields_ = [("batch", c_int32), ("seq_len", c_int32), ("num_q_heads", c_int32),
                ("num_kv_heads", c_int32), ("head_dim", c_int32), ("dtype", c_int32),
                ("decision_bias", c_float), ("temperature", c_float), ("window", c_int32),
                ("omega_src", c_int32)]


class DMCError(RuntimeError):
    def __init__(self, status, message):
        super().__init__(f"{STATUS_NAMES.get(status, status)}: {message}")
        self.status = status


def _load():
    # torch first: its HIP runtime is then the one the library binds to (one
    # runtime per process; loading the library first can bring in a second
    # copy, which then finds no device)
    import torch  # noqa: F401
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "or python paper_2403_09636_amd/csrc/build.py")
    lib = ctypes.CDLL(LIB_PATH)
    i64p = POINTER(c_int64)
    lib.dmc_cache_workspace_bytes.argtypes = [POINTER(CacheConfig)]
    lib.dmc_cache_workspace_bytes.restype = c_size_t
    lib.dmc_cache_alloc.argtypes = [POINTER(CacheConfig), c_void_p, c_size_t, c_void_p,
                                    POINTER(c_void_p)]
    lib.dmc_cache_free.argtypes = [c_void_p]
    lib.dmc_cache_reset.argtypes = [c_void_p, c_void_p]
    lib.dmc_prefill_compress.argtypes = [c_void_p, c_int32, c_void_p, i64p, c_void_p, i64p,
                                         c_void_p, i64p, c_int32, c_void_p, c_void_p, c_void_p]
    lib.dmc_prefill_attend.argtypes = [c_void_p, c_int32, c_void_p, i64p, c_void_p, i64p,
                                       c_void_p, i64p, c_int32, c_void_p, c_void_p, i64p,
                                       c_void_p, c_void_p]
    lib.dmc_decode_step.argtypes = [c_void_p, c_int32, c_void_p, c_void_p, c_void_p, c_void_p,
                                    c_void_p, c_void_p]
    lib.dmc_decode_step_static.argtypes = lib.dmc_decode_step.argtypes
    lib.dmc_cache_lengths.argtypes = [c_void_p, c_int32, c_void_p, c_void_p]
    lib.dmc_cache_export.argtypes = [c_void_p, c_int32, c_void_p, c_void_p, c_int32, c_void_p,
                                     c_void_p]
    lib.dmc_cache_import.argtypes = [c_void_p, c_int32, c_void_p, c_void_p, c_int32, c_void_p,
                                     c_void_p, c_void_p]
    lib.dmc_cache_check.argtypes = [c_void_p, c_void_p]
    lib.dmc_cache_pages_used.argtypes = [c_void_p, i64p, c_void_p]
    lib.dmc_last_error.argtypes = []
    lib.dmc_last_error.restype = c_char_p
    lib.dmc_train_workspace_bytes.argtypes = [POINTER(TrainConfig)]
    lib.dmc_train_workspace_bytes.restype = c_size_t
    lib.dmc_train_forward.argtypes = [POINTER(TrainConfig), c_void_p, c_void_p, c_void_p, c_void_p,
                                      c_void_p, c_void_p, c_void_p, c_size_t, c_void_p]
    lib.dmc_train_backward.argtypes = [POINTER(TrainConfig), c_void_p, c_void_p, c_void_p, c_void_p,
                                       c_void_p, c_void_p, c_void_p, c_void_p, c_void_p, c_void_p,
                                       c_void_p, c_size_t, c_void_p]
    for name in EXPORTS:
        if name not in ("dmc_cache_workspace_bytes", "dmc_last_error", "dmc_train_workspace_bytes"):
            getattr(lib, name).restype = c_int32
    return lib


lib = _load()


def last_error() -> str:
    msg = lib.dmc_last_error()
    return msg.decode() if msg else ""


def check(status: int):
    if status != DMC_OK:
        raise DMCError(status, last_error())


def make_config(num_layers, batch, num_q_heads, num_kv_heads, head_dim, dtype="bf16",
                page_size=32, max_slots_per_seq=4096, num_pages=None, decision_bias=0.0,
                omega_src="lead", split_tile=0, max_prompt_len=0,
                decision_src="per_head", window=0) -> CacheConfig:
    """A dmc_cache_config; num_pages defaults to room for every unit at capacity.

    omega_src: 'lead' | 'group_mean' | 'uniform'; decision_src: 'per_head' |
    'shared_layer' (DMC-HardC); window: 0 (exact) or the window-grouping width."""
    units = num_layers * batch * num_kv_heads
    if num_pages is None:
        num_pages = units * -(-max_slots_per_seq // page_size)
    return CacheConfig(num_layers, batch, num_q_heads, num_kv_heads, head_dim,
                       DMC_FP32 if dtype in ("fp32", "float32") else DMC_BF16, page_size,
                       max_slots_per_seq, num_pages, decision_bias, OMEGA_SRC[omega_src],
                       split_tile, max_prompt_len, DECISION_SRC[decision_src], window)


def workspace_bytes(cfg: CacheConfig) -> int:
    n = lib.dmc_cache_workspace_bytes(ctypes.byref(cfg))
    if n == 0:
        raise DMCError(DMC_ERR_INVALID_ARG, last_error())
    return n


def _ptr(t):
    return None if t is None else c_void_p(t.data_ptr())


# -- argument validation ------------------------------------------------------
# The C ABI receives raw pointers and cannot see shapes, dtypes or devices, so
# everything the header requires of a tensor is checked here, before any call
# into the library.  Checks run in a fixed order (dtype, shape, layout,
# alignment, then device), so each rejection can be exercised with CPU tensors.

def _fail(msg):
    raise DMCError(DMC_ERR_INVALID_ARG, msg)


def cache_dtype(cfg):
    import torch
    return torch.float32 if cfg.dtype == DMC_FP32 else torch.bfloat16


def _check(name, t, dtype, shape=None, contiguous=True, align16=True,
           last_dim_contiguous=False, stride_mult=None):
    """Validate one tensor argument (not its device, see _on_device); shape
    entries of None match any size."""
    import torch
    if not isinstance(t, torch.Tensor):
        _fail(f"{name} must be a torch.Tensor")
    if t.dtype != dtype:
        _fail(f"{name} has dtype {t.dtype}, expected {dtype}")
    if shape is not None:
        if t.dim() != len(shape) or any(w is not None and g != w for g, w in zip(t.shape, shape)):
            want = "[" + ", ".join("*" if w is None else str(w) for w in shape) + "]"
            _fail(f"{name} has shape {list(t.shape)}, expected {want}")
    if contiguous and not t.is_contiguous():
        _fail(f"{name} must be contiguous")
    if last_dim_contiguous and t.dim() > 0 and t.shape[-1] > 1 and t.stride(-1) != 1:
        _fail(f"{name} must have a contiguous last dimension")
    if stride_mult and any(st % stride_mult for st in t.stride()[:-1]):
        _fail(f"{name} strides {tuple(t.stride())} must be multiples of {stride_mult} elements")
    if align16 and t.numel() > 0 and t.data_ptr() % 16:
        _fail(f"{name} must be 16-byte aligned")


def _on_device(device, **tensors):
    """Last check of every entry point: all tensors on the cache's device."""
    for name, t in tensors.items():
        if t is not None and t.device != device:
            _fail(f"{name} is on {t.device}, the cache is on {device}")


def check_decode_args(cfg, device, q, k, v, out, slot_index=None):
    """dmc_decode_step: q, out [B, Hq, d]; k, v [B, Hkv, d]; contiguous, cache
    dtype, 16-byte aligned; slot_index int32 [B, Hkv]."""
    import torch
    dt = cache_dtype(cfg)
    B, Hq, Hkv, d = cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    _check("q", q, dt, (B, Hq, d))
    _check("k", k, dt, (B, Hkv, d))
    _check("v", v, dt, (B, Hkv, d))
    _check("out", out, dt, (B, Hq, d))
    if slot_index is not None:
        _check("slot_index", slot_index, torch.int32, (B, Hkv), align16=False)
    for name, t in (("q", q), ("k", k), ("v", v)):
        if _overlap(out, t):
            _fail(f"out overlaps {name}")
    _on_device(device, q=q, k=k, v=v, out=out, slot_index=slot_index)


def _overlap(x, y):
    if x.numel() == 0 or y.numel() == 0:
        return False
    x0, x1 = x.data_ptr(), x.data_ptr() + x.numel() * x.element_size()
    y0, y1 = y.data_ptr(), y.data_ptr() + y.numel() * y.element_size()
    return x0 < y1 and y0 < x1


def check_prefill_args(cfg, device, k, v, q, n, prompt_lens=None, slot_index=None,
                       full_q=False, out=None):
    """dmc_prefill_compress / dmc_prefill_attend: k, v [B, >= n, Hkv, d] with a
    contiguous last dimension and strides that are multiples of 8 elements,
    16-byte aligned; q [B, >= n, Hq, d] likewise when every element is read
    (prompt attention, full_q), else [B, >= n, Hq] or [B, >= n, Hq, *] (only
    element 0 is read); out like q; prompt_lens int32 [B]; slot_index int32
    [B, Hkv, n] contiguous."""
    import torch
    dt = cache_dtype(cfg)
    B, Hq, Hkv, d = cfg.batch, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    maxn = cfg.max_prompt_len if cfg.max_prompt_len > 0 else cfg.max_slots_per_seq
    if not 0 <= n <= maxn:
        _fail(f"prompt length {n} outside [0, {maxn}]")
    for name, t in (("k", k), ("v", v)):
        _check(name, t, dt, (B, None, Hkv, d), contiguous=False, last_dim_contiguous=True,
               stride_mult=8)
        if t.shape[1] < n:
            _fail(f"{name} holds {t.shape[1]} tokens, fewer than n = {n}")
    if full_q:
        _check("q", q, dt, (B, None, Hq, d), contiguous=False, last_dim_contiguous=True,
               stride_mult=8)
    else:
        if q.dim() == 3:
            _check("q", q, dt, (B, None, Hq), contiguous=False, align16=False)
        else:
            _check("q", q, dt, (B, None, Hq, None), contiguous=False, align16=False)
    if q.shape[1] < n:
        _fail(f"q holds {q.shape[1]} tokens, fewer than n = {n}")
    if out is not None:
        _check("out", out, dt, (B, None, Hq, d), contiguous=False,
               last_dim_contiguous=True, stride_mult=8)
        if out.shape[1] < n:
            _fail(f"out holds {out.shape[1]} tokens, fewer than n = {n}")
        for name, t in (("q", q), ("k", k), ("v", v)):
            if _overlap(out, t):
                _fail(f"out overlaps {name}")
    if prompt_lens is not None:
        _check("prompt_lens", prompt_lens, torch.int32, (B,), align16=False)
    if slot_index is not None:
        _check("slot_index", slot_index, torch.int32, (B, Hkv, n), align16=False)
    _on_device(device, k=k, v=v, q=q, out=out, prompt_lens=prompt_lens, slot_index=slot_index)


def check_import_args(cfg, device, K, V, lengths, z):
    """dmc_cache_import: K, V [B, Hkv, dense_slots, d] contiguous cache dtype,
    16-byte aligned; lengths int32 [B, Hkv]; z float32 [B, Hkv]."""
    import torch
    dt = cache_dtype(cfg)
    B, Hkv, d = cfg.batch, cfg.num_kv_heads, cfg.head_dim
    _check("K", K, dt, (B, Hkv, None, d))
    _check("V", V, dt, (B, Hkv, K.shape[2], d))
    _check("lengths", lengths, torch.int32, (B, Hkv), align16=False)
    _check("z", z, torch.float32, (B, Hkv), align16=False)
    _on_device(device, K=K, V=V, lengths=lengths, z=z)


def check_train_args(cfg, device, q, k, v, noise, extra=()):
    """dmc_train_forward / dmc_train_backward: q-shaped [B, n, Hq, d] and
    k-shaped [B, n, Hkv, d] tensors contiguous in the config dtype and 16-byte
    aligned; noise and the per-token fp32 arrays [B, n, Hkv] contiguous.
    extra: (name, tensor, kind) with kind 'q', 'k' or 'tok' (None tensors skip)."""
    import torch
    dt = torch.float32 if cfg.dtype == DMC_FP32 else torch.bfloat16
    B, n, Hq, Hkv, d = cfg.batch, cfg.seq_len, cfg.num_q_heads, cfg.num_kv_heads, cfg.head_dim
    shapes = {"q": (dt, (B, n, Hq, d), True), "k": (dt, (B, n, Hkv, d), True),
              "tok": (torch.float32, (B, n, Hkv), False)}
    items = [("q", q, "q"), ("k", k, "k"), ("v", v, "k"), ("noise", noise, "tok"), *extra]
    for name, t, kind in items:
        if t is None:
            continue
        dtype, shape, a16 = shapes[kind]
        _check(name, t, dtype, shape, align16=a16)
    _on_device(device, **{name: t for name, t, _ in items})


def _stream(stream):
    import torch
    s = torch.cuda.current_stream() if stream is None else stream
    return c_void_p(s.cuda_stream)


def _cuda_device(device):
    import torch
    dev = torch.device(device)
    if dev.type == "cuda" and dev.index is None:
        dev = torch.device("cuda", torch.cuda.current_device())
    return dev


class DMCCache:
    """A paged DMC cache in one torch-allocated workspace on the current GPU.

    Thin wrapper over the C ABI.  The library checks pointers, alignment,
    strides, layer and prompt length; the shapes, dtypes, devices and layouts
    of the tensors, which it cannot see, are checked here before each call
    (check_*_args), raising DMCError.
    """

    def __init__(self, cfg: CacheConfig, device="cuda", stream=None):
        import torch
        self.cfg = cfg
        self.device = _cuda_device(device)
        self.dtype = torch.float32 if cfg.dtype == DMC_FP32 else torch.bfloat16
        self.G = cfg.num_q_heads // cfg.num_kv_heads
        nbytes = workspace_bytes(cfg)
        self.workspace = torch.empty(nbytes + 256, dtype=torch.uint8, device=self.device)
        base = self.workspace.data_ptr()
        self._ws_ptr = (base + 255) // 256 * 256
        self._ws_bytes = nbytes
        handle = c_void_p()
        check(lib.dmc_cache_alloc(ctypes.byref(cfg), c_void_p(self._ws_ptr), nbytes,
                                  _stream(stream), ctypes.byref(handle)))
        self.handle = handle

    def close(self):
        if getattr(self, "handle", None):
            lib.dmc_cache_free(self.handle)
            self.handle = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    # -- hot path -------------------------------------------------------------
    def decode_step(self, layer, q, k, v, out=None, slot_index=None, stream=None):
        """Algorithm 1 update + attention for one layer; returns out [B, Hq, d]."""
        if out is None:
            out = torch_empty_like(q)
        check_decode_args(self.cfg, self.device, q, k, v, out, slot_index)
        check(lib.dmc_decode_step(self.handle, layer, _ptr(q), _ptr(k), _ptr(v), _ptr(out),
                                  _ptr(slot_index), _stream(stream)))
        return out

    def decode_step_static(self, layer, q, k, v, out, slot_index=None, stream=None):
        """dmc_decode_step_static: as decode_step, with the split-K records in the
        library's static device scratch; allocates nothing (`out` is required)."""
        check_decode_args(self.cfg, self.device, q, k, v, out, slot_index)
        check(lib.dmc_decode_step_static(self.handle, layer, _ptr(q), _ptr(k), _ptr(v),
                                         _ptr(out), _ptr(slot_index), _stream(stream)))
        return out

    def prefill(self, layer, k, v, q, n=None, prompt_lens=None, slot_index=None, stream=None):
        """Compress a prompt: k, v [B, n, Hkv, d] (strided), q [B, n, Hq, (d)]."""
        n = k.shape[1] if n is None else n
        check_prefill_args(self.cfg, self.device, k, v, q, n, prompt_lens, slot_index)
        ks = (c_int64 * 3)(k.stride(0), k.stride(1), k.stride(2))
        vs = (c_int64 * 3)(v.stride(0), v.stride(1), v.stride(2))
        qs = (c_int64 * 3)(q.stride(0), q.stride(1), q.stride(2))
        check(lib.dmc_prefill_compress(self.handle, layer, _ptr(k), ks, _ptr(v), vs, _ptr(q), qs,
                                       n, _ptr(prompt_lens), _ptr(slot_index), _stream(stream)))

    def prefill_attend(self, layer, k, v, q, out=None, n=None, prompt_lens=None, slot_index=None,
                       stream=None):
        """Compress a prompt and attend every prompt query: k, v [B, n, Hkv, d],
        q [B, n, Hq, d] (strided, d contiguous); returns out [B, n, Hq, d]."""
        n = k.shape[1] if n is None else n
        if out is None:
            import torch
            out = torch.empty((q.shape[0], n, q.shape[2], q.shape[3]), dtype=q.dtype,
                              device=q.device)
        check_prefill_args(self.cfg, self.device, k, v, q, n, prompt_lens, slot_index,
                           full_q=True, out=out)
        ks = (c_int64 * 3)(k.stride(0), k.stride(1), k.stride(2))
        vs = (c_int64 * 3)(v.stride(0), v.stride(1), v.stride(2))
        qs = (c_int64 * 3)(q.stride(0), q.stride(1), q.stride(2))
        os_ = (c_int64 * 3)(out.stride(0), out.stride(1), out.stride(2))
        check(lib.dmc_prefill_attend(self.handle, layer, _ptr(k), ks, _ptr(v), vs, _ptr(q), qs, n,
                                     _ptr(prompt_lens), _ptr(out), os_, _ptr(slot_index),
                                     _stream(stream)))
        return out

    # -- accessors --------------------------------------------------------------
    def lengths(self, layer, stream=None):
        import torch
        out = torch.empty((self.cfg.batch, self.cfg.num_kv_heads), dtype=torch.int32,
                          device=self.device)
        check(lib.dmc_cache_lengths(self.handle, layer, _ptr(out), _stream(stream)))
        return out

    def export(self, layer, dense_slots=None, stream=None):
        import torch
        dense_slots = self.cfg.max_slots_per_seq if dense_slots is None else dense_slots
        shape = (self.cfg.batch, self.cfg.num_kv_heads, dense_slots, self.cfg.head_dim)
        K = torch.empty(shape, dtype=self.dtype, device=self.device)
        V = torch.empty(shape, dtype=self.dtype, device=self.device)
        z = torch.empty(shape[:2], dtype=torch.float32, device=self.device)
        check(lib.dmc_cache_export(self.handle, layer, _ptr(K), _ptr(V), dense_slots, _ptr(z),
                                   _stream(stream)))
        return K, V, z

    def import_(self, layer, K, V, lengths, z, stream=None):
        check_import_args(self.cfg, self.device, K, V, lengths, z)
        check(lib.dmc_cache_import(self.handle, layer, _ptr(K), _ptr(V), K.shape[2],
                                   _ptr(lengths), _ptr(z), _stream(stream)))

    def check(self, stream=None):
        check(lib.dmc_cache_check(self.handle, _stream(stream)))

    def status(self, stream=None) -> int:
        return lib.dmc_cache_check(self.handle, _stream(stream))

    def pages_used(self, stream=None) -> int:
        n = c_int64()
        check(lib.dmc_cache_pages_used(self.handle, ctypes.byref(n), _stream(stream)))
        return n.value

    def reset(self, stream=None):
        check(lib.dmc_cache_reset(self.handle, _stream(stream)))


def torch_empty_like(t):
    import torch
    return torch.empty_like(t, memory_format=torch.contiguous_format)


def make_train_config(batch, seq_len, num_q_heads, num_kv_heads, head_dim, dtype="bf16",
                      decision_bias=5.0, temperature=0.1, window=12, omega_src="lead") -> TrainConfig:
    """A dmc_train_config (defaults: the paper's c = 5, tau = 0.1, w = 12)."""
    return TrainConfig(batch, seq_len, num_q_heads, num_kv_heads, head_dim,
                       DMC_FP32 if dtype in ("fp32", "float32") else DMC_BF16, decision_bias,
                       temperature, window, OMEGA_SRC[omega_src])


class DMCTrainer:
    """Training-time DMC attention of one layer shape (forward + backward)
    with its workspace in one torch allocation on the current GPU."""

    def __init__(self, cfg: TrainConfig, device="cuda"):
        import torch
        self.cfg = cfg
        n = lib.dmc_train_workspace_bytes(ctypes.byref(cfg))
        if n == 0:
            raise DMCError(DMC_ERR_INVALID_ARG, last_error())
        self.device = _cuda_device(device)
        self.workspace = torch.empty(n + 256, dtype=torch.uint8, device=self.device)
        self._ws = c_void_p((self.workspace.data_ptr() + 255) // 256 * 256)
        self._ws_bytes = n

    def forward(self, q, k, v, noise, out=None, alpha=None, stream=None):
        """out [B, n, Hq, d] (and alpha [B, n, Hkv] fp32 if given)."""
        if out is None:
            out = torch_empty_like(q)
        check_train_args(self.cfg, self.device, q, k, v, noise,
                         (("out", out, "q"), ("alpha", alpha, "tok")))
        check(lib.dmc_train_forward(ctypes.byref(self.cfg), _ptr(q), _ptr(k), _ptr(v), _ptr(noise),
                                    _ptr(out), _ptr(alpha), self._ws, self._ws_bytes,
                                    _stream(stream)))
        return out

    def backward(self, q, k, v, noise, out, dout, dalpha=None, dq=None, dk=None, dv=None,
                 stream=None):
        """(dq, dk, dv) of sum(out * dout) + sum(alpha * dalpha)."""
        dq = torch_empty_like(q) if dq is None else dq
        dk = torch_empty_like(k) if dk is None else dk
        dv = torch_empty_like(v) if dv is None else dv
        check_train_args(self.cfg, self.device, q, k, v, noise,
                         (("out", out, "q"), ("dout", dout, "q"), ("dalpha", dalpha, "tok"),
                          ("dq", dq, "q"), ("dk", dk, "k"), ("dv", dv, "k")))
        check(lib.dmc_train_backward(ctypes.byref(self.cfg), _ptr(q), _ptr(k), _ptr(v),
                                     _ptr(noise), _ptr(out), _ptr(dout), _ptr(dalpha), _ptr(dq),
                                     _ptr(dk), _ptr(dv), self._ws, self._ws_bytes,
                                     _stream(stream)))
        return dq, dk, dv
