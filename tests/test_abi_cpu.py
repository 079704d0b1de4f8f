"""The C ABI without a GPU: the library loads, exports every symbol the
header declares, sizes workspaces, and rejects invalid arguments before any
HIP call."""
import ctypes
import os
import re
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "dmc.h")


def _declared():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(dmc_[a-z_]+)\s*\(", text)))


@pytest.fixture(scope="module")
def P():
    import paper_2403_09636_amd as P
    return P


def test_header_symbols_exported(P):
    names = _declared()
    assert names, "no declarations found"
    assert sorted(P.EXPORTS) == names
    lib = ctypes.CDLL(P.LIB_PATH)
    for n in names:
        assert hasattr(lib, n), f"{n} not exported"
    out = subprocess.run(["nm", "-D", "--defined-only", P.LIB_PATH], capture_output=True,
                         text=True).stdout
    exported = set(re.findall(r"\bT (dmc_\w+)", out))
    assert set(names) <= exported


def test_config_struct_matches_header(P):
    text = open(HEADER).read()
    body = re.search(r"typedef struct dmc_cache_config \{(.*?)\} dmc_cache_config;", text, re.S)
    fields = re.findall(r"^\s*(?:int32_t|int64_t|float)\s+([a-z_, ]+);", body.group(1), re.M)
    names = [f.strip() for grp in fields for f in grp.split(",")]
    assert names == [f[0] for f in P.CacheConfig._fields_]
    assert ctypes.sizeof(P.CacheConfig) == 64


def test_workspace_bytes(P):
    cfg = P.make_config(32, 64, 32, 32, 128, max_slots_per_seq=4160, num_pages=2_200_000)
    n = P.workspace_bytes(cfg)
    pool = 2_200_000 * 2 * 32 * 128 * 2
    assert pool < n < pool * 1.02
    cfg2 = P.make_config(32, 64, 32, 32, 128, max_slots_per_seq=4160, num_pages=2_200_001)
    assert P.workspace_bytes(cfg2) > n


@pytest.mark.parametrize("field,value,msg", [
    ("num_kv_heads", 3, "multiple"), ("head_dim", 96, "head_dim"), ("page_size", 48, "page_size"),
    ("page_size", 4, "page_size"), ("dtype", 7, "dtype"), ("num_pages", 0, "num_pages"),
    ("num_pages", 1 << 31, "num_pages"), ("max_slots_per_seq", 0, "max_slots"),
    ("omega_src", 5, "omega"), ("split_tile", -1, "split_tile"), ("max_prompt_len", 99999, "prompt"),
    ("decision_src", 2, "decision_src"), ("window", -1, "window"), ("window", 65, "window"),
    ("page_size", 131072, "page_size"),
    ("batch", 0, ">= 1"), ("num_q_heads", 48, "group"),
])
def test_invalid_config(P, field, value, msg):
    cfg = P.make_config(2, 4, 16, 4, 128, max_slots_per_seq=1024)
    setattr(cfg, field, value)
    assert P.binding.lib.dmc_cache_workspace_bytes(ctypes.byref(cfg)) == 0
    assert msg in P.binding.last_error()


def test_too_many_units_for_decode_table(P):
    """Layers whose slot-space table would not fit in LDS keep every g-th entry
    (g up to 64); beyond that, and beyond 2^20 units, they are refused."""
    assert P.binding.lib.dmc_cache_workspace_bytes(ctypes.byref(P.make_config(1, 4096, 8, 8, 128))) > 0
    assert P.binding.lib.dmc_cache_workspace_bytes(ctypes.byref(P.make_config(1, 512, 32, 32, 128))) > 0
    huge = P.make_config(1, 1 << 18, 8, 8, 64, max_slots_per_seq=8, num_pages=1024)   # 2^21 units
    assert P.binding.lib.dmc_cache_workspace_bytes(ctypes.byref(huge)) == 0
    assert "units" in P.binding.last_error()


def test_windowed_cache_needs_the_full_table(P):
    big = P.make_config(1, 512, 32, 32, 128, window=12)       # 16384 units: over 64 KB with the
                                                              # windowed means beside the table
    assert P.binding.lib.dmc_cache_workspace_bytes(ctypes.byref(big)) == 0
    assert "units" in P.binding.last_error()
    assert P.binding.lib.dmc_cache_workspace_bytes(
        ctypes.byref(P.make_config(1, 470, 32, 32, 128, window=12))) > 0


def test_matrix_core_cache_unit_limit(P):
    """bf16 grouped-query caches (G >= 4, 32-slot pages) decode with a 128 KB
    chunk ring in LDS at d = 128; the slot-space table beside it holds 8176
    entries, i.e. up to 8175 units with one entry each, and up to 64 times
    that with grouped entries.  fp32 caches run the vector kernel."""
    for batch in (1021, 1024, 65400):                         # 8168, 8192, 523200 units
        cfg = P.make_config(1, batch, 64, 8, 128, "bf16", max_slots_per_seq=8, num_pages=1024)
        assert P.binding.lib.dmc_cache_workspace_bytes(ctypes.byref(cfg)) > 0, batch
    big = P.make_config(1, 65401, 64, 8, 128, "bf16", max_slots_per_seq=8, num_pages=1024)
    assert P.binding.lib.dmc_cache_workspace_bytes(ctypes.byref(big)) == 0
    assert "units" in P.binding.last_error()
    vec = P.make_config(1, 65401, 64, 8, 128, "fp32", max_slots_per_seq=8, num_pages=1024)
    assert P.binding.lib.dmc_cache_workspace_bytes(ctypes.byref(vec)) > 0


def test_alloc_rejects_before_hip(P):
    lib = P.binding.lib
    cfg = P.make_config(1, 2, 2, 2, 64, max_slots_per_seq=64)
    out = ctypes.c_void_p()
    n = P.workspace_bytes(cfg)
    assert lib.dmc_cache_alloc(ctypes.byref(cfg), None, n, None, ctypes.byref(out)) == 1
    assert "workspace" in P.binding.last_error()
    assert lib.dmc_cache_alloc(ctypes.byref(cfg), ctypes.c_void_p(0x1008), n, None,
                               ctypes.byref(out)) == 1
    assert "aligned" in P.binding.last_error()
    assert lib.dmc_cache_alloc(ctypes.byref(cfg), ctypes.c_void_p(0x1000), n - 1, None,
                               ctypes.byref(out)) == 1
    assert "needs" in P.binding.last_error()
    assert lib.dmc_cache_alloc(ctypes.byref(cfg), ctypes.c_void_p(0x1000), n, None, None) == 1
    bad = P.make_config(1, 2, 2, 2, 65)
    assert lib.dmc_cache_alloc(ctypes.byref(bad), ctypes.c_void_p(0x1000), n, None,
                               ctypes.byref(out)) == 2
    assert out.value is None


def test_entry_points_reject_null_cache(P):
    lib = P.binding.lib
    s = (ctypes.c_int64 * 3)(0, 0, 0)
    i64 = ctypes.c_int64()
    calls = {
        "dmc_decode_step": lambda: lib.dmc_decode_step(None, 0, None, None, None, None, None, None),
        "dmc_prefill_compress": lambda: lib.dmc_prefill_compress(None, 0, None, s, None, s, None,
                                                                 s, 0, None, None, None),
        "dmc_prefill_attend": lambda: lib.dmc_prefill_attend(None, 0, None, s, None, s, None, s,
                                                             0, None, None, s, None, None),
        "dmc_cache_lengths": lambda: lib.dmc_cache_lengths(None, 0, None, None),
        "dmc_cache_export": lambda: lib.dmc_cache_export(None, 0, None, None, 0, None, None),
        "dmc_cache_import": lambda: lib.dmc_cache_import(None, 0, None, None, 0, None, None, None),
        "dmc_cache_check": lambda: lib.dmc_cache_check(None, None),
        "dmc_cache_pages_used": lambda: lib.dmc_cache_pages_used(None, ctypes.byref(i64), None),
        "dmc_cache_reset": lambda: lib.dmc_cache_reset(None, None),
        "dmc_cache_free": lambda: lib.dmc_cache_free(None),
    }
    for name, call in calls.items():
        assert call() == 1, name
        assert "NULL" in P.binding.last_error(), name


def test_product_path_never_imports_oracle():
    pkg = os.path.join(ROOT, "paper_2403_09636_amd")
    for dirpath, _, files in os.walk(pkg):
        for f in files:
            if f.endswith((".py", ".cpp", ".hip", ".h")):
                text = open(os.path.join(dirpath, f)).read()
                assert not re.search(r"^\s*(from|import)\s+oracle", text, re.M), f
                assert "dmc_oracle" not in text, f


def test_missing_library_fails_loudly(tmp_path):
    dst = tmp_path / "paper_2403_09636_amd"
    shutil.copytree(os.path.join(ROOT, "paper_2403_09636_amd"), dst,
                    ignore=shutil.ignore_patterns("*.so", "__pycache__", "csrc"))
    res = subprocess.run([sys.executable, "-c", "import paper_2403_09636_amd"], cwd=tmp_path,
                         capture_output=True, text=True)
    assert res.returncode != 0 and "not built" in res.stderr


def test_build_runs_on_a_tree_without_the_library(tmp_path):
    """build() must reach the compiler on a fresh checkout, where no libdmc.so exists yet.

    A stand-in hipcc writes an empty file, so the build "succeeds" and only the final import
    (loading that empty file) fails: "built" must be printed before it.
    """
    for item in ("__graft_entry__.py", "include", "paper_2403_09636_amd"):
        src = os.path.join(ROOT, item)
        if os.path.isdir(src):
            shutil.copytree(src, tmp_path / item,
                            ignore=shutil.ignore_patterns("*.so", "__pycache__"))
        else:
            shutil.copy(src, tmp_path / item)
    fake = tmp_path / "rocm" / "bin"
    fake.mkdir(parents=True)
    (fake / "hipcc").write_text('#!/bin/sh\nwhile [ "$1" != "-o" ]; do shift; done\n: > "$2"\n')
    (fake / "hipcc").chmod(0o755)
    env = dict(os.environ, ROCM_PATH=str(tmp_path / "rocm"))
    res = subprocess.run([sys.executable, "-c", "import __graft_entry__ as g; g.build()"],
                         cwd=tmp_path, env=env, capture_output=True, text=True)
    assert "built " in res.stdout, res.stdout + res.stderr


def test_train_config_struct_matches_header(P):
    text = open(HEADER).read()
    body = re.search(r"typedef struct dmc_train_config \{(.*?)\} dmc_train_config;", text, re.S)
    fields = re.findall(r"^\s*(?:int32_t|int64_t|float)\s+([a-z_, ]+);", body.group(1), re.M)
    names = [f.strip() for grp in fields for f in grp.split(",")]
    assert names == [f[0] for f in P.TrainConfig._fields_]
    assert ctypes.sizeof(P.TrainConfig) == 40


@pytest.mark.parametrize("field,value,msg", [
    ("num_kv_heads", 3, "multiple"), ("head_dim", 96, "head_dim"), ("dtype", 9, "dtype"),
    ("temperature", 0.0, "temperature"), ("temperature", -1.0, "temperature"),
    ("window", 0, "window"), ("window", 65, "window"), ("omega_src", 1, "omega_src"),
    ("seq_len", 0, ">= 1"), ("num_q_heads", 24, "group"),
])
def test_invalid_train_config(P, field, value, msg):
    cfg = P.make_train_config(2, 128, 16, 4, 128)
    assert P.binding.lib.dmc_train_workspace_bytes(ctypes.byref(cfg)) > 0
    setattr(cfg, field, value)
    assert P.binding.lib.dmc_train_workspace_bytes(ctypes.byref(cfg)) == 0
    assert msg in P.binding.last_error()


def test_train_entry_points_reject_before_hip(P):
    lib = P.binding.lib
    cfg = P.make_train_config(1, 64, 4, 2, 64, window=12)
    n = lib.dmc_train_workspace_bytes(ctypes.byref(cfg))
    a = ctypes.c_void_p(0x1000)
    ws = ctypes.c_void_p(0x10000)
    assert lib.dmc_train_forward(ctypes.byref(cfg), None, a, a, a, a, None, ws, n, None) == 1
    assert "NULL" in P.binding.last_error()
    assert lib.dmc_train_forward(ctypes.byref(cfg), a, a, a, a, a, None, ws, n - 1, None) == 1
    assert "needs" in P.binding.last_error()
    assert lib.dmc_train_forward(ctypes.byref(cfg), ctypes.c_void_p(0x1008), a, a, a, a, None, ws,
                                 n, None) == 1
    assert "aligned" in P.binding.last_error()
    assert lib.dmc_train_backward(ctypes.byref(cfg), a, a, a, a, a, a, None, None, a, a, ws, n,
                                  None) == 1
    assert "NULL" in P.binding.last_error()
    assert lib.dmc_train_backward(None, a, a, a, a, a, a, None, a, a, a, ws, n, None) == 1
