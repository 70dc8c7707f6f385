"""The C ABI on the CPU: symbols, validation codes, sizes, argument errors.

Nothing here launches a kernel; device entry points are only called with
arguments the host checks reject before anything is enqueued.
"""

import ctypes
import os
import re
import shutil
import subprocess

import pytest

from paper_2601_22379_amd import spla

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "spla.h")


def declared_functions():
    text = open(HEADER).read()
    return sorted(set(re.findall(r"^\s*(?:const char\*|int32_t)\s+(spla_\w+)\(", text, re.M)))


def test_binding_lists_every_declared_function():
    assert sorted(spla.EXPORTS) == declared_functions()


@pytest.mark.parametrize("path", [spla.LIB_PATH, spla.HOST_LIB_PATH])
def test_library_exports_every_declared_symbol(path):
    if not os.path.exists(path):
        pytest.skip("library not built")
    out = subprocess.run(["nm", "-D", "--defined-only", path], capture_output=True, text=True,
                         check=True).stdout
    syms = set(re.findall(r"\bT (spla_\w+)", out))
    want = declared_functions() if path == spla.LIB_PATH else sorted(spla.HOST_EXPORTS)
    assert set(want) <= syms


def test_hip_library_loads_and_resolves_symbols():
    lib = spla.lib()
    for s in spla.EXPORTS:
        assert getattr(lib, s) is not None


def _cfg(**kw):
    base = dict(batch=4, n_q_heads=32, n_kv_heads=8, head_dim=128, block_size=64, top_k=32,
                max_seq_len=131072, dtype="bf16")
    base.update(kw)
    return spla.make_config(**base)


@pytest.mark.parametrize("libname", ["hip", "host"])
@pytest.mark.parametrize("kw,want", [
    ({}, 0),
    (dict(n_q_heads=30), -1),
    (dict(n_q_heads=8 * 17), -2),
    (dict(head_dim=96), -2),
    (dict(block_size=16, max_seq_len=1024), -2),
    (dict(top_k=4), -1),
    (dict(top_k=257), -3),
    (dict(max_seq_len=1000), -1),
    (dict(max_seq_len=64 * 32769), -3),
    (dict(dtype=5), -1),
    (dict(rms_eps=float("nan")), -1),
    (dict(flags=16), -1),
    (dict(n_sink=0, n_local=0, top_k=1), 0),
    (dict(n_q_heads=40, n_kv_heads=8), 0),
    (dict(sel_window=32, sel_stride=16), 0),                   # the paper's windows
    (dict(sel_window=64, sel_stride=32), 0),
    (dict(sel_window=16, sel_stride=16), 0),
    (dict(sel_window=32, sel_stride=0), -1),
    (dict(sel_window=8, sel_stride=16), -1),
    (dict(sel_window=48, sel_stride=24), -2),                  # stride does not divide B
    (dict(sel_window=40, sel_stride=16), -2),                  # window not a multiple
    (dict(sel_window=80, sel_stride=16), -2),                  # more than 4 strides
    (dict(sel_window=32, sel_stride=16, max_seq_len=16 * 16385 // 64 * 64 + 64), -3),
    (dict(kv_pages=100), 0),                                   # paged KV pool
    (dict(kv_pages=-1), -1),
    (dict(kv_pages=(1 << 24) + 1), -3),
])
def test_validate_codes(libname, kw, want):
    lib = spla.lib() if libname == "hip" else spla.host_lib()
    assert spla.validate(_cfg(**kw), lib) == want


def test_sizes_follow_documented_layout():
    c = _cfg()
    b = spla.cache_bytes(c)
    assert b[0] == 4 * 8 * 131072 * 128 * 2
    assert b[1] == 4 * 8 * 2048 * 128 * 64 * 2
    assert b[2] == 4 * 8 * 32 * 2 * 32 * 64 * 4 * 4
    assert b[3] == 4 * 8 * 128 * 128 * 4 and b[4] == 4 * 8 * 128 * 4 and b[5] == 16
    assert spla.workspace_bytes(c) % 256 == 0
    assert spla.append_workspace_bytes(c, 1) > 0
    # strided selection: one statistics entry per window (131072 / 16 = 8192)
    w = spla.cache_bytes(_cfg(sel_window=32, sel_stride=16))
    assert w[2] == 4 * 8 * 128 * 2 * 32 * 64 * 4 * 4
    assert w[:2] == b[:2] and w[3:] == b[3:]
    # paged pool: one page of B rows per KV head and page
    pg = spla.cache_bytes(_cfg(kv_pages=1000))
    assert pg[0] == pg[1] == 1000 * 8 * 64 * 128 * 2
    assert pg[2:] == b[2:]


def test_device_calls_reject_bad_arguments_before_launch():
    lib = spla.lib()
    c = _cfg()
    null_cache = spla.SplaCacheStruct()
    assert lib.spla_decode(ctypes.byref(c), ctypes.byref(null_cache), None, None, None, None,
                           None, 0, None) == -1
    assert lib.spla_decode(None, None, None, None, None, None, None, 0, None) == -1
    fake = spla.SplaCacheStruct(*([256] * 6), None)
    # valid-looking cache, missing workspace
    assert lib.spla_decode(ctypes.byref(c), ctypes.byref(fake), 256, 256, 512, None, None, 0,
                           None) == -4
    # misaligned workspace
    assert lib.spla_decode(ctypes.byref(c), ctypes.byref(fake), 256, 256, 512, None, 8,
                           1 << 40, None) == -4
    # prefill: a negative token count, and missing token rows, are rejected;
    # no tokens is a no-op
    assert lib.spla_prefill(ctypes.byref(c), ctypes.byref(fake), -1, 256, 256, 256, 256, 512,
                            None, 256, 1 << 40, None) == -1
    assert lib.spla_prefill(ctypes.byref(c), ctypes.byref(fake), 3, None, 256, 256, 256, 512,
                            None, 256, 1 << 40, None) == -1
    assert lib.spla_prefill(ctypes.byref(c), ctypes.byref(fake), 0, None, None, 256, 256, 512,
                            None, 256, 1 << 40, None) == 0
    # a paged pool needs its block table, and a contiguous cache has none
    paged = _cfg(kv_pages=64)
    assert lib.spla_decode(ctypes.byref(paged), ctypes.byref(fake), 256, 256, 512, None, 256,
                           1 << 40, None) == -1
    tabled = spla.SplaCacheStruct(*([256] * 6), None, 256)
    assert lib.spla_decode(ctypes.byref(c), ctypes.byref(tabled), 256, 256, 512, None, 256,
                           1 << 40, None) == -1
    # out aliasing q
    assert lib.spla_decode(ctypes.byref(c), ctypes.byref(fake), 256, 256, 256, None, 256,
                           1 << 40, None) == -1
    assert lib.spla_append(ctypes.byref(c), ctypes.byref(fake), 256, 256, -1, None, None, 0,
                           None) == -1
    assert lib.spla_append(ctypes.byref(c), ctypes.byref(fake), 256, 256, 131073, None, None, 0,
                           None) == -3
    assert lib.spla_append(ctypes.byref(c), ctypes.byref(fake), 256, 256, 16, None, None, 0,
                           None) == -4
    bad = _cfg(top_k=2)
    assert lib.spla_step(ctypes.byref(bad), ctypes.byref(fake), 256, 256, 256, 256, 512, None,
                         256, 1 << 40, None) == -1
    assert lib.spla_reset(ctypes.byref(bad), ctypes.byref(fake), None) == -1


def test_binding_fails_loudly_without_library(monkeypatch, tmp_path):
    monkeypatch.setattr(spla, "LIB_PATH", str(tmp_path / "missing.so"))
    monkeypatch.setattr(spla, "_LIB", None)
    with pytest.raises(ImportError):
        spla.lib()


@pytest.mark.skipif(shutil.which("g++") is None, reason="no g++")
def test_header_and_host_code_under_sanitizers(tmp_path):
    exe = tmp_path / "abi_check"
    cmd = ["g++", "-std=c++17", "-x", "c++", os.path.join(ROOT, "tests", "native", "abi_check.c"),
           "-x", "c++", os.path.join(ROOT, "paper_2601_22379_amd", "csrc", "spla_host.cpp"),
           "-I", os.path.join(ROOT, "include"), "-fsanitize=address,undefined",
           "-fno-sanitize-recover=all", "-g", "-o", str(exe)]
    subprocess.run(cmd, check=True, capture_output=True)
    r = subprocess.run([str(exe)], capture_output=True, text=True)
    assert r.returncode == 0, r.stdout + r.stderr
    assert "ALL OK" in r.stdout
    # the header is valid C too
    r2 = subprocess.run(["gcc", "-std=c99", "-fsyntax-only", "-I", os.path.join(ROOT, "include"),
                         os.path.join(ROOT, "tests", "native", "abi_check.c")],
                        capture_output=True, text=True)
    assert r2.returncode == 0, r2.stderr


@pytest.mark.parametrize("libname", ["hip", "host"])
@pytest.mark.parametrize("kw,single", [
    ({}, True),                                              # the 128K benchmark shape
    (dict(n_q_heads=40, n_kv_heads=8), True),                # G = 5
    (dict(block_size=128, max_seq_len=65536), True),
    (dict(max_seq_len=64 * 8192), True),                     # largest single-launch block count
    (dict(max_seq_len=64 * 8193), False),
    (dict(n_q_heads=64, n_kv_heads=8), False),               # G = 8
    (dict(head_dim=64), False),
    (dict(dtype="f32"), False),
    (dict(flags=spla.FLAG_SEPARATE_KERNELS), False),
    (dict(sel_window=32, sel_stride=16), False),             # strided selection
    (dict(kv_pages=4096), True),                             # paged KV pool
    (dict(batch=16), True),                                  # 128 units: the limit
    (dict(batch=17), False),
    (dict(batch=64, block_size=128, max_seq_len=65536, top_k=16), False),  # high batch
])
def test_decode_phase_mask(libname, kw, single):
    lib = spla.lib() if libname == "hip" else spla.host_lib()
    got = spla.decode_phases(_cfg(**kw), lib)
    assert got == (["decode"] if single else ["score", "select", "sparse", "merge"])



def test_noalloc_rejects_before_launch():
    """spla_decode_noalloc checks its arguments and the scratch size on the
    host; a shape whose workspace exceeds the scratch is rejected."""
    lib = spla.lib()
    fake = spla.SplaCacheStruct(*([256] * 6), None)
    big = spla.make_config(128, 32, 8, 128, 64, 256, 1 << 21)
    assert spla.workspace_bytes(big) > 64 << 20
    assert lib.spla_decode_noalloc(ctypes.byref(big), ctypes.byref(fake), 256, 256, 512, None,
                                   None) == -4
    c = _cfg()
    assert lib.spla_decode_noalloc(ctypes.byref(c), ctypes.byref(fake), 256, 256, 256, None,
                                   None) == -1
    assert lib.spla_decode_noalloc(ctypes.byref(c), None, 256, 256, 512, None, None) == -1
