"""CPU-only checks of the C ABI: the library loads, exports every symbol the
header declares, and rejects every malformed input on the host with the
documented status before touching a device."""
import os
import re
import subprocess

import numpy as np
import pytest

import paper_2606_16264_amd as mx
import workload as wl
from helpers import mx_batch, mx_cfg, mx_shape

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADER = os.path.join(ROOT, "include", "mx.h")


def declared_functions():
    text = open(HEADER).read()
    text = re.sub(r"/\*.*?\*/", "", text, flags=re.S)
    return sorted(set(re.findall(r"\b(mx_[a-z_0-9]+)\s*\(", text)))


def test_header_symbols_exported():
    names = declared_functions()
    assert "mx_layer_step" in names and "mx_paged_attn" in names and "mx_kv_append" in names
    out = subprocess.run(["nm", "-D", "--defined-only", mx.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (mx_[a-z_0-9]+)", out))
    missing = [n for n in names if n not in exported]
    assert not missing, f"declared but not exported: {missing}"
    assert sorted(mx.EXPORTED) == names
    for n in names:
        assert hasattr(mx.lib(), n)


def test_status_strings():
    assert mx.lib().mx_status_str(0).decode() == "MX_OK"
    assert mx.lib().mx_status_str(2).decode() == "MX_ERR_NO_SPACE"
    assert mx.mx_version() >> 16 == 1


def shape64(pool=64, nq=4, nkv=4, d=64):
    return mx.attn_shape(nq, nkv, d, pool)


def one(phase, n_new, ctx, pages):
    return mx.Batch([phase], [n_new], [ctx], [pages])


@pytest.mark.parametrize("batch,status", [
    (one(7, 1, 5, [0]), mx.MX_ERR_INVALID),                    # bad phase
    (one(mx.MX_PREFILL, 0, 0, [0]), mx.MX_ERR_INVALID),        # n_new = 0
    (one(mx.MX_DECODE, 2, 5, [0]), mx.MX_ERR_INVALID),         # decode with 2 tokens
    (one(mx.MX_DECODE, 1, 0, [0]), mx.MX_ERR_INVALID),         # decode without context
    (one(mx.MX_PREFILL, 3, -1, [0]), mx.MX_ERR_INVALID),       # negative context
    (one(mx.MX_PREFILL, 2, 15, [3]), mx.MX_ERR_NO_SPACE),      # position 16 needs a 2nd page
    (one(mx.MX_DECODE, 1, 16, [1]), mx.MX_ERR_NO_SPACE),       # decode at a page boundary
    (one(mx.MX_PREFILL, 4, 0, [64]), mx.MX_ERR_INVALID),       # page id out of range
    (one(mx.MX_PREFILL, 4, 0, [-1]), mx.MX_ERR_INVALID),       # negative page id
    (mx.Batch([0, 1], [3, 1], [0, 2], [[5], [5]]), mx.MX_ERR_INVALID),  # same slot written twice
])
def test_validation_errors(batch, status):
    assert mx.mx_batch_validate(batch, shape64()) == status
    assert mx.last_error() != ""


def test_validation_accepts_shared_prefix_and_boundaries():
    # two decodes reading the same (shared, read-only) first page, writing distinct slots
    b = mx.Batch([1, 1, 0], [1, 1, 16], [16, 17, 0], [[2, 3], [2, 4], [9]])
    assert mx.mx_batch_validate(b, shape64()) == mx.MX_OK
    assert mx.mx_batch_validate(mx.Batch([], [], [], []), shape64()) == mx.MX_OK


@pytest.mark.parametrize("shape,status", [
    (mx.attn_shape(4, 3, 64, 64), mx.MX_ERR_INVALID),      # nq % nkv != 0
    (mx.attn_shape(4, 4, 96, 64), mx.MX_ERR_UNSUPPORTED),  # head_dim
    (mx.attn_shape(4, 4, 64, 64, page_size=32), mx.MX_ERR_UNSUPPORTED),
    (mx.attn_shape(0, 4, 64, 64), mx.MX_ERR_INVALID),
    (mx.attn_shape(4, 4, 64, 0), mx.MX_ERR_INVALID),
])
def test_shape_errors(shape, status):
    assert mx.mx_batch_validate(one(0, 4, 0, [1]), shape) == status


def test_errors_precede_any_device_work():
    """On this GPU-less host any HIP call fails with MX_ERR_HIP, so an entry
    point that returns its own validation status has enqueued nothing."""
    cfg = wl.CONFIGS["c1"]
    c = mx_cfg(mx, cfg, 64)
    bad = one(mx.MX_PREFILL, 2, 15, [3])
    fake = type("T", (), {"data_ptr": lambda self: 0x1000, "numel": lambda self: 1 << 30,
                          "element_size": lambda self: 1})()
    st = mx.lib().mx_layer_step(bad.ptr, mx.ctypes.byref(c), 0x1000, 0x2000, 0x3000, 0x4000,
                                0x5000, 0x6000, 1 << 30, None)
    assert st == mx.MX_ERR_NO_SPACE
    st = mx.lib().mx_paged_attn(bad.ptr, mx.ctypes.byref(c.attn), 0x1000, 0x2000, 0x3000,
                                0x4000, 0x6000, 1 << 30, None)
    assert st == mx.MX_ERR_NO_SPACE
    good = one(mx.MX_PREFILL, 4, 0, [1])
    st = mx.lib().mx_kv_append(good.ptr, mx.ctypes.byref(c.attn), None, 0x2000, 0x3000, 0x4000,
                               0x6000, 1 << 30, None)
    assert st == mx.MX_ERR_NULL
    st = mx.lib().mx_layer_step(good.ptr, mx.ctypes.byref(c), 0x1000, 0x2000, 0x3000, 0x4000,
                                0x5000, 0x6000, 16, None)
    assert st == mx.MX_ERR_TOO_LARGE
    st = mx.lib().mx_layer_step(good.ptr, mx.ctypes.byref(c), 0x1000, 0x2000, 0x2000, 0x4000,
                                0x5000, 0x6000, 1 << 30, None)
    assert st == mx.MX_ERR_INVALID     # y aliases x
    # an empty batch is a no-op that touches nothing
    empty = mx.Batch([], [], [], [])
    st = mx.lib().mx_layer_step(empty.ptr, mx.ctypes.byref(c), 0, 0, 0, 0, 0, 0, 0, None)
    assert st == mx.MX_OK
    del fake


def test_cfg_errors():
    c = mx.layer_cfg(250, 1024, 4, 4, 64, 64)
    assert mx.lib().mx_packed_weights_bytes(mx.ctypes.byref(c)) == 0
    c = mx.layer_cfg(256, 1000, 4, 4, 64, 64)
    assert mx.lib().mx_packed_weights_bytes(mx.ctypes.byref(c)) == 0


@pytest.mark.parametrize("key,P", [("c1", 128), ("c2", 512), ("c3", 4096), ("c4", 2048),
                                   ("c5", 8192)])
def test_workspace_bound_covers_batch(key, P):
    cfg = wl.CONFIGS[key]
    b = wl.make_batch(key, P)
    c = mx_cfg(mx, cfg, b.pool_pages)
    need = mx.mx_workspace_bytes_for(mx_batch(mx, b), cfg=c)
    bound = mx.mx_workspace_bytes(c, None, b.T, b.R, int(sum(len(t) for t in b.page_tables)))
    assert 0 < need <= bound
    need_attn = mx.mx_workspace_bytes_for(mx_batch(mx, b), shape=mx_shape(mx, cfg, b.pool_pages))
    assert need_attn < need
    assert mx.mx_packed_weights_bytes(c) >= 2 * cfg.params


@pytest.mark.parametrize("args,status", [
    ((64, 256, 256, 0, 5, 1), "MX_ERR_INVALID"),       # tile shape out of range
    ((64, 256, 256, 0, -2, 1), "MX_ERR_INVALID"),
    ((64, 256, 256, 0, 0, 0), "MX_ERR_INVALID"),       # forced shape without a split count
    ((64, 256, 256, 0, 0, 5), "MX_ERR_INVALID"),       # more splits than 64-wide K chunks
    ((64, 256, 160, 0, 0, 1), "MX_ERR_UNSUPPORTED"),   # K not a multiple of 64
    ((-1, 256, 256, 0, 0, 1), "MX_ERR_INVALID"),       # negative M
    ((64, 96, 256, 2, 0, 1), "MX_ERR_UNSUPPORTED"),    # SwiGLU needs N % 64 == 0
    ((64, 256, 256, 3, 0, 1), "MX_ERR_INVALID"),       # the QKV epilogue is not exposed here
    ((64, 256, 512, 0, 0, 2), "MX_ERR_TOO_LARGE"),     # split scratch larger than ws
    ((64, 256, 256, 1, 0, 1), "MX_ERR_INVALID"),       # residual R overlapping C (0x4000 in [0x3000, +32K))
])
def test_debug_gemm_config_errors(args, status):
    M, N, K, epi, cfg, ks = args
    st = mx.lib().mx_debug_gemm_config(M, N, K, 0x1000, 0x2000, 0x3000, 0x4000, epi, cfg, ks,
                                       0x5000, 16, None)
    assert st == getattr(mx, status), st


@pytest.mark.parametrize("args,status", [
    ((64, 264, 256, 0, 0, 1), "MX_ERR_UNSUPPORTED"),   # tiled weights need N % 16 == 0
    ((64, 256, 160, 0, 0, 1), "MX_ERR_UNSUPPORTED"),   # K not a multiple of 64
    ((64, 256, 256, 0, 5, 1), "MX_ERR_INVALID"),       # tile shape out of range
])
def test_debug_gemm_tiled_errors(args, status):
    M, N, K, epi, cfg, ks = args
    st = mx.lib().mx_debug_gemm_tiled(M, N, K, 0x1000, 0x2000, 0x3000, 0x4000, epi, cfg, ks,
                                      0x5000, 16, None)
    assert st == getattr(mx, status), st


def test_misaligned_pointers_rejected_before_device_work():
    cfg = wl.CONFIGS["c1"]
    c = mx_cfg(mx, cfg, 64)
    good = one(mx.MX_PREFILL, 4, 0, [1])
    # x off by 8 bytes
    st = mx.lib().mx_layer_step(good.ptr, mx.ctypes.byref(c), 0x1000, 0x2008, 0x3000, 0x4000,
                                0x5000, 0x6000, 1 << 30, None)
    assert st == mx.MX_ERR_INVALID
    st = mx.lib().mx_paged_attn(good.ptr, mx.ctypes.byref(c.attn), 0x1000, 0x2000, 0x3002,
                                0x4000, 0x6000, 1 << 30, None)
    assert st == mx.MX_ERR_INVALID
    st = mx.lib().mx_kv_append(good.ptr, mx.ctypes.byref(c.attn), 0x1000, 0x2000, 0x3000, 0x4000,
                               0x6004, 1 << 30, None)
    assert st == mx.MX_ERR_INVALID
    st = mx.lib().mx_debug_gemm_config(64, 256, 256, 0x1000, 0x2000, 0x3006, None, 0, 0, 1,
                                       0x5000, 1 << 20, None)
    assert st == mx.MX_ERR_INVALID


def test_one_hip_runtime_whatever_the_import_order():
    """Importing the binding before torch must not leave two HIP runtimes in
    the process (the library's and torch's): streams and pointers handed from
    one to the other are invalid.  Checked in a fresh interpreter that imports
    the binding first, then torch, then the input generator library."""
    code = (
        "import paper_2606_16264_amd, torch, workload.device as d; d.lib()\n"
        "maps = open('/proc/self/maps').read().split('\\n')\n"
        "paths = {l.split()[-1] for l in maps if 'libamdhip64' in l}\n"
        "print(len(paths)); print(sorted(paths))\n")
    out = subprocess.run([__import__("sys").executable, "-c", code], cwd=ROOT, capture_output=True,
                         text=True, timeout=300)
    assert out.returncode == 0, out.stderr[-2000:]
    n = int(out.stdout.split()[0])
    assert n == 1, out.stdout
