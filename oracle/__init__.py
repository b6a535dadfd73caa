"""Python view of the fp64 CPU oracle (``oracle/oracle.c``).

TEST INFRASTRUCTURE ONLY: the tests, the smoke check and the CPU-baseline leg of
the benchmark use this package; the product library and its binding never
import it.  It loads ``liboracle.so`` with ctypes and marshals numpy arrays; all
arithmetic is in the C file.
"""
from __future__ import annotations

import ctypes
import os
import subprocess
from dataclasses import dataclass

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
_LIB_PATH = os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "oracle.c")


CFLAGS = ["-O2", "-march=x86-64-v3", "-fopenmp"]


def build(verbose: bool = False) -> str:
    """Compile liboracle.so with gcc (plain C, OpenMP)."""
    cmd = ["gcc"] + CFLAGS + ["-fPIC", "-shared", "-std=c11",
                              "-Wall", "-Wextra", "-Wno-unused-parameter", "-o", _LIB_PATH + ".tmp",
                              _SRC, "-lm"]
    if verbose:
        print(" ".join(cmd))
    subprocess.run(cmd, check=True)
    os.replace(_LIB_PATH + ".tmp", _LIB_PATH)
    return _LIB_PATH


_lib = None


class using:
    """Context manager that routes every call to another build of oracle.c
    (the mutation tests compile deliberately broken copies on the CPU)."""

    def __init__(self, path: str):
        self.path = path

    def __enter__(self):
        global _lib
        self.saved = _lib
        alt = ctypes.CDLL(self.path)
        _declare(alt)
        _lib = alt
        return alt

    def __exit__(self, *exc):
        global _lib
        _lib = self.saved
        return False


def build_variant(src_text: str, out_path: str) -> str:
    """Compile a modified copy of oracle.c (CPU only, for mutation tests)."""
    d = os.path.dirname(out_path)
    src = os.path.join(d, "oracle_variant.c")
    with open(src, "w") as f:
        f.write(src_text)
    subprocess.run(["gcc", "-O1", "-fopenmp", "-fPIC", "-shared", "-std=c11", "-I", _HERE,
                    "-o", out_path, src, "-lm"], check=True)
    return out_path


def source_text() -> str:
    with open(_SRC) as f:
        return f.read()


def lib() -> ctypes.CDLL:
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB_PATH) or os.path.getmtime(_LIB_PATH) < os.path.getmtime(_SRC):
            build()
        _lib = ctypes.CDLL(_LIB_PATH)
        _declare(_lib)
    return _lib


_P = ctypes.c_void_p
_I32 = ctypes.c_int32
_I64 = ctypes.c_int64
_D = ctypes.c_double


class _LayerCfg(ctypes.Structure):
    _fields_ = [("hidden", _I32), ("ffn", _I32), ("n_q_heads", _I32), ("n_kv_heads", _I32),
                ("head_dim", _I32), ("rms_eps", _D), ("rope_theta", _D), ("scale", _D)]


def _declare(L: ctypes.CDLL) -> None:
    L.orc_bf16_to_double.argtypes = [ctypes.c_uint16]
    L.orc_bf16_to_double.restype = _D
    L.orc_num_threads.restype = ctypes.c_int
    L.orc_token_map.argtypes = [_I32, _P, _P, _P, _P, _I32, _P, _P, _P, _P]
    L.orc_token_map.restype = ctypes.c_int
    L.orc_rmsnorm.argtypes = [_I64, _I64, _P, _P, _D, _P]
    L.orc_linear.argtypes = [_I64, _I64, _I64, _P, _P, _P]
    L.orc_rope.argtypes = [_I64, _I32, _I32, _P, _D, _P]
    L.orc_silu_mul.argtypes = [_I64, _I64, _P, _P]
    L.orc_attention_contig.argtypes = [_I32, _P, _P, _I32, _I32, _I32, _D, _P, _P, _P, _P, _P]
    L.orc_attention_paged.argtypes = [_I32, _P, _P, _I32, _I32, _I32, _D, _P, _P, _P, _I64,
                                      _I32, _P, _P, _P]
    L.orc_attention_paged.restype = ctypes.c_int
    L.orc_attention_weights.argtypes = [_I32, _P, _P, _I32, _I32, _I32, _D, _P, _P, _P, _I64,
                                        _I32, _P]
    L.orc_attention_weights.restype = _I64
    L.orc_layer_step.argtypes = [ctypes.POINTER(_LayerCfg), _I32, _P, _P] + [_P] * 9 + \
        [_I64, _P] + [_P] * 9
    L.orc_layer_step.restype = ctypes.c_int
    L.orc_kv_append.argtypes = [_I32, _P, _P, _P, _P, _I32, _I32, _I32, _P, _P, _P, _P, _I64]
    L.orc_kv_append.restype = ctypes.c_int


def _c(a, dtype):
    """Contiguous array of the given dtype (a copy only if needed)."""
    return np.ascontiguousarray(a, dtype=dtype)


def _p(a) -> int:
    return a.ctypes.data if a is not None else None


def num_threads() -> int:
    return int(lib().orc_num_threads())


def bf16_to_double(bits: int) -> float:
    return float(lib().orc_bf16_to_double(int(bits)))


@dataclass
class TokenMap:
    cu_q: np.ndarray
    tok_req: np.ndarray
    tok_pos: np.ndarray
    tok_slot: np.ndarray


def _tables(page_tables):
    page_off = np.zeros(len(page_tables) + 1, dtype=np.int64)
    for r, tbl in enumerate(page_tables):
        page_off[r + 1] = page_off[r] + len(tbl)
    flat = np.concatenate([np.asarray(t, dtype=np.int32) for t in page_tables]) \
        if page_tables else np.zeros(0, dtype=np.int32)
    return page_off, _c(flat if flat.size else np.zeros(1, np.int32), np.int32)


def token_map(n_new, ctx_len, page_tables, page_size: int = 16) -> TokenMap:
    n_new = _c(n_new, np.int32)
    ctx_len = _c(ctx_len, np.int32)
    R = len(n_new)
    page_off, flat = _tables(page_tables)
    T = int(n_new.sum())
    cu_q = np.zeros(R + 1, np.int32)
    tok_req = np.zeros(max(T, 1), np.int32)
    tok_pos = np.zeros(max(T, 1), np.int32)
    tok_slot = np.zeros(max(T, 1), np.int64)
    rc = lib().orc_token_map(R, _p(n_new), _p(ctx_len), _p(page_off), _p(flat), page_size,
                             _p(cu_q), _p(tok_req), _p(tok_pos), _p(tok_slot))
    if rc != 0:
        raise ValueError("page table too short for the request's positions")
    return TokenMap(cu_q, tok_req[:T], tok_pos[:T], tok_slot[:T])


def rmsnorm(x, g, eps: float) -> np.ndarray:
    x = _c(x, np.float64)
    g = _c(g, np.float64)
    T, H = x.shape
    out = np.empty_like(x)
    lib().orc_rmsnorm(T, H, _p(x), _p(g), eps, _p(out))
    return out


def linear(a, w_bf16) -> np.ndarray:
    a = _c(a, np.float64)
    w = _c(w_bf16, np.uint16)
    T, K = a.shape
    N, K2 = w.shape
    assert K == K2
    out = np.empty((T, N), np.float64)
    lib().orc_linear(T, K, N, _p(a), _p(w), _p(out))
    return out


def rope(u, pos, theta: float) -> np.ndarray:
    u = np.array(u, dtype=np.float64, copy=True, order="C")
    pos = _c(pos, np.int32)
    T, nh, d = u.shape
    lib().orc_rope(T, nh, d, _p(pos), theta, _p(u))
    return u


def silu_mul(gu) -> np.ndarray:
    gu = _c(gu, np.float64)
    T, F2 = gu.shape
    F = F2 // 2
    a = np.empty((T, F), np.float64)
    lib().orc_silu_mul(T, F, _p(gu), _p(a))
    return a


def attention_contig(n_new, ctx_len, q, kc, vc, kv_off, scale: float) -> np.ndarray:
    """q [T,nq,d]; kc/vc [sum kv_len, nkv, d]; kv_off [R] token offset per request."""
    n_new = _c(n_new, np.int32)
    ctx_len = _c(ctx_len, np.int32)
    q = _c(q, np.float64)
    kc = _c(kc, np.float64)
    vc = _c(vc, np.float64)
    kv_off = _c(kv_off, np.int64)
    T, nq, d = q.shape
    nkv = kc.shape[1]
    o = np.empty_like(q)
    lib().orc_attention_contig(len(n_new), _p(n_new), _p(ctx_len), nq, nkv, d, scale, _p(q),
                               _p(kc), _p(vc), _p(kv_off), _p(o))
    return o


def attention_paged(n_new, ctx_len, q, k_pool, v_pool, page_tables, scale: float) -> np.ndarray:
    """q [T,nq,d]; pools [pool_pages, nkv, page_size, d] (float64)."""
    n_new = _c(n_new, np.int32)
    ctx_len = _c(ctx_len, np.int32)
    q = _c(q, np.float64)
    k_pool = _c(k_pool, np.float64)
    v_pool = _c(v_pool, np.float64)
    T, nq, d = q.shape
    pool_pages, nkv, ps, d2 = k_pool.shape
    assert d2 == d
    page_off, flat = _tables(page_tables)
    o = np.empty_like(q)
    rc = lib().orc_attention_paged(len(n_new), _p(n_new), _p(ctx_len), nq, nkv, d, scale,
                                   _p(q), _p(k_pool), _p(v_pool), pool_pages, ps,
                                   _p(page_off), _p(flat), _p(o))
    if rc != 0:
        raise ValueError("invalid page table")
    return o


def attention_weights(n_new, ctx_len, q, kc, kv_off, scale: float, t: int, h: int) -> np.ndarray:
    n_new = _c(n_new, np.int32)
    ctx_len = _c(ctx_len, np.int32)
    q = _c(q, np.float64)
    kc = _c(kc, np.float64)
    kv_off = _c(kv_off, np.int64)
    T, nq, d = q.shape
    nkv = kc.shape[1]
    w = np.empty(int(kc.shape[0]) + 1, np.float64)
    n = lib().orc_attention_weights(len(n_new), _p(n_new), _p(ctx_len), nq, nkv, d, scale,
                                    _p(q), _p(kc), _p(kv_off), t, h, _p(w))
    if n < 0:
        raise ValueError("token out of range")
    return w[:n]


@dataclass
class LayerOut:
    h: np.ndarray
    k_new: np.ndarray
    v_new: np.ndarray
    q: np.ndarray
    o: np.ndarray
    x1: np.ndarray
    h2: np.ndarray
    a: np.ndarray
    y: np.ndarray
    rows: np.ndarray


def layer_step(cfg: dict, n_new, ctx_len, x, weights: dict, k_prior, v_prior,
               rows=None) -> LayerOut:
    """One layer iteration.  ``x`` and every weight are bf16 bit arrays (uint16);
    ``k_prior``/``v_prior`` are bf16 bits [sum ctx_len, nkv, d], request-major.
    ``rows``: token indices to evaluate (default: all)."""
    n_new = _c(n_new, np.int32)
    ctx_len = _c(ctx_len, np.int32)
    H, F = cfg["hidden"], cfg["ffn"]
    nq, nkv, d = cfg["n_q_heads"], cfg["n_kv_heads"], cfg["head_dim"]
    T = int(n_new.sum())
    x = _c(x, np.uint16).reshape(T, H)
    w = {k: _c(weights[k], np.uint16) for k in ("g1", "w_qkv", "w_o", "g2", "w_gu", "w_down")}
    kp = _c(k_prior, np.uint16).reshape(-1) if np.size(k_prior) else np.zeros(1, np.uint16)
    vp = _c(v_prior, np.uint16).reshape(-1) if np.size(v_prior) else np.zeros(1, np.uint16)
    if rows is None:
        rows_arr = np.arange(T, dtype=np.int64)
    else:
        rows_arr = _c(np.sort(np.asarray(rows)), np.int64)
    nr = len(rows_arr)
    c = _LayerCfg(H, F, nq, nkv, d, float(cfg["rms_eps"]), float(cfg["rope_theta"]),
                  float(cfg.get("scale", 1.0 / np.sqrt(d))))
    h = np.empty((T, H), np.float64)
    k_new = np.empty((T, nkv, d), np.float64)
    v_new = np.empty((T, nkv, d), np.float64)
    q = np.empty((nr, nq, d), np.float64)
    o = np.empty((nr, nq * d), np.float64)
    x1 = np.empty((nr, H), np.float64)
    h2 = np.empty((nr, H), np.float64)
    a = np.empty((nr, F), np.float64)
    y = np.empty((nr, H), np.float64)
    rc = lib().orc_layer_step(ctypes.byref(c), len(n_new), _p(n_new), _p(ctx_len), _p(x),
                              _p(w["g1"]), _p(w["w_qkv"]), _p(w["w_o"]), _p(w["g2"]),
                              _p(w["w_gu"]), _p(w["w_down"]), _p(kp), _p(vp), nr,
                              _p(rows_arr), _p(h), _p(k_new), _p(v_new), _p(q), _p(o),
                              _p(x1), _p(h2), _p(a), _p(y))
    if rc != 0:
        raise ValueError("orc_layer_step rejected its arguments")
    return LayerOut(h, k_new, v_new, q, o, x1, h2, a, y, rows_arr)


def kv_append(n_new, ctx_len, page_tables, k_new_bits, v_new_bits, k_pool_bits, v_pool_bits,
              page_size: int = 16):
    """Returns new (k_pool, v_pool) uint16 arrays with the new rows copied in."""
    n_new = _c(n_new, np.int32)
    ctx_len = _c(ctx_len, np.int32)
    kn = _c(k_new_bits, np.uint16)
    vn = _c(v_new_bits, np.uint16)
    kpool = np.array(k_pool_bits, dtype=np.uint16, copy=True, order="C")
    vpool = np.array(v_pool_bits, dtype=np.uint16, copy=True, order="C")
    pool_pages, nkv, ps, d = kpool.shape
    assert ps == page_size
    page_off, flat = _tables(page_tables)
    rc = lib().orc_kv_append(len(n_new), _p(n_new), _p(ctx_len), _p(page_off), _p(flat),
                             page_size, nkv, d, _p(kn), _p(vn), _p(kpool), _p(vpool),
                             pool_pages)
    if rc != 0:
        raise ValueError("invalid page table")
    return kpool, vpool
