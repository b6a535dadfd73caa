"""Device-side synthetic pool fill (wraps workload/libmxgen.so).  Input
generation only; the values are those of ``workload.hash_bf16`` at each
element's canonical index."""
from __future__ import annotations

import ctypes
import os

import numpy as np

import workload as wl

_LIB = os.path.join(os.path.dirname(os.path.abspath(__file__)), "libmxgen.so")
_lib = None


def lib():
    global _lib
    if _lib is None:
        if not os.path.exists(_LIB):
            raise ImportError(f"{_LIB} is not built; run __graft_entry__.build()")
        import torch  # noqa: F401  (torch's HIP runtime must be the one loaded first)
        L = ctypes.CDLL(_LIB)
        P, I32, I64, U64 = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_uint64
        L.mxgen_fill_pool.argtypes = [P, P, I64, I32, I32, U64, U64, P, P]
        L.mxgen_fill_pool.restype = ctypes.c_int
        L.mxgen_poison_slots.argtypes = [P, P, P, I64, I32, I32, P]
        L.mxgen_poison_slots.restype = ctypes.c_int
        _lib = L
    return _lib


def alloc_pools(cfg: wl.LayerConfig, pool_pages: int, device="cuda"):
    import torch
    # keys: each page blocked by 32 dims, [page][head][dim / 32][slot][32]
    k = torch.empty((pool_pages, cfg.n_kv_heads, cfg.head_dim // 32, 16, 32),
                    dtype=torch.uint16, device=device)
    # values: each page stored transposed, [page][head][dim][slot]
    v = torch.empty((pool_pages, cfg.n_kv_heads, cfg.head_dim, 16), dtype=torch.uint16,
                    device=device)
    return k, v


def fill_pools(k_pool, v_pool, cfg: wl.LayerConfig, batch: wl.Batch, seed: int,
               poison: bool = True) -> None:
    """Hash values everywhere; bf16 NaN on pages no request owns and on slots at
    or beyond each request's ctx_len (when ``poison``).  V is written in the
    transposed page layout and K in the blocked one."""
    import torch
    stream = torch.cuda.current_stream().cuda_stream
    owned = None
    if poison:
        owned = torch.from_numpy(wl.owned_pages_mask(batch)).to(k_pool.device)
    rc = lib().mxgen_fill_pool(k_pool.data_ptr(), v_pool.data_ptr(), batch.pool_pages,
                               cfg.n_kv_heads, cfg.head_dim, int(wl.stream_key(seed, 0)),
                               int(wl.stream_key(seed, 1)),
                               owned.data_ptr() if owned is not None else None, stream)
    if rc != 0:
        raise RuntimeError(f"mxgen_fill_pool failed ({rc})")
    if poison:
        slots = wl.poison_slots(batch)
        if len(slots):
            ts = torch.from_numpy(slots.astype(np.int64)).to(k_pool.device)
            rc = lib().mxgen_poison_slots(k_pool.data_ptr(), v_pool.data_ptr(), ts.data_ptr(),
                                          len(slots), cfg.n_kv_heads, cfg.head_dim, stream)
            if rc != 0:
                raise RuntimeError(f"mxgen_poison_slots failed ({rc})")
            torch.cuda.current_stream().synchronize()


def _host(t) -> np.ndarray:
    a = t.cpu().numpy() if hasattr(t, "cpu") else np.asarray(t)
    return a.view(np.uint16)


def k_pool_canonical(k_pool_b):
    """Device K pool [pages][nkv][d/32][16][32] (blocked pages) -> numpy uint16
    [pages][nkv][16][d]."""
    a = _host(k_pool_b)
    p, g, nb = a.shape[:3]
    return np.ascontiguousarray(a.transpose(0, 1, 3, 2, 4).reshape(p, g, 16, nb * 32))


def k_pool_blocked(k_canon: np.ndarray) -> np.ndarray:
    """Canonical [pages][nkv][16][d] -> the device's blocked K page layout
    [pages][nkv][d/32][16][32]."""
    p, g, s, d = k_canon.shape
    return np.ascontiguousarray(k_canon.reshape(p, g, s, d // 32, 32).transpose(0, 1, 3, 2, 4))


def v_pool_canonical(v_pool_t):
    """Device V pool [pages][nkv][d][16] (transposed pages) -> numpy uint16
    [pages][nkv][16][d]."""
    a = v_pool_t.cpu().numpy() if hasattr(v_pool_t, "cpu") else np.asarray(v_pool_t)
    return np.ascontiguousarray(a.view(np.uint16).transpose(0, 1, 3, 2))
