"""Python binding of libmx, the gfx950 HIP library declared in ``include/mx.h``.

Argument marshalling only: every step of the layer iteration runs in the HIP
kernels of ``libmx.so``.  PyTorch supplies device memory (``tensor.data_ptr()``)
and streams.  Importing this module fails loudly if ``libmx.so`` has not been
built (``python -m paper_2606_16264_amd.build`` or ``__graft_entry__.build()``);
there is no fallback implementation.
"""
from __future__ import annotations

import ctypes
import os
from dataclasses import dataclass
from typing import Optional, Sequence

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# MX_LIB_PATH selects another build of the same library (the host-sanitized
# one); by default the in-tree libmx.so.
LIB_PATH = os.environ.get("MX_LIB_PATH") or os.path.join(_HERE, "libmx.so")

MX_OK, MX_ERR_INVALID, MX_ERR_NO_SPACE, MX_ERR_TOO_LARGE, MX_ERR_UNSUPPORTED, MX_ERR_NULL, \
    MX_ERR_HIP = range(7)
MX_PREFILL, MX_DECODE = 0, 1

EXPORTED = [
    "mx_status_str", "mx_last_error", "mx_version", "mx_batch_validate", "mx_workspace_bytes_for",
    "mx_workspace_bytes", "mx_packed_weights_bytes", "mx_pack_weights", "mx_kv_append",
    "mx_paged_attn", "mx_layer_step", "mx_layer_workspace_offsets", "mx_debug_token_map",
    "mx_debug_gather", "mx_debug_gemm_ws_bytes", "mx_debug_gemm", "mx_debug_gemm_config",
    "mx_debug_gemm_tiled", "mx_debug_gemm_plan", "mx_debug_gemm_rows",
    "mx_debug_reduce_residual_rmsnorm", "mx_paged_attn_static", "mx_paged_attn_static_max_bytes",
    "mx_profile_enable", "mx_profile_read",
]


class MxError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_status_name(status)}: {msg}")
        self.status = status


class _Request(ctypes.Structure):
    _fields_ = [("phase", ctypes.c_int32), ("n_new", ctypes.c_int32), ("ctx_len", ctypes.c_int32),
                ("n_pages", ctypes.c_int32), ("pages", ctypes.POINTER(ctypes.c_int32))]


class _Batch(ctypes.Structure):
    _fields_ = [("num_reqs", ctypes.c_int32), ("reqs", ctypes.POINTER(_Request))]


class AttnShape(ctypes.Structure):
    _fields_ = [("n_q_heads", ctypes.c_int32), ("n_kv_heads", ctypes.c_int32),
                ("head_dim", ctypes.c_int32), ("page_size", ctypes.c_int32),
                ("pool_pages", ctypes.c_int64), ("scale", ctypes.c_float)]


class LayerCfg(ctypes.Structure):
    _fields_ = [("hidden", ctypes.c_int32), ("ffn", ctypes.c_int32), ("attn", AttnShape),
                ("rms_eps", ctypes.c_float), ("rope_theta", ctypes.c_float)]


class _Weights(ctypes.Structure):
    _fields_ = [(n, ctypes.c_void_p) for n in ("ln1_g", "w_qkv", "w_o", "ln2_g", "w_gate_up", "w_down")]


def _load() -> ctypes.CDLL:
    if not os.path.exists(LIB_PATH):
        raise ImportError(f"{LIB_PATH} is not built; run __graft_entry__.build() "
                          "(there is no fallback implementation)")
    # torch first: it loads the HIP runtime it ships with, and libmx.so's own
    # dependency on libamdhip64.so.7 then binds to that same runtime.  Loaded
    # the other way round, the process ends up with two HIP runtimes (the
    # system one for libmx.so, torch's for torch), and streams and pointers
    # passed between them are invalid.
    import torch  # noqa: F401
    L = ctypes.CDLL(LIB_PATH)
    P, I32, I64, SZ = ctypes.c_void_p, ctypes.c_int32, ctypes.c_int64, ctypes.c_size_t
    BP = ctypes.POINTER(_Batch)
    SP = ctypes.POINTER(AttnShape)
    CP = ctypes.POINTER(LayerCfg)
    sig = {
        "mx_status_str": ([ctypes.c_int], ctypes.c_char_p),
        "mx_last_error": ([], ctypes.c_char_p),
        "mx_version": ([], ctypes.c_uint32),
        "mx_batch_validate": ([BP, SP], ctypes.c_int),
        "mx_workspace_bytes_for": ([BP, SP, CP], SZ),
        "mx_workspace_bytes": ([CP, SP, I32, I32, I64], SZ),
        "mx_packed_weights_bytes": ([CP], SZ),
        "mx_pack_weights": ([CP, ctypes.POINTER(_Weights), P, SZ, P], ctypes.c_int),
        "mx_kv_append": ([BP, SP, P, P, P, P, P, SZ, P], ctypes.c_int),
        "mx_paged_attn": ([BP, SP, P, P, P, P, P, SZ, P], ctypes.c_int),
        "mx_layer_step": ([BP, CP, P, P, P, P, P, P, SZ, P], ctypes.c_int),
        "mx_paged_attn_static": ([BP, SP, P, P, P, P, P], ctypes.c_int),
        "mx_paged_attn_static_max_bytes": ([], SZ),
        "mx_layer_workspace_offsets": ([BP, CP, ctypes.POINTER(SZ)], ctypes.c_int),
        "mx_debug_token_map": ([BP, SP, P, P, P, P, SZ, P], ctypes.c_int),
        "mx_debug_gather": ([BP, SP, I32, P, P, P, P, P, SZ, P], ctypes.c_int),
        "mx_debug_gemm_ws_bytes": ([I32, I32, I32], SZ),
        "mx_debug_gemm": ([I32, I32, I32, P, P, P, P, I32, P, SZ, P], ctypes.c_int),
        "mx_debug_gemm_config": ([I32, I32, I32, P, P, P, P, I32, I32, I32, P, SZ, P], ctypes.c_int),
        "mx_debug_gemm_tiled": ([I32, I32, I32, P, P, P, P, I32, I32, I32, P, SZ, P], ctypes.c_int),
        "mx_debug_gemm_plan": ([I32, I32, I32, ctypes.POINTER(I32)], ctypes.c_int),
        "mx_debug_gemm_rows": ([I32, I32, I32, P, P, P, P, I32, I32, I32, I32, I32, P, SZ, P],
                               ctypes.c_int),
        "mx_debug_reduce_residual_rmsnorm": ([P, I32, P, P, P, P, I32, I32, ctypes.c_float, I32, P],
                                             ctypes.c_int),
        "mx_profile_enable": ([I32], ctypes.c_int),
        "mx_profile_read": ([ctypes.POINTER(ctypes.c_char_p), ctypes.POINTER(ctypes.c_float),
                             ctypes.POINTER(ctypes.c_int32), I32], I32),
    }
    for name, (args, res) in sig.items():
        fn = getattr(L, name)
        fn.argtypes = args
        fn.restype = res
    return L


_lib = _load()


def lib() -> ctypes.CDLL:
    return _lib


def _status_name(s: int) -> str:
    return _lib.mx_status_str(int(s)).decode()


def last_error() -> str:
    return _lib.mx_last_error().decode()


def _check(status: int) -> None:
    if status != MX_OK:
        raise MxError(status, last_error())


# ----------------------------------------------------------------- batch marshalling
class Batch:
    """A mixed batch in the C layout.  Holds the host arrays alive while in use."""

    def __init__(self, phase: Sequence[int], n_new: Sequence[int], ctx_len: Sequence[int],
                 page_tables: Sequence[Sequence[int]]):
        R = len(n_new)
        self._tables = [np.ascontiguousarray(t, dtype=np.int32) for t in page_tables]
        self._reqs = (_Request * max(R, 1))()
        for r in range(R):
            t = self._tables[r]
            self._reqs[r].phase = int(phase[r])
            self._reqs[r].n_new = int(n_new[r])
            self._reqs[r].ctx_len = int(ctx_len[r])
            self._reqs[r].n_pages = len(t)
            self._reqs[r].pages = t.ctypes.data_as(ctypes.POINTER(ctypes.c_int32)) if len(t) else None
        self._batch = _Batch(R, self._reqs)
        self.R = R
        self.T = int(sum(int(n) for n in n_new))

    @property
    def ptr(self):
        return ctypes.byref(self._batch)


def attn_shape(n_q_heads, n_kv_heads, head_dim, pool_pages, scale=0.0, page_size=16) -> AttnShape:
    return AttnShape(n_q_heads, n_kv_heads, head_dim, page_size, int(pool_pages), float(scale))


def layer_cfg(hidden, ffn, n_q_heads, n_kv_heads, head_dim, pool_pages, rms_eps=1e-5,
              rope_theta=1e4, scale=0.0) -> LayerCfg:
    return LayerCfg(hidden, ffn, attn_shape(n_q_heads, n_kv_heads, head_dim, pool_pages, scale),
                    float(rms_eps), float(rope_theta))


def _ptr(t) -> Optional[int]:
    return None if t is None else t.data_ptr()


def _stream(stream) -> Optional[int]:
    if stream is None:
        import torch
        return torch.cuda.current_stream().cuda_stream
    return getattr(stream, "cuda_stream", stream)


# ----------------------------------------------------------------- entry points
def mx_version() -> int:
    return int(_lib.mx_version())


def mx_batch_validate(batch: Batch, shape: AttnShape) -> int:
    """Returns the status code (host only)."""
    return int(_lib.mx_batch_validate(batch.ptr, ctypes.byref(shape)))


def mx_workspace_bytes_for(batch: Batch, shape: Optional[AttnShape] = None,
                           cfg: Optional[LayerCfg] = None) -> int:
    n = _lib.mx_workspace_bytes_for(batch.ptr, ctypes.byref(shape) if shape else None,
                                    ctypes.byref(cfg) if cfg else None)
    if n == 0:
        raise MxError(MX_ERR_INVALID, last_error())
    return int(n)


def mx_workspace_bytes(cfg: Optional[LayerCfg], shape: Optional[AttnShape], max_tokens: int,
                       max_reqs: int, max_pages: int) -> int:
    n = _lib.mx_workspace_bytes(ctypes.byref(cfg) if cfg else None,
                                ctypes.byref(shape) if shape else None, max_tokens, max_reqs,
                                max_pages)
    if n == 0:
        raise MxError(MX_ERR_INVALID, last_error())
    return int(n)


def mx_packed_weights_bytes(cfg: LayerCfg) -> int:
    n = _lib.mx_packed_weights_bytes(ctypes.byref(cfg))
    if n == 0:
        raise MxError(MX_ERR_INVALID, last_error())
    return int(n)


def mx_pack_weights(cfg: LayerCfg, weights: dict, packed, stream=None) -> None:
    """weights: device tensors g1, w_qkv, w_o, g2, w_gu, w_down (bf16 or uint16 views)."""
    w = _Weights(_ptr(weights["g1"]), _ptr(weights["w_qkv"]), _ptr(weights["w_o"]),
                 _ptr(weights["g2"]), _ptr(weights["w_gu"]), _ptr(weights["w_down"]))
    _check(_lib.mx_pack_weights(ctypes.byref(cfg), ctypes.byref(w), _ptr(packed),
                                packed.numel() * packed.element_size(), _stream(stream)))


def mx_kv_append(batch: Batch, shape: AttnShape, k_new, v_new, k_pool, v_pool, ws,
                 stream=None) -> None:
    _check(_lib.mx_kv_append(batch.ptr, ctypes.byref(shape), _ptr(k_new), _ptr(v_new),
                             _ptr(k_pool), _ptr(v_pool), _ptr(ws), ws.numel(), _stream(stream)))


def mx_paged_attn(batch: Batch, shape: AttnShape, q, k_pool, v_pool, out, ws, stream=None) -> None:
    _check(_lib.mx_paged_attn(batch.ptr, ctypes.byref(shape), _ptr(q), _ptr(k_pool), _ptr(v_pool),
                              _ptr(out), _ptr(ws), ws.numel(), _stream(stream)))


def mx_paged_attn_static(batch: Batch, shape: AttnShape, q, k_pool, v_pool, out,
                         stream=None) -> None:
    """mx_paged_attn with the library's static device scratch instead of a
    workspace (no allocation); calls on one GPU must not overlap."""
    _check(_lib.mx_paged_attn_static(batch.ptr, ctypes.byref(shape), _ptr(q), _ptr(k_pool),
                                     _ptr(v_pool), _ptr(out), _stream(stream)))


def mx_paged_attn_static_max_bytes() -> int:
    return int(_lib.mx_paged_attn_static_max_bytes())


def mx_layer_step(batch: Batch, cfg: LayerCfg, packed, x, y, k_pool, v_pool, ws,
                  stream=None) -> None:
    _check(_lib.mx_layer_step(batch.ptr, ctypes.byref(cfg), _ptr(packed), _ptr(x), _ptr(y),
                              _ptr(k_pool), _ptr(v_pool), _ptr(ws), ws.numel(), _stream(stream)))


def mx_layer_workspace_offsets(batch: Batch, cfg: LayerCfg) -> dict:
    off = (ctypes.c_size_t * 5)()
    _check(_lib.mx_layer_workspace_offsets(batch.ptr, ctypes.byref(cfg), off))
    return dict(zip(("h", "q", "o", "x1", "a"), [int(v) for v in off]))


def mx_debug_token_map(batch: Batch, shape: AttnShape, tok_req, tok_pos, tok_slot, ws,
                       stream=None) -> None:
    _check(_lib.mx_debug_token_map(batch.ptr, ctypes.byref(shape), _ptr(tok_req), _ptr(tok_pos),
                                   _ptr(tok_slot), _ptr(ws), ws.numel(), _stream(stream)))


def mx_debug_gather(batch: Batch, shape: AttnShape, req: int, k_pool, v_pool, k_out, v_out, ws,
                    stream=None) -> None:
    _check(_lib.mx_debug_gather(batch.ptr, ctypes.byref(shape), int(req), _ptr(k_pool),
                                _ptr(v_pool), _ptr(k_out), _ptr(v_out), _ptr(ws), ws.numel(),
                                _stream(stream)))


EPI_STORE, EPI_RESIDUAL, EPI_SWIGLU = 0, 1, 2


def mx_debug_gemm_ws_bytes(M: int, N: int, K: int) -> int:
    return int(_lib.mx_debug_gemm_ws_bytes(M, N, K))


def mx_debug_gemm(A, B, C, R=None, epilogue: int = EPI_STORE, ws=None, stream=None,
                  tile_cfg: int = -1, ksplit: int = 0, tiled: bool = False, M: int = None,
                  N: int = None, K: int = None) -> None:
    """C = epi(A B^T); A [M][K], B [N][K], C [M][N] (or [M][N/2] for SwiGLU).
    tile_cfg >= 0 forces a tile shape and K split (tuning).  tiled: the
    operands in the layer step's layouts (mx_debug_gemm_tiled: A and B in the
    16 x 32 tile layout, the SwiGLU output too; any tensor shapes, pass M, N, K)."""
    if tiled:
        if M is None or N is None or K is None:
            raise ValueError("tiled needs M, N and K")
        fn = _lib.mx_debug_gemm_tiled
    else:
        M, K = A.shape
        N = B.shape[0]
        fn = _lib.mx_debug_gemm_config
    _check(fn(M, N, K, _ptr(A), _ptr(B), _ptr(C), _ptr(R), epilogue, tile_cfg, ksplit, _ptr(ws),
              0 if ws is None else ws.numel(), _stream(stream)))


def mx_debug_gemm_plan(M: int, N: int, K: int) -> dict:
    """The cost model's plan of an M x N x K projection (host only)."""
    out = (ctypes.c_int32 * 5)()
    _check(_lib.mx_debug_gemm_plan(M, N, K, out))
    return {"cfg": out[0], "ksplit": out[1], "m_main": out[2], "tail_cfg": out[3],
            "tail_ksplit": out[4]}


def mx_debug_gemm_rows(A, B_tiled, C, R, epilogue: int, M: int, N: int, K: int, m_main: int,
                       main_cfg: int, tail_cfg: int, tail_ksplit: int, ws=None,
                       stream=None) -> None:
    """A forced row split (operands in the layer's layouts, as mx_debug_gemm
    with tiled=True): rows [0, m_main) with tile shape main_cfg, the rest with
    tail_cfg split tail_ksplit ways over K."""
    _check(_lib.mx_debug_gemm_rows(M, N, K, _ptr(A), _ptr(B_tiled), _ptr(C), _ptr(R), epilogue,
                                   m_main, main_cfg, tail_cfg, tail_ksplit, _ptr(ws),
                                   0 if ws is None else ws.numel(), _stream(stream)))


def mx_debug_reduce_residual_rmsnorm(partial, ksplit: int, R, x1, g, h, eps: float = 1e-5,
                                     split_row: int = 0, stream=None) -> None:
    """The output projection's fused split-K reduce + residual + RMSNorm."""
    M, H = R.shape
    _check(_lib.mx_debug_reduce_residual_rmsnorm(_ptr(partial), ksplit, _ptr(R), _ptr(x1), _ptr(g),
                                                 _ptr(h), M, H, eps, split_row, _stream(stream)))


def mx_profile_enable(on: bool = True) -> None:
    _check(_lib.mx_profile_enable(1 if on else 0))


def mx_profile_read(max_entries: int = 64) -> dict:
    """{tag: (total_ms, launches)} accumulated since the last read."""
    names = (ctypes.c_char_p * max_entries)()
    ms = (ctypes.c_float * max_entries)()
    cnt = (ctypes.c_int32 * max_entries)()
    n = _lib.mx_profile_read(names, ms, cnt, max_entries)
    return {names[i].decode(): (float(ms[i]), int(cnt[i])) for i in range(n)}
