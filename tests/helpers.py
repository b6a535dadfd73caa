"""Shared test helpers: tolerance metric, batch/shape marshalling, device setup.
The oracle side and the HIP side never meet here except through the seeded
inputs of ``workload``."""
from __future__ import annotations

import math

import numpy as np

import workload as wl

TOL = 2e-2  # max relative error per row (bf16 compute, fp32 accumulate)


def rel_err_rows(got, exp) -> np.ndarray:
    """Per row: max_j |got - exp| / max_j |exp| (rows = leading axis)."""
    got = np.asarray(got, np.float64).reshape(len(got), -1)
    exp = np.asarray(exp, np.float64).reshape(len(exp), -1)
    num = np.abs(got - exp).max(axis=1)
    den = np.abs(exp).max(axis=1)
    return num / np.maximum(den, 1e-30)


def assert_rows_close(got, exp, tol=TOL, what=""):
    got = np.asarray(got, np.float64)
    assert np.isfinite(got).all(), f"{what}: non-finite values in the GPU result"
    err = rel_err_rows(got, exp)
    worst = int(np.argmax(err)) if len(err) else 0
    assert len(err) == 0 or err.max() <= tol, \
        f"{what}: max per-row relative error {err.max():.3e} (row {worst}) > {tol}"
    return float(err.max()) if len(err) else 0.0


def mx_batch(mx, b: wl.Batch):
    return mx.Batch(b.phase, b.n_new, b.ctx_len, b.page_tables)


def mx_shape(mx, cfg: wl.LayerConfig, pool_pages: int):
    return mx.attn_shape(cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim, pool_pages)


def mx_cfg(mx, cfg: wl.LayerConfig, pool_pages: int):
    return mx.layer_cfg(cfg.hidden, cfg.ffn, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim,
                        pool_pages, cfg.rms_eps, cfg.rope_theta)


def dev(bits, device="cuda"):
    import torch
    return torch.from_numpy(np.ascontiguousarray(bits, dtype=np.uint16)).to(device)


def host_bits(t) -> np.ndarray:
    return t.cpu().numpy().view(np.uint16)


def bits_to_f64(t) -> np.ndarray:
    return wl.bf16_bits_to_f64(host_bits(t))


def tile_elems(M, K) -> int:
    """Elements of an M x K matrix in the projection-input tile layout: ceil(M/16)
    tile rows of K/32 one-kilobyte tiles plus one unused tile each."""
    return -(-M // 16) * (16 * K + 512)


def to_tiles(a, pad=0x7FC0) -> np.ndarray:
    """[M][K] uint16 -> the projection-input tile layout (flat): tile rows of
    [K/32 + 1][16][32], the last tile of each unused; the padding rows of the
    last tile row and the unused tiles are filled with `pad` (a NaN: a kernel
    that read them would show it)."""
    a = np.asarray(a, np.uint16)
    M, K = a.shape
    M16 = -(-M // 16) * 16
    p = np.full((M16, K + 32), pad, np.uint16)
    p[:M, :K] = a
    return np.ascontiguousarray(p.reshape(M16 // 16, 16, K // 32 + 1, 32).transpose(0, 2, 1, 3)).reshape(-1)


def from_tiles(t, M, K) -> np.ndarray:
    """The inverse of to_tiles: tile layout (device tensor or array) -> [M][K] uint16."""
    a = (host_bits(t) if hasattr(t, "cpu") else np.asarray(t).view(np.uint16)).reshape(-1)
    M16 = -(-M // 16) * 16
    a = a[:tile_elems(M, K)].reshape(M16 // 16, K // 32 + 1, 16, 32)[:, :K // 32]
    return np.ascontiguousarray(a.transpose(0, 2, 1, 3).reshape(M16, K)[:M])


def tiles_unwritten(t, M, K) -> np.ndarray:
    """The elements of a tile-layout buffer that hold no matrix element (padding
    rows, unused tiles), as uint16."""
    a = (host_bits(t) if hasattr(t, "cpu") else np.asarray(t).view(np.uint16)).reshape(-1)
    real = to_tiles(np.ones((M, K), np.uint16), pad=0).astype(bool)
    return a[:len(real)][~real]


def sample_rows(b: wl.Batch, rng, n_decode=16, n_prefill_random=62):
    """All decode rows of n_decode random decode requests, plus the first, the
    last and n_prefill_random random rows of every prefill chunk."""
    start = np.concatenate([[0], np.cumsum(b.n_new)])
    dec = [r for r in range(b.R) if b.phase[r] == wl.DECODE]
    rows = [int(start[r]) for r in rng.choice(dec, size=min(n_decode, len(dec)), replace=False)]
    for r in range(b.R):
        if b.phase[r] != wl.PREFILL:
            continue
        n = int(b.n_new[r])
        pick = {0, n - 1}
        pick.update(rng.choice(n, size=min(n_prefill_random, n), replace=False).tolist())
        rows += [int(start[r]) + i for i in sorted(pick)]
    return np.array(sorted(set(rows)), np.int64)


def truncated_subbatch(b: wl.Batch, rows):
    """The requests that own the sampled rows, each cut after its last sampled
    row (later tokens cannot influence earlier rows: attention is causal).
    Returns (sub_batch, request ids, row indices inside the sub-batch, token
    indices in the full batch of the sub-batch's tokens)."""
    start = np.concatenate([[0], np.cumsum(b.n_new)])
    req_of = np.searchsorted(start, rows, side="right") - 1
    reqs = sorted(set(req_of.tolist()))
    n_new, tok_idx, sub_rows, off = [], [], [], 0
    for r in reqs:
        last = int(max(rows[req_of == r])) - int(start[r])
        n_new.append(last + 1)
        tok_idx += list(range(int(start[r]), int(start[r]) + last + 1))
        for t in rows[req_of == r]:
            sub_rows.append(off + int(t) - int(start[r]))
        off += last + 1
    sub = b.subset(reqs)
    sub.n_new = np.array(n_new, np.int32)
    return sub, reqs, np.array(sub_rows, np.int64), np.array(tok_idx, np.int64)


def bf16_half_ulp(v) -> np.ndarray:
    """Half the bf16 ulp at each value's binade (8 significant bits): the most
    that rounding a real number to the stored bf16 value v can have moved it."""
    v = np.abs(np.asarray(v, np.float64))
    e = np.floor(np.log2(np.maximum(v, 2.0 ** -126)))
    return 2.0 ** (e - 8)


def branch_err_rows(got_branch, exp_branch, allowance) -> tuple:
    """Per-row error of a residual branch recovered from bf16-stored sums.
    The GPU stores base + branch rounded once to bf16, so the branch read back
    as (stored - base) carries up to `allowance` (half an ulp of each stored
    value involved) per element on top of the kernel's own error.  Returns
    (raw, net): max_j |got - exp| / max_j |exp| without and with the allowance
    taken off each element's difference."""
    got = np.asarray(got_branch, np.float64).reshape(len(got_branch), -1)
    exp = np.asarray(exp_branch, np.float64).reshape(len(exp_branch), -1)
    al = np.asarray(allowance, np.float64).reshape(got.shape)
    diff = np.abs(got - exp)
    den = np.maximum(np.abs(exp).max(axis=1), 1e-30)
    return diff.max(axis=1) / den, np.maximum(diff - al, 0.0).max(axis=1) / den
