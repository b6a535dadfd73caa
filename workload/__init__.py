"""Seeded synthetic inputs for the multiplexed layer step.

This module is shared by the oracle side (tests, CPU baseline) and the HIP side
(tests, benchmark).  It holds no arithmetic of the method: it only draws
weights, activations, batch shapes, page tables and cached key/value contents.

Inputs are shaped like the chat-style serving iterations the paper studies
(Section 3.1: long-tailed prompt lengths; Section 5.1: chunked prefill with
2048-token chunks, decode batches of running requests).  The paper measures on a
production trace that is not available here; these synthetic batches stand in
for the per-iteration shape of that trace and reproduce none of its records.

Cached key/value contents are a counter-based function of the physical pool
location (SplitMix64, Steele, Lea and Flood 2014, "Fast splittable pseudorandom
number generators"), implemented once here in numpy and once in
``csrc/mxgen.hip`` for device-side bulk fills; tests check the two agree bit
for bit.
"""
from __future__ import annotations

import math
from dataclasses import dataclass, field
from typing import Dict, List, Optional

import numpy as np

PAGE_SIZE = 16
BF16_NAN = np.uint16(0x7FC0)


# --------------------------------------------------------------------------
# bf16 bit helpers (input encoding only)
# --------------------------------------------------------------------------
def f32_to_bf16_bits(a) -> np.ndarray:
    """Round float32 values to bfloat16, round-to-nearest-even; returns uint16 bits."""
    a = np.ascontiguousarray(a, dtype=np.float32)
    u = a.view(np.uint32).astype(np.uint64)
    rounding = ((u >> np.uint64(16)) & np.uint64(1)) + np.uint64(0x7FFF)
    out = ((u + rounding) >> np.uint64(16)).astype(np.uint16)
    nan = np.isnan(a)
    if nan.any():
        out[nan] = BF16_NAN
    return out


def bf16_bits_to_f32(b) -> np.ndarray:
    b = np.ascontiguousarray(b, dtype=np.uint16)
    return (b.astype(np.uint32) << np.uint32(16)).view(np.float32)


def bf16_bits_to_f64(b) -> np.ndarray:
    return bf16_bits_to_f32(b).astype(np.float64)


# --------------------------------------------------------------------------
# SplitMix64 counter-based generator (host side)
# --------------------------------------------------------------------------
GAMMA = np.uint64(0x9E3779B97F4A7C15)
_M1 = np.uint64(0xBF58476D1CE4E5B9)
_M2 = np.uint64(0x94D049BB133111EB)


def mix64(z):
    """SplitMix64 output function (Stafford variant 13 finaliser)."""
    z = np.asarray(z, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = (z ^ (z >> np.uint64(30))) * _M1
        z = (z ^ (z >> np.uint64(27))) * _M2
    return z ^ (z >> np.uint64(31))


def stream_key(seed: int, kv: int) -> np.uint64:
    """Key of the K (kv=0) or V (kv=1) stream of a pool fill."""
    return np.uint64(mix64(np.uint64((int(seed) * 2 + int(kv)) & 0xFFFFFFFFFFFFFFFF)))


def hash_bf16(key: np.uint64, counter) -> np.ndarray:
    """bf16 bits of the value at ``counter`` of stream ``key``:
    z = mix64(key + (counter + 1) * GAMMA); u = (z >> 40) - 2^23 (a 24-bit signed
    integer); value = float32(u * 2^-23) * float32(sqrt 3), rounded to bf16.
    The value is uniform on [-sqrt 3, sqrt 3), unit variance."""
    c = np.asarray(counter, dtype=np.uint64)
    with np.errstate(over="ignore"):
        z = mix64(np.uint64(key) + (c + np.uint64(1)) * GAMMA)
    u = (z >> np.uint64(40)).astype(np.int64) - 8388608
    f = u.astype(np.float32) * np.float32(2.0 ** -23)
    v = f * np.float32(1.7320508)
    return f32_to_bf16_bits(v)


def pool_counter(page, head, slot, dim, nkv: int, d: int, page_size: int = PAGE_SIZE):
    """Flat element index of pool[page][head][slot][dim]."""
    page = np.asarray(page, dtype=np.uint64)
    return ((page * np.uint64(nkv) + np.uint64(head)) * np.uint64(page_size)
            + np.asarray(slot, dtype=np.uint64)) * np.uint64(d) + np.asarray(dim, dtype=np.uint64)


# --------------------------------------------------------------------------
# Layer shapes
# --------------------------------------------------------------------------
@dataclass(frozen=True)
class LayerConfig:
    name: str
    hidden: int
    ffn: int
    n_q_heads: int
    n_kv_heads: int
    head_dim: int
    rms_eps: float = 1e-5
    rope_theta: float = 1e4
    page_size: int = PAGE_SIZE

    @property
    def scale(self) -> float:
        return 1.0 / math.sqrt(self.head_dim)

    @property
    def qkv_rows(self) -> int:
        return (self.n_q_heads + 2 * self.n_kv_heads) * self.head_dim

    @property
    def kv_bytes_per_token(self) -> int:
        return 2 * self.n_kv_heads * self.head_dim * 2

    @property
    def params(self) -> int:
        H, F = self.hidden, self.ffn
        return (self.qkv_rows * H + H * self.n_q_heads * self.head_dim + 2 * F * H + H * F
                + 2 * H)

    def as_dict(self) -> dict:
        return dict(hidden=self.hidden, ffn=self.ffn, n_q_heads=self.n_q_heads,
                    n_kv_heads=self.n_kv_heads, head_dim=self.head_dim,
                    rms_eps=self.rms_eps, rope_theta=self.rope_theta, scale=self.scale)


# The five layer shapes of the benchmark (tiny parity layer, then 7B, 13B,
# Llama-3-8B and 70B shapes).
CONFIGS: Dict[str, LayerConfig] = {
    "c1": LayerConfig("tiny-256", 256, 1024, 4, 4, 64),
    "c2": LayerConfig("llama7b", 4096, 11008, 32, 32, 128),
    "c3": LayerConfig("llama13b", 5120, 13824, 40, 40, 128),
    "c4": LayerConfig("llama3-8b", 4096, 14336, 32, 8, 128, rope_theta=5e5),
    "c5": LayerConfig("llama70b", 8192, 28672, 64, 8, 128),
}
CONFIG_INDEX = {"c1": 0, "c2": 1, "c3": 2, "c4": 3, "c5": 4}

# Default mixed-prefill sweep per shape.
SWEEPS = {
    "c1": [128],
    "c2": [0, 512],
    "c3": [0, 256, 512, 1024, 2048, 4096],
    "c4": [0, 2048],
    "c5": [0, 1024, 2048, 3072, 4096, 5120, 6144, 7168, 8192],
}

C5_POOL_PAGES = 150_000_000_000 // (PAGE_SIZE * 4096)  # ~150 GB of K+V at 4 KB/token


# --------------------------------------------------------------------------
# Batches
# --------------------------------------------------------------------------
PREFILL, DECODE = 0, 1


@dataclass
class Batch:
    phase: np.ndarray          # int32 [R]
    n_new: np.ndarray          # int32 [R]
    ctx_len: np.ndarray        # int32 [R]
    page_tables: List[np.ndarray]
    pool_pages: int
    page_size: int = PAGE_SIZE
    info: dict = field(default_factory=dict)

    @property
    def R(self) -> int:
        return int(len(self.n_new))

    @property
    def T(self) -> int:
        return int(self.n_new.sum())

    @property
    def prefill_tokens(self) -> int:
        return int(self.n_new[self.phase == PREFILL].sum())

    @property
    def kv_len(self) -> np.ndarray:
        return self.ctx_len + self.n_new

    def page_off(self) -> np.ndarray:
        off = np.zeros(self.R + 1, np.int64)
        for r, t in enumerate(self.page_tables):
            off[r + 1] = off[r] + len(t)
        return off

    def flat_pages(self) -> np.ndarray:
        if not self.page_tables:
            return np.zeros(0, np.int32)
        return np.concatenate(self.page_tables).astype(np.int32)

    def subset(self, reqs) -> "Batch":
        reqs = list(reqs)
        return Batch(self.phase[reqs].copy(), self.n_new[reqs].copy(), self.ctx_len[reqs].copy(),
                     [self.page_tables[r] for r in reqs], self.pool_pages, self.page_size,
                     dict(self.info))


def _pages_needed(kv_len, page_size=PAGE_SIZE):
    return (np.asarray(kv_len, np.int64) + page_size - 1) // page_size


def assign_pages(rng: np.random.Generator, kv_len: np.ndarray, pool_pages: Optional[int],
                 page_size: int = PAGE_SIZE):
    """Page tables drawn from a random permutation of the pool (shuffled pool)."""
    need = _pages_needed(kv_len, page_size)
    total = int(need.sum())
    if pool_pages is None:
        pool_pages = max(2 * total, 1)
    if total > pool_pages:
        raise ValueError("batch does not fit the pool")
    if pool_pages <= 4_000_000:
        chosen = rng.permutation(pool_pages)[:total]
    else:
        chosen = rng.choice(pool_pages, size=total, replace=False)
    tables, off = [], 0
    for n in need:
        tables.append(chosen[off:off + n].astype(np.int32))
        off += int(n)
    return tables, pool_pages


def lognormal_int(rng, median, sigma, lo, hi, size):
    v = np.round(rng.lognormal(mean=math.log(median), sigma=sigma, size=size))
    return np.clip(v, lo, hi).astype(np.int32)


def split_prompts(rng, P: int, median: float, sigma: float) -> List[int]:
    """Prompt lengths ~ round(lognormal(ln median, sigma)), clipped to [1, remaining],
    drawn until they sum to P (the last one truncated)."""
    out, left = [], P
    while left > 0:
        L = int(np.clip(np.round(rng.lognormal(math.log(median), sigma)), 1, left))
        out.append(L)
        left -= L
    return out


def make_batch(cfg_key: str, P: Optional[int] = None, sigma: float = 1.0,
               decode_ctx: Optional[List[int]] = None,
               prefill_lens: Optional[List[int]] = None,
               prefill_ctx: Optional[List[int]] = None,
               pool_pages: Optional[int] = None) -> Batch:
    """Batch of one of the benchmark shapes.  Decode requests come first, then
    prefill chunks.  Explicit ``decode_ctx``/``prefill_lens``/``prefill_ctx``
    override the drawn values (used by tests)."""
    idx = CONFIG_INDEX[cfg_key]
    ss = np.random.SeedSequence(1000 + idx).spawn(6)
    rng_ctx = np.random.default_rng(ss[3])
    rng_len = np.random.default_rng(ss[4])
    rng_pages = np.random.default_rng(ss[5])
    if P is None:
        P = SWEEPS[cfg_key][-1]
    if decode_ctx is None:
        if cfg_key == "c1":
            decode_ctx = rng_ctx.integers(64, 257, size=4)
        elif cfg_key == "c2":
            decode_ctx = rng_ctx.integers(512, 2049, size=64)
        elif cfg_key == "c3":
            decode_ctx = lognormal_int(rng_ctx, 700, sigma, 32, 4096, 128)
        elif cfg_key == "c4":
            decode_ctx = lognormal_int(rng_ctx, 1500, sigma, 32, 8192, 256)
        else:
            decode_ctx = rng_ctx.integers(1024, 16385, size=256)
    decode_ctx = [int(c) for c in decode_ctx]
    if prefill_lens is None:
        if P == 0:
            prefill_lens = []
        elif cfg_key == "c3":
            prefill_lens = split_prompts(rng_len, P, 600, sigma)
        else:
            prefill_lens = [P]
    prefill_lens = [int(v) for v in prefill_lens]
    if prefill_ctx is None:
        prefill_ctx = [0] * len(prefill_lens)
    phase = [DECODE] * len(decode_ctx) + [PREFILL] * len(prefill_lens)
    n_new = [1] * len(decode_ctx) + prefill_lens
    ctx = decode_ctx + [int(c) for c in prefill_ctx]
    phase = np.array(phase, np.int32)
    n_new = np.array(n_new, np.int32)
    ctx = np.array(ctx, np.int32)
    if pool_pages is None:
        if cfg_key == "c1":
            pool_pages = 64
            # redraw the decode contexts until the batch fits in the pool
            while int(_pages_needed(ctx + n_new).sum()) > pool_pages:
                redraw = rng_ctx.integers(64, 257, size=len(decode_ctx))
                ctx[: len(decode_ctx)] = redraw
        elif cfg_key == "c5":
            pool_pages = C5_POOL_PAGES
    tables, pool_pages = assign_pages(rng_pages, ctx + n_new, pool_pages)
    info = dict(config=cfg_key, P=int(sum(prefill_lens)), sigma=sigma,
                n_decode=len(decode_ctx), n_prefill=len(prefill_lens))
    return Batch(phase, n_new, ctx, tables, int(pool_pages), PAGE_SIZE, info)


def custom_batch(rng: np.random.Generator, decode_ctx, prefill, pool_pages=None,
                 page_size: int = PAGE_SIZE) -> Batch:
    """Batch from explicit lists: ``decode_ctx`` contexts, ``prefill`` = list of
    (n_new, ctx_len).  Pages drawn from a shuffled pool (2x need by default)."""
    decode_ctx = [int(c) for c in decode_ctx]
    phase = [DECODE] * len(decode_ctx) + [PREFILL] * len(prefill)
    n_new = [1] * len(decode_ctx) + [int(n) for n, _ in prefill]
    ctx = decode_ctx + [int(c) for _, c in prefill]
    phase = np.array(phase, np.int32)
    n_new = np.array(n_new, np.int32)
    ctx = np.array(ctx, np.int32)
    tables, pool_pages = assign_pages(rng, ctx + n_new, pool_pages, page_size)
    return Batch(phase, n_new, ctx, tables, int(pool_pages), page_size, {})


# --------------------------------------------------------------------------
# Weights and activations
# --------------------------------------------------------------------------
def _streams(cfg_key: str):
    idx = CONFIG_INDEX.get(cfg_key, 7)
    return np.random.SeedSequence(1000 + idx).spawn(6)


def make_weights(cfg: LayerConfig, seed_key: str, std: float = 0.02) -> Dict[str, np.ndarray]:
    """Canonical bf16 weights: rows of w_qkv ordered q, k, v heads; w_gu gate then up.
    Values ~ N(0, std); RMSNorm gains 1 + 0.1 N(0, 1)."""
    ss = _streams(seed_key)
    rw = np.random.default_rng(ss[0])
    rg = np.random.default_rng(ss[1])
    H, F = cfg.hidden, cfg.ffn
    nqd = cfg.n_q_heads * cfg.head_dim

    def normal(shape):
        return f32_to_bf16_bits(rw.standard_normal(shape, dtype=np.float32) * np.float32(std))

    w = {
        "w_qkv": normal((cfg.qkv_rows, H)),
        "w_o": normal((H, nqd)),
        "w_gu": normal((2 * F, H)),
        "w_down": normal((H, F)),
    }
    w["g1"] = f32_to_bf16_bits(1.0 + 0.1 * rg.standard_normal(H, dtype=np.float32))
    w["g2"] = f32_to_bf16_bits(1.0 + 0.1 * rg.standard_normal(H, dtype=np.float32))
    return w


def make_x(cfg: LayerConfig, T: int, seed_key: str) -> np.ndarray:
    rx = np.random.default_rng(_streams(seed_key)[2])
    return f32_to_bf16_bits(rx.standard_normal((T, cfg.hidden), dtype=np.float32))


def kv_seed(cfg_key: str) -> int:
    return 1000 + CONFIG_INDEX.get(cfg_key, 7)


def prior_kv(cfg: LayerConfig, batch: Batch, r: int, seed: int):
    """Host copy of request r's cached keys/values (positions < ctx_len), as the
    pool fill defines them: bf16 bits [ctx_len, nkv, d] for K and for V."""
    n = int(batch.ctx_len[r])
    nkv, d, ps = cfg.n_kv_heads, cfg.head_dim, batch.page_size
    if n == 0:
        z = np.zeros((0, nkv, d), np.uint16)
        return z, z.copy()
    j = np.arange(n)
    page = batch.page_tables[r][j // ps].astype(np.uint64)
    slot = (j % ps).astype(np.uint64)
    c = pool_counter(page[:, None, None], np.arange(nkv, dtype=np.uint64)[None, :, None],
                     slot[:, None, None], np.arange(d, dtype=np.uint64)[None, None, :], nkv, d, ps)
    return hash_bf16(stream_key(seed, 0), c), hash_bf16(stream_key(seed, 1), c)


def prior_kv_concat(cfg: LayerConfig, batch: Batch, seed: int, reqs=None):
    """Cached K/V of the given requests (default all), request-major."""
    reqs = range(batch.R) if reqs is None else reqs
    ks, vs = [], []
    for r in reqs:
        k, v = prior_kv(cfg, batch, r, seed)
        ks.append(k)
        vs.append(v)
    if not ks:
        z = np.zeros((0, cfg.n_kv_heads, cfg.head_dim), np.uint16)
        return z, z.copy()
    return np.concatenate(ks), np.concatenate(vs)


def host_pool(cfg: LayerConfig, batch: Batch, seed: int, poison: bool = True):
    """Whole host pool image (small pools only): hash values at every element,
    bf16 NaN on pages no request owns and on slots at or beyond ctx_len of the
    owning request (when ``poison``).  Returns (k_pool, v_pool) uint16
    [pool_pages, nkv, page_size, d]."""
    nkv, d, ps = cfg.n_kv_heads, cfg.head_dim, batch.page_size
    shape = (batch.pool_pages, nkv, ps, d)
    c = np.arange(int(np.prod(shape)), dtype=np.uint64).reshape(shape)
    k = hash_bf16(stream_key(seed, 0), c)
    v = hash_bf16(stream_key(seed, 1), c)
    if poison:
        for slot in poison_slots(batch):
            k[slot // ps, :, slot % ps, :] = BF16_NAN
            v[slot // ps, :, slot % ps, :] = BF16_NAN
        owned = np.zeros(batch.pool_pages, bool)
        for t in batch.page_tables:
            owned[t] = True
        k[~owned] = BF16_NAN
        v[~owned] = BF16_NAN
    return k, v


def poison_slots(batch: Batch) -> np.ndarray:
    """Slots of owned pages at positions >= ctx_len (not yet valid context)."""
    ps = batch.page_size
    out = []
    for r in range(batch.R):
        tbl = batch.page_tables[r].astype(np.int64)
        pos = np.arange(int(batch.ctx_len[r]), len(tbl) * ps)
        out.append(tbl[pos // ps] * ps + pos % ps)
    return np.concatenate(out) if out else np.zeros(0, np.int64)


def owned_pages_mask(batch: Batch) -> np.ndarray:
    owned = np.zeros(batch.pool_pages, np.uint8)
    for t in batch.page_tables:
        owned[t] = 1
    return owned
