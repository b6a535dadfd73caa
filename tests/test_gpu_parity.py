"""GPU parity of the HIP path (through the C ABI) against the fp64 oracle on the
same seeded inputs.  Integer/byte work is compared bit for bit; floating point
per row with max relative error 2e-2 (bf16 compute, fp32 accumulate).

Unused pool slots (pages no request owns, and slots at or beyond each request's
cached length before the step) are filled with bf16 NaN, so any read of a slot
outside a request's keys poisons the result and fails the finiteness check."""
import math
import sys

import numpy as np
import pytest

import oracle
import workload as wl
from helpers import (TOL, assert_rows_close, bf16_half_ulp, bits_to_f64, branch_err_rows, dev,
                     from_tiles, host_bits, mx_batch, mx_cfg, mx_shape, rel_err_rows,
                     sample_rows, tile_elems, tiles_unwritten, to_tiles, truncated_subbatch)

pytestmark = pytest.mark.gpu

torch = pytest.importorskip("torch")
if not torch.cuda.is_available():
    pytest.skip("no GPU", allow_module_level=True)

import paper_2606_16264_amd as mx  # noqa: E402
import workload.device as wdev      # noqa: E402


def say(*a):
    print(*a, flush=True)
    sys.stdout.flush()


def ws_tensor(nbytes):
    return torch.empty(int(nbytes), dtype=torch.uint8, device="cuda")


def sync():
    torch.cuda.synchronize()


# ----------------------------------------------------------------------- generator
def test_device_pool_fill_matches_host():
    cfg = wl.CONFIGS["c1"]
    b = wl.make_batch("c1")
    say("case: device pool fill c1")
    k, v = wdev.alloc_pools(cfg, b.pool_pages)
    wdev.fill_pools(k, v, cfg, b, 1000, poison=True)
    sync()
    hk, hv = wl.host_pool(cfg, b, 1000, poison=True)
    np.testing.assert_array_equal(wdev.k_pool_canonical(k), hk)
    np.testing.assert_array_equal(wdev.v_pool_canonical(v), hv)


# ----------------------------------------------------------------------- token map
TOKEN_MAP_CASES = [("c1", 128), ("c2", 512), ("c3", 4096), ("c4", 2048), ("c5", 8192)]


@pytest.mark.parametrize("key,P", TOKEN_MAP_CASES)
def test_token_map_bit_exact(key, P):
    say(f"case: token map {key} P={P}")
    cfg = wl.CONFIGS[key]
    b = wl.make_batch(key, P)
    mb = mx_batch(mx, b)
    shape = mx_shape(mx, cfg, b.pool_pages)
    ws = ws_tensor(mx.mx_workspace_bytes_for(mb, shape=shape))
    T = b.T
    tr = torch.empty(T, dtype=torch.int32, device="cuda")
    tp = torch.empty(T, dtype=torch.int32, device="cuda")
    ts = torch.empty(T, dtype=torch.int64, device="cuda")
    mx.mx_debug_token_map(mb, shape, tr, tp, ts, ws)
    sync()
    ref = oracle.token_map(b.n_new, b.ctx_len, b.page_tables, 16)
    np.testing.assert_array_equal(tr.cpu().numpy(), ref.tok_req)
    np.testing.assert_array_equal(tp.cpu().numpy(), ref.tok_pos)
    np.testing.assert_array_equal(ts.cpu().numpy(), ref.tok_slot)


def boundary_batch(rng, pool=None):
    """Decodes at and around page boundaries, prefills with and without a cached prefix."""
    return wl.custom_batch(rng, [1, 15, 16, 17, 31, 32, 33, 100, 255, 256, 1000],
                           [(1, 0), (7, 0), (16, 0), (64, 0), (65, 0), (130, 0), (50, 17),
                            (33, 48), (16, 16)], pool_pages=pool)


# ----------------------------------------------------------------------- KV append / gather
@pytest.mark.parametrize("nkv,d", [(4, 64), (8, 128), (2, 128)])
def test_kv_append_bit_exact(nkv, d):
    say(f"case: kv append nkv={nkv} d={d}")
    rng = np.random.default_rng(20 + nkv + d)
    cfg = wl.LayerConfig("t", 256, 256, nkv, nkv, d)
    b = boundary_batch(rng)
    k, v = wdev.alloc_pools(cfg, b.pool_pages)
    wdev.fill_pools(k, v, cfg, b, 7, poison=True)
    sync()
    k0, v0 = wdev.k_pool_canonical(k), wdev.v_pool_canonical(v)
    kn = rng.integers(0, 65536, (b.T, nkv, d), dtype=np.uint16)
    vn = rng.integers(0, 65536, (b.T, nkv, d), dtype=np.uint16)
    mb = mx_batch(mx, b)
    shape = mx_shape(mx, cfg, b.pool_pages)
    ws = ws_tensor(mx.mx_workspace_bytes_for(mb, shape=shape))
    mx.mx_kv_append(mb, shape, dev(kn), dev(vn), k, v, ws)
    sync()
    ek, ev = oracle.kv_append(b.n_new, b.ctx_len, b.page_tables, kn, vn, k0, v0)
    np.testing.assert_array_equal(wdev.k_pool_canonical(k), ek)
    np.testing.assert_array_equal(wdev.v_pool_canonical(v), ev)


def test_gather_bit_exact():
    say("case: gather")
    rng = np.random.default_rng(31)
    cfg = wl.LayerConfig("t", 256, 256, 4, 4, 128)
    b = boundary_batch(rng)
    k, v = wdev.alloc_pools(cfg, b.pool_pages)
    wdev.fill_pools(k, v, cfg, b, 9, poison=False)
    sync()
    mb = mx_batch(mx, b)
    shape = mx_shape(mx, cfg, b.pool_pages)
    ws = ws_tensor(mx.mx_workspace_bytes_for(mb, shape=shape))
    hk, hv = wl.host_pool(cfg, b, 9, poison=False)
    for r in (0, 3, 10, 13, 17, 19):
        L = int(b.kv_len[r])
        ko = torch.empty((L, 4, 128), dtype=torch.uint16, device="cuda")
        vo = torch.empty((L, 4, 128), dtype=torch.uint16, device="cuda")
        mx.mx_debug_gather(mb, shape, r, k, v, ko, vo, ws)
        sync()
        j = np.arange(L)
        pg = b.page_tables[r][j // 16]
        np.testing.assert_array_equal(host_bits(ko), hk[pg, :, j % 16])
        np.testing.assert_array_equal(host_bits(vo), hv[pg, :, j % 16])


# ----------------------------------------------------------------------- attention
def attention_case(cfg, b, seed, rng, needle=False):
    """Pools filled (NaN-poisoned), new K/V appended through the ABI, random q.
    Returns device tensors and the oracle's expected output."""
    k, v = wdev.alloc_pools(cfg, b.pool_pages)
    wdev.fill_pools(k, v, cfg, b, seed, poison=True)
    nq, nkv, d = cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    kn = wl.f32_to_bf16_bits(rng.uniform(-math.sqrt(3), math.sqrt(3), (b.T, nkv, d)))
    vn = wl.f32_to_bf16_bits(rng.uniform(-math.sqrt(3), math.sqrt(3), (b.T, nkv, d)))
    qf = rng.standard_normal((b.T, nq, d)).astype(np.float32)
    kp, vp = wl.prior_kv_concat(cfg, b, seed)
    if needle:
        # per request: the key of one cached position is set to 20x the first
        # q head's direction (scaled by sqrt(d)), so the softmax is dominated by it
        start = np.concatenate([[0], np.cumsum(b.n_new)])
        pstart = np.concatenate([[0], np.cumsum(b.ctx_len)])
        for r in range(b.R):
            if b.ctx_len[r] == 0:
                continue
            j = int(rng.integers(0, int(b.ctx_len[r])))
            t = int(start[r])
            for g in range(nkv):
                h0 = g * (nq // nkv)
                qd = qf[t:t + int(b.n_new[r]), h0].mean(axis=0)
                qf[t:t + int(b.n_new[r]), g * (nq // nkv):(g + 1) * (nq // nkv)] = qd
                kp[pstart[r] + j, g] = wl.f32_to_bf16_bits(20.0 * qd / np.linalg.norm(qd) * math.sqrt(d) / 4)
        # write the needle keys into the device pool
        kh = wdev.k_pool_canonical(k)
        for r in range(b.R):
            for j in range(int(b.ctx_len[r])):
                page = b.page_tables[r][j // 16]
                kh[page, :, j % 16] = kp[pstart[r] + j]
        k.copy_(torch.from_numpy(wdev.k_pool_blocked(kh)).cuda())
    q = wl.f32_to_bf16_bits(qf)
    mb = mx_batch(mx, b)
    shape = mx_shape(mx, cfg, b.pool_pages)
    ws = ws_tensor(mx.mx_workspace_bytes_for(mb, shape=shape))
    mx.mx_kv_append(mb, shape, dev(kn), dev(vn), k, v, ws)
    # oracle inputs: cached prefix then the new tokens, per request
    ks, vs, t0, p0 = [], [], 0, 0
    for r in range(b.R):
        c, n = int(b.ctx_len[r]), int(b.n_new[r])
        ks += [kp[p0:p0 + c], kn[t0:t0 + n]]
        vs += [vp[p0:p0 + c], vn[t0:t0 + n]]
        t0 += n
        p0 += c
    kc = wl.bf16_bits_to_f64(np.concatenate(ks))
    vc = wl.bf16_bits_to_f64(np.concatenate(vs))
    off = np.concatenate([[0], np.cumsum(b.kv_len)])[:-1]
    exp = oracle.attention_contig(b.n_new, b.ctx_len, wl.bf16_bits_to_f64(q), kc, vc, off,
                                  cfg.scale)
    return dict(k=k, v=v, q=dev(q), mb=mb, shape=shape, ws=ws, exp=exp, vc=vc, off=off)


ATTN_SHAPES = [(4, 4, 64), (8, 8, 128), (32, 8, 128), (16, 2, 128), (32, 1, 64), (64, 8, 128)]


@pytest.mark.parametrize("nq,nkv,d", ATTN_SHAPES)
def test_paged_attn_boundaries(nq, nkv, d):
    say(f"case: paged attn boundaries nq={nq} nkv={nkv} d={d}")
    rng = np.random.default_rng(100 + nq + nkv + d)
    cfg = wl.LayerConfig("t", 256, 256, nq, nkv, d)
    b = boundary_batch(rng)
    c = attention_case(cfg, b, 11, rng)
    out = torch.empty((b.T, nq, d), dtype=torch.uint16, device="cuda")
    mx.mx_paged_attn(c["mb"], c["shape"], c["q"], c["k"], c["v"], out, c["ws"])
    sync()
    err = assert_rows_close(bits_to_f64(out).reshape(b.T * nq, d), c["exp"].reshape(b.T * nq, d),
                            what="attention")
    say(f"  max row rel err {err:.2e}")


# Prefill tiles of 128 query rows (two blocks of 16 per wave): chunks that
# fill a tile exactly, spill one row into the next, end inside a wave's second
# block, and continue a cached prefix
@pytest.mark.parametrize("nq,nkv,d", [(8, 8, 128), (32, 8, 128), (4, 4, 64)])
def test_paged_attn_prefill_tiles(nq, nkv, d):
    say(f"case: paged attn prefill tiles nq={nq} nkv={nkv} d={d}")
    rng = np.random.default_rng(200 + nq + nkv + d)
    cfg = wl.LayerConfig("t", 256, 256, nq, nkv, d)
    b = wl.custom_batch(rng, [5, 600], [(128, 0), (129, 40), (256, 7), (383, 300), (17, 0), (48, 1)])
    c = attention_case(cfg, b, 14, rng)
    out = torch.empty((b.T, nq, d), dtype=torch.uint16, device="cuda")
    mx.mx_paged_attn(c["mb"], c["shape"], c["q"], c["k"], c["v"], out, c["ws"])
    sync()
    err = assert_rows_close(bits_to_f64(out).reshape(b.T * nq, d), c["exp"].reshape(b.T * nq, d),
                            what="attention")
    say(f"  max row rel err {err:.2e}")


@pytest.mark.parametrize("key", ["c2", "c4"])
def test_paged_attn_long_contexts_split(key):
    """Long decode contexts (several key splits and the merge) at a real shape."""
    say(f"case: paged attn long contexts {key}")
    rng = np.random.default_rng(5)
    cfg = wl.CONFIGS[key]
    b = wl.custom_batch(rng, [3000, 8191, 16384, 777, 4096, 2048, 16, 5000],
                        [(300, 0), (128, 900)])
    c = attention_case(cfg, b, 12, rng)
    out = torch.empty((b.T, cfg.n_q_heads, cfg.head_dim), dtype=torch.uint16, device="cuda")
    mx.mx_paged_attn(c["mb"], c["shape"], c["q"], c["k"], c["v"], out, c["ws"])
    sync()
    n = cfg.n_q_heads
    assert_rows_close(bits_to_f64(out).reshape(-1, cfg.head_dim),
                      c["exp"].reshape(-1, cfg.head_dim), what="attention")
    # deterministic: a second launch is bit-identical
    out2 = torch.empty_like(out)
    mx.mx_paged_attn(c["mb"], c["shape"], c["q"], c["k"], c["v"], out2, c["ws"])
    sync()
    assert torch.equal(out, out2)


def test_paged_attn_needle():
    say("case: paged attn needle")
    rng = np.random.default_rng(6)
    cfg = wl.LayerConfig("t", 256, 256, 8, 2, 128)
    b = wl.custom_batch(rng, [40, 300, 1000, 33], [(20, 70)])
    c = attention_case(cfg, b, 13, rng, needle=True)
    out = torch.empty((b.T, 8, 128), dtype=torch.uint16, device="cuda")
    mx.mx_paged_attn(c["mb"], c["shape"], c["q"], c["k"], c["v"], out, c["ws"])
    sync()
    assert_rows_close(bits_to_f64(out).reshape(-1, 128), c["exp"].reshape(-1, 128),
                      what="attention (needle)")


# ----------------------------------------------------------------------- GEMM
CANARY = 0x7FC1  # a NaN pattern no GEMM output takes


def gemm_case(M, N, K, epi, tile_cfg=-1, ksplit=0, b_tiled=False):
    """C = epi(A B^T) through the C-ABI against the oracle; C sits between two
    canary rows on each side, which must come back untouched.  b_tiled: the
    weights go in as the layer step's packed 16 x 32 tiles."""
    say(f"case: gemm M={M} N={N} K={K} epi={epi} cfg={tile_cfg} ksplit={ksplit} tiled={b_tiled}")
    rng = np.random.default_rng(M + N + K + epi)
    a = wl.f32_to_bf16_bits(rng.standard_normal((M, K), dtype=np.float32))
    w = wl.f32_to_bf16_bits(rng.standard_normal((N, K), dtype=np.float32) * 0.02)
    r = wl.f32_to_bf16_bits(rng.standard_normal((M, N), dtype=np.float32))
    ncol = N // 2 if epi == 2 else N
    # filled and checked through the int16 view: few device ops exist for uint16;
    # C starts 16-byte aligned after at least two canary rows
    lead = -(-2 * ncol // 8) * 8
    buf16 = torch.full((lead + (M + 2) * ncol,), CANARY, dtype=torch.int16, device="cuda")
    C = buf16.view(torch.uint16)[lead:lead + M * ncol].view(M, ncol)
    need = mx.mx_debug_gemm_ws_bytes(M, N, K) if tile_cfg < 0 else \
        (ksplit * M * N * 4 if ksplit > 1 else 0)
    ws = ws_tensor(max(need, 256))
    n_c = M * ncol
    if b_tiled:
        # the layer's layouts: A (NaN in its padding rows and unused tiles, never
        # read) and the SwiGLU output in the tile layout
        wt = np.ascontiguousarray(w.reshape(N // 16, 16, K // 32, 32).transpose(0, 2, 1, 3))
        n_c = tile_elems(M, ncol) if epi == 2 else M * ncol
        buf16 = torch.full((lead + n_c + 2 * ncol,), CANARY, dtype=torch.int16, device="cuda")
        C = buf16.view(torch.uint16)[lead:lead + n_c]
        if epi != 2:
            C = C.view(M, ncol)
        mx.mx_debug_gemm(dev(to_tiles(a)), dev(wt.reshape(-1)), C, dev(r) if epi == 1 else None,
                         epi, ws, tile_cfg=tile_cfg, ksplit=ksplit, tiled=True, M=M, N=N, K=K)
    else:
        mx.mx_debug_gemm(dev(a), dev(w), C, dev(r) if epi == 1 else None, epi, ws,
                         tile_cfg=tile_cfg, ksplit=ksplit)
    sync()
    guard = torch.cat([buf16[:lead], buf16[lead + n_c:]]).cpu().numpy()
    assert (guard == CANARY).all(), "GEMM wrote outside C"
    if b_tiled and epi == 2:
        assert (tiles_unwritten(C, M, ncol).view(np.int16) == CANARY).all(), \
            "GEMM wrote a padding row or an unused tile of C"
        C = torch.from_numpy(from_tiles(C, M, ncol))
    # every row at small shapes, sampled rows keep the fp64 reference cheap at large ones
    if M * N * K <= (1 << 31):
        rows = np.arange(M)
    else:
        rows = np.unique(np.concatenate([[0, M - 1], rng.integers(0, M, size=min(M, 48))]))
    acc = oracle.linear(wl.bf16_bits_to_f64(a[rows]), w)
    if epi == 1:
        exp = acc + wl.bf16_bits_to_f64(r[rows])
    elif epi == 2:
        # packed rows: 32-row blocks alternate gate and up of the same features
        blocks = acc.reshape(len(rows), N // 64, 2, 32)
        exp = oracle.silu_mul(np.concatenate([blocks[:, :, 0].reshape(len(rows), -1),
                                              blocks[:, :, 1].reshape(len(rows), -1)], axis=1))
    else:
        exp = acc
    assert_rows_close(bits_to_f64(C)[rows], exp, what="gemm")


@pytest.mark.parametrize("M,N,K,epi", [
    (1, 768, 256, 0), (64, 12288, 4096, 0), (132, 1024, 256, 1), (576, 4096, 4096, 1),
    (577, 2048, 512, 2), (1000, 22016, 4096, 2), (2304, 6144, 4096, 0), (256, 4096, 11008, 1),
    (8, 256, 1024, 2),
])
def test_gemm_matches_oracle(M, N, K, epi):
    gemm_case(M, N, K, epi)


# every tile shape with every epilogue, ragged M and N edges, with and without a K split
@pytest.mark.parametrize("tile_cfg", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("M,N,K,epi,ksplit", [
    (577, 2048, 512, 2, 1), (300, 1344, 768, 0, 1), (131, 1088, 512, 1, 1),
    (97, 640, 1024, 2, 2), (33, 384, 2048, 1, 4), (257, 320, 256, 0, 2),
])
def test_gemm_forced_tile_shapes(tile_cfg, M, N, K, epi, ksplit):
    gemm_case(M, N, K, epi, tile_cfg=tile_cfg, ksplit=ksplit)


# The packed 16 x 32 weight tiles the layer step reads, through every tile shape:
# ragged M and N (N a multiple of 16 only), every epilogue, with and without a K split
@pytest.mark.parametrize("tile_cfg", [0, 1, 2, 3, 4])
@pytest.mark.parametrize("M,N,K,epi,ksplit", [
    (577, 1040, 512, 0, 1), (131, 2048, 1024, 2, 2), (64, 4096, 2048, 1, 4), (300, 784, 768, 1, 1),
])
def test_gemm_tiled_weights(tile_cfg, M, N, K, epi, ksplit):
    gemm_case(M, N, K, epi, tile_cfg=tile_cfg, ksplit=ksplit, b_tiled=True)


# N not a multiple of 4: the element-wise split-K reduce (plain and residual)
@pytest.mark.parametrize("tile_cfg", [0, 3])
@pytest.mark.parametrize("M,N,K,epi,ksplit", [(131, 1090, 512, 1, 2), (70, 775, 1024, 0, 4)])
def test_gemm_ragged_n_split(tile_cfg, M, N, K, epi, ksplit):
    gemm_case(M, N, K, epi, tile_cfg=tile_cfg, ksplit=ksplit)


# K splits that do not divide the K / 64 chunks: split z takes chunks
# [z C / S, (z + 1) C / S), so the splits differ in length by one chunk
@pytest.mark.parametrize("tile_cfg,b_tiled", [(3, False), (1, False), (3, True), (0, True)])
@pytest.mark.parametrize("M,N,K,epi,ksplit", [
    (70, 640, 320, 1, 3), (131, 1024, 1344, 0, 8), (64, 2048, 11008, 1, 8), (33, 768, 704, 2, 5),
])
def test_gemm_uneven_split(tile_cfg, b_tiled, M, N, K, epi, ksplit):
    gemm_case(M, N, K, epi, tile_cfg=tile_cfg, ksplit=ksplit, b_tiled=b_tiled)


# More 256 x 256 tiles than the chip holds workgroups at once (several rounds
# of the XCD-grouped tile order over a ragged tile grid): ragged M and N edges,
# every epilogue, row-major and tiled operands, short K (8 to 16 slices of the
# four-stage ring, one of them not a multiple of four).
@pytest.mark.parametrize("M,N,K,epi,b_tiled", [
    (4112, 4160, 256, 0, False), (4100, 4352, 384, 1, False), (4112, 4160, 512, 1, True),
    (4097, 8320, 256, 2, True), (4112, 4160, 320, 0, True),
])
def test_gemm_many_tiles_per_workgroup(M, N, K, epi, b_tiled):
    gemm_case(M, N, K, epi, tile_cfg=0, ksplit=1, b_tiled=b_tiled)


# ----------------------------------------------------------------------- layer step
def pack_layer(cfg, b, w):
    c = mx_cfg(mx, cfg, b.pool_pages)
    packed = torch.empty(mx.mx_packed_weights_bytes(c), dtype=torch.uint8, device="cuda")
    dw = {k: dev(v) for k, v in w.items()}
    mx.mx_pack_weights(c, dw, packed)
    sync()
    return c, packed


def run_layer(cfg, b, w, x, seed, reps=1, keep_before=False):
    c, packed = pack_layer(cfg, b, w)
    if b.pool_pages * cfg.kv_bytes_per_token * 16 > (16 << 30):
        # a pool of this size (the 70B shape's is ~150 GB) must not land next
        # to a cached block of an earlier one: hand cached memory back first
        torch.cuda.empty_cache()
    k, v = wdev.alloc_pools(cfg, b.pool_pages)
    wdev.fill_pools(k, v, cfg, b, seed, poison=True)
    before = dict(k0=k.clone(), v0=v.clone()) if keep_before else {}
    mb = mx_batch(mx, b)
    ws = ws_tensor(mx.mx_workspace_bytes_for(mb, cfg=c))
    xd = dev(x)
    y = torch.empty_like(xd)
    for _ in range(reps):
        mx.mx_layer_step(mb, c, packed, xd, y, k, v, ws)
    sync()
    off = mx.mx_layer_workspace_offsets(mb, c)
    T, H, F = b.T, cfg.hidden, cfg.ffn
    nqd = cfg.n_q_heads * cfg.head_dim

    def view(name, cols):
        o = off[name]
        return ws[o:o + T * cols * 2].view(torch.uint16).reshape(T, cols)

    def view_tiled(name, cols):  # a projection input: tile rows of [cols/32 + 1][16][32]
        o = off[name]
        T16 = -(-T // 16) * 16
        t = ws[o:o + tile_elems(T, cols) * 2].view(torch.int16)
        t = t.reshape(T16 // 16, cols // 32 + 1, 16, 32)[:, :cols // 32]
        return t.permute(0, 2, 1, 3).reshape(T16, cols)[:T].contiguous().view(torch.uint16)

    return dict(y=y, k=k, v=v, q=view("q", nqd), o=view_tiled("o", nqd), x1=view("x1", H),
                a=view_tiled("a", F), h2=view_tiled("h", H), **before)


def staged_attention(cfg, sub, x_sub, w, kp, vp, sub_rows):
    """Attention output of the evaluated rows from an oracle pipeline that
    stores each stage boundary in bf16 exactly where the HIP path does
    (RMSNorm output h; post-RoPE q and k; v), with every step computed by the
    pinned oracle functions (rmsnorm, linear, rope, attention) in fp64.  This
    isolates the attention kernel's own arithmetic (bf16 probabilities, fp32
    accumulation) from the bf16 storage of its inputs, which attention can
    amplify for short, sharply peaked contexts.  Oracle values only."""
    rnd = lambda a: wl.bf16_bits_to_f64(wl.f32_to_bf16_bits(np.asarray(a, np.float32)))
    H, nq, nkv, d = cfg.hidden, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    start = np.concatenate([[0], np.cumsum(sub.n_new)])
    pstart = np.concatenate([[0], np.cumsum(sub.ctx_len)])
    pos_all = np.concatenate([np.arange(c, c + n) for n, c in zip(sub.n_new, sub.ctx_len)])
    h = rnd(oracle.rmsnorm(wl.bf16_bits_to_f64(x_sub), wl.bf16_bits_to_f64(w["g1"]), cfg.rms_eps))
    k = oracle.linear(h, w["w_qkv"][nq * d:(nq + nkv) * d]).reshape(-1, nkv, d)
    v = oracle.linear(h, w["w_qkv"][(nq + nkv) * d:]).reshape(-1, nkv, d)
    k = rnd(oracle.rope(k, pos_all, cfg.rope_theta))
    v = rnd(v)
    q = oracle.linear(h[sub_rows], w["w_qkv"][:nq * d]).reshape(-1, nq, d)
    q = rnd(oracle.rope(q, pos_all[sub_rows], cfg.rope_theta))
    ks, vs = [], []
    for r in range(sub.R):
        c, n = int(sub.ctx_len[r]), int(sub.n_new[r])
        ks += [wl.bf16_bits_to_f64(kp[pstart[r]:pstart[r] + c]), k[start[r]:start[r] + n]]
        vs += [wl.bf16_bits_to_f64(vp[pstart[r]:pstart[r] + c]), v[start[r]:start[r] + n]]
    kc, vc = np.concatenate(ks), np.concatenate(vs)
    koff = np.concatenate([[0], np.cumsum(sub.ctx_len + sub.n_new)])
    req_of = np.searchsorted(start, sub_rows, side="right") - 1
    return oracle.attention_contig(np.ones(len(sub_rows), np.int32),
                                   pos_all[sub_rows].astype(np.int32), q, kc, vc, koff[req_of],
                                   cfg.scale)


def check_layer(cfg, b, got, exp, rows_gpu, what, o_ref=None, x=None, branch_allowance=True):
    """Stage-by-stage comparison of the GPU iteration with the oracle on the
    evaluated rows.  Gated at 2e-2 (max relative error per row) against the
    exact oracle: q, x1, h2, the SwiGLU output a, the layer output y, and the
    residual branches with the residual stripped: the attention branch x1 - x,
    the MLP branch y - x1 and their sum y - x (x: the bf16 input bits of the
    whole batch).  A branch can be small next to the residual x ~ N(0, 1), so
    an error in it would hide under y or x1 alone.  The GPU stores x1 and y in
    bf16, rounded once; a branch read back from them carries up to half an ulp
    of each stored value involved, which is taken off each element's
    difference before the 2e-2 gate (branch_allowance; False gates the raw
    difference).  The attention output o is gated at 2e-2 per head row against
    the stage-emulating oracle pipeline (o_ref, see staged_attention); its
    error against the exact oracle is reported per head row and per token row."""
    d = cfg.head_dim
    n = len(rows_gpu)
    g = lambda name: bits_to_f64(got[name])[rows_gpu]
    errs = {
        "q": rel_err_rows(g("q").reshape(-1, d), exp.q.reshape(-1, d)).max(),
        "o_vs_exact": rel_err_rows(g("o").reshape(-1, d), exp.o.reshape(-1, d)).max(),
        "o_row_vs_exact": rel_err_rows(g("o").reshape(n, -1), exp.o.reshape(n, -1)).max(),
        "x1": rel_err_rows(g("x1"), exp.x1).max(),
        "h2": rel_err_rows(g("h2"), exp.h2).max(),
        "a": rel_err_rows(g("a"), exp.a).max(),
        "y": rel_err_rows(g("y"), exp.y).max(),
    }
    if o_ref is not None:
        errs["o"] = rel_err_rows(g("o").reshape(-1, d), o_ref.reshape(-1, d)).max()
    branches = {}
    if x is not None:
        xr = wl.bf16_bits_to_f64(np.asarray(x)[rows_gpu])
        x1g, yg = g("x1"), g("y")
        hx1, hy = bf16_half_ulp(x1g), bf16_half_ulp(yg)
        branches = {"x1-x": (x1g - xr, exp.x1 - xr, hx1),
                    "y-x1": (yg - x1g, exp.y - exp.x1, hy),
                    "y-x": (yg - xr, exp.y - xr, hx1 + hy)}
        for name, (gb, eb, al) in branches.items():
            raw, net = branch_err_rows(gb, eb, al if branch_allowance else np.zeros_like(al))
            errs[f"{name}_raw"] = raw.max()
            errs[name] = net.max()
    say(f"  {what} stage errors: " + ", ".join(f"{k}={v:.2e}" for k, v in errs.items()))
    for name in ("q", "x1", "h2", "a", "y"):
        assert_rows_close(g(name).reshape(n, -1), getattr(exp, name).reshape(n, -1),
                          what=f"{what} {name}")
    for name in branches:
        assert np.isfinite(errs[name]) and errs[name] <= TOL, \
            f"{what} branch {name}: max per-row relative error {errs[name]:.3e} > {TOL}"
    if o_ref is not None:
        assert_rows_close(g("o").reshape(-1, d), o_ref.reshape(-1, d), what=f"{what} attention o")
    return errs


def check_pool_rows(cfg, b, got, exp_k, exp_v, tok_idx):
    """New keys/values at their slots (tolerance) for the given tokens."""
    tm = oracle.token_map(b.n_new, b.ctx_len, b.page_tables, 16)
    slots = tm.tok_slot[tok_idx]
    pg = torch.from_numpy(slots // 16).cuda()
    sl = torch.from_numpy(slots % 16).cuda()
    # uint16 tensors cannot be gathered on the device; gather their int16 view
    kk = got["k"].view(torch.int16)[pg, :, :, sl].view(torch.uint16)  # [n][nkv][d/32][32]
    vv = got["v"].view(torch.int16)[pg, :, :, sl].view(torch.uint16)
    assert_rows_close(bits_to_f64(kk).reshape(-1, cfg.head_dim),
                      exp_k.reshape(-1, cfg.head_dim), what="appended k")
    assert_rows_close(bits_to_f64(vv).reshape(-1, cfg.head_dim),
                      exp_v.reshape(-1, cfg.head_dim), what="appended v")


def test_layer_step_c1_full():
    say("case: layer step c1 (all rows)")
    cfg = wl.CONFIGS["c1"]
    b = wl.make_batch("c1")
    w = wl.make_weights(cfg, "c1")
    x = wl.make_x(cfg, b.T, "c1")
    got = run_layer(cfg, b, w, x, wl.kv_seed("c1"), reps=2)
    kp, vp = wl.prior_kv_concat(cfg, b, wl.kv_seed("c1"))
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = np.arange(b.T)
    o_ref = staged_attention(cfg, b, x, w, kp, vp, rows)
    errs = check_layer(cfg, b, got, exp, rows, "c1", o_ref, x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, rows)
    say("  errors", {k: f"{v:.2e}" for k, v in errs.items()})


SMALL_GQA = wl.LayerConfig("small-gqa", 512, 1408, 8, 2, 128, rope_theta=5e5)


def test_layer_step_small_gqa_full():
    say("case: layer step small GQA (all rows)")
    cfg = SMALL_GQA
    rng = np.random.default_rng(77)
    b = wl.custom_batch(rng, [1, 16, 33, 500, 1500, 64, 17], [(200, 0), (70, 33), (1, 0)])
    ws = {k: wl.f32_to_bf16_bits(rng.standard_normal(s, dtype=np.float32) * 0.02) for k, s in (
        ("w_qkv", (cfg.qkv_rows, cfg.hidden)), ("w_o", (cfg.hidden, 1024)),
        ("w_gu", (2 * cfg.ffn, cfg.hidden)), ("w_down", (cfg.hidden, cfg.ffn)))}
    ws["g1"] = wl.f32_to_bf16_bits(1 + 0.1 * rng.standard_normal(cfg.hidden, dtype=np.float32))
    ws["g2"] = wl.f32_to_bf16_bits(1 + 0.1 * rng.standard_normal(cfg.hidden, dtype=np.float32))
    x = wl.f32_to_bf16_bits(rng.standard_normal((b.T, cfg.hidden), dtype=np.float32))
    got = run_layer(cfg, b, ws, x, 4242)
    kp, vp = wl.prior_kv_concat(cfg, b, 4242)
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, ws, kp, vp)
    rows = np.arange(b.T)
    check_layer(cfg, b, got, exp, rows, "small-gqa", staged_attention(cfg, b, x, ws, kp, vp, rows), x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, rows)


def small_weights(rng, cfg):
    ws = {k: wl.f32_to_bf16_bits(rng.standard_normal(s, dtype=np.float32) * 0.02) for k, s in (
        ("w_qkv", (cfg.qkv_rows, cfg.hidden)), ("w_o", (cfg.hidden, cfg.n_q_heads * cfg.head_dim)),
        ("w_gu", (2 * cfg.ffn, cfg.hidden)), ("w_down", (cfg.hidden, cfg.ffn)))}
    ws["g1"] = wl.f32_to_bf16_bits(1 + 0.1 * rng.standard_normal(cfg.hidden, dtype=np.float32))
    ws["g2"] = wl.f32_to_bf16_bits(1 + 0.1 * rng.standard_normal(cfg.hidden, dtype=np.float32))
    return ws


def changed_slots(before, after, transposed):
    """Slots (page * 16 + s) where a pool differs bitwise between two images."""
    diff = before.view(torch.int16) != after.view(torch.int16)
    # keys [page][kv head][d/32][16][32], values [page][kv head][d][16]
    if transposed:
        per_slot = diff.any(dim=2).any(dim=1)
    else:
        per_slot = diff.any(dim=4).any(dim=2).any(dim=1)
    pg, sl = torch.nonzero(per_slot, as_tuple=True)
    return set((pg.cpu().numpy().astype(np.int64) * 16 + sl.cpu().numpy()).tolist())


@pytest.mark.parametrize("cfg", [SMALL_GQA, wl.LayerConfig("small-mha64", 256, 704, 4, 4, 64)],
                         ids=lambda c: c.name)
def test_layer_step_aligned_value_runs(cfg):
    """Eight decodes put the first prefill row on an 8-aligned row and slot, so
    the QKV epilogue writes whole 16-byte runs of the value pages; a chunk with
    40 cached tokens stays aligned across page boundaries, and a 5-token chunk
    ends on a partial run that mixes two requests.  Every row and every new
    slot is checked, and no pool entry outside the new slots may change."""
    say(f"case: layer step aligned value runs {cfg.name}")
    rng = np.random.default_rng(91)
    b = wl.custom_batch(rng, [3, 16, 40, 100, 7, 64, 15, 31], [(200, 0), (77, 40), (5, 3)])
    w = small_weights(rng, cfg)
    x = wl.f32_to_bf16_bits(rng.standard_normal((b.T, cfg.hidden), dtype=np.float32))
    got = run_layer(cfg, b, w, x, 4343, keep_before=True)
    kp, vp = wl.prior_kv_concat(cfg, b, 4343)
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = np.arange(b.T)
    check_layer(cfg, b, got, exp, rows, cfg.name, staged_attention(cfg, b, x, w, kp, vp, rows), x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, rows)
    written = set(oracle.token_map(b.n_new, b.ctx_len, b.page_tables, 16).tok_slot.tolist())
    assert changed_slots(got["k0"], got["k"], False) <= written
    assert changed_slots(got["v0"], got["v"], True) <= written


def test_layer_step_value_runs_any_alignment():
    """Chunks whose first row falls at different offsets in the 32-row blocks
    of the QKV epilogue and whose cached lengths put their first slot at every
    offset 0 .. 7 within a group of 8: the value runs are found from the slots
    themselves (a run may start at any row of a block and cross into the next
    page's group), the tokens left over go one at a time.  Every row and every
    new slot is checked, and no pool entry outside the new slots may change."""
    say("case: layer step value runs at every alignment")
    cfg = SMALL_GQA
    rng = np.random.default_rng(93)
    # first rows 5, 42, 87, 116, 182, 223, 284, 311; first slots 3, 5, 6, 7, 2, 1, 4, 0 mod 8
    b = wl.custom_batch(rng, [9, 30, 100, 250, 17],
                        [(37, 3), (45, 21), (29, 14), (66, 7), (41, 26), (61, 9), (27, 12), (50, 32)])
    w = small_weights(rng, cfg)
    x = wl.f32_to_bf16_bits(rng.standard_normal((b.T, cfg.hidden), dtype=np.float32))
    got = run_layer(cfg, b, w, x, 4545, keep_before=True)
    kp, vp = wl.prior_kv_concat(cfg, b, 4545)
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = np.arange(b.T)
    check_layer(cfg, b, got, exp, rows, "any-alignment", staged_attention(cfg, b, x, w, kp, vp, rows), x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, rows)
    written = set(oracle.token_map(b.n_new, b.ctx_len, b.page_tables, 16).tok_slot.tolist())
    assert changed_slots(got["k0"], got["k"], False) <= written
    assert changed_slots(got["v0"], got["v"], True) <= written


MEDIUM_MHA = wl.LayerConfig("medium-mha", 1536, 2816, 12, 12, 128)


def test_layer_step_split_reduces_all_rows():
    """A 90-row batch of a 1536-wide layer on which every projection is split
    over K (QKV three ways, gate/up four, down seven: 44 K chunks in uneven
    splits), so every split reduce runs: the QKV one with RoPE and the KV
    append, the SwiGLU one, the residual one, and the output projection's
    reduce fused with the residual and the second RMSNorm.  Every row of every
    stage and every new slot is checked against the oracle."""
    say("case: layer step, every projection split over K (all rows)")
    cfg = MEDIUM_MHA
    rng = np.random.default_rng(17)
    b = wl.custom_batch(rng, rng.integers(8, 300, size=60), [(30, 0)])
    w = small_weights(rng, cfg)
    x = wl.f32_to_bf16_bits(rng.standard_normal((b.T, cfg.hidden), dtype=np.float32))
    got = run_layer(cfg, b, w, x, 2929)
    kp, vp = wl.prior_kv_concat(cfg, b, 2929)
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = np.arange(b.T)
    check_layer(cfg, b, got, exp, rows, cfg.name, staged_attention(cfg, b, x, w, kp, vp, rows), x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, rows)


def test_layer_step_streams_and_ring():
    """Twelve layer steps (more than the eight pinned staging buffers), on the
    null stream and on torch streams that are dropped between calls: every
    output equals the first null-stream step bit for bit (the step is
    deterministic and appends the same keys to the same slots)."""
    say("case: layer step across streams and the staging ring")
    cfg = wl.CONFIGS["c1"]
    b = wl.make_batch("c1")
    w = wl.make_weights(cfg, "c1")
    x = wl.make_x(cfg, b.T, "c1")
    c, packed = pack_layer(cfg, b, w)
    k, v = wdev.alloc_pools(cfg, b.pool_pages)
    wdev.fill_pools(k, v, cfg, b, wl.kv_seed("c1"), poison=True)
    mb = mx_batch(mx, b)
    ws = ws_tensor(mx.mx_workspace_bytes_for(mb, cfg=c))
    xd = dev(x)
    ref = torch.empty_like(xd)
    mx.mx_layer_step(mb, c, packed, xd, ref, k, v, ws)
    sync()
    for i, kind in enumerate(["null", "null", "side", "null", "side", "side", "null", "null",
                              "null", "side", "null", "null"]):
        y = torch.empty_like(xd)
        if kind == "null":
            mx.mx_layer_step(mb, c, packed, xd, y, k, v, ws)
            sync()
        else:
            s = torch.cuda.Stream()
            s.wait_stream(torch.cuda.current_stream())
            mx.mx_layer_step(mb, c, packed, xd, y, k, v, ws, stream=s)
            s.synchronize()
            del s
        assert torch.equal(y.view(torch.int16), ref.view(torch.int16)), f"step {i} ({kind})"


# Degenerate batches: a lone decode (T = 1), one-token prefills with and
# without a cached prefix, a prefill-only batch, a chunk of exactly one tile,
# and a batch whose only decode sits on a page boundary
DEGENERATE = {
    "lone-decode": ([37], []),
    "one-token-prefill": ([], [(1, 0)]),
    "one-token-chunk-after-cache": ([], [(1, 300)]),
    "prefill-only": ([], [(33, 0), (64, 16), (2, 31)]),
    "one-tile-chunk": ([], [(64, 0)]),
    "decode-at-page-edge": ([16], [(15, 0)]),
}


@pytest.mark.parametrize("case", list(DEGENERATE))
def test_layer_step_degenerate_batches(case):
    say(f"case: layer step degenerate batch {case}")
    cfg = SMALL_GQA
    rng = np.random.default_rng(sum(map(ord, case)))
    dec, pre = DEGENERATE[case]
    b = wl.custom_batch(rng, dec, pre)
    w = small_weights(rng, cfg)
    x = wl.f32_to_bf16_bits(rng.standard_normal((b.T, cfg.hidden), dtype=np.float32))
    got = run_layer(cfg, b, w, x, 515, keep_before=True)
    kp, vp = wl.prior_kv_concat(cfg, b, 515)
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = np.arange(b.T)
    check_layer(cfg, b, got, exp, rows, case, staged_attention(cfg, b, x, w, kp, vp, rows), x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, rows)
    written = set(oracle.token_map(b.n_new, b.ctx_len, b.page_tables, 16).tok_slot.tolist())
    assert changed_slots(got["k0"], got["k"], False) <= written
    assert changed_slots(got["v0"], got["v"], True) <= written


def gemm_plans(cfg, T):
    """The cost model's plan of each projection of the layer at T rows."""
    H, F, nq, nkv, d = cfg.hidden, cfg.ffn, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    return {name: mx.mx_debug_gemm_plan(T, N, K) for name, (N, K) in (
        ("qkv", ((nq + 2 * nkv) * d, H)), ("o", (H, nq * d)), ("gate_up", (2 * F, H)),
        ("down", (H, F)))}


# Every sweep point of the 13B and 70B shapes that the benchmark reports
# beyond the chunk-free points (the 70B shape at P = 0, 4096 and 8192 is its
# headline curve's start, middle and end), plus a chunk after 6144 cached tokens.
SAMPLED_CASES = [("c2", 512, 0), ("c2", 0, 0), ("c3", 256, 0), ("c3", 1024, 0), ("c3", 2048, 0),
                 ("c3", 4096, 0), ("c4", 2048, 0), ("c4", 2048, 6144), ("c5", 0, 0),
                 ("c5", 1024, 0), ("c5", 4096, 0), ("c5", 8192, 0)]


@pytest.mark.parametrize("key,P,ctx", SAMPLED_CASES)
def test_layer_step_sampled(key, P, ctx):
    """Full-size layer iteration (the benchmark's launch configuration),
    checked on sampled rows: the oracle evaluates the requests that own them,
    cut after their last sampled row.  ctx > 0: the P-token chunk continues a
    prompt with ctx tokens already cached (a later chunk of a chunked prefill,
    as in the chunk-index sweep)."""
    say(f"case: layer step {key} P={P} ctx={ctx} (sampled rows)")
    cfg = wl.CONFIGS[key]
    b = wl.make_batch(key, P, prefill_lens=[P], prefill_ctx=[ctx]) if ctx else wl.make_batch(key, P)
    w = wl.make_weights(cfg, key)
    x = wl.make_x(cfg, b.T, key)
    seed = wl.kv_seed(key)
    say(f"  T={b.T} plans: {gemm_plans(cfg, b.T)}")
    got = run_layer(cfg, b, w, x, seed)
    rng = np.random.default_rng(3)
    # the 70B shape's contexts reach 16384 tokens: fewer sampled requests keep
    # the oracle's host copy of their cached keys and values small
    big = key == "c5"
    rows = sample_rows(b, rng, n_decode=4 if big else 16, n_prefill_random=8 if big else 30)
    if big and b.T > 8192:
        # rows on both sides of the row split of the 70B projections (8192 rows
        # in whole rounds of tiles, the rest as a GEMM of their own)
        rows = np.unique(np.concatenate([rows, [8191, 8192, 8193]]))
    sub, reqs, sub_rows, tok_idx = truncated_subbatch(b, rows)
    kp, vp = wl.prior_kv_concat(cfg, sub, seed)
    exp = oracle.layer_step(cfg.as_dict(), sub.n_new, sub.ctx_len, x[tok_idx], w, kp, vp,
                            rows=sub_rows)
    o_ref = staged_attention(cfg, sub, x[tok_idx], w, kp, vp, sub_rows)
    errs = check_layer(cfg, b, got, exp, rows, key, o_ref, x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, tok_idx)
    say("  errors", {k: f"{v:.2e}" for k, v in errs.items()})


def test_layer_step_small_residual_branches():
    """The residual x scaled down 16-fold (an exact power of two), so that the
    attention and MLP branches dominate x1 and y: the branches x1 - x, y - x1
    and y - x are gated at 2e-2 against the exact oracle on the raw
    difference, with no allowance for the bf16 storage of x1 and y.  (RMSNorm
    makes h, and so every branch input, nearly independent of x's scale.)"""
    say("case: layer step with a small residual (branches gated raw)")
    cfg = SMALL_GQA
    rng = np.random.default_rng(4545)
    b = wl.custom_batch(rng, [5, 16, 300, 1000, 2047, 64], [(150, 0), (40, 96), (1, 0)])
    w = small_weights(rng, cfg)
    x = wl.f32_to_bf16_bits(rng.standard_normal((b.T, cfg.hidden), dtype=np.float32) / 16.0)
    got = run_layer(cfg, b, w, x, 616)
    kp, vp = wl.prior_kv_concat(cfg, b, 616)
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = np.arange(b.T)
    check_layer(cfg, b, got, exp, rows, "small-residual", staged_attention(cfg, b, x, w, kp, vp, rows),
                x=x, branch_allowance=False)


# ----------------------------------------------------------------------- GEMM row split
# A GEMM whose rows run as two launches: rows [0, m_main) in whole rounds of
# tiles, the rest as a GEMM of its own (split over K or not).  Every epilogue
# of the debug entry point, ragged tails, weights in the packed tile layout.
@pytest.mark.parametrize("M,N,K,epi,m_main,main_cfg,tail_cfg,tail_ks", [
    (700, 2048, 1024, 0, 512, 0, 3, 4), (700, 2048, 1024, 1, 512, 1, 1, 1),
    (577, 1024, 2048, 2, 512, 2, 3, 8), (1100, 1040, 512, 1, 1024, 0, 0, 3),
    (300, 4096, 4096, 1, 256, 0, 1, 8), (300, 768, 704, 2, 256, 4, 2, 5),
])
def test_gemm_row_split(M, N, K, epi, m_main, main_cfg, tail_cfg, tail_ks):
    say(f"case: gemm row split M={M} N={N} K={K} epi={epi} m_main={m_main} "
        f"cfg={main_cfg} tail={tail_cfg}/{tail_ks}")
    rng = np.random.default_rng(M + 3 * N + K + epi)
    a = wl.f32_to_bf16_bits(rng.standard_normal((M, K), dtype=np.float32))
    w = wl.f32_to_bf16_bits(rng.standard_normal((N, K), dtype=np.float32) * 0.02)
    r = wl.f32_to_bf16_bits(rng.standard_normal((M, N), dtype=np.float32))
    ncol = N // 2 if epi == 2 else N
    lead = -(-2 * ncol // 8) * 8
    n_c = tile_elems(M, ncol) if epi == 2 else M * ncol  # the SwiGLU output in the tile layout
    buf16 = torch.full((lead + n_c + 2 * ncol,), CANARY, dtype=torch.int16, device="cuda")
    C = buf16.view(torch.uint16)[lead:lead + n_c]
    if epi != 2:
        C = C.view(M, ncol)
    ws = ws_tensor(max(tail_ks * (M - m_main) * N * 4 if tail_ks > 1 else 0, 256))
    wt = np.ascontiguousarray(w.reshape(N // 16, 16, K // 32, 32).transpose(0, 2, 1, 3))
    mx.mx_debug_gemm_rows(dev(to_tiles(a)), dev(wt.reshape(-1)), C, dev(r) if epi == 1 else None,
                          epi, M, N, K, m_main, main_cfg, tail_cfg, tail_ks, ws)
    sync()
    guard = torch.cat([buf16[:lead], buf16[lead + n_c:]]).cpu().numpy()
    assert (guard == CANARY).all(), "GEMM wrote outside C"
    if epi == 2:
        assert (tiles_unwritten(C, M, ncol).view(np.int16) == CANARY).all(), \
            "GEMM wrote a padding row or an unused tile of C"
        C = torch.from_numpy(from_tiles(C, M, ncol))
    acc = oracle.linear(wl.bf16_bits_to_f64(a), w)
    if epi == 1:
        exp = acc + wl.bf16_bits_to_f64(r)
    elif epi == 2:
        blocks = acc.reshape(M, N // 64, 2, 32)
        exp = oracle.silu_mul(np.concatenate([blocks[:, :, 0].reshape(M, -1),
                                              blocks[:, :, 1].reshape(M, -1)], axis=1))
    else:
        exp = acc
    assert_rows_close(bits_to_f64(C), exp, what="gemm row split")


def test_gemm_plan_rows_at_benchmark_point():
    """The 70B-shaped projections at 8448 rows (the benchmark's headline
    point): down, O and QKV run 8192 rows in whole rounds of 256 x 256 tiles
    and the last 256 rows as a GEMM of their own split over K; gate/up, whose
    tiles fill 28.9 rounds, runs as one launch."""
    plans = gemm_plans(wl.CONFIGS["c5"], 8448)
    say(f"  plans: {plans}")
    for name in ("qkv", "o", "down"):
        assert plans[name]["m_main"] == 8192 and plans[name]["cfg"] == 0, name
        assert plans[name]["tail_ksplit"] > 1, name
    assert plans["gate_up"]["m_main"] == 8448


# ----------------------------------------------------------------------- fused O reduce + RMSNorm
@pytest.mark.parametrize("H", [1536, 5120, 8192])
@pytest.mark.parametrize("ks,split_row", [(2, 0), (8, 0), (9, 0), (4, 37)])
def test_reduce_residual_rmsnorm(H, ks, split_row):
    """The output projection's split-K reduce fused with the residual and the
    second RMSNorm: a partly filled second register chunk (H = 5120), both
    chunks full (8192), more planes than are loaded ahead (9 > 8), and rows
    completed by the GEMM itself (split_row > 0: the row split).  x1 against
    the fp64 sum of the planes and the residual (one bf16 rounding: within
    half an ulp plus the fp32 sums' error); h against the oracle's RMSNorm of
    the GPU's x1 at 2e-2, and x1 bit for bit where rows were complete."""
    say(f"case: reduce+rmsnorm H={H} ks={ks} split_row={split_row}")
    M = 97
    rng = np.random.default_rng(H + ks + split_row)
    planes = (rng.standard_normal((ks, M - split_row, H)) * 0.5).astype(np.float32)
    r = wl.f32_to_bf16_bits(rng.standard_normal((M, H), dtype=np.float32))
    x1_done = wl.f32_to_bf16_bits(rng.standard_normal((M, H), dtype=np.float32))
    g = wl.f32_to_bf16_bits(1 + 0.1 * rng.standard_normal(H, dtype=np.float32))
    x1 = dev(x1_done)
    h = torch.empty((tile_elems(M, H),), dtype=torch.uint16, device="cuda")  # tile layout
    mx.mx_debug_reduce_residual_rmsnorm(torch.from_numpy(planes).cuda(), ks, dev(r), x1, dev(g), h,
                                        eps=1e-5, split_row=split_row)
    sync()
    got_x1 = bits_to_f64(x1)
    np.testing.assert_array_equal(host_bits(x1)[:split_row], x1_done[:split_row])
    exact = planes.astype(np.float64).sum(axis=0) + wl.bf16_bits_to_f64(r[split_row:])
    tail = got_x1[split_row:]
    # fp32 sums of ks planes and the residual: each partial sum's rounding is at
    # most 2^-24 of the summands' magnitude sum; then one rounding to bf16
    mag = np.abs(planes.astype(np.float64)).sum(axis=0) + np.abs(wl.bf16_bits_to_f64(r[split_row:]))
    bound = bf16_half_ulp(tail) + (ks + 1) * mag * 2.0 ** -24 + 1e-30
    assert (np.abs(tail - exact) <= bound).all(), "x1 off by more than one rounding"
    exp_h = oracle.rmsnorm(got_x1, wl.bf16_bits_to_f64(g), 1e-5)
    assert_rows_close(wl.bf16_bits_to_f64(from_tiles(h, M, H)), exp_h, what="h")


# ----------------------------------------------------------------------- row split in the layer
G2048 = wl.LayerConfig("gqa-2048", 2048, 5632, 16, 4, 128)


def test_layer_step_row_split_all_rows():
    """A 2696-row iteration of a 2048-wide GQA layer on which the QKV
    projection runs its first 2688 rows in whole rounds and the last 8 as a GEMM
    of their own split over K: the fused QKV epilogue (RoPE, q, and the KV
    append) of those rows runs in the split reduce with the rotary table,
    token slots and q rows taken from row 2688 on.  Every row of every stage
    and every new slot against the oracle."""
    say("case: layer step with row-split projections (all rows)")
    cfg = G2048
    rng = np.random.default_rng(2696)
    dec = rng.integers(8, 600, size=100)
    b = wl.custom_batch(rng, dec, [(1000, 0), (900, 37), (696, 5)])
    assert b.T == 2696
    plans = gemm_plans(cfg, b.T)
    say(f"  plans: {plans}")
    assert plans["qkv"]["m_main"] < b.T and plans["qkv"]["tail_ksplit"] > 1
    w = small_weights(rng, cfg)
    x = wl.f32_to_bf16_bits(rng.standard_normal((b.T, cfg.hidden), dtype=np.float32))
    got = run_layer(cfg, b, w, x, 2696, keep_before=True)
    kp, vp = wl.prior_kv_concat(cfg, b, 2696)
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = np.arange(b.T)
    check_layer(cfg, b, got, exp, rows, cfg.name, staged_attention(cfg, b, x, w, kp, vp, rows), x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, rows)
    written = set(oracle.token_map(b.n_new, b.ctx_len, b.page_tables, 16).tok_slot.tolist())
    assert changed_slots(got["k0"], got["k"], False) <= written
    assert changed_slots(got["v0"], got["v"], True) <= written


# ----------------------------------------------------------------------- randomised batches
from hypothesis import HealthCheck, given, settings  # noqa: E402
from hypothesis import strategies as st  # noqa: E402

RANDOM_SETTINGS = dict(derandomize=True, deadline=None, database=None,
                       suppress_health_check=[HealthCheck.too_slow, HealthCheck.data_too_large,
                                              HealthCheck.function_scoped_fixture])


@st.composite
def ctx_near_page_edge(draw, lo_pages=0, hi_pages=64):
    """A cached length that ends on a page boundary or one token short of it."""
    k = draw(st.integers(lo_pages, hi_pages))
    return max(16 * k + draw(st.sampled_from([0, 15])), 0)


@st.composite
def mixed_batch(draw, max_prefill=300):
    """Decodes (1..8, cached lengths at or just below page edges) and prefill
    chunks (0..3, with or without a cached prefix), in random order."""
    dec = [max(1, draw(ctx_near_page_edge(0, 80))) for _ in range(draw(st.integers(0, 8)))]
    pre = [(draw(st.integers(1, max_prefill)), draw(ctx_near_page_edge(0, 20)) * draw(st.integers(0, 1)))
           for _ in range(draw(st.integers(0 if dec else 1, 3)))]
    seed = draw(st.integers(0, 2 ** 31 - 1))
    return dec, pre, seed


HEADS = st.sampled_from([(4, 4, 64), (8, 8, 128), (8, 2, 128), (16, 4, 64), (16, 2, 128),
                         (32, 4, 128), (8, 1, 64)])


@settings(max_examples=24, **RANDOM_SETTINGS)
@given(batch=mixed_batch(), heads=HEADS)
def test_paged_attn_random_batches(batch, heads):
    """mx_paged_attn against the exact oracle (same bf16 q, k, v on both sides)
    on random mixed batches: request count and phases, chunk lengths, cached
    lengths at page edges, GQA group sizes 1, 4 and 8, head_dim 64 and 128."""
    dec, pre, seed = batch
    nq, nkv, d = heads
    say(f"case: random attention nq={nq} nkv={nkv} d={d} decodes={dec} prefills={pre} seed={seed}")
    rng = np.random.default_rng(seed)
    cfg = wl.LayerConfig("t", 256, 256, nq, nkv, d)
    b = wl.custom_batch(rng, dec, pre)
    c = attention_case(cfg, b, seed % 1000 + 1, rng)
    out = torch.empty((b.T, nq, d), dtype=torch.uint16, device="cuda")
    mx.mx_paged_attn(c["mb"], c["shape"], c["q"], c["k"], c["v"], out, c["ws"])
    sync()
    assert_rows_close(bits_to_f64(out).reshape(b.T * nq, d), c["exp"].reshape(b.T * nq, d),
                      what="attention")


@settings(max_examples=10, **RANDOM_SETTINGS)
@given(batch=mixed_batch(max_prefill=200), heads=HEADS)
def test_layer_step_random_batches(batch, heads):
    """mx_layer_step on random mixed batches of a small layer (hidden 512):
    every row of every stage and the branch sums against the exact oracle,
    every new slot in the pools."""
    dec, pre, seed = batch
    nq, nkv, d = heads
    say(f"case: random layer nq={nq} nkv={nkv} d={d} decodes={dec} prefills={pre} seed={seed}")
    rng = np.random.default_rng(seed)
    cfg = wl.LayerConfig("rand", 512, 704, nq, nkv, d)
    b = wl.custom_batch(rng, dec, pre)
    w = small_weights(rng, cfg)
    x = wl.f32_to_bf16_bits(rng.standard_normal((b.T, cfg.hidden), dtype=np.float32))
    got = run_layer(cfg, b, w, x, seed % 1000 + 1)
    kp, vp = wl.prior_kv_concat(cfg, b, seed % 1000 + 1)
    exp = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = np.arange(b.T)
    check_layer(cfg, b, got, exp, rows, "random", staged_attention(cfg, b, x, w, kp, vp, rows), x=x)
    check_pool_rows(cfg, b, got, exp.k_new, exp.v_new, rows)


@st.composite
def gemm_problem(draw):
    """A random GEMM of the debug entry points: ragged M, N a multiple of 16
    (64 for SwiGLU), K a multiple of 64, any epilogue, row-major operands or
    the layer's layouts, the library's plan or a forced tile shape and K split."""
    epi = draw(st.sampled_from([0, 1, 2]))
    M = draw(st.integers(1, 640))
    unit = 64 if epi == 2 else 16
    N = unit * draw(st.integers(1, 2048 // unit))
    K = 64 * draw(st.integers(1, 32))
    tiled = draw(st.booleans())
    cfg = draw(st.sampled_from([-1, 0, 1, 2, 3, 4]))
    ks = draw(st.integers(1, min(8, K // 64))) if cfg >= 0 else 0
    return M, N, K, epi, tiled, cfg, ks


@settings(max_examples=30, **RANDOM_SETTINGS)
@given(p=gemm_problem())
def test_gemm_random_problems(p):
    """The GEMM against the oracle, with canaries around C, on random shapes,
    epilogues, layouts, tile shapes and K splits."""
    M, N, K, epi, tiled, cfg, ks = p
    gemm_case(M, N, K, epi, tile_cfg=cfg, ksplit=ks, b_tiled=tiled)
