"""Pins of the fp64 CPU oracle against things other than itself: hand-worked
fixtures (tests/golden), closed forms, invariants, brute force and independent
library routines (numpy / torch CPU in float64).  CPU only."""
import json
import math
import os

import numpy as np
import pytest
import torch
import torch.nn.functional as F
from hypothesis import given, settings, strategies as st, HealthCheck

import oracle
import workload as wl

GOLD = os.path.join(os.path.dirname(__file__), "golden")


def load(name):
    with open(os.path.join(GOLD, name)) as f:
        return json.load(f)


def bf16(a):
    return wl.f32_to_bf16_bits(np.asarray(a, np.float32))


def f64(bits):
    return wl.bf16_bits_to_f64(bits)


# --------------------------------------------------------------------------- token map
def test_token_map_golden():
    g = load("token_map_small.json")
    reqs = g["requests"]
    tm = oracle.token_map([r["n_new"] for r in reqs], [r["ctx_len"] for r in reqs],
                          [r["pages"] for r in reqs], g["page_size"])
    assert tm.cu_q.tolist() == g["cu_q"]
    assert tm.tok_req.tolist() == g["tok_req"]
    assert tm.tok_pos.tolist() == g["tok_pos"]
    assert tm.tok_slot.tolist() == g["tok_slot"]


def brute_token_map(n_new, ctx, tables, ps):
    req, pos, slot = [], [], []
    for r in range(len(n_new)):
        for i in range(n_new[r]):
            p = ctx[r] + i
            req.append(r)
            pos.append(p)
            slot.append(int(tables[r][p // ps]) * ps + p % ps)
    return req, pos, slot


@settings(max_examples=60, deadline=None)
@given(st.lists(st.tuples(st.integers(1, 40), st.integers(0, 70)), min_size=1, max_size=9),
       st.integers(0, 2**31 - 1))
def test_token_map_brute_force(reqs, seed):
    rng = np.random.default_rng(seed)
    n_new = [n for n, _ in reqs]
    ctx = [c for _, c in reqs]
    b = wl.custom_batch(rng, [], [(n, c) for n, c in reqs])
    tm = oracle.token_map(b.n_new, b.ctx_len, b.page_tables, 16)
    req, pos, slot = brute_token_map(n_new, ctx, b.page_tables, 16)
    assert tm.tok_req.tolist() == req
    assert tm.tok_pos.tolist() == pos
    assert tm.tok_slot.tolist() == slot
    assert tm.cu_q.tolist() == [0] + list(np.cumsum(n_new))
    # written slots are unique
    assert len(set(slot)) == len(slot)


def test_token_map_short_table():
    with pytest.raises(ValueError):
        oracle.token_map([2], [15], [[3]], 16)   # position 16 needs a second page


# --------------------------------------------------------------------------- RMSNorm
def test_rmsnorm_golden():
    g = load("rmsnorm_small.json")
    for case in g["cases"]:
        out = oracle.rmsnorm(np.array([g["x"]]), np.array(g["g"]), case["eps"])
        np.testing.assert_allclose(out[0], case["expected"], rtol=1e-15)


def test_rmsnorm_numpy_and_invariants():
    rng = np.random.default_rng(1)
    x = rng.standard_normal((7, 96))
    g = 1 + 0.1 * rng.standard_normal(96)
    eps = 1e-5
    out = oracle.rmsnorm(x, g, eps)
    ref = x / np.sqrt((x * x).mean(axis=1, keepdims=True) + eps) * g
    np.testing.assert_allclose(out, ref, rtol=1e-13)
    # rms of out / g is one (eps = 0) and the map is scale invariant
    o0 = oracle.rmsnorm(x, g, 0.0)
    np.testing.assert_allclose(np.sqrt(((o0 / g) ** 2).mean(axis=1)), 1.0, rtol=1e-13)
    np.testing.assert_allclose(oracle.rmsnorm(3.7 * x, g, 0.0), o0, rtol=1e-13)
    # torch's own rms_norm in float64
    t = F.rms_norm(torch.from_numpy(x), (96,), weight=torch.from_numpy(g), eps=eps).numpy()
    np.testing.assert_allclose(out, t, rtol=1e-12)


# --------------------------------------------------------------------------- linear
def test_linear_matches_numpy():
    rng = np.random.default_rng(2)
    a = rng.standard_normal((5, 48))
    w = bf16(rng.standard_normal((33, 48)) * 0.1)
    out = oracle.linear(a, w)
    np.testing.assert_allclose(out, a @ f64(w).T, rtol=1e-12, atol=1e-14)


def test_bf16_widening_exact():
    for bits in (0x0000, 0x3F80, 0xBF80, 0x4049, 0x0001, 0x7F7F, 0xC2F7):
        expect = float(np.array([bits], np.uint16).astype(np.uint32).__lshift__(16).view(np.float32)[0])
        assert oracle.bf16_to_double(bits) == expect
    assert oracle.bf16_to_double(0x3F80) == 1.0
    assert oracle.bf16_to_double(0xC000) == -2.0


# --------------------------------------------------------------------------- RoPE
def test_rope_golden():
    g = load("rope_small.json")
    u = np.array(g["u"], np.float64).reshape(1, 1, g["d"])
    out = oracle.rope(u, [g["pos"]], g["theta"])
    np.testing.assert_allclose(out.reshape(-1), g["expected"], rtol=1e-15, atol=1e-15)


def rope_complex(u, pos, theta):
    """Independent formulation: pair (u_i, u_{i+d/2}) as the complex number
    u_i + i u_{i+d/2} and multiply by exp(i * pos * theta^(-2i/d))."""
    T, nh, d = u.shape
    half = d // 2
    z = u[..., :half] + 1j * u[..., half:]
    inv = theta ** (-2.0 * np.arange(half) / d)
    rot = np.exp(1j * np.asarray(pos, np.float64)[:, None, None] * inv[None, None, :])
    w = z * rot
    return np.concatenate([w.real, w.imag], axis=-1)


def test_rope_properties():
    rng = np.random.default_rng(3)
    T, nh, d = 6, 3, 64
    u = rng.standard_normal((T, nh, d))
    pos = np.array([0, 1, 17, 255, 4096, 16383], np.int32)
    out = oracle.rope(u, pos, 1e4)
    # angles reach 1.6e4 rad, where one fp64 ulp of the angle is 3.6e-12 rad
    np.testing.assert_allclose(out, rope_complex(u, pos, 1e4), rtol=1e-10, atol=1e-10)
    # position 0 is the identity; norms are preserved
    np.testing.assert_array_equal(out[0], u[0])
    np.testing.assert_allclose(np.linalg.norm(out, axis=-1), np.linalg.norm(u, axis=-1), rtol=1e-13)
    # <R(m) q, R(n) k> depends only on m - n
    q = rng.standard_normal((1, 1, d))
    k = rng.standard_normal((1, 1, d))
    dots = []
    for m, n in ((10, 3), (107, 100), (7, 0)):
        dots.append(float((oracle.rope(q, [m], 5e5) * oracle.rope(k, [n], 5e5)).sum()))
    np.testing.assert_allclose(dots, dots[0], rtol=1e-12)


def test_rope_d2_is_plain_rotation():
    u = np.array([[[1.0, 0.0]]])
    for p in (1, 2, 5):
        out = oracle.rope(u, [p], 1e4)
        np.testing.assert_allclose(out.reshape(-1), [math.cos(p), math.sin(p)], rtol=1e-15, atol=1e-15)


# --------------------------------------------------------------------------- SwiGLU
def test_silu_mul_golden_and_torch():
    g = load("swiglu_small.json")
    gu = np.array([g["gate"] + g["up"]])
    np.testing.assert_allclose(oracle.silu_mul(gu)[0], g["expected"], rtol=1e-15, atol=1e-300)
    rng = np.random.default_rng(4)
    gu = rng.standard_normal((4, 2 * 40)) * 4
    ref = (F.silu(torch.from_numpy(gu[:, :40])) * torch.from_numpy(gu[:, 40:])).numpy()
    np.testing.assert_allclose(oracle.silu_mul(gu), ref, rtol=1e-13, atol=1e-15)
    # limits: silu(z) -> z for z >> 0, -> 0 for z << 0
    big = np.array([[60.0, -60.0, 1.0, 1.0]])
    np.testing.assert_allclose(oracle.silu_mul(big)[0], [60.0, -60.0 * math.exp(-60.0)], rtol=1e-12)


# --------------------------------------------------------------------------- attention
def test_attention_golden():
    g = load("attention_small.json")
    q = np.array(g["q"]).reshape(2, 1, 2)
    k = np.array(g["k"]).reshape(2, 1, 2)
    v = np.array(g["v"]).reshape(2, 1, 2)
    scale = 1 / math.sqrt(2)
    o = oracle.attention_contig([2], [0], q, k, v, [0], scale)
    np.testing.assert_allclose(o.reshape(2, 2), g["expected_prefill"], rtol=1e-14, atol=1e-14)
    o = oracle.attention_contig([1], [1], q[1:], k, v, [0], scale)
    np.testing.assert_allclose(o.reshape(2), g["expected_decode"], rtol=1e-14, atol=1e-14)


def rand_attention_case(rng, reqs, nq, nkv, d):
    """reqs = [(n_new, ctx_len)]; returns q, kc, vc, kv_off."""
    T = sum(n for n, _ in reqs)
    L = sum(n + c for n, c in reqs)
    q = rng.standard_normal((T, nq, d))
    kc = rng.standard_normal((L, nkv, d))
    vc = rng.standard_normal((L, nkv, d))
    kv_off = np.cumsum([0] + [n + c for n, c in reqs])[:-1]
    return q, kc, vc, kv_off


def sdpa_reference(reqs, q, kc, vc, kv_off, scale):
    """torch scaled_dot_product_attention (float64, CPU) per request with an
    explicit causal mask; kv heads repeated for grouped queries."""
    nq, nkv = q.shape[1], kc.shape[1]
    out, t0 = [], 0
    for (n, c), off in zip(reqs, kv_off):
        L = n + c
        qq = torch.from_numpy(q[t0:t0 + n]).permute(1, 0, 2)          # [nq, n, d]
        kk = torch.from_numpy(kc[off:off + L]).permute(1, 0, 2)
        vv = torch.from_numpy(vc[off:off + L]).permute(1, 0, 2)
        kk = kk.repeat_interleave(nq // nkv, dim=0)
        vv = vv.repeat_interleave(nq // nkv, dim=0)
        mask = torch.arange(L)[None, :] <= (c + torch.arange(n))[:, None]
        o = F.scaled_dot_product_attention(qq, kk, vv, attn_mask=mask, scale=scale)
        out.append(o.permute(1, 0, 2).numpy())
        t0 += n
    return np.concatenate(out)


@pytest.mark.parametrize("nq,nkv,d", [(4, 4, 64), (8, 2, 64), (8, 1, 128)])
def test_attention_matches_sdpa(nq, nkv, d):
    rng = np.random.default_rng(5 + nq + nkv)
    reqs = [(1, 37), (9, 0), (1, 1), (5, 23), (1, 80), (17, 16)]
    q, kc, vc, off = rand_attention_case(rng, reqs, nq, nkv, d)
    scale = 1 / math.sqrt(d)
    o = oracle.attention_contig([n for n, _ in reqs], [c for _, c in reqs], q, kc, vc, off, scale)
    ref = sdpa_reference(reqs, q, kc, vc, off, scale)
    np.testing.assert_allclose(o, ref, rtol=1e-11, atol=1e-12)


def test_paged_equals_contiguous_bitwise():
    rng = np.random.default_rng(6)
    nq, nkv, d, ps = 6, 3, 64, 16
    reqs = [(1, 47), (20, 0), (3, 29), (1, 15), (1, 16)]
    b = wl.custom_batch(rng, [], reqs, pool_pages=64)
    q, kc, vc, off = rand_attention_case(rng, reqs, nq, nkv, d)
    kpool = np.full((64, nkv, ps, d), np.nan)
    vpool = np.full((64, nkv, ps, d), np.nan)
    for r, (n, c) in enumerate(reqs):
        for j in range(n + c):
            page = b.page_tables[r][j // ps]
            kpool[page, :, j % ps] = kc[off[r] + j]
            vpool[page, :, j % ps] = vc[off[r] + j]
    n_new = [n for n, _ in reqs]
    ctx = [c for _, c in reqs]
    oc = oracle.attention_contig(n_new, ctx, q, kc, vc, off, 0.125)
    op = oracle.attention_paged(n_new, ctx, q, kpool, vpool, b.page_tables, 0.125)
    assert np.isfinite(op).all()          # no NaN slot (unused page slot) was read
    np.testing.assert_array_equal(op, oc)


def test_decode_equals_last_prefill_row_bitwise():
    rng = np.random.default_rng(7)
    nq, nkv, d, n = 4, 2, 64, 33
    q, kc, vc, off = rand_attention_case(rng, [(n, 0)], nq, nkv, d)
    full = oracle.attention_contig([n], [0], q, kc, vc, [0], 0.125)
    dec = oracle.attention_contig([1], [n - 1], q[n - 1:], kc, vc, [0], 0.125)
    np.testing.assert_array_equal(dec[0], full[n - 1])


def test_softmax_rows_sum_to_one():
    rng = np.random.default_rng(8)
    reqs = [(1, 200), (12, 5)]
    q, kc, vc, off = rand_attention_case(rng, reqs, 4, 2, 64)
    q *= 3
    for t in (0, 1, 7, 12):
        for h in (0, 3):
            w = oracle.attention_weights([1, 12], [200, 5], q, kc, off, 0.125, t, h)
            assert abs(w.sum() - 1.0) <= 1e-12
            assert (w >= 0).all()
    assert len(oracle.attention_weights([1, 12], [200, 5], q, kc, off, 0.125, 0, 0)) == 201
    assert len(oracle.attention_weights([1, 12], [200, 5], q, kc, off, 0.125, 1, 0)) == 6


def test_attention_special_cases():
    rng = np.random.default_rng(9)
    d = 64
    # a single key: o = v
    q = rng.standard_normal((1, 2, d))
    k = rng.standard_normal((1, 2, d))
    v = rng.standard_normal((1, 2, d))
    o = oracle.attention_contig([1], [0], q, k, v, [0], 0.125)
    np.testing.assert_allclose(o, v, rtol=1e-15)
    # q = 0: uniform weights, o = mean of the visible values
    L = 40
    k = rng.standard_normal((L, 1, d))
    v = rng.standard_normal((L, 1, d))
    o = oracle.attention_contig([1], [L - 1], np.zeros((1, 1, d)), k, v, [0], 0.125)
    np.testing.assert_allclose(o[0, 0], v[:, 0].mean(axis=0), rtol=1e-12, atol=1e-14)
    # needle: one key aligned with q, scaled x20, dominates
    qv = rng.standard_normal(d)
    qv /= np.linalg.norm(qv)
    k = rng.standard_normal((L, 1, d)) * 0.1
    k[13, 0] = 20 * math.sqrt(d) * qv * 2
    o = oracle.attention_contig([1], [L - 1], qv.reshape(1, 1, d), k, v, [0], 1 / math.sqrt(d))
    np.testing.assert_allclose(o[0, 0], v[13, 0], rtol=1e-6, atol=1e-6)


# --------------------------------------------------------------------------- KV append
def test_kv_append_brute_force():
    rng = np.random.default_rng(10)
    nkv, d = 2, 64
    reqs = [(1, 31), (18, 0), (4, 14)]
    b = wl.custom_batch(rng, [], reqs, pool_pages=40)
    T = b.T
    kn = rng.integers(0, 65535, (T, nkv, d), dtype=np.uint16)
    vn = rng.integers(0, 65535, (T, nkv, d), dtype=np.uint16)
    kp = rng.integers(0, 65535, (40, nkv, 16, d), dtype=np.uint16)
    vp = rng.integers(0, 65535, (40, nkv, 16, d), dtype=np.uint16)
    ko, vo = oracle.kv_append(b.n_new, b.ctx_len, b.page_tables, kn, vn, kp, vp)
    ke, ve = kp.copy(), vp.copy()
    t = 0
    for r, (n, c) in enumerate(reqs):
        for i in range(n):
            p = c + i
            page = b.page_tables[r][p // 16]
            ke[page, :, p % 16] = kn[t]
            ve[page, :, p % 16] = vn[t]
            t += 1
    np.testing.assert_array_equal(ko, ke)
    np.testing.assert_array_equal(vo, ve)


# --------------------------------------------------------------------------- whole layer
def torch_layer(cfg, n_new, ctx, x_bits, w, kprior_bits, vprior_bits):
    """Independent composition from torch CPU float64 library routines:
    rms_norm, linear, complex-number RoPE, scaled_dot_product_attention, silu."""
    H, Fd, nq, nkv, d = cfg.hidden, cfg.ffn, cfg.n_q_heads, cfg.n_kv_heads, cfg.head_dim
    t = lambda bits: torch.from_numpy(f64(bits))
    x = t(x_bits)
    h = F.rms_norm(x, (H,), weight=t(w["g1"]), eps=cfg.rms_eps)
    qkv = F.linear(h, t(w["w_qkv"]))
    T = x.shape[0]
    q = qkv[:, : nq * d].reshape(T, nq, d).numpy()
    k = qkv[:, nq * d:(nq + nkv) * d].reshape(T, nkv, d).numpy()
    v = qkv[:, (nq + nkv) * d:].reshape(T, nkv, d).numpy()
    pos = np.concatenate([np.arange(c, c + n) for n, c in zip(n_new, ctx)])
    q = rope_complex(q, pos, cfg.rope_theta)
    k = rope_complex(k, pos, cfg.rope_theta)
    kp, vp = f64(kprior_bits), f64(vprior_bits)
    kcs, vcs, t0, p0 = [], [], 0, 0
    for n, c in zip(n_new, ctx):
        kcs += [kp[p0:p0 + c], k[t0:t0 + n]]
        vcs += [vp[p0:p0 + c], v[t0:t0 + n]]
        t0 += n
        p0 += c
    kc, vc = np.concatenate(kcs), np.concatenate(vcs)
    reqs = list(zip(n_new, ctx))
    off = np.cumsum([0] + [n + c for n, c in reqs])[:-1]
    o = torch.from_numpy(sdpa_reference(reqs, q, kc, vc, off, cfg.scale).reshape(T, nq * d))
    x1 = x + F.linear(o, t(w["w_o"]))
    h2 = F.rms_norm(x1, (H,), weight=t(w["g2"]), eps=cfg.rms_eps)
    gu = F.linear(h2, t(w["w_gu"]))
    a = F.silu(gu[:, :Fd]) * gu[:, Fd:]
    y = x1 + F.linear(a, t(w["w_down"]))
    return dict(h=h.numpy(), k=k, v=v, q=q, o=o.numpy(), x1=x1.numpy(), h2=h2.numpy(),
                a=a.numpy(), y=y.numpy())


SMALL = wl.LayerConfig("test-small", 128, 320, 4, 2, 32, rope_theta=1e4)


@pytest.mark.parametrize("cfg", [SMALL, wl.CONFIGS["c1"]], ids=["gqa-small", "c1"])
def test_layer_matches_torch_composition(cfg):
    rng = np.random.default_rng(11)
    if cfg.name == "tiny-256":
        b = wl.make_batch("c1")
        w = wl.make_weights(cfg, "c1")
    else:
        b = wl.custom_batch(rng, [5, 16, 33], [(9, 0), (6, 7)])
        w = {k: bf16(rng.standard_normal(s) * sc) for k, s, sc in (
            ("w_qkv", (cfg.qkv_rows, cfg.hidden), 0.05),
            ("w_o", (cfg.hidden, cfg.n_q_heads * cfg.head_dim), 0.05),
            ("w_gu", (2 * cfg.ffn, cfg.hidden), 0.05), ("w_down", (cfg.hidden, cfg.ffn), 0.05))}
        w["g1"] = bf16(1 + 0.1 * rng.standard_normal(cfg.hidden))
        w["g2"] = bf16(1 + 0.1 * rng.standard_normal(cfg.hidden))
    x = bf16(rng.standard_normal((b.T, cfg.hidden)))
    kp, vp = wl.prior_kv_concat(cfg, b, 1234)
    out = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    ref = torch_layer(cfg, b.n_new.tolist(), b.ctx_len.tolist(), x, w, kp, vp)
    for name, got in (("h", out.h), ("k", out.k_new), ("v", out.v_new), ("q", out.q),
                      ("o", out.o), ("x1", out.x1), ("h2", out.h2), ("a", out.a), ("y", out.y)):
        np.testing.assert_allclose(got, ref[name], rtol=1e-9, atol=1e-11, err_msg=name)


def test_layer_row_subset_equals_full():
    cfg = SMALL
    rng = np.random.default_rng(12)
    b = wl.custom_batch(rng, [3, 40], [(21, 0), (5, 18)])
    w = {k: bf16(rng.standard_normal(s) * 0.05) for k, s in (
        ("w_qkv", (cfg.qkv_rows, cfg.hidden)), ("w_o", (cfg.hidden, cfg.n_q_heads * cfg.head_dim)),
        ("w_gu", (2 * cfg.ffn, cfg.hidden)), ("w_down", (cfg.hidden, cfg.ffn)))}
    w["g1"] = bf16(np.ones(cfg.hidden))
    w["g2"] = bf16(np.ones(cfg.hidden))
    x = bf16(rng.standard_normal((b.T, cfg.hidden)))
    kp, vp = wl.prior_kv_concat(cfg, b, 99)
    full = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp)
    rows = [0, 1, 2, 9, 22, 27]
    sub = oracle.layer_step(cfg.as_dict(), b.n_new, b.ctx_len, x, w, kp, vp, rows=rows)
    for name in ("q", "o", "x1", "h2", "a", "y"):
        np.testing.assert_array_equal(getattr(sub, name), getattr(full, name)[rows], err_msg=name)
