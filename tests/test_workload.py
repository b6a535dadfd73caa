"""Seeded input generators: encodings, determinism and batch shapes (CPU only)."""
import numpy as np
import torch

import workload as wl


def test_bf16_rounding_matches_torch():
    rng = np.random.default_rng(0)
    a = np.concatenate([rng.standard_normal(10000).astype(np.float32) * 10,
                        np.array([0.0, -0.0, 1.0, 1.00390625, 1.01171875, 65504.0, 1e-30], np.float32)])
    ours = wl.f32_to_bf16_bits(a)
    ref = torch.from_numpy(a).to(torch.bfloat16).view(torch.int16).numpy().view(np.uint16)
    np.testing.assert_array_equal(ours, ref)
    np.testing.assert_array_equal(wl.bf16_bits_to_f32(ours),
                                  torch.from_numpy(a).to(torch.bfloat16).float().numpy())


def test_splitmix64_reference_values():
    # SplitMix64 sequence from state 0: first outputs of the published generator
    # (state += golden gamma, then the variant-13 finaliser).
    out = [int(wl.mix64(np.uint64((i * 0x9E3779B97F4A7C15) & (2**64 - 1)))) for i in (1, 2, 3)]
    assert out == [0xE220A8397B1DCDAF, 0x6E789E6AA1B965F4, 0x06C45D188009454F]


def test_hash_values_uniform_unit_variance():
    c = np.arange(200000, dtype=np.uint64)
    v = wl.bf16_bits_to_f64(wl.hash_bf16(wl.stream_key(1001, 0), c))
    assert abs(v.mean()) < 0.01
    assert abs(v.var() - 1.0) < 0.01
    # sqrt(3) rounds up to 1.734375 in bf16
    assert v.min() >= -1.734375 and v.max() <= 1.734375
    w = wl.bf16_bits_to_f64(wl.hash_bf16(wl.stream_key(1001, 1), c))
    assert abs(np.corrcoef(v, w)[0, 1]) < 0.01


def test_batches_shapes():
    b = wl.make_batch("c1")
    assert b.T == 132 and b.R == 5 and b.pool_pages == 64
    assert sum(len(t) for t in b.page_tables) <= 64
    assert ((b.ctx_len[:4] >= 64) & (b.ctx_len[:4] <= 256)).all()
    b = wl.make_batch("c2", 512)
    assert b.T == 576 and b.R == 65 and b.prefill_tokens == 512
    b = wl.make_batch("c3", 4096)
    assert b.prefill_tokens == 4096 and b.T == 4096 + 128
    assert ((b.ctx_len[:128] >= 32) & (b.ctx_len[:128] <= 4096)).all()
    b = wl.make_batch("c4", 2048)
    assert b.T == 2304
    b = wl.make_batch("c5", 0)
    assert b.T == 256 and b.pool_pages == wl.C5_POOL_PAGES
    # same seed, same batch; pages unique across requests
    b2 = wl.make_batch("c5", 0)
    assert (b.ctx_len == b2.ctx_len).all()
    flat = b.flat_pages()
    assert len(np.unique(flat)) == len(flat)


def test_prior_kv_matches_host_pool():
    cfg = wl.CONFIGS["c1"]
    b = wl.make_batch("c1")
    kp, vp = wl.host_pool(cfg, b, 1000)
    for r in range(b.R):
        k, v = wl.prior_kv(cfg, b, r, 1000)
        for j in range(int(b.ctx_len[r])):
            page = b.page_tables[r][j // 16]
            np.testing.assert_array_equal(k[j], kp[page, :, j % 16])
            np.testing.assert_array_equal(v[j], vp[page, :, j % 16])


def test_bf16_half_ulp_bounds_rounding():
    """The branch gates of the layer parity tests take half an ulp of each
    stored bf16 value off the difference: that must bound the error of
    rounding any real number to that value (and be no looser than needed)."""
    import numpy as np
    from helpers import bf16_half_ulp
    rng = np.random.default_rng(8)
    v = np.concatenate([rng.standard_normal(100000) * 10.0 ** rng.integers(-6, 6, 100000),
                        [1.0, -2.0, 0.5, 255.9, 256.0, 1e-3]])
    r = wl.bf16_bits_to_f64(wl.f32_to_bf16_bits(v.astype(np.float32)))
    err = np.abs(r - v.astype(np.float32).astype(np.float64))
    hu = bf16_half_ulp(r)
    assert (err <= hu).all()
    # tight: at 1.0 the bf16 spacing is 2^-7, so half an ulp is 2^-8
    assert bf16_half_ulp(np.array([1.0, 1.5, 2.0]))[0] == 2.0 ** -8
    assert bf16_half_ulp(np.array([2.0]))[0] == 2.0 ** -7


def test_key_page_layout_conversions():
    """The device's blocked key pages [page][head][d/32][16][32] and the
    canonical [page][head][16][d] order: element (slot s, dim e) of a page sits
    at (e / 32) * 512 + s * 32 + e % 32, and the two conversions are inverses."""
    import workload.device as wdev
    rng = np.random.default_rng(3)
    for d in (64, 128):
        canon = rng.integers(0, 65536, (3, 2, 16, d), dtype=np.uint16)
        blocked = wdev.k_pool_blocked(canon)
        assert blocked.shape == (3, 2, d // 32, 16, 32)
        flat = blocked.reshape(3, 2, -1)
        for s, e in ((0, 0), (5, 33), (15, d - 1), (7, 31)):
            assert flat[1, 1, (e // 32) * 512 + s * 32 + e % 32] == canon[1, 1, s, e]
        np.testing.assert_array_equal(wdev.k_pool_canonical(blocked), canon)
