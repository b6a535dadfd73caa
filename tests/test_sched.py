"""Host-side scheduling layer: the latency predictor's features and fit."""
import numpy as np
import pytest

from paper_2606_16264_amd.sched import FEATURES, LatencyModel, batch_features


def brute_features(n_new, ctx, dec):
    T = sum(n_new)
    kv = sum(c + 1 for c, d in zip(ctx, dec) if d)
    pairs = 0
    for t, p, d in zip(n_new, ctx, dec):
        if d:
            continue
        for i in range(t):            # new token i sits at position p + i ...
            for j in range(p + i + 1):  # ... and attends to keys 0 .. p + i
                pairs += 1
    return [1.0, T, kv, pairs, len(n_new)]


def test_features_hand_example():
    f = batch_features([1, 1, 4], [10, 20, 3], [True, True, False])
    assert list(f) == [1.0, 6.0, 32.0, 22.0, 3.0]
    assert FEATURES == ("one", "tokens", "decode_kv", "prefill_pairs", "requests")


@pytest.mark.parametrize("seed", range(5))
def test_features_match_brute_force(seed):
    rng = np.random.default_rng(seed)
    n_dec, n_pre = int(rng.integers(0, 6)), int(rng.integers(0, 4))
    n_new = [1] * n_dec + [int(v) for v in rng.integers(1, 40, size=n_pre)]
    ctx = [int(v) for v in rng.integers(0, 60, size=n_dec + n_pre)]
    ctx[:n_dec] = [max(1, c) for c in ctx[:n_dec]]
    dec = [True] * n_dec + [False] * n_pre
    assert list(batch_features(n_new, ctx, dec)) == brute_features(n_new, ctx, dec)


def synthetic(rng, n, coef, noise=0.0):
    feats, lat = [], []
    for _ in range(n):
        n_dec = int(rng.integers(1, 200))
        P = int(rng.choice([0, 256, 1024, 4096]))
        n_new = [1] * n_dec + ([P] if P else [])
        ctx = list(rng.integers(64, 4097, size=n_dec)) + ([int(rng.choice([0, 2048]))] if P else [])
        f = batch_features(n_new, ctx, [True] * n_dec + ([False] if P else []))
        feats.append(f)
        lat.append(float(f @ coef) * (1.0 + noise * rng.standard_normal()))
    return feats, lat


def test_fit_recovers_exact_coefficients():
    rng = np.random.default_rng(7)
    coef = np.array([150.0, 0.08, 1.9e-4, 3.0e-7, 0.4])
    feats, lat = synthetic(rng, 40, coef)
    m = LatencyModel.fit(feats, lat)
    np.testing.assert_allclose(m.coef, coef, rtol=1e-6)
    r = m.residuals(feats, lat)
    assert r["max_abs_rel"] < 1e-9
    f = feats[3]
    assert m.predict_batch([1, 1, 512], [100, 200, 0], [True, True, False]) == pytest.approx(
        float(batch_features([1, 1, 512], [100, 200, 0], [True, True, False]) @ coef))
    assert LatencyModel.from_dict(m.as_dict()).predict(f)[0] == pytest.approx(m.predict(f)[0])


def test_fit_with_noise_has_small_residuals():
    rng = np.random.default_rng(8)
    coef = np.array([150.0, 0.08, 1.9e-4, 3.0e-7, 0.4])
    feats, lat = synthetic(rng, 60, coef, noise=0.01)
    m = LatencyModel.fit(feats[:30], lat[:30])
    assert m.residuals(feats[30:], lat[30:])["median_abs_rel"] < 0.02


def test_fit_needs_enough_samples():
    with pytest.raises(ValueError):
        LatencyModel.fit([np.ones(5)] * 3, [1.0, 2.0, 3.0])
