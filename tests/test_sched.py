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
    return [1.0, T, max(T - 256, 0), kv, pairs, len(n_new)]


def test_features_hand_example():
    f = batch_features([1, 1, 4], [10, 20, 3], [True, True, False])
    assert list(f) == [1.0, 6.0, 0.0, 32.0, 22.0, 3.0]
    f = batch_features([1, 300], [10, 0], [True, False])
    assert list(f) == [1.0, 301.0, 45.0, 11.0, 300 * 301 / 2, 2.0]
    assert FEATURES == ("one", "tokens", "tokens_beyond_knot", "decode_kv", "prefill_pairs",
                        "requests")


@pytest.mark.parametrize("seed", range(5))
def test_features_match_brute_force(seed):
    rng = np.random.default_rng(seed)
    n_dec, n_pre = int(rng.integers(0, 6)), int(rng.integers(0, 4))
    n_new = [1] * n_dec + [int(v) for v in rng.integers(1, 400, size=n_pre)]
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
    coef = np.array([150.0, 0.02, 0.08, 1.9e-4, 3.0e-7, 0.4])
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
    coef = np.array([150.0, 0.02, 0.08, 1.9e-4, 3.0e-7, 0.4])
    feats, lat = synthetic(rng, 60, coef, noise=0.01)
    m = LatencyModel.fit(feats[:30], lat[:30])
    assert m.residuals(feats[30:], lat[30:])["median_abs_rel"] < 0.02


def test_fit_needs_enough_samples():
    with pytest.raises(ValueError):
        LatencyModel.fit([np.ones(6)] * 3, [1.0, 2.0, 3.0])


# ---------------------------------------------------------------- SLO and slack
from paper_2606_16264_amd.sched import (SLO, Cluster, Request, Simulator, admits_chunk,  # noqa: E402
                                        attainment, synthetic_requests)


def done_request(rid, arrival, first, decode_time, output):
    r = Request(rid, arrival, 10, output)
    r.first_token, r.decode_time = first, decode_time
    return r


def test_attainment_eq1_to_3():
    slo = SLO(ttft=100.0, tpot=10.0)
    reqs = [done_request(0, 0.0, 100.0, 100.0, 10),    # TTFT = 100 ok, TPOT = 10 ok
            done_request(1, 5.0, 106.0, 50.0, 10),     # TTFT 101 misses
            done_request(2, 0.0, 50.0, 101.0, 10),     # TPOT 10.1 misses
            done_request(3, 0.0, 20.0, 90.0, 10)]      # both ok
    a = attainment(reqs, slo)
    assert a["attainment"] == 0.5
    assert a["ttft_attainment"] == 0.75 and a["tpot_attainment"] == 0.75


def test_slack_accumulates_per_decode_step():
    r = Request(0, 0.0, 10, 20)
    for t in (60.0, 60.0, 80.0):
        r.decode_time += t
        r.decode_steps += 1
    assert r.slack(100.0) == 300.0 - 200.0


def test_admission_fig7():
    """A decode iteration of 60 against a TPOT SLO of 100 leaves 40 of slack per
    token; a prefill that makes the iteration 160 fits once the slack reaches
    60, i.e. it is piggybacked on the iteration producing the third token, and
    the decode request's running TPOT stays within the SLO."""
    slo = SLO(ttft=1e9, tpot=100.0)
    r0 = Request(0, 0.0, 10, 20)
    admitted_at = None
    for step in range(4):
        if admitted_at is None and admits_chunk([r0], 60.0, 160.0, slo):
            admitted_at = step
            t = 160.0
        else:
            t = 60.0
        r0.decode_time += t
        r0.decode_steps += 1
        assert r0.decode_time <= r0.decode_steps * slo.tpot
    assert admitted_at == 2   # steps 0, 1 produce tokens 2 and 3; admission at the third decode step


def test_admission_gates():
    slo = SLO(ttft=1e9, tpot=100.0, busy_fraction=0.9, hbm_watermark=0.8)
    r = Request(0, 0.0, 10, 20)
    r.decode_steps, r.decode_time = 10, 100.0          # lots of slack
    assert admits_chunk([r], 50.0, 150.0, slo)
    assert not admits_chunk([r], 90.0, 150.0, slo)    # decode batch alone at 90% of the SLO
    assert not admits_chunk([r], 50.0, 150.0, slo, kv_use=81.0, kv_capacity=100.0)
    fresh = Request(1, 0.0, 10, 20)                    # no slack yet: one SLO of budget
    assert admits_chunk([fresh], 50.0, 100.0, slo) and not admits_chunk([fresh], 50.0, 100.5, slo)


# ---------------------------------------------------------------- simulator
TOY = LatencyModel(coef=np.array([50.0, 10.0, 0.0, 0.0, 0.0, 0.0]))   # 50 + 10 per token, per layer


def test_simulator_fig7_scenario():
    """One prefill worker and one multiplexing worker.  R0 is prefilled and
    then decodes on the multiplexing worker at 60 per token (TPOT SLO 100); a
    long prompt occupies the prefill worker; a short prompt that the prefill
    worker cannot serve within its TTFT SLO waits until R0 has built up the
    slack for it, and is then prefilled on the multiplexing worker without
    pushing R0 over its TPOT SLO."""
    slo = SLO(ttft=1000.0, tpot=100.0)
    cl = Cluster(workers=2, prefill_workers=1, chunk=64, layers=1,
                 kv_bytes_per_token=1.0, link_bytes_per_us=1e12, kv_capacity=1e12)
    reqs = [Request(0, 0.0, 5, 10), Request(1, 1.0, 1000, 2), Request(2, 150.0, 10, 2)]
    sim = Simulator(TOY, cl, slo, trace=True)
    res = sim.run(reqs)
    admits = [(t, w, rid) for t, w, kind, rid in sim.log if kind == "admit"]
    assert admits == [(pytest.approx(220.0), 1, 2)]
    r0 = next(r for r in sim.done if r.rid == 0)
    assert r0.tpot <= slo.tpot
    r2 = next(r for r in sim.done if r.rid == 2)
    assert r2.ttft <= slo.ttft
    assert res["requests"] == 3


@pytest.mark.parametrize("prefill_workers", [1, 2, 3])
def test_simulator_conserves_requests(prefill_workers):
    reqs = synthetic_requests(rate_per_s=20.0, n=120, seed=5, prompt_median=512, output_median=32)
    slo = SLO(ttft=2e6, tpot=4e4)
    model = LatencyModel(coef=np.array([250.0, 0.5, 0.0, 1.5e-3, 7e-5, 1.0]))
    sim = Simulator(model, Cluster(workers=4, prefill_workers=prefill_workers, chunk=512), slo,
                    seed=1)
    res = sim.run(reqs)
    assert res["requests"] == len(reqs)
    for r in sim.done:
        assert r.generated == r.output and r.first_token >= r.arrival
        assert r.decode_steps == r.output - 1 and r.finish >= r.first_token


def test_light_load_meets_every_slo():
    model = LatencyModel(coef=np.array([250.0, 0.5, 0.0, 1.5e-3, 7e-5, 1.0]))
    from paper_2606_16264_amd.sched import light_load_slo
    slo = light_load_slo(model, 32, 512, 512)
    reqs = synthetic_requests(rate_per_s=0.2, n=30, seed=6, prompt_median=512, output_median=16,
                              max_prompt=2048)
    for prefill_workers in (1, 2, 3):
        res = Simulator(model, Cluster(workers=4, prefill_workers=prefill_workers), slo).run(reqs)
        assert res["attainment"] == 1.0, (prefill_workers, res)


# ---------------------------------------------------------------- committed fits
@pytest.mark.parametrize("key", ["c2", "c4"])
def test_committed_latency_model_refits_from_its_samples(key):
    """The fitted latency model in profiles/ follows from its own recorded
    samples: the seeded batches regenerate with the recorded sizes, and a refit
    on their features and the recorded latencies (even samples; odd ones held
    out) predicts what the committed coefficients predict, with the committed
    held-out error."""
    import json
    import os

    import bench
    import workload as wl
    path = os.path.join(os.path.dirname(os.path.dirname(os.path.abspath(__file__))), "profiles",
                        f"latency_model_layer_step_{key}.json")
    rec = json.load(open(path))["latency_model"]
    samples = rec["samples"]
    feats = []
    for s, (r, b) in zip(samples, bench.predictor_batches(key, len(samples))):
        assert {k: s[k] for k in r} == r
        feats.append(batch_features(b.n_new, b.ctx_len, b.phase == wl.DECODE))
    lat = [s["us"] for s in samples]
    train, test = list(range(0, len(lat), 2)), list(range(1, len(lat), 2))
    m = LatencyModel.fit([feats[i] for i in train], [lat[i] for i in train])
    committed = LatencyModel.from_dict(rec["coef_us"])
    got, want = m.predict(np.array(feats)), committed.predict(np.array(feats))
    assert np.max(np.abs(got - want) / np.array(lat)) < 1e-3
    held = m.residuals([feats[i] for i in test], [lat[i] for i in test])
    assert held["median_abs_rel"] == pytest.approx(rec["held_out_residuals"]["median_abs_rel"],
                                                   abs=1e-3)
