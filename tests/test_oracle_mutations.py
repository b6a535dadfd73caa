"""Plants plausible mistakes in copies of oracle.c (on the CPU) and checks that
at least one pin of tests/test_oracle.py fails for each: evidence that the pins
constrain every step of the oracle, not just its happy path."""
import json
import os
import subprocess
import sys

import pytest

import oracle

HERE = os.path.dirname(os.path.abspath(__file__))

PIN_NAMES = """
    pins.test_token_map_golden,
    pins.test_rmsnorm_golden,
    pins.test_rmsnorm_numpy_and_invariants,
    pins.test_linear_matches_numpy,
    pins.test_rope_golden,
    pins.test_rope_properties,
    pins.test_rope_d2_is_plain_rotation,
    pins.test_silu_mul_golden_and_torch,
    pins.test_attention_golden,
    lambda: pins.test_attention_matches_sdpa(8, 2, 64),
    pins.test_paged_equals_contiguous_bitwise,
    pins.test_decode_equals_last_prefill_row_bitwise,
    pins.test_softmax_rows_sum_to_one,
    pins.test_attention_special_cases,
    pins.test_kv_append_brute_force,
    lambda: pins.test_layer_matches_torch_composition(pins.SMALL),
"""

RUNNER = """
import json, sys
sys.path.insert(0, %r)
sys.path.insert(0, %r)
import oracle
import test_oracle as pins
PINS = [%s]
failed = []
with oracle.using(sys.argv[1]):
    for pin in PINS:
        try:
            pin()
        except (AssertionError, ValueError) as e:
            failed.append(getattr(pin, "__name__", "lambda"))
print(json.dumps(failed))
"""

MUTATIONS = {
    "rmsnorm-drops-gain": ("out[t * H + i] = xr[i] * inv * g[i];", "out[t * H + i] = xr[i] * inv;"),
    "rmsnorm-drops-eps": ("sqrt(ss / (double)H + eps)", "sqrt(ss / (double)H)"),
    "rmsnorm-sum-not-mean": ("sqrt(ss / (double)H + eps)", "sqrt(ss + eps)"),
    "linear-wrong-row": ("wrow[k] = orc_bf16_to_double(W[n * K + k]);",
                         "wrow[k] = orc_bf16_to_double(W[(n ^ 1) < N ? (n ^ 1) * K + k : n * K + k]);"),
    "rope-sign": ("v[i] = a0 * c - a1 * s;", "v[i] = a0 * c + a1 * s;"),
    "rope-frequency": ("pow(theta, -2.0 * (double)i / (double)d)", "pow(theta, -1.0 * (double)i / (double)d)"),
    "rope-pairing": ("double a0 = v[i], a1 = v[i + half];", "double a0 = v[i], a1 = v[i ^ 1];"),
    "silu-sign": ("a[t * F + f] = g / (1.0 + exp(-g)) * up;", "a[t * F + f] = g / (1.0 + exp(g)) * up;"),
    "swiglu-swapped": ("double g = gu[t * 2 * F + f];\n      double up = gu[t * 2 * F + F + f];",
                       "double up = gu[t * 2 * F + f];\n      double g = gu[t * 2 * F + F + f];"),
    "attn-causal-off-by-one": ("int64_t p = ctx_len[r] + (t - first[r]);",
                               "int64_t p = ctx_len[r] + (t - first[r]) - 1;"),
    "attn-gqa-mapping": ("kv_rows(&src, h / group, p + 1", "kv_rows(&src, h % nkv, p + 1"),
    "attn-no-normalise": ("for (int32_t i = 0; i < d; i++) out[i] /= l;", ""),
    "attn-no-scale": ("    s *= scale;\n", "\n"),
    "paged-slot": ("base = ((page * src->nkv + g) * src->page_size + j % src->page_size) * src->d;",
                   "base = ((page * src->nkv + g) * src->page_size + (j + 1) % src->page_size) * src->d;"),
    "token-map-slot": ("* page_size + p % page_size;", "* page_size + (p + 1) % page_size;"),
    "kv-append-slot": ("int64_t s = p % page_size;", "int64_t s = (p + 1) % page_size;"),
    "layer-drops-residual": ("for (int64_t e = 0; e < H; e++) x1[i * H + e] += xd[row_idx[i] * H + e];", ";"),
    "layer-rope-on-v": ("orc_rope(T, (int32_t)nkv, (int32_t)d, pos, c->rope_theta, k_new);",
                        "orc_rope(T, (int32_t)nkv, (int32_t)d, pos, c->rope_theta, k_new);\n  orc_rope(T, (int32_t)nkv, (int32_t)d, pos, c->rope_theta, v_new);"),
    "layer-norm2-gain-g1": ("orc_rmsnorm(nr, H, x1, g2d, c->rms_eps, h2);",
                            "orc_rmsnorm(nr, H, x1, g1d, c->rms_eps, h2);"),
    "layer-k-from-v-rows": ("orc_linear(T, H, nkv * d, h, w_qkv + nq * d * H, k_new);",
                            "orc_linear(T, H, nkv * d, h, w_qkv + (nq + nkv) * d * H, k_new);"),
    "layer-q-no-rope": ("  orc_rope(nr, (int32_t)nq, (int32_t)d, pos_r, c->rope_theta, q);\n", "\n"),
    "layer-row-misses-own-key": ("row_ctx[i] = pos_r[i];", "row_ctx[i] = pos_r[i] > 0 ? pos_r[i] - 1 : 0;"),
    "layer-down-residual-x": ("for (int64_t i = 0; i < nr * H; i++) y[i] += x1[i];",
                              "for (int64_t i = 0; i < nr; i++)\n    for (int64_t e = 0; e < H; e++) y[i * H + e] += xd[row_idx[i] * H + e];"),
    "layer-gu-no-down": ("for (int64_t i = 0; i < nr * H; i++) y[i] += x1[i];", ""),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_planted_mistake_is_caught(name, tmp_path):
    old, new = MUTATIONS[name]
    src = oracle.source_text()
    assert src.count(old) == 1, f"mutation anchor for {name} not unique in oracle.c"
    so = oracle.build_variant(src.replace(old, new), str(tmp_path / "liboracle_mut.so"))
    # each mutant runs in its own process so that a crash cannot pass as a catch
    script = RUNNER % (os.path.dirname(HERE), HERE, PIN_NAMES)
    res = subprocess.run([sys.executable, "-c", script, so], capture_output=True, text=True,
                         timeout=600)
    assert res.returncode == 0, f"mutant {name} crashed the pins: {res.stderr[-2000:]}"
    failed = json.loads(res.stdout.strip().splitlines()[-1])
    assert failed, f"no pin caught the planted mistake {name}"
