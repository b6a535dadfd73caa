"""Iteration-latency predictor (the offline-profiled execution-time estimate
the multiplexing toggle relies on, Section 4.3; prefill and decode execution
times are taken as highly predictable there, which the fit's residuals test).

A mixed iteration's latency is modelled as linear in the work its parts do:

    t = c0 + c_tok * T + c_big * max(T - T_KNOT, 0) + c_kv * KV + c_pair * PAIRS + c_req * R

T      tokens in the iteration (every projection streams them);
max(T - T_KNOT, 0)
       the tokens beyond one 256-row GEMM tile: up to about that many rows
       the projections stream their weights from HBM once and cost little
       more per token, beyond it they are bound by the matrix cores and cost
       a fixed amount per token (a hinge at T_KNOT, so that one fit spans
       decode-only and prefill-heavy batches);
KV     cached keys read by the decode rows, sum over decodes of ctx + 1
       (decode attention streams the KV cache);
PAIRS  query-key pairs of the prefill chunks, sum over chunks of
       t * p + t (t + 1) / 2 for a chunk of t tokens after p cached ones
       (prefill attention is quadratic in the chunk and linear in its prior);
R      requests in the batch (per-request setup).

The fit is an ordinary least-squares solve over measured (batch, latency)
samples of one layer shape; relative residuals are reported by `residuals`.
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Dict, Iterable, List, Sequence

import numpy as np

FEATURES = ("one", "tokens", "tokens_beyond_knot", "decode_kv", "prefill_pairs", "requests")
T_KNOT = 256


def batch_features(n_new: Sequence[int], ctx_len: Sequence[int], is_decode: Sequence[bool]) -> np.ndarray:
    """Feature vector of one iteration's batch, in FEATURES order."""
    n_new = np.asarray(n_new, np.float64)
    ctx = np.asarray(ctx_len, np.float64)
    dec = np.asarray(is_decode, bool)
    T = n_new.sum()
    kv = (ctx[dec] + 1.0).sum()
    t, p = n_new[~dec], ctx[~dec]
    pairs = (t * p + t * (t + 1.0) / 2.0).sum()
    return np.array([1.0, T, max(T - T_KNOT, 0.0), kv, pairs, float(len(n_new))])


@dataclass
class LatencyModel:
    """Linear latency model of one layer shape (coefficients in microseconds
    per unit of each feature)."""
    coef: np.ndarray = field(default_factory=lambda: np.zeros(len(FEATURES)))
    layers: int = 1

    @classmethod
    def fit(cls, feats: Iterable[np.ndarray], lat_us: Iterable[float], layers: int = 1) -> "LatencyModel":
        X = np.vstack(list(feats))
        y = np.asarray(list(lat_us), np.float64)
        if X.shape[0] < X.shape[1]:
            raise ValueError(f"{X.shape[0]} samples cannot fit {X.shape[1]} coefficients")
        coef, *_ = np.linalg.lstsq(X, y, rcond=None)
        return cls(coef=coef, layers=layers)

    def predict(self, feats: np.ndarray) -> np.ndarray:
        """Predicted latency in microseconds of one layer times `layers`."""
        return (np.atleast_2d(feats) @ self.coef) * self.layers

    def predict_batch(self, n_new, ctx_len, is_decode) -> float:
        return float(self.predict(batch_features(n_new, ctx_len, is_decode))[0])

    def residuals(self, feats: Iterable[np.ndarray], lat_us: Iterable[float]) -> Dict[str, float]:
        X = np.vstack(list(feats))
        y = np.asarray(list(lat_us), np.float64)
        rel = (X @ self.coef * self.layers - y) / y
        return {"median_abs_rel": float(np.median(np.abs(rel))), "max_abs_rel": float(np.abs(rel).max()),
                "mean_rel": float(rel.mean()), "n": int(len(y))}

    def as_dict(self) -> Dict[str, float]:
        return {name: float(c) for name, c in zip(FEATURES, self.coef)}

    @classmethod
    def from_dict(cls, d: Dict[str, float], layers: int = 1) -> "LatencyModel":
        return cls(coef=np.array([float(d[n]) for n in FEATURES]), layers=layers)
