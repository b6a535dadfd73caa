"""SLO accounting and the TPOT-slack admission test of SLO-aware multiplexing.

SLO attainment (Section 2.2, Eq. 1-3): a request meets its TTFT SLO when the
time from its arrival to its first token is within TTFT_SLO, and its TPOT SLO
when the total time of its decode iterations divided by its generation length
L_r is within TPOT_SLO; attainment is the fraction of requests meeting both.

TPOT slack (Sections 2.2 and 4.2): every decode iteration of a request that
takes less than TPOT_SLO adds the difference to the request's slack.  A
prefill chunk may be piggybacked onto the next decode iteration of a
multiplexing worker only if, for every decode request running there, the
predicted iteration time with the chunk fits in one TPOT_SLO plus the slack
the request has accumulated (so its running TPOT stays within the SLO), and
only if the decode batch alone is not already close to the SLO and the
worker's decode KV-cache use is under its HBM watermark (Section 4.3).
"""
from __future__ import annotations

from dataclasses import dataclass, field
from typing import Iterable, List, Optional, Sequence

import numpy as np


@dataclass
class Request:
    rid: int
    arrival: float            # microseconds
    prompt: int               # prompt tokens
    output: int               # tokens to generate, L_r >= 1 (the first comes with the prefill)
    prefilled: int = 0        # prompt tokens processed so far
    first_token: Optional[float] = None
    generated: int = 0        # tokens generated so far
    decode_time: float = 0.0  # sum of the iteration times of its decode steps
    decode_steps: int = 0
    finish: Optional[float] = None
    worker: int = -1          # worker holding its KV cache (decode)
    ready: float = 0.0        # earliest time it may decode (after a KV migration)
    ttft_slo: Optional[float] = None   # this request's TTFT SLO, when SLOs are per request

    @property
    def ttft(self) -> float:
        return self.first_token - self.arrival

    @property
    def tpot(self) -> float:
        return self.decode_time / self.output

    def slack(self, tpot_slo: float) -> float:
        """Accumulated TPOT slack: decode steps so far times the SLO minus
        the time they took."""
        return self.decode_steps * tpot_slo - self.decode_time


@dataclass
class SLO:
    ttft: float               # microseconds (used when a request carries no TTFT SLO of its own)
    tpot: float               # microseconds
    busy_fraction: float = 0.9   # decode batch alone at or above this share of TPOT_SLO: no multiplexing
    hbm_watermark: float = 0.9   # decode KV use above this share of the KV capacity: no multiplexing

    def ttft_of(self, r: "Request") -> float:
        return r.ttft_slo if r.ttft_slo is not None else self.ttft


def attainment(reqs: Sequence[Request], slo: SLO) -> dict:
    """Eq. 1-3 over finished requests, plus the latency percentiles."""
    ttft = np.array([r.ttft for r in reqs])
    tpot = np.array([r.tpot for r in reqs])
    ok_ttft = ttft <= np.array([slo.ttft_of(r) for r in reqs])
    ok_tpot = tpot <= slo.tpot
    n = len(reqs)
    return {
        "attainment": float((ok_ttft & ok_tpot).sum() / n) if n else 1.0,
        "ttft_attainment": float(ok_ttft.mean()) if n else 1.0,
        "tpot_attainment": float(ok_tpot.mean()) if n else 1.0,
        "ttft_p50_us": float(np.percentile(ttft, 50)) if n else 0.0,
        "ttft_p90_us": float(np.percentile(ttft, 90)) if n else 0.0,
        "tpot_p50_us": float(np.percentile(tpot, 50)) if n else 0.0,
        "tpot_p90_us": float(np.percentile(tpot, 90)) if n else 0.0,
        "requests": n,
    }


def admits_chunk(decodes: Iterable[Request], t_base: float, t_with_chunk: float, slo: SLO,
                 kv_use: float = 0.0, kv_capacity: float = float("inf")) -> bool:
    """May a prefill chunk join the next decode iteration of this worker?

    t_base: predicted time of the decode-only iteration; t_with_chunk: with
    the chunk.  Every running decode must keep its TPOT within the SLO after
    this iteration (t_with_chunk <= TPOT_SLO + its accumulated slack); the
    decode batch alone must not already be close to the SLO; the worker's
    decode KV use must be under the watermark."""
    if t_base >= slo.busy_fraction * slo.tpot:
        return False
    if kv_use > slo.hbm_watermark * kv_capacity:
        return False
    for r in decodes:
        if t_with_chunk > slo.tpot + r.slack(slo.tpot):
            return False
    return True
