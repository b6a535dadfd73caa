"""Discrete-event simulator of SLO-aware prefill/decode multiplexing on a group
of workers, driven by the iteration-latency model (per layer, times the model's
layers).

Workers (Section 4.2): prefill workers and multiplexing workers.  A
multiplexing worker runs its decodes and piggybacks a prefill chunk onto its
next decode iteration only when the TPOT-slack test and the decode-batch and HBM
gates pass (slo.admits_chunk); a prefill worker takes a queued request only
when the predicted queueing plus execution time fits the request's remaining
TTFT budget; a request no worker can serve within its SLO any more goes to the
least-loaded prefill worker.  Requests prefilled on a prefill worker migrate to
the multiplexing worker with the fewest unfinished tokens; requests prefilled on
a multiplexing worker decode where they are.

Every decode iteration's time (including the piggybacked chunk) is added to
the decode time of each request in it, so interference shows up in TPOT.
Iteration times are the model's prediction times (1 + e), e drawn from a
normal distribution with the measured relative residual as its deviation;
the scheduler itself decides on the noise-free prediction.
"""
from __future__ import annotations

import heapq
from collections import deque
from dataclasses import dataclass, field
from typing import Dict, List, Optional, Sequence

import numpy as np

from .predictor import LatencyModel, batch_features
from .slo import SLO, Request, admits_chunk, attainment


@dataclass
class Cluster:
    workers: int = 4               # total workers
    prefill_workers: int = 2       # how many of them are prefill workers
    chunk: int = 2048              # chunk size of chunked prefill
    max_batch: int = 256           # running decodes per worker
    layers: int = 32
    kv_bytes_per_token: float = 131072.0   # all layers
    kv_capacity: float = 150e9             # bytes of KV cache per worker
    link_bytes_per_us: float = 153e3       # KV migration bandwidth (one xGMI link)
    noise: float = 0.0                     # relative deviation of actual vs predicted iteration time
    scan: int = 16                         # queued requests a multiplexing worker looks at


@dataclass
class _Worker:
    wid: int
    role: str                      # "prefill" | "mux"
    queue: deque = field(default_factory=deque)     # prefill requests assigned to it
    running: List[Request] = field(default_factory=list)
    pending: deque = field(default_factory=deque)   # waiting for KV room / migration
    prefill: Optional[Request] = None               # request being chunked here
    busy_until: float = 0.0
    busy: bool = False
    kv_use: float = 0.0


class Simulator:
    def __init__(self, model: LatencyModel, cluster: Cluster, slo: SLO, seed: int = 0,
                 trace: bool = False):
        self.m = model
        self.trace = trace
        self.c = cluster
        self.slo = slo
        self.rng = np.random.default_rng(seed)
        if not 1 <= cluster.prefill_workers < cluster.workers:
            raise ValueError("need at least one prefill and one multiplexing worker")
        roles = ["prefill"] * cluster.prefill_workers + ["mux"] * (cluster.workers - cluster.prefill_workers)
        self.w = [_Worker(i, r) for i, r in enumerate(roles)]
        self.toggle: deque = deque()   # requests not yet placed
        self.done: List[Request] = []
        self.events: list = []
        self.seq = 0
        self.log: List[tuple] = []     # (time, worker, kind, detail) for tests

    # ------------------------------------------------------------ latency
    def predict(self, decodes: Sequence[Request], chunk: Optional[tuple] = None) -> float:
        """Predicted iteration time (us) of decodes plus an optional chunk
        (tokens, cached tokens before it)."""
        n_new = [1] * len(decodes)
        ctx = [r.prompt + r.generated - 1 for r in decodes]
        dec = [True] * len(decodes)
        if chunk is not None:
            n_new.append(chunk[0])
            ctx.append(chunk[1])
            dec.append(False)
        if not n_new:
            return 0.0
        return self.m.predict_batch(n_new, ctx, dec) * self.c.layers

    def actual(self, t: float) -> float:
        if self.c.noise <= 0:
            return t
        return t * max(0.5, 1.0 + self.c.noise * self.rng.standard_normal())

    # ------------------------------------------------------------ helpers
    def _push(self, t, kind, payload):
        heapq.heappush(self.events, (t, self.seq, kind, payload))
        self.seq += 1

    def _unfinished(self, w: _Worker) -> float:
        q = sum(r.prompt - r.prefilled for r in w.queue)
        if w.prefill is not None:
            q += w.prefill.prompt - w.prefill.prefilled
        return q + sum(r.output - r.generated for r in w.running) + \
            sum(r.output - r.generated for r in w.pending)

    def _prefill_time(self, r: Request) -> float:
        t = r.prompt - r.prefilled
        return self.m.predict_batch([t], [r.prefilled], [False]) * self.c.layers

    def _queue_time(self, w: _Worker, now: float) -> float:
        start = max(now, w.busy_until) if w.busy else now
        return start - now + sum(self._prefill_time(r) for r in w.queue)

    def _place_decode(self, r: Request, now: float):
        """A request prefilled on a prefill worker: its KV cache migrates to the
        multiplexing worker with the fewest unfinished tokens."""
        w = min((w for w in self.w if w.role == "mux"), key=self._unfinished)
        r.ready = now + r.prompt * self.c.kv_bytes_per_token / self.c.link_bytes_per_us
        r.worker = w.wid
        w.pending.append(r)
        self._kick(w, now)

    def _admit_pending(self, w: _Worker, now: float):
        keep = deque()
        while w.pending:
            r = w.pending.popleft()
            need = (r.prompt + r.output) * self.c.kv_bytes_per_token
            fits = len(w.running) < self.c.max_batch and w.kv_use + need <= self.c.kv_capacity
            if r.ready <= now and (fits or not w.running):  # an idle worker always makes progress
                w.running.append(r)
                w.kv_use += need
            else:
                keep.append(r)
        w.pending = keep

    def _finish_token(self, r: Request, w: _Worker, now: float):
        if r.generated >= r.output:
            r.finish = now
            w.running.remove(r)
            w.kv_use -= (r.prompt + r.output) * self.c.kv_bytes_per_token
            self.done.append(r)

    # ------------------------------------------------------------ dispatch
    def _dispatch(self, now: float):
        # prefill workers take a request when it fits its TTFT budget
        keep = deque()
        while self.toggle:
            r = self.toggle.popleft()
            pws = [w for w in self.w if w.role == "prefill"]
            best = min(pws, key=lambda w: self._queue_time(w, now))
            finish = now + self._queue_time(best, now) + self._prefill_time(r)
            budget = self.slo.ttft_of(r)
            if finish - r.arrival <= budget or now + self._prefill_time(r) - r.arrival > budget:
                # competent, or lost for its SLO anyway: best effort on the least-loaded
                best.queue.append(r)
                self._kick(best, now)
            else:
                keep.append(r)
        self.toggle = keep
        for w in self.w:
            if w.role == "mux":
                self._kick(w, now)

    # ------------------------------------------------------------ iterations
    def _kick(self, w: _Worker, now: float):
        if w.busy:
            return
        self._admit_pending(w, now)
        chunk = None
        prefill_req = None
        decodes = list(w.running)
        if w.role == "prefill":
            if not w.queue:
                return
            prefill_req = w.queue.popleft()
            chunk = (prefill_req.prompt - prefill_req.prefilled, prefill_req.prefilled)
            decodes = []
        else:
            t_base = self.predict(decodes) if decodes else 0.0
            cand = []
            if w.prefill is not None:
                cand = [w.prefill]
            else:
                cand = list(self.toggle)[: self.c.scan]
            for r in cand:
                ch = (min(self.c.chunk, r.prompt - r.prefilled), r.prefilled)
                t_with = self.predict(decodes, ch)
                if admits_chunk(decodes, t_base, t_with, self.slo, w.kv_use, self.c.kv_capacity):
                    if w.prefill is None:
                        self.toggle.remove(r)
                        w.prefill = r
                        if self.trace:
                            self.log.append((now, w.wid, "admit", r.rid))
                    prefill_req, chunk = r, ch
                    break
            if not decodes and chunk is None:
                if w.pending:
                    self._push(min(r.ready for r in w.pending), "wake", w.wid)
                return
        t = self.actual(self.predict(decodes, chunk))
        w.busy = True
        w.busy_until = now + t
        if self.trace:
            self.log.append((now, w.wid, "iter", (len(decodes), chunk)))
        self._push(now + t, "done", (w.wid, decodes, prefill_req, chunk, t))

    def _iteration_done(self, now: float, payload):
        wid, decodes, preq, chunk, t = payload
        w = self.w[wid]
        w.busy = False
        for r in decodes:
            r.generated += 1
            r.decode_time += t
            r.decode_steps += 1
            self._finish_token(r, w, now)
        if preq is not None:
            preq.prefilled += chunk[0]
            if preq.prefilled >= preq.prompt:
                preq.first_token = now
                preq.generated = 1
                if w.role == "mux":
                    w.prefill = None
                if preq.output <= 1:
                    preq.finish = now
                    self.done.append(preq)
                elif w.role == "prefill":
                    self._place_decode(preq, now)
                else:
                    preq.worker = w.wid
                    preq.ready = now
                    w.pending.append(preq)
        if w.role == "prefill":
            self._dispatch(now)
        self._kick(w, now)

    # ------------------------------------------------------------ run
    def run(self, requests: Sequence[Request]) -> Dict:
        for r in requests:
            self._push(r.arrival, "arrive", r)
        while self.events:
            now, _, kind, payload = heapq.heappop(self.events)
            if kind == "arrive":
                self.toggle.append(payload)
                self._dispatch(now)
            elif kind == "done":
                self._iteration_done(now, payload)
            elif kind == "wake":
                self._kick(self.w[payload], now)
            if self.toggle:
                self._dispatch(now)
        if len(self.done) != len(requests):
            raise RuntimeError(f"{len(requests) - len(self.done)} requests never finished")
        return attainment(self.done, self.slo)


def synthetic_requests(rate_per_s: float, n: int, seed: int, prompt_median: float = 2048,
                       output_median: float = 128, sigma_prompt: float = 1.0, sigma_output: float = 0.8,
                       max_prompt: int = 16384, max_output: int = 1024) -> List[Request]:
    """Poisson arrivals with long-tailed (lognormal) prompt and output lengths:
    a synthetic stand-in for a production trace."""
    rng = np.random.default_rng(seed)
    gaps = rng.exponential(1e6 / rate_per_s, size=n)
    t = np.cumsum(gaps)
    p = np.clip(np.round(rng.lognormal(np.log(prompt_median), sigma_prompt, n)), 32, max_prompt).astype(int)
    o = np.clip(np.round(rng.lognormal(np.log(output_median), sigma_output, n)), 1, max_output).astype(int)
    return [Request(i, float(t[i]), int(p[i]), int(o[i])) for i in range(n)]


def light_load_slo(model: LatencyModel, layers: int, prompt_median: int, ctx_median: int,
                   factor: float = 5.0, **gates) -> SLO:
    """SLOs at `factor` times the light-load latency of each phase: the median
    prompt's prefill alone, and one decode step of one request (Section 5.1
    sets them at five times the light-load latency)."""
    ttft = model.predict_batch([prompt_median], [0], [False]) * layers
    tpot = model.predict_batch([1], [ctx_median], [True]) * layers
    return SLO(ttft=factor * ttft, tpot=factor * tpot, **gates)


def per_request_ttft(model: LatencyModel, layers: int, reqs: Sequence[Request], factor: float = 5.0):
    """Give every request a TTFT SLO of `factor` times its own prefill alone
    (the light-load latency of its prefill phase)."""
    for r in reqs:
        r.ttft_slo = factor * model.predict_batch([r.prompt], [0], [False]) * layers


def attainment_sweep(model: LatencyModel, rates: Sequence[float], n: int = 1500, seed: int = 11,
                     workers: int = 4, prefill_workers: int = 2, layers: int = 32, chunk: int = 2048,
                     kv_bytes_per_token: float = 131072.0, kv_capacity: float = 250e9,
                     noise: float = 0.0, prompt_median: int = 2048, output_median: int = 128,
                     slo_factor: float = 5.0) -> Dict:
    """SLO attainment of multiplexed serving over a sweep of arrival rates, one
    synthetic request stream per rate."""
    slo = light_load_slo(model, layers, prompt_median, prompt_median, slo_factor)
    rows = []
    for rate in rates:
        reqs = synthetic_requests(rate, n, seed, prompt_median, output_median)
        per_request_ttft(model, layers, reqs, slo_factor)
        cl = Cluster(workers=workers, prefill_workers=prefill_workers, chunk=chunk, layers=layers,
                     kv_bytes_per_token=kv_bytes_per_token, kv_capacity=kv_capacity, noise=noise)
        rows.append(Simulator(model, cl, slo, seed=seed).run(reqs))
    return {"slo_us": {"ttft_of_median_prompt": slo.ttft, "tpot": slo.tpot,
                       "ttft_rule": f"{slo_factor} x each request's own prefill time alone"},
            "rates": list(rates), "attainment": rows}
