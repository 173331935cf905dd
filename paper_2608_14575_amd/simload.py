"""Seeded inputs of the closed-loop serving simulation (inputs only).

The paper evaluates routers on a vLLM deployment of five models on two H100
GPUs (Table 3), under three arrival patterns -- Poisson, micro-burst and
sustained overload -- at 15-21 requests per second (Sec. 5).  That cluster,
its trained predictor and its prompt sets are not available; this module
draws stand-ins of the same structure for ``hwr_sim_run`` (include/hwr_sim.h):

* the pool: Table 3's placement -- Phi-3-mini (3.8 B) and Qwen2.5-14B on GPU 0;
  Qwen2.5-3B, Mistral-7B and Llama-3.1-8B on GPU 1 -- one pair per model;
* a serving model per pair, from its parameter count P (billions):
  prefill 20 ms + 2 P us per prompt token, decode 4 + 0.5 P ms per token at one
  running request plus 2% of that per further request running on the same GPU,
  16 batch slots and 30,000 KV-cache tokens (all slots busy, the pool serves
  about 21 requests per second);
* requests: prompt length clip(round(exp(N(6, 1))), 16, 8192), output length
  U{64..512} (given to the router as N_out: a two-head predictor), embedding
  N(0, 1)^384 normalised (the paper's encoder width) and rounded to bf16;
* the latency bound of Sec. 5: B = a + b p + d TPOT_SLO with a = 0.3 s,
  b = 1e-4 s per prompt token and TPOT_SLO = 20 ms (d = output tokens); the
  router uses the same form with its N_out, the evaluation the true d;
* arrivals over ``duration_s`` at mean rate ``rate`` per second:
  ``poisson`` -- exponential gaps; ``micro_burst`` -- each second, 40% of the
  rate arrives in its first 100 ms and 60% in the rest (Poisson counts,
  uniform times); ``sustained_overload`` -- one request every 1/rate s with a
  uniform jitter of one gap (no lulls; rates above the pool's capacity);
* predictor weights set by hand (the trained predictor is not available, and a
  randomly drawn one knows nothing about this serving model), a load-aware
  predictor of the paper's form (Eq. 1: two ReLU layers, softplus heads) with
  TTFT ~ ttft_avg (1 + waiting) (p / 512)^(1/2) and
  TPOT ~ tpot_avg (1 + running)^(1/2) (see ``handset_predictor``);
* quality heads Wq ~ N(0, 0.1^2), bq = 0.40 + 0.06 ln P (larger models score
  higher on average).
"""
from __future__ import annotations

import math
from dataclasses import dataclass
from typing import Optional

import numpy as np

from . import synth as S

# Table 3 of the paper: (model, parameters in billions, GPU)
POOL = (("Phi-3-mini", 3.8, 0), ("Qwen2.5-14B", 14.0, 0),
        ("Qwen2.5-3B", 3.0, 1), ("Mistral-7B", 7.0, 1), ("Llama-3.1-8B", 8.0, 1))
SIM_SLO = dict(ttft_slo_a=0.3, ttft_slo_b=1e-4, tpot_slo=0.020)
PATTERNS = ("poisson", "micro_burst", "sustained_overload")

# numpy mirror of hwr_sim_pair (32 bytes)
PAIR_DTYPE = np.dtype([("gpu", "<i4"), ("max_running", "<i4"), ("kv_capacity", "<i8"),
                       ("prefill_base_us", "<i4"), ("prefill_per_token_ns", "<i4"),
                       ("tpot_base_us", "<i4"), ("tpot_per_running_us", "<i4")])
assert PAIR_DTYPE.itemsize == 32

_K_SIM_REQ, _K_SIM_ARR, _K_SIM_W = 10, 11, 12


def sim_spec(dtype: str = "bf16", hidden: int = 64, embed_dim: int = 384) -> S.Spec:
    """Routing problem of the simulated pool (5 models, 2 GPUs, one pair each)."""
    return S.Spec("SIM", 1, 1, len(POOL), 2, embed_dim, 24, hidden, dtype, gpu_width=3,
                  slo_kind="fixed", slo_value=6.0, bound_mode=1, **SIM_SLO)


def handset_predictor(F: int, H: int, A: int, Gw: int):
    """W1 [F][H], b1 [H], W2 [H][H], W3 [H][2] and b3 [2] of the load-aware
    predictor (module docstring).  Feature slots follow include/hwr.h:
    b = A + Gw; b+1 ln(p)/8, b+2 ln(1+running)/2, b+3 ln(1+waiting)/2,
    b+6 ln(ttft_avg)/4, b+7 ln(tpot_avg)/4.

    Layer 1 forms s = ln(ttft_avg) + ln(1 + waiting) + (ln p - ln 512) / 2 as
    ReLU(s) - ReLU(-s) plus hinge units ReLU(s - t_k) at knots t_k; layer 2
    passes them on (identity); the TTFT head sums them into the piecewise-linear
    interpolant of softplus^-1(e^s), so softplus(z) ~ e^s over s in [-3, 8]
    (e^s from 0.05 s to 50 min).  TPOT stays in the region where softplus(z) ~ e^z:
    z = ln(tpot_avg) + ln(1 + running) / 2."""
    b = A + Gw
    knots = np.arange(-3.0, 8.0 + 1e-9, 0.5)
    assert 4 + knots.size <= H and b + 7 < F
    w1 = np.zeros((F, H), np.float32)
    b1 = np.zeros(H, np.float32)
    w2 = np.eye(H, dtype=np.float32)
    w3 = np.zeros((H, 2), np.float32)
    s_terms = ((b + 6, 4.0), (b + 3, 2.0), (b + 1, 4.0))     # s = sum of coef * feature + s0
    s0 = -0.5 * math.log(512.0)
    units = [(+1.0, 0.0), (-1.0, 0.0)] + [(+1.0, -t) for t in knots]   # (sign, knot offset)
    for j, (sign, off) in enumerate(units):
        for slot, c in s_terms:
            w1[slot, j] = sign * c
        b1[j] = sign * s0 + off
    # the target f(s) = softplus^-1(e^s) - s, interpolated linearly between knots
    y = np.exp(knots)
    f = y + np.log(-np.expm1(-y)) - knots          # softplus^-1(y) = y + ln(1 - e^-y)
    slopes = np.diff(f) / np.diff(knots)
    w3[0, 0], w3[1, 0] = 1.0, -1.0
    prev = 0.0
    for k in range(slopes.size):
        w3[2 + k, 0] = slopes[k] - prev
        prev = slopes[k]
    jt = 2 + knots.size
    for j, sign in ((jt, 1.0), (jt + 1, -1.0)):
        w1[b + 7, j], w1[b + 2, j] = 4.0 * sign, 1.0 * sign
        w3[j, 1] = sign
    b3 = np.array([f[0], 0.0], np.float32)
    return w1, b1, w2, w3, b3


@dataclass
class SimWorkload:
    problem: S.Problem
    pairs: np.ndarray            # PAIR_DTYPE [N]
    n_gpus: int
    prior_ttft_s: np.ndarray     # float32 [N]
    prior_tpot_s: np.ndarray     # float32 [N]
    arrival_us: np.ndarray       # int64 [R]
    input_len: np.ndarray        # int32 [R]
    output_len: np.ndarray       # int32 [R]
    slo_us: np.ndarray           # int64 [R]
    queries: S.Queries           # what the router sees (expected_out_len = output_len)
    tick_us: int = 1000
    monitor_period_us: int = 250_000
    max_time_us: int = 0
    pattern: str = "poisson"
    rate: float = 0.0
    duration_s: float = 0.0

    @property
    def n_requests(self) -> int:
        return int(self.arrival_us.shape[0])


def arrivals(pattern: str, rate: float, duration_s: float, rng: np.random.Generator) -> np.ndarray:
    """Arrival times in microseconds, sorted (module docstring)."""
    if pattern == "poisson":
        n_max = int(rate * duration_s * 2 + 64)
        t = np.cumsum(rng.exponential(1.0 / rate, n_max))
        t = t[t < duration_s]
    elif pattern == "micro_burst":
        parts = []
        for k in range(int(math.ceil(duration_s))):
            nb, nl = rng.poisson(0.4 * rate), rng.poisson(0.6 * rate)
            parts.append(k + rng.uniform(0.0, 0.1, nb))
            parts.append(k + rng.uniform(0.1, 1.0, nl))
        t = np.sort(np.concatenate(parts)) if parts else np.zeros(0)
        t = t[t < duration_s]
    elif pattern == "sustained_overload":
        n = int(rate * duration_s)
        t = (np.arange(n) + rng.uniform(0.0, 1.0, n)) / rate
        t = np.sort(t[t < duration_s])
    else:
        raise ValueError(f"unknown arrival pattern {pattern!r}")
    return np.floor(t * 1e6).astype(np.int64)


def make_sim(seed: int = 1, pattern: str = "sustained_overload", rate: float = 18.0,
             duration_s: float = 60.0, dtype: str = "bf16", drain_s: float = 600.0,
             monitor_period_us: int = 250_000, tick_us: int = 1000,
             n_requests: Optional[int] = None) -> SimWorkload:
    """The simulated pool and a request stream (``n_requests`` truncates it)."""
    sp = sim_spec(dtype)
    M, D, F, H = sp.n_models, sp.embed_dim, sp.feat_dim, sp.hidden
    params = np.array([p for _, p, _ in POOL], np.float32)
    gpu = np.array([g for _, _, g in POOL], np.int32)
    rw = S._rng(seed, _K_SIM_W)
    wq = rw.standard_normal((D, M)) * 0.1
    bq = (0.40 + 0.06 * np.log(params.astype(np.float64))).astype(np.float32)
    w1, b1, w2, w3, b3 = handset_predictor(F, H, sp.arch_width, sp.gpu_width)
    w1v, w1b = S._round_to(dtype, w1)
    w2v, w2b = S._round_to(dtype, w2)
    w3v, w3b = S._round_to(dtype, w3)
    wqv, wqb = S._round_to(dtype, wq)
    pb = S.Problem(sp, seed, np.arange(M, dtype=np.int32), gpu, (np.arange(M) % sp.arch_width).astype(np.int32),
                   params, wqv, w1v, w2v, w3v, wqb, w1b, w2b, w3b, bq, b1, np.zeros(H, np.float32), b3)

    pairs = np.zeros(M, PAIR_DTYPE)
    pairs["gpu"] = gpu
    pairs["max_running"] = 16
    pairs["kv_capacity"] = 30_000
    pairs["prefill_base_us"] = 20_000
    pairs["prefill_per_token_ns"] = np.rint(2000.0 * params).astype(np.int32)
    tpot = np.rint(4000.0 + 500.0 * params).astype(np.int32)
    pairs["tpot_base_us"] = tpot
    pairs["tpot_per_running_us"] = np.rint(0.02 * tpot).astype(np.int32)
    prior_ttft = ((pairs["prefill_base_us"] + 512 * pairs["prefill_per_token_ns"] // 1000) / 1e6).astype(np.float32)
    prior_tpot = (tpot / 1e6).astype(np.float32)

    t = arrivals(pattern, rate, duration_s, S._rng(seed, _K_SIM_ARR))
    if n_requests is not None:
        t = t[:n_requests]
    R = t.shape[0]
    rr = S._rng(seed, _K_SIM_REQ)
    e = rr.standard_normal((R, D), dtype=np.float32)
    nrm = np.sqrt(np.einsum("ij,ij->i", e, e, dtype=np.float32)).astype(np.float32)
    e /= np.maximum(nrm, np.float32(1e-30))[:, None]
    ev, eb = S._round_to(dtype, e)
    input_len = np.clip(np.rint(np.exp(rr.normal(6.0, 1.0, R))), 16, 8192).astype(np.int32)
    output_len = rr.integers(64, 513, R).astype(np.int32)
    a, b, ts = SIM_SLO["ttft_slo_a"], SIM_SLO["ttft_slo_b"], SIM_SLO["tpot_slo"]
    slo_us = np.rint(1e6 * (a + b * input_len.astype(np.float64) + ts * output_len)).astype(np.int64)
    q = S.Queries(ev, eb, input_len, output_len.copy(), np.full(R, sp.slo_value, np.float32))
    return SimWorkload(pb, pairs, 2, prior_ttft, prior_tpot, t, input_len, output_len, slo_us, q,
                       tick_us=tick_us, monitor_period_us=monitor_period_us,
                       max_time_us=int((duration_s + drain_s) * 1e6), pattern=pattern, rate=rate,
                       duration_s=duration_s)
