"""Seeded synthetic routing workloads (inputs only).

This module draws every input of the routing problem of HW-Router (Sec. 3.1:
a set of model-GPU pairs and a batch of queries; Sec. 3.2 / Table 2: the
runtime signals the hardware monitor caches per pair) and nothing else.  It
holds none of the method's arithmetic: no feature assembly, no predictor, no
cost, no utility.  Both the CPU oracle (tests) and the HIP path (bench, tests)
take their inputs from here, so neither depends on the other.

The paper's workloads (MiniLM-embedded MixInstruct + LongBench prompts on a
five-pair, two-GPU pool) are not available; the distributions below stand in
for them:

* query embedding e ~ N(0, 1)^D, L2-normalised in fp32 (the paper embeds with a
  384-wide sentence encoder, Sec. 4), rounded to bf16 for bf16 workloads;
* input length = clip(round(exp(N(mu, sigma))), lo, hi) (short instructions
  mixed with long-context prompts);
* expected output length ~ U{64..512};
* per-pair state: running ~ Poisson(4), waiting ~ Poisson(2), kv ~ U[0,1],
  gpu_util ~ U[0,1], recent TTFT ~ lognormal(log 0.2 s, 0.5), recent TPOT ~
  lognormal(log 0.03 s, 0.4); an optional overloaded subset draws waiting ~
  Poisson(20) and kv ~ U[0.8, 1];
* model attributes: parameter count from {1.5, 7, 14, 32, 72} B, architecture
  id = model index mod 4; pairs are the full model x GPU-type product,
  model-major (d = m * G + g);
* predictor weights He-normal (N(0, 2 / fan_in)), hidden biases 0, output bias
  b3 from a stored calibration table (see ``b3_for``); quality head
  Wq ~ N(0, 0.1^2), bq ~ U[0.4, 0.8].

Seeds: ``SeedSequence(seed)`` children with fixed spawn keys, one per draw
group (models, weights, state, state walk, query chunk c), so any chunk can be
regenerated alone.
"""
from __future__ import annotations

import json
import math
import os
from dataclasses import dataclass, field, replace
from typing import Optional

import numpy as np

PARAMS_SET_B = (1.5, 7.0, 14.0, 32.0, 72.0)

# numpy mirror of the 24-byte per-pair runtime record passed to the library.
STATE_DTYPE = np.dtype([
    ("running_q", "<i4"), ("waiting_q", "<i4"),
    ("kv_util", "<f4"), ("gpu_util", "<f4"),
    ("ttft_avg_s", "<f4"), ("tpot_avg_s", "<f4"),
])
assert STATE_DTYPE.itemsize == 24

# spawn-key groups
_K_MODELS, _K_WEIGHTS, _K_STATE, _K_WALK, _K_QUERIES = 0, 1, 2, 3, 4

# targets of the output-bias calibration (recent-TTFT median of the state
# distribution; a per-token latency that makes a few hundred tokens cost ~1-2 s)
B3_TARGET_TTFT_S = 0.2
B3_TARGET_TPOT_S = 0.005
B3_TARGET_NOUT = 288.0          # median of U{64..512}: the given N_out's median
NOUT_HEAD_SCALE = 100.0         # weight scale of the N_out head (tokens per unit)
# The paper's SLO form for the synthetic workloads: TTFT_SLO(p) = a + b p with
# the 1.2x slack folded in (1.2 x (0.2 s + 5e-5 s/token)), TPOT_SLO = 6 ms
# (about the 70th percentile of the calibrated TPOT predictions).
PAPER_SLO = dict(bound_mode=1, ttft_slo_a=0.24, ttft_slo_b=6e-5, tpot_slo=0.006)


@dataclass(frozen=True)
class Spec:
    """Shape and distribution recipe of one synthetic routing workload."""
    name: str
    n_queries: int              # queries per chunk
    n_chunks: int               # chunks (total queries = n_queries * n_chunks)
    n_models: int               # M
    n_gpu_types: int            # G  (pairs N = M * G)
    embed_dim: int              # D
    feat_dim: int               # F (24 or 32)
    hidden: int                 # H
    dtype: str                  # "f32" or "bf16" (embeddings and weights)
    arch_width: int = 4
    gpu_width: int = 3
    cost_weight: float = 0.5    # alpha in u = Q - alpha * E2E / SLO
    slo_kind: str = "fixed"     # fixed | choice | uniform
    slo_value: float = 2.0
    slo_choices: tuple = ()
    slo_range: tuple = ()
    len_mu: float = 6.0
    len_sigma: float = 1.0
    len_lo: int = 16
    len_hi: int = 8192
    nout_lo: int = 64
    nout_hi: int = 512
    overload_frac: float = 0.0
    walk_steps: int = 0
    n_heads: int = 2            # 3: the predictor also predicts N_out (Eq. 1)
    # decision rule: score 0: u = Q - w C / B, 1: u = (1 - w) Q - w C (Sec. 3.1);
    # bound 0: B = the query's SLO, 1: B = a + b p + N_out tpot_slo
    score_mode: int = 0
    bound_mode: int = 0
    ttft_slo_a: float = 0.0
    ttft_slo_b: float = 0.0
    tpot_slo: float = 0.0

    @property
    def n_deployments(self) -> int:
        return self.n_models * self.n_gpu_types

    @property
    def total_queries(self) -> int:
        return self.n_queries * self.n_chunks


SPECS = {
    # 64 queries x 8 pairs (4 models x 2 GPU types), fp32 everywhere
    "C1": Spec("C1", 64, 1, 4, 2, 384, 24, 64, "f32", gpu_width=3,
               slo_kind="fixed", slo_value=2.0),
    # 4096 queries x 16 pairs, bf16 embeddings and weights, fp32 accumulate
    "C2": Spec("C2", 4096, 1, 8, 2, 768, 24, 128, "bf16", gpu_width=3,
               slo_kind="fixed", slo_value=1.5),
    # 65536 queries x 64 pairs, 20% of pairs overloaded, per-query SLO set
    "C3": Spec("C3", 65536, 1, 16, 4, 1024, 32, 256, "bf16", gpu_width=8,
               slo_kind="choice", slo_choices=(0.5, 1.0, 2.0, 5.0),
               overload_frac=0.2),
    # single query x 32 pairs, 10,000 sequential calls with a state walk
    "C4": Spec("C4", 1, 1, 16, 2, 768, 24, 128, "bf16", gpu_width=3,
               slo_kind="fixed", slo_value=1.5, walk_steps=10000),
    # 1,048,576 queries (16 x 65536) x 256 pairs, heavy-tailed input length
    "C5": Spec("C5", 65536, 16, 32, 8, 1536, 32, 256, "bf16", gpu_width=8,
               slo_kind="uniform", slo_range=(0.3, 10.0),
               len_mu=7.0, len_sigma=1.5, len_hi=32768),
}


def spec(name: str, **overrides) -> Spec:
    """A named workload spec, optionally with fields replaced."""
    return replace(SPECS[name], **overrides)


# ---------------------------------------------------------------- bf16 bits
def f32_to_bf16_bits(x: np.ndarray) -> np.ndarray:
    """Round finite fp32 values to the nearest bf16 (ties to even); return raw
    bits.  (For finite inputs the 32-bit sum below cannot overflow.)"""
    u = np.ascontiguousarray(x, dtype=np.float32).view(np.uint32)
    if not np.isfinite(x).all():
        raise ValueError("non-finite input")
    r = u + (np.uint32(0x7FFF) + ((u >> np.uint32(16)) & np.uint32(1)))
    return (r >> np.uint32(16)).astype(np.uint16)


def bf16_bits_to_f32(b: np.ndarray) -> np.ndarray:
    return (np.ascontiguousarray(b, dtype=np.uint16).astype(np.uint32) << np.uint32(16)).view(np.float32)


def _round_to(dtype: str, x: np.ndarray):
    """(values as fp32, bits to hand to the library) for storage dtype."""
    x = np.ascontiguousarray(x, dtype=np.float32)
    if dtype == "bf16":
        bits = f32_to_bf16_bits(x)
        return bf16_bits_to_f32(bits), bits
    return x, x


# ---------------------------------------------------------------- b3 table
_B3_PATH = os.path.join(os.path.dirname(__file__), "b3_table.json")
_B3_CACHE: Optional[dict] = None


def _b3_table() -> dict:
    global _B3_CACHE
    if _B3_CACHE is None:
        try:
            with open(_B3_PATH) as f:
                _B3_CACHE = json.load(f)
        except FileNotFoundError:
            _B3_CACHE = {}
    return _B3_CACHE


def softplus_inverse(y: float) -> float:
    return math.log(math.expm1(y))


def b3_targets(n_heads: int = 2) -> list:
    t = [B3_TARGET_TTFT_S, B3_TARGET_TPOT_S]
    return t + [B3_TARGET_NOUT] if n_heads == 3 else t


def b3_default(n_heads: int = 2) -> np.ndarray:
    return np.array([softplus_inverse(t) for t in b3_targets(n_heads)], dtype=np.float32)


def b3_for(sp: Spec, seed: int) -> np.ndarray:
    """Output bias for (spec, seed).

    The stored table holds, per named workload and seed, the bias that puts the
    median predicted TTFT / TPOT (and N_out with three heads) at the initial
    state on the targets above (written by tests/golden/make_b3_table.py,
    which runs the CPU oracle).  Any other (spec, seed) gets
    softplus^-1(target) with no calibration.
    """
    ent = _b3_table().get(b3_key(sp, seed))
    if ent is None:
        return b3_default(sp.n_heads)
    return np.array(ent, dtype=np.float32)


def b3_key(sp: Spec, seed: int) -> str:
    key = f"{sp.name}:{seed}:{sp.embed_dim}:{sp.feat_dim}:{sp.hidden}:{sp.n_models}x{sp.n_gpu_types}"
    return key + ":h3" if sp.n_heads == 3 else key


# ---------------------------------------------------------------- draws
def _rng(seed: int, *key: int) -> np.random.Generator:
    return np.random.default_rng(np.random.SeedSequence(seed, spawn_key=tuple(key)))


@dataclass
class Problem:
    """Everything hwr_init takes: pairs, model attributes, weights."""
    spec: Spec
    seed: int
    dep_model: np.ndarray       # int32 [N]
    dep_gpu: np.ndarray         # int32 [N]
    model_arch: np.ndarray      # int32 [M]
    model_params_b: np.ndarray  # float32 [M]
    # weights as fp32 values (exactly the bf16 values for bf16 workloads) ...
    wq: np.ndarray              # [D, M]
    w1: np.ndarray              # [F, H]
    w2: np.ndarray              # [H, H]
    w3: np.ndarray              # [H, n_heads]
    # ... and as the bits handed to the library (uint16 for bf16, else float32)
    wq_bits: np.ndarray
    w1_bits: np.ndarray
    w2_bits: np.ndarray
    w3_bits: np.ndarray
    bq: np.ndarray              # float32 [M]
    b1: np.ndarray              # float32 [H]
    b2: np.ndarray              # float32 [H]
    b3: np.ndarray              # float32 [n_heads]

    @property
    def n_deployments(self) -> int:
        return int(self.dep_model.shape[0])


@dataclass
class Queries:
    emb: np.ndarray             # float32 [n, D] values (bf16-exact for bf16)
    emb_bits: np.ndarray        # uint16 [n, D] (bf16) or float32 [n, D]
    input_len: np.ndarray       # int32 [n]
    expected_out_len: np.ndarray  # int32 [n]
    slo_s: np.ndarray           # float32 [n]

    @property
    def n(self) -> int:
        return int(self.input_len.shape[0])

    def slice(self, a: int, b: int) -> "Queries":
        return Queries(self.emb[a:b], self.emb_bits[a:b], self.input_len[a:b],
                       self.expected_out_len[a:b], self.slo_s[a:b])

    def take(self, idx) -> "Queries":
        idx = np.asarray(idx)
        return Queries(self.emb[idx], self.emb_bits[idx], self.input_len[idx],
                       self.expected_out_len[idx], self.slo_s[idx])


def make_problem(sp: Spec, seed: int, b3: Optional[np.ndarray] = None) -> Problem:
    M, G, D, F, H = sp.n_models, sp.n_gpu_types, sp.embed_dim, sp.feat_dim, sp.hidden
    rm = _rng(seed, _K_MODELS)
    params = rm.choice(np.array(PARAMS_SET_B), size=M).astype(np.float32)
    arch = (np.arange(M) % sp.arch_width).astype(np.int32)
    dep_model = np.repeat(np.arange(M, dtype=np.int32), G)
    dep_gpu = np.tile(np.arange(G, dtype=np.int32), M)

    rw = _rng(seed, _K_WEIGHTS)
    w1 = rw.standard_normal((F, H)) * math.sqrt(2.0 / F)
    w2 = rw.standard_normal((H, H)) * math.sqrt(2.0 / H)
    w3 = rw.standard_normal((H, 2)) * math.sqrt(2.0 / H)
    wq = rw.standard_normal((D, M)) * 0.1
    bq = rw.uniform(0.4, 0.8, size=M).astype(np.float32)
    if sp.n_heads == 3:
        # the N_out head is drawn after everything else, so the other weights
        # equal the two-head problem's; it works in tokens, hence the scale
        w3 = np.hstack([w3, rw.standard_normal((H, 1)) * math.sqrt(2.0 / H) * NOUT_HEAD_SCALE])
    elif sp.n_heads != 2:
        raise ValueError("n_heads must be 2 or 3")
    w1v, w1b = _round_to(sp.dtype, w1)
    w2v, w2b = _round_to(sp.dtype, w2)
    w3v, w3b = _round_to(sp.dtype, w3)
    wqv, wqb = _round_to(sp.dtype, wq)
    if b3 is None:
        b3 = b3_for(sp, seed)
    return Problem(sp, seed, dep_model, dep_gpu, arch, params,
                   wqv, w1v, w2v, w3v, wqb, w1b, w2b, w3b, bq,
                   np.zeros(H, np.float32), np.zeros(H, np.float32),
                   np.asarray(b3, dtype=np.float32).copy())


def make_state(sp: Spec, seed: int) -> np.ndarray:
    """Initial per-pair runtime signals (Table 2 plus GPU utilisation)."""
    N = sp.n_deployments
    r = _rng(seed, _K_STATE)
    st = np.zeros(N, dtype=STATE_DTYPE)
    st["running_q"] = r.poisson(4.0, N)
    st["waiting_q"] = r.poisson(2.0, N)
    st["kv_util"] = r.uniform(0.0, 1.0, N)
    st["gpu_util"] = r.uniform(0.0, 1.0, N)
    st["ttft_avg_s"] = np.exp(r.normal(math.log(0.2), 0.5, N))
    st["tpot_avg_s"] = np.exp(r.normal(math.log(0.03), 0.4, N))
    if sp.overload_frac > 0.0:
        k = int(round(sp.overload_frac * N))
        over = r.permutation(N)[:k]
        st["waiting_q"][over] = r.poisson(20.0, k)
        st["kv_util"][over] = r.uniform(0.8, 1.0, k)
    return st


def overloaded_pairs(sp: Spec, seed: int) -> np.ndarray:
    """Indices of the overloaded subset drawn by make_state (empty if none)."""
    N = sp.n_deployments
    if sp.overload_frac <= 0.0:
        return np.zeros(0, np.int64)
    r = _rng(seed, _K_STATE)
    r.poisson(4.0, N); r.poisson(2.0, N); r.uniform(0.0, 1.0, N); r.uniform(0.0, 1.0, N)
    r.normal(0.0, 0.5, N); r.normal(0.0, 0.4, N)
    k = int(round(sp.overload_frac * N))
    return np.sort(r.permutation(N)[:k])


class StateWalk:
    """Random walk of the runtime signals between sequential single-query
    calls: queue lengths move by U{-1, 0, +1} (clipped at 0), KV utilisation
    drifts by N(0, 0.02) (clipped to [0, 1]); other signals are held."""

    def __init__(self, sp: Spec, seed: int, state0: Optional[np.ndarray] = None):
        self.state = (make_state(sp, seed) if state0 is None else state0).copy()
        self._r = _rng(seed, _K_WALK)

    def step(self) -> np.ndarray:
        N = self.state.shape[0]
        r = self._r
        dr = r.integers(-1, 2, N)
        dw = r.integers(-1, 2, N)
        dk = r.normal(0.0, 0.02, N)
        st = self.state
        st["running_q"] = np.maximum(st["running_q"] + dr, 0)
        st["waiting_q"] = np.maximum(st["waiting_q"] + dw, 0)
        st["kv_util"] = np.clip(st["kv_util"] + dk, 0.0, 1.0).astype(np.float32)
        return st.copy()


def make_queries(sp: Spec, seed: int, chunk: int = 0, n: Optional[int] = None) -> Queries:
    """Queries of chunk ``chunk`` (independent stream per chunk)."""
    if n is None:
        n = sp.n_queries
    D = sp.embed_dim
    r = _rng(seed, _K_QUERIES, chunk)
    e = r.standard_normal((n, D), dtype=np.float32)
    nrm = np.sqrt(np.einsum("ij,ij->i", e, e, dtype=np.float32)).astype(np.float32)
    e /= np.maximum(nrm, np.float32(1e-30))[:, None]
    ev, eb = _round_to(sp.dtype, e)
    ln = np.rint(np.exp(r.normal(sp.len_mu, sp.len_sigma, n)))
    input_len = np.clip(ln, sp.len_lo, sp.len_hi).astype(np.int32)
    nout = r.integers(sp.nout_lo, sp.nout_hi + 1, n).astype(np.int32)
    if sp.slo_kind == "fixed":
        slo = np.full(n, sp.slo_value, np.float32)
    elif sp.slo_kind == "choice":
        slo = r.choice(np.array(sp.slo_choices, np.float32), size=n).astype(np.float32)
    elif sp.slo_kind == "uniform":
        slo = r.uniform(sp.slo_range[0], sp.slo_range[1], n).astype(np.float32)
    else:
        raise ValueError(sp.slo_kind)
    return Queries(ev, eb, input_len, nout, slo)


def custom_spec(name="custom", **kw) -> Spec:
    """Small ad-hoc workloads for tests (any field of Spec)."""
    base = dict(n_queries=16, n_chunks=1, n_models=3, n_gpu_types=2, embed_dim=64,
                feat_dim=24, hidden=64, dtype="f32", gpu_width=3)
    base.update(kw)
    return Spec(name, **base)
