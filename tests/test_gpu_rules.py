"""GPU parity of the decision rules beyond the default: the paper's own score
u = (1 - lambda) Q - lambda C (Sec. 3.1), the evaluation's SLO form
B = a + b * input_len + N_out * tpot_slo as the bound of Eq. 3, and several
cost weights scored in one call (a lambda sweep reusing the predictions).
Each weight's decisions are checked against the oracle at that weight, and,
given the GPU's own predictions, against the oracle's decision step exactly."""
import numpy as np
import pytest

from paper_2608_14575_amd import hwr
from paper_2608_14575_amd import synth as S

import gpu_util as G
from test_gpu_decide_exact import _exact

pytestmark = pytest.mark.gpu

RULES = {"paper score": dict(score_mode=1, cost_weight=0.3),
         "paper bound": dict(S.PAPER_SLO),
         "paper both": dict(S.PAPER_SLO, score_mode=1, cost_weight=0.1)}
PER_QUERY = ("choice", "feasible", "utility", "e2e_s", "ttft_s", "tpot_s", "nout")


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    hwr.load()
    yield


def _report(name, rep):
    print(f"[parity] {name}: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:8]


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
@pytest.mark.parametrize("heads", [2, 3])
@pytest.mark.parametrize("rule", sorted(RULES))
def test_rule_parity_and_exact_decisions(rule, heads, pipeline):
    sp = S.spec("C3", n_queries=300, n_heads=heads, **RULES[rule])
    pb, st, qs = S.make_problem(sp, 13), S.make_state(sp, 13), S.make_queries(sp, 13)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    out = G.route_device(r, qs, sp.dtype)
    _report(f"{rule}, {heads} heads, {pipeline}", G.check(pb, st, qs, out))
    _exact(out, pb, qs, sp.cost_weight)


@pytest.mark.parametrize("rule", sorted(RULES))
def test_rule_fp32_host(rule):
    sp = S.spec("C1", n_heads=3, **RULES[rule])
    pb, st, qs = S.make_problem(sp, 1), S.make_state(sp, 1), S.make_queries(sp, 1)
    r = G.make_router(pb)
    r.update(st)
    out = r.route_host(qs.emb_bits, qs.input_len, None, qs.slo_s, candidates=True)
    _report(f"C1 fp32 {rule}", G.check(pb, st, qs, out))
    _exact(out, pb, qs, sp.cost_weight)


SWEEPS = {"lambda (paper score)": (1, [0.0, 0.05, 0.1, 0.3, 0.6, 1.0]),
          "alpha (normalised score)": (0, [0.0, 0.25, 0.5, 2.0])}


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
@pytest.mark.parametrize("heads", [2, 3])
@pytest.mark.parametrize("sweep", sorted(SWEEPS))
def test_weight_sweep(sweep, heads, pipeline):
    """K weights in one call: outputs [n][K]; weight k equals a one-weight
    route at that weight (oracle parity and exact decisions)."""
    mode, ws = SWEEPS[sweep]
    sp = S.spec("C2", n_queries=600, n_heads=heads, score_mode=mode)
    pb, st, qs = S.make_problem(sp, 14), S.make_state(sp, 14), S.make_queries(sp, 14)
    r = G.make_router(pb, pipeline=pipeline, cost_weights=ws)
    r.update(st)
    out = G.route_device(r, qs, sp.dtype)
    assert out["choice"].shape == (qs.n, len(ws))
    for k, w in enumerate(ws):
        sub = {key: out[key][:, k] for key in PER_QUERY}
        sub.update({key: v for key, v in out.items() if key.startswith("cand_")})
        _report(f"{sweep} w={w} {heads} heads {pipeline}", G.check(pb, st, qs, sub, alpha=w))
        _exact(sub, pb, qs, w)
    if mode == 1:
        # lambda = 0 ranks by quality alone, lambda = 1 by cost alone
        rows = np.arange(qs.n)
        c0, c1 = out["choice"][:, 0], out["choice"][:, -1]
        feas_both = out["feasible"][:, 0].astype(bool) & out["feasible"][:, -1].astype(bool)
        Q = out["cand_quality"][:, pb.dep_model]
        assert (Q[rows, c0] >= Q[rows, c1])[feas_both].all()
        assert (out["e2e_s"][:, -1] <= out["e2e_s"][:, 0])[feas_both].all()


@pytest.mark.parametrize("flags", [0, hwr.HWR_FLAG_GRAPH])
@pytest.mark.parametrize("heads", [2, 3])
@pytest.mark.parametrize("rule", sorted(RULES))
def test_single_query_rules(rule, heads, flags):
    """The single-query kernel with each rule (H = 128, 32 pairs)."""
    sp = S.spec("C4", n_queries=40, n_heads=heads, **RULES[rule])
    pb, st, qs = S.make_problem(sp, 15), S.make_state(sp, 15), S.make_queries(sp, 15)
    r = G.make_router(pb, flags=flags)
    r.update(st)
    outs = [r.route_host(one.emb_bits, one.input_len, one.expected_out_len, one.slo_s)
            for one in (qs.slice(i, i + 1) for i in range(qs.n))]
    got = {k: np.concatenate([o[k] for o in outs]) for k in outs[0]}
    _report(f"single {rule} {heads} heads flags={flags}", G.check(pb, st, qs, got))


def test_weight_sweep_single_host_query():
    """One host query with several weights takes the batch path."""
    ws = [0.1, 0.5, 0.9]
    sp = S.spec("C4", n_queries=8, score_mode=1)
    pb, st, qs = S.make_problem(sp, 16), S.make_state(sp, 16), S.make_queries(sp, 16)
    r = G.make_router(pb, cost_weights=ws)
    r.update(st)
    for i in range(qs.n):
        one = qs.slice(i, i + 1)
        got = r.route_host(one.emb_bits, one.input_len, one.expected_out_len, one.slo_s)
        assert got["choice"].shape == (1, 3)
        for k, w in enumerate(ws):
            sub = {key: got[key][:, k] for key in PER_QUERY}
            _report(f"single host query w={w}", G.check(pb, st, one, sub, alpha=w))
