"""Closed-loop simulator with the HIP router in the loop (hwr_sim_run with a
library context): every routing call is checked against the CPU oracle on
the snapshot that call saw (the acceptance rule of tests/parity.py), and the
reference simulation, replaying the GPU's choices, reproduces every request
time, snapshot and metric bit for bit."""
import numpy as np
import pytest

from oracle import oracle as O
from oracle import sim_ref
from paper_2608_14575_amd import hwr, simload

import gpu_util as GU
import parity
from test_sim_cpu import METRIC_KEYS, assert_same, sim_args

pytestmark = pytest.mark.gpu


def run_gpu(w, freeze=False, **kw):
    r = GU.make_router(w.problem, **kw)
    try:
        out = hwr.simulate(r, **sim_args(w), emb=w.queries.emb_bits, emb_dtype=hwr.HWR_BF16,
                           expected_out_len=w.queries.expected_out_len, freeze_state=freeze,
                           max_samples=10**6)
    finally:
        r.close()
    return out


def check_calls(w, out, freeze):
    """Each request was routed at the start of its step with the snapshot of
    the latest monitor instant (the first one when frozen)."""
    assert out["n_samples"] == len(out["samples"])
    step = w.arrival_us // w.tick_us * w.tick_us
    snap_id = np.zeros_like(step) if freeze else step // w.monitor_period_us
    prob = O.OracleProblem.from_synth(w.problem)
    q = w.queries
    eligible = total = 0
    for k in np.unique(snap_id):
        idx = np.nonzero(snap_id == k)[0]
        orc = O.route(prob, out["samples"][k], q.emb[idx], q.input_len[idx], q.expected_out_len[idx],
                      q.slo_s[idx], candidates=True)
        got = dict(choice=out["pair"][idx], utility=out["utility"][idx], e2e_s=out["pred_e2e_s"][idx])
        rep = parity.compare(got, orc, slo=q.slo_s[idx], alpha=prob.alpha, dep_model=w.problem.dep_model,
                             rtol=1e-2, query_ids=idx, score_mode=prob.score_mode)
        assert rep.ok, rep.failures[:5]
        eligible += rep.eligible
        total += rep.n
    assert total == w.n_requests
    return eligible / total


def replay(w, out, freeze):
    def route(snapshot, r0, r1):
        return out["pair"][r0:r1], out["utility"][r0:r1], out["pred_e2e_s"][r0:r1]
    return sim_ref.simulate(w.pairs, w.n_gpus, w.tick_us, w.monitor_period_us, w.max_time_us,
                            w.prior_ttft_s, w.prior_tpot_s, w.arrival_us, w.input_len, w.output_len,
                            w.slo_us, route, freeze_state=freeze)


@pytest.mark.parametrize("pattern,rate,freeze", [("sustained_overload", 21.0, False),
                                                 ("micro_burst", 18.0, False),
                                                 ("poisson", 15.0, True)])
def test_gpu_router_in_the_loop(pattern, rate, freeze):
    w = simload.make_sim(7, pattern, rate, duration_s=12.0, dtype="bf16")
    out = run_gpu(w, freeze)
    print(f"sim {pattern} rate {rate} freeze {freeze}: {w.n_requests} requests, "
          f"{out['route_calls']} routing calls, p50 {out['route_us_p50']:.1f} us", flush=True)
    assert out["n_completed"] == w.n_requests > 100
    frac = check_calls(w, out, freeze)
    assert frac > 0.5
    ref = replay(w, out, freeze)
    assert_same(out, ref)


def test_gpu_loop_live_state_beats_frozen():
    w = simload.make_sim(8, "sustained_overload", 21.0, duration_s=20.0, dtype="bf16")
    live, frozen = run_gpu(w), run_gpu(w, freeze=True)
    for o, fz in ((live, False), (frozen, True)):
        check_calls(w, o, fz)
    assert live["load_skew"] < frozen["load_skew"]
    assert live["slo_attainment"] > frozen["slo_attainment"]
    assert live["mean_latency_s"] < frozen["mean_latency_s"]


def test_gpu_loop_with_staged_pipeline_matches_fused():
    """The library's two pipelines route the same calls (host batches of
    several queries); choices may differ only inside the epsilon-set, so the
    checks are per call, against the oracle."""
    w = simload.make_sim(9, "micro_burst", 21.0, duration_s=6.0, dtype="bf16")
    for pipe in ("fused", "staged"):
        out = run_gpu(w, pipeline=pipe)
        check_calls(w, out, False)
        assert_same(out, replay(w, out, False))
