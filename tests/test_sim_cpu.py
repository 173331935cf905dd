"""Closed-loop simulator (include/hwr_sim.h) on the CPU: the library's
hwr_sim_run, driven by the CPU routing oracle through its router callback,
against the reference simulation (oracle/sim_ref.py) -- every request time,
snapshot and metric bit for bit -- and both against closed forms of the
service model on hand-built cases."""
import numpy as np
import pytest

from oracle import oracle as O
from oracle import sim_ref
from paper_2608_14575_amd import hwr, simload

INT_KEYS = ("pair", "first_token_us", "finish_us")
METRIC_KEYS = [k for k in hwr.SIM_METRICS if not k.startswith("route_us")]


def oracle_router(w):
    prob = O.OracleProblem.from_synth(w.problem)
    q = w.queries

    def route(snapshot, r0, r1):
        res = O.route(prob, snapshot, q.emb[r0:r1], q.input_len[r0:r1], q.expected_out_len[r0:r1],
                      q.slo_s[r0:r1], candidates=False)
        return res.choice, res.utility, res.e2e_s
    return route


def sim_args(w):
    return dict(pairs=w.pairs, n_gpus=w.n_gpus, tick_us=w.tick_us, monitor_period_us=w.monitor_period_us,
                max_time_us=w.max_time_us, prior_ttft_s=w.prior_ttft_s, prior_tpot_s=w.prior_tpot_s,
                arrival_us=w.arrival_us, input_len=w.input_len, output_len=w.output_len, slo_us=w.slo_us)


def run_both(w, router, freeze=False):
    lib = hwr.simulate(None, **sim_args(w), router=router, freeze_state=freeze, max_samples=100000)
    ref = sim_ref.simulate(w.pairs, w.n_gpus, w.tick_us, w.monitor_period_us, w.max_time_us,
                           w.prior_ttft_s, w.prior_tpot_s, w.arrival_us, w.input_len, w.output_len,
                           w.slo_us, router, freeze_state=freeze)
    return lib, ref


def assert_same(lib, ref):
    for k in INT_KEYS:
        np.testing.assert_array_equal(lib[k], ref[k], err_msg=k)
    for k in ("utility", "pred_e2e_s"):
        np.testing.assert_array_equal(lib[k].view(np.uint32), ref[k].view(np.uint32), err_msg=k)
    assert lib["samples"].shape == ref["samples"].shape
    assert lib["samples"].tobytes() == ref["samples"].tobytes()
    for k in METRIC_KEYS:
        assert lib[k] == ref[k], (k, lib[k], ref[k])


@pytest.mark.parametrize("pattern,rate,freeze", [("sustained_overload", 18.0, False),
                                                 ("micro_burst", 15.0, False),
                                                 ("poisson", 21.0, True)])
def test_library_matches_reference(pattern, rate, freeze):
    w = simload.make_sim(3, pattern, rate, duration_s=6.0, dtype="f32")
    lib, ref = run_both(w, oracle_router(w), freeze)
    assert lib["n_completed"] == w.n_requests > 50
    assert_same(lib, ref)


def one_pair(max_running=4, kv=100000, pf0=1000, pfn=2000, tp0=500, tpr=100, gpu=0, n=1):
    p = np.zeros(n, simload.PAIR_DTYPE)
    p["gpu"], p["max_running"], p["kv_capacity"] = gpu, max_running, kv
    p["prefill_base_us"], p["prefill_per_token_ns"] = pf0, pfn
    p["tpot_base_us"], p["tpot_per_running_us"] = tp0, tpr
    return p


def fixed_router(choice):
    def route(snapshot, r0, r1):
        n = r1 - r0
        return np.full(n, choice, np.int32), np.zeros(n, np.float32), np.zeros(n, np.float32)
    return route


def run_case(pairs, arrival, inl, outl, slo=None, router=None, n_gpus=1, tick=1000, period=250000,
             max_time=10_000_000, **kw):
    R = len(arrival)
    args = dict(pairs=pairs, n_gpus=n_gpus, tick_us=tick, monitor_period_us=period, max_time_us=max_time,
                prior_ttft_s=np.full(len(pairs), 0.1, np.float32), prior_tpot_s=np.full(len(pairs), 0.01, np.float32),
                arrival_us=np.asarray(arrival, np.int64), input_len=np.asarray(inl, np.int32),
                output_len=np.asarray(outl, np.int32),
                slo_us=np.asarray(slo if slo is not None else [10**9] * R, np.int64))
    router = router or fixed_router(0)
    lib = hwr.simulate(None, **args, router=router, max_samples=10000, **kw)
    ref = sim_ref.simulate(args["pairs"], n_gpus, tick, period, max_time, args["prior_ttft_s"],
                           args["prior_tpot_s"], args["arrival_us"], args["input_len"], args["output_len"],
                           args["slo_us"], router, freeze_state=kw.get("freeze_state", False))
    assert_same(lib, ref)
    return lib


def test_single_request_closed_form():
    # prefill = 1000 us + 300 tokens * 2 us = 1600 us from the arrival (mid-step);
    # then 49 further tokens at 500 us each (one request running)
    a, p, d = 12_345, 300, 50
    out = run_case(one_pair(), [a], [p], [d])
    assert out["first_token_us"][0] == a + 1000 + p * 2000 // 1000
    assert out["finish_us"][0] == a + 1600 + (d - 1) * 500
    assert out["mean_latency_s"] == (1600 + 49 * 500) / 1e6
    assert out["n_completed"] == 1 and out["route_calls"] == 1


def test_single_token_request_ends_with_its_first_token():
    out = run_case(one_pair(), [0], [10], [1])
    assert out["finish_us"][0] == out["first_token_us"][0] == 1000 + 20


def test_batching_slows_every_running_request():
    # two requests together on one pair: B = 2, every token takes 500 + 100 us
    out = run_case(one_pair(), [0, 0], [0 + 1, 1], [11, 11])
    ft = 1000 + 2          # 1 token of prompt: 2000 ns
    np.testing.assert_array_equal(out["first_token_us"], [ft, ft])
    np.testing.assert_array_equal(out["finish_us"], [ft + 10 * 600, ft + 10 * 600])


def test_slots_and_fifo_queueing():
    # one slot: the second request waits for the first to end (its slot frees
    # at the end of that step) and is admitted at the next step boundary
    out = run_case(one_pair(max_running=1), [0, 100], [1, 1], [3, 3])
    f0 = 1002 + 2 * 500
    assert out["finish_us"][0] == f0
    start1 = (f0 // 1000 + 1) * 1000
    assert out["first_token_us"][1] == start1 + 1002
    assert out["finish_us"][1] == start1 + 1002 + 2 * 500


def test_kv_capacity_blocks_admission_but_never_deadlocks():
    # each request needs 60 + 40 = 100 KV tokens; capacity 150 admits one at a
    # time; a lone request larger than the capacity is still admitted
    out = run_case(one_pair(max_running=8, kv=150), [0, 0, 0], [60, 60, 500], [40, 40, 40])
    assert out["n_completed"] == 3
    f = out["finish_us"]
    assert f[0] < out["first_token_us"][1] and f[1] < out["first_token_us"][2]


def test_monitor_snapshot_definition():
    # one request finished inside the first window: the snapshot at 250 ms has
    # its TTFT and TPOT as the window means; GPU utilisation = busy steps / steps
    # (a second request at 300 ms keeps the run going past the 250 ms snapshot)
    a, p, d = 0, 100, 21
    out = run_case(one_pair(), [a, 300_000], [p, p], [d, d], period=250_000, max_time=600_000)
    s = out["samples"]
    ft, fin = out["first_token_us"][0], out["finish_us"][0]
    assert s[0]["ttft_avg_s"] == np.float32(0.1) and s[0]["gpu_util"] == 0.0
    assert s[1]["ttft_avg_s"] == np.float32((ft - a) / 1e6)
    assert s[1]["tpot_avg_s"] == np.float32((fin - ft) / 1e6 / (d - 1))
    busy_steps = fin // 1000 + 1           # steps [0, 1 ms), ... that had the request running
    assert s[1]["gpu_util"] == np.float32(busy_steps / 250)
    assert s[1]["running_q"] == 0 and s[1]["waiting_q"] == 0 and s[1]["kv_util"] == 0.0


def test_load_skew_when_everything_goes_to_one_gpu():
    pairs = np.concatenate([one_pair(max_running=1, gpu=0), one_pair(max_running=1, gpu=1)])
    arrival = np.arange(40) * 20_000          # faster than one slot can serve
    out = run_case(pairs, arrival, [100] * 40, [200] * 40, n_gpus=2, router=fixed_router(0))
    s = out["samples"]
    q0 = (s["running_q"][:, 0].astype(np.int64) + s["waiting_q"][:, 0]).sum() / len(s)
    assert out["load_skew"] == q0 and out["avg_load"] == q0 / 2
    assert out["running_skew"] == s["running_q"][:, 0].sum() / len(s)
    assert out["waiting_skew"] == s["waiting_q"][:, 0].sum() / len(s)
    assert 0.0 < out["running_fraction"] < 0.5


def test_frozen_router_sees_only_the_first_snapshot():
    seen = []

    def rec(snapshot, r0, r1):
        seen.append(snapshot.tobytes())
        return fixed_router(0)(snapshot, r0, r1)
    arrival = np.arange(30) * 50_000
    run_case(one_pair(), arrival, [50] * 30, [100] * 30, router=rec, freeze_state=True)
    assert len(set(seen)) == 1
    seen.clear()
    run_case(one_pair(), arrival, [50] * 30, [100] * 30, router=rec)
    assert len(set(seen)) > 1


def test_slo_attainment_counts_unfinished_requests_as_missed():
    # the run stops at 50 ms: the second request cannot finish
    out = run_case(one_pair(max_running=1), [0, 0], [1, 1], [20, 200], slo=[10**6, 10**6],
                   max_time=50_000)
    assert out["n_completed"] == 1 and out["n_met_slo"] == 1 and out["slo_attainment"] == 0.5
    assert out["finish_us"][1] == -1


@pytest.mark.parametrize("bad", [
    dict(tick_us=0), dict(monitor_period_us=1500), dict(pairs_gpu=3), dict(arrival=[5, 1]),
    dict(output_len=[0, 1]), dict(prior=float("nan"))])
def test_invalid_arguments_are_status_codes(bad):
    pairs = one_pair()
    if "pairs_gpu" in bad:
        pairs["gpu"] = bad["pairs_gpu"]
    args = dict(pairs=pairs, n_gpus=1, tick_us=bad.get("tick_us", 1000),
                monitor_period_us=bad.get("monitor_period_us", 250_000), max_time_us=10**6,
                prior_ttft_s=np.full(1, bad.get("prior", 0.1), np.float32), prior_tpot_s=np.full(1, 0.01, np.float32),
                arrival_us=np.asarray(bad.get("arrival", [0, 1]), np.int64), input_len=np.ones(2, np.int32),
                output_len=np.asarray(bad.get("output_len", [1, 1]), np.int32), slo_us=np.zeros(2, np.int64))
    with pytest.raises(hwr.HwrError) as e:
        hwr.simulate(None, **args, router=fixed_router(0))
    assert e.value.status == hwr.HWR_ERR_INVALID_ARG


def test_router_errors_abort_the_run():
    def bad(snapshot, r0, r1):
        n = r1 - r0
        return np.full(n, 7, np.int32), np.zeros(n, np.float32), np.zeros(n, np.float32)
    with pytest.raises(hwr.HwrError):
        run_case(one_pair(), [0], [1], [1], router=bad)


def test_live_state_balances_the_pool_better_than_a_frozen_one():
    """The paper's claim in this model: with the monitor's signals the router
    spreads a sustained overload over the pool; with the initial snapshot it
    keeps sending each query where the static estimate looks best."""
    w = simload.make_sim(5, "sustained_overload", 21.0, duration_s=20.0, dtype="f32")
    r = oracle_router(w)
    live = hwr.simulate(None, **sim_args(w), router=r)
    frozen = hwr.simulate(None, **sim_args(w), router=r, freeze_state=True)
    assert live["n_completed"] == frozen["n_completed"] == w.n_requests
    assert live["load_skew"] < frozen["load_skew"]
    assert live["running_fraction"] > frozen["running_fraction"]
    assert live["slo_attainment"] > frozen["slo_attainment"]
    assert live["mean_latency_s"] < frozen["mean_latency_s"]


def test_empty_request_stream_and_zero_horizon():
    pairs = one_pair()
    base = dict(pairs=pairs, n_gpus=1, tick_us=1000, monitor_period_us=250_000,
                prior_ttft_s=np.full(1, 0.1, np.float32), prior_tpot_s=np.full(1, 0.01, np.float32),
                arrival_us=np.zeros(0, np.int64), input_len=np.zeros(0, np.int32),
                output_len=np.zeros(0, np.int32), slo_us=np.zeros(0, np.int64))
    out = hwr.simulate(None, **base, max_time_us=10**6, router=fixed_router(0), max_samples=10)
    assert out["n_completed"] == 0 and out["route_calls"] == 0 and out["slo_attainment"] == 0.0
    assert out["n_samples"] == 1 and out["end_us"] == 1000
    out = hwr.simulate(None, **dict(base, arrival_us=np.zeros(1, np.int64), input_len=np.ones(1, np.int32),
                                    output_len=np.ones(1, np.int32), slo_us=np.zeros(1, np.int64)),
                       max_time_us=0, router=fixed_router(0))
    assert out["n_samples"] == 0 and out["route_calls"] == 0 and out["finish_us"][0] == -1
