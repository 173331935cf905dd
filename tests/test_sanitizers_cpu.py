"""Host code under AddressSanitizer and UndefinedBehaviourSanitizer.

tests/sanitize/driver.cpp is built with gcc/g++ and -fsanitize=address,undefined
(no recovery: any report aborts it) together with the CPU oracle
(oracle/hwr_oracle.c) and the closed-loop simulator
(paper_2608_14575_amd/csrc/hwr_sim.cpp).  It runs the oracle over whole
routing problems (two and three heads, both decision rules, bf16 emulation
and fp32) plus bf16 / softplus sweeps, and the simulator with the oracle as
its router callback; every output must equal, bit for bit, what the
unsanitized builds give on the same inputs (the oracle through
oracle/oracle.py, the simulator through the library's hwr_sim_run).  No
device is needed and no GPU code is built."""
import os
import shutil
import subprocess

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_14575_amd import hwr, simload
from paper_2608_14575_amd import synth as S

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SAN = ["-fsanitize=address,undefined", "-fno-sanitize-recover=all", "-fno-omit-frame-pointer", "-g", "-O1",
       "-ffp-contract=off"]


@pytest.fixture(scope="module")
def driver(tmp_path_factory):
    if shutil.which("gcc") is None or shutil.which("g++") is None:
        pytest.skip("gcc/g++ not available")
    d = tmp_path_factory.mktemp("san")
    inc = ["-I", os.path.join(ROOT, "oracle"), "-I", os.path.join(ROOT, "include")]
    orc = str(d / "hwr_oracle.o")
    sim = str(d / "hwr_sim.o")
    exe = str(d / "driver")
    subprocess.run(["gcc", "-std=c11", *SAN, *inc, "-c", os.path.join(ROOT, "oracle", "hwr_oracle.c"), "-o", orc],
                   check=True)
    subprocess.run(["g++", "-std=c++17", *SAN, *inc, "-c",
                    os.path.join(ROOT, "paper_2608_14575_amd", "csrc", "hwr_sim.cpp"), "-o", sim], check=True)
    subprocess.run(["g++", "-std=c++17", *SAN, *inc, os.path.join(ROOT, "tests", "sanitize", "driver.cpp"),
                    orc, sim, "-lm", "-o", exe], check=True)
    # the instrumentation is really in: both runtimes' entry points are linked
    syms = subprocess.run(["nm", exe], capture_output=True, text=True).stdout
    assert "__asan_init" in syms and "__ubsan_handle" in syms
    return exe


def _write(d, **arrays):
    for k, v in arrays.items():
        np.ascontiguousarray(v).tofile(os.path.join(d, f"{k}.bin"))


def _write_problem(d, prob: O.OracleProblem, extra: dict):
    D, M = np.shape(prob.wq)
    F, H = np.shape(prob.w1)
    meta = dict(M=M, G=prob.n_gpu_types, N=len(prob.dep_model), D=D, F=F, H=H, arch_width=prob.arch_width,
                gpu_width=prob.gpu_width, bf16=int(prob.bf16), n_heads=prob.n_heads, alpha=prob.alpha,
                score_mode=prob.score_mode, bound_mode=prob.bound_mode, ttft_slo_a=prob.ttft_slo_a,
                ttft_slo_b=prob.ttft_slo_b, tpot_slo=prob.tpot_slo, **extra)
    with open(os.path.join(d, "meta.txt"), "w") as fh:
        for k, v in meta.items():
            fh.write(f"{k} {float(v)!r}\n")
    f32 = lambda a: np.asarray(a, np.float32)
    i32 = lambda a: np.asarray(a, np.int32)
    _write(d, dep_model=i32(prob.dep_model), dep_gpu=i32(prob.dep_gpu), model_arch=i32(prob.model_arch),
           model_params_b=f32(prob.model_params_b), wq=f32(prob.wq), bq=f32(prob.bq), w1=f32(prob.w1),
           b1=f32(prob.b1), w2=f32(prob.w2), b2=f32(prob.b2), w3=f32(prob.w3), b3=f32(prob.b3))


def _run(exe, mode, d):
    env = dict(os.environ, ASAN_OPTIONS="detect_leaks=1:abort_on_error=1", UBSAN_OPTIONS="print_stacktrace=1")
    r = subprocess.run([exe, mode, str(d)], capture_output=True, text=True, env=env)
    assert r.returncode == 0, f"sanitized driver failed ({r.returncode}):\n{r.stderr[-4000:]}"


def _read(d, name, dtype):
    return np.fromfile(os.path.join(d, name), dtype=dtype)


def _sweep():
    rng = np.random.default_rng(7)
    vals = [rng.standard_normal(4000).astype(np.float32) * 30,
            np.array([0.0, -0.0, 1.0, -1.0, np.inf, -np.inf, 1e-40, -1e-40, 3.0e38, -3.0e38, 88.0, -88.0,
                      1.00390625, 1.01171875, 1.0 + 2 ** -8, 1.0 + 3 * 2 ** -9], np.float32),
            (np.arange(2000, dtype=np.uint32) * 0x00010000 + 0x00008000).view(np.float32)]   # bf16 ties
    v = np.concatenate(vals).astype(np.float32)
    return v[np.isfinite(v) | np.isinf(v)]


@pytest.mark.parametrize("name,kw,seed", [
    ("C1", dict(), 1),                                              # fp32, two heads
    ("C2", dict(n_queries=48, hidden=64), 2),                       # bf16 emulation
    ("C2", dict(n_queries=40, hidden=64, n_heads=3), 6),            # three heads
    ("C3", dict(n_queries=24, hidden=64, n_models=4, n_gpu_types=2), 3),   # per-query SLO set
])
def test_oracle_under_sanitizers(driver, tmp_path, name, kw, seed):
    sp = S.spec(name, **kw)
    pb, st, qs = S.make_problem(sp, seed), S.make_state(sp, seed), S.make_queries(sp, seed)
    prob = O.OracleProblem.from_synth(pb)
    d = tmp_path
    _write_problem(d, prob, {})
    _write(d, running_q=st["running_q"].astype(np.int32), waiting_q=st["waiting_q"].astype(np.int32),
           kv_util=st["kv_util"].astype(np.float32), gpu_util=st["gpu_util"].astype(np.float32),
           ttft_avg_s=st["ttft_avg_s"].astype(np.float32), tpot_avg_s=st["tpot_avg_s"].astype(np.float32),
           emb=np.asarray(qs.emb, np.float32), input_len=qs.input_len.astype(np.int32),
           expected_out_len=qs.expected_out_len.astype(np.int32), slo_s=qs.slo_s.astype(np.float32),
           sweep=_sweep())
    _run(driver, "route", d)
    ref = O.route_synth(pb, st, qs, candidates=True)
    n, N, M = qs.n, len(pb.dep_model), pb.wq.shape[1]
    np.testing.assert_array_equal(_read(d, "out_choice.bin", np.int32), ref.choice)
    np.testing.assert_array_equal(_read(d, "out_feasible.bin", np.uint8), ref.feasible)
    for fname, arr in (("out_utility.bin", ref.utility), ("out_e2e.bin", ref.e2e_s),
                       ("out_cand_z.bin", ref.cand_z), ("out_cand_ttft.bin", ref.cand_ttft),
                       ("out_cand_tpot.bin", ref.cand_tpot), ("out_cand_u.bin", ref.cand_u),
                       ("out_quality.bin", ref.quality)):
        got = _read(d, fname, np.float32)
        assert got.size == np.size(arr), fname
        assert np.array_equal(got.view(np.uint32), np.ascontiguousarray(arr, np.float32).ravel().view(np.uint32)), fname
    # the decision step alone reproduces the route's decisions
    np.testing.assert_array_equal(_read(d, "dec_choice.bin", np.int32), ref.choice)
    assert np.array_equal(_read(d, "dec_utility.bin", np.float32).view(np.uint32), ref.utility.view(np.uint32))
    sw = _sweep()
    assert np.array_equal(_read(d, "out_bf16.bin", np.float32).view(np.uint32), O.bf16_array(sw).view(np.uint32))
    sp_ref = np.array([O.softplus(float(x)) for x in sw], np.float32)
    assert np.array_equal(_read(d, "out_softplus.bin", np.float32).view(np.uint32), sp_ref.view(np.uint32))
    assert n * N > 0 and M > 0


@pytest.mark.parametrize("pattern,rate,freeze", [("sustained_overload", 18.0, False), ("micro_burst", 15.0, True)])
def test_simulator_under_sanitizers(driver, tmp_path, pattern, rate, freeze):
    w = simload.make_sim(4, pattern, rate, duration_s=3.0, dtype="f32")
    prob = O.OracleProblem.from_synth(w.problem)
    q = w.queries
    d = tmp_path
    max_samples = 1000
    _write_problem(d, prob, dict(n_gpus=w.n_gpus, tick_us=w.tick_us, monitor_period_us=w.monitor_period_us,
                                 max_time_us=w.max_time_us, freeze_state=int(freeze), max_samples=max_samples))
    _write(d, pairs=w.pairs, prior_ttft_s=np.asarray(w.prior_ttft_s, np.float32),
           prior_tpot_s=np.asarray(w.prior_tpot_s, np.float32), arrival_us=np.asarray(w.arrival_us, np.int64),
           input_len=np.asarray(w.input_len, np.int32), output_len=np.asarray(w.output_len, np.int32),
           slo_us=np.asarray(w.slo_us, np.int64), emb=np.asarray(q.emb, np.float32),
           expected_out_len=np.asarray(q.expected_out_len, np.int32), route_slo_s=np.asarray(q.slo_s, np.float32))
    _run(driver, "sim", d)

    def router(snapshot, r0, r1):
        res = O.route(prob, snapshot, q.emb[r0:r1], q.input_len[r0:r1], q.expected_out_len[r0:r1],
                      q.slo_s[r0:r1], candidates=False)
        return res.choice, res.utility, res.e2e_s

    ref = hwr.simulate(None, pairs=w.pairs, n_gpus=w.n_gpus, tick_us=w.tick_us,
                       monitor_period_us=w.monitor_period_us, max_time_us=w.max_time_us,
                       prior_ttft_s=w.prior_ttft_s, prior_tpot_s=w.prior_tpot_s, arrival_us=w.arrival_us,
                       input_len=w.input_len, output_len=w.output_len, slo_us=w.slo_us, router=router,
                       freeze_state=freeze, max_samples=max_samples)
    np.testing.assert_array_equal(_read(d, "sim_pair.bin", np.int32), ref["pair"])
    np.testing.assert_array_equal(_read(d, "sim_first_token_us.bin", np.int64), ref["first_token_us"])
    np.testing.assert_array_equal(_read(d, "sim_finish_us.bin", np.int64), ref["finish_us"])
    for k in ("utility", "pred_e2e_s"):
        assert np.array_equal(_read(d, f"sim_{k}.bin", np.float32).view(np.uint32), ref[k].view(np.uint32)), k
    assert _read(d, "sim_samples.bin", np.uint8).tobytes() == ref["samples"].tobytes()
    m = _read(d, "sim_metrics.bin", np.float64)
    keys = ("n_completed", "n_met_slo", "slo_attainment", "mean_latency_s", "p99_latency_s", "running_fraction",
            "load_skew", "waiting_skew", "mean_utility")
    for k, v in zip(keys, m):
        assert v == float(ref[k]), (k, v, ref[k])
    assert ref["n_completed"] > 20
