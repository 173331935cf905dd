"""Benchmark: batched routing-score evaluation on one MI355X.

Step = one call of hwr_route_batch over the whole throughput workload
(1,048,576 queries x 256 model-GPU pairs, 16 chunks of 65,536 queries on one
stream, inputs resident in HBM).  Prints one JSON line with candidates
scored per second, the roofline position of the dominant kernel (the fused
predictor, MFMA-bound) measured with HIP events on the launch stream, the
single-query latency path (p50 / p99 over 10,000 sequential calls with a
state update between calls), and the CPU oracle timed on a bounded sample.

    python bench.py [--gpus 1] [--steps 10] [--warmup 2]
"""
from __future__ import annotations

import argparse
import ctypes as C
import glob
import hashlib
import json
import os
import re
import sys
import time

import numpy as np

ROOT = os.path.dirname(os.path.abspath(__file__))
sys.path.insert(0, ROOT)

# The HIP runtime's replay of captured graphs: with its packet capture off, a
# one-kernel graph (the single-query graph launch mode) launches about 5 us
# sooner on this stack.  Read when the runtime starts, so set before torch is
# imported; an explicit setting in the environment is kept.
GRAPH_ENV = ("DEBUG_CLR_GRAPH_PACKET_CAPTURE", "0")
os.environ.setdefault(*GRAPH_ENV)

METRIC = "routing candidates scored/sec (query×deployment) at 1 MI355X; p50 1-query route µs"
PEAK_BF16_TFLOPS = 2500.0      # MI355X dense bf16 MFMA
PEAK_HBM_GBS = 8000.0          # MI355X HBM3E
PROFILE_EVERY = 4              # kernel timing samples one launch in four of each kernel


TRAFFIC_FILE = os.path.join(ROOT, "profiles", "hbm_traffic_C5_1Mx256.json")
KERNEL_NAMES = {   # as the profiler names them
    "fused": "void hwr::k_mlp_bf16<256, false, 2, true, 4, true>(hwr::MlpArgs)",
    "mlp": "void hwr::k_mlp_bf16<256, true, 2, true, 4, false>(hwr::MlpArgs)",
    "quality": "hwr::k_quality_bf16_lds(hwr::QualityArgs)",
    "gather": "hwr::k_gather(hwr::GatherArgs)",
    "epilogue": "void hwr::k_epilogue<false, false, false, false>(hwr::EpilogueArgs)",
}


def source_hash() -> str:
    """sha256 of the library's HIP sources with comments and whitespace
    removed: changes to code change it, changes to comments do not."""
    h = hashlib.sha256()
    csrc = os.path.join(ROOT, "paper_2608_14575_amd", "csrc")
    for f in sorted(glob.glob(os.path.join(csrc, "*.hip")) + glob.glob(os.path.join(csrc, "*.hpp"))):
        with open(f) as fh:
            text = fh.read()
        text = re.sub(r"/\*.*?\*/", " ", text, flags=re.S)
        text = re.sub(r"//[^\n]*", " ", text)
        h.update(os.path.basename(f).encode())
        h.update(" ".join(text.split()).encode())
    return h.hexdigest()


def counter_traffic(workload: str) -> dict:
    """HBM bytes per launch (FETCH_SIZE + WRITE_SIZE, scaled by the copy
    calibration) from the committed counter summary of this workload -- only
    while the kernel sources are the ones the counters were taken on."""
    if workload != "C5" or not os.path.exists(TRAFFIC_FILE):
        return {}
    with open(TRAFFIC_FILE) as fh:
        rec = json.load(fh)
    if rec.get("source_sha256") != source_hash():
        return {}
    per = {k: v["fetch_bytes"] + v["write_bytes"] for k, v in rec["kernels"].items()}
    return {short: per[name] for short, name in KERNEL_NAMES.items() if name in per}


def log(msg: str) -> None:
    print(f"[bench] {msg}", file=sys.stderr, flush=True)


def predictor_flops(F: int, H: int) -> int:
    """Algorithmic flops of the Eq. 1 predictor per candidate: 2(FH + H^2 + 2H)."""
    return 2 * (F * H + H * H + 2 * H)


def prepare(args, S, torch):
    """The throughput workload, generated chunk by chunk and made resident in
    HBM before any timing."""
    sp = S.spec(args.workload)
    pb, st = S.make_problem(sp, args.seed), S.make_state(sp, args.seed)
    n, D = sp.total_queries, sp.embed_dim
    dev = torch.device("cuda:0")
    emb = torch.empty((n, D), dtype=torch.int16, device=dev)
    il = torch.empty(n, dtype=torch.int32, device=dev)
    no = torch.empty(n, dtype=torch.int32, device=dev)
    slo = torch.empty(n, dtype=torch.float32, device=dev)
    sample = None
    for c in range(sp.n_chunks):
        qs = S.make_queries(sp, args.seed, chunk=c)
        a, b = c * sp.n_queries, (c + 1) * sp.n_queries
        emb[a:b] = torch.from_numpy(qs.emb_bits.view(np.int16)).to(dev)
        il[a:b] = torch.from_numpy(qs.input_len).to(dev)
        no[a:b] = torch.from_numpy(qs.expected_out_len).to(dev)
        slo[a:b] = torch.from_numpy(qs.slo_s).to(dev)
        if c == 0:
            sample = qs.slice(0, args.cpu_sample)
            sample_wide = qs.slice(0, 4 * args.cpu_sample)
        log(f"generated chunk {c + 1}/{sp.n_chunks}")
    return dict(sp=sp, pb=pb, st=st, emb=emb, il=il, no=no, slo=slo, sample=sample, sample_wide=sample_wide)


def hbm_line(nbytes: float, avg_ms: float, kernel: str, traffic=None, direction: str = "read") -> dict:
    gbs = nbytes / (avg_ms / 1e3) / 1e9 if avg_ms > 0 else 0.0
    return {"bound": "hbm", "achieved": gbs, "peak": PEAK_HBM_GBS, "unit": "GB/s",
            "frac": gbs / PEAK_HBM_GBS, "traffic": traffic, "bytes_per_launch": nbytes,
            "avg_launch_ms": avg_ms, "kernel": kernel, "hbm_dir": direction}


def throughput(args, hwr, torch, w, pipeline, steps, warmup):
    """Time `steps` calls of hwr_route_batch over the whole workload with one
    pipeline; per-kernel durations from the library's HIP events on the
    stream the kernels run on."""
    sp = w["sp"]
    n, N, M, D = sp.total_queries, sp.n_deployments, sp.n_models, sp.embed_dim
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    r = hwr.Router.from_problem(w["pb"], max_chunk=sp.n_queries, pipeline=pipeline,
                                stream=int(stream.cuda_stream))
    r.update(w["st"])
    out = dict(choice=torch.empty(n, dtype=torch.int32, device=dev),
               feasible=torch.empty(n, dtype=torch.uint8, device=dev),
               utility=torch.empty(n, dtype=torch.float32, device=dev),
               e2e_s=torch.empty(n, dtype=torch.float32, device=dev),
               ttft_s=torch.empty(n, dtype=torch.float32, device=dev),
               tpot_s=torch.empty(n, dtype=torch.float32, device=dev))

    def step():
        r.route(w["emb"], w["il"], w["no"], w["slo"], mem=hwr.HWR_MEM_DEVICE, **out)

    for _ in range(warmup):
        step()
    torch.cuda.synchronize()
    log(f"{pipeline}: warmup done ({warmup} steps)")
    # one launch in four of each kernel carries the dispatch-recorded events:
    # a timed launch is dispatched a few microseconds later, which on 32
    # back-to-back launches per step would cost the step about 0.7%
    r.profile(PROFILE_EVERY)
    r.profile_read(reset=True)
    ev = [torch.cuda.Event(enable_timing=True) for _ in range(steps + 1)]
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    ev[0].record(stream)
    for i in range(steps):
        step()
        ev[i + 1].record(stream)
    torch.cuda.synchronize()
    wall = time.perf_counter() - t0
    kt = r.profile_read(reset=True)
    r.profile(False)
    gpu_ms = ev[0].elapsed_time(ev[-1])
    per_step = np.array([ev[i].elapsed_time(ev[i + 1]) for i in range(steps)])
    log(f"{pipeline}: timed {steps} steps: {gpu_ms:.2f} ms (events), {wall * 1e3:.2f} ms (host)")
    choice = out["choice"].cpu().numpy()
    assert (choice >= 0).all() and (choice < N).all(), "choice out of range"
    r.close()
    ms_step = max(gpu_ms, wall * 1e3) / steps
    value = n * N / (ms_step / 1e3)

    def avg(k):
        ms, cnt = kt[k]
        return ms / cnt if cnt else 0.0

    kname = "fused" if pipeline == "fused" else "mlp"
    k_avg_ms = avg(kname)
    traffic = counter_traffic(args.workload)
    nq = sp.n_queries
    chunk_cands = nq * N
    flops = predictor_flops(sp.feat_dim, sp.hidden) * chunk_cands
    achieved = flops / (k_avg_ms / 1e3) / 1e12
    qflops = 2 * nq * D * M
    qk_ms = k_avg_ms + avg("quality")
    with_q = (flops + qflops) / (qk_ms / 1e3) / 1e12 if qk_ms > 0 else 0.0
    stages = {k: {"avg_ms": (v[0] / v[1]) if v[1] else 0.0, "timed_launches": v[1]}
              for k, v in kt.items() if v[1]}
    res = dict(
        value=value, ms_per_step=ms_step, stages=stages,
        step_ms={"median": float(np.median(per_step)), "p10": float(np.percentile(per_step, 10)),
                 "p90": float(np.percentile(per_step, 90)), "steps": steps},
        roofline={"bound": "mfma", "achieved": achieved, "peak": PEAK_BF16_TFLOPS, "unit": "TFLOP/s",
                  "frac": achieved / PEAK_BF16_TFLOPS, "traffic": traffic.get(kname),
                  "kernel": f"k_mlp_bf16<{sp.hidden}> ({pipeline})",
                  "flop_per_launch": flops, "avg_launch_ms": k_avg_ms,
                  # the predictor and the quality GEMM together, per chunk
                  "with_quality": {"achieved": with_q, "frac": with_q / PEAK_BF16_TFLOPS,
                                   "flop_per_chunk": flops + qflops}},
        # per chunk: embeddings read, Q matrix written, heads read once
        quality_roofline=hbm_line(nq * (D * 2 + M * 4) + D * 32 * 2, avg("quality"), "k_quality_bf16_lds",
                                  traffic.get("quality")),
        config={"workload": f"{sp.name} throughput stress: {n} queries x {N} pairs ({M} models x "
                            f"{sp.n_gpu_types} GPU types), embed {D} bf16, predictor "
                            f"{sp.feat_dim}-{sp.hidden}-{sp.hidden}-2 bf16/fp32-acc, "
                            f"{sp.n_chunks} chunks of {nq} on one stream",
                "queries": n, "pairs": N, "chunk": nq, "pipeline": pipeline, "seed": args.seed},
    )
    if pipeline == "staged":
        # gather: writes the feature matrix X (64 B per candidate), reads the
        # input lengths and the pair rows; epilogue: reads TTFT and TPOT
        # (8 B per candidate), the Q matrix, N_out and the bound, writes
        # choice, feasible and four floats per query
        res["gather_roofline"] = hbm_line(chunk_cands * 64 + nq * 4 + N * 64, avg("gather"), "k_gather",
                                          traffic.get("gather"), "write")
        res["epilogue_roofline"] = hbm_line(chunk_cands * 8 + nq * (M * 4 + 8 + 21), avg("epilogue"),
                                            "k_epilogue", traffic.get("epilogue"))
    return res


def single_query(args, S, hwr, torch, flags=0):
    """p50 / p99 of hwr_route_batch for one host query, with the runtime
    signals updated (random walk) between calls; host clock around the call.
    flags = 0: plain kernel launch; HWR_FLAG_GRAPH: graph launch."""
    sp = S.spec("C4")
    pb = S.make_problem(sp, 4)
    walk = S.StateWalk(sp, 4)
    r = hwr.Router.from_problem(pb, stream=int(torch.cuda.current_stream().cuda_stream), flags=flags)
    r.update(walk.state)
    calls = args.c4_calls
    qs = S.make_queries(sp, 4, n=calls)
    L = hwr.load()
    emb = np.zeros((1, sp.embed_dim), np.uint16)
    il = np.zeros(1, np.int32)
    no = np.zeros(1, np.int32)
    slo = np.zeros(1, np.float32)
    outs = [np.zeros(1, np.int32), np.zeros(1, np.uint8)] + [np.zeros(1, np.float32) for _ in range(4)]
    b = hwr.hwr_query_batch(1, hwr.HWR_MEM_HOST, emb.ctypes.data, il.ctypes.data, no.ctypes.data,
                            slo.ctypes.data)
    res = hwr.hwr_route_result(choice=outs[0].ctypes.data, feasible=outs[1].ctypes.data,
                               utility=outs[2].ctypes.data, e2e_s=outs[3].ctypes.data,
                               ttft_s=outs[4].ctypes.data, tpot_s=outs[5].ctypes.data)
    bref, rref = C.byref(b), C.byref(res)
    ctx = r.ctx
    route_ns = np.zeros(calls, np.int64)
    upd_ns = np.zeros(calls, np.int64)
    for i in range(calls + 100):
        k = i % calls
        st = walk.step()
        t0 = time.perf_counter_ns()
        rc = L.hwr_update_hw_state(ctx, st.ctypes.data, st.shape[0])
        t1 = time.perf_counter_ns()
        assert rc == 0, hwr.hwr_last_error(ctx)
        emb[0] = qs.emb_bits[k]
        il[0], no[0], slo[0] = qs.input_len[k], qs.expected_out_len[k], qs.slo_s[k]
        t2 = time.perf_counter_ns()
        rc = L.hwr_route_batch(ctx, bref, rref)
        t3 = time.perf_counter_ns()
        assert rc == 0, hwr.hwr_last_error(ctx)
        if i >= 100:                     # the first 100 calls warm up
            route_ns[k], upd_ns[k] = t3 - t2, t1 - t0
    r.close()
    us = route_ns / 1e3
    return {"calls": calls, "p50_us": float(np.percentile(us, 50)), "p99_us": float(np.percentile(us, 99)),
            "mean_us": float(us.mean()), "update_p50_us": float(np.percentile(upd_ns / 1e3, 50)),
            "workload": "C4: 1 query x 32 pairs (16 models x 2 GPU types), embed 768 bf16, "
                        "predictor 24-128-128-2, host I/O, "
                        + {0: "kernel launch", hwr.HWR_FLAG_GRAPH: "graph launch",
                           hwr.HWR_FLAG_RESIDENT: "resident kernel (no launch per call)"}[flags],
            "timing": "host clock around hwr_route_batch (ctypes call included)"}


def batch_latency(args, S, hwr, torch):
    """Latency of one hwr_route_batch call on device-resident inputs for the
    smaller routing workloads (C1 fp32; C2, C3 bf16), one chunk each: the C
    function called directly (argument structs built once, as a C caller
    would), HIP events on the call's stream around each call; median and p99
    over `--batch-calls` calls after 10 untimed ones."""
    L = hwr.load()
    dev = torch.device("cuda:0")
    stream = torch.cuda.current_stream()
    res = {}
    for name in ("C1", "C2", "C3"):
        sp = S.spec(name)
        pb, st, qs = S.make_problem(sp, args.seed), S.make_state(sp, args.seed), S.make_queries(sp, args.seed)
        emb_np = qs.emb_bits.view(np.int16) if sp.dtype == "bf16" else np.ascontiguousarray(qs.emb_bits, np.float32)
        emb = torch.from_numpy(np.ascontiguousarray(emb_np)).to(dev)
        il = torch.from_numpy(np.ascontiguousarray(qs.input_len)).to(dev)
        no = torch.from_numpy(np.ascontiguousarray(qs.expected_out_len)).to(dev)
        slo = torch.from_numpy(np.ascontiguousarray(qs.slo_s)).to(dev)
        n, N = qs.n, sp.n_deployments
        out = dict(choice=torch.empty(n, dtype=torch.int32, device=dev),
                   feasible=torch.empty(n, dtype=torch.uint8, device=dev),
                   utility=torch.empty(n, dtype=torch.float32, device=dev),
                   e2e_s=torch.empty(n, dtype=torch.float32, device=dev),
                   ttft_s=torch.empty(n, dtype=torch.float32, device=dev),
                   tpot_s=torch.empty(n, dtype=torch.float32, device=dev))
        r = hwr.Router.from_problem(pb, max_chunk=n, stream=int(stream.cuda_stream))
        r.update(st)
        qb = hwr.hwr_query_batch(n, hwr.HWR_MEM_DEVICE, emb.data_ptr(), il.data_ptr(), no.data_ptr(),
                                 slo.data_ptr())
        rr = hwr.hwr_route_result(**{k: v.data_ptr() for k, v in out.items()})
        qref, rref, ctx = C.byref(qb), C.byref(rr), r.ctx
        calls = args.batch_calls
        ev = [(torch.cuda.Event(enable_timing=True), torch.cuda.Event(enable_timing=True)) for _ in range(calls)]
        for _ in range(10):
            assert L.hwr_route_batch(ctx, qref, rref) == 0, hwr.hwr_last_error(ctx)
        torch.cuda.synchronize()
        for a, b in ev:
            a.record(stream)
            rc = L.hwr_route_batch(ctx, qref, rref)
            b.record(stream)
            assert rc == 0, hwr.hwr_last_error(ctx)
        torch.cuda.synchronize()
        choice = out["choice"].cpu().numpy()
        assert (choice >= 0).all() and (choice < N).all(), "choice out of range"
        r.close()
        us = np.array([a.elapsed_time(b) * 1e3 for a, b in ev])
        p50 = float(np.percentile(us, 50))
        res[name] = {"queries": n, "pairs": N, "candidates": n * N, "dtype": sp.dtype,
                     "predictor": f"{sp.feat_dim}-{sp.hidden}-{sp.hidden}-2", "embed_dim": sp.embed_dim,
                     "calls": calls, "p50_us": p50, "p99_us": float(np.percentile(us, 99)),
                     "candidates_per_s_at_p50": n * N / (p50 / 1e6),
                     "timing": "HIP events on the stream around each C call (host enqueue included)"}
        log(f"batch latency {name}: {n} x {N}, p50 {p50:.1f} us")
    return res


def closed_loop(args, hwr, torch):
    """The closed-loop serving simulation (include/hwr_sim.h) with the library
    routing every step's arrivals: Table 3's pool of five models on two GPUs,
    each arrival pattern at one rate, with the monitor's signals refreshed
    every 250 ms (live) or held at the first snapshot (frozen).  Reports the
    paper's Sec. 5 metrics and the host time of each routing call."""
    from paper_2608_14575_amd import simload
    keys = ("slo_attainment", "mean_latency_s", "p99_latency_s", "mean_ttft_s", "running_fraction",
            "avg_load", "load_skew", "running_skew", "waiting_skew", "n_completed", "route_calls",
            "route_us_p50", "route_us_p99")
    out = {}
    runs = [(p, args.sim_rate) for p in simload.PATTERNS]
    runs += [("sustained_overload", float(x)) for x in args.sim_overload_rates.split(",") if x
             and float(x) != args.sim_rate]
    for pattern, rate in runs:
        w = simload.make_sim(11, pattern, rate, duration_s=args.sim_seconds, dtype="bf16")
        row = {"requests": w.n_requests, "rate": rate}
        for mode, freeze in (("live", False), ("frozen", True)):
            r = hwr.Router.from_problem(w.problem, stream=int(torch.cuda.current_stream().cuda_stream))
            t0 = time.perf_counter()
            o = hwr.simulate(r, pairs=w.pairs, n_gpus=w.n_gpus, tick_us=w.tick_us,
                             monitor_period_us=w.monitor_period_us, max_time_us=w.max_time_us,
                             prior_ttft_s=w.prior_ttft_s, prior_tpot_s=w.prior_tpot_s,
                             arrival_us=w.arrival_us, input_len=w.input_len, output_len=w.output_len,
                             slo_us=w.slo_us, emb=w.queries.emb_bits, emb_dtype=hwr.HWR_BF16,
                             expected_out_len=w.queries.expected_out_len, freeze_state=freeze)
            wall = time.perf_counter() - t0
            r.close()
            row[mode] = {k: o[k] for k in keys}
            row[mode]["wall_s"] = wall
        out[pattern if rate == args.sim_rate else f"{pattern}@{rate:g}"] = row
        log(f"closed loop {pattern} at {rate} req/s: SLO attainment live "
            f"{row['live']['slo_attainment']:.3f} / frozen {row['frozen']['slo_attainment']:.3f}, "
            f"load skew {row['live']['load_skew']:.2f} / {row['frozen']['load_skew']:.2f}, "
            f"routing call p50 {row['live']['route_us_p50']:.1f} us")
    return {"workload": f"Table 3 pool (5 models, 2 GPUs), {args.sim_seconds:g} s of arrivals at "
                        f"{args.sim_rate:g} req/s per pattern (sustained overload also at "
                        f"{args.sim_overload_rates} req/s), 1 ms steps, monitor every 250 ms, "
                        f"hand-set load-aware predictor 24-64-64-2 bf16, embed 384",
            "timing": "host clock around each hwr_route_batch call of the simulation (host batches)",
            "patterns": out}


def closed_loop_pareto(args, hwr, torch):
    """The quality-latency trade-off of the paper's Fig. 4(a), in the closed
    loop: sustained overload on Table 3's pool, one simulation per cost weight,
    live and frozen monitor.  The quality of each served request is the
    library's own Q for the chosen pair's model (one device batch with the
    per-model quality output after the run)."""
    from paper_2608_14575_amd import simload
    w = simload.make_sim(12, "sustained_overload", args.pareto_rate, duration_s=args.sim_seconds, dtype="bf16")
    dev = torch.device("cuda:0")
    stream = int(torch.cuda.current_stream().cuda_stream)
    q = w.queries
    emb = torch.from_numpy(q.emb_bits.view(np.int16)).to(dev)
    il = torch.from_numpy(q.input_len).to(dev)
    no = torch.from_numpy(q.expected_out_len).to(dev)
    R, M = w.n_requests, w.problem.wq.shape[1]
    rows = []
    for alpha in [float(x) for x in args.pareto_weights.split(",") if x]:
        r = hwr.Router.from_problem(w.problem, cost_weight=alpha, stream=stream)
        r.update(_idle_state(w, hwr))
        qual = torch.empty((R, M), dtype=torch.float32, device=dev)
        choice = torch.empty(R, dtype=torch.int32, device=dev)
        r.route(emb, il, no, None, mem=hwr.HWR_MEM_DEVICE, choice=choice, cand_quality=qual)
        torch.cuda.synchronize()
        qual = qual.cpu().numpy()
        row = {"cost_weight": alpha}
        for mode, freeze in (("live", False), ("frozen", True)):
            o = hwr.simulate(r, pairs=w.pairs, n_gpus=w.n_gpus, tick_us=w.tick_us,
                             monitor_period_us=w.monitor_period_us, max_time_us=w.max_time_us,
                             prior_ttft_s=w.prior_ttft_s, prior_tpot_s=w.prior_tpot_s,
                             arrival_us=w.arrival_us, input_len=w.input_len, output_len=w.output_len,
                             slo_us=w.slo_us, emb=q.emb_bits, emb_dtype=hwr.HWR_BF16,
                             expected_out_len=q.expected_out_len, freeze_state=freeze)
            chosen_model = w.problem.dep_model[o["pair"]]
            row[mode] = {"mean_quality": float(qual[np.arange(R), chosen_model].mean()),
                         "mean_latency_s": o["mean_latency_s"], "p99_latency_s": o["p99_latency_s"],
                         "slo_attainment": o["slo_attainment"], "load_skew": o["load_skew"]}
        r.close()
        rows.append(row)
        log(f"pareto weight {alpha}: live quality {row['live']['mean_quality']:.4f} latency "
            f"{row['live']['mean_latency_s']:.2f} s / frozen {row['frozen']['mean_quality']:.4f} "
            f"{row['frozen']['mean_latency_s']:.2f} s")
    return {"workload": f"Table 3 pool, sustained overload at {args.pareto_rate:g} req/s for "
                        f"{args.sim_seconds:g} s, one run per cost weight",
            "quality": "the library's Q of the chosen pair's model (per-model quality output)",
            "points": rows}


def host_batches(args, hwr, torch, w):
    """Host-memory batches (HWR_MEM_HOST) of the first `--host-chunks` C5
    chunks, PCIe-inclusive (never `value`): the same queries routed from
    pageable and from pinned host memory, best of three calls each; both
    give the same bits."""
    sp, k = w["sp"], args.host_chunks
    n = k * sp.n_queries
    emb = w["emb"][:n].cpu().numpy().view(np.uint16)
    il, no, slo = (w[x][:n].cpu().numpy() for x in ("il", "no", "slo"))
    r = hwr.Router.from_problem(w["pb"], max_chunk=sp.n_queries)
    r.update(w["st"])
    res, outs = {}, {}
    pin = lambda x: torch.from_numpy(np.ascontiguousarray(x)).pin_memory().numpy()
    for name, arrays in (("pageable", (emb, il, no, slo)),
                         ("pinned", (pin(emb.view(np.int16)).view(np.uint16), pin(il), pin(no), pin(slo)))):
        r.route_host(*(a[:sp.n_queries] for a in arrays))       # first use: staging set up
        best = None
        for _ in range(3):
            t0 = time.perf_counter()
            outs[name] = r.route_host(*arrays)
            dt = time.perf_counter() - t0
            best = dt if best is None else min(best, dt)
        res[name] = {"ms": best * 1e3, "candidates_per_s": n * sp.n_deployments / best,
                     "embedding_gb_per_s": emb.nbytes / best / 1e9}
        log(f"host batch ({name}): {n} queries in {best * 1e3:.1f} ms, {res[name]['candidates_per_s']:.3e} "
            f"candidates/s, {res[name]['embedding_gb_per_s']:.1f} GB/s of embeddings")
    r.close()
    assert all(np.array_equal(outs["pageable"][x], outs["pinned"][x]) for x in outs["pinned"])
    res["workload"] = f"{k} C5 chunks ({n} queries x {sp.n_deployments} pairs, {emb.nbytes / 1e6:.0f} MB of embeddings)"
    res["timing"] = "host clock around hwr_route_batch (HWR_MEM_HOST), upload and copy-back included"
    return res


def _idle_state(w, hwr):
    """The monitor's first snapshot of an idle pool (what the simulation
    starts from), for the quality-only batch before a run."""
    st = np.zeros(len(w.pairs), hwr.STATE_DTYPE)
    st["ttft_avg_s"], st["tpot_avg_s"] = w.prior_ttft_s, w.prior_tpot_s
    return st


def cpu_baseline(pb, st, sample, sp, sample_wide=None):
    """The CPU oracle (plain C, one thread) on a bounded sample of the same
    workload: the first queries of chunk 0 against all pairs.  With
    `sample_wide`, also the same oracle on all host threads (up to 16, the
    CPU share of one GPU): one shard of the wider sample per thread (the C
    call releases the interpreter lock)."""
    from oracle import oracle as O
    O.build(force=False)
    O.lib()
    t0 = time.perf_counter()
    O.route_synth(pb, st, sample, candidates=False)
    dt = time.perf_counter() - t0
    cands = sample.n * sp.n_deployments
    wide = None
    if sample_wide is not None:
        from concurrent.futures import ThreadPoolExecutor
        threads = max(1, min(os.cpu_count() or 1, 16))
        bounds = np.linspace(0, sample_wide.n, threads + 1).astype(int)
        shards = [sample_wide.slice(int(a), int(b)) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]
        t1 = time.perf_counter()
        with ThreadPoolExecutor(max_workers=len(shards)) as ex:
            list(ex.map(lambda q: O.route_synth(pb, st, q, candidates=False), shards))
        dtw = time.perf_counter() - t1
        wc = sample_wide.n * sp.n_deployments
        wide = {"value": wc / dtw, "unit": "candidates/s", "cores": len(shards),
                "sample": f"first {sample_wide.n} queries of chunk 0 x {sp.n_deployments} pairs "
                          f"({wc} candidates, {dtw:.1f} s, {len(shards)} threads)"}
    cpu = "unknown"
    try:
        with open("/proc/cpuinfo") as fh:
            cpu = next(line.split(":", 1)[1].strip() for line in fh if line.startswith("model name"))
    except (OSError, StopIteration):
        pass
    return {"value": cands / dt, "unit": "candidates/s", "cores": 1, "kind": "oracle",
            "sample": f"first {sample.n} queries of chunk 0 x {sp.n_deployments} pairs "
                      f"({cands} candidates, {dt:.1f} s, one thread)",
            "host_cpu": cpu, "host_threads": os.cpu_count(), "all_cores": wide}


PROBE_READ_BYTES = 4 << 30     # read-ceiling buffer: 16x the last-level cache


def peak_probes(hwr, torch) -> dict:
    """Achievable ceilings of this device, measured now with the library's
    probe kernels: the register-fed bf16 MFMA rate (the better of one and two
    waves per SIMD; launches of ~4 ms, long enough for the power limit to
    act) and the streaming read rate of a 4 GiB buffer (the best of 1, 2, 4
    and 8 waves per SIMD).  Each figure is the median of its timed launches."""
    mfma_clk = {w: hwr.hwr_probe_mfma_bf16(0, w, 16384, 9) for w in (1, 2)}
    mfma = {w: v[0] for w, v in mfma_clk.items()}
    buf = torch.ones(PROBE_READ_BYTES // 4, dtype=torch.int32, device="cuda:0")
    read = {w: hwr.hwr_probe_hbm_read(0, buf.data_ptr(), PROBE_READ_BYTES, w, 9) for w in (1, 2, 4, 8)}
    write = {w: hwr.hwr_probe_hbm_write(0, buf.data_ptr(), PROBE_READ_BYTES, w, 9) for w in (1, 2, 4, 8)}
    del buf
    torch.cuda.synchronize()
    res = {"mfma_bf16_tflops": max(mfma.values()),
           "mfma_bf16_by_waves_per_simd": {str(k): v for k, v in mfma.items()},
           # shader clock during the product loops (the published peak
           # assumes 2.4 GHz)
           "mfma_clock_mhz_by_waves_per_simd": {str(k): v[1] for k, v in mfma_clk.items()},
           "hbm_read_gbs": max(read.values()),
           "hbm_read_by_waves_per_simd": {str(k): v for k, v in read.items()},
           "hbm_write_gbs": max(write.values()),
           "hbm_write_by_waves_per_simd": {str(k): v for k, v in write.items()},
           "probes": "hwr_probe_mfma_bf16 (32x32x16 bf16, register operands, 8 chains per wave), "
                     f"hwr_probe_hbm_read ({PROBE_READ_BYTES >> 30} GiB streaming read, non-temporal 16-byte loads), "
                     f"hwr_probe_hbm_write (the same buffer, 16-byte stores)"}
    log(f"ceilings: MFMA bf16 {res['mfma_bf16_tflops']:.0f} TFLOP/s at "
        f"{mfma_clk[max(mfma, key=mfma.get)][1]:.0f} MHz "
        f"({res['mfma_bf16_tflops'] / PEAK_BF16_TFLOPS:.3f} of nominal), HBM read "
        f"{res['hbm_read_gbs']:.0f} GB/s ({res['hbm_read_gbs'] / PEAK_HBM_GBS:.3f} of nominal), HBM write "
        f"{res['hbm_write_gbs']:.0f} GB/s ({res['hbm_write_gbs'] / PEAK_HBM_GBS:.3f} of nominal)")
    return res


def with_achievable(line: dict, ceilings: dict) -> dict:
    """Adds the fraction of the measured ceiling of the line's bound next to
    the fraction of the published peak: the MFMA ceiling, or the HBM read or
    write ceiling by the kernel's dominant direction (`hbm_dir`)."""
    if line is None or not ceilings:
        return line
    if line["bound"] == "mfma":
        peak = ceilings["mfma_bf16_tflops"]
    else:
        peak = ceilings["hbm_write_gbs" if line.get("hbm_dir") == "write" else "hbm_read_gbs"]
    line["achievable_peak"] = peak
    line["achievable_frac"] = line["achieved"] / peak if peak > 0 else None
    if "with_quality" in line:
        line["with_quality"]["achievable_frac"] = line["with_quality"]["achieved"] / peak if peak > 0 else None
    return line


def copy_probe(torch) -> int:
    """A plain device-to-device copy of 1 GiB, three times: the reference
    for scaling the FETCH_SIZE / WRITE_SIZE counters to bytes."""
    nbytes = 1 << 30
    src = torch.ones(nbytes // 4, dtype=torch.float32, device="cuda:0")
    dst = torch.empty_like(src)
    for _ in range(3):
        dst.copy_(src)
    torch.cuda.synchronize()
    print(json.dumps({"copy_probe_bytes_read": nbytes, "copy_probe_bytes_written": nbytes,
                      "launches": 3}), flush=True)
    return 0


def main() -> int:
    ap = argparse.ArgumentParser()
    ap.add_argument("--gpus", type=int, default=1)
    ap.add_argument("--steps", type=int, default=10)
    ap.add_argument("--warmup", type=int, default=2)
    ap.add_argument("--workload", default="C5")
    ap.add_argument("--pipeline", default="fused", choices=["fused", "staged"])
    ap.add_argument("--seed", type=int, default=5)
    ap.add_argument("--staged-steps", type=int, default=5,
                    help="steps of the staged pipeline (gather / epilogue HBM figures); 0 skips it")
    ap.add_argument("--c4-calls", type=int, default=10000)
    ap.add_argument("--cpu-sample", type=int, default=1024)
    ap.add_argument("--host-chunks", type=int, default=4,
                    help="C5 chunks routed from host memory, pageable and pinned (0: skip)")
    ap.add_argument("--batch-calls", type=int, default=200,
                    help="timed calls per workload for the C1-C3 batch latencies (0: skip)")
    ap.add_argument("--no-cpu-baseline", action="store_true")
    ap.add_argument("--no-single", action="store_true")
    ap.add_argument("--no-sim", action="store_true", help="skip the closed-loop simulation")
    ap.add_argument("--sim-rate", type=float, default=21.0)
    ap.add_argument("--sim-seconds", type=float, default=60.0)
    ap.add_argument("--pareto-weights", default="0,0.25,0.5,1,2,4",
                    help="cost weights of the closed-loop quality-latency sweep ('' skips it)")
    ap.add_argument("--pareto-rate", type=float, default=18.0)
    ap.add_argument("--sim-overload-rates", default="15,18,21",
                    help="extra sustained-overload arrival rates (the paper sweeps 15, 18, 21 req/s)")
    ap.add_argument("--copy-probe", action="store_true",
                    help="only run a plain device copy of known size (counter calibration)")
    ap.add_argument("--peak-probe", action="store_true",
                    help="only measure the achievable MFMA and HBM-read ceilings and print them")
    ap.add_argument("--no-peak-probe", action="store_true",
                    help="skip the ceiling probes (rooflines carry the nominal fraction only)")
    args = ap.parse_args()
    if args.gpus != 1 or int(os.environ.get("WORLD_SIZE", "1")) != 1:
        print("bench.py measures one GPU only: the library has no multi-GPU path "
              "(run with --gpus 1)", file=sys.stderr)
        return 2
    import torch
    from paper_2608_14575_amd import hwr
    from paper_2608_14575_amd import synth as S
    if not torch.cuda.is_available():
        print("bench.py needs a GPU", file=sys.stderr)
        return 2
    torch.cuda.set_device(0)
    if args.copy_probe:
        return copy_probe(torch)
    hwr.load()
    if args.peak_probe:
        print(json.dumps(peak_probes(hwr, torch)), flush=True)
        return 0
    w = prepare(args, S, torch)
    res = throughput(args, hwr, torch, w, args.pipeline, args.steps, args.warmup)
    log(f"throughput {res['value']:.3e} candidates/s, predictor {res['roofline']['achieved']:.1f} TFLOP/s")
    staged = None
    if args.pipeline == "fused" and args.staged_steps > 0:
        sr = throughput(args, hwr, torch, w, "staged", args.staged_steps, 1)
        staged = {"value": sr["value"], "unit": "candidates/s", "ms_per_step": sr["ms_per_step"],
                  "steps": args.staged_steps, "gather_roofline": sr["gather_roofline"],
                  "epilogue_roofline": sr["epilogue_roofline"], "mlp_roofline": sr["roofline"],
                  "stages": sr["stages"]}
        log(f"staged: gather {sr['gather_roofline']['frac']:.2f} of HBM, "
            f"epilogue {sr['epilogue_roofline']['frac']:.2f} of HBM")
    # ceilings measured right after the throughput steps, in the same power
    # and thermal state
    ceilings = None if args.no_peak_probe else peak_probes(hwr, torch)
    if ceilings:
        with_achievable(res["roofline"], ceilings)
        with_achievable(res["quality_roofline"], ceilings)
        if staged:
            for k in ("gather_roofline", "epilogue_roofline", "mlp_roofline"):
                with_achievable(staged[k], ceilings)
    single = None if args.no_single else single_query(args, S, hwr, torch)
    single_graph = None if args.no_single else single_query(args, S, hwr, torch, hwr.HWR_FLAG_GRAPH)
    if single_graph:
        single_graph["runtime_env"] = f"{GRAPH_ENV[0]}={os.environ.get(GRAPH_ENV[0])}"
    single_res = None if args.no_single else single_query(args, S, hwr, torch, hwr.HWR_FLAG_RESIDENT)
    floor = None
    if not args.no_single:
        # what a launch answered through pinned host memory costs with no work
        # in it: the floor under the plain and the graph-launched single query
        fp, fg = hwr.hwr_probe_launch_floor(0, False, 2000), hwr.hwr_probe_launch_floor(0, True, 2000)
        floor = {"plain_launch": {"p50_us": fp[0], "p99_us": fp[1]},
                 "graph_launch": {"p50_us": fg[0], "p99_us": fg[1]},
                 "probe": "hwr_probe_launch_floor: one wave echoes a pinned request number, 2000 calls",
                 "runtime_env": f"{GRAPH_ENV[0]}={os.environ.get(GRAPH_ENV[0])}"}
        log(f"launch floor: plain p50 {fp[0]:.1f} us, graph p50 {fg[0]:.1f} us")
    if single:
        log(f"single query (kernel launch) p50 {single['p50_us']:.1f} us p99 {single['p99_us']:.1f} us; "
            f"(graph launch) p50 {single_graph['p50_us']:.1f} us p99 {single_graph['p99_us']:.1f} us; "
            f"(resident) p50 {single_res['p50_us']:.1f} us p99 {single_res['p99_us']:.1f} us")
    batch = batch_latency(args, S, hwr, torch) if args.batch_calls > 0 else None
    hostb = host_batches(args, hwr, torch, w) if args.host_chunks > 0 else None
    sim = None if args.no_sim else closed_loop(args, hwr, torch)
    pareto = None if args.no_sim or not args.pareto_weights else closed_loop_pareto(args, hwr, torch)
    cpu = None if args.no_cpu_baseline else cpu_baseline(w["pb"], w["st"], w["sample"], w["sp"], w["sample_wide"])
    line = {
        "metric": METRIC, "value": res["value"], "unit": "candidates/s", "n_gpus": 1,
        "steps": args.steps, "warmup": args.warmup, "ms_per_step": res["ms_per_step"],
        "higher_is_better": True, "scaling": "weak", "vs_baseline": None, "dtype": "bf16",
        "data": "synthetic (seeded; stands in for the paper's embedded prompt sets)",
        "config": res["config"], "roofline": res["roofline"], "cpu_baseline": cpu,
        "single_query": single, "single_query_graph_launch": single_graph,
        "single_query_resident": single_res, "single_query_launch_floor": floor,
        "step_ms": res["step_ms"], "quality_roofline": res["quality_roofline"], "stages": res["stages"],
        "staged_pipeline": staged, "ceilings": ceilings, "batch_latency": batch, "host_batches": hostb,
        "closed_loop": sim, "closed_loop_pareto": pareto,
    }
    print(json.dumps(line), flush=True)
    return 0


if __name__ == "__main__":
    sys.exit(main())
