"""Reference closed-loop serving simulation.  TEST INFRASTRUCTURE ONLY.

A plain, slow Python statement of the simulation that include/hwr_sim.h
defines, written from that definition (not from the library's C++), used to
check hwr_sim_run step for step.  The router is a callable handed the cached
monitor snapshot; the tests pass the CPU routing oracle (oracle.route) or a
replay of the choices a GPU run made.

What it follows (paper): the monitor polls the runtime signals of every pair
every 200-300 ms and the router reads that cache (Sec. 3.2, item 1); the
metrics are Sec. 5's: SLO attainment, queue composition (running vs waiting)
and load / running / waiting skew, the paper's |Qbar_0 - Qbar_1| taken as
max - min over GPUs.  Everything that steers the trajectory is integer
arithmetic; floats are single IEEE operations on exact integers, or sums in
request / pair order, so the library must agree bit for bit.
"""
from __future__ import annotations

import math
from collections import deque

import numpy as np

STATE_FIELDS = ("running_q", "waiting_q", "kv_util", "gpu_util", "ttft_avg_s", "tpot_avg_s")
STATE_DTYPE = np.dtype([("running_q", "<i4"), ("waiting_q", "<i4"), ("kv_util", "<f4"),
                        ("gpu_util", "<f4"), ("ttft_avg_s", "<f4"), ("tpot_avg_s", "<f4")])


def _pct(sorted_vals, q):
    if not sorted_vals:
        return 0.0
    return sorted_vals[int(math.floor(q * (len(sorted_vals) - 1)))]


def simulate(pairs, n_gpus, tick_us, monitor_period_us, max_time_us, prior_ttft_s, prior_tpot_s,
             arrival_us, input_len, output_len, slo_us, router, freeze_state=False):
    """Run the simulation.  ``pairs``: records with gpu, max_running,
    kv_capacity, prefill_base_us, prefill_per_token_ns, tpot_base_us,
    tpot_per_running_us.  ``router(snapshot, r0, r1)`` returns (choice,
    utility, e2e) for requests r0..r1-1.  Returns per-request arrays, the
    snapshots and the metrics (the names of hwr_sim_result)."""
    N, G, R = len(pairs), int(n_gpus), len(arrival_us)
    arr = [int(x) for x in arrival_us]
    pin = [int(x) for x in input_len]
    pout = [int(x) for x in output_len]
    slo = [int(x) for x in slo_us]
    gpu = [int(p["gpu"]) for p in pairs]
    slots = [int(p["max_running"]) for p in pairs]
    cap = [int(p["kv_capacity"]) for p in pairs]
    pf0 = [int(p["prefill_base_us"]) for p in pairs]
    pfn = [int(p["prefill_per_token_ns"]) for p in pairs]
    tp0 = [int(p["tpot_base_us"]) for p in pairs]
    tpr = [int(p["tpot_per_running_us"]) for p in pairs]

    waiting = [deque() for _ in range(N)]
    running = [[] for _ in range(N)]     # each: [r, delay, prefill_left, first_done, acc, tokens_left]
    kv_used = [0] * N
    ttft_sum, ttft_n = [0] * N, [0] * N
    tpot_sum, tpot_n = [0.0] * N, [0] * N
    ttft_avg = [float(np.float32(x)) for x in prior_ttft_s]
    tpot_avg = [float(np.float32(x)) for x in prior_tpot_s]
    busy = [0] * G
    window = 0
    pair = [-1] * R
    util = [0.0] * R
    pe2e = [0.0] * R
    first = [-1] * R
    finish = [-1] * R
    samples = []
    cache = None
    route_calls = 0

    T, nxt, live = 0, 0, 0
    while T < max_time_us:
        if T % monitor_period_us == 0:
            snap = np.zeros(N, STATE_DTYPE)
            for d in range(N):
                if ttft_n[d] > 0:
                    ttft_avg[d] = float(np.float32(ttft_sum[d] / ttft_n[d] / 1e6))
                if tpot_n[d] > 0:
                    tpot_avg[d] = float(np.float32(tpot_sum[d] / tpot_n[d]))
                snap[d]["running_q"] = len(running[d])
                snap[d]["waiting_q"] = len(waiting[d])
                snap[d]["kv_util"] = np.float32(min(kv_used[d] / cap[d], 1.0))
                snap[d]["gpu_util"] = np.float32(busy[gpu[d]] / window) if window > 0 else np.float32(0.0)
                snap[d]["ttft_avg_s"] = np.float32(ttft_avg[d])
                snap[d]["tpot_avg_s"] = np.float32(tpot_avg[d])
                ttft_sum[d] = ttft_n[d] = 0
                tpot_sum[d], tpot_n[d] = 0.0, 0
            samples.append(snap)
            if not freeze_state or cache is None:
                cache = snap.copy()
            busy = [0] * G
            window = 0
        # arrivals of [T, T + tick) are routed together, then queue FIFO
        r0 = nxt
        while nxt < R and arr[nxt] < T + tick_us:
            nxt += 1
        if nxt > r0:
            ch, u, c = router(cache.copy(), r0, nxt)
            route_calls += 1
            for i, r in enumerate(range(r0, nxt)):
                pair[r] = int(ch[i])
                util[r] = float(np.float32(u[i]))
                pe2e[r] = float(np.float32(c[i]))
                assert 0 <= pair[r] < N
                waiting[pair[r]].append(r)
            live += nxt - r0
        # admission
        for d in range(N):
            while waiting[d] and len(running[d]) < slots[d]:
                r = waiting[d][0]
                need = pin[r] + pout[r]
                if kv_used[d] + need > cap[d] and running[d]:
                    break
                waiting[d].popleft()
                kv_used[d] += need
                delay = arr[r] - T if arr[r] > T else 0
                running[d].append([r, delay, pf0[d] + pin[r] * pfn[d] // 1000, False, 0, pout[r] - 1])
        on_gpu = [0] * G
        for d in range(N):
            on_gpu[gpu[d]] += len(running[d])
        # service
        for d in range(N):
            if not running[d]:
                continue
            tpot = tp0[d] + tpr[d] * (on_gpu[gpu[d]] - 1)
            for a in running[d]:
                r = a[0]
                avail = tick_us - a[1]
                a[1] = 0
                if not a[3]:
                    used = min(avail, a[2])
                    a[2] -= used
                    avail -= used
                    if a[2] > 0:
                        continue
                    a[3] = True
                    first[r] = T + (tick_us - avail)
                    ttft_sum[d] += first[r] - arr[r]
                    ttft_n[d] += 1
                end = -1
                if a[5] == 0:
                    end = first[r]
                else:
                    a[4] += avail
                    k = min(a[4] // tpot, a[5])
                    a[4] -= k * tpot
                    a[5] -= k
                    if a[5] == 0:
                        end = T + tick_us - a[4]
                if end >= 0:
                    finish[r] = end
                    if pout[r] > 1:
                        tpot_sum[d] += (end - first[r]) / 1e6 / (pout[r] - 1)
                        tpot_n[d] += 1
            keep = []
            for a in running[d]:
                if finish[a[0]] >= 0:
                    kv_used[d] -= pin[a[0]] + pout[a[0]]
                    live -= 1
                else:
                    keep.append(a)
            running[d] = keep
        window += 1
        for g in range(G):
            if on_gpu[g] > 0:
                busy[g] += 1
        T += tick_us
        if nxt == R and live == 0:
            break

    # metrics (Sec. 5)
    lat = sorted(finish[r] - arr[r] for r in range(R) if finish[r] >= 0)
    met = sum(1 for r in range(R) if finish[r] >= 0 and finish[r] - arr[r] <= slo[r])
    ft = [first[r] - arr[r] for r in range(R) if first[r] >= 0]
    S = len(samples) if samples else 1
    run_g, wait_g = [0] * G, [0] * G
    sum_run = sum_wait = 0
    for snap in samples:
        for d in range(N):
            run_g[gpu[d]] += int(snap[d]["running_q"])
            wait_g[gpu[d]] += int(snap[d]["waiting_q"])
            sum_run += int(snap[d]["running_q"])
            sum_wait += int(snap[d]["waiting_q"])
    qb = [(run_g[g] + wait_g[g]) / S for g in range(G)]
    rb = [run_g[g] / S for g in range(G)]
    wb = [wait_g[g] / S for g in range(G)]
    usum, routed = 0.0, 0
    for r in range(R):
        if pair[r] >= 0:
            usum += util[r]
            routed += 1
    qsum = 0.0
    for v in qb:
        qsum += v
    m = dict(
        n_samples=len(samples), end_us=T, n_completed=len(lat), n_met_slo=met, route_calls=route_calls,
        slo_attainment=met / R if R else 0.0,
        mean_latency_s=(sum(lat) / len(lat) / 1e6) if lat else 0.0,
        p50_latency_s=_pct(lat, 0.5) / 1e6 if lat else 0.0,
        p99_latency_s=_pct(lat, 0.99) / 1e6 if lat else 0.0,
        mean_ttft_s=(sum(ft) / len(ft) / 1e6) if ft else 0.0,
        mean_running=sum_run / S, mean_waiting=sum_wait / S,
        running_fraction=sum_run / (sum_run + sum_wait) if sum_run + sum_wait else 0.0,
        avg_load=qsum / G, load_skew=max(qb) - min(qb), running_skew=max(rb) - min(rb),
        waiting_skew=max(wb) - min(wb), mean_utility=usum / routed if routed else 0.0)
    m.update(pair=np.array(pair, np.int32), utility=np.array(util, np.float32),
             pred_e2e_s=np.array(pe2e, np.float32), first_token_us=np.array(first, np.int64),
             finish_us=np.array(finish, np.int64),
             samples=np.stack(samples) if samples else np.zeros((0, N), STATE_DTYPE))
    return m
