"""Kernel timing of the library (hwr_profile_enable / hwr_profile_read): every
kernel launch is counted, with a positive duration, the durations fit inside
the wall time, and timing changes no result (a timed launch goes through the
dispatch that records its events, an untimed one through a plain launch)."""
import time

import numpy as np
import pytest

from paper_2608_14575_amd import hwr
from paper_2608_14575_amd import synth as S

import gpu_util as G

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    hwr.load()
    yield


def _case(seed=21, n=3000):
    sp = S.spec("C2", n_queries=n)
    return S.make_problem(sp, seed), S.make_state(sp, seed), S.make_queries(sp, seed)


@pytest.mark.parametrize("pipeline,kinds", [("fused", ("quality", "fused")),
                                            ("staged", ("quality", "gather", "mlp", "epilogue"))])
def test_every_launch_is_timed_and_results_do_not_change(pipeline, kinds):
    import torch
    pb, st, qs = _case()
    r = G.make_router(pb, pipeline=pipeline, max_chunk=1024)      # 3 chunks
    r.update(st)
    ref = G.route_device(r, qs, "bf16")
    r.profile(True)
    r.profile_read(reset=True)
    torch.cuda.synchronize()
    t0 = time.perf_counter()
    got = G.route_device(r, qs, "bf16")
    wall_ms = (time.perf_counter() - t0) * 1e3
    kt = r.profile_read(reset=True)
    r.profile(False)
    again = G.route_device(r, qs, "bf16")
    r.close()
    for k in ref:
        assert np.array_equal(ref[k], got[k]), k
        assert np.array_equal(ref[k], again[k]), k
    total = 0.0
    for k in kinds:
        ms, n = kt[k]
        assert n == 3, (k, n)
        assert ms > 0.0, k
        total += ms
    assert total <= wall_ms, (total, wall_ms)
    # small chunks may split the pairs over several workgroups and merge them
    extra = {"state", "merge"} if pipeline == "fused" else {"state"}
    assert sum(n for k, (_, n) in kt.items() if k not in kinds and k not in extra) == 0
    assert kt["merge"][1] in (0, 3) and kt["state"][1] <= 1


def test_sampled_timing_counts_one_launch_in_k():
    """hwr_profile_enable(ctx, k > 1) times the first launch of each kind and
    every k-th after it; results are unchanged, and k < 0 is refused."""
    import torch
    pb, st, qs = _case()
    r = G.make_router(pb, max_chunk=1024)         # 3 chunks: launches 0, 1, 2 of each kind
    r.update(st)
    ref = G.route_device(r, qs, "bf16")
    r.profile(2)
    r.profile_read(reset=True)
    got = G.route_device(r, qs, "bf16")
    kt = r.profile_read(reset=True)
    for k in ("quality", "fused"):
        assert kt[k][1] == 2 and kt[k][0] > 0.0, (k, kt[k])
    r.profile(5)
    got5 = G.route_device(r, qs, "bf16")
    kt5 = r.profile_read(reset=True)
    assert kt5["fused"][1] == 1 and kt5["quality"][1] == 1
    with pytest.raises(hwr.HwrError) as e:
        r.profile(-1)
    assert e.value.status == hwr.HWR_ERR_INVALID_ARG
    r.profile(False)
    r.close()
    torch.cuda.synchronize()
    for k in ref:
        assert np.array_equal(ref[k], got[k]), k
        assert np.array_equal(ref[k], got5[k]), k


@pytest.mark.parametrize("flags", [0, hwr.HWR_FLAG_GRAPH])
def test_single_query_launches_are_timed(flags):
    pb, st, qs = _case(n=8)
    r = G.make_router(pb, flags=flags)
    r.update(st)
    plain = [r.route_host(qs.emb_bits[i:i + 1], qs.input_len[i:i + 1], qs.expected_out_len[i:i + 1],
                          qs.slo_s[i:i + 1]) for i in range(4)]
    r.profile(True)
    r.profile_read(reset=True)
    timed = [r.route_host(qs.emb_bits[i:i + 1], qs.input_len[i:i + 1], qs.expected_out_len[i:i + 1],
                          qs.slo_s[i:i + 1]) for i in range(4)]
    kt = r.profile_read(reset=True)
    r.close()
    ms, n = kt["single"]
    assert n == 4 and ms > 0.0
    for a, b in zip(plain, timed):
        for k in a:
            assert np.array_equal(a[k], b[k]), k
