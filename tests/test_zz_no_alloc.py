"""hwr_route_batch_static (the entry point that allocates nothing: its work
space is a static device array of the library) against hwr_route_batch on
the same context: identical outputs, bit for bit, on two calls in a row, the
second with fewer queries (and other queries), through the C ABI.  Covers
the fused predictor in its split (small batch) and unsplit (full chunk)
launches, three heads, the staged pipeline in several scratch-sized chunks,
several cost weights, and the fp32 path; no device memory is allocated
during the calls; host batches are refused."""
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


CASES = [
    # (config, overrides, router keywords, first and second batch sizes)
    ("C2", dict(), dict(), 3000, 700),                          # fused, split launches
    ("C3", dict(n_queries=65536), dict(), 65536, 40000),        # fused H = 256, unsplit four-tile launch
    ("C2", dict(n_heads=3), dict(), 1500, 333),                 # three heads
    ("C5", dict(n_queries=5000), dict(pipeline="staged"), 5000, 1234),   # staged: chunks of the scratch
    ("C2", dict(), dict(cost_weights=[0.0, 0.5, 2.0]), 1200, 200),        # several cost weights
    ("C1", dict(n_queries=900), dict(), 900, 64),               # fp32 path
]


def _outputs(r, n, candidates):
    return G.dev_outputs(n, r.N, r.M, candidates, r.n_heads, r.n_weights)


@pytest.mark.parametrize("name,kw,rkw,n1,n2", CASES)
def test_static_entry_matches_route_batch(name, kw, rkw, n1, n2):
    import torch
    sp = S.spec(name, **kw)
    pb, st = S.make_problem(sp, 17), S.make_state(sp, 17)
    r = G.make_router(pb, **rkw)
    r.update(st)
    candidates = name != "C3"
    for call, (n, seed) in enumerate(((n1, 17), (n2, 18))):
        qs = S.make_queries(sp, seed, n=n)
        emb, il, no, slo = G.to_dev_inputs(qs, sp.dtype)
        no_arg = None if sp.n_heads == 3 else no
        ref = _outputs(r, n, candidates)
        r.route(emb, il, no_arg, slo, mem=hwr.HWR_MEM_DEVICE, **ref)
        got = _outputs(r, n, candidates)
        for v in got.values():       # stale values would show up as differences
            v.fill_(7)
        torch.cuda.synchronize()
        free0 = torch.cuda.mem_get_info()[0]
        r.route(emb, il, no_arg, slo, mem=hwr.HWR_MEM_DEVICE, static=True, **got)
        torch.cuda.synchronize()
        if call == 1:                # after a first call of every kernel: nothing is allocated
            assert torch.cuda.mem_get_info()[0] >= free0
        for k in ref:
            a, b = ref[k].cpu().numpy(), got[k].cpu().numpy()
            assert a.tobytes() == b.tobytes(), (name, call, k)
        print(f"[static] {name} {rkw} call {call}: {n} queries identical", flush=True)
    r.close()


def test_static_entry_refuses_host_batches():
    sp = S.spec("C2", n_queries=8)
    pb, st, qs = S.make_problem(sp, 3), S.make_state(sp, 3), S.make_queries(sp, 3)
    r = G.make_router(pb)
    r.update(st)
    out = dict(choice=np.zeros(qs.n, np.int32))
    with pytest.raises(hwr.HwrError) as e:
        r.route(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s, mem=hwr.HWR_MEM_HOST,
                static=True, **out)
    assert e.value.status == hwr.HWR_ERR_INVALID_ARG
    assert "device-memory batches only" in str(e.value)
    r.close()
