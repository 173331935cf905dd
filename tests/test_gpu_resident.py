"""The resident single-query path (HWR_FLAG_RESIDENT): one workgroup stays on
the device between calls and serves each new request record it finds.  Its
decisions equal the plain launch's bit for bit (same arithmetic), and match
the oracle under a state walk.  It leaves after its idle polls and the next
call brings it back; hwr_free stops it; batches on the same context are not
affected."""
import time

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_14575_amd import hwr
from paper_2608_14575_amd import synth as S

import gpu_util as G
import parity

pytestmark = pytest.mark.gpu


@pytest.fixture(scope="module", autouse=True)
def _device():
    import torch
    assert torch.cuda.is_available(), "GPU tests need a device"
    hwr.load()
    yield


def _one(r, qs, i):
    one = qs.slice(i, i + 1)
    return r.route_host(one.emb_bits, one.input_len, one.expected_out_len, one.slo_s)


@pytest.mark.parametrize("name,kw", [
    ("C4", dict()),                                   # H = 128, 32 pairs
    ("C4", dict(n_heads=3)),                          # predicted N_out
    ("C2", dict(hidden=64)),                          # H = 64, 16 pairs
    ("C3", dict()),                                   # H = 256, 64 pairs (2 tiles)
])
def test_resident_equals_plain_and_matches_oracle(name, kw):
    sp = S.spec(name, n_queries=60, **kw)
    pb = S.make_problem(sp, 23)
    qs = S.make_queries(sp, 23)
    res = G.make_router(pb, flags=hwr.HWR_FLAG_RESIDENT)
    plain = G.make_router(pb)
    walk = S.StateWalk(sp, 23)
    got, ref, states = [], [], []
    for i in range(qs.n):
        st = walk.step()
        states.append(st)
        res.update(st)
        plain.update(st)
        got.append(_one(res, qs, i))
        ref.append(_one(plain, qs, i))
    res.close()
    plain.close()
    for a, b in zip(got, ref):
        for k in a:
            assert np.array_equal(a[k], b[k]), k
    ok = 0
    for i in range(qs.n):
        one = qs.slice(i, i + 1)
        rep = parity.compare(got[i], O.route_synth(pb, states[i], one), slo=one.slo_s, alpha=sp.cost_weight,
                             dep_model=pb.dep_model, rtol=1e-2, heads=sp.n_heads)
        assert rep.ok, (i, rep.failures[:3])
        ok += 1
    print(f"[parity] resident {name} {kw}: {ok}/{qs.n} queries match the oracle", flush=True)


def test_resident_leaves_when_idle_and_comes_back():
    sp = S.spec("C4", n_queries=6)
    pb, st, qs = S.make_problem(sp, 24), S.make_state(sp, 24), S.make_queries(sp, 24)
    res = G.make_router(pb, flags=hwr.HWR_FLAG_RESIDENT)
    plain = G.make_router(pb)
    res.update(st)
    plain.update(st)
    for i in range(qs.n):
        a = _one(res, qs, i)
        b = _one(plain, qs, i)
        for k in a:
            assert np.array_equal(a[k], b[k]), (i, k)
        time.sleep(0.25 if i % 2 == 0 else 0.0)      # longer than the kernel's idle polls
    res.close()
    plain.close()


def test_free_stops_the_resident_kernel():
    sp = S.spec("C4", n_queries=2)
    pb, st, qs = S.make_problem(sp, 25), S.make_state(sp, 25), S.make_queries(sp, 25)
    for _ in range(3):
        res = G.make_router(pb, flags=hwr.HWR_FLAG_RESIDENT)
        res.update(st)
        _one(res, qs, 0)
        t0 = time.perf_counter()
        res.close()
        assert time.perf_counter() - t0 < 1.0


def test_batches_beside_the_resident_kernel():
    sp = S.spec("C2", n_queries=500)
    pb, st, qs = S.make_problem(sp, 26), S.make_state(sp, 26), S.make_queries(sp, 26)
    res = G.make_router(pb, flags=hwr.HWR_FLAG_RESIDENT)
    plain = G.make_router(pb)
    res.update(st)
    plain.update(st)
    want = G.route_device(plain, qs, "bf16")
    for i in range(3):
        a = _one(res, qs, i)
        got = G.route_device(res, qs, "bf16")
        for k in want:
            assert np.array_equal(want[k], got[k]), k
        assert a["choice"][0] == _one(plain, qs, i)["choice"][0]
    res.close()
    plain.close()


def test_unknown_flags_are_rejected():
    sp = S.spec("C4", n_queries=1)
    pb = S.make_problem(sp, 27)
    with pytest.raises(hwr.HwrError) as e:
        G.make_router(pb, flags=4)
    assert e.value.status == hwr.HWR_ERR_INVALID_ARG
