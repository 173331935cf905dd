"""Hidden-layer biases on the GPU.  The generator's predictors have b1 = b2 = 0
(the weights are drawn, not trained), so these cases draw non-zero biases
and check the HIP path against the oracle.  The bf16 predictor carries b1
inside its first MFMA layer when three feature slots past the signals are
free and b1 splits exactly into three bf16 parts; the other cases (a wide
one-hot layout, a bias too small to split exactly) keep b1 as the
accumulator start.  Both paths are covered, fused, staged and single query."""
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


CASES = {
    # name: (spec, folds)
    "C2": (S.spec("C2", n_queries=1500), True),
    "C3": (S.spec("C3", n_queries=700), True),
    "wide one-hot": (S.custom_spec("wide", n_queries=600, n_models=3, n_gpu_types=2, gpu_width=18,
                                   feat_dim=32, hidden=128, embed_dim=128, dtype="bf16"), False),
    "tiny bias": (S.spec("C2", n_queries=600), False),
}


def biased_problem(name, seed=41):
    sp, _ = CASES[name]
    pb = S.make_problem(sp, seed)
    rng = np.random.default_rng(seed)
    H = sp.hidden
    pb.b1 = rng.normal(0.0, 0.3, H).astype(np.float32)
    pb.b2 = rng.normal(0.0, 0.3, H).astype(np.float32)
    if name == "tiny bias":
        pb.b1[3] = np.float32(1e-40)         # subnormal: no exact three-part bf16 split
    return sp, pb


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
@pytest.mark.parametrize("name", sorted(CASES))
def test_biases_match_the_oracle(name, pipeline):
    sp, pb = biased_problem(name)
    st, qs = S.make_state(sp, 41), S.make_queries(sp, 41)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    got = G.route_device(r, qs, sp.dtype)
    r.close()
    rep = G.check(pb, st, qs, got)
    print(f"{name} {pipeline}: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]


@pytest.mark.parametrize("name", sorted(CASES))
def test_biases_single_query(name):
    sp, pb = biased_problem(name)
    st, qs = S.make_state(sp, 42), S.make_queries(sp, 42, n=6)
    r = G.make_router(pb)
    r.update(st)
    for i in range(qs.n):
        one = qs.slice(i, i + 1)
        got = r.route_host(one.emb_bits, one.input_len, one.expected_out_len, one.slo_s)
        rep = G.check(pb, st, one, got)
        assert rep.ok, (i, rep.failures[:3])
    r.close()


def test_biases_fp32_path():
    sp = S.spec("C1")
    pb = S.make_problem(sp, 43)
    rng = np.random.default_rng(43)
    pb.b1 = rng.normal(0.0, 0.3, sp.hidden).astype(np.float32)
    pb.b2 = rng.normal(0.0, 0.3, sp.hidden).astype(np.float32)
    st, qs = S.make_state(sp, 43), S.make_queries(sp, 43)
    r = G.make_router(pb)
    r.update(st)
    got = r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s, candidates=True)
    r.close()
    rep = G.check(pb, st, qs, got)
    assert rep.ok, rep.failures[:5]
