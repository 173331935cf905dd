"""The decision step on the GPU is exact: given the GPU's own predictions
(TTFT, TPOT per candidate) and qualities, the oracle's Eq. 2 / Eq. 3 step
reproduces every GPU decision bit for bit: choice, feasibility, utility and
cost, in every pipeline.  Unlike the parity tests there is no tolerance:
the cost, the division C / SLO and the utility are each rounded once in
fp32 on both sides, and ties go to the lower pair index."""
import numpy as np
import pytest

from oracle import oracle as O
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


def _exact(out, pb, qs, alpha):
    sp = pb.spec
    d = O.decide(pb.dep_model, out["cand_ttft"], out["cand_tpot"], out["cand_quality"],
                 qs.expected_out_len, qs.slo_s, alpha, cand_nout=out.get("cand_nout"),
                 input_len=qs.input_len, score_mode=sp.score_mode, bound_mode=sp.bound_mode,
                 ttft_slo_a=sp.ttft_slo_a, ttft_slo_b=sp.ttft_slo_b, tpot_slo=sp.tpot_slo)
    assert np.array_equal(out["choice"], d["choice"])
    assert np.array_equal(out["feasible"], d["feasible"])
    assert np.array_equal(out["utility"].view(np.int32), d["utility"].view(np.int32))
    assert np.array_equal(out["e2e_s"].view(np.int32), d["e2e_s"].view(np.int32))
    # the reported TTFT / TPOT are the chosen candidate's
    rows = np.arange(qs.n)
    assert np.array_equal(out["ttft_s"], out["cand_ttft"][rows, out["choice"]])
    assert np.array_equal(out["tpot_s"], out["cand_tpot"][rows, out["choice"]])
    # and the N_out used for it: predicted (three heads) or the query's own
    want_n = (out["cand_nout"][rows, out["choice"]] if "cand_nout" in out
              else qs.expected_out_len.astype(np.float32))
    assert np.array_equal(out["nout"], want_n)


CASES = {
    "C2": ("C2", dict(n_queries=1000), 2),
    "C3 ragged": ("C3", dict(n_queries=333), 3),
    "C5 shape": ("C5", dict(n_queries=300), 5),
    "15 pairs": ("C2", dict(n_queries=257, n_models=5, n_gpu_types=3), 8),
    "C2 3 heads": ("C2", dict(n_queries=1000, n_heads=3), 2),
    "C3 3 heads": ("C3", dict(n_queries=333, n_heads=3), 3),
    "H=64 15 pairs 3 heads": ("C2", dict(n_queries=200, n_models=5, n_gpu_types=3, hidden=64, n_heads=3), 9),
}


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
@pytest.mark.parametrize("case", sorted(CASES))
def test_device_decisions_are_exact(case, pipeline):
    name, kw, seed = CASES[case]
    sp = S.spec(name, **kw)
    pb, st, qs = S.make_problem(sp, seed), S.make_state(sp, seed), S.make_queries(sp, seed)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    _exact(G.route_device(r, qs, sp.dtype), pb, qs, sp.cost_weight)


@pytest.mark.parametrize("heads", [2, 3])
def test_fp32_host_decisions_are_exact(heads):
    sp = S.spec("C1", n_heads=heads)
    pb, st, qs = S.make_problem(sp, 1), S.make_state(sp, 1), S.make_queries(sp, 1)
    r = G.make_router(pb)
    r.update(st)
    out = r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s, candidates=True)
    _exact(out, pb, qs, sp.cost_weight)


def test_extreme_bounds_take_the_division_fallback():
    """Bounds far outside [2^-20, 2^20] s take the plain IEEE division; the
    decisions stay exact."""
    sp = S.spec("C2", n_queries=200)
    pb, st, qs = S.make_problem(sp, 11), S.make_state(sp, 11), S.make_queries(sp, 11)
    qs.slo_s[::2] = np.float32(1e-30)
    qs.slo_s[1::2] = np.float32(1e30)
    r = G.make_router(pb)
    r.update(st)
    _exact(G.route_device(r, qs, sp.dtype), pb, qs, sp.cost_weight)
