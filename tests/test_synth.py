"""The seeded input generator: ranges, determinism, chunk independence, and
the workload statistics the calibrated output bias is meant to give."""
import math

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_14575_amd import synth as S


@pytest.mark.parametrize("name", ["C1", "C2", "C3", "C4", "C5"])
def test_ranges_and_shapes(name):
    sp = S.spec(name)
    pb = S.make_problem(sp, 1)
    st = S.make_state(sp, 1)
    n = min(sp.n_queries, 2048)
    qs = S.make_queries(sp, 1, n=n)
    N = sp.n_deployments
    assert pb.dep_model.shape == (N,) and pb.dep_gpu.shape == (N,)
    assert np.array_equal(pb.dep_model * sp.n_gpu_types + pb.dep_gpu, np.arange(N))
    assert set(pb.model_params_b.tolist()) <= set(S.PARAMS_SET_B)
    assert pb.wq.shape == (sp.embed_dim, sp.n_models)
    assert pb.w1.shape == (sp.feat_dim, sp.hidden) and pb.w2.shape == (sp.hidden, sp.hidden)
    assert (st["running_q"] >= 0).all() and (st["waiting_q"] >= 0).all()
    assert ((st["kv_util"] >= 0) & (st["kv_util"] <= 1)).all()
    assert (st["ttft_avg_s"] > 0).all() and (st["tpot_avg_s"] > 0).all()
    assert (qs.input_len >= sp.len_lo).all() and (qs.input_len <= sp.len_hi).all()
    assert (qs.expected_out_len >= 64).all() and (qs.expected_out_len <= 512).all()
    assert (qs.slo_s > 0).all()
    norms = np.linalg.norm(qs.emb.astype(np.float64), axis=1)
    tol = 1e-5 if sp.dtype == "f32" else 2e-2
    np.testing.assert_allclose(norms, 1.0, atol=tol)
    if sp.dtype == "bf16":
        assert qs.emb_bits.dtype == np.uint16
        assert np.array_equal(S.bf16_bits_to_f32(qs.emb_bits), qs.emb)
        assert np.array_equal(S.bf16_bits_to_f32(pb.w2_bits), pb.w2)
    if sp.slo_kind == "choice":
        assert set(np.unique(qs.slo_s).tolist()) <= set(sp.slo_choices)
    if sp.slo_kind == "uniform":
        assert qs.slo_s.min() >= sp.slo_range[0] and qs.slo_s.max() <= sp.slo_range[1]


def test_distribution_moments():
    sp = S.spec("C2")
    st = np.concatenate([S.make_state(sp, s) for s in range(200)])
    assert abs(st["running_q"].mean() - 4.0) < 0.2
    assert abs(st["waiting_q"].mean() - 2.0) < 0.15
    assert abs(np.median(st["ttft_avg_s"]) - 0.2) < 0.02
    assert abs(np.median(st["tpot_avg_s"]) - 0.03) < 0.003
    qs = S.make_queries(sp, 3)
    assert abs(np.median(np.log(qs.input_len)) - 6.0) < 0.1


def test_overload_subset():
    sp = S.spec("C3")
    st = S.make_state(sp, 2)
    over = S.overloaded_pairs(sp, 2)
    assert len(over) == round(0.2 * sp.n_deployments)
    assert (st["kv_util"][over] >= 0.8).all()
    assert st["waiting_q"][over].mean() > 3 * st["waiting_q"][np.setdiff1d(np.arange(64), over)].mean()


def test_determinism_and_chunks():
    sp = S.spec("C5", n_queries=64, embed_dim=128)
    a = S.make_queries(sp, 5, chunk=3)
    b = S.make_queries(sp, 5, chunk=3)
    c = S.make_queries(sp, 5, chunk=4)
    assert np.array_equal(a.emb_bits, b.emb_bits) and np.array_equal(a.slo_s, b.slo_s)
    assert not np.array_equal(a.emb_bits, c.emb_bits)
    p1, p2 = S.make_problem(sp, 5), S.make_problem(sp, 5)
    assert np.array_equal(p1.w2_bits, p2.w2_bits)


def test_bf16_rounding_of_inputs():
    import torch
    x = np.random.default_rng(0).standard_normal(100000).astype(np.float32)
    ours = S.bf16_bits_to_f32(S.f32_to_bf16_bits(x))
    ref = torch.from_numpy(x).to(torch.bfloat16).float().numpy()
    assert np.array_equal(ours, ref)


def test_state_walk():
    sp = S.spec("C4")
    w = S.StateWalk(sp, 4)
    s0 = w.state.copy()
    s1 = w.step()
    assert (np.abs(s1["running_q"] - s0["running_q"]) <= 1).all()
    assert ((s1["kv_util"] >= 0) & (s1["kv_util"] <= 1)).all()
    assert np.array_equal(s1["ttft_avg_s"], s0["ttft_avg_s"])


@pytest.mark.parametrize("name", ["C1", "C2", "C3"])
def test_calibrated_workload_statistics(name):
    """The stored output bias puts the median predicted TTFT / TPOT on the
    targets, and the SLO test is neither vacuous nor saturated."""
    sp = S.spec(name)
    assert S.b3_key(sp, 1) in S._b3_table()
    pb, st = S.make_problem(sp, 1), S.make_state(sp, 1)
    qs = S.make_queries(sp, 1, n=min(sp.n_queries, 128))
    r = O.route_synth(pb, st, qs)
    assert abs(np.median(r.cand_ttft) / S.B3_TARGET_TTFT_S - 1) < 0.1
    assert abs(np.median(r.cand_tpot) / S.B3_TARGET_TPOT_S - 1) < 0.1
    frac = r.cand_feasible.mean()
    print(f"{name}: feasible fraction {frac:.2f}, median C {np.median(r.cand_e2e):.2f} s, "
          f"distinct choices {len(set(r.choice.tolist()))}")
    assert 0.2 < frac < 0.95
    assert len(set(r.choice.tolist())) >= 3
    assert math.isfinite(float(r.utility.sum()))
