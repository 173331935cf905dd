"""GPU parity: the HIP library (through its C ABI) against the CPU oracle on
seeded workloads of the synthetic configurations, under the acceptance rule
in tests/parity.py (fp32 1e-4, bf16 1e-2 relative)."""
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


def _report(name, rep):
    print(f"[parity] {name}: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:8]


def test_c1_fp32_host_full():
    sp = S.spec("C1")
    pb, st, qs = S.make_problem(sp, 1), S.make_state(sp, 1), S.make_queries(sp, 1)
    r = G.make_router(pb)
    r.update(st)
    out = r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s, candidates=True)
    rep = G.check(pb, st, qs, out)
    _report("C1 fp32 host", rep)
    assert rep.max_rel_ttft < 1e-5 and rep.max_rel_tpot < 1e-5


@pytest.mark.parametrize("hidden,heads,nq,models,D", [
    (64, 2, 1, 4, 384),          # one query: one workgroup, one busy wave of the quality kernel
    (64, 2, 1027, 4, 384),       # 8,216 candidates: waves loop over candidates; ragged workgroups
    (128, 2, 301, 32, 192),      # H = 128 (two units per lane), 32 models, D = 3 x 64
    (128, 3, 523, 6, 448),       # three heads: N_out predicted per candidate
])
def test_fp32_device_shapes(hidden, heads, nq, models, D):
    """fp32 predictor (one wave per candidate) and quality (one wave per
    query) at shapes past C1: H = 128, three heads, 32 models, batches
    larger than one pass of the grid, ragged query counts."""
    sp = S.spec("C1", n_queries=nq, hidden=hidden, n_heads=heads, n_models=models, embed_dim=D)
    pb, st, qs = S.make_problem(sp, 11), S.make_state(sp, 11), S.make_queries(sp, 11)
    r = G.make_router(pb)
    r.update(st)
    out = G.route_device(r, qs, sp.dtype)
    rep = G.check(pb, st, qs, out)
    _report(f"fp32 H={hidden} heads={heads} nq={nq} M={models} D={D}", rep)
    assert rep.max_rel_ttft < 1e-5 and rep.max_rel_tpot < 1e-5


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
def test_c2_bf16_device_full(pipeline):
    sp = S.spec("C2")
    pb, st, qs = S.make_problem(sp, 2), S.make_state(sp, 2), S.make_queries(sp, 2)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    out = G.route_device(r, qs, sp.dtype)
    rep = G.check(pb, st, qs, out)
    _report(f"C2 bf16 {pipeline}", rep)
    # the oracle rounds at the same points, so errors sit far below the bound
    assert rep.max_rel_ttft < 2e-3 and rep.max_rel_tpot < 2e-3


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
def test_hidden_64_bf16(pipeline):
    """H = 64 (two row tiles): the shallowest software pipeline."""
    sp = S.spec("C2", n_queries=700, hidden=64)
    pb, st, qs = S.make_problem(sp, 6), S.make_state(sp, 6), S.make_queries(sp, 6)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    out = G.route_device(r, qs, sp.dtype)
    _report(f"H=64 bf16 {pipeline}", G.check(pb, st, qs, out))


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
def test_c3_shape_ragged_tail(pipeline):
    """H = 256, 64 pairs, 300 queries: two workgroups, the second ragged."""
    sp = S.spec("C3", n_queries=300)
    pb, st, qs = S.make_problem(sp, 3), S.make_state(sp, 3), S.make_queries(sp, 3)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    out = G.route_device(r, qs, sp.dtype)
    _report(f"C3-shape ragged {pipeline}", G.check(pb, st, qs, out))


def test_c3_full_size_sampled():
    sp = S.spec("C3")
    pb, st, qs = S.make_problem(sp, 1), S.make_state(sp, 1), S.make_queries(sp, 1)
    r = G.make_router(pb)
    r.update(st)
    out = G.route_device(r, qs, sp.dtype, candidates=False)
    idx = np.arange(0, qs.n, 256) + (np.arange(qs.n // 256) % 256)
    sub = {k: v[idx] for k, v in out.items()}
    _report("C3 full, sampled", G.check(pb, st, qs.take(idx), sub, query_ids=idx))


def test_c5_full_size_sampled():
    """1,048,576 queries x 256 pairs in 65,536-query chunks, the launch
    configuration the benchmark times; parity on a strided sample."""
    import torch
    sp = S.spec("C5")
    pb, st = S.make_problem(sp, 5), S.make_state(sp, 5)
    r = G.make_router(pb, max_chunk=sp.n_queries)
    r.update(st)
    n = sp.total_queries
    dev = torch.device("cuda")
    emb = torch.empty((n, sp.embed_dim), dtype=torch.int16, device=dev)
    il = torch.empty(n, dtype=torch.int32, device=dev)
    no = torch.empty(n, dtype=torch.int32, device=dev)
    slo = torch.empty(n, dtype=torch.float32, device=dev)
    samples = []
    for c in range(sp.n_chunks):
        qs = S.make_queries(sp, 5, chunk=c)
        a, b = c * sp.n_queries, (c + 1) * sp.n_queries
        emb[a:b] = torch.from_numpy(qs.emb_bits.view(np.int16)).to(dev)
        il[a:b] = torch.from_numpy(qs.input_len).to(dev)
        no[a:b] = torch.from_numpy(qs.expected_out_len).to(dev)
        slo[a:b] = torch.from_numpy(qs.slo_s).to(dev)
        local = np.arange(7 * c % 4096, sp.n_queries, 4096)[:16]
        samples.append((a + local, qs.take(local)))
    out = G.dev_outputs(n, r.N, r.M, False)
    r.route(emb, il, no, slo, mem=hwr.HWR_MEM_DEVICE, **out)
    torch.cuda.synchronize()
    out = {k: v.cpu().numpy() for k, v in out.items()}
    idx = np.concatenate([s[0] for s in samples])
    qsub = S.Queries(*(np.concatenate([getattr(s[1], f) for s in samples])
                       for f in ("emb", "emb_bits", "input_len", "expected_out_len", "slo_s")))
    sub = {k: v[idx] for k, v in out.items()}
    _report("C5 full, sampled", G.check(pb, st, qsub, sub, query_ids=idx))
    assert (out["choice"] >= 0).all() and (out["choice"] < r.N).all()


@pytest.mark.parametrize("flags", [0, hwr.HWR_FLAG_GRAPH])
def test_c4_single_query_walk(flags):
    """Sequential single-query calls with a state update between each."""
    sp = S.spec("C4")
    pb = S.make_problem(sp, 4)
    walk = S.StateWalk(sp, 4)
    r = G.make_router(pb, flags=flags)
    qs_all = S.make_queries(sp, 4, n=200)
    from oracle import oracle as O
    import parity
    exact = elig = 0
    for i in range(200):
        st = walk.step()
        r.update(st)
        qs = qs_all.slice(i, i + 1)
        out = r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s)
        orc = O.route_synth(pb, st, qs)
        rep = parity.compare(out, orc, slo=qs.slo_s, alpha=sp.cost_weight, dep_model=pb.dep_model,
                             rtol=1e-2)
        assert rep.ok, (i, rep.failures)
        elig += rep.eligible
        exact += rep.exact
    print(f"[parity] C4 single-query walk flags={flags}: eligible {elig}/200 exact {exact}", flush=True)
    assert elig > 100


# ---------------------------------------------------------------- three heads
@pytest.mark.parametrize("pipeline", ["fused", "staged"])
@pytest.mark.parametrize("name,kw,seed", [
    ("C2", dict(n_queries=2048), 2),                  # H = 128
    ("C3", dict(n_queries=300), 3),                   # H = 256, ragged tail
    ("C2", dict(n_queries=500, hidden=64), 6),        # H = 64
])
def test_three_heads_predicted_output_length(name, kw, seed, pipeline):
    """Eq. 1 with the third head: N_out predicted per candidate and used in
    Eq. 2; the query's given expected_out_len is not passed at all."""
    sp = S.spec(name, n_heads=3, **kw)
    pb, st, qs = S.make_problem(sp, seed), S.make_state(sp, seed), S.make_queries(sp, seed)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    import torch
    emb, il, _, slo = G.to_dev_inputs(qs, sp.dtype)
    out = G.dev_outputs(qs.n, r.N, r.M, True, 3)
    r.route(emb, il, None, slo, mem=hwr.HWR_MEM_DEVICE, **out)
    torch.cuda.synchronize()
    out = {k: v.cpu().numpy() for k, v in out.items()}
    rep = G.check(pb, st, qs, out)
    _report(f"{name} 3 heads {pipeline}", rep)
    assert rep.max_rel_nout < 2e-3
    rows = np.arange(qs.n)
    assert np.array_equal(out["nout"], out["cand_nout"][rows, out["choice"]])


def test_three_heads_fp32_host():
    sp = S.spec("C1", n_heads=3)
    pb, st, qs = S.make_problem(sp, 1), S.make_state(sp, 1), S.make_queries(sp, 1)
    r = G.make_router(pb)
    r.update(st)
    out = r.route_host(qs.emb_bits, qs.input_len, None, qs.slo_s, candidates=True)
    rep = G.check(pb, st, qs, out)
    _report("C1 3 heads fp32 host", rep)
    assert rep.max_rel_nout < 1e-5


REPLICATES = [
    # (config, overrides, pipeline): each run at seeds 100 + id and 200 + id
    ("C1", dict(), "fused"),
    ("C2", dict(n_queries=1111), "fused"),
    ("C2", dict(n_queries=1111), "staged"),
    ("C3", dict(n_queries=777), "fused"),
    ("C3", dict(n_queries=777), "staged"),
]


@pytest.mark.parametrize("offset", [100, 200])
@pytest.mark.parametrize("name,kw,pipeline", REPLICATES)
def test_replicate_seeds(name, kw, pipeline, offset):
    """Replicate draws of C1-C3 (weights, state and queries all redrawn) at
    seeds 100 + id and 200 + id, ragged query counts, through the device path."""
    seed = offset + int(name[1:])
    sp = S.spec(name, **kw)
    pb, st, qs = S.make_problem(sp, seed), S.make_state(sp, seed), S.make_queries(sp, seed)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    out = G.route_device(r, qs, sp.dtype)
    r.close()
    _report(f"{name} seed {seed} {pipeline}", G.check(pb, st, qs, out))

