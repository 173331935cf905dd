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


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
def test_c3_full_size_per_candidate(pipeline):
    """65,536 queries x 64 pairs in one chunk (fused: 256 workgroups, the
    unsplit launch; staged: gather, four-tile predictor and epilogue at full
    size): every prediction and quality of every 16th query compared with the
    oracle, and every choice of the sample under the acceptance rule."""
    import torch
    sp = S.spec("C3")
    pb, st, qs = S.make_problem(sp, 1), S.make_state(sp, 1), S.make_queries(sp, 1)
    r = G.make_router(pb, pipeline=pipeline)
    r.update(st)
    emb, il, no, slo = G.to_dev_inputs(qs, sp.dtype)
    out = G.dev_outputs(qs.n, r.N, r.M, True)
    r.route(emb, il, no, slo, mem=hwr.HWR_MEM_DEVICE, **out)
    lean = G.dev_outputs(qs.n, r.N, r.M, False)
    r.route(emb, il, no, slo, mem=hwr.HWR_MEM_DEVICE, **lean)
    torch.cuda.synchronize()
    for k, v in lean.items():     # the form without per-candidate outputs decides identically
        assert torch.equal(v, out[k]), k
    idx = np.arange(0, qs.n, 16)
    sub = {k: v[torch.from_numpy(idx).to(v.device)].cpu().numpy() for k, v in out.items()}
    q = qs.take(idx)
    rep = G.check_against(pb, q, sub, G.oracle_threaded(pb, st, q), query_ids=idx)
    _report(f"C3 full {pipeline}, every 16th query ({idx.size} x {r.N} candidates)", rep)
    assert rep.max_rel_ttft < 2e-3 and rep.max_rel_tpot < 2e-3


def _c5_inputs(sp, seed, dev):
    import torch
    n = sp.total_queries
    emb = torch.empty((n, sp.embed_dim), dtype=torch.int16, device=dev)
    il = torch.empty(n, dtype=torch.int32, device=dev)
    no = torch.empty(n, dtype=torch.int32, device=dev)
    slo = torch.empty(n, dtype=torch.float32, device=dev)
    chunks = []
    for c in range(sp.n_chunks):
        qs = S.make_queries(sp, seed, chunk=c)
        a, b = c * sp.n_queries, (c + 1) * sp.n_queries
        emb[a:b] = torch.from_numpy(qs.emb_bits.view(np.int16)).to(dev)
        il[a:b] = torch.from_numpy(qs.input_len).to(dev)
        no[a:b] = torch.from_numpy(qs.expected_out_len).to(dev)
        slo[a:b] = torch.from_numpy(qs.slo_s).to(dev)
        chunks.append(qs)
    return emb, il, no, slo, chunks


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
def test_c5_full_size_per_candidate(pipeline):
    """1,048,576 queries x 256 pairs in 65,536-query chunks -- the launch
    configuration the benchmark times (fused: one unsplit launch per chunk;
    staged: the staged pipeline's line of the benchmark).  The batch is
    routed twice: without per-candidate outputs (the benchmark's kernel form)
    and with them; both give identical decisions.  Every 256th query across
    all 16 chunks (4,096 queries x 256 pairs) is compared with the oracle
    candidate by candidate, and its choice under the acceptance rule."""
    import torch
    sp = S.spec("C5")
    pb, st = S.make_problem(sp, 5), S.make_state(sp, 5)
    r = G.make_router(pb, max_chunk=sp.n_queries, pipeline=pipeline)
    r.update(st)
    dev = torch.device("cuda")
    emb, il, no, slo, chunks = _c5_inputs(sp, 5, dev)
    n = sp.total_queries
    lean = G.dev_outputs(n, r.N, r.M, False)
    r.route(emb, il, no, slo, mem=hwr.HWR_MEM_DEVICE, **lean)
    out = G.dev_outputs(n, r.N, r.M, True)
    r.route(emb, il, no, slo, mem=hwr.HWR_MEM_DEVICE, **out)
    torch.cuda.synchronize()
    for k, v in lean.items():
        assert torch.equal(v, out[k]), k
    choice = lean["choice"].cpu().numpy()
    assert (choice >= 0).all() and (choice < r.N).all()
    idx = np.arange(0, n, 256)
    sub = {k: v[torch.from_numpy(idx).to(dev)].cpu().numpy() for k, v in out.items()}
    del out, lean
    torch.cuda.empty_cache()
    per = sp.n_queries
    qsub = S.Queries(*(np.concatenate([getattr(chunks[c].take(idx[idx // per == c] - c * per), f)
                                       for c in range(sp.n_chunks)])
                       for f in ("emb", "emb_bits", "input_len", "expected_out_len", "slo_s")))
    rep = G.check_against(pb, qsub, sub, G.oracle_threaded(pb, st, qsub), query_ids=idx)
    _report(f"C5 full {pipeline}, every 256th query ({idx.size} x {r.N} candidates)", rep)
    assert rep.max_rel_ttft < 2e-3 and rep.max_rel_tpot < 2e-3


@pytest.fixture(scope="module")
def c4_walk():
    """The C4 workload: 10,000 sequential queries, the runtime signals taking
    one random-walk step before each; the oracle's result for every step."""
    sp = S.spec("C4")
    pb = S.make_problem(sp, 4)
    walk = S.StateWalk(sp, 4)
    steps = 10000
    qs = S.make_queries(sp, 4, n=steps)
    states = [walk.step() for _ in range(steps)]
    from concurrent.futures import ThreadPoolExecutor
    from oracle import oracle as O
    O.lib()
    with ThreadPoolExecutor(max_workers=16) as ex:
        parts = list(ex.map(lambda i: O.route_synth(pb, states[i], qs.slice(i, i + 1)), range(steps)))
    return sp, pb, qs, states, G.stack_results(parts)


@pytest.mark.parametrize("flags", [0, hwr.HWR_FLAG_GRAPH, hwr.HWR_FLAG_RESIDENT])
def test_c4_single_query_walk(c4_walk, flags):
    """All 10,000 sequential single-query calls of the C4 workload with a
    state update before each, in each launch mode (kernel launch, captured
    graph, resident kernel), against the oracle under the acceptance rule."""
    sp, pb, qs, states, orc = c4_walk
    r = G.make_router(pb, flags=flags)
    keys = ("choice", "feasible", "utility", "e2e_s", "ttft_s", "tpot_s")
    got = {k: np.zeros(qs.n, np.uint8 if k == "feasible" else (np.int32 if k == "choice" else np.float32))
           for k in keys}
    for i in range(qs.n):
        r.update(states[i])
        o = r.route_host(qs.emb_bits[i:i + 1], qs.input_len[i:i + 1], qs.expected_out_len[i:i + 1],
                         qs.slo_s[i:i + 1])
        for k in keys:
            got[k][i] = o[k][0]
    r.close()
    rep = G.check_against(pb, qs, got, orc)
    _report(f"C4 single-query walk, {qs.n} steps, flags={flags}", rep)
    assert rep.eligible > qs.n // 2


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



@pytest.mark.parametrize("kw,pipeline", [
    (dict(), "fused"),                                           # H = 128, lean and non-lean
    (dict(n_heads=3), "staged"),                                 # H = 128, three heads
    (dict(hidden=256), "staged"),                                # H = 256 staged
    (dict(hidden=256, n_heads=3), "fused"),                      # H = 256, three heads
    (dict(score_mode=1, cost_weight=0.3, **S.PAPER_SLO), "fused"),   # H = 128, the paper's rules
])
def test_four_tile_form_equals_two_tile_form(kw, pipeline):
    """A chunk that gives every compute unit a workgroup (256 queries each)
    takes the four-column-tile, one-wave-per-SIMD predictor at H = 128 and
    256; half that chunk takes the two-tile form (the pair range split over
    workgroups).  Both give the same bits -- decisions, per-candidate
    predictions, the Q matrix -- and the four-tile form's decisions are the
    same with and without per-candidate outputs (its lean and full
    instantiations).  Every 64th query is also checked against the oracle
    (Sec. 3.2 Eq. 1-3)."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 256 * cus
    sp = S.spec("C2", n_queries=n, **kw)
    pb, st, qs = S.make_problem(sp, 17), S.make_state(sp, 17), S.make_queries(sp, 17)
    four = G.make_router(pb, pipeline=pipeline, max_chunk=n)
    two = G.make_router(pb, pipeline=pipeline, max_chunk=n // 2)
    for r in (four, two):
        r.update(st)
    a = G.route_device(four, qs, "bf16")
    b = G.route_device(two, qs, "bf16")
    lean = G.route_device(four, qs, "bf16", candidates=False)
    for k in a:
        assert np.array_equal(a[k].view(np.uint8), b[k].view(np.uint8)), k
    for k in lean:
        assert np.array_equal(a[k].view(np.uint8), lean[k].view(np.uint8)), k
    idx = np.arange(0, n, 64)
    rep = G.check(pb, st, qs.take(idx), {k: v[idx] for k, v in a.items()}, query_ids=idx)
    _report(f"four-tile form {kw} {pipeline}, every 64th of {n} queries", rep)
