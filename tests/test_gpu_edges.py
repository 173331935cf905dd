"""GPU edge cases and invariants of the C ABI: error paths, empty and ragged
batches, chunking and workgroup-split invariance (bit-exact), fused vs
staged, host vs device memory, degenerate decisions, maximum sizes."""
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


def _same(a: dict, b: dict, keys=None):
    for k in keys or a.keys():
        assert np.array_equal(a[k], b[k]), k


def _case(name="C2", seed=9, **kw):
    sp = S.spec(name, **kw)
    return sp, S.make_problem(sp, seed), S.make_state(sp, seed), S.make_queries(sp, seed)


def test_route_before_state_and_bad_state():
    sp, pb, st, qs = _case(n_queries=64)
    r = G.make_router(pb)
    with pytest.raises(hwr.HwrError) as e:
        r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s)
    assert e.value.status == hwr.HWR_ERR_STATE
    r.update(st)
    before = r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s)
    for field, val in (("kv_util", 1.5), ("ttft_avg_s", np.nan), ("waiting_q", -1), ("tpot_avg_s", 0.0)):
        bad = st.copy()
        bad[field][3] = val
        with pytest.raises(hwr.HwrError) as e:
            r.update(bad)
        assert e.value.status == hwr.HWR_ERR_INVALID_ARG
    with pytest.raises(hwr.HwrError):
        r.update(st[:-1])
    after = r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s)
    _same(before, after)


def test_bad_host_queries_rejected():
    sp, pb, st, qs = _case(n_queries=8)
    r = G.make_router(pb)
    r.update(st)
    il = qs.input_len.copy()
    il[2] = 0
    with pytest.raises(hwr.HwrError):
        r.route_host(qs.emb_bits, il, qs.expected_out_len, qs.slo_s)
    slo = qs.slo_s.copy()
    slo[1] = -1.0
    with pytest.raises(hwr.HwrError):
        r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, slo)
    # a device buffer passed as host memory (the C ABI, past the binding's own
    # checks) is rejected before anything reads it
    import ctypes as C
    import torch
    emb_dev = torch.from_numpy(qs.emb_bits.view(np.int16)).to("cuda:0")
    il, no, slo = (np.ascontiguousarray(x) for x in (qs.input_len, qs.expected_out_len, qs.slo_s))
    choice = np.zeros(qs.n, np.int32)
    b = hwr.hwr_query_batch(qs.n, hwr.HWR_MEM_HOST, emb_dev.data_ptr(), il.ctypes.data, no.ctypes.data,
                            slo.ctypes.data)
    res = hwr.hwr_route_result(choice=choice.ctypes.data)
    assert hwr.load().hwr_route_batch(r.ctx, C.byref(b), C.byref(res)) == hwr.HWR_ERR_INVALID_ARG
    assert "device pointer" in hwr.hwr_last_error(r.ctx)


def test_empty_batch_is_noop():
    sp, pb, st, qs = _case(n_queries=4)
    r = G.make_router(pb)
    r.update(st)
    out = r.route_host(qs.emb_bits[:0], qs.input_len[:0], qs.expected_out_len[:0], qs.slo_s[:0])
    assert out["choice"].shape == (0,)


@pytest.mark.parametrize("pipeline", ["fused", "staged"])
@pytest.mark.parametrize("chunk", [100, 101])
def test_chunking_is_invisible(pipeline, chunk):
    """333 queries in one chunk and in chunks of 100 or 101 (pair-major rows
    then padded to 104 queries, the last chunk to 36 or 32)."""
    sp, pb, st, qs = _case(n_queries=333)
    a = G.make_router(pb, pipeline=pipeline)
    b = G.make_router(pb, pipeline=pipeline, max_chunk=chunk)
    a.update(st)
    b.update(st)
    _same(G.route_device(a, qs, "bf16"), G.route_device(b, qs, "bf16"))


@pytest.mark.parametrize("embed_dim", [768, 576])
def test_quality_unroll_is_invisible(embed_dim):
    """The quality GEMM has three forms with one MFMA chain order: small
    grids load four embedding slices ahead (one wave per workgroup); large
    ones stream rows through LDS when D is a multiple of 256 (768), else load
    one slice at a time (576).  A batch routed in one large chunk and in
    small chunks gives bit-identical outputs, Q matrix included."""
    import torch
    cus = torch.cuda.get_device_properties(0).multi_processor_count
    n = 128 * cus + 5                       # one chunk: grid above the CU count
    sp, pb, st, qs = _case(n_queries=n, seed=13, embed_dim=embed_dim)
    big = G.make_router(pb, max_chunk=n)
    small = G.make_router(pb, max_chunk=128 * (cus // 2))
    big.update(st)
    small.update(st)
    _same(G.route_device(big, qs, "bf16"), G.route_device(small, qs, "bf16"))


@pytest.mark.parametrize("kw", [dict(), dict(n_heads=3), dict(n_heads=3, **S.PAPER_SLO, score_mode=1)])
def test_fp32_chunking_is_invisible(kw):
    """fp32 path (quality, predictor, decision epilogue): 1500 queries in one
    chunk, in three chunks of 500 and in 38 chunks of at most 40 give the same
    outputs, candidates and Q matrix included; two and three heads, the
    paper's rules.  Chunks of 40 are small enough for the predictor launch to
    run the quality rows as well (no quality launch of their own)."""
    sp, pb, st, qs = _case("C1", n_queries=1500, seed=14, **kw)
    routers = [G.make_router(pb, max_chunk=m) for m in (1500, 500, 40)]
    for r in routers:
        r.update(st)
    routers[2].profile(True)
    outs = [G.route_device(r, qs, "f32") for r in routers]
    kt = routers[2].profile_read(reset=True)
    for r in routers:
        r.close()
    assert kt["quality"][1] == 0 and kt["mlp"][1] == 38, kt
    _same(outs[0], outs[1])
    _same(outs[0], outs[2])


def test_fused_equals_staged_and_split_equals_unsplit():
    """Same arithmetic per candidate in every mode: bit-identical outputs.
    40 queries over 64 pairs makes the fused kernel split the pairs over
    workgroups and merge their keys."""
    sp, pb, st, qs = _case("C3", n_queries=40, seed=12)
    f = G.make_router(pb, pipeline="fused")
    s = G.make_router(pb, pipeline="staged")
    f.update(st)
    s.update(st)
    of, os_ = G.route_device(f, qs, "bf16"), G.route_device(s, qs, "bf16")
    _same(of, os_)
    rep = G.check(pb, st, qs, of)
    assert rep.ok, rep.failures[:5]


def test_debug_outputs_do_not_change_decisions_and_repeat_exactly():
    sp, pb, st, qs = _case(n_queries=500)
    r = G.make_router(pb)
    r.update(st)
    with_c = G.route_device(r, qs, "bf16", candidates=True)
    without = G.route_device(r, qs, "bf16", candidates=False)
    again = G.route_device(r, qs, "bf16", candidates=False)
    _same(without, {k: with_c[k] for k in without})
    _same(without, again)


def test_host_equals_device():
    sp, pb, st, qs = _case(n_queries=257)
    r = G.make_router(pb)
    r.update(st)
    d = G.route_device(r, qs, "bf16", candidates=True)
    h = r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s, candidates=True)
    _same(d, h)


@pytest.mark.parametrize("name,kw", [
    ("C2", dict(pipeline="fused")),
    ("C2", dict(pipeline="staged")),
    ("C2", dict(pipeline="fused", cost_weights=[0.1, 0.5, 2.0])),
    ("C1", dict()),
])
def test_host_batches_in_several_chunks(name, kw):
    """Host-memory batches stream their chunks through two input sets (the
    next chunk's upload overlaps this chunk's kernels): 333 queries in chunks
    of 100, against the device path in one chunk, bit for bit, candidates
    included; and the same router routes a second, shorter batch."""
    heads = 3 if kw.get("cost_weights") is None and name == "C2" and kw["pipeline"] == "staged" else 2
    sp, pb, st, qs = _case(name, n_queries=333, n_heads=heads)
    one = G.make_router(pb, **kw)
    many = G.make_router(pb, max_chunk=100, **kw)
    one.update(st)
    many.update(st)
    d = G.route_device(one, qs, sp.dtype, candidates=True)
    h = many.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s, candidates=True)
    _same(d, h)
    sub = qs.slice(0, 150)
    h2 = many.route_host(sub.emb_bits, sub.input_len, sub.expected_out_len, sub.slo_s, candidates=True)
    _same({k: v[:150] for k, v in d.items()}, h2)


@pytest.mark.parametrize("pinned", [False, True])
def test_large_host_batches_through_the_pinned_ring(pinned):
    """A pageable host batch of at least 16 MB of embeddings passes through the
    library's pinned ring (filled by its copy threads); a pinned one is
    uploaded directly.  20,000 C3 queries (41 MB) in chunks of 3,000, so the
    ring of four 32 MB slots wraps, against the device path in one chunk, bit
    for bit; then a second batch through the same router."""
    import torch
    sp, pb, st, qs = _case("C3", n_queries=20000)
    one = G.make_router(pb)
    many = G.make_router(pb, max_chunk=3000)
    one.update(st)
    many.update(st)
    d = G.route_device(one, qs, sp.dtype, candidates=False)
    emb = qs.emb_bits
    if pinned:
        emb = torch.from_numpy(np.ascontiguousarray(emb)).pin_memory().numpy()
    assert emb.nbytes >= 16 << 20
    for _ in range(2):
        h = many.route_host(emb, qs.input_len, qs.expected_out_len, qs.slo_s)
        _same(d, h)


def test_default_slo_used_when_absent():
    sp, pb, st, qs = _case(n_queries=64)
    r = G.make_router(pb, default_slo_s=1.5)
    r.update(st)
    a = G.route_device(r, qs, "bf16", with_slo=False)
    qs.slo_s[:] = 1.5
    b = G.route_device(r, qs, "bf16")
    _same(a, b)


def test_all_infeasible_falls_back():
    sp, pb, st, qs = _case(n_queries=128)
    qs.slo_s[:] = 1e-4
    r = G.make_router(pb)
    r.update(st)
    out = G.route_device(r, qs, "bf16")
    assert not out["feasible"].any()
    rep = G.check(pb, st, qs, out)
    assert rep.ok, rep.failures[:5]


def test_duplicate_pairs_go_to_lowest_index():
    sp = S.spec("C2", n_queries=96, n_models=2, n_gpu_types=2)
    pb, st, qs = S.make_problem(sp, 14), S.make_state(sp, 14), S.make_queries(sp, 14)
    pb.dep_model[:] = [0, 0, 1, 1]
    pb.dep_gpu[:] = [0, 0, 1, 1]
    st[1] = st[0]
    st[3] = st[2]
    r = G.make_router(pb)
    r.update(st)
    out = G.route_device(r, qs, "bf16")
    assert set(np.unique(out["choice"]).tolist()) <= {0, 2}
    assert np.array_equal(out["cand_ttft"][:, 0], out["cand_ttft"][:, 1])


def test_single_pair():
    sp, pb, st, qs = _case(n_queries=50, n_models=1, n_gpu_types=1)
    r = G.make_router(pb)
    r.update(st)
    assert (G.route_device(r, qs, "bf16")["choice"] == 0).all()


def test_pair_permutation_maps_choice():
    sp, pb, st, qs = _case(n_queries=200, seed=21)
    r = G.make_router(pb)
    r.update(st)
    base = G.route_device(r, qs, "bf16")
    perm = np.random.default_rng(3).permutation(pb.n_deployments)
    pb2 = S.make_problem(sp, 21)
    pb2.dep_model, pb2.dep_gpu = pb.dep_model[perm].copy(), pb.dep_gpu[perm].copy()
    r2 = G.make_router(pb2)
    r2.update(st[perm].copy())
    out = G.route_device(r2, qs, "bf16")
    # identical per-candidate arithmetic -> identical decisions up to the relabelling
    assert np.array_equal(perm[out["choice"]], base["choice"])


def test_maximum_shape():
    """1024 pairs (32 models x 8 GPU types, each pair listed 4 times with its
    own state), D = 8192, H = 256; ragged query count."""
    sp = S.spec("C5", n_queries=37, embed_dim=8192)
    pb = S.make_problem(sp, 31)
    pb.dep_model = np.tile(pb.dep_model, 4)
    pb.dep_gpu = np.tile(pb.dep_gpu, 4)
    st = np.concatenate([S.make_state(sp, 31 + k) for k in range(4)])
    qs = S.make_queries(sp, 31)
    r = G.make_router(pb)
    r.update(st)
    out = G.route_device(r, qs, "bf16")
    rep = G.check(pb, st, qs, out)
    print(f"[parity] max shape: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]


def test_maximum_shape_fp32():
    """fp32 at its largest: 1024 pairs (32 models x 8 GPU types, listed four
    times with their own states), 32 models, D = 8192, H = 128, three heads;
    ragged query count."""
    sp = S.spec("C1", n_queries=37, n_models=32, n_gpu_types=8, gpu_width=8, embed_dim=8192,
                hidden=128, n_heads=3)
    pb = S.make_problem(sp, 32)
    pb.dep_model = np.tile(pb.dep_model, 4)
    pb.dep_gpu = np.tile(pb.dep_gpu, 4)
    st = np.concatenate([S.make_state(sp, 32 + k) for k in range(4)])
    qs = S.make_queries(sp, 32)
    r = G.make_router(pb)
    r.update(st)
    out = G.route_device(r, qs, "f32")
    rep = G.check(pb, st, qs, out)
    print(f"[parity] fp32 max shape: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]


def test_unsupported_shapes_are_rejected():
    sp = S.spec("C2", n_queries=4, hidden=96)
    pb = S.make_problem(sp, 1)
    with pytest.raises(hwr.HwrError) as e:
        G.make_router(pb)
    assert e.value.status == hwr.HWR_ERR_UNSUPPORTED


def _wide(seed: int, n_queries: int):
    """1024 pairs: the 32 x 8 pair grid listed four times, each copy with its
    own runtime signals (several pair slices per epilogue lane)."""
    sp = S.spec("C5", n_queries=n_queries)
    pb = S.make_problem(sp, seed)
    pb.dep_model = np.tile(pb.dep_model, 4)
    pb.dep_gpu = np.tile(pb.dep_gpu, 4)
    st = np.concatenate([S.make_state(sp, seed + k) for k in range(4)])
    return sp, pb, st, S.make_queries(sp, seed)


@pytest.mark.parametrize("shape", ["15 pairs", "1 pair", "1024 pairs"])
def test_staged_epilogue_shapes(shape):
    """The staged decision epilogue against the fused path (bit-exact) and the
    oracle, for pair counts that take its scalar path (N % 4 != 0), a
    one-lane group, and several 4-pair slices per lane."""
    if shape == "1024 pairs":
        sp, pb, st, qs = _wide(41, 70)
    else:
        kw = dict(n_models=5, n_gpu_types=3) if shape == "15 pairs" else dict(n_models=1, n_gpu_types=1)
        sp, pb, st, qs = _case(n_queries=301, seed=40, **kw)
    f = G.make_router(pb, pipeline="fused")
    s = G.make_router(pb, pipeline="staged")
    f.update(st)
    s.update(st)
    of, os_ = G.route_device(f, qs, "bf16"), G.route_device(s, qs, "bf16")
    _same(of, os_, keys=["choice", "feasible", "utility", "e2e_s", "ttft_s", "tpot_s"])
    rep = G.check(pb, st, qs, os_)
    print(f"[parity] staged {shape}: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]


def test_staged_epilogue_unaligned_candidate_buffers():
    """Caller candidate buffers 4 bytes off a 16-byte boundary: the epilogue
    must fall back to element loads and give the same decisions."""
    import torch
    sp, pb, st, qs = _case(n_queries=257, seed=42)
    r = G.make_router(pb, pipeline="staged")
    r.update(st)
    ref = G.route_device(r, qs, "bf16")
    emb, il, no, slo = G.to_dev_inputs(qs, "bf16")
    out = G.dev_outputs(qs.n, r.N, r.M, False)
    n, N = qs.n, r.N
    tt = torch.zeros(n * N + 1, dtype=torch.float32, device="cuda")
    tp = torch.zeros(n * N + 1, dtype=torch.float32, device="cuda")
    assert tt[1:].data_ptr() % 16 != 0
    r.route(emb, il, no, slo, mem=hwr.HWR_MEM_DEVICE, cand_ttft=tt[1:], cand_tpot=tp[1:], **out)
    torch.cuda.synchronize()
    got = {k: v.cpu().numpy() for k, v in out.items()}
    _same(got, ref, keys=list(got))
    assert np.array_equal(tt[1:].cpu().numpy().reshape(n, N), ref["cand_ttft"])


def test_contexts_on_threads_are_independent():
    """Three contexts, each created and used by its own host thread on its
    own stream at the same time (a fused and a staged host batch, each over
    16 MB of pageable embeddings, so each context runs its own pinned ring and
    copy threads, and a run of single queries), give the same bits as each
    context alone."""
    import threading
    import torch
    work = []
    for name, seed, n, pipe in (("C2", 40, 12000, "fused"), ("C3", 41, 9000, "staged"), ("C4", 42, 40, "fused")):
        sp, pb, st, qs = _case(name, seed=seed, n_queries=n)
        work.append((pb, st, qs, pipe, name == "C4"))

    def run(pb, st, qs, pipe, single, stream):
        r = hwr.Router.from_problem(pb, pipeline=pipe, stream=stream)
        r.update(st)
        if single:
            outs = [r.route_host(qs.emb_bits[i:i + 1], qs.input_len[i:i + 1], qs.expected_out_len[i:i + 1],
                                 qs.slo_s[i:i + 1]) for i in range(qs.n)]
            out = {k: np.concatenate([o[k] for o in outs]) for k in outs[0]}
        else:
            out = r.route_host(qs.emb_bits, qs.input_len, qs.expected_out_len, qs.slo_s)
        r.close()
        return out

    ref = [run(*w, stream=G.torch_stream()) for w in work]
    got = [[] for _ in work]
    errors = []

    def worker(i):
        try:
            torch.cuda.set_device(0)
            s = torch.cuda.Stream()
            for _ in range(4):
                got[i].append(run(*work[i], stream=int(s.cuda_stream)))
            s.synchronize()
        except Exception as e:          # reported by the main thread
            errors.append((i, repr(e)))

    threads = [threading.Thread(target=worker, args=(i,)) for i in range(len(work))]
    for t in threads:
        t.start()
    for t in threads:
        t.join(timeout=120)
    assert not any(t.is_alive() for t in threads), "a routing thread did not finish"
    assert not errors, errors
    for i in range(len(work)):
        assert len(got[i]) == 4
        for out in got[i]:
            _same(out, ref[i])
