"""GPU parity of the single-query latency path (one host query, all pairs in
one workgroup, graph or plain launch) for every hidden width and for pair
counts spanning several 32-pair tiles, against the CPU oracle."""
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


@pytest.mark.parametrize("name,kw", [
    ("C2", dict(hidden=64)),                          # H = 64, 16 pairs
    ("C3", dict()),                                   # H = 256, 64 pairs (2 tiles), D = 1024
    ("C5", dict()),                                   # H = 256, 256 pairs (8 tiles), D = 1536, M = 32
    ("C2", dict(n_models=5, n_gpu_types=3)),          # 15 pairs, odd model count
    ("C4", dict(n_heads=3)),                          # predicted N_out (third head), H = 128
    ("C3", dict(n_heads=3)),                          # predicted N_out, H = 256, 2 tiles
])
@pytest.mark.parametrize("flags", [0, hwr.HWR_FLAG_GRAPH])
def test_single_query_matches_oracle(name, kw, flags):
    sp = S.spec(name, n_queries=40, **kw)
    pb, st, qs = S.make_problem(sp, 17), S.make_state(sp, 17), S.make_queries(sp, 17)
    r = G.make_router(pb, flags=flags)
    r.update(st)
    outs = []
    for i in range(qs.n):
        one = qs.slice(i, i + 1)
        outs.append(r.route_host(one.emb_bits, one.input_len, one.expected_out_len, one.slo_s))
    got = {k: np.concatenate([o[k] for o in outs]) for k in outs[0]}
    orc = O.route_synth(pb, st, qs)
    rep = parity.compare(got, orc, slo=qs.slo_s, alpha=sp.cost_weight, dep_model=pb.dep_model,
                         rtol=1e-2, heads=sp.n_heads)
    print(f"[parity] single {name} {kw} flags={flags}: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]
    # the batch path on the same queries agrees on every eligible choice
    batch = G.route_device(r, qs, "bf16", candidates=False)
    assert (batch["choice"] == got["choice"]).mean() > 0.9
    if sp.n_heads == 2:
        assert np.array_equal(got["nout"], qs.expected_out_len.astype(np.float32))


@pytest.mark.parametrize("flags", [0, hwr.HWR_FLAG_RESIDENT])
def test_single_query_maximum_shape(flags):
    """The single-query kernel at the largest shape: 1024 pairs (32 models x 8
    GPU types, each listed four times with its own state), D = 8192, H = 256.
    Every fallback of the kernel runs: pair rows past the first 32, quality
    weight pieces past the eight held per lane, the second pass of models."""
    sp = S.spec("C5", n_queries=8, embed_dim=8192)
    pb = S.make_problem(sp, 41)
    pb.dep_model = np.tile(pb.dep_model, 4)
    pb.dep_gpu = np.tile(pb.dep_gpu, 4)
    st = np.concatenate([S.make_state(sp, 41 + k) for k in range(4)])
    qs = S.make_queries(sp, 41)
    r = G.make_router(pb, flags=flags)
    r.update(st)
    outs = [r.route_host(qs.emb_bits[i:i + 1], qs.input_len[i:i + 1], qs.expected_out_len[i:i + 1],
                         qs.slo_s[i:i + 1]) for i in range(qs.n)]
    r.close()
    got = {k: np.concatenate([o[k] for o in outs]) for k in outs[0]}
    orc = O.route_synth(pb, st, qs)
    rep = parity.compare(got, orc, slo=qs.slo_s, alpha=sp.cost_weight, dep_model=pb.dep_model,
                         rtol=1e-2, heads=sp.n_heads)
    print(f"[parity] single max shape flags={flags}: {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]
