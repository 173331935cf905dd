"""Helpers for the GPU tests: run the HIP library on generator workloads
(device batches through torch tensors) and the oracle beside it."""
from __future__ import annotations

import os

import numpy as np

from oracle import oracle as O
from paper_2608_14575_amd import hwr
from paper_2608_14575_amd import synth as S

import parity


def torch_stream() -> int:
    import torch
    return int(torch.cuda.current_stream().cuda_stream)


def make_router(pb, **kw) -> hwr.Router:
    kw.setdefault("stream", torch_stream())
    return hwr.Router.from_problem(pb, **kw)


def to_dev_inputs(qs, dtype: str):
    import torch
    dev = torch.device("cuda")
    if dtype == "bf16":
        emb = torch.from_numpy(np.ascontiguousarray(qs.emb_bits).view(np.int16)).to(dev)
    else:
        emb = torch.from_numpy(np.ascontiguousarray(qs.emb_bits, np.float32)).to(dev)
    il = torch.from_numpy(np.ascontiguousarray(qs.input_len)).to(dev)
    no = torch.from_numpy(np.ascontiguousarray(qs.expected_out_len)).to(dev)
    slo = torch.from_numpy(np.ascontiguousarray(qs.slo_s)).to(dev)
    return emb, il, no, slo


def dev_outputs(n: int, N: int, M: int, candidates: bool, heads: int = 2, weights: int = 1):
    import torch
    dev = torch.device("cuda")
    sh = (n,) if weights == 1 else (n, weights)
    out = dict(choice=torch.full(sh, -1, dtype=torch.int32, device=dev),
               feasible=torch.zeros(sh, dtype=torch.uint8, device=dev),
               utility=torch.zeros(sh, dtype=torch.float32, device=dev),
               e2e_s=torch.zeros(sh, dtype=torch.float32, device=dev),
               ttft_s=torch.zeros(sh, dtype=torch.float32, device=dev),
               tpot_s=torch.zeros(sh, dtype=torch.float32, device=dev),
               nout=torch.zeros(sh, dtype=torch.float32, device=dev))
    if candidates:
        out.update(cand_ttft=torch.zeros((n, N), dtype=torch.float32, device=dev),
                   cand_tpot=torch.zeros((n, N), dtype=torch.float32, device=dev),
                   cand_quality=torch.zeros((n, M), dtype=torch.float32, device=dev))
        if heads == 3:
            out["cand_nout"] = torch.zeros((n, N), dtype=torch.float32, device=dev)
    return out


def route_device(router: hwr.Router, qs, dtype: str, candidates: bool = True, with_slo: bool = True):
    import torch
    emb, il, no, slo = to_dev_inputs(qs, dtype)
    out = dev_outputs(qs.n, router.N, router.M, candidates, router.n_heads, router.n_weights)
    router.route(emb, il, no, slo if with_slo else None, mem=hwr.HWR_MEM_DEVICE, **out)
    torch.cuda.synchronize()
    return {k: v.cpu().numpy() for k, v in out.items()}


def rtol_for(dtype: str) -> float:
    return 1e-2 if dtype == "bf16" else 1e-4


def check(pb, state, qs, gpu: dict, rtol: float = None, query_ids=None, alpha=None) -> parity.ParityReport:
    sp = pb.spec
    rtol = rtol_for(sp.dtype) if rtol is None else rtol
    alpha = sp.cost_weight if alpha is None else alpha
    orc = O.route_synth(pb, state, qs, candidates=True, alpha=alpha)
    return parity.compare(gpu, orc, slo=qs.slo_s, alpha=alpha, dep_model=pb.dep_model,
                          rtol=rtol, emb=qs.emb, wq=pb.wq, bq=pb.bq, query_ids=query_ids,
                          heads=sp.n_heads, score_mode=sp.score_mode)


def oracle_threaded(pb, state, qs, candidates: bool = True, alpha=None, threads: int = 16):
    """The oracle on ``qs`` split into per-thread shards (the C call releases
    the interpreter lock), concatenated back in query order: the same
    results as one call, in a fraction of the time on a many-core host."""
    from concurrent.futures import ThreadPoolExecutor
    threads = max(1, min(threads, os.cpu_count() or 1, qs.n))
    bounds = np.linspace(0, qs.n, threads + 1).astype(int)
    shards = [qs.slice(int(a), int(b)) for a, b in zip(bounds[:-1], bounds[1:]) if b > a]
    O.lib()
    with ThreadPoolExecutor(max_workers=len(shards)) as ex:
        parts = list(ex.map(lambda q: O.route_synth(pb, state, q, candidates=candidates, alpha=alpha), shards))
    return stack_results(parts)


def stack_results(parts):
    """Concatenate oracle results of consecutive query ranges."""
    out = {}
    for f in O.OracleResult.__dataclass_fields__:
        vals = [getattr(r, f) for r in parts]
        out[f] = None if any(v is None for v in vals) else np.concatenate(vals, axis=0)
    return O.OracleResult(**out)


def check_against(pb, qs, gpu: dict, orc, rtol: float = None, query_ids=None, alpha=None) -> parity.ParityReport:
    """``check`` with a precomputed oracle result."""
    sp = pb.spec
    rtol = rtol_for(sp.dtype) if rtol is None else rtol
    alpha = sp.cost_weight if alpha is None else alpha
    return parity.compare(gpu, orc, slo=qs.slo_s, alpha=alpha, dep_model=pb.dep_model, rtol=rtol,
                          emb=qs.emb, wq=pb.wq, bq=pb.bq, query_ids=query_ids, heads=sp.n_heads,
                          score_mode=sp.score_mode)
