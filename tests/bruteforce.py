"""Brute-force routing in pure Python (stdlib only), for tiny inputs.

An independent cross-check of the C oracle: every candidate (query, pair) is
evaluated with exact rational sums (``fractions``) rounded once to fp32 at the
documented rounding points, the full candidate tuples are sorted, and the top
tuple is the choice.  The selection rule of Eq. 3 is applied by sorting on
(feasible, u, -pair) rather than by a running maximum.
"""
from __future__ import annotations

import math
import struct
from fractions import Fraction


def f32(x: float) -> float:
    """Nearest fp32 value of a Python float (ties to even)."""
    return struct.unpack("<f", struct.pack("<f", x))[0]


def _f32_neighbours(x: float):
    b = struct.unpack("<I", struct.pack("<f", f32(x)))[0]
    up = struct.unpack("<f", struct.pack("<I", b + 1))[0] if b != 0x7F7FFFFF else float("inf")
    dn = struct.unpack("<f", struct.pack("<I", b - 1))[0] if b not in (0, 0x80000000) else -0.0
    return dn, f32(x), up


def f32_exact(q: Fraction) -> float:
    """Round an exact rational to the nearest fp32 (ties to even), without the
    double rounding a pass through fp64 could cause."""
    best = None
    for c in _f32_neighbours(float(q)):
        if math.isinf(c):
            continue
        dist = abs(Fraction(c) - q)
        even = (struct.unpack("<I", struct.pack("<f", c))[0] & 1) == 0
        key = (dist, not even)
        if best is None or key < best[0]:
            best = (key, c)
    return best[1]


def bf16(x: float) -> float:
    """Nearest bf16 value of an fp32 value (ties to even), via the fp32 bits."""
    b = struct.unpack("<I", struct.pack("<f", x))[0]
    kept, dropped = b >> 16, b & 0xFFFF
    if dropped > 0x8000 or (dropped == 0x8000 and kept & 1):
        kept += 1
    return struct.unpack("<f", struct.pack("<I", (kept << 16) & 0xFFFFFFFF))[0]


def _dot(a, b, bias) -> float:
    return f32_exact(sum((Fraction(x) * Fraction(y) for x, y in zip(a, b)), Fraction(bias)))


def route(prob: dict, state: list, queries: list):
    """prob: dict of plain lists (weights row-major as nested lists),
    state: list of dicts per pair, queries: list of dicts.
    Returns (choices, per-query sorted candidate tuples)."""
    M, N, F, H = prob["M"], prob["N"], prob["F"], prob["H"]
    A, Gw = prob["arch_width"], prob["gpu_width"]
    use_bf16 = prob["bf16"]
    rnd = (lambda v: bf16(f32(v))) if use_bf16 else f32
    choices, ranked = [], []
    for q in queries:
        qual = [_dot(q["emb"], [prob["wq"][k][m] for k in range(len(q["emb"]))], prob["bq"][m])
                for m in range(M)]
        cands = []
        for d in range(N):
            m, g, s = prob["dep_model"][d], prob["dep_gpu"][d], state[d]
            x = [0.0] * F
            x[prob["model_arch"][m]] = 1.0
            x[A + g] = 1.0
            b = A + Gw
            x[b + 0] = rnd(math.log(prob["model_params_b"][m]) / 4)
            x[b + 1] = rnd(math.log(q["input_len"]) / 8)
            x[b + 2] = rnd(math.log(1 + s["running_q"]) / 2)
            x[b + 3] = rnd(math.log(1 + s["waiting_q"]) / 2)
            x[b + 4] = rnd(s["kv_util"])
            x[b + 5] = rnd(s["gpu_util"])
            x[b + 6] = rnd(math.log(s["ttft_avg_s"]) / 4)
            x[b + 7] = rnd(math.log(s["tpot_avg_s"]) / 4)
            h1 = []
            for j in range(H):
                a = _dot([prob["w1"][f][j] for f in range(F)], x, prob["b1"][j])
                h1.append(bf16(max(a, 0.0)) if use_bf16 else max(a, 0.0))
            h2 = []
            for j in range(H):
                a = _dot([prob["w2"][i][j] for i in range(H)], h1, prob["b2"][j])
                h2.append(bf16(max(a, 0.0)) if use_bf16 else max(a, 0.0))
            NH = prob.get("n_heads", 2)
            z = [_dot([prob["w3"][i][k] for i in range(H)], h2, prob["b3"][k]) for k in range(NH)]
            sp = [f32(max(v, 0.0) + math.log1p(math.exp(-abs(v)))) for v in z]
            ttft, tpot = sp[0], sp[1]
            nout = sp[2] if NH == 3 else q["expected_out_len"]   # Eq. 1 third head, else given
            e2e = f32_exact(Fraction(tpot) * Fraction(nout) + Fraction(ttft))
            slo = f32(q["slo_s"])
            feas = 1 if e2e <= slo else 0
            t = f32_exact(Fraction(e2e) / Fraction(slo))
            at = f32_exact(Fraction(f32(prob["alpha"])) * Fraction(t))
            u = f32_exact(Fraction(qual[m]) - Fraction(at))
            cands.append((feas, u, -d, dict(d=d, ttft=ttft, tpot=tpot, nout=nout, e2e=e2e, u=u, z=z,
                                              feasible=feas, quality=qual[m])))
        order = sorted(cands, key=lambda c: (c[0], c[1], c[2]), reverse=True)
        choices.append(order[0][3]["d"])
        ranked.append(order)
    return choices, ranked


def from_synth(pb, state, qs, alpha=None):
    """Plain-list copies of generator objects."""
    sp = pb.spec
    prob = dict(M=sp.n_models, N=pb.n_deployments, F=sp.feat_dim, H=sp.hidden,
                arch_width=sp.arch_width, gpu_width=sp.gpu_width, bf16=sp.dtype == "bf16",
                n_heads=sp.n_heads,
                alpha=sp.cost_weight if alpha is None else alpha,
                dep_model=[int(v) for v in pb.dep_model], dep_gpu=[int(v) for v in pb.dep_gpu],
                model_arch=[int(v) for v in pb.model_arch],
                model_params_b=[float(v) for v in pb.model_params_b],
                wq=pb.wq.tolist(), bq=[float(v) for v in pb.bq], w1=pb.w1.tolist(),
                b1=[float(v) for v in pb.b1], w2=pb.w2.tolist(), b2=[float(v) for v in pb.b2],
                w3=pb.w3.tolist(), b3=[float(v) for v in pb.b3])
    st = [dict(running_q=int(s["running_q"]), waiting_q=int(s["waiting_q"]),
               kv_util=float(s["kv_util"]), gpu_util=float(s["gpu_util"]),
               ttft_avg_s=float(s["ttft_avg_s"]), tpot_avg_s=float(s["tpot_avg_s"])) for s in state]
    qq = [dict(emb=[float(v) for v in qs.emb[i]], input_len=int(qs.input_len[i]),
               expected_out_len=int(qs.expected_out_len[i]), slo_s=float(qs.slo_s[i]))
          for i in range(qs.n)]
    return prob, st, qq
