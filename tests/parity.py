"""Acceptance rule for GPU routing results against the CPU oracle.

Predictions: every candidate's TTFT and TPOT within ``rtol`` relative of the
oracle; qualities within ``rtol`` of their dot-product error scale
sum_k |e_k Wq_km| + |bq_m|.

With a third head the predicted N_out of every candidate is compared the
same way, and the cost C = TTFT + N_out * TPOT then carries two uncertain
factors, so its share of the uncertainty below is doubled (k = 2, else 1).

Decisions: floating point decides the choice, so the choice is compared
exactly only where the oracle's decision is robust to errors of that size
(B_c is the candidate's bound: the query's SLO, or the paper form):
  tau_c = rtol * (|Q_c| + k * alpha * C_c / B_c)      (utility uncertainty;
          rtol * ((1 - alpha) |Q_c| + k * alpha * C_c) for the paper score)
  ambiguous_c = |C_c - B_c| <= rtol * (k * C_c + B_c) (bound test uncertain)
A query is *eligible* for a bit-exact choice when its winner b is not
ambiguous, no ambiguous candidate could enter or leave the feasible set in a
way that changes the winner, and every other competitor c has
u_b - u_c > tau_b + tau_c.  Otherwise the GPU's choice g must be one some
admissible perturbation could produce (the epsilon-set):
  - if some candidate is surely feasible (feasible, not ambiguous):
    g is feasible or ambiguous, and u_g >= max over surely feasible c of
    (u_c - tau_c) - tau_g;
  - else g is ambiguous, or u_g >= max over all c of (u_c - tau_c) - tau_g.
"""
from __future__ import annotations

from dataclasses import dataclass, field

import numpy as np


@dataclass
class ParityReport:
    n: int
    eligible: int = 0
    exact: int = 0
    eps_ok: int = 0
    max_rel_ttft: float = 0.0
    max_rel_tpot: float = 0.0
    max_rel_quality: float = 0.0
    max_rel_nout: float = 0.0
    max_rel_chosen: float = 0.0
    failures: list = field(default_factory=list)

    @property
    def ok(self) -> bool:
        return not self.failures

    def summary(self) -> str:
        return (f"n={self.n} eligible={self.eligible / max(self.n, 1):.3f} "
                f"exact={self.exact}/{self.eligible} eps={self.eps_ok}/{self.n - self.eligible} "
                f"max_rel ttft={self.max_rel_ttft:.2e} tpot={self.max_rel_tpot:.2e} "
                f"quality={self.max_rel_quality:.2e} nout={self.max_rel_nout:.2e} "
                f"chosen={self.max_rel_chosen:.2e}")


def compare(gpu: dict, orc, *, slo: np.ndarray, alpha: float, dep_model: np.ndarray, rtol: float,
            emb: np.ndarray = None, wq: np.ndarray = None, bq: np.ndarray = None,
            query_ids=None, heads: int = 2, score_mode: int = 0) -> ParityReport:
    """gpu: dict of numpy outputs (choice, feasible, utility, e2e_s, ttft_s,
    tpot_s, optional cand_ttft / cand_tpot / cand_quality), rows aligned
    with the oracle result ``orc`` (oracle.OracleResult with candidates)."""
    n = len(orc.choice)
    rep = ParityReport(n)
    qid = np.arange(n) if query_ids is None else np.asarray(query_ids)
    tt_o, tp_o = orc.cand_ttft.astype(np.float64), orc.cand_tpot.astype(np.float64)
    if gpu.get("cand_ttft") is not None:
        e1 = np.abs(gpu["cand_ttft"] - tt_o) / tt_o
        e2 = np.abs(gpu["cand_tpot"] - tp_o) / tp_o
        rep.max_rel_ttft, rep.max_rel_tpot = float(e1.max()), float(e2.max())
        if rep.max_rel_ttft > rtol or rep.max_rel_tpot > rtol:
            bad = np.argwhere((e1 > rtol) | (e2 > rtol))[:5]
            rep.failures.append(f"predictions beyond rtol at (query, pair) {bad.tolist()}")
    if heads == 3 and gpu.get("cand_nout") is not None:
        no_o = orc.cand_nout.astype(np.float64)
        en = np.abs(gpu["cand_nout"] - no_o) / no_o
        rep.max_rel_nout = float(en.max())
        if rep.max_rel_nout > rtol:
            rep.failures.append(f"N_out predictions beyond rtol (max {rep.max_rel_nout:.3e})")
    if gpu.get("cand_quality") is not None and emb is not None:
        scale = np.abs(emb.astype(np.float64)) @ np.abs(wq.astype(np.float64)) + np.abs(bq)
        eq = np.abs(gpu["cand_quality"] - orc.quality) / scale
        rep.max_rel_quality = float(eq.max())
        if rep.max_rel_quality > rtol:
            rep.failures.append(f"quality beyond rtol (max {rep.max_rel_quality:.3e})")

    Q = orc.quality[:, dep_model].astype(np.float64)
    C = orc.cand_e2e.astype(np.float64)
    u = orc.cand_u.astype(np.float64)
    S = (orc.cand_bound.astype(np.float64) if getattr(orc, "cand_bound", None) is not None
         else np.broadcast_to(slo.astype(np.float64)[:, None], C.shape))
    k = 2.0 if heads == 3 else 1.0
    if score_mode == 1:
        tau = rtol * ((1.0 - alpha) * np.abs(Q) + k * alpha * C)
    else:
        tau = rtol * (np.abs(Q) + k * alpha * C / S)
    amb = np.abs(C - S) <= rtol * (k * C + S)
    feas = orc.cand_feasible.astype(bool)
    sure = feas & ~amb
    g_all = np.asarray(gpu["choice"]).astype(np.int64)
    N = C.shape[1]
    for i in range(n):
        b = int(orc.choice[i])
        g = int(g_all[i])
        if not (0 <= g < N):
            rep.failures.append(f"query {qid[i]}: choice {g} out of range")
            continue
        others = np.arange(N) != b
        if feas[i, b]:
            comp = others & (feas[i] | amb[i])
        else:
            comp = others
        eligible = (not amb[i, b]) and bool(np.all(u[i, b] - u[i, comp] > tau[i, b] + tau[i, comp]))
        if not feas[i, b] and amb[i].any():
            eligible = False
        if eligible:
            rep.eligible += 1
            if g == b:
                rep.exact += 1
                fl = gpu.get("feasible")
                if fl is not None and int(fl[i]) != int(orc.feasible[i]):
                    rep.failures.append(f"query {qid[i]}: feasible flag differs")
            else:
                rep.failures.append(f"query {qid[i]}: eligible, oracle {b} (u={u[i, b]:.6f}) gpu {g} "
                                    f"(u={u[i, g]:.6f})")
            continue
        if sure[i].any():
            floor = np.max(u[i, sure[i]] - tau[i, sure[i]])
            ok = (feas[i, g] or amb[i, g]) and u[i, g] >= floor - tau[i, g]
        else:
            floor = np.max(u[i] - tau[i])
            ok = amb[i, g] or u[i, g] >= floor - tau[i, g]
        if ok:
            rep.eps_ok += 1
        else:
            rep.failures.append(f"query {qid[i]}: gpu {g} outside the epsilon-set (oracle {b})")
    # values reported for the chosen pair agree with the oracle's for that pair
    rows = np.arange(n)
    refs = [("ttft_s", tt_o), ("tpot_s", tp_o), ("e2e_s", C)]
    if heads == 3:
        refs.append(("nout", orc.cand_nout.astype(np.float64)))
    for key, ref in refs:
        if gpu.get(key) is not None:
            r = ref[rows, g_all]
            err = np.abs(np.asarray(gpu[key], np.float64) - r) / np.abs(r)
            rep.max_rel_chosen = max(rep.max_rel_chosen, float(err.max()))
    if gpu.get("utility") is not None:
        err = np.abs(np.asarray(gpu["utility"], np.float64) - u[rows, g_all]) / (tau[rows, g_all] / rtol)
        rep.max_rel_chosen = max(rep.max_rel_chosen, float(err.max()))
    if rep.max_rel_chosen > rtol:
        rep.failures.append(f"values of the chosen pair beyond rtol ({rep.max_rel_chosen:.3e})")
    return rep
