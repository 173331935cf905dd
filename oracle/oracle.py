"""ctypes front of the C oracle (hwr_oracle.c).  TEST INFRASTRUCTURE ONLY.

Only the tests, ``__graft_entry__.smoke()`` and the CPU-baseline leg of
``bench.py`` use this module.  It takes numpy arrays (weights and embeddings
as fp32 values; bf16 workloads pass their bf16 values exactly) and returns
numpy arrays.  It shares no code with the HIP library.
"""
from __future__ import annotations

import ctypes as C
import os
import subprocess
from dataclasses import dataclass
from typing import Optional

import numpy as np

_HERE = os.path.dirname(os.path.abspath(__file__))
# ORACLE_LIB_OVERRIDE points the pins at a deliberately broken copy of the
# oracle (tests/test_oracle_mutations.py checks that the pins catch it).
LIB_PATH = os.environ.get("ORACLE_LIB_OVERRIDE") or os.path.join(_HERE, "liboracle.so")
_SRC = os.path.join(_HERE, "hwr_oracle.c")

CFLAGS = ["-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off", "-fno-fast-math"]


def _stale() -> bool:
    if not os.path.exists(LIB_PATH):
        return True
    if os.environ.get("ORACLE_LIB_OVERRIDE"):
        return False
    t = os.path.getmtime(LIB_PATH)
    return any(os.path.getmtime(os.path.join(_HERE, f)) > t for f in ("hwr_oracle.c", "hwr_oracle.h"))


def build(force: bool = True) -> str:
    """Compile liboracle.so with gcc (plain C, contraction off); without
    ``force``, only when it is missing or older than its sources."""
    if force or _stale():
        tmp = LIB_PATH + ".tmp"
        subprocess.check_call(["gcc", *CFLAGS, "-o", tmp, _SRC, "-lm"])
        os.replace(tmp, LIB_PATH)
    return LIB_PATH


_i32p = C.POINTER(C.c_int32)
_f32p = C.POINTER(C.c_float)
_u8p = C.POINTER(C.c_uint8)


class _Problem(C.Structure):
    _fields_ = [("M", C.c_int32), ("G", C.c_int32), ("N", C.c_int32), ("D", C.c_int32),
                ("F", C.c_int32), ("H", C.c_int32), ("arch_width", C.c_int32),
                ("gpu_width", C.c_int32), ("bf16", C.c_int32), ("n_heads", C.c_int32),
                ("alpha", C.c_float), ("score_mode", C.c_int32), ("bound_mode", C.c_int32),
                ("ttft_slo_a", C.c_float), ("ttft_slo_b", C.c_float), ("tpot_slo", C.c_float),
                ("dep_model", _i32p), ("dep_gpu", _i32p), ("model_arch", _i32p),
                ("model_params_b", _f32p), ("wq", _f32p), ("bq", _f32p),
                ("w1", _f32p), ("b1", _f32p), ("w2", _f32p), ("b2", _f32p),
                ("w3", _f32p), ("b3", _f32p)]


class _State(C.Structure):
    _fields_ = [("running_q", _i32p), ("waiting_q", _i32p), ("kv_util", _f32p),
                ("gpu_util", _f32p), ("ttft_avg_s", _f32p), ("tpot_avg_s", _f32p)]


class _Rule(C.Structure):
    _fields_ = [("score_mode", C.c_int32), ("bound_mode", C.c_int32), ("w", C.c_float),
                ("ttft_slo_a", C.c_float), ("ttft_slo_b", C.c_float), ("tpot_slo", C.c_float)]


class _Queries(C.Structure):
    _fields_ = [("n", C.c_int32), ("emb", _f32p), ("input_len", _i32p),
                ("expected_out_len", _i32p), ("slo_s", _f32p)]


class _Result(C.Structure):
    _fields_ = [("choice", _i32p), ("feasible", _u8p), ("utility", _f32p),
                ("e2e_s", _f32p), ("ttft_s", _f32p), ("tpot_s", _f32p), ("nout", _f32p),
                ("cand_z", _f32p), ("cand_nout", _f32p), ("cand_ttft", _f32p), ("cand_tpot", _f32p),
                ("cand_e2e", _f32p), ("cand_u", _f32p), ("cand_bound", _f32p), ("cand_feasible", _u8p),
                ("quality", _f32p)]


_lib = None


def lib():
    global _lib
    if _lib is None:
        if _stale():
            build(force=False)
        L = C.CDLL(LIB_PATH)
        L.orc_bf16.restype = C.c_float
        L.orc_bf16.argtypes = [C.c_float]
        L.orc_bf16_n.restype = None
        L.orc_bf16_n.argtypes = [_f32p, _f32p, C.c_int64]
        L.orc_softplus.restype = C.c_float
        L.orc_softplus.argtypes = [C.c_float]
        L.orc_features.restype = None
        L.orc_features.argtypes = [C.POINTER(_Problem), C.POINTER(_State), C.c_int32, C.c_int32, _f32p]
        L.orc_quality.restype = C.c_float
        L.orc_quality.argtypes = [C.POINTER(_Problem), _f32p, C.c_int32]
        L.orc_mlp.restype = None
        L.orc_mlp.argtypes = [C.POINTER(_Problem), _f32p, _f32p]
        L.orc_decide.restype = C.c_int
        L.orc_decide.argtypes = [C.c_int32, C.c_int32, C.c_int32, _i32p, _f32p, _f32p, _f32p, _f32p,
                                 _i32p, _i32p, _f32p, C.POINTER(_Rule), _i32p, _u8p, _f32p, _f32p]
        L.orc_route.restype = C.c_int
        L.orc_route.argtypes = [C.POINTER(_Problem), C.POINTER(_State), C.POINTER(_Queries),
                                C.POINTER(_Result)]
        _lib = L
    return _lib


def _ptr(a: Optional[np.ndarray], ct):
    if a is None:
        return C.cast(None, C.POINTER(ct))
    return a.ctypes.data_as(C.POINTER(ct))


def _f32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.float32)


def _i32(a) -> np.ndarray:
    return np.ascontiguousarray(a, dtype=np.int32)


@dataclass
class OracleProblem:
    """Plain description of the routing problem (oracle-side)."""
    dep_model: np.ndarray
    dep_gpu: np.ndarray
    model_arch: np.ndarray
    model_params_b: np.ndarray
    wq: np.ndarray      # [D, M]
    bq: np.ndarray      # [M]
    w1: np.ndarray      # [F, H]
    b1: np.ndarray
    w2: np.ndarray      # [H, H]
    b2: np.ndarray
    w3: np.ndarray      # [H, 2]
    b3: np.ndarray      # [2]
    arch_width: int
    gpu_width: int
    n_gpu_types: int
    bf16: bool
    alpha: float = 0.5
    n_heads: int = 2
    score_mode: int = 0          # 0: u = Q - w C / B; 1: u = (1 - w) Q - w C
    bound_mode: int = 0          # 0: B = the query's SLO; 1: B = a + b p + N_out tpot_slo
    ttft_slo_a: float = 0.0
    ttft_slo_b: float = 0.0
    tpot_slo: float = 0.0

    @classmethod
    def from_synth(cls, pb, alpha: Optional[float] = None) -> "OracleProblem":
        sp = pb.spec
        return cls(pb.dep_model, pb.dep_gpu, pb.model_arch, pb.model_params_b,
                   pb.wq, pb.bq, pb.w1, pb.b1, pb.w2, pb.b2, pb.w3, pb.b3,
                   sp.arch_width, sp.gpu_width, sp.n_gpu_types, sp.dtype == "bf16",
                   sp.cost_weight if alpha is None else alpha, sp.n_heads, sp.score_mode,
                   sp.bound_mode, sp.ttft_slo_a, sp.ttft_slo_b, sp.tpot_slo)

    def _struct(self, keep: list) -> _Problem:
        arrs = dict(dep_model=_i32(self.dep_model), dep_gpu=_i32(self.dep_gpu),
                    model_arch=_i32(self.model_arch), model_params_b=_f32(self.model_params_b),
                    wq=_f32(self.wq), bq=_f32(self.bq), w1=_f32(self.w1), b1=_f32(self.b1),
                    w2=_f32(self.w2), b2=_f32(self.b2), w3=_f32(self.w3), b3=_f32(self.b3))
        keep.append(arrs)
        D, M = arrs["wq"].shape
        F, H = arrs["w1"].shape
        NH = int(self.n_heads)
        assert arrs["w2"].shape == (H, H) and arrs["w3"].shape == (H, NH) and arrs["b3"].shape == (NH,)
        N = arrs["dep_model"].shape[0]
        s = _Problem(M, int(self.n_gpu_types), N, D, F, H, int(self.arch_width),
                     int(self.gpu_width), int(bool(self.bf16)), NH, float(self.alpha),
                     int(self.score_mode), int(self.bound_mode), float(self.ttft_slo_a),
                     float(self.ttft_slo_b), float(self.tpot_slo))
        for k in ("dep_model", "dep_gpu", "model_arch"):
            setattr(s, k, _ptr(arrs[k], C.c_int32))
        for k in ("model_params_b", "wq", "bq", "w1", "b1", "w2", "b2", "w3", "b3"):
            setattr(s, k, _ptr(arrs[k], C.c_float))
        return s


def _state_struct(state: np.ndarray, keep: list) -> _State:
    arrs = dict(running_q=_i32(state["running_q"]), waiting_q=_i32(state["waiting_q"]),
                kv_util=_f32(state["kv_util"]), gpu_util=_f32(state["gpu_util"]),
                ttft_avg_s=_f32(state["ttft_avg_s"]), tpot_avg_s=_f32(state["tpot_avg_s"]))
    keep.append(arrs)
    s = _State()
    for k in ("running_q", "waiting_q"):
        setattr(s, k, _ptr(arrs[k], C.c_int32))
    for k in ("kv_util", "gpu_util", "ttft_avg_s", "tpot_avg_s"):
        setattr(s, k, _ptr(arrs[k], C.c_float))
    return s


def bf16(x: float) -> float:
    return float(lib().orc_bf16(float(x)))


def bf16_array(x) -> np.ndarray:
    xx = _f32(np.ravel(x))
    y = np.empty_like(xx)
    lib().orc_bf16_n(_ptr(xx, C.c_float), _ptr(y, C.c_float), xx.size)
    return y.reshape(np.shape(x))


def softplus(z: float) -> float:
    return float(lib().orc_softplus(float(z)))


def features(prob: OracleProblem, state: np.ndarray, d: int, input_len: int) -> np.ndarray:
    keep: list = []
    p = prob._struct(keep)
    s = _state_struct(state, keep)
    x = np.zeros(np.asarray(prob.w1).shape[0], np.float32)
    lib().orc_features(C.byref(p), C.byref(s), int(d), int(input_len), _ptr(x, C.c_float))
    return x


def quality(prob: OracleProblem, emb_row: np.ndarray, m: int) -> float:
    keep: list = []
    p = prob._struct(keep)
    e = _f32(emb_row)
    return float(lib().orc_quality(C.byref(p), _ptr(e, C.c_float), int(m)))


def mlp(prob: OracleProblem, x: np.ndarray) -> np.ndarray:
    keep: list = []
    p = prob._struct(keep)
    xx = _f32(x)
    z = np.zeros(int(prob.n_heads), np.float32)
    lib().orc_mlp(C.byref(p), _ptr(xx, C.c_float), _ptr(z, C.c_float))
    return z


@dataclass
class OracleResult:
    choice: np.ndarray
    feasible: np.ndarray
    utility: np.ndarray
    e2e_s: np.ndarray
    ttft_s: np.ndarray
    tpot_s: np.ndarray
    nout: Optional[np.ndarray] = None        # [n] N_out used for the chosen pair
    cand_z: Optional[np.ndarray] = None      # [n, N, n_heads]
    cand_nout: Optional[np.ndarray] = None   # [n, N] N_out used per candidate
    cand_ttft: Optional[np.ndarray] = None   # [n, N]
    cand_tpot: Optional[np.ndarray] = None
    cand_e2e: Optional[np.ndarray] = None
    cand_u: Optional[np.ndarray] = None
    cand_bound: Optional[np.ndarray] = None   # [n, N] the bound B of each candidate
    cand_feasible: Optional[np.ndarray] = None
    quality: Optional[np.ndarray] = None     # [n, M]


def route(prob: OracleProblem, state: np.ndarray, emb: np.ndarray, input_len, expected_out_len,
          slo_s, candidates: bool = True) -> OracleResult:
    """Run the whole path on the CPU.  ``candidates`` also returns every
    per-candidate intermediate (needed by the acceptance rule)."""
    keep: list = []
    p = prob._struct(keep)
    s = _state_struct(state, keep)
    emb = _f32(emb)
    n = emb.shape[0]
    N = p.N
    M = p.M
    il, no, slo = _i32(input_len), _i32(expected_out_len), _f32(slo_s)
    assert il.shape == (n,) and no.shape == (n,) and slo.shape == (n,)
    assert emb.shape[1] == p.D
    q = _Queries(n, _ptr(emb, C.c_float), _ptr(il, C.c_int32), _ptr(no, C.c_int32),
                 _ptr(slo, C.c_float))
    out = OracleResult(np.zeros(n, np.int32), np.zeros(n, np.uint8), np.zeros(n, np.float32),
                       np.zeros(n, np.float32), np.zeros(n, np.float32), np.zeros(n, np.float32))
    out.nout = np.zeros(n, np.float32)
    r = _Result()
    r.choice = _ptr(out.choice, C.c_int32)
    r.feasible = _ptr(out.feasible, C.c_uint8)
    for k in ("utility", "e2e_s", "ttft_s", "tpot_s", "nout"):
        setattr(r, k, _ptr(getattr(out, k), C.c_float))
    if candidates:
        out.cand_z = np.zeros((n, N, int(prob.n_heads)), np.float32)
        for k in ("cand_nout", "cand_ttft", "cand_tpot", "cand_e2e", "cand_u", "cand_bound"):
            setattr(out, k, np.zeros((n, N), np.float32))
        out.cand_feasible = np.zeros((n, N), np.uint8)
        out.quality = np.zeros((n, M), np.float32)
        for k in ("cand_z", "cand_nout", "cand_ttft", "cand_tpot", "cand_e2e", "cand_u", "cand_bound",
                  "quality"):
            setattr(r, k, _ptr(getattr(out, k), C.c_float))
        r.cand_feasible = _ptr(out.cand_feasible, C.c_uint8)
    rc = lib().orc_route(C.byref(p), C.byref(s), C.byref(q), C.byref(r))
    if rc != 0:
        raise ValueError("oracle rejected the problem sizes")
    return out


def decide(dep_model, cand_ttft, cand_tpot, quality, expected_out_len, slo_s, alpha: float,
           cand_nout=None, input_len=None, score_mode: int = 0, bound_mode: int = 0,
           ttft_slo_a: float = 0.0, ttft_slo_b: float = 0.0, tpot_slo: float = 0.0) -> dict:
    """Eq. 2 and Eq. 3 on given predictions (the decision step alone, same
    arithmetic and tie rule as ``route``): per query the choice, feasibility,
    utility and cost.  Inputs: TTFT / TPOT [n, N], quality [n, M]; N_out per
    candidate [n, N] (three heads) or None (the queries' expected_out_len);
    the rule (weight ``alpha``, score and bound modes) as in ``orc_rule``."""
    tt, tp, qual = _f32(cand_ttft), _f32(cand_tpot), _f32(quality)
    cn = None if cand_nout is None else _f32(cand_nout)
    n, N = tt.shape
    M = qual.shape[1]
    dm, no, slo = _i32(dep_model), _i32(expected_out_len), _f32(slo_s)
    il = _i32(np.ones(tt.shape[0]) if input_len is None else input_len)
    rule = _Rule(int(score_mode), int(bound_mode), float(alpha), float(ttft_slo_a), float(ttft_slo_b),
                 float(tpot_slo))
    assert tp.shape == (n, N) and qual.shape[0] == n and dm.shape == (N,)
    assert no.shape == (n,) and slo.shape == (n,) and (cn is None or cn.shape == (n, N))
    out = {"choice": np.zeros(n, np.int32), "feasible": np.zeros(n, np.uint8),
           "utility": np.zeros(n, np.float32), "e2e_s": np.zeros(n, np.float32)}
    rc = lib().orc_decide(n, N, M, _ptr(dm, C.c_int32), _ptr(tt, C.c_float), _ptr(tp, C.c_float),
                          _ptr(cn, C.c_float), _ptr(qual, C.c_float), _ptr(il, C.c_int32), _ptr(no, C.c_int32),
                          _ptr(slo, C.c_float), C.byref(rule), _ptr(out["choice"], C.c_int32), _ptr(out["feasible"], C.c_uint8),
                          _ptr(out["utility"], C.c_float), _ptr(out["e2e_s"], C.c_float))
    if rc != 0:
        raise ValueError("oracle rejected the sizes")
    return out


def route_synth(pb, state, qs, candidates: bool = True, alpha: Optional[float] = None) -> OracleResult:
    """Convenience: route generator objects (synth.Problem / synth.Queries)."""
    return route(OracleProblem.from_synth(pb, alpha), state, qs.emb, qs.input_len,
                 qs.expected_out_len, qs.slo_s, candidates)
