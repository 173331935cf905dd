"""ctypes binding of libhwr (include/hwr.h): the same entry points, argument
marshalling only.  Every step of the routing path runs in the library's HIP
kernels; if libhwr.so is missing this module raises instead of falling back.

``Router`` is a convenience wrapper that fills ``hwr_config`` from numpy
arrays and routes numpy (host) or torch (device) batches.
"""
from __future__ import annotations

import ctypes as C
import os
from typing import Optional

import numpy as np

_PKG = os.path.dirname(os.path.abspath(__file__))
LIB_PATH = os.path.join(_PKG, "libhwr.so")

HWR_OK, HWR_ERR_INVALID_ARG, HWR_ERR_OOM, HWR_ERR_HIP, HWR_ERR_STATE, HWR_ERR_UNSUPPORTED = 0, -1, -2, -3, -4, -5
HWR_F32, HWR_BF16 = 0, 1
HWR_MEM_DEVICE, HWR_MEM_HOST = 0, 1
HWR_PIPE_FUSED, HWR_PIPE_STAGED = 0, 1
HWR_FLAG_GRAPH = 1
HWR_FLAG_RESIDENT = 2
HWR_SCORE_NORMALIZED, HWR_SCORE_PAPER = 0, 1
HWR_BOUND_GIVEN, HWR_BOUND_PAPER = 0, 1
HWR_MAX_WEIGHTS = 8
HWR_K_STATE, HWR_K_QUALITY, HWR_K_GATHER, HWR_K_MLP, HWR_K_EPILOGUE, HWR_K_FUSED, HWR_K_MERGE, HWR_K_SINGLE = range(8)
HWR_K_COUNT = 8
KERNEL_NAMES = ["state", "quality", "gather", "mlp", "epilogue", "fused", "merge", "single"]

EXPORTS = ["hwr_init", "hwr_update_hw_state", "hwr_route_batch", "hwr_route_batch_static", "hwr_free",
           "hwr_last_error",
           "hwr_profile_enable", "hwr_profile_read", "hwr_sim_run", "hwr_sim_last_error",
           "hwr_probe_mfma_bf16", "hwr_probe_hbm_read", "hwr_probe_hbm_write", "hwr_probe_launch_floor",
           "hwr_probe_feature_log"]

_STATUS = {0: "HWR_OK", -1: "HWR_ERR_INVALID_ARG", -2: "HWR_ERR_OOM", -3: "HWR_ERR_HIP",
           -4: "HWR_ERR_STATE", -5: "HWR_ERR_UNSUPPORTED"}


class HwrError(RuntimeError):
    def __init__(self, status: int, msg: str):
        super().__init__(f"{_STATUS.get(status, status)}: {msg}")
        self.status = status


_vp = C.c_void_p
_i32p = C.POINTER(C.c_int32)
_f32p = C.POINTER(C.c_float)
_u8p = C.POINTER(C.c_uint8)


class hwr_hw_state(C.Structure):
    _fields_ = [("running_q", C.c_int32), ("waiting_q", C.c_int32), ("kv_util", C.c_float),
                ("gpu_util", C.c_float), ("ttft_avg_s", C.c_float), ("tpot_avg_s", C.c_float)]


class hwr_config(C.Structure):
    _fields_ = [("n_models", C.c_int32), ("n_gpu_types", C.c_int32), ("n_deployments", C.c_int32),
                ("arch_width", C.c_int32), ("gpu_width", C.c_int32), ("embed_dim", C.c_int32),
                ("feat_dim", C.c_int32), ("hidden", C.c_int32), ("emb_dtype", C.c_int32),
                ("weight_dtype", C.c_int32), ("pipeline", C.c_int32), ("max_chunk", C.c_int32),
                ("cost_weight", C.c_float), ("default_slo_s", C.c_float), ("device", C.c_int32),
                ("flags", C.c_int32), ("n_heads", C.c_int32), ("score_mode", C.c_int32),
                ("bound_mode", C.c_int32), ("ttft_slo_a", C.c_float), ("ttft_slo_b", C.c_float),
                ("tpot_slo", C.c_float), ("n_weights", C.c_int32),
                ("dep_model", _i32p), ("dep_gpu", _i32p), ("model_arch", _i32p),
                ("model_params_b", _f32p), ("wq", _vp), ("bq", _f32p), ("w1", _vp), ("b1", _f32p),
                ("w2", _vp), ("b2", _f32p), ("w3", _vp), ("b3", _f32p), ("cost_weights", _f32p),
                ("stream", _vp)]


class hwr_query_batch(C.Structure):
    _fields_ = [("n", C.c_int32), ("mem", C.c_int32), ("emb", _vp), ("input_len", _vp),
                ("expected_out_len", _vp), ("slo_s", _vp)]


class hwr_route_result(C.Structure):
    _fields_ = [("choice", _vp), ("feasible", _vp), ("utility", _vp), ("e2e_s", _vp),
                ("ttft_s", _vp), ("tpot_s", _vp), ("nout", _vp), ("cand_ttft", _vp), ("cand_tpot", _vp),
                ("cand_nout", _vp), ("cand_quality", _vp)]


class hwr_kernel_times(C.Structure):
    _fields_ = [("ms", C.c_double * HWR_K_COUNT), ("launches", C.c_int64 * HWR_K_COUNT)]


# ---- include/hwr_sim.h
class hwr_sim_pair(C.Structure):
    _fields_ = [("gpu", C.c_int32), ("max_running", C.c_int32), ("kv_capacity", C.c_int64),
                ("prefill_base_us", C.c_int32), ("prefill_per_token_ns", C.c_int32),
                ("tpot_base_us", C.c_int32), ("tpot_per_running_us", C.c_int32)]


class hwr_sim_config(C.Structure):
    _fields_ = [("n_pairs", C.c_int32), ("n_gpus", C.c_int32), ("pairs", _vp), ("tick_us", C.c_int32),
                ("monitor_period_us", C.c_int32), ("max_time_us", C.c_int64), ("freeze_state", C.c_int32),
                ("prior_ttft_s", _vp), ("prior_tpot_s", _vp)]


class hwr_sim_requests(C.Structure):
    _fields_ = [("n", C.c_int32), ("arrival_us", _vp), ("input_len", _vp), ("output_len", _vp),
                ("slo_us", _vp), ("emb", _vp), ("embed_dim", C.c_int32), ("emb_dtype", C.c_int32),
                ("expected_out_len", _vp), ("route_slo_s", _vp)]


SIM_METRICS = ["n_samples", "end_us", "n_completed", "n_met_slo", "route_calls", "slo_attainment",
               "mean_latency_s", "p50_latency_s", "p99_latency_s", "mean_ttft_s", "mean_running",
               "mean_waiting", "running_fraction", "avg_load", "load_skew", "running_skew",
               "waiting_skew", "mean_utility", "route_us_mean", "route_us_p50", "route_us_p99"]


class hwr_sim_result(C.Structure):
    _fields_ = ([("pair", _vp), ("utility", _vp), ("pred_e2e_s", _vp), ("first_token_us", _vp),
                 ("finish_us", _vp), ("max_samples", C.c_int32), ("samples", _vp), ("n_samples", C.c_int32)]
                + [(k, C.c_int64) for k in ("end_us", "n_completed", "n_met_slo", "route_calls")]
                + [(k, C.c_double) for k in SIM_METRICS[5:]])


hwr_sim_router_fn = C.CFUNCTYPE(C.c_int32, C.c_void_p, C.POINTER(hwr_hw_state), C.c_int32, C.c_int32,
                                C.c_int32, _i32p, _f32p, _f32p)
STATE_DTYPE = np.dtype([("running_q", "<i4"), ("waiting_q", "<i4"), ("kv_util", "<f4"),
                        ("gpu_util", "<f4"), ("ttft_avg_s", "<f4"), ("tpot_avg_s", "<f4")])


_lib = None


def load(path: Optional[str] = None) -> C.CDLL:
    """Load libhwr.so (in-tree).  Raises if it has not been built."""
    global _lib
    if _lib is not None and path is None:
        return _lib
    p = path or LIB_PATH
    if not os.path.exists(p):
        raise RuntimeError(f"libhwr.so not found at {p}: build it first "
                           "(python -m paper_2608_14575_amd.build); there is no fallback")
    # torch carries its own copy of the HIP runtime under the same soname as
    # the one the library is linked against.  Loaded first, that copy is the
    # one the library binds to; loaded after the library, it would be a
    # second runtime in the process, and the second to start finds no GPU.
    try:
        import torch  # noqa: F401
    except ImportError:
        pass
    L = C.CDLL(p)
    L.hwr_init.restype = C.c_int
    L.hwr_init.argtypes = [C.POINTER(hwr_config), C.POINTER(_vp)]
    L.hwr_update_hw_state.restype = C.c_int
    L.hwr_update_hw_state.argtypes = [_vp, _vp, C.c_int32]
    L.hwr_route_batch.restype = C.c_int
    L.hwr_route_batch.argtypes = [_vp, C.POINTER(hwr_query_batch), C.POINTER(hwr_route_result)]
    L.hwr_route_batch_static.restype = C.c_int
    L.hwr_route_batch_static.argtypes = [_vp, C.POINTER(hwr_query_batch), C.POINTER(hwr_route_result)]
    L.hwr_free.restype = None
    L.hwr_free.argtypes = [_vp]
    L.hwr_last_error.restype = C.c_char_p
    L.hwr_last_error.argtypes = [_vp]
    L.hwr_profile_enable.restype = C.c_int
    L.hwr_profile_enable.argtypes = [_vp, C.c_int32]
    L.hwr_profile_read.restype = C.c_int
    L.hwr_profile_read.argtypes = [_vp, C.POINTER(hwr_kernel_times), C.c_int32]
    L.hwr_sim_run.restype = C.c_int
    L.hwr_sim_run.argtypes = [_vp, C.POINTER(hwr_sim_config), C.POINTER(hwr_sim_requests),
                              hwr_sim_router_fn, _vp, C.POINTER(hwr_sim_result)]
    L.hwr_sim_last_error.restype = C.c_char_p
    L.hwr_sim_last_error.argtypes = []
    L.hwr_probe_mfma_bf16.restype = C.c_int
    L.hwr_probe_mfma_bf16.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_double),
                                      C.POINTER(C.c_double)]
    L.hwr_probe_hbm_read.restype = C.c_int
    L.hwr_probe_hbm_read.argtypes = [C.c_int32, _vp, C.c_uint64, C.c_int32, C.c_int32, C.POINTER(C.c_double)]
    L.hwr_probe_launch_floor.restype = C.c_int
    L.hwr_probe_launch_floor.argtypes = [C.c_int32, C.c_int32, C.c_int32, C.POINTER(C.c_double),
                                         C.POINTER(C.c_double)]
    L.hwr_probe_hbm_write.restype = C.c_int
    L.hwr_probe_hbm_write.argtypes = [C.c_int32, _vp, C.c_uint64, C.c_int32, C.c_int32, C.POINTER(C.c_double)]
    L.hwr_probe_feature_log.restype = C.c_int
    L.hwr_probe_feature_log.argtypes = [C.c_int32, _vp, C.c_int64, _vp]
    if path is None:
        _lib = L
    return L


def _check(status: int, ctx) -> None:
    if status != HWR_OK:
        raise HwrError(status, hwr_last_error(ctx))


# ---------------------------------------------------------------- the C ABI, 1:1
def hwr_init(cfg: hwr_config):
    ctx = _vp()
    st = load().hwr_init(C.byref(cfg), C.byref(ctx))
    _check(st, None)
    return ctx


def hwr_update_hw_state(ctx, state: np.ndarray) -> None:
    state = np.ascontiguousarray(state)
    assert state.dtype.itemsize == 24
    _check(load().hwr_update_hw_state(ctx, state.ctypes.data, int(state.shape[0])), ctx)


def hwr_route_batch(ctx, batch: hwr_query_batch, result: hwr_route_result) -> None:
    _check(load().hwr_route_batch(ctx, C.byref(batch), C.byref(result)), ctx)


def hwr_route_batch_static(ctx, batch: hwr_query_batch, result: hwr_route_result) -> None:
    _check(load().hwr_route_batch_static(ctx, C.byref(batch), C.byref(result)), ctx)


def hwr_probe_mfma_bf16(device: int, waves_per_simd: int, iters: int, reps: int) -> tuple:
    """Register-fed bf16 MFMA rate of the device in TFLOP/s and the shader
    clock in MHz it ran at (medians over the timed launches)."""
    out, mhz = C.c_double(), C.c_double()
    _check(load().hwr_probe_mfma_bf16(device, waves_per_simd, iters, reps, C.byref(out), C.byref(mhz)), None)
    return out.value, mhz.value


def hwr_probe_hbm_read(device: int, buf_ptr: int, nbytes: int, waves_per_simd: int, reps: int) -> float:
    """Streaming read rate in GB/s of nbytes of device memory at buf_ptr."""
    out = C.c_double()
    _check(load().hwr_probe_hbm_read(device, buf_ptr, nbytes, waves_per_simd, reps, C.byref(out)), None)
    return out.value


def hwr_probe_hbm_write(device: int, buf_ptr: int, nbytes: int, waves_per_simd: int, reps: int) -> float:
    """Streaming write rate in GB/s into nbytes of device memory at buf_ptr
    (overwritten)."""
    out = C.c_double()
    _check(load().hwr_probe_hbm_write(device, buf_ptr, nbytes, waves_per_simd, reps, C.byref(out)), None)
    return out.value


def hwr_probe_launch_floor(device: int, use_graph: bool, calls: int) -> tuple:
    """Host-clock p50 and p99 in µs of a launch of one wave answered through
    pinned host memory (plain or graph launch)."""
    p50, p99 = C.c_double(), C.c_double()
    _check(load().hwr_probe_launch_floor(device, int(use_graph), calls, C.byref(p50), C.byref(p99)), None)
    return p50.value, p99.value


def hwr_probe_feature_log(device: int, x: np.ndarray) -> np.ndarray:
    """ln(x) as the device's feature logarithm computes it (x: positive,
    finite, normal doubles)."""
    x = np.ascontiguousarray(x, np.float64)
    y = np.empty_like(x)
    _check(load().hwr_probe_feature_log(device, x.ctypes.data, x.size, y.ctypes.data), None)
    return y


def hwr_free(ctx) -> None:
    load().hwr_free(ctx)


def hwr_last_error(ctx) -> str:
    m = load().hwr_last_error(ctx)
    return m.decode() if m else ""


def hwr_profile_enable(ctx, enable) -> None:
    """enable: False / 0 off, True / 1 every launch, k > 1 one launch in k of each kernel."""
    _check(load().hwr_profile_enable(ctx, int(enable)), ctx)


def hwr_profile_read(ctx, reset: bool = True) -> dict:
    t = hwr_kernel_times()
    _check(load().hwr_profile_read(ctx, C.byref(t), 1 if reset else 0), ctx)
    return {KERNEL_NAMES[k]: (t.ms[k], int(t.launches[k])) for k in range(HWR_K_COUNT)}


# ---------------------------------------------------------------- convenience
def _ptr(a) -> int:
    if a is None:
        return 0
    if isinstance(a, np.ndarray):
        return a.ctypes.data
    return int(a.data_ptr())   # torch tensor


# element kinds of the buffers of a batch: accepted numpy dtypes / torch dtype names
_KINDS = {
    "i32": ({np.dtype(np.int32)}, {"torch.int32"}),
    "f32": ({np.dtype(np.float32)}, {"torch.float32"}),
    "u8": ({np.dtype(np.uint8)}, {"torch.uint8"}),
    "b16": ({np.dtype(np.uint16), np.dtype(np.int16)}, {"torch.int16", "torch.uint16", "torch.bfloat16"}),
}


def check_buffer(name: str, a, kind: str, count: int, mem: int, device: int = 0) -> None:
    """Raise HwrError(HWR_ERR_INVALID_ARG) unless ``a`` can hold ``count``
    elements of ``kind`` contiguously in the memory space ``mem``: a numpy
    array (or CPU tensor) for HWR_MEM_HOST, a tensor on GPU ``device`` for
    HWR_MEM_DEVICE.  The library reads and writes raw pointers, so a short,
    strided or misplaced buffer would otherwise reach the kernels."""
    def bad(msg):
        raise HwrError(HWR_ERR_INVALID_ARG, f"{name}: {msg}")
    np_kinds, torch_kinds = _KINDS[kind]
    if isinstance(a, np.ndarray):
        if mem == HWR_MEM_DEVICE:
            bad("a device batch needs device tensors, got a numpy array")
        if a.dtype not in np_kinds:
            bad(f"dtype {a.dtype} (expected {kind})")
        if not a.flags.c_contiguous:
            bad("not contiguous")
        size = a.size
    elif hasattr(a, "data_ptr") and hasattr(a, "is_contiguous"):
        dev = a.device
        if mem == HWR_MEM_DEVICE and (dev.type != "cuda" or (dev.index if dev.index is not None else 0) != device):
            bad(f"on {dev}, expected cuda:{device}")
        if mem == HWR_MEM_HOST and dev.type != "cpu":
            bad(f"on {dev}, a host batch needs host memory")
        if str(a.dtype) not in torch_kinds:
            bad(f"dtype {a.dtype} (expected {kind})")
        if not a.is_contiguous():
            bad("not contiguous")
        size = a.numel()
    else:
        bad(f"unsupported buffer type {type(a).__name__}")
    if size < count:
        bad(f"{size} elements, needs {count}")


def check_batch(*, n: int, D: int, M: int, N: int, K: int, dtype: str, n_heads: int, mem: int, device: int,
                emb, input_len, expected_out_len, slo_s, choice, feasible=None, utility=None, e2e_s=None,
                ttft_s=None, tpot_s=None, nout=None, cand_ttft=None, cand_tpot=None, cand_nout=None,
                cand_quality=None) -> None:
    """Every buffer of a route call checked against the context's shapes
    (D embedding width, M models, N pairs, K cost weights) before the call."""
    if mem not in (HWR_MEM_DEVICE, HWR_MEM_HOST):
        raise HwrError(HWR_ERR_INVALID_ARG, f"unknown mem {mem}")
    if n == 0:
        return
    check_buffer("emb", emb, "b16" if dtype == "bf16" else "f32", n * D, mem, device)
    check_buffer("input_len", input_len, "i32", n, mem, device)
    if expected_out_len is not None or n_heads == 2:
        check_buffer("expected_out_len", expected_out_len, "i32", n, mem, device)
    if slo_s is not None:
        check_buffer("slo_s", slo_s, "f32", n, mem, device)
    check_buffer("choice", choice, "i32", n * K, mem, device)
    for name, a, kind, count in (("feasible", feasible, "u8", n * K), ("utility", utility, "f32", n * K),
                                 ("e2e_s", e2e_s, "f32", n * K), ("ttft_s", ttft_s, "f32", n * K),
                                 ("tpot_s", tpot_s, "f32", n * K), ("nout", nout, "f32", n * K),
                                 ("cand_ttft", cand_ttft, "f32", n * N), ("cand_tpot", cand_tpot, "f32", n * N),
                                 ("cand_nout", cand_nout, "f32", n * N),
                                 ("cand_quality", cand_quality, "f32", n * M)):
        if a is not None:
            check_buffer(name, a, kind, count, mem, device)


class Router:
    """Owns one hwr context.  Arrays follow include/hwr.h: weights row-major
    ([D][M], [F][H], [H][H], [H][n_heads]) as uint16 bf16 bits (bf16) or
    float32."""

    def __init__(self, *, dep_model, dep_gpu, model_arch, model_params_b, wq, bq, w1, b1, w2, b2,
                 w3, b3, arch_width: int, gpu_width: int, n_gpu_types: int, dtype: str,
                 cost_weight: float = 0.5, default_slo_s: float = 1.0, pipeline: str = "fused",
                 max_chunk: int = 65536, stream: int = 0, flags: int = 0, device: int = 0,
                 n_heads: int = 2, score_mode: int = 0, bound_mode: int = 0, ttft_slo_a: float = 0.0,
                 ttft_slo_b: float = 0.0, tpot_slo: float = 0.0, cost_weights=None):
        wdt = np.uint16 if dtype == "bf16" else np.float32
        keep = dict(dep_model=np.ascontiguousarray(dep_model, np.int32),
                    dep_gpu=np.ascontiguousarray(dep_gpu, np.int32),
                    model_arch=np.ascontiguousarray(model_arch, np.int32),
                    model_params_b=np.ascontiguousarray(model_params_b, np.float32),
                    wq=np.ascontiguousarray(wq, wdt), bq=np.ascontiguousarray(bq, np.float32),
                    w1=np.ascontiguousarray(w1, wdt), b1=np.ascontiguousarray(b1, np.float32),
                    w2=np.ascontiguousarray(w2, wdt), b2=np.ascontiguousarray(b2, np.float32),
                    w3=np.ascontiguousarray(w3, wdt), b3=np.ascontiguousarray(b3, np.float32))
        D, M = keep["wq"].shape
        F, H = keep["w1"].shape
        N = keep["dep_model"].shape[0]
        if n_heads not in (2, 3) or keep["w3"].shape != (H, n_heads) or keep["b3"].shape != (n_heads,):
            raise ValueError(f"w3 must be [H][n_heads] and b3 [n_heads] with n_heads 2 or 3 "
                             f"(got {keep['w3'].shape}, {keep['b3'].shape}, n_heads={n_heads})")
        cfg = hwr_config()
        cfg.n_models, cfg.n_gpu_types, cfg.n_deployments = M, int(n_gpu_types), N
        cfg.arch_width, cfg.gpu_width = int(arch_width), int(gpu_width)
        cfg.embed_dim, cfg.feat_dim, cfg.hidden = D, F, H
        cfg.emb_dtype = cfg.weight_dtype = HWR_BF16 if dtype == "bf16" else HWR_F32
        cfg.pipeline = HWR_PIPE_STAGED if pipeline == "staged" else HWR_PIPE_FUSED
        cfg.max_chunk = int(max_chunk)
        cfg.cost_weight, cfg.default_slo_s = float(cost_weight), float(default_slo_s)
        cfg.device, cfg.flags, cfg.n_heads = int(device), int(flags), int(n_heads)
        cfg.score_mode, cfg.bound_mode = int(score_mode), int(bound_mode)
        cfg.ttft_slo_a, cfg.ttft_slo_b, cfg.tpot_slo = float(ttft_slo_a), float(ttft_slo_b), float(tpot_slo)
        if cost_weights is not None:
            keep["cost_weights"] = np.ascontiguousarray(cost_weights, np.float32).ravel()
            cfg.n_weights = int(keep["cost_weights"].size)
            cfg.cost_weights = keep["cost_weights"].ctypes.data_as(_f32p)
        for k in ("dep_model", "dep_gpu", "model_arch"):
            setattr(cfg, k, keep[k].ctypes.data_as(_i32p))
        for k in ("model_params_b", "bq", "b1", "b2", "b3"):
            setattr(cfg, k, keep[k].ctypes.data_as(_f32p))
        for k in ("wq", "w1", "w2", "w3"):
            setattr(cfg, k, keep[k].ctypes.data)
        cfg.stream = int(stream)
        self.M, self.N, self.D, self.dtype, self.n_heads = M, N, D, dtype, int(n_heads)
        self.device = int(device)
        self.n_weights = 1 if cost_weights is None else int(np.size(cost_weights))
        self.ctx = hwr_init(cfg)

    @classmethod
    def from_problem(cls, pb, **kw) -> "Router":
        """Build from a generator problem (paper_2608_14575_amd.synth.Problem)."""
        sp = pb.spec
        kw.setdefault("cost_weight", sp.cost_weight)
        kw.setdefault("default_slo_s", sp.slo_value)
        kw.setdefault("n_heads", sp.n_heads)
        for k in ("score_mode", "bound_mode", "ttft_slo_a", "ttft_slo_b", "tpot_slo"):
            kw.setdefault(k, getattr(sp, k))
        return cls(dep_model=pb.dep_model, dep_gpu=pb.dep_gpu, model_arch=pb.model_arch,
                   model_params_b=pb.model_params_b, wq=pb.wq_bits, bq=pb.bq, w1=pb.w1_bits,
                   b1=pb.b1, w2=pb.w2_bits, b2=pb.b2, w3=pb.w3_bits, b3=pb.b3,
                   arch_width=sp.arch_width, gpu_width=sp.gpu_width, n_gpu_types=sp.n_gpu_types,
                   dtype=sp.dtype, **kw)

    def close(self) -> None:
        if getattr(self, "ctx", None):
            hwr_free(self.ctx)
            self.ctx = None

    def __del__(self):
        try:
            self.close()
        except Exception:
            pass

    def update(self, state: np.ndarray) -> None:
        hwr_update_hw_state(self.ctx, state)

    def profile(self, enable=True) -> None:
        """Kernel timing: False off, True every launch, k > 1 one launch in k of each kernel."""
        hwr_profile_enable(self.ctx, enable)

    def profile_read(self, reset: bool = True) -> dict:
        return hwr_profile_read(self.ctx, reset)

    def route(self, emb, input_len, expected_out_len, slo_s=None, *, mem: int,
              choice, feasible=None, utility=None, e2e_s=None, ttft_s=None, tpot_s=None, nout=None,
              cand_ttft=None, cand_tpot=None, cand_nout=None, cand_quality=None, static: bool = False) -> None:
        """Route into caller-owned outputs (numpy for HWR_MEM_HOST, torch
        tensors on the device for HWR_MEM_DEVICE).  Every buffer is checked
        (kind, contiguity, memory space, size) before the library is called;
        a mismatch raises HwrError(HWR_ERR_INVALID_ARG).  ``static``: through
        hwr_route_batch_static (no allocation during the call; device
        batches only)."""
        n = int(input_len.shape[0])
        check_batch(n=n, D=self.D, M=self.M, N=self.N, K=self.n_weights, dtype=self.dtype,
                    n_heads=self.n_heads, mem=mem, device=self.device, emb=emb, input_len=input_len,
                    expected_out_len=expected_out_len, slo_s=slo_s, choice=choice, feasible=feasible,
                    utility=utility, e2e_s=e2e_s, ttft_s=ttft_s, tpot_s=tpot_s, nout=nout,
                    cand_ttft=cand_ttft, cand_tpot=cand_tpot, cand_nout=cand_nout, cand_quality=cand_quality)
        b = hwr_query_batch(n, mem, _ptr(emb), _ptr(input_len), _ptr(expected_out_len), _ptr(slo_s))
        r = hwr_route_result(_ptr(choice), _ptr(feasible), _ptr(utility), _ptr(e2e_s), _ptr(ttft_s),
                             _ptr(tpot_s), _ptr(nout), _ptr(cand_ttft), _ptr(cand_tpot), _ptr(cand_nout),
                             _ptr(cand_quality))
        (hwr_route_batch_static if static else hwr_route_batch)(self.ctx, b, r)

    def route_host(self, emb, input_len, expected_out_len, slo_s=None, candidates: bool = False) -> dict:
        """Route numpy inputs; returns numpy outputs (synchronous)."""
        n = int(np.shape(input_len)[0])
        wdt = np.uint16 if self.dtype == "bf16" else np.float32
        emb = np.ascontiguousarray(emb, wdt)
        il = np.ascontiguousarray(input_len, np.int32)
        no = None if expected_out_len is None else np.ascontiguousarray(expected_out_len, np.int32)
        slo = None if slo_s is None else np.ascontiguousarray(slo_s, np.float32)
        shape = (n,) if self.n_weights == 1 else (n, self.n_weights)   # [n][K] with K weights
        out = dict(choice=np.full(shape, -1, np.int32), feasible=np.zeros(shape, np.uint8),
                   utility=np.zeros(shape, np.float32), e2e_s=np.zeros(shape, np.float32),
                   ttft_s=np.zeros(shape, np.float32), tpot_s=np.zeros(shape, np.float32),
                   nout=np.zeros(shape, np.float32))
        if candidates:
            out.update(cand_ttft=np.zeros((n, self.N), np.float32),
                       cand_tpot=np.zeros((n, self.N), np.float32),
                       cand_quality=np.zeros((n, self.M), np.float32))
            if self.n_heads == 3:
                out["cand_nout"] = np.zeros((n, self.N), np.float32)
        self.route(emb, il, no, slo, mem=HWR_MEM_HOST, **out)
        return out


# ---------------------------------------------------------------- simulator
def simulate(ctx, *, pairs: np.ndarray, n_gpus: int, tick_us: int, monitor_period_us: int,
             max_time_us: int, prior_ttft_s, prior_tpot_s, arrival_us, input_len, output_len, slo_us,
             emb=None, emb_dtype: int = HWR_BF16, expected_out_len=None, route_slo_s=None,
             freeze_state: bool = False, router=None, max_samples: int = 0) -> dict:
    """hwr_sim_run (include/hwr_sim.h).  ``ctx``: a Router or an hwr context
    handle routes through the library; or ``router(snapshot, r0, r1)`` -- a
    Python callable given the cached snapshot (STATE_DTYPE [N]) that returns
    (choice, utility, e2e_s) for requests [r0, r1) -- with ctx None.  ``pairs``
    has the hwr_sim_pair layout (simload.PAIR_DTYPE).  Returns the per-request
    outputs, the stored snapshots and the metrics."""
    if isinstance(ctx, Router):
        ctx = ctx.ctx
    N = int(pairs.shape[0])
    R = int(np.shape(arrival_us)[0])
    keep = dict(pairs=np.ascontiguousarray(pairs), pt=np.ascontiguousarray(prior_ttft_s, np.float32),
                pp=np.ascontiguousarray(prior_tpot_s, np.float32),
                arr=np.ascontiguousarray(arrival_us, np.int64), il=np.ascontiguousarray(input_len, np.int32),
                ol=np.ascontiguousarray(output_len, np.int32), slo=np.ascontiguousarray(slo_us, np.int64))
    if keep["pairs"].dtype.itemsize != C.sizeof(hwr_sim_pair):
        raise ValueError("pairs must have the hwr_sim_pair layout")
    cfg = hwr_sim_config(N, int(n_gpus), keep["pairs"].ctypes.data, int(tick_us), int(monitor_period_us),
                         int(max_time_us), int(bool(freeze_state)), keep["pt"].ctypes.data,
                         keep["pp"].ctypes.data)
    req = hwr_sim_requests()
    req.n = R
    req.arrival_us, req.input_len = keep["arr"].ctypes.data, keep["il"].ctypes.data
    req.output_len, req.slo_us = keep["ol"].ctypes.data, keep["slo"].ctypes.data
    if emb is not None:
        keep["emb"] = np.ascontiguousarray(emb, np.uint16 if emb_dtype == HWR_BF16 else np.float32)
        req.emb, req.embed_dim, req.emb_dtype = keep["emb"].ctypes.data, int(keep["emb"].shape[1]), int(emb_dtype)
    if expected_out_len is not None:
        keep["no"] = np.ascontiguousarray(expected_out_len, np.int32)
        req.expected_out_len = keep["no"].ctypes.data
    if route_slo_s is not None:
        keep["rslo"] = np.ascontiguousarray(route_slo_s, np.float32)
        req.route_slo_s = keep["rslo"].ctypes.data
    out = dict(pair=np.full(R, -1, np.int32), utility=np.zeros(R, np.float32),
               pred_e2e_s=np.zeros(R, np.float32), first_token_us=np.full(R, -1, np.int64),
               finish_us=np.full(R, -1, np.int64), samples=np.zeros((max(max_samples, 0), N), STATE_DTYPE))
    res = hwr_sim_result()
    for k in ("pair", "utility", "pred_e2e_s", "first_token_us", "finish_us", "samples"):
        setattr(res, k, out[k].ctypes.data)
    res.max_samples = int(max_samples)
    errors = []

    def _cb(user, snap, n_pairs, r0, r1, choice, utility, e2e):
        try:
            st = np.ctypeslib.as_array(C.cast(snap, C.POINTER(C.c_uint8)), (n_pairs * 24,)).view(STATE_DTYPE).copy()
            ch, u, c = router(st, int(r0), int(r1))
            n = r1 - r0
            np.ctypeslib.as_array(choice, (n,))[:] = ch
            np.ctypeslib.as_array(utility, (n,))[:] = u
            np.ctypeslib.as_array(e2e, (n,))[:] = c
            return 0
        except Exception as ex:    # reported after the call returns
            errors.append(ex)
            return 1

    cb = hwr_sim_router_fn(_cb) if router is not None else hwr_sim_router_fn()
    st = load().hwr_sim_run(ctx, C.byref(cfg), C.byref(req), cb, None, C.byref(res))
    if errors:
        raise errors[0]
    if st != HWR_OK:
        raise HwrError(st, load().hwr_sim_last_error().decode())
    for k in SIM_METRICS:
        out[k] = getattr(res, k)
    out["samples"] = out["samples"][:min(res.n_samples, max(max_samples, 0))]
    return out
