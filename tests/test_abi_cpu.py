"""C-ABI contract checks that need no GPU: the library loads and exports every
function include/*.h declares, the ctypes structures match the C layout,
and argument errors come back as status codes (no device touched)."""
import ctypes as C
import glob
import os
import re
import subprocess

import numpy as np
import pytest

from paper_2608_14575_amd import hwr

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
HEADERS = sorted(glob.glob(os.path.join(ROOT, "include", "*.h")))


@pytest.fixture(scope="module")
def lib():
    if not os.path.exists(hwr.LIB_PATH):
        from paper_2608_14575_amd import build
        build.build()
    return hwr.load()


def _declared():
    names = set()
    for h in HEADERS:
        txt = open(h).read()
        names |= set(re.findall(r"^\s*(?:hwr_status|void|const char \*)\s*(hwr_\w+)\s*\(", txt, re.M))
    return sorted(names)


def test_every_declared_symbol_is_exported(lib):
    names = _declared()
    assert set(names) == set(hwr.EXPORTS), names
    out = subprocess.run(["nm", "-D", "--defined-only", hwr.LIB_PATH], capture_output=True,
                         text=True, check=True).stdout
    exported = set(re.findall(r"\bT (hwr_\w+)", out))
    for n in names:
        assert n in exported, n
        assert hasattr(lib, n)


def test_constants_match_header(tmp_path):
    """Every HWR_ enumerator and macro of include/*.h, as the C compiler sees
    it, has a binding constant of the same name and value."""
    names = set()
    for h in HEADERS:
        txt = open(h).read()
        names |= set(re.findall(r"^#define (HWR_[A-Z0-9_]+)\s+\S", txt, re.M))
        for body in re.findall(r"enum\s*(?:\w+\s*)?\{(.*?)\}", txt, re.S):
            names |= set(re.findall(r"\b(HWR_[A-Z0-9_]+)\s*(?:=|,|$)", body, re.M))
    names.discard("HWR_H")
    names = {n for n in names if not n.endswith("_H")}
    assert len(names) > 20, names
    src = ['#include <stdio.h>', '#include "hwr.h"', '#include "hwr_sim.h"', "int main(void) {"]
    src += [f'printf("{n} %lld\\n", (long long)({n}));' for n in sorted(names)]
    src.append("return 0; }")
    c = tmp_path / "consts.c"
    c.write_text("\n".join(src))
    exe = tmp_path / "consts"
    subprocess.check_call(["gcc", "-std=c11", f"-I{os.path.join(ROOT, 'include')}", str(c), "-o", str(exe)])
    got = dict(line.split() for line in subprocess.check_output([str(exe)], text=True).splitlines())
    missing = sorted(n for n in names if not hasattr(hwr, n))
    assert not missing, missing
    for n, v in got.items():
        assert getattr(hwr, n) == int(v), (n, getattr(hwr, n), v)


def test_struct_layout_matches_header(tmp_path):
    """offsetof / sizeof from the C compiler against the ctypes mirror."""
    fields = {
        "hwr_hw_state": [f for f, _ in hwr.hwr_hw_state._fields_],
        "hwr_config": [f for f, _ in hwr.hwr_config._fields_],
        "hwr_query_batch": [f for f, _ in hwr.hwr_query_batch._fields_],
        "hwr_route_result": [f for f, _ in hwr.hwr_route_result._fields_],
        "hwr_kernel_times": [f for f, _ in hwr.hwr_kernel_times._fields_],
        "hwr_sim_pair": [f for f, _ in hwr.hwr_sim_pair._fields_],
        "hwr_sim_config": [f for f, _ in hwr.hwr_sim_config._fields_],
        "hwr_sim_requests": [f for f, _ in hwr.hwr_sim_requests._fields_],
        "hwr_sim_result": [f for f, _ in hwr.hwr_sim_result._fields_],
    }
    src = ['#include <stdio.h>', '#include <stddef.h>', '#include "hwr.h"', '#include "hwr_sim.h"',
           "int main(void) {"]
    for s, fl in fields.items():
        src.append(f'printf("{s} sizeof %zu\\n", sizeof({s}));')
        for f in fl:
            src.append(f'printf("{s} {f} %zu\\n", offsetof({s}, {f}));')
    src.append("return 0; }")
    c = tmp_path / "layout.c"
    c.write_text("\n".join(src))
    exe = tmp_path / "layout"
    subprocess.check_call(["gcc", "-std=c11", f"-I{os.path.join(ROOT, 'include')}", str(c), "-o", str(exe)])
    got = {}
    for line in subprocess.check_output([str(exe)], text=True).splitlines():
        s, f, v = line.split()
        got[(s, f)] = int(v)
    for s, fl in fields.items():
        cls = getattr(hwr, s)
        assert got[(s, "sizeof")] == C.sizeof(cls), s
        for f in fl:
            assert got[(s, f)] == getattr(cls, f).offset, (s, f)
    assert got[("hwr_hw_state", "sizeof")] == 24


def _valid_cfg(keep):
    M, G, N, D, F, H = 2, 2, 4, 64, 24, 64
    keep.update(dep_model=np.array([0, 0, 1, 1], np.int32), dep_gpu=np.array([0, 1, 0, 1], np.int32),
                arch=np.array([0, 1], np.int32), params=np.array([7.0, 14.0], np.float32),
                wq=np.zeros((D, M), np.uint16), bq=np.zeros(M, np.float32),
                w1=np.zeros((F, H), np.uint16), w2=np.zeros((H, H), np.uint16),
                w3=np.zeros((H, 2), np.uint16), b=np.zeros(H, np.float32), b3=np.zeros(2, np.float32))
    cfg = hwr.hwr_config()
    cfg.n_models, cfg.n_gpu_types, cfg.n_deployments = M, G, N
    cfg.arch_width, cfg.gpu_width, cfg.embed_dim, cfg.feat_dim, cfg.hidden = 4, 3, D, F, H
    cfg.emb_dtype = cfg.weight_dtype = hwr.HWR_BF16
    cfg.cost_weight, cfg.default_slo_s = 0.5, 1.5
    i32 = C.POINTER(C.c_int32)
    f32 = C.POINTER(C.c_float)
    cfg.dep_model = keep["dep_model"].ctypes.data_as(i32)
    cfg.dep_gpu = keep["dep_gpu"].ctypes.data_as(i32)
    cfg.model_arch = keep["arch"].ctypes.data_as(i32)
    cfg.model_params_b = keep["params"].ctypes.data_as(f32)
    cfg.wq, cfg.w1, cfg.w2, cfg.w3 = (keep[k].ctypes.data for k in ("wq", "w1", "w2", "w3"))
    cfg.bq = keep["bq"].ctypes.data_as(f32)
    cfg.b1 = cfg.b2 = keep["b"].ctypes.data_as(f32)
    cfg.b3 = keep["b3"].ctypes.data_as(f32)
    return cfg


@pytest.mark.parametrize("mutate,status", [
    (lambda c, k: setattr(c, "n_deployments", 0), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: k["dep_model"].__setitem__(2, 5), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: k["dep_gpu"].__setitem__(0, -1), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: k["arch"].__setitem__(1, 4), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: k["params"].__setitem__(0, 0.0), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: setattr(c, "feat_dim", 14), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: setattr(c, "default_slo_s", float("nan")), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: setattr(c, "cost_weight", -1.0), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: setattr(c, "w2", None), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: setattr(c, "hidden", 96), hwr.HWR_ERR_UNSUPPORTED),
    (lambda c, k: setattr(c, "embed_dim", 100), hwr.HWR_ERR_UNSUPPORTED),
    (lambda c, k: setattr(c, "feat_dim", 40), hwr.HWR_ERR_UNSUPPORTED),
    (lambda c, k: setattr(c, "emb_dtype", hwr.HWR_F32), hwr.HWR_ERR_UNSUPPORTED),
    (lambda c, k: setattr(c, "n_heads", 4), hwr.HWR_ERR_INVALID_ARG),
    (lambda c, k: setattr(c, "n_heads", 1), hwr.HWR_ERR_INVALID_ARG),
])
def test_config_errors_are_status_codes(lib, mutate, status):
    keep = {}
    cfg = _valid_cfg(keep)
    mutate(cfg, keep)
    ctx = C.c_void_p()
    st = lib.hwr_init(C.byref(cfg), C.byref(ctx))
    assert st == status
    assert not ctx.value
    assert lib.hwr_last_error(None)


def test_null_arguments(lib):
    ctx = C.c_void_p()
    assert lib.hwr_init(None, C.byref(ctx)) == hwr.HWR_ERR_INVALID_ARG
    assert lib.hwr_update_hw_state(None, None, 0) == hwr.HWR_ERR_INVALID_ARG
    assert lib.hwr_route_batch(None, None, None) == hwr.HWR_ERR_INVALID_ARG
    assert lib.hwr_route_batch_static(None, None, None) == hwr.HWR_ERR_INVALID_ARG
    assert lib.hwr_profile_enable(None, 1) == hwr.HWR_ERR_INVALID_ARG
    lib.hwr_free(None)


def test_probe_argument_errors(lib):
    """The ceiling probes reject bad arguments before touching a device."""
    out = C.c_double(-1.0)
    bad_mfma = [(0, 1, 16, 3, None, None), (-1, 1, 16, 3, C.byref(out), None),
                (0, 0, 16, 3, C.byref(out), None), (0, 3, 16, 3, C.byref(out), None),
                (0, 1, 0, 3, C.byref(out), None), (0, 1, 16, 0, C.byref(out), None),
                (0, 1, 16, 65, C.byref(out), None)]
    for args in bad_mfma:
        assert lib.hwr_probe_mfma_bf16(*args) == hwr.HWR_ERR_INVALID_ARG, args
    buf = 1 << 20    # never dereferenced: every call below fails its checks first
    bad_read = [(0, None, 1 << 20, 2, 3, C.byref(out)), (0, buf, 0, 2, 3, C.byref(out)),
                (0, buf, 1000, 2, 3, C.byref(out)), (0, buf + 8, 1 << 20, 2, 3, C.byref(out)),
                (0, buf, 1 << 20, 0, 3, C.byref(out)), (0, buf, 1 << 20, 9, 3, C.byref(out)),
                (0, buf, 1 << 20, 2, 0, C.byref(out)), (0, buf, 1 << 20, 2, 3, None),
                (-1, buf, 1 << 20, 2, 3, C.byref(out))]
    for args in bad_read:
        assert lib.hwr_probe_hbm_read(*args) == hwr.HWR_ERR_INVALID_ARG, args
        assert lib.hwr_probe_hbm_write(*args) == hwr.HWR_ERR_INVALID_ARG, args
    p99 = C.c_double(-1.0)
    for args in [(0, 0, 10, None, C.byref(p99)), (0, 0, 10, C.byref(out), None), (-1, 0, 10, C.byref(out), C.byref(p99)),
                 (0, 2, 10, C.byref(out), C.byref(p99)), (0, 0, 0, C.byref(out), C.byref(p99)),
                 (0, 1, 100001, C.byref(out), C.byref(p99))]:
        assert lib.hwr_probe_launch_floor(*args) == hwr.HWR_ERR_INVALID_ARG, args
    assert out.value == -1.0 and p99.value == -1.0
    # the feature logarithm: every argument checked on the host first
    x = np.array([2.0, 3.0], np.float64)
    y = np.full(2, -7.0)
    for args in [(0, None, 2, y.ctypes.data), (0, x.ctypes.data, 2, None), (-1, x.ctypes.data, 2, y.ctypes.data),
                 (0, x.ctypes.data, 0, y.ctypes.data), (0, x.ctypes.data, (1 << 26) + 1, y.ctypes.data)]:
        assert lib.hwr_probe_feature_log(*args) == hwr.HWR_ERR_INVALID_ARG, args
    for bad in (0.0, -1.0, np.inf, np.nan, 1e-310):     # outside: positive, finite, normal
        xb = np.array([2.0, bad], np.float64)
        assert lib.hwr_probe_feature_log(0, xb.ctypes.data, 2, y.ctypes.data) == hwr.HWR_ERR_INVALID_ARG, bad
    assert (y == -7.0).all()


def test_no_device_is_a_clean_error(lib):
    import torch
    if torch.cuda.is_available():
        pytest.skip("a device is present")
    keep = {}
    cfg = _valid_cfg(keep)
    ctx = C.c_void_p()
    assert lib.hwr_init(C.byref(cfg), C.byref(ctx)) == hwr.HWR_ERR_HIP
    assert b"device" in lib.hwr_last_error(None)


def test_binding_fails_loudly_without_library(tmp_path):
    with pytest.raises(RuntimeError, match="no fallback"):
        hwr.load(str(tmp_path / "missing.so"))


def test_router_checks_head_shapes():
    """The binding refuses W3 / b3 whose shapes disagree with n_heads (the
    library reads H x n_heads weights)."""
    from paper_2608_14575_amd import synth as S
    pb = S.make_problem(S.spec("C2", n_queries=4), 1)
    with pytest.raises(ValueError):
        hwr.Router.from_problem(pb, n_heads=3)
