"""The C ABI from plain C: tests/c_client/route_file.c links libhwr.so and
routes a host batch with hwr_init / hwr_update_hw_state / hwr_route_batch /
hwr_free alone (no Python, no torch in that process).  On the CPU it must
compile against include/hwr.h; on the GPU its decisions must pass the oracle
acceptance rule."""
import os
import subprocess

import numpy as np
import pytest

from oracle import oracle as O
from paper_2608_14575_amd import hwr
from paper_2608_14575_amd import synth as S

import parity

HERE = os.path.dirname(os.path.abspath(__file__))
ROOT = os.path.dirname(HERE)
SRC = os.path.join(HERE, "c_client", "route_file.c")
PKG = os.path.dirname(hwr.LIB_PATH)


def build_client(tmp_path) -> str:
    if not os.path.exists(hwr.LIB_PATH):
        from paper_2608_14575_amd import build
        build.build()
    exe = str(tmp_path / "route_file")
    subprocess.check_call(["gcc", "-std=c11", "-Wall", "-Wextra", "-Werror", "-O2",
                           f"-I{os.path.join(ROOT, 'include')}", SRC, f"-L{PKG}", "-lhwr",
                           f"-Wl,-rpath,{PKG}", "-o", exe])
    return exe


def test_client_compiles_against_the_header(tmp_path):
    exe = build_client(tmp_path)
    assert os.path.exists(exe)
    r = subprocess.run([exe], capture_output=True, text=True)
    assert r.returncode == 2 and "usage" in r.stderr


def write_input(path, sp, pb, st, qs, pipeline: int):
    i32 = lambda a: np.ascontiguousarray(a, np.int32).tobytes()
    f32 = lambda a: np.ascontiguousarray(a, np.float32).tobytes()
    u16 = lambda a: np.ascontiguousarray(a, np.uint16).tobytes()
    hdr = [sp.n_models, sp.n_gpu_types, pb.n_deployments, sp.arch_width, sp.gpu_width, sp.embed_dim,
           sp.feat_dim, sp.hidden, qs.n, pipeline]
    with open(path, "wb") as f:
        f.write(i32(hdr))
        f.write(f32([sp.cost_weight, sp.slo_value]))
        for part in (i32(pb.dep_model), i32(pb.dep_gpu), i32(pb.model_arch), f32(pb.model_params_b),
                     u16(pb.wq_bits), f32(pb.bq), u16(pb.w1_bits), f32(pb.b1), u16(pb.w2_bits), f32(pb.b2),
                     u16(pb.w3_bits), f32(pb.b3), np.ascontiguousarray(st).tobytes(),
                     u16(qs.emb_bits), i32(qs.input_len), i32(qs.expected_out_len), f32(qs.slo_s)):
            f.write(part)


@pytest.mark.gpu
@pytest.mark.parametrize("pipeline,n", [(hwr.HWR_PIPE_FUSED, 3000), (hwr.HWR_PIPE_STAGED, 700), (hwr.HWR_PIPE_FUSED, 1)])
def test_c_client_routes_like_the_oracle(tmp_path, pipeline, n):
    sp = S.spec("C2", n_queries=n)
    pb, st, qs = S.make_problem(sp, 31), S.make_state(sp, 31), S.make_queries(sp, 31)
    exe = build_client(tmp_path)
    fin, fout = str(tmp_path / "in.bin"), str(tmp_path / "out.bin")
    write_input(fin, sp, pb, st, qs, pipeline)
    r = subprocess.run([exe, fin, fout], capture_output=True, text=True, timeout=120)
    assert r.returncode == 0, r.stderr
    raw = open(fout, "rb").read()
    choice = np.frombuffer(raw, np.int32, n, 0)
    feasible = np.frombuffer(raw, np.uint8, n, 4 * n)
    vals = np.frombuffer(raw, np.float32, 4 * n, 5 * n).reshape(4, n)
    got = dict(choice=choice, feasible=feasible, utility=vals[0], e2e_s=vals[1], ttft_s=vals[2], tpot_s=vals[3])
    orc = O.route_synth(pb, st, qs, candidates=True)
    rep = parity.compare(got, orc, slo=qs.slo_s, alpha=sp.cost_weight, dep_model=pb.dep_model, rtol=1e-2)
    print(f"C client ({'staged' if pipeline else 'fused'}, n={n}): {rep.summary()}", flush=True)
    assert rep.ok, rep.failures[:5]
