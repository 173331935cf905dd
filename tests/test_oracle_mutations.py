"""The oracle pins must catch plausible mistakes: each case plants one mistake
in a temporary copy of the oracle source (CPU only), rebuilds it, and expects
the pin suite to fail against it."""
import os
import shutil
import subprocess
import sys

import pytest

ROOT = os.path.dirname(os.path.dirname(os.path.abspath(__file__)))
SRC = os.path.join(ROOT, "oracle", "hwr_oracle.c")

MUTATIONS = {
    "swap_running_waiting": (
        "x[b + 2] = store(p, log(1.0 + (double)s->running_q[d]) / 2.0);\n"
        "    x[b + 3] = store(p, log(1.0 + (double)s->waiting_q[d]) / 2.0);",
        "x[b + 3] = store(p, log(1.0 + (double)s->running_q[d]) / 2.0);\n"
        "    x[b + 2] = store(p, log(1.0 + (double)s->waiting_q[d]) / 2.0);"),
    "input_len_scale": ("log((double)input_len) / 8.0", "log((double)input_len) / 4.0"),
    "w2_transposed": ("p->w2[(size_t)i * H + j]", "p->w2[(size_t)j * H + i]"),
    "dropped_b2": ("float a = (float)(acc + (double)p->b2[j]);", "float a = (float)(acc);"),
    "no_second_relu": ("h2[j] = store(p, a > 0.0f ? a : 0.0f);", "h2[j] = store(p, a);"),
    "w3_heads_swapped": ("p->w3[(size_t)i * NH + k]", "p->w3[(size_t)i * NH + (k < 2 ? 1 - k : k)]"),
    "w3_row_stride_two": ("p->w3[(size_t)i * NH + k]", "p->w3[(size_t)i * 2 + k]"),
    "nout_head_ignored": ("NH == 3 ? orc_softplus(z[2]) : nout_given", "NH == 3 ? (float)q->expected_out_len[iq] : nout_given"),
    "nout_from_tpot_head": ("NH == 3 ? orc_softplus(z[2]) : nout_given", "NH == 3 ? orc_softplus(z[1]) : nout_given"),
    "cost_without_nout": ("fmaf(tpot, nout, ttft)", "(tpot + ttft)"),
    "strict_bound": ("(c <= bound)", "(c < bound)"),
    "utility_sign": ("u = q - at;", "u = q + at;"),
    "ties_to_highest": ("(feas == best_f && u > best_u)", "(feas == best_f && u >= best_u)"),
    "bound_ignored": ("feas > best_f || ", ""),
    "wq_transposed": ("p->wq[(size_t)k * p->M + m]", "p->wq[(size_t)m * p->D + k]"),
    "gpu_onehot_offset": ("x[A + p->dep_gpu[d]] = 1.0f;", "x[p->dep_gpu[d]] = 1.0f;"),
    "bf16_truncates": (
        "if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u))) kept += 1u;", ""),
    "softplus_sign": ("log1p(exp(-fabs(v)))", "log1p(exp(fabs(v)))"),
    "wrong_model_of_pair": ("qual[p->dep_model[d]]", "qual[d % M]"),
    "decide_cost_terms_swapped": ("fmaf(cand_tpot[ci], nout, cand_ttft[ci])", "fmaf(cand_ttft[ci], nout, cand_tpot[ci])"),
    "paper_score_sign": ("u = wq - wc;", "u = wq + wc;"),
    "paper_score_weights_swapped": ("const float w1 = 1.0f - r->w;", "const float w1 = r->w;"),
    "paper_bound_drops_slope": ("fmaf(r->ttft_slo_b, (float)input_len, r->ttft_slo_a)", "r->ttft_slo_a"),
    "paper_bound_drops_nout": ("return fmaf(nout, r->tpot_slo, base);", "return base + r->tpot_slo;"),
    "decide_model_of_pair": ("quality[(size_t)iq * M + dep_model[d]]", "quality[(size_t)iq * M + d % M]"),
}


@pytest.mark.parametrize("name", sorted(MUTATIONS))
def test_pins_catch_planted_mistake(name, tmp_path):
    src = open(SRC).read()
    a, b = MUTATIONS[name]
    assert a in src, "mutation anchor no longer in the oracle source"
    (tmp_path / "hwr_oracle.c").write_text(src.replace(a, b))
    shutil.copy(os.path.join(ROOT, "oracle", "hwr_oracle.h"), tmp_path / "hwr_oracle.h")
    so = tmp_path / "liboracle.so"
    subprocess.check_call(["gcc", "-O2", "-std=c11", "-fPIC", "-shared", "-ffp-contract=off",
                           "-o", str(so), str(tmp_path / "hwr_oracle.c"), "-lm"])
    env = dict(os.environ, ORACLE_LIB_OVERRIDE=str(so))
    r = subprocess.run([sys.executable, "-m", "pytest", os.path.join(ROOT, "tests", "test_oracle_pins.py"),
                        "-q", "-x", "-p", "no:cacheprovider"], env=env, cwd=ROOT,
                       capture_output=True, text=True, timeout=300)
    assert r.returncode != 0, f"planted mistake {name!r} passed every pin:\n{r.stdout[-2000:]}"
