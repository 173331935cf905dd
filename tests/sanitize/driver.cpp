// Host-only test driver built with AddressSanitizer and UndefinedBehaviour-
// Sanitizer (tests/test_sanitizers_cpu.py builds and runs it): the CPU oracle
// (oracle/hwr_oracle.c) over a whole routing problem, and the closed-loop
// simulator (paper_2608_14575_amd/csrc/hwr_sim.cpp) with the oracle as its
// router callback.  It reads raw little-endian arrays from a directory and
// writes its outputs there; the test compares them with the unsanitized
// builds bit for bit.  Any sanitizer report aborts the run (nonzero exit).
//
//   driver route <dir>     oracle: orc_route with every per-candidate output,
//                          orc_decide on its predictions, bf16 and softplus sweeps
//   driver sim <dir>       hwr_sim_run with the oracle routing each step
#include <cstdint>
#include <cstdio>
#include <cstdlib>
#include <map>
#include <string>
#include <vector>

#include "hwr_oracle.h"
#include "hwr_sim.h"

// The simulator's library mode is not exercised here (it needs a device
// context); these stand-ins satisfy the link and fail if ever called.
extern "C" hwr_status hwr_update_hw_state(hwr_ctx *, const hwr_hw_state *, int32_t) { return HWR_ERR_UNSUPPORTED; }
extern "C" hwr_status hwr_route_batch(hwr_ctx *, const hwr_query_batch *, hwr_route_result *) { return HWR_ERR_UNSUPPORTED; }
extern "C" const char *hwr_last_error(const hwr_ctx *) { return "no library context in the sanitizer driver"; }

namespace {

std::string g_dir;

template <class T>
std::vector<T> load(const std::string &name) {
    const std::string path = g_dir + "/" + name;
    FILE *f = std::fopen(path.c_str(), "rb");
    if (!f) { std::fprintf(stderr, "missing %s\n", path.c_str()); std::exit(2); }
    std::fseek(f, 0, SEEK_END);
    const long bytes = std::ftell(f);
    std::fseek(f, 0, SEEK_SET);
    std::vector<T> v(static_cast<size_t>(bytes) / sizeof(T));
    if (!v.empty() && std::fread(v.data(), sizeof(T), v.size(), f) != v.size()) std::exit(2);
    std::fclose(f);
    return v;
}

template <class T>
void save(const std::string &name, const std::vector<T> &v) {
    const std::string path = g_dir + "/" + name;
    FILE *f = std::fopen(path.c_str(), "wb");
    if (!f || (!v.empty() && std::fwrite(v.data(), sizeof(T), v.size(), f) != v.size())) std::exit(3);
    std::fclose(f);
}

std::map<std::string, double> meta() {
    std::map<std::string, double> m;
    FILE *f = std::fopen((g_dir + "/meta.txt").c_str(), "r");
    if (!f) std::exit(2);
    char key[64];
    double val;
    while (std::fscanf(f, "%63s %lf", key, &val) == 2) m[key] = val;
    std::fclose(f);
    return m;
}

// The routing problem and its arrays (kept alive for the pointers).
struct Problem {
    std::vector<int32_t> dep_model, dep_gpu, model_arch;
    std::vector<float> params, wq, bq, w1, b1, w2, b2, w3, b3;
    orc_problem p{};
};

void load_problem(Problem &P, std::map<std::string, double> &m) {
    P.dep_model = load<int32_t>("dep_model.bin");
    P.dep_gpu = load<int32_t>("dep_gpu.bin");
    P.model_arch = load<int32_t>("model_arch.bin");
    P.params = load<float>("model_params_b.bin");
    P.wq = load<float>("wq.bin");
    P.bq = load<float>("bq.bin");
    P.w1 = load<float>("w1.bin");
    P.b1 = load<float>("b1.bin");
    P.w2 = load<float>("w2.bin");
    P.b2 = load<float>("b2.bin");
    P.w3 = load<float>("w3.bin");
    P.b3 = load<float>("b3.bin");
    orc_problem &p = P.p;
    p.M = static_cast<int32_t>(m["M"]);
    p.G = static_cast<int32_t>(m["G"]);
    p.N = static_cast<int32_t>(m["N"]);
    p.D = static_cast<int32_t>(m["D"]);
    p.F = static_cast<int32_t>(m["F"]);
    p.H = static_cast<int32_t>(m["H"]);
    p.arch_width = static_cast<int32_t>(m["arch_width"]);
    p.gpu_width = static_cast<int32_t>(m["gpu_width"]);
    p.bf16 = static_cast<int32_t>(m["bf16"]);
    p.n_heads = static_cast<int32_t>(m["n_heads"]);
    p.alpha = static_cast<float>(m["alpha"]);
    p.score_mode = static_cast<int32_t>(m["score_mode"]);
    p.bound_mode = static_cast<int32_t>(m["bound_mode"]);
    p.ttft_slo_a = static_cast<float>(m["ttft_slo_a"]);
    p.ttft_slo_b = static_cast<float>(m["ttft_slo_b"]);
    p.tpot_slo = static_cast<float>(m["tpot_slo"]);
    p.dep_model = P.dep_model.data();
    p.dep_gpu = P.dep_gpu.data();
    p.model_arch = P.model_arch.data();
    p.model_params_b = P.params.data();
    p.wq = P.wq.data();
    p.bq = P.bq.data();
    p.w1 = P.w1.data();
    p.b1 = P.b1.data();
    p.w2 = P.w2.data();
    p.b2 = P.b2.data();
    p.w3 = P.w3.data();
    p.b3 = P.b3.data();
}

int run_route() {
    auto m = meta();
    Problem P;
    load_problem(P, m);
    const orc_problem &p = P.p;
    auto running = load<int32_t>("running_q.bin"), waiting = load<int32_t>("waiting_q.bin");
    auto kv = load<float>("kv_util.bin"), gu = load<float>("gpu_util.bin");
    auto tt = load<float>("ttft_avg_s.bin"), tp = load<float>("tpot_avg_s.bin");
    const orc_state s{running.data(), waiting.data(), kv.data(), gu.data(), tt.data(), tp.data()};
    auto emb = load<float>("emb.bin");
    auto il = load<int32_t>("input_len.bin"), no = load<int32_t>("expected_out_len.bin");
    auto slo = load<float>("slo_s.bin");
    const int32_t n = static_cast<int32_t>(il.size()), N = p.N, M = p.M, NH = p.n_heads;
    const orc_queries q{n, emb.data(), il.data(), no.data(), slo.data()};
    std::vector<int32_t> choice(n);
    std::vector<uint8_t> feas(n), cfeas(static_cast<size_t>(n) * N);
    std::vector<float> u(n), e2e(n), ttft(n), tpot(n), nout(n), cz(static_cast<size_t>(n) * N * NH);
    std::vector<float> cn(static_cast<size_t>(n) * N), ctt(cn.size()), ctp(cn.size()), ce(cn.size()),
        cu(cn.size()), cb(cn.size()), qual(static_cast<size_t>(n) * M);
    orc_result r{choice.data(), feas.data(), u.data(), e2e.data(), ttft.data(), tpot.data(), nout.data(),
                 cz.data(), cn.data(), ctt.data(), ctp.data(), ce.data(), cu.data(), cb.data(), cfeas.data(),
                 qual.data()};
    if (orc_route(&p, &s, &q, &r) != 0) return 4;
    save("out_choice.bin", choice);
    save("out_feasible.bin", feas);
    save("out_utility.bin", u);
    save("out_e2e.bin", e2e);
    save("out_cand_z.bin", cz);
    save("out_cand_ttft.bin", ctt);
    save("out_cand_tpot.bin", ctp);
    save("out_cand_u.bin", cu);
    save("out_quality.bin", qual);
    // the decision step alone on the oracle's own predictions
    const orc_rule rule{p.score_mode, p.bound_mode, p.alpha, p.ttft_slo_a, p.ttft_slo_b, p.tpot_slo};
    std::vector<int32_t> dch(n);
    std::vector<uint8_t> dfe(n);
    std::vector<float> du(n), de(n);
    if (orc_decide(n, N, M, p.dep_model, ctt.data(), ctp.data(), NH == 3 ? cn.data() : nullptr, qual.data(),
                   il.data(), no.data(), slo.data(), &rule, dch.data(), dfe.data(), du.data(), de.data()) != 0)
        return 5;
    save("dec_choice.bin", dch);
    save("dec_utility.bin", du);
    // element functions over sweeps (ties, subnormals, infinities included)
    auto sweep = load<float>("sweep.bin");
    std::vector<float> sb(sweep.size()), ss(sweep.size());
    orc_bf16_n(sweep.data(), sb.data(), static_cast<int64_t>(sweep.size()));
    for (size_t i = 0; i < sweep.size(); ++i) ss[i] = orc_softplus(sweep[i]);
    save("out_bf16.bin", sb);
    save("out_softplus.bin", ss);
    return 0;
}

struct SimRouter {
    const orc_problem *p;
    const std::vector<float> *emb;
    const std::vector<int32_t> *il, *no;
    const std::vector<float> *slo;
};

int32_t sim_route(void *user, const hwr_hw_state *snap, int32_t n_pairs, int32_t r0, int32_t r1,
                  int32_t *choice, float *utility, float *e2e_s) {
    const SimRouter &R = *static_cast<const SimRouter *>(user);
    std::vector<int32_t> run(n_pairs), wai(n_pairs);
    std::vector<float> kv(n_pairs), gu(n_pairs), tt(n_pairs), tp(n_pairs);
    for (int d = 0; d < n_pairs; ++d) {
        run[d] = snap[d].running_q;
        wai[d] = snap[d].waiting_q;
        kv[d] = snap[d].kv_util;
        gu[d] = snap[d].gpu_util;
        tt[d] = snap[d].ttft_avg_s;
        tp[d] = snap[d].tpot_avg_s;
    }
    const orc_state s{run.data(), wai.data(), kv.data(), gu.data(), tt.data(), tp.data()};
    const int32_t n = r1 - r0;
    const orc_queries q{n, R.emb->data() + static_cast<size_t>(r0) * R.p->D, R.il->data() + r0,
                        R.no->data() + r0, R.slo->data() + r0};
    orc_result r{};
    r.choice = choice;
    r.utility = utility;
    r.e2e_s = e2e_s;
    return orc_route(R.p, &s, &q, &r) == 0 ? 0 : 1;
}

int run_sim() {
    auto m = meta();
    Problem P;
    load_problem(P, m);
    auto pairs = load<hwr_sim_pair>("pairs.bin");
    auto pt = load<float>("prior_ttft_s.bin"), pp = load<float>("prior_tpot_s.bin");
    auto arr = load<int64_t>("arrival_us.bin");
    auto il = load<int32_t>("input_len.bin"), ol = load<int32_t>("output_len.bin");
    auto slo_us = load<int64_t>("slo_us.bin");
    auto emb = load<float>("emb.bin");
    auto no = load<int32_t>("expected_out_len.bin");
    auto rslo = load<float>("route_slo_s.bin");
    const int32_t R = static_cast<int32_t>(arr.size()), N = static_cast<int32_t>(pairs.size());
    const hwr_sim_config cfg{N, static_cast<int32_t>(m["n_gpus"]), pairs.data(), static_cast<int32_t>(m["tick_us"]),
                             static_cast<int32_t>(m["monitor_period_us"]), static_cast<int64_t>(m["max_time_us"]),
                             static_cast<int32_t>(m["freeze_state"]), pt.data(), pp.data()};
    hwr_sim_requests rq{};
    rq.n = R;
    rq.arrival_us = arr.data();
    rq.input_len = il.data();
    rq.output_len = ol.data();
    rq.slo_us = slo_us.data();
    SimRouter sr{&P.p, &emb, &il, &no, &rslo};
    std::vector<int32_t> pair(R);
    std::vector<float> u(R), pe(R);
    std::vector<int64_t> ft(R), fin(R);
    const int32_t max_samples = static_cast<int32_t>(m["max_samples"]);
    std::vector<hwr_hw_state> samples(static_cast<size_t>(max_samples) * N);
    hwr_sim_result res{};
    res.pair = pair.data();
    res.utility = u.data();
    res.pred_e2e_s = pe.data();
    res.first_token_us = ft.data();
    res.finish_us = fin.data();
    res.max_samples = max_samples;
    res.samples = samples.data();
    const hwr_status st = hwr_sim_run(nullptr, &cfg, &rq, sim_route, &sr, &res);
    if (st != HWR_OK) {
        std::fprintf(stderr, "hwr_sim_run: %s\n", hwr_sim_last_error());
        return 6;
    }
    save("sim_pair.bin", pair);
    save("sim_utility.bin", u);
    save("sim_pred_e2e_s.bin", pe);
    save("sim_first_token_us.bin", ft);
    save("sim_finish_us.bin", fin);
    samples.resize(static_cast<size_t>(std::min(res.n_samples, max_samples)) * N);
    save("sim_samples.bin", samples);
    const std::vector<double> metrics{static_cast<double>(res.n_completed), static_cast<double>(res.n_met_slo),
                                      res.slo_attainment, res.mean_latency_s, res.p99_latency_s,
                                      res.running_fraction, res.load_skew, res.waiting_skew, res.mean_utility};
    save("sim_metrics.bin", metrics);
    return 0;
}

}  // namespace

int main(int argc, char **argv) {
    if (argc != 3) return 1;
    g_dir = argv[2];
    const std::string mode = argv[1];
    if (mode == "route") return run_route();
    if (mode == "sim") return run_sim();
    return 1;
}
