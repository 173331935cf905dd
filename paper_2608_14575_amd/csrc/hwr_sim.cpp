// Closed-loop serving simulator around the routing path (host code).  The
// semantics (step order, service model, monitor snapshot, metrics) are stated
// in hwr_sim.h; this file follows them literally.  Everything that decides
// the trajectory is integer arithmetic, and every floating-point value is one
// IEEE operation on exactly converted integers (or a plain sum in a fixed
// order), so a run can be reproduced bit for bit.
#include "hwr_sim.h"

#include <algorithm>
#include <chrono>
#include <cmath>
#include <deque>
#include <string>
#include <vector>

#include "c_boundary.hpp"

namespace {

thread_local std::string g_sim_err = "no error";

hwr_status sim_fail(hwr_status st, const std::string &msg) {
    g_sim_err = msg;
    return st;
}

struct Active {
    int32_t r;              // request index
    int64_t delay;          // offset of the arrival into the step it was admitted in
    int64_t prefill_left;   // prefill microseconds still to run
    bool first_done;        // first token emitted
    int64_t acc;            // microseconds accumulated since the last token
    int32_t tokens_left;    // tokens after the first still to generate
};

struct PairState {
    std::deque<int32_t> waiting;
    std::vector<Active> running;
    int64_t kv_used = 0;
    int64_t ttft_sum_us = 0, ttft_n = 0;   // first tokens of the monitor window
    double tpot_sum_s = 0.0;
    int64_t tpot_n = 0;                    // completions of the monitor window
    float ttft_avg = 0.0f, tpot_avg = 0.0f;
};

double percentile(const std::vector<int64_t> &sorted, double q) {
    if (sorted.empty()) return 0.0;
    const size_t i = static_cast<size_t>(std::floor(q * static_cast<double>(sorted.size() - 1)));
    return static_cast<double>(sorted[i]) / 1e6;
}

double percentile_d(std::vector<double> v, double q) {
    if (v.empty()) return 0.0;
    std::sort(v.begin(), v.end());
    return v[static_cast<size_t>(std::floor(q * static_cast<double>(v.size() - 1)))];
}

bool positive_finite(float x) { return std::isfinite(x) && x > 0.0f; }

hwr_status validate(const hwr_ctx *ctx, const hwr_sim_config *cfg, const hwr_sim_requests *rq,
                    hwr_sim_router_fn router, const hwr_sim_result *res) {
    const hwr_status bad = HWR_ERR_INVALID_ARG;
    if (!cfg || !rq || !res) return sim_fail(bad, "cfg, requests and result are required");
    if (!router && !ctx) return sim_fail(bad, "a library context or a router callback is required");
    if (cfg->n_pairs < 1 || cfg->n_gpus < 1 || !cfg->pairs) return sim_fail(bad, "n_pairs, n_gpus >= 1 and pairs are required");
    for (int d = 0; d < cfg->n_pairs; ++d) {
        const hwr_sim_pair &p = cfg->pairs[d];
        if (p.gpu < 0 || p.gpu >= cfg->n_gpus || p.max_running < 1 || p.kv_capacity < 1 ||
            p.prefill_base_us < 1 || p.prefill_per_token_ns < 0 || p.tpot_base_us < 1 ||
            p.tpot_per_running_us < 0)
            return sim_fail(bad, "pair " + std::to_string(d) + ": out-of-range serving parameters");
    }
    if (cfg->tick_us < 1 || cfg->monitor_period_us < cfg->tick_us || cfg->monitor_period_us % cfg->tick_us != 0)
        return sim_fail(bad, "tick_us >= 1 and monitor_period_us a positive multiple of it are required");
    if (cfg->max_time_us < 0) return sim_fail(bad, "max_time_us < 0");
    if (!cfg->prior_ttft_s || !cfg->prior_tpot_s) return sim_fail(bad, "prior_ttft_s and prior_tpot_s are required");
    for (int d = 0; d < cfg->n_pairs; ++d)
        if (!positive_finite(cfg->prior_ttft_s[d]) || !positive_finite(cfg->prior_tpot_s[d]))
            return sim_fail(bad, "priors must be finite and > 0");
    if (rq->n < 0) return sim_fail(bad, "n < 0");
    if (rq->n > 0) {
        if (!rq->arrival_us || !rq->input_len || !rq->output_len || !rq->slo_us)
            return sim_fail(bad, "arrival_us, input_len, output_len and slo_us are required");
        for (int r = 0; r < rq->n; ++r) {
            if (rq->arrival_us[r] < 0 || (r > 0 && rq->arrival_us[r] < rq->arrival_us[r - 1]))
                return sim_fail(bad, "arrival_us must be >= 0 and non-decreasing");
            if (rq->input_len[r] < 1 || rq->output_len[r] < 1 || rq->slo_us[r] < 0)
                return sim_fail(bad, "input_len, output_len >= 1 and slo_us >= 0 are required");
        }
        if (!router) {
            if (!rq->emb || rq->embed_dim < 1 || (rq->emb_dtype != HWR_F32 && rq->emb_dtype != HWR_BF16))
                return sim_fail(bad, "emb, embed_dim and emb_dtype are required with a library router");
        }
    }
    if (res->max_samples < 0) return sim_fail(bad, "max_samples < 0");
    if (res->max_samples > 0 && !res->samples) return sim_fail(bad, "samples is NULL");
    return HWR_OK;
}

hwr_status sim_run(hwr_ctx *ctx, const hwr_sim_config *cfg, const hwr_sim_requests *rq,
                   hwr_sim_router_fn router, void *user, hwr_sim_result *res) {
    hwr_status st = validate(ctx, cfg, rq, router, res);
    if (st != HWR_OK) return st;
    const int N = cfg->n_pairs, G = cfg->n_gpus, R = rq->n;
    const int64_t tick = cfg->tick_us, period = cfg->monitor_period_us;

    std::vector<PairState> ps(N);
    for (int d = 0; d < N; ++d) {
        ps[d].ttft_avg = cfg->prior_ttft_s[d];
        ps[d].tpot_avg = cfg->prior_tpot_s[d];
    }
    std::vector<int32_t> pair(R, -1);
    std::vector<float> util(R, 0.0f), pe2e(R, 0.0f);
    std::vector<int64_t> first(R, -1), finish(R, -1);
    std::vector<hwr_hw_state> snap(N), cache(N);
    std::vector<int64_t> busy(G, 0), sum_run_g(G, 0), sum_wait_g(G, 0);
    std::vector<int32_t> gpu_running(G, 0);
    int64_t window_ticks = 0, sum_run = 0, sum_wait = 0;
    int32_t n_samples = 0;
    std::vector<double> route_us;
    std::vector<int32_t> done;          // finished requests of the current pair and step
    const size_t esz = rq->emb_dtype == HWR_BF16 ? 2 : 4;

    int64_t T = 0;
    int32_t next = 0;
    int64_t live = 0;                   // routed and not finished
    while (T < cfg->max_time_us) {
        // 1. monitor snapshot, handed to the router
        if (T % period == 0) {
            for (int d = 0; d < N; ++d) {
                PairState &p = ps[d];
                const hwr_sim_pair &sp = cfg->pairs[d];
                if (p.ttft_n > 0)
                    p.ttft_avg = static_cast<float>(static_cast<double>(p.ttft_sum_us) / static_cast<double>(p.ttft_n) / 1e6);
                if (p.tpot_n > 0) p.tpot_avg = static_cast<float>(p.tpot_sum_s / static_cast<double>(p.tpot_n));
                double kv = static_cast<double>(p.kv_used) / static_cast<double>(sp.kv_capacity);
                if (kv > 1.0) kv = 1.0;
                hwr_hw_state &s = snap[d];
                s.running_q = static_cast<int32_t>(p.running.size());
                s.waiting_q = static_cast<int32_t>(p.waiting.size());
                s.kv_util = static_cast<float>(kv);
                s.gpu_util = window_ticks > 0
                                 ? static_cast<float>(static_cast<double>(busy[sp.gpu]) / static_cast<double>(window_ticks))
                                 : 0.0f;
                s.ttft_avg_s = p.ttft_avg;
                s.tpot_avg_s = p.tpot_avg;
                sum_run += s.running_q;
                sum_wait += s.waiting_q;
                sum_run_g[sp.gpu] += s.running_q;
                sum_wait_g[sp.gpu] += s.waiting_q;
                p.ttft_sum_us = p.ttft_n = 0;
                p.tpot_sum_s = 0.0;
                p.tpot_n = 0;
            }
            if (n_samples < res->max_samples)
                std::copy(snap.begin(), snap.end(), res->samples + static_cast<size_t>(n_samples) * N);
            if (!cfg->freeze_state || n_samples == 0) {
                cache = snap;
                if (!router) {
                    st = hwr_update_hw_state(ctx, cache.data(), N);
                    if (st != HWR_OK) return sim_fail(st, std::string("hwr_update_hw_state: ") + hwr_last_error(ctx));
                }
            }
            ++n_samples;
            std::fill(busy.begin(), busy.end(), 0);
            window_ticks = 0;
        }
        // 2. route this step's arrivals in one call; they join their pair's queue
        const int32_t r0 = next;
        while (next < R && rq->arrival_us[next] < T + tick) ++next;
        if (next > r0) {
            const int32_t n = next - r0;
            const auto t0 = std::chrono::steady_clock::now();
            if (router) {
                if (router(user, cache.data(), N, r0, next, pair.data() + r0, util.data() + r0, pe2e.data() + r0) != 0)
                    return sim_fail(HWR_ERR_INVALID_ARG, "the router callback failed");
            } else {
                hwr_query_batch b{};
                b.n = n;
                b.mem = HWR_MEM_HOST;
                b.emb = static_cast<const char *>(rq->emb) + static_cast<size_t>(r0) * rq->embed_dim * esz;
                b.input_len = rq->input_len + r0;
                b.expected_out_len = rq->expected_out_len ? rq->expected_out_len + r0 : nullptr;
                b.slo_s = rq->route_slo_s ? rq->route_slo_s + r0 : nullptr;
                hwr_route_result out{};
                out.choice = pair.data() + r0;
                out.utility = util.data() + r0;
                out.e2e_s = pe2e.data() + r0;
                st = hwr_route_batch(ctx, &b, &out);
                if (st != HWR_OK) return sim_fail(st, std::string("hwr_route_batch: ") + hwr_last_error(ctx));
            }
            route_us.push_back(std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count());
            for (int32_t r = r0; r < next; ++r) {
                if (pair[r] < 0 || pair[r] >= N) return sim_fail(HWR_ERR_INVALID_ARG, "the router chose a pair out of range");
                ps[pair[r]].waiting.push_back(r);
            }
            live += n;
        }
        // 3. admission, FIFO, while a slot and KV room are free
        for (int d = 0; d < N; ++d) {
            PairState &p = ps[d];
            const hwr_sim_pair &sp = cfg->pairs[d];
            while (!p.waiting.empty() && static_cast<int32_t>(p.running.size()) < sp.max_running) {
                const int32_t r = p.waiting.front();
                const int64_t need = static_cast<int64_t>(rq->input_len[r]) + rq->output_len[r];
                if (p.kv_used + need > sp.kv_capacity && !p.running.empty()) break;
                p.waiting.pop_front();
                p.kv_used += need;
                Active a;
                a.r = r;
                a.delay = rq->arrival_us[r] > T ? rq->arrival_us[r] - T : 0;
                a.prefill_left = sp.prefill_base_us + static_cast<int64_t>(rq->input_len[r]) * sp.prefill_per_token_ns / 1000;
                a.first_done = false;
                a.acc = 0;
                a.tokens_left = rq->output_len[r] - 1;
                p.running.push_back(a);
            }
        }
        std::fill(gpu_running.begin(), gpu_running.end(), 0);
        for (int d = 0; d < N; ++d) gpu_running[cfg->pairs[d].gpu] += static_cast<int32_t>(ps[d].running.size());
        // 4. service for one step; finished requests leave at its end
        for (int d = 0; d < N; ++d) {
            PairState &p = ps[d];
            const hwr_sim_pair &sp = cfg->pairs[d];
            if (p.running.empty()) continue;
            const int64_t tpot = sp.tpot_base_us + static_cast<int64_t>(sp.tpot_per_running_us) * (gpu_running[sp.gpu] - 1);
            done.clear();
            for (Active &a : p.running) {
                const int32_t r = a.r;
                int64_t avail = tick - a.delay;
                a.delay = 0;
                if (!a.first_done) {
                    const int64_t used = std::min(avail, a.prefill_left);
                    a.prefill_left -= used;
                    avail -= used;
                    if (a.prefill_left > 0) continue;
                    a.first_done = true;
                    first[r] = T + (tick - avail);
                    p.ttft_sum_us += first[r] - rq->arrival_us[r];
                    ++p.ttft_n;
                }
                int64_t t_end = -1;
                if (a.tokens_left == 0) {
                    t_end = first[r];
                } else {
                    a.acc += avail;
                    const int64_t k = std::min<int64_t>(a.acc / tpot, a.tokens_left);
                    a.acc -= k * tpot;
                    a.tokens_left -= static_cast<int32_t>(k);
                    if (a.tokens_left == 0) t_end = T + tick - a.acc;
                }
                if (t_end >= 0) {
                    finish[r] = t_end;
                    if (rq->output_len[r] > 1) {
                        p.tpot_sum_s += static_cast<double>(t_end - first[r]) / 1e6 / static_cast<double>(rq->output_len[r] - 1);
                        ++p.tpot_n;
                    }
                    done.push_back(r);
                }
            }
            if (!done.empty()) {
                size_t w = 0;
                for (size_t i = 0; i < p.running.size(); ++i) {
                    const int32_t r = p.running[i].r;
                    if (finish[r] >= 0) {
                        p.kv_used -= static_cast<int64_t>(rq->input_len[r]) + rq->output_len[r];
                        --live;
                    } else {
                        p.running[w++] = p.running[i];
                    }
                }
                p.running.resize(w);
            }
        }
        ++window_ticks;
        for (int g = 0; g < G; ++g)
            if (gpu_running[g] > 0) ++busy[g];
        T += tick;
        if (next == R && live == 0) break;
    }

    // metrics (Sec. 5)
    std::vector<int64_t> lat;
    int64_t met = 0, ttft_sum = 0, ttft_n = 0, lat_sum = 0, routed = 0;
    double usum = 0.0;
    for (int r = 0; r < R; ++r) {
        if (pair[r] >= 0) {
            usum += static_cast<double>(util[r]);
            ++routed;
        }
        if (first[r] >= 0) {
            ttft_sum += first[r] - rq->arrival_us[r];
            ++ttft_n;
        }
        if (finish[r] >= 0) {
            const int64_t l = finish[r] - rq->arrival_us[r];
            lat.push_back(l);
            lat_sum += l;
            if (l <= rq->slo_us[r]) ++met;
        }
    }
    std::sort(lat.begin(), lat.end());
    res->n_samples = n_samples;
    res->end_us = T;
    res->n_completed = static_cast<int64_t>(lat.size());
    res->n_met_slo = met;
    res->route_calls = static_cast<int64_t>(route_us.size());
    res->slo_attainment = R > 0 ? static_cast<double>(met) / static_cast<double>(R) : 0.0;
    res->mean_latency_s = lat.empty() ? 0.0 : static_cast<double>(lat_sum) / static_cast<double>(lat.size()) / 1e6;
    res->p50_latency_s = percentile(lat, 0.5);
    res->p99_latency_s = percentile(lat, 0.99);
    res->mean_ttft_s = ttft_n > 0 ? static_cast<double>(ttft_sum) / static_cast<double>(ttft_n) / 1e6 : 0.0;
    const double S = n_samples > 0 ? static_cast<double>(n_samples) : 1.0;
    res->mean_running = static_cast<double>(sum_run) / S;
    res->mean_waiting = static_cast<double>(sum_wait) / S;
    res->running_fraction = sum_run + sum_wait > 0 ? static_cast<double>(sum_run) / static_cast<double>(sum_run + sum_wait) : 0.0;
    double qsum = 0.0, qmax = 0.0, qmin = 0.0, rmax = 0.0, rmin = 0.0, wmax = 0.0, wmin = 0.0;
    for (int g = 0; g < G; ++g) {
        const double qb = static_cast<double>(sum_run_g[g] + sum_wait_g[g]) / S;
        const double rb = static_cast<double>(sum_run_g[g]) / S;
        const double wb = static_cast<double>(sum_wait_g[g]) / S;
        qsum += qb;
        if (g == 0 || qb > qmax) qmax = qb;
        if (g == 0 || qb < qmin) qmin = qb;
        if (g == 0 || rb > rmax) rmax = rb;
        if (g == 0 || rb < rmin) rmin = rb;
        if (g == 0 || wb > wmax) wmax = wb;
        if (g == 0 || wb < wmin) wmin = wb;
    }
    res->avg_load = qsum / static_cast<double>(G);
    res->load_skew = qmax - qmin;
    res->running_skew = rmax - rmin;
    res->waiting_skew = wmax - wmin;
    res->mean_utility = routed > 0 ? usum / static_cast<double>(routed) : 0.0;
    double rsum = 0.0;
    for (double v : route_us) rsum += v;
    res->route_us_mean = route_us.empty() ? 0.0 : rsum / static_cast<double>(route_us.size());
    res->route_us_p50 = percentile_d(route_us, 0.5);
    res->route_us_p99 = percentile_d(route_us, 0.99);
    if (res->pair) std::copy(pair.begin(), pair.end(), res->pair);
    if (res->utility) std::copy(util.begin(), util.end(), res->utility);
    if (res->pred_e2e_s) std::copy(pe2e.begin(), pe2e.end(), res->pred_e2e_s);
    if (res->first_token_us) std::copy(first.begin(), first.end(), res->first_token_us);
    if (res->finish_us) std::copy(finish.begin(), finish.end(), res->finish_us);
    g_sim_err = "no error";
    return HWR_OK;
}

}  // namespace

extern "C" hwr_status hwr_sim_run(hwr_ctx *ctx, const hwr_sim_config *cfg, const hwr_sim_requests *rq,
                                  hwr_sim_router_fn router, void *user, hwr_sim_result *res) {
    return hwr::c_boundary([&] { return sim_run(ctx, cfg, rq, router, user, res); },
                           [](const char *m) { g_sim_err = m; });
}

extern "C" const char *hwr_sim_last_error(void) { return g_sim_err.c_str(); }
