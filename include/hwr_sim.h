/*
 * hwr_sim.h -- closed-loop serving simulator around the routing path.
 *
 * HW-Router routes every arriving query with the runtime signals that a
 * hardware monitor polls every 200-300 ms and caches (Sec. 3.2, item 1), and
 * the paper judges a router by what then happens in the serving cluster
 * (Sec. 5): the SLO attainment, the queue composition (running vs waiting
 * requests) and the load skew between GPUs.  This simulator closes that loop
 * on the host: requests arrive, are routed in batches through a router, queue
 * at their pair, are served by a simple continuous-batching model, and the
 * monitor's snapshots are fed back to the router.  With a library context the
 * router is hwr_update_hw_state + hwr_route_batch (host batches, one call per
 * simulation step that has arrivals); a callback can stand in for it.
 *
 * Time is integer microseconds and the service model is integer arithmetic,
 * so a run is deterministic and exactly reproducible.  One step of tick_us:
 *   1. at multiples of monitor_period_us, the monitor takes a snapshot of
 *      every pair (running / waiting counts, KV-cache use, GPU utilisation over
 *      the window, mean TTFT of first tokens and mean TPOT of completions in
 *      the window, or the previous value when the window saw none) and hands
 *      it to the router (kept from the first snapshot on with freeze_state);
 *   2. the requests arriving in [T, T + tick_us) are routed in one call and
 *      join their pair's waiting queue in request order (FIFO);
 *   3. each pair admits from the head of its queue while it has a free slot
 *      and KV room for input_len + output_len tokens (a pair with nothing
 *      running always admits its head);
 *   4. each running request is served for tick_us: prefill takes
 *      prefill_base_us + input_len * prefill_per_token_ns / 1000 and ends with
 *      the first token; every further token takes
 *      tpot_base_us + tpot_per_running_us * (B - 1), B = requests running on
 *      the pair's GPU; a request ends after output_len tokens and frees its
 *      slot and KV at the end of the step.
 *
 * Metrics (Sec. 5): a request meets its SLO if finish - arrival <= slo_us;
 * attainment = met / n_requests (unfinished requests do not meet it).  Queue
 * composition and load use the monitor snapshots: mean running and waiting
 * summed over pairs, running fraction = running / (running + waiting), and
 * per GPU the mean total queue Qbar_g (running + waiting of its pairs); load
 * skew = max_g Qbar_g - min_g Qbar_g (the paper's |Qbar_0 - Qbar_1| for two
 * GPUs), running and waiting skew likewise.  Percentiles are the sorted
 * values at index floor(q * (n - 1)).
 */
#ifndef HWR_SIM_H
#define HWR_SIM_H

#include <stdint.h>

#include "hwr.h"

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {                      /* serving model of one model-GPU pair      */
    int32_t gpu;                      /* physical GPU of the pair, [0, n_gpus)     */
    int32_t max_running;              /* batch slots, >= 1                         */
    int64_t kv_capacity;              /* KV-cache tokens, >= 1                     */
    int32_t prefill_base_us;          /* >= 0                                      */
    int32_t prefill_per_token_ns;     /* >= 0                                      */
    int32_t tpot_base_us;             /* time per output token, one request, >= 1  */
    int32_t tpot_per_running_us;      /* added per further running request, >= 0  */
} hwr_sim_pair;

typedef struct {
    int32_t n_pairs;                  /* N, equal to the router's pair count       */
    int32_t n_gpus;                   /* physical GPUs, >= 1                       */
    const hwr_sim_pair *pairs;        /* [N]                                       */
    int32_t tick_us;                  /* step, >= 1                                */
    int32_t monitor_period_us;        /* a positive multiple of tick_us            */
    int64_t max_time_us;              /* the run stops here, finished or not       */
    int32_t freeze_state;             /* 1: the router keeps the first snapshot    */
    const float *prior_ttft_s;        /* [N] cached TTFT / TPOT before any         */
    const float *prior_tpot_s;        /* [N] observation, > 0                      */
} hwr_sim_config;

typedef struct {                      /* host memory, sorted by arrival            */
    int32_t n;                        /* R requests, >= 0                          */
    const int64_t *arrival_us;        /* [R] non-decreasing, >= 0                  */
    const int32_t *input_len;         /* [R] prompt tokens, >= 1                   */
    const int32_t *output_len;        /* [R] tokens generated, >= 1                */
    const int64_t *slo_us;            /* [R] latency bound of the evaluation       */
    /* what the router sees (an hwr_query_batch per step):                         */
    const void    *emb;               /* [R][embed_dim], the context's emb_dtype   */
    int32_t        embed_dim;
    int32_t        emb_dtype;         /* hwr_dtype                                 */
    const int32_t *expected_out_len;  /* [R] (two-head predictors)                 */
    const float   *route_slo_s;       /* [R] bound for the router, or NULL         */
} hwr_sim_requests;

/* A router other than the library's: choose pairs for requests [r0, r1) from
 * the cached snapshot (N records); write choice (in [0, N)), utility and
 * predicted cost per request; return 0, or nonzero to abort the run. */
typedef int32_t (*hwr_sim_router_fn)(void *user, const hwr_hw_state *snapshot, int32_t n_pairs,
                                     int32_t r0, int32_t r1, int32_t *choice, float *utility,
                                     float *e2e_s);

typedef struct {
    /* per request [R], caller-owned */
    int32_t *pair;                    /* chosen pair, -1 if never routed           */
    float   *utility;                 /* router's utility of the choice            */
    float   *pred_e2e_s;              /* router's predicted cost C of the choice   */
    int64_t *first_token_us;          /* -1 if not reached                         */
    int64_t *finish_us;               /* -1 if not finished                        */
    /* monitor snapshots [max_samples][N], caller-owned (may be NULL)             */
    int32_t max_samples;
    hwr_hw_state *samples;
    /* outputs */
    int32_t n_samples;                /* snapshots taken (all count in metrics)    */
    int64_t end_us;                   /* time the run stopped                      */
    int64_t n_completed, n_met_slo, route_calls;
    double  slo_attainment;
    double  mean_latency_s, p50_latency_s, p99_latency_s, mean_ttft_s;
    double  mean_running, mean_waiting, running_fraction;
    double  avg_load, load_skew, running_skew, waiting_skew;
    double  mean_utility;
    /* host clock around each router call (not part of the deterministic state) */
    double  route_us_mean, route_us_p50, route_us_p99;
} hwr_sim_result;

/* Run the simulation.  ctx: the router (router == NULL), or NULL with a
 * callback router.  The context must have n_pairs pairs; its cached state is
 * replaced by the simulator's snapshots.  Samples beyond max_samples are still
 * taken and counted in the metrics but not stored.  HWR_ERR_INVALID_ARG for
 * inconsistent sizes or values, the router's status if a route fails. */
hwr_status hwr_sim_run(hwr_ctx *ctx, const hwr_sim_config *cfg, const hwr_sim_requests *req,
                       hwr_sim_router_fn router, void *user, hwr_sim_result *res);

/* Message of the last hwr_sim_run error on this thread.  Never NULL. */
const char *hwr_sim_last_error(void);

#ifdef __cplusplus
}
#endif
#endif /* HWR_SIM_H */
