/*
 * CPU oracle for HW-Router's batched routing-score path.  TEST INFRASTRUCTURE
 * ONLY: the tests, the smoke check and the benchmark's CPU-baseline leg call
 * it; the HIP library never does, and the two share no code.
 *
 * It computes, for every query x and every model-GPU pair i, literally and one
 * candidate at a time:
 *   - the feature vector feat(x, M_i, S_i)                     (Sec. 3.2, Eq. 1)
 *   - the cost predictor f_cost -> TTFT_i(x), TPOT_i(x)        (Sec. 3.2, Eq. 1)
 *   - the cost C_i(x) = TTFT_i(x) + N_out(x) * TPOT_i(x)       (Sec. 3.2, Eq. 2)
 *   - the hardware-independent quality Q_i(x)                  (Sec. 3.2, item 3)
 *   - the SLO-constrained argmax of the trade-off score        (Sec. 3.1; Eq. 3)
 * Accumulation is in fp64; values are rounded to fp32 (and to bf16 where the
 * workload stores bf16) at the points documented in hwr_oracle.c.
 *
 * Parity pins: see tests/test_oracle_pins.py (every function here is pinned).
 */
#ifndef HWR_ORACLE_H
#define HWR_ORACLE_H
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct {
    int32_t M, G, N, D, F, H;          /* models, GPU types, pairs, embed, feat, hidden */
    int32_t arch_width, gpu_width;     /* one-hot widths                                 */
    int32_t bf16;                      /* 1: round x, h1, h2 to bf16 before next layer  */
    int32_t n_heads;                   /* 2 (or 0): N_out given; 3: predicted (Eq. 1)    */
    float   alpha;                     /* cost weight w of the score (see orc_rule)      */
    int32_t score_mode;                /* see orc_rule                                   */
    int32_t bound_mode;
    float   ttft_slo_a, ttft_slo_b, tpot_slo;
    const int32_t *dep_model, *dep_gpu;     /* [N]                                   */
    const int32_t *model_arch;              /* [M]                                   */
    const float   *model_params_b;          /* [M] (billions)                        */
    const float   *wq, *bq;                 /* [D*M] row-major [D][M], [M]           */
    const float   *w1, *b1;                 /* [F*H] row-major [F][H], [H]           */
    const float   *w2, *b2;                 /* [H*H] row-major [H_in][H_out], [H]    */
    const float   *w3, *b3;                 /* [H*NH] row-major [H][NH], [NH]        */
} orc_problem;

typedef struct {                            /* per pair, Table 2 + GPU utilisation  */
    const int32_t *running_q, *waiting_q;
    const float   *kv_util, *gpu_util, *ttft_avg_s, *tpot_avg_s;
} orc_state;

typedef struct {
    int32_t n;
    const float   *emb;                     /* [n*D]                                 */
    const int32_t *input_len;               /* [n]                                   */
    const int32_t *expected_out_len;        /* [n]                                   */
    const float   *slo_s;                   /* [n]                                   */
} orc_queries;

/* Decision rule (Sec. 3.1 score, Eq. 3 bound; the bound's paper form is the
 * evaluation's SLO definition):
 *   score_mode 0: u = Q - w * (C / B)        1: u = (1 - w) * Q - w * C
 *   bound_mode 0: B = the query's SLO        1: B = a + b * p + N_out * tpot_slo
 * with p the input length and N_out the candidate's (given or predicted);
 * a pair is feasible iff C <= B.  Every fp32 operation is rounded once. */
typedef struct {
    int32_t score_mode, bound_mode;
    float   w;
    float   ttft_slo_a, ttft_slo_b, tpot_slo;
} orc_rule;

typedef struct {                            /* any pointer may be NULL (not written) */
    int32_t *choice;                        /* [n]                                   */
    uint8_t *feasible;                      /* [n]                                   */
    float   *utility, *e2e_s, *ttft_s, *tpot_s;   /* [n], of the chosen pair         */
    float   *nout;                          /* [n] N_out used for the chosen pair    */
    float   *cand_z;                        /* [n*N*NH] predictor outputs before softplus */
    float   *cand_nout;                     /* [n*N] N_out used per candidate        */
    float   *cand_ttft, *cand_tpot, *cand_e2e, *cand_u;   /* [n*N]                   */
    float   *cand_bound;                    /* [n*N] the bound B of each candidate    */
    uint8_t *cand_feasible;                 /* [n*N]                                 */
    float   *quality;                       /* [n*M]                                 */
} orc_result;

/* fp32 -> nearest bf16 value (ties to even), returned as fp32. */
float orc_bf16(float x);
void  orc_bf16_n(const float *x, float *y, int64_t n);
/* softplus in fp64, rounded to fp32. */
float orc_softplus(float z);
/* feature vector of (query with input_len, pair d) into x[F]. */
void  orc_features(const orc_problem *p, const orc_state *s, int32_t d,
                   int32_t input_len, float *x);
/* quality of model m for one embedding row. */
float orc_quality(const orc_problem *p, const float *emb_row, int32_t m);
/* predictor on one feature vector: z[NH] before softplus (NH = 2 or 3). */
void  orc_mlp(const orc_problem *p, const float *x, float *z);
/* Eq. 2 and Eq. 3 alone, on given predictions: for each of n queries, the
 * candidates' TTFT and TPOT ([n*N]), their N_out ([n*N]; NULL: the query's
 * expected_out_len) and the per-model quality ([n*M], mapped to pairs through
 * dep_model) -> the choice and its feasibility, utility and cost, with the
 * same arithmetic and tie rule as orc_route.  Returns 0, or -1 on bad sizes. */
int   orc_decide(int32_t n, int32_t N, int32_t M, const int32_t *dep_model,
                 const float *cand_ttft, const float *cand_tpot, const float *cand_nout,
                 const float *quality, const int32_t *input_len, const int32_t *expected_out_len,
                 const float *slo_s, const orc_rule *rule,
                 int32_t *choice, uint8_t *feasible, float *utility_out, float *e2e_out);
/* the whole path over a batch of queries.  Returns 0, or -1 on bad sizes. */
int   orc_route(const orc_problem *p, const orc_state *s, const orc_queries *q,
                orc_result *r);

#ifdef __cplusplus
}
#endif
#endif
