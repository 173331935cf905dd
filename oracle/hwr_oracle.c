/*
 * CPU oracle for HW-Router's routing-score path.  TEST INFRASTRUCTURE ONLY
 * (tests, smoke check, CPU-baseline leg of the benchmark); no product code
 * links or calls it.  Plain loops, one candidate at a time, fp64 accumulation.
 *
 * Readings of the paper used here (the paper fixes none of these numbers):
 *  - Feature vector (Eq. 1 says: query features, one-hot model/GPU identifiers
 *    and the runtime signals S_i of Table 2, concatenated).  With
 *    A = arch_width, Gw = gpu_width, b = A + Gw:
 *      x[model_arch[m]] = 1, x[A + gpu] = 1,
 *      x[b+0] = ln(params_B)/4,   x[b+1] = ln(input_len)/8,
 *      x[b+2] = ln(1+running)/2,  x[b+3] = ln(1+waiting)/2,
 *      x[b+4] = kv_util,          x[b+5] = gpu_util,
 *      x[b+6] = ln(ttft_avg_s)/4, x[b+7] = ln(tpot_avg_s)/4, rest 0.
 *    Each value is computed in fp64 and rounded to fp32 (then bf16).
 *  - Predictor (Eq. 1: two hidden ReLU layers): h1 = ReLU(W1^T x + b1),
 *    h2 = ReLU(W2^T h1 + b2), z = W3^T h2 + b3, TTFT = softplus(z0),
 *    TPOT = softplus(z1), and with three heads N_out = softplus(z2), in
 *    tokens.  Each layer output is accumulated in fp64, rounded to fp32, and
 *    (bf16 workloads) h1, h2 are rounded to bf16.
 *  - Cost (Eq. 2): C = TTFT + N_out * TPOT, one fp32 rounding, with N_out the
 *    third head's prediction for the candidate, or (two heads) the output
 *    length given per query.
 *  - Quality (Sec. 3.2 item 3, hardware-independent): Q = e . Wq[:, m] + bq[m].
 *  - Decision (Sec. 3.1 score, Eq. 3): by default u = Q - w * C / B in fp32
 *    (w = 0.5 is the paper's score with lambda = 1/3 and C normalised by
 *    the bound, scaled by 2/3: the argmax is the same); or the paper's own
 *    score u = (1 - w) Q - w C (w = lambda, C in seconds).  B is the query's
 *    SLO, or the evaluation's SLO form a + b p + N_out tpot_slo (p input
 *    tokens).  A pair is feasible iff C <= B; choose the feasible pair with
 *    the largest u, ties to the lowest pair index; if no pair is feasible,
 *    the largest u over all pairs.
 */
#include "hwr_oracle.h"

#include <math.h>
#include <stdlib.h>
#include <string.h>

/* Round-to-nearest-even onto the bf16 grid (8 significand bits), from the
 * definition: keep the top 16 bits of the fp32 pattern; add one unit in the
 * last kept place when the dropped half is above one half, or exactly one half
 * with an odd kept part. */
float orc_bf16(float x) {
    uint32_t u;
    memcpy(&u, &x, 4);
    if ((u & 0x7F800000u) == 0x7F800000u) {          /* inf or NaN */
        if (u & 0x007FFFFFu) u |= 0x00400000u;       /* stay NaN   */
        u &= 0xFFFF0000u;
    } else {
        uint32_t kept = u >> 16, dropped = u & 0xFFFFu;
        if (dropped > 0x8000u || (dropped == 0x8000u && (kept & 1u))) kept += 1u;
        u = kept << 16;
    }
    float y;
    memcpy(&y, &u, 4);
    return y;
}

void orc_bf16_n(const float *x, float *y, int64_t n) {
    for (int64_t i = 0; i < n; ++i) y[i] = orc_bf16(x[i]);
}

float orc_softplus(float z) {
    double v = (double)z;
    double r = (v > 0.0 ? v : 0.0) + log1p(exp(-fabs(v)));
    return (float)r;
}

static float store(const orc_problem *p, double v) {
    float f = (float)v;
    return p->bf16 ? orc_bf16(f) : f;
}

void orc_features(const orc_problem *p, const orc_state *s, int32_t d,
                  int32_t input_len, float *x) {
    const int32_t m = p->dep_model[d];
    const int32_t A = p->arch_width, b = p->arch_width + p->gpu_width;
    for (int32_t f = 0; f < p->F; ++f) x[f] = 0.0f;
    x[p->model_arch[m]] = 1.0f;
    x[A + p->dep_gpu[d]] = 1.0f;
    x[b + 0] = store(p, log((double)p->model_params_b[m]) / 4.0);
    x[b + 1] = store(p, log((double)input_len) / 8.0);
    x[b + 2] = store(p, log(1.0 + (double)s->running_q[d]) / 2.0);
    x[b + 3] = store(p, log(1.0 + (double)s->waiting_q[d]) / 2.0);
    x[b + 4] = store(p, (double)s->kv_util[d]);
    x[b + 5] = store(p, (double)s->gpu_util[d]);
    x[b + 6] = store(p, log((double)s->ttft_avg_s[d]) / 4.0);
    x[b + 7] = store(p, log((double)s->tpot_avg_s[d]) / 4.0);
}

float orc_quality(const orc_problem *p, const float *emb_row, int32_t m) {
    double acc = 0.0;
    for (int32_t k = 0; k < p->D; ++k)
        acc += (double)emb_row[k] * (double)p->wq[(size_t)k * p->M + m];
    return (float)(acc + (double)p->bq[m]);
}

void orc_mlp(const orc_problem *p, const float *x, float *z) {
    const int32_t F = p->F, H = p->H;
    float *h1 = (float *)malloc(sizeof(float) * (size_t)H);
    float *h2 = (float *)malloc(sizeof(float) * (size_t)H);
    for (int32_t j = 0; j < H; ++j) {
        double acc = 0.0;
        for (int32_t f = 0; f < F; ++f)
            acc += (double)p->w1[(size_t)f * H + j] * (double)x[f];
        float a = (float)(acc + (double)p->b1[j]);
        h1[j] = store(p, a > 0.0f ? a : 0.0f);
    }
    for (int32_t j = 0; j < H; ++j) {
        double acc = 0.0;
        for (int32_t i = 0; i < H; ++i)
            acc += (double)p->w2[(size_t)i * H + j] * (double)h1[i];
        float a = (float)(acc + (double)p->b2[j]);
        h2[j] = store(p, a > 0.0f ? a : 0.0f);
    }
    const int32_t NH = p->n_heads == 3 ? 3 : 2;
    for (int32_t k = 0; k < NH; ++k) {
        double acc = 0.0;
        for (int32_t i = 0; i < H; ++i)
            acc += (double)p->w3[(size_t)i * NH + k] * (double)h2[i];
        z[k] = (float)(acc + (double)p->b3[k]);
    }
    free(h1);
    free(h2);
}

/* u in fp32, each operation rounded once (the file is built with contraction
 * off): score 0: t = C / B, u = Q - w * t; score 1: u = (1 - w) * Q - w * C.
 * -0 -> +0, NaN -> -inf. */
static float utility(const orc_rule *r, float q, float c, float bound) {
    float u;
    if (r->score_mode == 1) {
        const float w1 = 1.0f - r->w;
        const float wq = w1 * q;
        const float wc = r->w * c;
        u = wq - wc;
    } else {
        const float t = c / bound;
        const float at = r->w * t;
        u = q - at;
    }
    if (u != u) u = -INFINITY;
    if (u == 0.0f) u = 0.0f;
    return u;
}

/* The latency bound B of a candidate: the query's SLO, or a + b p + N_out
 * tpot_slo (two fused multiply-adds, each rounded once). */
static float bound_of(const orc_rule *r, int32_t input_len, float nout, float slo) {
    if (r->bound_mode == 1) {
        const float base = fmaf(r->ttft_slo_b, (float)input_len, r->ttft_slo_a);
        return fmaf(nout, r->tpot_slo, base);
    }
    return slo;
}

static orc_rule rule_of(const orc_problem *p) {
    orc_rule r;
    r.score_mode = p->score_mode;
    r.bound_mode = p->bound_mode;
    r.w = p->alpha;
    r.ttft_slo_a = p->ttft_slo_a;
    r.ttft_slo_b = p->ttft_slo_b;
    r.tpot_slo = p->tpot_slo;
    return r;
}

int orc_route(const orc_problem *p, const orc_state *s, const orc_queries *q,
              orc_result *r) {
    const int32_t N = p->N, M = p->M, F = p->F;
    const int32_t NH = p->n_heads == 3 ? 3 : 2;
    if (N <= 0 || M <= 0 || F <= 0 || p->H <= 0 || q->n < 0) return -1;
    if (p->n_heads != 0 && p->n_heads != 2 && p->n_heads != 3) return -1;
    const orc_rule rule = rule_of(p);
    if (p->arch_width + p->gpu_width + 8 > F) return -1;
    float *x = (float *)malloc(sizeof(float) * (size_t)F);
    float *qual = (float *)malloc(sizeof(float) * (size_t)M);
    for (int32_t iq = 0; iq < q->n; ++iq) {
        const float *e = q->emb + (size_t)iq * p->D;
        const float slo = q->slo_s[iq];
        const float nout_given = NH == 2 ? (float)q->expected_out_len[iq] : 0.0f;
        for (int32_t m = 0; m < M; ++m) {
            qual[m] = orc_quality(p, e, m);
            if (r->quality) r->quality[(size_t)iq * M + m] = qual[m];
        }
        int32_t best = -1;
        int best_f = 0;
        float best_u = 0.0f, best_c = 0.0f, best_tt = 0.0f, best_tp = 0.0f, best_n = 0.0f;
        for (int32_t d = 0; d < N; ++d) {
            float z[3];
            orc_features(p, s, d, q->input_len[iq], x);
            orc_mlp(p, x, z);
            const float ttft = orc_softplus(z[0]);
            const float tpot = orc_softplus(z[1]);
            const float nout = NH == 3 ? orc_softplus(z[2]) : nout_given;
            const float c = fmaf(tpot, nout, ttft);
            const float bound = bound_of(&rule, q->input_len[iq], nout, slo);
            const int feas = (c <= bound);
            const float u = utility(&rule, qual[p->dep_model[d]], c, bound);
            const size_t ci = (size_t)iq * N + d;
            if (r->cand_bound) r->cand_bound[ci] = bound;
            if (r->cand_z)
                for (int32_t k = 0; k < NH; ++k) r->cand_z[NH * ci + k] = z[k];
            if (r->cand_nout) r->cand_nout[ci] = nout;
            if (r->cand_ttft) r->cand_ttft[ci] = ttft;
            if (r->cand_tpot) r->cand_tpot[ci] = tpot;
            if (r->cand_e2e) r->cand_e2e[ci] = c;
            if (r->cand_u) r->cand_u[ci] = u;
            if (r->cand_feasible) r->cand_feasible[ci] = (uint8_t)feas;
            /* lexicographic (feasible, u), earlier pair wins exact ties */
            if (best < 0 || feas > best_f || (feas == best_f && u > best_u)) {
                best = d; best_f = feas; best_u = u;
                best_c = c; best_tt = ttft; best_tp = tpot; best_n = nout;
            }
        }
        if (r->choice) r->choice[iq] = best;
        if (r->feasible) r->feasible[iq] = (uint8_t)best_f;
        if (r->utility) r->utility[iq] = best_u;
        if (r->e2e_s) r->e2e_s[iq] = best_c;
        if (r->ttft_s) r->ttft_s[iq] = best_tt;
        if (r->tpot_s) r->tpot_s[iq] = best_tp;
        if (r->nout) r->nout[iq] = best_n;
    }
    free(x);
    free(qual);
    return 0;
}

int orc_decide(int32_t n, int32_t N, int32_t M, const int32_t *dep_model,
               const float *cand_ttft, const float *cand_tpot, const float *cand_nout,
               const float *quality, const int32_t *input_len, const int32_t *expected_out_len,
               const float *slo_s, const orc_rule *rule,
               int32_t *choice, uint8_t *feasible, float *utility_out, float *e2e_out) {
    if (n < 0 || N <= 0 || M <= 0) return -1;
    for (int32_t iq = 0; iq < n; ++iq) {
        const float slo = slo_s[iq];
        int32_t best = -1;
        int best_f = 0;
        float best_u = 0.0f, best_c = 0.0f;
        for (int32_t d = 0; d < N; ++d) {
            const size_t ci = (size_t)iq * N + d;
            const float nout = cand_nout ? cand_nout[ci] : (float)expected_out_len[iq];
            const float c = fmaf(cand_tpot[ci], nout, cand_ttft[ci]);
            const float bound = bound_of(rule, input_len[iq], nout, slo);
            const int feas = (c <= bound);
            const float u = utility(rule, quality[(size_t)iq * M + dep_model[d]], c, bound);
            if (best < 0 || feas > best_f || (feas == best_f && u > best_u)) {
                best = d; best_f = feas; best_u = u; best_c = c;
            }
        }
        choice[iq] = best;
        feasible[iq] = (uint8_t)best_f;
        utility_out[iq] = best_u;
        e2e_out[iq] = best_c;
    }
    return 0;
}
