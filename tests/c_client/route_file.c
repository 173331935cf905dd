/*
 * A plain C client of libhwr (include/hwr.h): reads a routing problem and a
 * batch of host queries from a binary file, routes the batch, writes the
 * decisions.  No Python and no torch: the C ABI alone.
 *
 *   route_file <in.bin> <out.bin>
 *
 * in.bin, little-endian, every array contiguous in this order:
 *   int32  M, G, N, A, Gw, D, F, H, n, pipeline
 *   float  cost_weight, default_slo_s
 *   int32  dep_model[N], dep_gpu[N], model_arch[M]
 *   float  model_params_b[M]
 *   uint16 wq[D*M]   float bq[M]     (bf16 bit patterns)
 *   uint16 w1[F*H]   float b1[H]
 *   uint16 w2[H*H]   float b2[H]
 *   uint16 w3[H*2]   float b3[2]
 *   hwr_hw_state state[N]             (24 bytes each)
 *   uint16 emb[n*D]  int32 input_len[n]  int32 expected_out_len[n]  float slo_s[n]
 * out.bin: int32 choice[n], uint8 feasible[n], float utility[n], e2e_s[n],
 *   ttft_s[n], tpot_s[n].
 * Exit status 0 on success; otherwise a message on stderr.
 */
#include <stdint.h>
#include <stdio.h>
#include <stdlib.h>

#include "hwr.h"

static FILE *g_in;

static void *take(size_t bytes) {
    void *p = malloc(bytes ? bytes : 1);
    if (!p || fread(p, 1, bytes, g_in) != bytes) {
        fprintf(stderr, "route_file: short input\n");
        exit(2);
    }
    return p;
}

int main(int argc, char **argv) {
    if (argc != 3) {
        fprintf(stderr, "usage: route_file <in.bin> <out.bin>\n");
        return 2;
    }
    g_in = fopen(argv[1], "rb");
    if (!g_in) {
        fprintf(stderr, "route_file: cannot open %s\n", argv[1]);
        return 2;
    }
    const int32_t *hd = take(10 * sizeof(int32_t));
    const float *hf = take(2 * sizeof(float));
    const int32_t M = hd[0], G = hd[1], N = hd[2], D = hd[5], F = hd[6], H = hd[7], n = hd[8];
    hwr_config cfg = {0};
    cfg.n_models = M;
    cfg.n_gpu_types = G;
    cfg.n_deployments = N;
    cfg.arch_width = hd[3];
    cfg.gpu_width = hd[4];
    cfg.embed_dim = D;
    cfg.feat_dim = F;
    cfg.hidden = H;
    cfg.emb_dtype = cfg.weight_dtype = HWR_BF16;
    cfg.pipeline = hd[9];
    cfg.cost_weight = hf[0];
    cfg.default_slo_s = hf[1];
    cfg.n_heads = 2;
    cfg.dep_model = take(N * sizeof(int32_t));
    cfg.dep_gpu = take(N * sizeof(int32_t));
    cfg.model_arch = take(M * sizeof(int32_t));
    cfg.model_params_b = take(M * sizeof(float));
    cfg.wq = take((size_t)D * M * 2);
    cfg.bq = take(M * sizeof(float));
    cfg.w1 = take((size_t)F * H * 2);
    cfg.b1 = take(H * sizeof(float));
    cfg.w2 = take((size_t)H * H * 2);
    cfg.b2 = take(H * sizeof(float));
    cfg.w3 = take((size_t)H * 2 * 2);
    cfg.b3 = take(2 * sizeof(float));
    const hwr_hw_state *state = take(N * sizeof(hwr_hw_state));
    hwr_query_batch q = {0};
    q.n = n;
    q.mem = HWR_MEM_HOST;
    q.emb = take((size_t)n * D * 2);
    q.input_len = take(n * sizeof(int32_t));
    q.expected_out_len = take(n * sizeof(int32_t));
    q.slo_s = take(n * sizeof(float));
    fclose(g_in);

    hwr_ctx *ctx = NULL;
    hwr_status st = hwr_init(&cfg, &ctx);
    if (st != HWR_OK) {
        fprintf(stderr, "hwr_init: %d %s\n", (int)st, hwr_last_error(NULL));
        return 1;
    }
    st = hwr_update_hw_state(ctx, state, N);
    hwr_route_result r = {0};
    r.choice = malloc(n * sizeof(int32_t));
    r.feasible = malloc(n);
    float *vals = malloc(4 * (size_t)n * sizeof(float));
    r.utility = vals;
    r.e2e_s = vals + n;
    r.ttft_s = vals + 2 * (size_t)n;
    r.tpot_s = vals + 3 * (size_t)n;
    if (st == HWR_OK) st = hwr_route_batch(ctx, &q, &r);
    if (st != HWR_OK) {
        fprintf(stderr, "route: %d %s\n", (int)st, hwr_last_error(ctx));
        hwr_free(ctx);
        return 1;
    }
    hwr_free(ctx);
    FILE *out = fopen(argv[2], "wb");
    if (!out || fwrite(r.choice, sizeof(int32_t), n, out) != (size_t)n || fwrite(r.feasible, 1, n, out) != (size_t)n ||
        fwrite(vals, sizeof(float), 4 * (size_t)n, out) != 4 * (size_t)n) {
        fprintf(stderr, "route_file: cannot write %s\n", argv[2]);
        return 2;
    }
    fclose(out);
    return 0;
}
