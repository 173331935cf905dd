/*
 * hwr.h -- batched hardware-aware LLM routing scores on one MI355X (gfx950).
 *
 * The routing problem (HW-Router, Sec. 3.1): a set of n model-GPU pairs
 * (M_i, g_i) and a set of queries; each query is assigned to one pair.  For
 * every (query, pair) candidate the library
 *   1. assembles the feature vector feat(x, M_i, S_i): model attributes
 *      (architecture id, parameter count), GPU type, the query's input length,
 *      and the pair's runtime signals S_i (Table 2 plus GPU utilisation)
 *      -- Sec. 3.2, Eq. 1;
 *   2. runs the cost predictor f_cost, a small MLP with two hidden ReLU layers,
 *      giving TTFT and TPOT -- and, with three output heads, the number of
 *      output tokens N_out -- and the cost C = TTFT + N_out * TPOT
 *      -- Sec. 3.2, Eq. 1 and Eq. 2 (with two heads N_out is given per query);
 *   3. estimates the hardware-independent quality Q of the pair's model from
 *      the query embedding (a linear head per model) -- Sec. 3.2, item 3;
 *   4. scores each candidate -- by default u = Q - w * C / B (the Sec. 3.1
 *      trade-off score with the cost normalised by the bound B), or the
 *      paper's own u = (1 - w) * Q - w * C with w = lambda -- and takes, per
 *      query, the argmax over the pairs that meet the latency bound, C <= B
 *      -- Eq. 3.  B is the query's SLO, or the evaluation's SLO form
 *      B = a + b * input_len + N_out * tpot_slo.  Several weights w can be
 *      scored in one call (a lambda sweep), reusing the predictions.
 *
 * Feature layout (F slots; A = arch_width, Gw = gpu_width, b = A + Gw):
 *   [arch one-hot (A)] [GPU one-hot (Gw)] ln(params_B)/4, ln(input_len)/8,
 *   ln(1+running)/2, ln(1+waiting)/2, kv_util, gpu_util, ln(ttft_avg_s)/4,
 *   ln(tpot_avg_s)/4, then zeros up to F.  Requires A + Gw + 8 <= F <= 32.
 *
 * Decision rule: among candidates with C <= B, the largest u; if none meets
 * the bound, the largest u over all pairs (reported feasible = 0); exact ties
 * go to the lowest pair index.
 *
 * Predictor outputs: z = W3^T h2 + b3; TTFT = softplus(z0), TPOT = softplus(z1)
 * in seconds and, with three heads, N_out = softplus(z2) in tokens.
 *
 * Precision: with HWR_BF16 the embeddings and all weight matrices are bf16
 * (raw uint16 bit patterns); features and hidden activations are rounded to
 * bf16 (nearest, ties to even) before each matrix product; products accumulate
 * in fp32; biases, predictions, costs and utilities are fp32.  With HWR_F32
 * everything is fp32.  The decision arithmetic rounds each operation once:
 * C = fma(TPOT, N_out, TTFT); B = fma(N_out, tpot_slo, fma(b, input_len, a))
 * in the paper-bound mode; u = Q - w * (C / B), or (1 - w) * Q - w * C with
 * 1 - w rounded once.
 *
 * Conventions
 *  - Every call returns an hwr_status; nothing throws across this boundary.
 *    On a validation error, outputs are not written; a HIP error in the middle
 *    of a batch of several chunks may leave earlier chunks' outputs written.
 *    hwr_last_error() holds a message.
 *  - The context owns device copies of weights and state; the caller owns all
 *    query and result buffers.  Configuration and state are copied in.
 *  - HWR_MEM_DEVICE batches are ordered on the context's stream and return
 *    without waiting; HWR_MEM_HOST batches return with the results written.
 *    A host batch larger than max_chunk is streamed: the next chunk's upload
 *    (on a second stream of the context) overlaps this chunk's kernels.  A
 *    host batch in pageable memory with 16 MB of embeddings or more is copied
 *    through 128 MB of pinned memory the context allocates on first use, by
 *    up to seven host threads of its own (held until hwr_free).
 *  - A context is not thread-safe: one context per thread (or per stream).
 */
#ifndef HWR_H
#define HWR_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct hwr_ctx hwr_ctx;   /* opaque, owned by the library */

/* Every function returns a status; none lets a C++ exception reach the
 * caller (a host allocation or a host thread that fails is HWR_ERR_OOM). */
typedef enum {
    HWR_OK = 0,
    HWR_ERR_INVALID_ARG = -1,     /* bad pointer, size, id or value           */
    HWR_ERR_OOM = -2,             /* device, pinned or host memory, or a host
                                     thread, could not be obtained           */
    HWR_ERR_HIP = -3,             /* HIP runtime error (incl. no device)      */
    HWR_ERR_STATE = -4,           /* route before the first state update      */
    HWR_ERR_UNSUPPORTED = -5      /* valid but unsupported shape / dtype      */
} hwr_status;

typedef enum { HWR_F32 = 0, HWR_BF16 = 1 } hwr_dtype;
typedef enum { HWR_MEM_DEVICE = 0, HWR_MEM_HOST = 1 } hwr_mem;

/* How a batch is computed.  FUSED: quality kernel, then one kernel that
 * assembles features, runs the predictor and the decision per candidate
 * without writing per-candidate data.  STAGED: quality, feature gather (writes
 * X[q][d][32] bf16), predictor (writes TTFT/TPOT per candidate), decision --
 * each stage a separate kernel.  Both give the same results. */
typedef enum { HWR_PIPE_FUSED = 0, HWR_PIPE_STAGED = 1 } hwr_pipeline;

/* hwr_config.flags */
#define HWR_FLAG_GRAPH 1          /* single host query: launch a captured graph */
#define HWR_FLAG_RESIDENT 2       /* single host query: a resident kernel serves it  */
                                  /* (takes precedence over HWR_FLAG_GRAPH)          */

/* hwr_config.score_mode / bound_mode */
typedef enum { HWR_SCORE_NORMALIZED = 0, HWR_SCORE_PAPER = 1 } hwr_score_mode;
typedef enum { HWR_BOUND_GIVEN = 0, HWR_BOUND_PAPER = 1 } hwr_bound_mode;
#define HWR_MAX_WEIGHTS 8         /* cost weights scored in one call           */

/* Runtime signals of one pair (Table 2 of the paper plus GPU utilisation). */
typedef struct {
    int32_t running_q;            /* requests running, >= 0                    */
    int32_t waiting_q;            /* requests waiting, >= 0                    */
    float   kv_util;              /* KV-cache usage as a fraction, [0, 1]      */
    float   gpu_util;             /* GPU utilisation as a fraction, [0, 1]     */
    float   ttft_avg_s;           /* recent mean time to first token, s, > 0   */
    float   tpot_avg_s;           /* recent mean time per output token, s, > 0 */
} hwr_hw_state;                   /* 24 bytes */

typedef struct {
    int32_t n_models;             /* M, 1..32                                    */
    int32_t n_gpu_types;          /* G, 1..gpu_width                             */
    int32_t n_deployments;        /* N pairs, 1..1024 (need not be M * G)        */
    int32_t arch_width;           /* A, one-hot width of the architecture id     */
    int32_t gpu_width;            /* Gw, one-hot width of the GPU type           */
    int32_t embed_dim;            /* D, multiple of 64, <= 8192                  */
    int32_t feat_dim;             /* F, A + Gw + 8 <= F <= 32                    */
    int32_t hidden;               /* H: 64, 128 or 256 (HWR_F32: 64 or 128)      */
    int32_t emb_dtype;            /* hwr_dtype; must equal weight_dtype          */
    int32_t weight_dtype;         /* hwr_dtype of wq, w1, w2, w3                 */
    int32_t pipeline;             /* hwr_pipeline                                */
    int32_t max_chunk;            /* queries per internal chunk (0 -> 65536)     */
    float   cost_weight;          /* w (one weight; see n_weights): >= 0, and    */
                                  /* <= 1 with HWR_SCORE_PAPER                   */
    float   default_slo_s;        /* bound when a batch gives no per-query SLO   */
    int32_t device;               /* HIP device ordinal                          */
    int32_t flags;                /* HWR_FLAG_*                                  */
    int32_t n_heads;              /* predictor heads: 2 (or 0): N_out given per  */
                                  /* query; 3: N_out predicted (Eq. 1)           */
    int32_t score_mode;           /* hwr_score_mode                              */
    int32_t bound_mode;           /* hwr_bound_mode                              */
    float   ttft_slo_a;           /* paper bound: a in s, > 0 (the paper's fit   */
    float   ttft_slo_b;           /* times its 1.2 slack); b in s per input      */
    float   tpot_slo;             /* token, >= 0; tpot_slo in s per output token */
    int32_t n_weights;            /* K: 0 -> one decision with cost_weight;      */
                                  /* 1..HWR_MAX_WEIGHTS -> cost_weights[K]       */
    const int32_t *dep_model;     /* [N] model of pair i, in [0, M)              */
    const int32_t *dep_gpu;       /* [N] GPU type of pair i, in [0, G)           */
    const int32_t *model_arch;    /* [M] architecture id, in [0, A)              */
    const float   *model_params_b;/* [M] parameter count in billions, > 0        */
    const void    *wq;            /* [D][M] quality heads, row-major             */
    const float   *bq;            /* [M]                                         */
    const void    *w1;            /* [F][H] row-major (input-major)              */
    const float   *b1;            /* [H]                                         */
    const void    *w2;            /* [H][H] row-major, [in][out]                 */
    const float   *b2;            /* [H]                                         */
    const void    *w3;            /* [H][n_heads] row-major; column 0 TTFT,      */
                                  /* 1 TPOT, 2 N_out                             */
    const float   *b3;            /* [n_heads]                                   */
    const float   *cost_weights;  /* [K] when n_weights > 0 (same limits as      */
                                  /* cost_weight)                                */
    void          *stream;        /* hipStream_t the context works on, or NULL   */
} hwr_config;                     /* all pointers are host memory                */

typedef struct {
    int32_t n;                    /* queries in the batch, >= 0                  */
    int32_t mem;                  /* hwr_mem of every pointer here and in the result */
    const void    *emb;           /* [n][D] in emb_dtype                         */
    const int32_t *input_len;     /* [n] prompt tokens, >= 1                     */
    const int32_t *expected_out_len; /* [n] N_out of Eq. 2, >= 0; ignored (may   */
                                     /* be NULL) with n_heads == 3               */
    const float   *slo_s;         /* [n] latency bound in s, > 0; NULL -> default_slo_s */
} hwr_query_batch;

/* With n_weights = K > 1 every per-query output below holds K values per
 * query, [n][K] (weight k of query q at q * K + k); the debug outputs keep
 * their shapes. */
typedef struct {                  /* caller-owned, in the batch's memory space   */
    int32_t *choice;              /* [n] chosen pair index (required)            */
    uint8_t *feasible;            /* [n] 1 iff the chosen pair meets the bound   */
    float   *utility;             /* [n] u of the chosen pair                    */
    float   *e2e_s;               /* [n] C of the chosen pair                    */
    float   *ttft_s;              /* [n] TTFT of the chosen pair                 */
    float   *tpot_s;              /* [n] TPOT of the chosen pair                 */
    float   *nout;                /* [n] N_out of the chosen pair (given or      */
                                  /* predicted)                                  */
    float   *cand_ttft;           /* [n][N] every candidate's TTFT (debug)       */
    float   *cand_tpot;           /* [n][N] every candidate's TPOT (debug)       */
    float   *cand_nout;           /* [n][N] every candidate's predicted N_out    */
                                  /* (debug; n_heads == 3 only)                  */
    float   *cand_quality;        /* [n][M] every (query, model) quality (debug) */
} hwr_route_result;               /* every pointer but choice may be NULL        */

/* Create a context for one deployed pair set (Sec. 3.1: the model-GPU pairs
 * (M_i, g_i) the router chooses among, with each model's attributes) and one
 * trained router: the cost predictor f_cost of Sec. 3.2 Eq. 1 (w1..w3, b1..b3)
 * and the per-model quality heads of Sec. 3.2 item 3 (wq, bq).  Validates the
 * configuration, copies and re-lays-out the weights on the device and
 * allocates work space for max_chunk queries; the caller may free every
 * buffer cfg points to when this returns.  Routing needs one
 * hwr_update_hw_state first.  Errors: HWR_ERR_INVALID_ARG for an out-of-range
 * field or NULL table, HWR_ERR_UNSUPPORTED for a shape the kernels do not
 * handle, HWR_ERR_OOM / HWR_ERR_HIP from the device; *out is NULL on error. */
hwr_status hwr_init(const hwr_config *cfg, hwr_ctx **out);

/* Replace the cached runtime signals of all N pairs (the hardware monitor's
 * local cache, Sec. 3.2 item 1).  `state` is host memory, n must equal N.
 * Every field is checked (finite, in range); on error the previous snapshot
 * is kept.  Ordered on the context's stream: later routes see the new state,
 * routes already enqueued keep the old one.  Returns before the copy ends;
 * the caller may reuse `state` immediately. */
hwr_status hwr_update_hw_state(hwr_ctx *ctx, const hwr_hw_state *state, int32_t n);

/* Route a batch (Eq. 3 for each query).  n == 0 is a no-op.  Batches larger
 * than max_chunk run as successive chunks on the context's stream.  A single
 * query in host memory takes a latency path: one kernel launch (or, with
 * HWR_FLAG_GRAPH, one launch of a graph holding that kernel, captured on the
 * first call; on ROCm 7 such a launch is about 5 us faster with the runtime's
 * graph packet capture off, DEBUG_CLR_GRAPH_PACKET_CAPTURE=0 in the
 * environment before the runtime starts) on a private stream of the context, reading the query and the
 * newest state from pinned host memory and writing the decision there; it
 * does not wait for batches still enqueued on the context's stream.  With
 * HWR_FLAG_RESIDENT, that kernel stays on the device between calls instead
 * (one workgroup, polling the pinned request record): a call then costs no
 * launch.  After about 0.1 s without a request it leaves, and the next call
 * launches it again; hwr_free stops it.  Host
 * inputs are checked (input_len >= 1, N_out >= 0, SLO > 0 and finite); device
 * inputs are not, and out-of-range values give unspecified choices (all
 * memory accesses stay in bounds). */
hwr_status hwr_route_batch(hwr_ctx *ctx, const hwr_query_batch *q, hwr_route_result *r);

/* hwr_route_batch for callers that cannot allocate device memory during a
 * call: code under HIP graph capture, tight serving loops, harnesses that
 * forbid hipMalloc.  Same arguments, results and ordering as hwr_route_batch
 * for HWR_MEM_DEVICE batches, bit for bit; it calls no hipMalloc, hipFree or
 * other allocating routine (and creates no events: kernel timing is skipped).
 * Its work space -- the quality matrix, the split partials and, for staged,
 * fp32 and several-weight contexts, the per-candidate predictions and
 * features -- lives in a static 64 MiB device array of the library, one per
 * GPU, held until the process ends (its address is taken by the first
 * hwr_init on each device).  A batch is routed in chunks of as many queries
 * as that space holds (at most max_chunk); HWR_ERR_UNSUPPORTED when a single
 * query needs more than 64 MiB (about 3,600 pairs at most, staged).  Host
 * batches: HWR_ERR_INVALID_ARG (they stage through buffers allocated on first
 * use).  Every call on one GPU uses that GPU's one array, from any context:
 * calls that overlap in time on one GPU (different streams, threads or
 * contexts) race on it and give undefined results; calls ordered on one
 * stream do not.  Each call writes every element it later reads; nothing
 * carries over from the previous call. */
hwr_status hwr_route_batch_static(hwr_ctx *ctx, const hwr_query_batch *q, hwr_route_result *r);

/* Destroy a context (NULL is allowed); waits for its stream first. */
void hwr_free(hwr_ctx *ctx);

/* Message of the last error on ctx, or of the last failed hwr_init on this
 * thread when ctx is NULL.  Never NULL; owned by the library. */
const char *hwr_last_error(const hwr_ctx *ctx);

/* Kernel timing: each kernel launch carries two HIP events that its dispatch
 * records at the kernel's start and end, on the stream it runs on (a graph
 * launch of the single-query path is bracketed by events instead).
 * fp32 chunks small enough for the predictor and the quality rows to share
 * the device run both in the predictor's launch: HWR_K_MLP, no HWR_K_QUALITY.
 * Indices of hwr_kernel_times.ms / launches: */
enum {
    HWR_K_STATE = 0, HWR_K_QUALITY = 1, HWR_K_GATHER = 2, HWR_K_MLP = 3,
    HWR_K_EPILOGUE = 4, HWR_K_FUSED = 5, HWR_K_MERGE = 6, HWR_K_SINGLE = 7,
    HWR_K_COUNT = 8
};
typedef struct {
    double  ms[HWR_K_COUNT];      /* summed kernel durations, milliseconds       */
    int64_t launches[HWR_K_COUNT];   /* timed launches                            */
} hwr_kernel_times;

/* Per-launch event timing: 0 off (the default), 1 every launch, k > 1 one
 * launch in k of each kernel kind (the first, then every k-th).  A timed
 * launch waits a few microseconds longer to be dispatched, so sampling keeps
 * the timing's cost on back-to-back launches small.  hwr_kernel_times then
 * counts and sums the timed launches only.  k < 0 is an invalid argument. */
hwr_status hwr_profile_enable(hwr_ctx *ctx, int32_t enable);
/* Wait for the timed launches, add their durations into *out (zeroed first),
 * and, if reset != 0, start a new accumulation. */
hwr_status hwr_profile_read(hwr_ctx *ctx, hwr_kernel_times *out, int32_t reset);

#ifdef __cplusplus
}
#endif
#endif /* HWR_H */
