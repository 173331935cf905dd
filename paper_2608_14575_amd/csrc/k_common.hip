// State ingest, feature gather, decision epilogue, split merge and the fp32
// predictor / quality kernels of libhwr (gfx950).
#include <cfloat>
#include <cmath>

#include "hwr_device.hpp"
#include "hwr_probe.h"

namespace hwr {

// ------------------------------------------------------------ state ingest
// One thread per pair: the pair's slice of the Eq. 1 feature vector (model
// and GPU one-hots, parameter count, Table 2 signals, GPU utilisation), in
// fp32 and bf16.  The query slot (ln(input_len)/8) is left 0 here and filled
// per candidate.  Logs are evaluated in fp64 and rounded once to fp32.
__global__ __launch_bounds__(256) void k_state(StateArgs a) {
    const int d = blockIdx.x * blockDim.x + threadIdx.x;
    if (d >= a.N) return;
    const PairFeatures p = pair_features(a.src[d], a.pair_params[d], a.pair_arch[d], a.dep_gpu[d],
                                         a.arch_width, a.gpu_width);
    float *rf = a.dep_f32 + static_cast<size_t>(d) * kFeatPad;
    uint16_t *rb = a.dep_bf16 + static_cast<size_t>(d) * kFeatPad;
#pragma unroll
    for (int f = 0; f < kFeatPad; ++f) {
        const float v = p.slot(f);
        rf[f] = v;
        rb[f] = (a.fold_b1 && f >= kFoldSlot) ? uint16_t{0x3F80} : bf16_bits(v);   // 1.0
    }
}

hipError_t launch_state(const StateArgs &a, hipStream_t s) {
    return launch_kernel(k_state, dim3((a.N + 255) / 256), dim3(256), 0, s, a);
}

// ------------------------------------------------------------ fp32 quality
// Hardware-independent quality (Sec. 3.2 item 3): Q[q][m] = e_q . Wq[:, m] + bq[m].
// fp32 workloads; one wave per query.  Lane l accumulates every model over
// k = l, l + 64, ... (the embedding row and Wq's rows k, M consecutive
// floats each, are read lane-contiguously), then a DPP sum per model; lane m
// writes model m's value to dst[m].
__device__ __forceinline__ void quality_row_f32(const QualityArgs &a, int q, int lane, float *dst) {
    const float *e = static_cast<const float *>(a.emb) + static_cast<size_t>(q) * a.D;
    const int M = a.M;
    float acc[kMaxModels];
#pragma unroll
    for (int m = 0; m < kMaxModels; ++m) acc[m] = 0.0f;
    for (int k = lane; k < a.D; k += 64) {
        const float ev = e[k];
        const float *w = a.wq + static_cast<size_t>(k) * M;
#pragma unroll
        for (int m = 0; m < kMaxModels; ++m)
            if (m < M) acc[m] = fmaf(ev, w[m], acc[m]);
    }
#pragma unroll
    for (int m = 0; m < kMaxModels; ++m) {
        if (m < M) {
            const float v = wave_sum(acc[m]);
            if (lane == m) dst[m] = v + a.bq[m];
        }
    }
}

__global__ __launch_bounds__(256) void k_quality_f32(QualityArgs a) {
    const int lane = threadIdx.x & 63;
    const int q = blockIdx.x * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    if (q >= a.nq) return;                       // the whole wave
    quality_row_f32(a, q, lane, a.qmat + static_cast<size_t>(q) * a.M);
}

hipError_t launch_quality_f32(const QualityArgs &a, hipStream_t s) {
    return launch_kernel(k_quality_f32, dim3(static_cast<unsigned>((a.nq + 3) / 4)), dim3(256), 0, s, a);
}

// ------------------------------------------------------------ fp32 predictor
// Eq. 1 predictor in fp32, one wave per candidate (q, d).  Lane l holds
// hidden units l and (H = 128) l + 64.  Layer 1 reads the pair's feature row
// as wave-uniform values; layer 2 broadcasts each first-layer unit with
// readlane; the heads are DPP sums, then softplus.  Both hidden layers
// accumulate in input order from the bias, one rounding per fused
// multiply-add.  Weights staged in LDS as [input][unit] rows, so the lanes of
// a wave read consecutive words.
template <int H>
struct alignas(16) F32Weights {
    float w1[kFeatPad * H];
    float w2[H * H];
    float w3[H * kMaxHeads];
    float b1[H];
    float b2[H];
};

// Copy the weights into LDS (256 threads).  Trip counts are compile-time
// bounds and the copies move 16 bytes, so every load of a thread is issued
// before its first store: one memory round trip, not one per iteration.
template <int T, int CAP>
__device__ __forceinline__ void copy_f32x4(float *dst, const float *src, int count) {
    const int n4 = count / 4;                 // counts are multiples of 4 here
    f32x4 v[(CAP / 4 + T - 1) / T];
#pragma unroll
    for (int i = 0; i < (CAP / 4 + T - 1) / T; ++i) {
        const int k = threadIdx.x + i * T;
        if (k < n4) v[i] = reinterpret_cast<const f32x4 *>(src)[k];
    }
#pragma unroll
    for (int i = 0; i < (CAP / 4 + T - 1) / T; ++i) {
        const int k = threadIdx.x + i * T;
        if (k < n4) reinterpret_cast<f32x4 *>(dst)[k] = v[i];
    }
}

template <int H>
__device__ __forceinline__ void stage_f32(const MlpF32Args &a, F32Weights<H> &s) {
    copy_f32x4<256, kFeatPad * H>(s.w1, a.w1, a.F * H);
    copy_f32x4<256, H * H>(s.w2, a.w2, H * H);
    copy_f32x4<256, H * kMaxHeads>(s.w3, a.w3, H * a.nheads);
    copy_f32x4<256, H>(s.b1, a.b1, H);
    copy_f32x4<256, H>(s.b2, a.b2, H);
}

// Candidate (q, d) on one wave (q and d wave-uniform): TTFT, TPOT and the
// third head's N_out, the same value in every lane.
template <int H>
__device__ __forceinline__ void predict_f32(const MlpF32Args &a, const F32Weights<H> &s, long q, int d, int lane,
                                            float &tt, float &tp, float &nc) {
    constexpr int U = H / 64;
    const int NH = a.nheads;
    const float xl = len_feature(a.q.input_len[q]);
    const float *row = a.dep_f32 + static_cast<size_t>(d) * kFeatPad;
    float h1[U], h2[U];
#pragma unroll
    for (int u = 0; u < U; ++u) h1[u] = s.b1[lane + 64 * u];
    for (int f = 0; f < a.F; ++f) {
        const float x = (f == a.len_slot) ? xl : row[f];
#pragma unroll
        for (int u = 0; u < U; ++u) h1[u] = fmaf(s.w1[f * H + lane + 64 * u], x, h1[u]);
    }
#pragma unroll
    for (int u = 0; u < U; ++u) {
        h1[u] = fmaxf(h1[u], 0.0f);
        h2[u] = s.b2[lane + 64 * u];
    }
#pragma unroll
    for (int v = 0; v < U; ++v) {
        const int hv = __float_as_int(h1[v]);
#pragma unroll
        for (int i = 0; i < 64; ++i) {
            const float x = __int_as_float(__builtin_amdgcn_readlane(hv, i));
            const float *w = s.w2 + (64 * v + i) * H + lane;
#pragma unroll
            for (int u = 0; u < U; ++u) h2[u] = fmaf(w[64 * u], x, h2[u]);
        }
    }
    float z0 = 0.0f, z1 = 0.0f, z2 = 0.0f;
#pragma unroll
    for (int u = 0; u < U; ++u) {
        const float h = fmaxf(h2[u], 0.0f);
        const int j = lane + 64 * u;
        z0 = fmaf(s.w3[NH * j + 0], h, z0);
        z1 = fmaf(s.w3[NH * j + 1], h, z1);
        if (NH == 3) z2 = fmaf(s.w3[NH * j + 2], h, z2);
    }
    z0 = wave_sum(z0);
    z1 = wave_sum(z1);
    if (NH == 3) z2 = wave_sum(z2);
    tt = softplus_f32(z0 + a.b3_0);
    tp = softplus_f32(z1 + a.b3_1);
    nc = NH == 3 ? softplus_f32(z2 + a.b3_2) : 0.0f;
}

// Waves stride over the candidates of the chunk.  Workgroups past
// mlp_blocks, if any, run the chunk's quality rows instead (a wave per query),
// at the same time.
template <int H>
__global__ __launch_bounds__(256) void k_mlp_f32(MlpF32Args a) {
    if (static_cast<int>(blockIdx.x) >= a.mlp_blocks) {
        const int q = (blockIdx.x - a.mlp_blocks) * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
        if (q < a.quality.nq)
            quality_row_f32(a.quality, q, threadIdx.x & 63, a.quality.qmat + static_cast<size_t>(q) * a.quality.M);
        return;
    }
    __shared__ F32Weights<H> s;
    stage_f32<H>(a, s);
    __syncthreads();
    const int lane = threadIdx.x & 63;
    const long total = static_cast<long>(a.q.nq) * a.N;
    const long stride = static_cast<long>(a.mlp_blocks) * 4;
    for (long c = static_cast<long>(blockIdx.x) * 4 + __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
         c < total; c += stride) {
        const long q = c / a.N;
        const int d = static_cast<int>(c - q * a.N);
        float tt, tp, nc;
        predict_f32<H>(a, s, q, d, lane, tt, tp, nc);
        if (lane == 0) {                 // pair-major, as the epilogue reads it
            const size_t pm = static_cast<size_t>(d) * a.ldq + q;
            a.cand_ttft[pm] = tt;
            a.cand_tpot[pm] = tp;
            if (a.nheads == 3) a.cand_nout[pm] = nc;
        }
    }
}

// One wave per candidate, at most 1024 workgroups (each stages the weights once).
int mlp_f32_blocks(long candidates) {
    const long wgs = (candidates + 3) / 4;
    return static_cast<int>(wgs < 1024 ? (wgs < 1 ? 1 : wgs) : 1024);
}

hipError_t launch_mlp_f32(int H, const MlpF32Args &args, hipStream_t s) {
    MlpF32Args a = args;
    a.mlp_blocks = mlp_f32_blocks(static_cast<long>(a.q.nq) * a.N);
    const int qblocks = a.with_quality ? (a.quality.nq + 3) / 4 : 0;
    const dim3 grid(static_cast<unsigned>(a.mlp_blocks + qblocks));
    if (H == 64) return launch_kernel(k_mlp_f32<64>, grid, dim3(256), 0, s, a);
    if (H == 128) return launch_kernel(k_mlp_f32<128>, grid, dim3(256), 0, s, a);
    return hipErrorInvalidValue;
}

// ------------------------------------------------------------ feature gather
// Staged pipeline: X[d][q][0:32] (bf16, pair-major: for each pair the rows of
// consecutive queries are consecutive, which is how the staged predictor reads
// them) = the pair's feature row with the query's input-length slot filled
// in.  Each workgroup stages all pair rows in LDS once and broadcasts them
// over kGatherQ queries; consecutive threads write consecutive 16-byte pieces
// of one pair's kGatherQ-row block (16 KB contiguous per pair).  One
// workgroup per compute unit at 65,536 queries: streaming writes measured on
// this part reach their highest rate with one wave per SIMD.
__global__ __launch_bounds__(256) void k_gather(GatherArgs a) {
    extern __shared__ uint4 s_dep[];          // [N][4]
    __shared__ uint32_t s_xl[kGatherQ];
    const uint4 *g = reinterpret_cast<const uint4 *>(a.dep_bf16);
    for (int i = threadIdx.x; i < a.N * 4; i += blockDim.x) s_dep[i] = g[i];
    const int q0 = blockIdx.x * kGatherQ;
    if (threadIdx.x < kGatherQ && q0 + static_cast<int>(threadIdx.x) < a.q.nq)
        s_xl[threadIdx.x] = bf16_bits(len_feature(a.q.input_len[q0 + threadIdx.x]));
    __syncthreads();
    const int nqb = min(kGatherQ, a.q.nq - q0);
    const int per_d = nqb * 4;
    const int total = a.N * per_d;
    const int lpart = a.len_slot >> 3, lword = (a.len_slot & 7) >> 1, lhi = a.len_slot & 1;
    uint4 *X = reinterpret_cast<uint4 *>(a.X);
    for (int i = threadIdx.x; i < total; i += blockDim.x) {
        const int d = i / per_d;
        const int rem = i - d * per_d;
        const int qi = rem >> 2, part = rem & 3;
        uint4 v = s_dep[d * 4 + part];
        if (part == lpart) {
            const uint32_t xl = s_xl[qi];
            const uint32_t keep = lhi ? 0x0000FFFFu : 0xFFFF0000u;
            const uint32_t put = lhi ? (xl << 16) : xl;
            if (lword == 0) v.x = (v.x & keep) | put;
            if (lword == 1) v.y = (v.y & keep) | put;
            if (lword == 2) v.z = (v.z & keep) | put;
            if (lword == 3) v.w = (v.w & keep) | put;
        }
        X[(static_cast<size_t>(d) * a.ldq + q0 + qi) * 4 + part] = v;
    }
}

hipError_t launch_gather(const GatherArgs &a, hipStream_t s) {
    const unsigned grid = static_cast<unsigned>((a.q.nq + kGatherQ - 1) / kGatherQ);
    return launch_kernel(k_gather, dim3(grid), dim3(256), static_cast<uint32_t>(a.N) * 64, s, a);
}

// ------------------------------------------------------------ decision epilogue
// Per query: cost (Eq. 2), bound test and utility for every pair, then the
// Eq. 3 argmax -- once per cost weight (a lambda sweep; outputs are then
// [query][weight]).  Predictions are pair-major with 16-byte aligned pair
// rows: a workgroup takes kEpiQB consecutive queries, lane i of every wave
// the kEpiQL queries kEpiQL i .. kEpiQL i + kEpiQL - 1 of them (one load
// per pair and array, so each load of a wave reads 64 kEpiQL consecutive
// values of one pair's row), and wave w the pairs w, w + kEpiW, ... in
// increasing order.  The quality rows of the workgroup's queries are staged
// in LDS transposed ([model][query]), so the lane's values of one model are
// one LDS read; the pairs' models are staged too.  Each lane keeps the best
// candidate of each of its queries; the waves then compare packed decision
// keys through LDS (unique: they hold the pair index), and the wave holding
// the largest writes the outputs.  DBG also writes the caller's
// per-candidate outputs, [query][pair].  The predictions are read with
// non-temporal loads (each is read once), the first pair step's loads are
// issued before the LDS staging, and each later step's before the previous
// one is decided.  Shape measured at 65,536 x 256 (same box): two queries
// per lane and eight waves 31.6 us; four and sixteen 35.2 us; four and four
// 58.8 us; the two early loads took the chosen shape to 29.0 us and the
// step-ahead loads to 27.4 us (four pairs per step instead of two: 29.0 us
// without them, 31.3 us with).
constexpr int kEpiQL = 2;                  // queries per lane
typedef f32x2 EpiVec;                      // a lane's values of one pair: kEpiQL floats
constexpr int kEpiQB = 64 * kEpiQL;        // queries per workgroup
constexpr int kEpiW = 8;                   // waves per workgroup: pair classes mod kEpiW
constexpr int kEpiThreads = 64 * kEpiW;
constexpr int kEpiQS = kEpiQB + 4;         // LDS quality row stride (16-byte multiple, offset banks)
constexpr int kEpiUnroll = 2;              // pairs per wave loaded before any is used

template <bool PN, bool MULTI, bool GEN, bool DBG>
__global__ __launch_bounds__(kEpiThreads) void k_epilogue(EpilogueArgs a) {
    Rule rule = a.rule;
    if constexpr (!GEN) rule = Rule{};
    // [pair_stride(N)] models | [M][kEpiQS] quality | [kEpiW][kEpiQL][64 lanes] keys
    extern __shared__ __attribute__((aligned(16))) float s_ep[];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int32_t *s_model = reinterpret_cast<int32_t *>(s_ep);
    float *s_qt = s_ep + pair_stride(a.N);
    uint64_t *s_key = reinterpret_cast<uint64_t *>(s_qt + static_cast<size_t>(a.M) * kEpiQS);
    for (int i = tid; i < a.N; i += kEpiThreads) s_model[i] = a.dep_model[i];
    const int nq = a.q.nq;
    const int q0 = blockIdx.x * kEpiQB;
    const int nqb = min(kEpiQB, nq - q0);
    const int ql = kEpiQL * lane;              // the lane's first query, in the workgroup
    // lanes past the chunk's padded end read pair rows from their start
    const size_t col = q0 + ql < a.ldq ? static_cast<size_t>(q0 + ql) : 0;
    const size_t ld = static_cast<size_t>(a.ldq);
    auto load_step = [&](int d0, EpiVec (&t)[kEpiUnroll], EpiVec (&p)[kEpiUnroll], EpiVec (&v)[kEpiUnroll]) {
#pragma unroll
        for (int u = 0; u < kEpiUnroll; ++u) {
            const int d = d0 + kEpiW * u;
            const size_t ci = static_cast<size_t>(d < a.N ? d : 0) * ld + col;
            t[u] = __builtin_nontemporal_load(reinterpret_cast<const EpiVec *>(a.cand_ttft + ci));
            p[u] = __builtin_nontemporal_load(reinterpret_cast<const EpiVec *>(a.cand_tpot + ci));
            if constexpr (PN) v[u] = __builtin_nontemporal_load(reinterpret_cast<const EpiVec *>(a.cand_nout + ci));
        }
    };
    // the first pair step's predictions are requested before the staging
    EpiVec t0[kEpiUnroll], p0[kEpiUnroll], v0[kEpiUnroll];
    load_step(wave, t0, p0, v0);
    for (int i = tid; i < nqb * a.M; i += kEpiThreads) {
        const int r = i / a.M, m = i - r * a.M;
        s_qt[m * kEpiQS + r] = a.qmat[static_cast<size_t>(q0) * a.M + i];
    }
    __syncthreads();
    bool valid[kEpiQL];
    float nout[kEpiQL], slo[kEpiQL];
    int32_t len[kEpiQL];
#pragma unroll
    for (int j = 0; j < kEpiQL; ++j) {
        valid[j] = ql + j < nqb;
        const int qc = valid[j] ? q0 + ql + j : 0;
        const int32_t no = PN ? 0 : a.q.nout[qc];
        nout[j] = static_cast<float>(no < 0 ? 0 : no);
        slo[j] = a.q.slo ? a.q.slo[qc] : a.q.default_slo;
        len[j] = GEN ? a.q.input_len[qc] : 0;
    }
    const int nw = MULTI ? a.nw : 1;
    for (int kw = 0; kw < nw; ++kw) {
        QueryRule qrule[kEpiQL];
        Best best[kEpiQL];
#pragma unroll
        for (int j = 0; j < kEpiQL; ++j) {
            qrule[j] = query_rule(rule, slo[j], len[j], nout[j], a.w[kw]);
            best[j] = best_none();
        }
        for (int d0 = wave; d0 < a.N; d0 += kEpiW * kEpiUnroll) {
            EpiVec tv[kEpiUnroll], pv[kEpiUnroll], nv[kEpiUnroll];
#pragma unroll
            for (int u = 0; u < kEpiUnroll; ++u) {
                tv[u] = t0[u];
                pv[u] = p0[u];
                if constexpr (PN) nv[u] = v0[u];
            }
            // request the next step before deciding this one: this weight's
            // next pairs, else the next weight's first
            int dn = d0 + kEpiW * kEpiUnroll;
            bool more = dn < a.N;
            if (!more && kw + 1 < nw) {
                dn = wave;
                more = true;
            }
            if (more) load_step(dn, t0, p0, v0);
#pragma unroll
            for (int u = 0; u < kEpiUnroll; ++u) {
                const int d = d0 + kEpiW * u;
                if (d < a.N) {
                    const EpiVec qv = *reinterpret_cast<const EpiVec *>(s_qt + s_model[d] * kEpiQS + ql);
                    // every query of the lane is decided (a query past the
                    // chunk's end only reads padding, and is never written)
#pragma unroll
                    for (int j = 0; j < kEpiQL; ++j) {
                        const float nc = PN ? nv[u][j] : nout[j];
                        if (DBG && kw == 0 && valid[j]) {
                            const size_t co = static_cast<size_t>(q0 + ql + j) * a.N + d;
                            if (a.dbg_ttft) a.dbg_ttft[co] = tv[u][j];
                            if (a.dbg_tpot) a.dbg_tpot[co] = pv[u][j];
                            if (PN && a.dbg_nout) a.dbg_nout[co] = nc;
                        }
                        offer(best[j], decide(tv[u][j], pv[u][j], nc, rule, qrule[j], qv[j]), d, tv[u][j], pv[u][j], nc);
                    }
                }
            }
        }
        uint64_t key[kEpiQL];
#pragma unroll
        for (int j = 0; j < kEpiQL; ++j) {
            key[j] = best_key(best[j]);
            s_key[(wave * kEpiQL + j) * 64 + lane] = key[j];   // lane-contiguous: no bank conflicts
        }
        __syncthreads();
#pragma unroll
        for (int j = 0; j < kEpiQL; ++j) {
            uint64_t top = 0;
#pragma unroll
            for (int v = 0; v < kEpiW; ++v) {
                const uint64_t o = s_key[(v * kEpiQL + j) * 64 + lane];
                top = o > top ? o : top;
            }
            if (valid[j] && key[j] == top)
                write_outputs(a.out, (q0 + ql + j) * nw + kw, key[j], best[j].u, best[j].e2e, best[j].tt, best[j].tp,
                              best[j].n);
        }
        __syncthreads();                       // the next weight reuses the keys
    }
}

template <bool PN, bool MULTI, bool GEN, bool DBG>
static hipError_t launch_epilogue_t(const EpilogueArgs &a, dim3 g, size_t lds, hipStream_t s) {
    return launch_kernel(k_epilogue<PN, MULTI, GEN, DBG>, g, dim3(kEpiThreads), static_cast<uint32_t>(lds), s, a);
}

hipError_t launch_epilogue(const EpilogueArgs &a, hipStream_t s) {
    using Launch = hipError_t (*)(const EpilogueArgs &, dim3, size_t, hipStream_t);
    static const Launch table[16] = {
        launch_epilogue_t<false, false, false, false>, launch_epilogue_t<false, false, false, true>,
        launch_epilogue_t<false, false, true, false>, launch_epilogue_t<false, false, true, true>,
        launch_epilogue_t<false, true, false, false>, launch_epilogue_t<false, true, false, true>,
        launch_epilogue_t<false, true, true, false>, launch_epilogue_t<false, true, true, true>,
        launch_epilogue_t<true, false, false, false>, launch_epilogue_t<true, false, false, true>,
        launch_epilogue_t<true, false, true, false>, launch_epilogue_t<true, false, true, true>,
        launch_epilogue_t<true, true, false, false>, launch_epilogue_t<true, true, false, true>,
        launch_epilogue_t<true, true, true, false>, launch_epilogue_t<true, true, true, true>,
    };
    const unsigned grid = static_cast<unsigned>((a.q.nq + kEpiQB - 1) / kEpiQB);
    const size_t lds = (static_cast<size_t>(pair_stride(a.N)) + static_cast<size_t>(a.M) * kEpiQS) * 4 +
                       static_cast<size_t>(kEpiW) * kEpiQB * 8;
    const bool gen = a.rule.score_paper || a.rule.bound_paper;
    const bool dbg = a.dbg_ttft || a.dbg_tpot || a.dbg_nout;
    const int idx = (a.cand_nout ? 8 : 0) + (a.nw > 1 ? 4 : 0) + (gen ? 2 : 0) + (dbg ? 1 : 0);
    return table[idx](a, dim3(grid), lds, s);
}

// ------------------------------------------------------------ split merge
// When the pairs of a chunk are split over several workgroups, each writes
// its best key and values; this picks the maximum key per query.
__global__ __launch_bounds__(256) void k_merge(MergeArgs a) {
    const int q = blockIdx.x * blockDim.x + threadIdx.x;
    if (q >= a.nq) return;
    uint64_t best = 0;
    int bs = 0;
    for (int s = 0; s < a.nsplit; ++s) {
        const uint64_t k = a.part_key[static_cast<size_t>(s) * a.nq + q];
        if (k > best) {
            best = k;
            bs = s;
        }
    }
    const float *v = a.part_val + (static_cast<size_t>(bs) * a.nq + q) * kPartVals;
    write_outputs(a.out, q, best, v[0], v[1], v[2], v[3], v[4]);
}

hipError_t launch_merge(const MergeArgs &a, hipStream_t s) {
    return launch_kernel(k_merge, dim3((a.nq + 255) / 256), dim3(256), 0, s, a);
}

}  // namespace hwr

// ------------------------------------------------------------ feature log check
namespace {
__global__ __launch_bounds__(256) void k_feature_log(const double *x, double *y, int64_t n) {
    const int64_t i = static_cast<int64_t>(blockIdx.x) * 256 + threadIdx.x;
    if (i < n) y[i] = hwr::ln_pos(x[i]);
}
}  // namespace

extern "C" hwr_status hwr_probe_feature_log(int32_t device, const double *x, int64_t n, double *y) {
    if (!x || !y || device < 0 || n < 1 || n > (int64_t{1} << 26)) return HWR_ERR_INVALID_ARG;
    for (int64_t i = 0; i < n; ++i)
        if (!(x[i] >= DBL_MIN && x[i] <= DBL_MAX)) return HWR_ERR_INVALID_ARG;   // positive, finite, normal
    int prev = -1;
    hipError_t e = hipGetDevice(&prev);
    if (e == hipSuccess) e = hipSetDevice(device);
    double *dx = nullptr, *dy = nullptr;
    const size_t bytes = static_cast<size_t>(n) * sizeof(double);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&dx), bytes);
    if (e == hipSuccess) e = hipMalloc(reinterpret_cast<void **>(&dy), bytes);
    if (e == hipSuccess) e = hipMemcpy(dx, x, bytes, hipMemcpyHostToDevice);
    if (e == hipSuccess) {
        hipLaunchKernelGGL(k_feature_log, dim3(static_cast<unsigned>((n + 255) / 256)), dim3(256), 0, nullptr, dx, dy, n);
        e = hipGetLastError();
    }
    if (e == hipSuccess) e = hipMemcpy(y, dy, bytes, hipMemcpyDeviceToHost);
    if (dx) (void)hipFree(dx);
    if (dy) (void)hipFree(dy);
    if (prev >= 0) (void)hipSetDevice(prev);
    if (e == hipSuccess) return HWR_OK;
    return e == hipErrorOutOfMemory ? HWR_ERR_OOM : HWR_ERR_HIP;
}
