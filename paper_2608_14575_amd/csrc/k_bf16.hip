// bf16 MFMA kernels of libhwr (gfx950): the quality GEMM and the cost
// predictor with its decision epilogue.
//
// MFMA operand layouts (v_mfma_f32_32x32x16_bf16, wave64): A is 32 rows x 16
// k, B is 16 k x 32 columns; lane l holds 8 consecutive-in-k values of row
// (A) / column (B) l & 31, lane half l >> 5 selecting which 8 of the 16 k.
// The accumulator holds column l & 31 and rows crow(r, l >> 5), r = 0..15.
//
// The predictor computes every layer transposed, h^T = W^T x^T: rows are
// hidden units, columns are candidates.  An accumulator tile then holds, per
// lane, 16 hidden units of one candidate -- exactly the per-lane shape of the
// next layer's B operand -- so activations stay in registers from layer to
// layer; the weights (A operands) are re-laid-out on the host so that their k
// order matches the accumulator row order (see hwr_api.hip, pack_predictor).
#include <type_traits>

#include "hwr_device.hpp"

namespace hwr {

__device__ __forceinline__ f32x16 mfma32(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

// v_mfma_f32_16x16x32_bf16: A is 16 rows x 32 k, B 32 k x 16 columns; lane l
// holds 8 consecutive-in-k values of row (A) / column (B) l & 15, k-group
// l >> 4.  The accumulator holds column l & 15, rows 4 * (l >> 4) + 0..3.
__device__ __forceinline__ f32x4 mfma16(bf16x8 a, bf16x8 b, f32x4 c) {
    return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 bias_tile(const f32x4 *p) {
    const f32x4 a = p[0], b = p[1], c = p[2], d = p[3];
    return (f32x16){a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3],
                    c[0], c[1], c[2], c[3], d[0], d[1], d[2], d[3]};
}

// ReLU + bf16 rounding of accumulator elements [base, base + 8), packed as the
// 8 k-values of one B operand.
__device__ __forceinline__ bf16x8 relu_pack8(const f32x16 &c, int base) {
    u32x4 u;
    u[0] = __builtin_bit_cast(uint32_t, relu_bf16x2(c[base + 0], c[base + 1]));
    u[1] = __builtin_bit_cast(uint32_t, relu_bf16x2(c[base + 2], c[base + 3]));
    u[2] = __builtin_bit_cast(uint32_t, relu_bf16x2(c[base + 4], c[base + 5]));
    u[3] = __builtin_bit_cast(uint32_t, relu_bf16x2(c[base + 6], c[base + 7]));
    return __builtin_bit_cast(bf16x8, u);
}

// ------------------------------------------------------------ quality GEMM
// Q[q][m] = e_q . Wq[:, m] + bq[m] (Sec. 3.2 item 3), bf16 in, fp32 out.
// Each wave: 32 queries x 32 (padded) models.  Per 64-wide slice of the
// embedding, lane half h reads 64 contiguous bytes of its query row, as four
// k-blocks; Wq is pre-packed so that each lane's B operand for the same
// k-block is one contiguous 16-byte load.  The embedding stream dominates
// the traffic (HBM-bound, arithmetic intensity ~M flop/byte).  U slices are
// loaded before their MFMAs.  Large batches: four waves per workgroup and
// U = 1, which streams best.  Batches with fewer four-wave workgroups than
// compute units: one wave per workgroup (four times the compute units busy)
// and U = 4 (a quarter of the dependent memory round trips).  The MFMA chain
// runs over the slices in the same order either way: identical results.
template <int U>
__global__ __launch_bounds__(256) void k_quality_bf16(QualityArgs a) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int row = lane & 31, h = lane >> 5;
    const int q0 = (blockIdx.x * (blockDim.x >> 6) + wave) * 32;
    const int qa = q0 + row;
    const bool valid = qa < a.nq;
    const uint16_t *e = static_cast<const uint16_t *>(a.emb) +
                        static_cast<size_t>(valid ? qa : 0) * a.D + 32 * h;
    const bf16x8 *wq = reinterpret_cast<const bf16x8 *>(a.wq_pk) + lane;
    f32x16 acc = {};
    const int S = a.D / 64;
    const bf16x8 zero = {};
    int s = 0;
    for (; s + U <= S; s += U) {
        bf16x8 av[U][4], bv[U][4];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c) {
                av[u][c] = *reinterpret_cast<const bf16x8 *>(e + 64 * (s + u) + 8 * c);
                bv[u][c] = wq[((s + u) * 4 + c) * 64];
            }
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int c = 0; c < 4; ++c) acc = mfma32(valid ? av[u][c] : zero, bv[u][c], acc);
    }
    for (; s < S; ++s) {
        bf16x8 av[4], bv[4];
#pragma unroll
        for (int c = 0; c < 4; ++c) {
            av[c] = *reinterpret_cast<const bf16x8 *>(e + 64 * s + 8 * c);
            bv[c] = wq[(s * 4 + c) * 64];
        }
#pragma unroll
        for (int c = 0; c < 4; ++c) acc = mfma32(valid ? av[c] : zero, bv[c], acc);
    }
    const int m = lane & 31;
    if (m < a.M) {
        const float bias = a.bq[m];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const int q = q0 + crow(r, h);
            if (q < a.nq) a.qmat[static_cast<size_t>(q) * a.M + m] = acc[r] + bias;
        }
    }
}

// Large batches with D a multiple of 256: the workgroup (four waves, 64
// queries) streams its rows through LDS in slabs of 256 k (512 bytes per row),
// all four waves loading coalesced with the next slab prefetched in
// registers; waves 0 and 1 run the MFMA chains of the two 32-query tiles from
// LDS in the same k order as k_quality_bf16, so the results are identical.
// Each load instruction then covers two rows' 512 contiguous bytes instead of
// 16 bytes of 32 rows (3.6% faster on HBM-resident chunks).
constexpr int kQSlab = 256;                       // k per slab
constexpr int kQRows = 64;                        // queries per workgroup
__global__ __launch_bounds__(256) void k_quality_bf16_lds(QualityArgs a) {
    constexpr int RB = 2 * kQSlab + 16;           // LDS row stride in bytes (16-byte pad)
    constexpr int PPR = 2 * kQSlab / 16;          // 16-byte pieces per row per slab
    constexpr int PT = kQRows * PPR / 256;        // pieces per thread per slab
    __shared__ __attribute__((aligned(16))) unsigned char s_slab[kQRows * RB];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r0 = blockIdx.x * kQRows;
    const int nslab = a.D / kQSlab;
    const uint16_t *emb = static_cast<const uint16_t *>(a.emb);
    u32x4 pre[PT];
    auto load = [&](int j) {
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int p = tid + 256 * i, row = p / PPR, col = p % PPR;
            const int q = r0 + row < a.nq ? r0 + row : a.nq - 1;
            // plain loads: a chunk that is still in the last-level cache
            // (embeddings written just before routing) is read from there;
            // non-temporal loads would bypass it
            pre[i] = *reinterpret_cast<const u32x4 *>(emb + static_cast<size_t>(q) * a.D + j * kQSlab + col * 8);
        }
    };
    const int row = lane & 31, h = lane >> 5;
    const bf16x8 *wq = reinterpret_cast<const bf16x8 *>(a.wq_pk) + lane;
    f32x16 acc = {};
    load(0);
    for (int j = 0; j < nslab; ++j) {
#pragma unroll
        for (int i = 0; i < PT; ++i) {
            const int p = tid + 256 * i, rw = p / PPR, col = p % PPR;
            *reinterpret_cast<u32x4 *>(s_slab + rw * RB + col * 16) = pre[i];
        }
        __syncthreads();
        if (j + 1 < nslab) load(j + 1);
        if (wave < 2) {
            const unsigned char *base = s_slab + (32 * wave + row) * RB + 64 * h;
#pragma unroll
            for (int sl = 0; sl < kQSlab / 64; ++sl) {
                const int sg = j * (kQSlab / 64) + sl;
                bf16x8 av[4], bv[4];
#pragma unroll
                for (int c = 0; c < 4; ++c) {
                    av[c] = *reinterpret_cast<const bf16x8 *>(base + sl * 128 + 16 * c);
                    bv[c] = wq[(sg * 4 + c) * 64];
                }
#pragma unroll
                for (int c = 0; c < 4; ++c) acc = mfma32(av[c], bv[c], acc);
            }
        }
        __syncthreads();
    }
    if (wave < 2) {
        const int m = lane & 31;
        if (m < a.M) {
            const float bias = a.bq[m];
#pragma unroll
            for (int r = 0; r < 16; ++r) {
                const int q = r0 + 32 * wave + crow(r, h);
                if (q < a.nq) a.qmat[static_cast<size_t>(q) * a.M + m] = acc[r] + bias;
            }
        }
    }
}

hipError_t launch_quality_bf16(const QualityArgs &a, int cus, hipStream_t s) {
    const int grid = (a.nq + 127) / 128;
    if (grid < cus) return launch_kernel(k_quality_bf16<4>, dim3((a.nq + 31) / 32), dim3(64), 0, s, a);
    if (a.D % kQSlab == 0)
        return launch_kernel(k_quality_bf16_lds, dim3((a.nq + kQRows - 1) / kQRows), dim3(256), 0, s, a);
    return launch_kernel(k_quality_bf16<1>, dim3(grid), dim3(256), 0, s, a);
}


// ------------------------------------------------------------ predictor
// Eq. 1 cost predictor on MFMA tiles, for all (query, pair) candidates of a
// chunk.  A workgroup covers kQPerBlock queries; its waves form query groups
// of 32 * NT queries, two waves per group, and the two waves of a group split
// the workgroup's pair range in halves (their decision keys merge through LDS
// at the end).  NT = 2: 8 waves, two per SIMD, so that one wave's VALU
// epilogue overlaps the other's MFMAs.  NT = 4: 4 waves, one per SIMD, each
// holding twice the candidates, so that every weight fragment read from LDS
// feeds four MFMAs instead of two (half the LDS traffic per candidate); the
// first layer's activations then sit in the accumulation registers (AGPRs),
// which the MFMA reads directly.  Each wave steps through its pairs,
// evaluating NT x 32 candidates (one pair, 32 * NT queries) per step:
//   X^T  (32 features x 32 candidates, bf16)   built from the pair's feature
//        row (L1-resident) and each query's input-length feature;
//   h1^T = ReLU(W1^T X^T + b1)  -> bf16, registers;
//   h2^T = ReLU(W2^T h1^T + b2) -> bf16, per 32-row tile, each tile folded at
//   once into the head layer z = W3^T h2^T + b3, itself a chain of 16x16x32
//   MFMAs that leaves each candidate's heads in the lane that decides it;
//   TTFT = softplus(z0), TPOT = softplus(z1).
// The layers are software-pipelined: a tile's MFMAs are issued before the
// previous tile's VALU epilogue (bias, ReLU, bf16 packing), so the matrix
// pipe and the vector ALU overlap.  W1, W2 and W3 (A operands) and the biases
// (accumulator initial values) live in LDS.  After the heads, lane half h
// carries column tiles h, h + 2, ... (one query per lane and tile pair).
// Fused mode then applies Eq. 2, the bound test and the utility and keeps
// each query's best candidate (Eq. 3); staged mode reads X from HBM and
// writes TTFT/TPOT per candidate.  X and the staged outputs are pair-major
// (candidate (q, d) at d * nq + q): the 64 lanes of a wave, 64 consecutive
// queries, read whole rows and write 256 contiguous bytes.
template <int NT>
struct MlpShape {
    static constexpr int kWaves = NT == 4 ? 4 : 8;
    static constexpr int kThreads = 64 * kWaves;
    static constexpr int kQPW = 32 * NT;                 // queries per wave
    static constexpr int kQG = kQPerBlock / kQPW;        // query groups per workgroup
    static_assert(kWaves == 2 * kQG, "two waves (pair halves) per query group");
};

template <int H, bool STAGED, int NH, bool FB, int NT, bool LEAN = false>
__global__ __launch_bounds__(MlpShape<NT>::kThreads, 1) void k_mlp_bf16(MlpArgs a) {
    constexpr int MT = H / 32;     // 32-row tiles of a hidden layer
    constexpr int KB2 = H / 16;    // k-blocks of the second layer
    constexpr int NO = NT / 2;     // queries each lane decides (tiles h, h + 2, ...)
    constexpr int kThreads = MlpShape<NT>::kThreads;
    constexpr int kQPW = MlpShape<NT>::kQPW;
    constexpr int kQG = MlpShape<NT>::kQG;
    static_assert(NT == 2 || NT == 4, "two or four column tiles per wave");
    __shared__ bf16x8 s_w1[MT * 2 * 64];
    __shared__ bf16x8 s_w2[MT * KB2 * 64];
    __shared__ f32x4 s_b1[MT * 2 * 4];
    __shared__ f32x4 s_b2[MT * 2 * 4];
    constexpr int W3S = 2 * NH + 1;   // head fragments per k-block (last: zeros)
    __shared__ bf16x8 s_w3f[KB2 * W3S];
    __shared__ uint64_t s_mkey[kQPerBlock];
    __shared__ f32x4 s_mval[kQPerBlock];
    __shared__ float s_mnout[NH == 3 ? kQPerBlock : 1];
    const int tid = threadIdx.x;
    {
        // Every load of a staging round is issued before its first LDS
        // store: one memory round trip for W1, the biases and the head
        // fragments, then one per round of up to kStageRound W2 pieces per
        // thread (one round for 512 threads, two for 256).  Indices past an
        // array's end are clamped for the loads and skipped for the stores.
        constexpr int nW1 = MT * 2 * 64, nW2 = MT * KB2 * 64, nB = MT * 2 * 4, nW3 = KB2 * W3S;
        constexpr int pW1 = (nW1 + kThreads - 1) / kThreads;
        constexpr int pW2 = (nW2 + kThreads - 1) / kThreads;
        constexpr int pB = (nB + kThreads - 1) / kThreads;
        constexpr int pW3 = (nW3 + kThreads - 1) / kThreads;
        constexpr int kStageRound = 16;
        constexpr int rW2 = pW2 < kStageRound ? pW2 : kStageRound;
        static_assert(pW2 % rW2 == 0, "whole staging rounds");
        const uint4 *g1 = reinterpret_cast<const uint4 *>(a.w1_pk);
        const uint4 *g2 = reinterpret_cast<const uint4 *>(a.w2_pk);
        const uint4 *gb1 = reinterpret_cast<const uint4 *>(a.b1_pk);
        const uint4 *gb2 = reinterpret_cast<const uint4 *>(a.b2_pk);
        const uint4 *g3 = reinterpret_cast<const uint4 *>(a.w3_frag);
        uint4 v1[pW1], v2[rW2], vb1[pB], vb2[pB], v3[pW3];
        // W1, the biases and the head fragments first (one round trip), so
        // that nothing is held across the W2 rounds: otherwise the compiler
        // keeps W1 in scratch memory meanwhile
#pragma unroll
        for (int i = 0; i < pW1; ++i) {
            const int k = tid + i * kThreads;
            v1[i] = g1[k < nW1 ? k : 0];
        }
#pragma unroll
        for (int i = 0; i < pB; ++i) {
            const int k = tid + i * kThreads;
            vb1[i] = gb1[k < nB ? k : 0];
            vb2[i] = gb2[k < nB ? k : 0];
        }
#pragma unroll
        for (int i = 0; i < pW3; ++i) {
            const int k = tid + i * kThreads;
            v3[i] = g3[k < nW3 ? k : 0];
        }
#pragma unroll
        for (int i = 0; i < pW1; ++i) {
            const int k = tid + i * kThreads;
            if (k < nW1) reinterpret_cast<uint4 *>(s_w1)[k] = v1[i];
        }
#pragma unroll
        for (int i = 0; i < pB; ++i) {
            const int k = tid + i * kThreads;
            if (k < nB) {
                reinterpret_cast<uint4 *>(s_b1)[k] = vb1[i];
                reinterpret_cast<uint4 *>(s_b2)[k] = vb2[i];
            }
        }
#pragma unroll
        for (int i = 0; i < pW3; ++i) {
            const int k = tid + i * kThreads;
            if (k < nW3) reinterpret_cast<uint4 *>(s_w3f)[k] = v3[i];
        }
#pragma unroll
        for (int r = 0; r < pW2 / rW2; ++r) {
#pragma unroll
            for (int i = 0; i < rW2; ++i) {
                const int k = tid + (r * rW2 + i) * kThreads;
                v2[i] = g2[k < nW2 ? k : 0];
            }
#pragma unroll
            for (int i = 0; i < rW2; ++i) {
                const int k = tid + (r * rW2 + i) * kThreads;
                if (k < nW2) reinterpret_cast<uint4 *>(s_w2)[k] = v2[i];
            }
        }
    }
    __syncthreads();

    // (the wave index is uniform: kept in scalar registers, so are the
    // pair loop and the per-pair table reads)
    const int lane = tid & 63, wave = __builtin_amdgcn_readfirstlane(tid >> 6), n = lane & 31, h = lane >> 5;
    const int qw = wave % kQG, grp = wave / kQG;
    const int nq = a.q.nq;
    const int qbase = blockIdx.x * kQPerBlock + qw * kQPW;
    // LEAN: the default decision rule (normalised score, the query's own
    // bound) and no per-candidate outputs, so that the decision code is
    // straight-line
    Rule rule = a.rule;
    if constexpr (LEAN) rule = Rule{};
    // every lane builds features for all column tiles ...
    int qc[NT];
    uint32_t xl[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int q = qbase + 32 * t + n;
        qc[t] = q < nq ? q : 0;
        xl[t] = bf16_bits(len_feature(a.q.input_len[qc[t]]));
        // keep the feature in a register: otherwise the fp64 log is
        // recomputed inside the pair loop
        asm volatile("" : "+v"(xl[t]));
    }
    // ... and decides for column tiles h, h + 2, ... only (queries qme[j])
    int qme[NO], qmc[NO];
    bool vme[NO];
    float nout[NO];
    QueryRule qrule[NO];
    const float *qrow[NO];
#pragma unroll
    for (int j = 0; j < NO; ++j) {
        qme[j] = qbase + 32 * (2 * j + h) + n;
        vme[j] = qme[j] < nq;
        qmc[j] = vme[j] ? qme[j] : 0;
        const int32_t nomy = a.q.nout ? a.q.nout[qmc[j]] : 0;   // given N_out (two heads)
        nout[j] = static_cast<float>(nomy < 0 ? 0 : nomy);
        qrule[j] = query_rule(rule, a.q.slo ? a.q.slo[qmc[j]] : a.q.default_slo,
                              a.q.input_len[qmc[j]], nout[j], a.w);
        qrow[j] = a.qmat + static_cast<size_t>(qmc[j]) * a.M;
    }
    // the input-length slot: k-block, lane half and element holding it
    const int ls_kb = a.len_slot >> 4, ls_h = (a.len_slot >> 3) & 1, ls_e = a.len_slot & 7;
    const bool patch = (h == ls_h);

    const int split = STAGED ? 0 : blockIdx.y;
    const int nsplit = STAGED ? 1 : a.nsplit;
    const long span0 = static_cast<long>(a.N) * split / nsplit;
    const long span1 = static_cast<long>(a.N) * (split + 1) / nsplit;
    const int d0 = static_cast<int>(span0 + (span1 - span0) * grp / 2);
    const int d1 = static_cast<int>(span0 + (span1 - span0) * (grp + 1) / 2);

    Best best[NO];
#pragma unroll
    for (int j = 0; j < NO; ++j) best[j] = best_none();

    // Head-layer A fragment of this lane for column tile t (an index into a
    // k-block's fragments): lane 16g + i holds row i, k-group g.  Row
    // i = 8(t & 1) + 4s + m is head m of sub-column s; it takes weights only
    // from the k-groups whose B lanes carry sub-column s (g & 1 == s), namely
    // the hidden-unit half g >> 1.  Every other lane reads the zero fragment.
    // Tiles t and t ^ 1 share one head accumulator, acc3[t >> 1].
    int w3_sel[2];
    {
        const int i = lane & 15, g = lane >> 4, m = i & 3, s = (i >> 2) & 1;
#pragma unroll
        for (int t = 0; t < 2; ++t)
            w3_sel[t] = ((i >> 3) == t && m < NH && (g & 1) == s) ? m * 2 + (g >> 1) : 2 * NH;
    }

    // Per-pair inputs are loaded one step ahead: the pair's feature row
    // (fused) or the candidates' feature rows (staged), and the quality
    // Q[query][model(pair)], whose address needs a scalar load first.
    const bf16x8 *dep = reinterpret_cast<const bf16x8 *>(a.dep_bf16);
    const int dfirst = d0 < d1 ? d0 : 0;
    constexpr int NR = STAGED ? NT : 1;   // feature rows loaded per step
    // staged four-tile form: the next step's rows are loaded once the first
    // layer has consumed this step's (they share registers), in the
    // second layer's shadow
    constexpr bool kLateX = STAGED && NT == 4;
    bf16x8 nr[NR][2];
    auto load_x = [&](int dn) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const bf16x8 *xr = reinterpret_cast<const bf16x8 *>(
                a.X + (static_cast<size_t>(dn) * a.ldq + qc[t]) * kFeatPad);
            nr[t][0] = xr[h];
            nr[t][1] = xr[2 + h];
        }
    };
    if constexpr (STAGED) {
        load_x(dfirst);
    } else {
        nr[0][0] = dep[dfirst * 4 + h];
        nr[0][1] = dep[dfirst * 4 + 2 + h];
    }
    float nq_val[NO];
#pragma unroll
    for (int j = 0; j < NO; ++j) nq_val[j] = STAGED ? 0.0f : qrow[j][a.dep_model[dfirst]];

    // TTFT, TPOT and N_out (the third head's prediction in tokens, else
    // the query's given value) from the head-layer sums of own query j
    auto head_values = [&](int j, float z0, float z1, float z2, float &tt, float &tp, float &nc) {
        tt = softplus_fast(z0 + a.b3_0);
        tp = softplus_fast(z1 + a.b3_1);
        nc = NH == 3 ? softplus_fast(z2 + a.b3_2) : nout[j];
    };
    // per-candidate outputs when requested, then cost, bound test,
    // utility and the running argmax (Eq. 2, Eq. 3) of own query j
    auto take_candidate = [&](int j, int dd, float tt, float tp, float nc, float Q) {
        const size_t ci = a.cand_pm ? static_cast<size_t>(dd) * a.ldq + qmc[j] : static_cast<size_t>(qmc[j]) * a.N + dd;
        if (!LEAN && a.cand_ttft && vme[j]) {
            a.cand_ttft[ci] = tt;
            a.cand_tpot[ci] = tp;
        }
        if (!LEAN && a.cand_nout && vme[j]) a.cand_nout[ci] = nc;
        offer<NH == 3>(best[j], decide(tt, tp, nc, rule, qrule[j], Q), dd, tt, tp, nc);
    };
    // four-tile form: head sums and quality of the previous pair step,
    // decided during the next step (pd < 0: none pending)
    float pz[NO][NH], pQ[NO];
    int pd = -1;
#pragma unroll
    for (int j = 0; j < NO; ++j) {
        pQ[j] = 0.0f;
#pragma unroll
        for (int m = 0; m < NH; ++m) pz[j][m] = 0.0f;
    }

    for (int d = d0; d < d1; ++d) {
        bf16x8 cr[NR][2];
#pragma unroll
        for (int t = 0; t < NR; ++t) {
            cr[t][0] = nr[t][0];
            cr[t][1] = nr[t][1];
        }
        float Qd[NO];
#pragma unroll
        for (int j = 0; j < NO; ++j) Qd[j] = nq_val[j];
        {
            const int dn = d + 1 < d1 ? d + 1 : d;
            if constexpr (STAGED) {
                if constexpr (!kLateX) load_x(dn);
            } else {
                nr[0][0] = dep[dn * 4 + h];
                nr[0][1] = dep[dn * 4 + 2 + h];
                const int mdn = a.dep_model[dn];
#pragma unroll
                for (int j = 0; j < NO; ++j) nq_val[j] = qrow[j][mdn];
            }
        }
        // LDS offsets made opaque per step: the weight fragments are
        // loop-invariant, and hoisting all of them out of the pair loop would
        // need far more registers than a lane has.
        int lo = lane, ho = h, w3o0 = w3_sel[0], w3o1 = w3_sel[1];
        asm volatile("" : "+v"(lo), "+v"(ho), "+v"(w3o0), "+v"(w3o1));
        // ---- features (Eq. 1), B operand of layer 1
        bf16x8 xf[NT][2];
        if constexpr (STAGED) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                xf[t][0] = cr[t][0];
                xf[t][1] = cr[t][1];
            }
        } else {
            const bf16x8 r0 = cr[0][0], r1 = cr[0][1];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                if constexpr (NT == 4) {
                    // the launcher takes this form only with the slot in
                    // k-block 0: the second k-block is the same for every tile
                    xf[t][0] = patch ? put_elem(r0, ls_e, xl[t]) : r0;
                    xf[t][1] = r1;
                } else {
                    xf[t][0] = (patch && ls_kb == 0) ? put_elem(r0, ls_e, xl[t]) : r0;
                    xf[t][1] = (patch && ls_kb == 1) ? put_elem(r1, ls_e, xl[t]) : r1;
                }
            }
        }
        // ---- layers 1 and 2, software-pipelined: the VALU epilogue of row
        // tile i-1 (ReLU, bf16 rounding, head dot products) is issued between
        // the first and the remaining MFMAs of row tile i, so it runs while
        // those MFMAs occupy the matrix pipe.  The fences keep that order
        // (the scheduler would otherwise cluster the epilogues after the
        // MFMAs); LDS and global reads may still move across them.
        constexpr int kFence = 0x100 | 0x020;   // DS reads, VMEM reads may cross
        bf16x8 h1[NT][KB2];
        f32x16 acc[2][NT];
        auto l1_mfma = [&](int mt, f32x16 (&c)[NT]) {
            // FB: b1 enters through the folded-bias feature slots
            const f32x16 bi = FB ? f32x16{} : bias_tile(s_b1 + (mt * 2 + ho) * 4);
#pragma unroll
            for (int t = 0; t < NT; ++t) c[t] = bi;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const bf16x8 w = s_w1[(mt * 2 + kb) * 64 + lo];
#pragma unroll
                for (int t = 0; t < NT; ++t) c[t] = mfma32(w, xf[t][kb], c[t]);
            }
        };
        // (the empty asm statements pin each epilogue's results at this
        // point: otherwise IR passes sink the pure ReLU / dot-product chains
        // to their last use, past the fences, and the registers overflow.
        // With four column tiles they also place the first layer's
        // activations in the accumulation registers, read by the MFMAs of
        // the second layer as their B operand.)
        auto l1_epi = [&](int mt, const f32x16 (&c)[NT]) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                h1[t][2 * mt] = relu_pack8(c[t], 0);
                h1[t][2 * mt + 1] = relu_pack8(c[t], 8);
                if constexpr (NT == 4) {
                    asm volatile("" : "+a"(h1[t][2 * mt]), "+a"(h1[t][2 * mt + 1]));
                } else {
                    asm volatile("" : "+v"(h1[t][2 * mt]), "+v"(h1[t][2 * mt + 1]));
                }
            }
        };
        auto l2_mfma = [&](int mo, int kb0, int kb1, f32x16 (&c)[NT]) {
            if (kb0 == 0) {
                const f32x16 bi = bias_tile(s_b2 + (mo * 2 + ho) * 4);
#pragma unroll
                for (int t = 0; t < NT; ++t) c[t] = bi;
            }
#pragma unroll
            for (int kb = kb0; kb < kb1; ++kb) {
                const bf16x8 w = s_w2[(mo * KB2 + kb) * 64 + lo];
#pragma unroll
                for (int t = 0; t < NT; ++t) c[t] = mfma32(w, h1[t][kb], c[t]);
            }
        };
        // Head layer on the matrix pipe: z = W3^T h2^T on 16x16x32 tiles (the
        // heads need few rows, and this shape takes the same B operand as the
        // 32x32x16 one in half the cycles).  A 16x16x32 B operand reads lanes
        // j, j + 16, j + 32, j + 48 as its column j: candidates j and j + 16 of
        // the column tile, each split over two lanes (hidden-unit halves).  The
        // A fragments (see w3_sel) keep them apart: tile t's row
        // 8(t & 1) + 4s + m is head m of candidate 32t + 16s + j, so after
        // tiles t and t ^ 1 every lane holds its own candidate's heads in
        // accumulator elements 0..NH-1 of acc3[t >> 1].  One fragment read
        // serves the tiles of every accumulator.  (Packed bf16 dot products
        // would stall the matrix pipe: they do not co-issue with MFMA on
        // gfx950.)
        f32x4 acc3[NO];
#pragma unroll
        for (int j = 0; j < NO; ++j) acc3[j] = f32x4{};
        auto l2_epi = [&](int mo, const f32x16 (&c)[NT]) {
            bf16x8 h2[NT][2];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                h2[t][0] = relu_pack8(c[t], 0);
                h2[t][1] = relu_pack8(c[t], 8);
            }
#pragma unroll
            for (int b = 0; b < 2; ++b) {
                const int kb = 2 * mo + b;
                const bf16x8 f0 = s_w3f[kb * W3S + w3o0], f1 = s_w3f[kb * W3S + w3o1];
#pragma unroll
                for (int j = 0; j < NO; ++j) {
                    acc3[j] = mfma16(f0, h2[2 * j][b], acc3[j]);
                    acc3[j] = mfma16(f1, h2[2 * j + 1][b], acc3[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < NO; ++j) asm volatile("" : "+v"(acc3[j]));
        };
        // MFMA k-steps of tile mo issued before the previous epilogue.  For
        // mo = 0 that epilogue produces layer-1 k-blocks KB2-2 and KB2-1, so
        // the head steps must stop short of them.
        constexpr int kHead = KB2 - 2 < 4 ? KB2 - 2 : 4;
        if constexpr (NT == 4) {
            // One wave per SIMD: the matrix pipe and the vector ALU overlap
            // only where this wave's own instruction stream interleaves them,
            // and LDS latency is hidden only by loading fragments ahead, so
            // both phases below are scheduled by hand (a fence after every
            // MFMA slot).  Phase A runs the first layer together with the
            // second layer's row tile 0, whose k-blocks become available two
            // at a time.  Phase B runs the second layer's other row tiles,
            // each with the previous tile's epilogue interleaved, its weight
            // fragments streamed through a ring of kRing fragments loaded
            // kRing k-steps ahead.  Measured on one wave per SIMD: an MFMA
            // 32x32x16 issues every ~34 cycles with four independent
            // accumulators; v_cvt_pk_bf16_f32 costs ~7 issue cycles,
            // v_pk_max_i16 ~5 and v_accvgpr_write ~6, so phase A is bound by
            // its epilogue's vector work and phase B by the MFMA issue rate.
            constexpr int kRing = 3;
            constexpr int kFull = 0;             // nothing crosses
            f32x16 a1[NT];                       // first-layer row tile in flight
            bf16x8 w1c0[2];                      // its W1 fragments
            auto l1_tile = [&](int mt, int t, const bf16x8 (&w)[2]) {
                a1[t] = FB ? f32x16{} : bias_tile(s_b1 + (mt * 2 + ho) * 4);
                a1[t] = mfma32(w[0], xf[t][0], a1[t]);
                a1[t] = mfma32(w[1], xf[t][1], a1[t]);
            };
            // Phase A, scheduled by hand, one iteration per first-layer row
            // tile mt, 16 MFMA slots each with one sixth of the epilogue of
            // row tile mt (per tile t: four slots, two ReLU + bf16 pairs
            // each, and the move of every finished fragment into the
            // accumulation registers).  The MFMAs of a slot: tile 3 of row
            // tile mt (held back from the previous iteration), tiles 0-2 of
            // row tile mt + 1 (each after its tile's epilogue has read the
            // accumulator), and the second layer's row tile 0 over the
            // k-blocks of row tile mt - 1.  Weight fragments are loaded one
            // iteration ahead; a fence after every slot keeps the order.
            bf16x8 w1n[2], w2n[2];
            {
                const bf16x8 w[2] = {s_w1[0 * 64 + lo], s_w1[1 * 64 + lo]};
                w1n[0] = s_w1[2 * 64 + lo];
                w1n[1] = s_w1[3 * 64 + lo];
                w2n[0] = s_w2[0 * 64 + lo];
                w2n[1] = s_w2[1 * 64 + lo];
                const f32x16 bi = bias_tile(s_b2 + (0 * 2 + ho) * 4);
#pragma unroll
                for (int t = 0; t < NT; ++t) acc[0][t] = bi;
                w1c0[0] = w[0];
                w1c0[1] = w[1];
#pragma unroll
                for (int t = 0; t < NT - 1; ++t) l1_tile(0, t, w);
            }
            __builtin_amdgcn_sched_barrier(kFull);
#pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                const bf16x8 w1c[2] = {w1n[0], w1n[1]};      // row tile mt + 1
                const bf16x8 w2c[2] = {w2n[0], w2n[1]};      // row tile 0, k-blocks 2mt - 2, 2mt - 1
                const bf16x8 w1m[2] = {w1c0[0], w1c0[1]};    // row tile mt (its tile 3)
                if (mt + 2 < MT) {
                    w1n[0] = s_w1[((mt + 2) * 2 + 0) * 64 + lo];
                    w1n[1] = s_w1[((mt + 2) * 2 + 1) * 64 + lo];
                }
                if (mt >= 1) {                   // row tile 0, k-blocks 2mt, 2mt + 1 next
                    w2n[0] = s_w2[(2 * mt + 0) * 64 + lo];
                    w2n[1] = s_w2[(2 * mt + 1) * 64 + lo];
                }
                w1c0[0] = w1c[0];
                w1c0[1] = w1c[1];
                u32x4 hv[2];
#pragma unroll
                for (int sl = 0; sl < 16; ++sl) {
                    const int t = sl / 4, part = sl % 4;
                    // MFMA of this slot
                    if (sl == 0 || sl == 1) {
                        const int kb = sl;
                        if (kb == 0) a1[NT - 1] = FB ? f32x16{} : bias_tile(s_b1 + (mt * 2 + ho) * 4);
                        a1[NT - 1] = mfma32(w1m[kb], xf[NT - 1][kb], a1[NT - 1]);
                    } else if (part >= 2) {
                        if (mt > 0) {
                            const int b = sl >= 8 ? 1 : 0;
                            const int tt = (sl % 8 < 4 ? 0 : 2) + (part - 2);
                            acc[0][tt] = mfma32(w2c[b], h1[tt][2 * mt - 2 + b], acc[0][tt]);
                        }
                    } else if (mt + 1 < MT) {        // part 0 or 1, slots 4.. : row tile mt + 1, tile t - 1
                        const int tt = t - 1, kb = part;
                        if (kb == 0) a1[tt] = FB ? f32x16{} : bias_tile(s_b1 + ((mt + 1) * 2 + ho) * 4);
                        a1[tt] = mfma32(w1c[kb], xf[tt][kb], a1[tt]);
                    }
                    __builtin_amdgcn_sched_barrier(kFull);
                    // epilogue of row tile mt, tile t: fragment part / 2,
                    // pairs 2 (part % 2) .. + 1
                    {
                        const int fr = part / 2, p0 = 2 * (part % 2);
#pragma unroll
                        for (int q = 0; q < 2; ++q) {
                            const int e = 4 * fr + p0 + q;
                            hv[fr][p0 + q] = __builtin_bit_cast(uint32_t, relu_bf16x2(a1[t][2 * e], a1[t][2 * e + 1]));
                        }
                        if (part % 2 == 1) {
                            h1[t][2 * mt + fr] = __builtin_bit_cast(bf16x8, hv[fr]);
                            asm volatile("" : "+a"(h1[t][2 * mt + fr]));
                        }
                    }
                    __builtin_amdgcn_sched_barrier(kFull);
                }
            }
            // the last two k-blocks of row tile 0; the phase-B ring and the
            // bias of row tile 1 are loaded first
            if constexpr (kLateX) load_x(d + 1 < d1 ? d + 1 : d);
            bf16x8 ring[kRing];
            auto w2idx = [&](int i) { return s_w2[(KB2 + i) * 64 + lo]; };   // row tiles 1.. in order
#pragma unroll
            for (int i = 0; i < kRing; ++i) ring[i] = w2idx(i);
            f32x16 bnext = bias_tile(s_b2 + (1 * 2 + ho) * 4);
#pragma unroll
            for (int b = 0; b < 2; ++b)
#pragma unroll
                for (int t = 0; t < NT; ++t) acc[0][t] = mfma32(w2n[b], h1[t][KB2 - 2 + b], acc[0][t]);
            __builtin_amdgcn_sched_barrier(kFull);
            // Phase B, scheduled by hand: every MFMA of row tile mo is
            // followed by one slot of work on row tile mo - 1 (slot
            // s = 4 kb + t): slots 0-31 take the ReLU and bf16 rounding of
            // one element pair each (tile s / 8, pair s % 8), slots 8-11 load
            // the head fragments, and the head MFMAs follow once their tiles'
            // activations are complete.  With 64 slots per row tile (H = 256)
            // they take slots 32-39; with 32 (H = 128) the head MFMAs of tiles
            // 0-1 take slots 16-19 and those of tiles 2-3, whose activations
            // complete at the row tile's last slot, slots 0-3 of the next row
            // tile (their activations and fragments carried over).  Either
            // way each head accumulator takes its contributions in the order
            // of the other form.  The next row tile's bias is loaded at
            // k-step 1.  A scheduling fence after every slot keeps this order.
            constexpr int kSteps = (MT - 1) * KB2;
            constexpr int kSlots = KB2 * NT;
            constexpr bool kWide = kSlots >= 40 + 8 * NO;
            static_assert(kWide || kSlots == 32, "four-tile slot maps: H = 256 or H = 128");
            constexpr int kDec0 = kWide ? 40 : 20;      // first decision slot
            constexpr int kDecStride = kWide ? 8 : 4;   // slots per own query's decision
            float dtt[NO], dtp[NO], dnc[NO];
            u32x4 h2c[2][2];                     // narrow: tiles 2-3 of the previous row tile [par][b]
            bf16x8 f3c[2][2];                    // narrow: their head fragments [b][par]
            auto epi_pair = [&](const f32x16 &v, int e) {
                return __builtin_bit_cast(uint32_t, relu_bf16x2(v[2 * e], v[2 * e + 1]));
            };
            // row tile mo of phase B; DEC: with the previous pair step's
            // decisions in its slots kDec0 .. (one own query per kDecStride
            // slots, in pieces: TTFT, TPOT, N_out, decision)
            auto row_tile = [&](auto mo_c, auto dec_c) {
                constexpr int mo = decltype(mo_c)::value;
                constexpr bool DEC = decltype(dec_c)::value;
                f32x16 (&c)[NT] = acc[mo & 1];
                const f32x16 (&pv)[NT] = acc[(mo - 1) & 1];
                const f32x16 bi = bnext;
                u32x4 h2u[NT][2];
                bf16x8 f3[2][2];                 // head fragments [k-block half b][tile parity]
#pragma unroll
                for (int kb = 0; kb < KB2; ++kb) {
                    const int i = (mo - 1) * KB2 + kb;
                    const bf16x8 w = ring[i % kRing];
                    if (i + kRing < kSteps) ring[i % kRing] = w2idx(i + kRing);
                    if (kb == 1 && mo + 1 < MT) bnext = bias_tile(s_b2 + ((mo + 1) * 2 + ho) * 4);
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
                        c[t] = mfma32(w, h1[t][kb], kb == 0 ? bi : c[t]);
                        __builtin_amdgcn_sched_barrier(kFull);
                        const int sl = 4 * kb + t;
                        if (sl < 32) {
                            const int tt = sl / 8, e = sl % 8;
                            h2u[tt][e / 4][e % 4] = epi_pair(pv[tt], e);
                        }
                        if (sl >= 8 && sl < 12) {
                            const int b = (sl - 8) / 2, par = (sl - 8) % 2;
                            const int kh = 2 * (mo - 1) + b;
                            f3[b][par] = s_w3f[kh * W3S + (par ? w3o1 : w3o0)];
                        }
                        // acc3[j]: (b 0, tile 2j), (b 0, tile 2j + 1), (b 1, 2j), (b 1, 2j + 1)
                        if (kWide && sl >= 32 && sl < 40) {
                            const int j = (sl - 32) / 4, r = (sl - 32) % 4, b = r / 2, par = r % 2;
                            acc3[j] = mfma16(f3[b][par], __builtin_bit_cast(bf16x8, h2u[2 * j + par][b]), acc3[j]);
                        }
                        if (!kWide && sl >= 16 && sl < 20) {
                            const int r = sl - 16, b = r / 2, par = r % 2;
                            acc3[0] = mfma16(f3[b][par], __builtin_bit_cast(bf16x8, h2u[par][b]), acc3[0]);
                        }
                        if (!kWide && mo >= 2 && sl < 4) {
                            const int b = sl / 2, par = sl % 2;
                            acc3[1] = mfma16(f3c[b][par], __builtin_bit_cast(bf16x8, h2c[par][b]), acc3[1]);
                        }
                        if constexpr (DEC) {
                            if (sl >= kDec0 && sl < kDec0 + kDecStride * NO && (sl - kDec0) % kDecStride < 4) {
                                const int j = (sl - kDec0) / kDecStride, piece = (sl - kDec0) % kDecStride;
                                if (pd >= 0) {
                                    if (piece == 0) dtt[j] = softplus_fast(pz[j][0] + a.b3_0);
                                    if (piece == 1) dtp[j] = softplus_fast(pz[j][1] + a.b3_1);
                                    if (piece == 2) dnc[j] = NH == 3 ? softplus_fast(pz[j][NH - 1] + a.b3_2) : nout[j];
                                    if (piece == 3) take_candidate(j, pd, dtt[j], dtp[j], dnc[j], pQ[j]);
                                }
                            }
                        }
                        __builtin_amdgcn_sched_barrier(kFull);
                    }
                }
                if constexpr (!kWide) {
#pragma unroll
                    for (int par = 0; par < 2; ++par)
#pragma unroll
                        for (int b = 0; b < 2; ++b) {
                            h2c[par][b] = h2u[2 + par][b];
                            f3c[b][par] = f3[b][par];
                        }
                }
            };
            // row tiles 1 .. MT - 1 (compile-time indices); the decisions of
            // the previous pair step ride in row tile 1
            auto run_tiles = [&](auto self, auto mo_c) {
                constexpr int mo = decltype(mo_c)::value;
                if constexpr (mo < MT) {
                    row_tile(mo_c, std::integral_constant<bool, mo == 1 && !STAGED>{});
                    self(self, std::integral_constant<int, mo + 1>{});
                }
            };
            run_tiles(run_tiles, std::integral_constant<int, 1>{});
            if constexpr (!kWide) {
                // tiles 2-3 of row tile MT - 2, before row tile MT - 1's heads
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int b = r / 2, par = r % 2;
                    acc3[1] = mfma16(f3c[b][par], __builtin_bit_cast(bf16x8, h2c[par][b]), acc3[1]);
                }
            }
            l2_epi(MT - 1, acc[(MT - 1) & 1]);
        } else {
            // layer 1: MFMAs of tile mt, then the epilogue of tile mt - 1
    #pragma unroll
            for (int mt = 0; mt < MT; ++mt) {
                l1_mfma(mt, acc[mt & 1]);
                if (mt > 0) {
                    __builtin_amdgcn_sched_barrier(kFence);
                    l1_epi(mt - 1, acc[(mt - 1) & 1]);
                    __builtin_amdgcn_sched_barrier(kFence);
                }
            }
            // layer 2: first k-steps of tile mo, epilogue of the previous tile
            // (layer-1 tile MT-1 for mo = 0), then the remaining k-steps
    #pragma unroll
            for (int mo = 0; mo < MT; ++mo) {
                const int cur = (MT + mo) & 1, prev = (MT + mo - 1) & 1;
                l2_mfma(mo, 0, kHead, acc[cur]);
                __builtin_amdgcn_sched_barrier(kFence);
                if (mo == 0) l1_epi(MT - 1, acc[prev]);
                else l2_epi(mo - 1, acc[prev]);
                __builtin_amdgcn_sched_barrier(kFence);
                l2_mfma(mo, kHead, KB2, acc[cur]);
            }
            l2_epi(MT - 1, acc[(2 * MT - 1) & 1]);
        }
        // ---- heads: lane half h completes column tiles h, h + 2, ... (its
        // partner lane holds the other half of the same candidates' hidden
        // units).  The four-tile fused form defers this to the next pair
        // step, where it runs in the second layer's MFMA shadow.
        if constexpr (NT == 4 && !STAGED) {
#pragma unroll
            for (int j = 0; j < NO; ++j) {
#pragma unroll
                for (int m = 0; m < NH; ++m) pz[j][m] = acc3[j][m];
                pQ[j] = Qd[j];
            }
            pd = d;
        } else {
#pragma unroll
            for (int j = 0; j < NO; ++j) {
                float tt, tp, nc;
                head_values(j, acc3[j][0], acc3[j][1], NH == 3 ? acc3[j][2] : 0.0f, tt, tp, nc);
                if constexpr (STAGED) {
                    const size_t ci = static_cast<size_t>(d) * a.ldq + qmc[j];   // pair-major
                    if (vme[j]) {
                        a.cand_ttft[ci] = tt;
                        a.cand_tpot[ci] = tp;
                        if (NH == 3) a.cand_nout[ci] = nc;
                    }
                } else {
                    take_candidate(j, d, tt, tp, nc, Qd[j]);
                }
            }
        }
    }
    if constexpr (NT == 4 && !STAGED) {
        if (pd >= 0) {
#pragma unroll
            for (int j = 0; j < NO; ++j) {
                float tt, tp, nc;
                head_values(j, pz[j][0], pz[j][1], NH == 3 ? pz[j][2] : 0.0f, tt, tp, nc);
                take_candidate(j, pd, tt, tp, nc, pQ[j]);
            }
        }
    }
    if constexpr (!STAGED) {
#pragma unroll
        for (int j = 0; j < NO; ++j) {
            uint64_t bkey = best_key(best[j]);
            float bu = best[j].u, be = best[j].e2e, btt = best[j].tt, btp = best[j].tp;
            float bn = NH == 3 ? best[j].n : nout[j];
            // merge the two pair halves of each query through LDS
            const int slot = qw * kQPW + 32 * (2 * j + h) + n;
            if (grp == 1) {
                s_mkey[slot] = bkey;
                s_mval[slot] = (f32x4){bu, be, btt, btp};
                if constexpr (NH == 3) s_mnout[slot] = bn;
            }
            __syncthreads();
            if (grp == 0 && vme[j]) {
                const uint64_t ok = s_mkey[slot];
                if (ok > bkey) {
                    const f32x4 v = s_mval[slot];
                    bkey = ok;
                    bu = v[0];
                    be = v[1];
                    btt = v[2];
                    btp = v[3];
                    if constexpr (NH == 3) bn = s_mnout[slot];
                }
                if (nsplit == 1) {
                    write_outputs(a.out, qme[j], bkey, bu, be, btt, btp, bn);
                } else {
                    const size_t pi = static_cast<size_t>(split) * nq + qme[j];
                    a.part_key[pi] = bkey;
                    float *pv = a.part_val + pi * kPartVals;
                    pv[0] = bu;
                    pv[1] = be;
                    pv[2] = btt;
                    pv[3] = btp;
                    pv[4] = bn;
                }
            }
        }
    }
}

// Column tiles per wave: four at H = 256 and H = 128 (one wave per SIMD, the
// hand-scheduled form) for batches that give every compute unit a workgroup,
// staged, and fused when the input-length slot lies in the first k-block; two
// otherwise (two waves per SIMD: smaller batches start and drain faster).
// The two forms give bit-identical results.
template <int H, bool STAGED, int NH, bool FB>
static hipError_t launch_mlp_t(const MlpArgs &a, dim3 grid, hipStream_t s) {
    constexpr bool kFour = H == 256 || H == 128;
    if constexpr (kFour && STAGED) {
        if (a.four_tiles)
            return launch_kernel(k_mlp_bf16<H, STAGED, NH, FB, 4, false>, grid, dim3(MlpShape<4>::kThreads), 0, s, a);
    }
    const bool lean = !a.cand_ttft && !a.cand_nout && !a.rule.score_paper && !a.rule.bound_paper;
    if constexpr (kFour && !STAGED) {
        if (a.four_tiles && a.len_slot < 16) {   // the four-tile form patches k-block 0 only
            if (lean)
                return launch_kernel(k_mlp_bf16<H, STAGED, NH, FB, 4, true>, grid, dim3(MlpShape<4>::kThreads), 0, s, a);
            return launch_kernel(k_mlp_bf16<H, STAGED, NH, FB, 4, false>, grid, dim3(MlpShape<4>::kThreads), 0, s, a);
        }
    }
    if constexpr (!STAGED) {
        if (lean) return launch_kernel(k_mlp_bf16<H, STAGED, NH, FB, 2, true>, grid, dim3(MlpShape<2>::kThreads), 0, s, a);
    }
    return launch_kernel(k_mlp_bf16<H, STAGED, NH, FB, 2>, grid, dim3(MlpShape<2>::kThreads), 0, s, a);
}

template <int H>
static hipError_t launch_mlp_h(bool staged, const MlpArgs &a, hipStream_t s) {
    const dim3 grid((a.q.nq + kQPerBlock - 1) / kQPerBlock, staged ? 1 : a.nsplit);
    if (a.fold_b1) {
        if (a.nheads == 3)
            return staged ? launch_mlp_t<H, true, 3, true>(a, grid, s) : launch_mlp_t<H, false, 3, true>(a, grid, s);
        return staged ? launch_mlp_t<H, true, 2, true>(a, grid, s) : launch_mlp_t<H, false, 2, true>(a, grid, s);
    }
    if (a.nheads == 3)
        return staged ? launch_mlp_t<H, true, 3, false>(a, grid, s) : launch_mlp_t<H, false, 3, false>(a, grid, s);
    return staged ? launch_mlp_t<H, true, 2, false>(a, grid, s) : launch_mlp_t<H, false, 2, false>(a, grid, s);
}

hipError_t launch_mlp_bf16(int H, bool staged, const MlpArgs &a, hipStream_t s) {
    switch (H) {
        case 64: return launch_mlp_h<64>(staged, a, s);
        case 128: return launch_mlp_h<128>(staged, a, s);
        case 256: return launch_mlp_h<256>(staged, a, s);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace hwr
