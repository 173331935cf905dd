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
// chunk.  Workgroup: 8 waves, two per SIMD.  Waves w and w + 4 take the same
// 64 queries and split the workgroup's pair range in two halves, so that one
// wave's VALU epilogue overlaps the other's MFMAs; their decision keys merge
// through LDS at the end.  Each wave steps through its pairs, evaluating
// 2 x 32 candidates (one pair, 64 queries) per step:
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
// carries column tile h alone (one query per lane).  Fused mode then applies
// Eq. 2, the bound test and the utility and keeps the query's best candidate
// (Eq. 3); staged mode reads X from HBM and writes TTFT/TPOT per candidate.
template <int H, bool STAGED, int NH, bool FB>
__global__ __launch_bounds__(kMlpThreads, 1) void k_mlp_bf16(MlpArgs a) {
    constexpr int MT = H / 32;     // 32-row tiles of a hidden layer
    constexpr int KB2 = H / 16;    // k-blocks of the second layer
    constexpr int NT = 2;          // 32-candidate column tiles per wave
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
        // Every load of the staging is issued before the first LDS store:
        // one memory round trip for the whole prologue.  Indices past an
        // array's end are clamped for the loads and skipped for the stores.
        constexpr int nW1 = MT * 2 * 64, nW2 = MT * KB2 * 64, nB = MT * 2 * 4, nW3 = KB2 * W3S;
        constexpr int pW1 = (nW1 + kMlpThreads - 1) / kMlpThreads;
        constexpr int pW2 = (nW2 + kMlpThreads - 1) / kMlpThreads;
        const uint4 *g1 = reinterpret_cast<const uint4 *>(a.w1_pk);
        const uint4 *g2 = reinterpret_cast<const uint4 *>(a.w2_pk);
        const uint4 *gb1 = reinterpret_cast<const uint4 *>(a.b1_pk);
        const uint4 *gb2 = reinterpret_cast<const uint4 *>(a.b2_pk);
        const uint4 *g3 = reinterpret_cast<const uint4 *>(a.w3_frag);
        uint4 v1[pW1], v2[pW2];
#pragma unroll
        for (int i = 0; i < pW1; ++i) {
            const int k = tid + i * kMlpThreads;
            v1[i] = g1[k < nW1 ? k : 0];
        }
#pragma unroll
        for (int i = 0; i < pW2; ++i) {
            const int k = tid + i * kMlpThreads;
            v2[i] = g2[k < nW2 ? k : 0];
        }
        static_assert(nB <= kMlpThreads && nW3 <= kMlpThreads, "one bias / head piece per thread");
        const uint4 vb1 = gb1[tid < nB ? tid : 0], vb2 = gb2[tid < nB ? tid : 0];
        const uint4 v3 = g3[tid < nW3 ? tid : 0];
#pragma unroll
        for (int i = 0; i < pW1; ++i) {
            const int k = tid + i * kMlpThreads;
            if (k < nW1) reinterpret_cast<uint4 *>(s_w1)[k] = v1[i];
        }
#pragma unroll
        for (int i = 0; i < pW2; ++i) {
            const int k = tid + i * kMlpThreads;
            if (k < nW2) reinterpret_cast<uint4 *>(s_w2)[k] = v2[i];
        }
        if (tid < nB) {
            reinterpret_cast<uint4 *>(s_b1)[tid] = vb1;
            reinterpret_cast<uint4 *>(s_b2)[tid] = vb2;
        }
        if (tid < nW3) reinterpret_cast<uint4 *>(s_w3f)[tid] = v3;
    }
    __syncthreads();

    const int lane = tid & 63, wave = tid >> 6, n = lane & 31, h = lane >> 5;
    const int qw = wave & 3, grp = wave >> 2;
    const int nq = a.q.nq;
    const int qbase = blockIdx.x * kQPerBlock + qw * kQPerWave;
    // every lane builds features for both column tiles ...
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
    // ... and decides for column tile h only (query qme)
    const int qme = qbase + 32 * h + n;
    const bool vme = qme < nq;
    const int qmc = vme ? qme : 0;
    const int32_t nomy = a.q.nout ? a.q.nout[qmc] : 0;   // given N_out (two heads)
    const float nout = static_cast<float>(nomy < 0 ? 0 : nomy);
    const QueryRule qrule = query_rule(a.rule, a.q.slo ? a.q.slo[qmc] : a.q.default_slo,
                                       a.q.input_len[qmc], nout, a.w);
    // the input-length slot: k-block, lane half and element holding it
    const int ls_kb = a.len_slot >> 4, ls_h = (a.len_slot >> 3) & 1, ls_e = a.len_slot & 7;
    const bool patch = (h == ls_h);

    const int split = STAGED ? 0 : blockIdx.y;
    const int nsplit = STAGED ? 1 : a.nsplit;
    const long span0 = static_cast<long>(a.N) * split / nsplit;
    const long span1 = static_cast<long>(a.N) * (split + 1) / nsplit;
    const int d0 = static_cast<int>(span0 + (span1 - span0) * grp / 2);
    const int d1 = static_cast<int>(span0 + (span1 - span0) * (grp + 1) / 2);

    Best best = best_none();

    // Head-layer A fragment of this lane for column tile t (an index into a
    // k-block's fragments): lane 16g + i holds row i, k-group g.  Row
    // i = 8t + 4s + m is head m of sub-column s; it takes weights only from
    // the k-groups whose B lanes carry sub-column s (g & 1 == s), namely the
    // hidden-unit half g >> 1.  Every other lane reads the zero fragment.
    int w3_sel[NT];
    {
        const int i = lane & 15, g = lane >> 4, m = i & 3, s = (i >> 2) & 1;
#pragma unroll
        for (int t = 0; t < NT; ++t)
            w3_sel[t] = ((i >> 3) == t && m < NH && (g & 1) == s) ? m * 2 + (g >> 1) : 2 * NH;
    }

    // Per-pair inputs are loaded one step ahead: the pair's feature row
    // (fused) or the candidates' feature rows (staged), and the quality
    // Q[query][model(pair)], whose address needs a scalar load first.
    const bf16x8 *dep = reinterpret_cast<const bf16x8 *>(a.dep_bf16);
    const float *qrow = a.qmat + static_cast<size_t>(qmc) * a.M;
    const int dfirst = d0 < d1 ? d0 : 0;
    bf16x8 nr[NT][2];
    if constexpr (STAGED) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const bf16x8 *xr = reinterpret_cast<const bf16x8 *>(
                a.X + (static_cast<size_t>(qc[t]) * a.N + dfirst) * kFeatPad);
            nr[t][0] = xr[h];
            nr[t][1] = xr[2 + h];
        }
    } else {
        nr[0][0] = dep[dfirst * 4 + h];
        nr[0][1] = dep[dfirst * 4 + 2 + h];
    }
    float nq_val = STAGED ? 0.0f : qrow[a.dep_model[dfirst]];

    for (int d = d0; d < d1; ++d) {
        bf16x8 cr[NT][2];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            cr[t][0] = nr[t][0];
            cr[t][1] = nr[t][1];
        }
        const float Qd = nq_val;
        {
            const int dn = d + 1 < d1 ? d + 1 : d;
            if constexpr (STAGED) {
#pragma unroll
                for (int t = 0; t < NT; ++t) {
                    const bf16x8 *xr = reinterpret_cast<const bf16x8 *>(
                        a.X + (static_cast<size_t>(qc[t]) * a.N + dn) * kFeatPad);
                    nr[t][0] = xr[h];
                    nr[t][1] = xr[2 + h];
                }
            } else {
                nr[0][0] = dep[dn * 4 + h];
                nr[0][1] = dep[dn * 4 + 2 + h];
                nq_val = qrow[a.dep_model[dn]];
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
                xf[t][0] = (patch && ls_kb == 0) ? put_elem(r0, ls_e, xl[t]) : r0;
                xf[t][1] = (patch && ls_kb == 1) ? put_elem(r1, ls_e, xl[t]) : r1;
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
        // to their last use, past the fences, and the registers overflow)
        auto l1_epi = [&](int mt, const f32x16 (&c)[NT]) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                h1[t][2 * mt] = relu_pack8(c[t], 0);
                h1[t][2 * mt + 1] = relu_pack8(c[t], 8);
                asm volatile("" : "+v"(h1[t][2 * mt]), "+v"(h1[t][2 * mt + 1]));
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
        // A fragments (see w3_sel) keep them apart: tile t's row 8t + 4s + m is
        // head m of candidate 32t + 16s + j, so after both tiles every lane
        // holds its own candidate's heads in accumulator elements 0..NH-1.
        // (Packed bf16 dot products would stall the matrix pipe: they do not
        // co-issue with MFMA on gfx950.)
        f32x4 acc3 = {};
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
                acc3 = mfma16(s_w3f[kb * W3S + w3o0], h2[0][b], acc3);
                acc3 = mfma16(s_w3f[kb * W3S + w3o1], h2[1][b], acc3);
            }
            asm volatile("" : "+v"(acc3));
        };
        // MFMA k-steps of tile mo issued before the previous epilogue.  For
        // mo = 0 that epilogue produces layer-1 k-blocks KB2-2 and KB2-1, so
        // the head steps must stop short of them.
        constexpr int kHead = KB2 - 2 < 4 ? KB2 - 2 : 4;
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
        // ---- heads: lane half h completes column tile h (its partner lane
        // holds the other 128 hidden units of the same candidates)
        const float tt = softplus_fast(acc3[0] + a.b3_0);
        const float tp = softplus_fast(acc3[1] + a.b3_1);
        // N_out: the third head's prediction (tokens), else the query's given value
        const float nc = NH == 3 ? softplus_fast(acc3[2] + a.b3_2) : nout;
        const size_t ci = static_cast<size_t>(qmc) * a.N + d;
        if constexpr (STAGED) {
            if (vme) {
                a.cand_ttft[ci] = tt;
                a.cand_tpot[ci] = tp;
                if (NH == 3) a.cand_nout[ci] = nc;
            }
        } else {
            if (a.cand_ttft && vme) {
                a.cand_ttft[ci] = tt;
                a.cand_tpot[ci] = tp;
            }
            if (a.cand_nout && vme) a.cand_nout[ci] = nc;
            // ---- cost, bound test, utility, running argmax (Eq. 2, Eq. 3)
            offer<NH == 3>(best, decide(tt, tp, nc, a.rule, qrule, Qd), d, tt, tp, nc);
        }
    }
    if constexpr (!STAGED) {
        uint64_t bkey = best_key(best);
        float bu = best.u, be = best.e2e, btt = best.tt, btp = best.tp;
        float bn = NH == 3 ? best.n : nout;
        // merge the two pair halves of each query through LDS
        const int slot = qw * kQPerWave + lane;
        if (grp == 1) {
            s_mkey[slot] = bkey;
            s_mval[slot] = (f32x4){bu, be, btt, btp};
            if constexpr (NH == 3) s_mnout[slot] = bn;
        }
        __syncthreads();
        if (grp == 0 && vme) {
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
                write_outputs(a.out, qme, bkey, bu, be, btt, btp, bn);
            } else {
                const size_t pi = static_cast<size_t>(split) * nq + qme;
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

template <int H>
static hipError_t launch_mlp_h(bool staged, const MlpArgs &a, hipStream_t s) {
    const dim3 grid((a.q.nq + kQPerBlock - 1) / kQPerBlock, staged ? 1 : a.nsplit);
    const dim3 block(kMlpThreads);
    if (a.fold_b1) {
        if (a.nheads == 3)
            return staged ? launch_kernel(k_mlp_bf16<H, true, 3, true>, grid, block, 0, s, a)
                          : launch_kernel(k_mlp_bf16<H, false, 3, true>, grid, block, 0, s, a);
        return staged ? launch_kernel(k_mlp_bf16<H, true, 2, true>, grid, block, 0, s, a)
                      : launch_kernel(k_mlp_bf16<H, false, 2, true>, grid, block, 0, s, a);
    }
    if (a.nheads == 3)
        return staged ? launch_kernel(k_mlp_bf16<H, true, 3, false>, grid, block, 0, s, a)
                      : launch_kernel(k_mlp_bf16<H, false, 3, false>, grid, block, 0, s, a);
    return staged ? launch_kernel(k_mlp_bf16<H, true, 2, false>, grid, block, 0, s, a)
                  : launch_kernel(k_mlp_bf16<H, false, 2, false>, grid, block, 0, s, a);
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
