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
// the traffic (HBM-bound, arithmetic intensity ~M flop/byte).
__global__ __launch_bounds__(256) void k_quality_bf16(QualityArgs a) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int row = lane & 31, h = lane >> 5;
    const int q0 = blockIdx.x * 128 + wave * 32;
    const int qa = q0 + row;
    const bool valid = qa < a.nq;
    const uint16_t *e = static_cast<const uint16_t *>(a.emb) +
                        static_cast<size_t>(valid ? qa : 0) * a.D + 32 * h;
    const bf16x8 *wq = reinterpret_cast<const bf16x8 *>(a.wq_pk) + lane;
    f32x16 acc = {};
    const int S = a.D / 64;
    const bf16x8 zero = {};
#pragma unroll 2
    for (int s = 0; s < S; ++s) {
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

hipError_t launch_quality_bf16(const QualityArgs &a, hipStream_t s) {
    hipLaunchKernelGGL(k_quality_bf16, dim3((a.nq + 127) / 128), dim3(256), 0, s, a);
    return hipGetLastError();
}

// ------------------------------------------------------------ predictor
// Eq. 1 cost predictor on MFMA tiles, for all (query, pair) candidates of a
// chunk.  Workgroup: 4 waves x 64 queries; each wave loops over the pairs of
// its range, evaluating 2 x 32 candidates (one pair, 64 queries) per step:
//   X^T  (32 features x 32 candidates, bf16)   built from the pair's feature
//        row (L1-resident) and each query's input-length feature;
//   h1^T = ReLU(W1^T X^T + b1)  -> bf16, registers;
//   h2^T = ReLU(W2^T h1^T + b2) -> bf16, per 32-row tile, folded at once into
//   z    = W3^T h2^T + b3 by packed bf16 dot products;
//   TTFT = softplus(z0), TPOT = softplus(z1).
// W1, W2 (A operands), biases (as accumulator initial values) and W3 pairs
// live in LDS.  Fused mode then applies Eq. 2, the bound test and the
// utility and keeps a running maximum decision key per query (Eq. 3); staged
// mode reads X from HBM and writes TTFT/TPOT per candidate instead.
template <int H, bool STAGED>
__global__ __launch_bounds__(256, 1) void k_mlp_bf16(MlpArgs a) {
    constexpr int MT = H / 32;     // 32-row tiles of a hidden layer
    constexpr int KB2 = H / 16;    // k-blocks of the second layer
    constexpr int NT = 2;          // 32-candidate column tiles per wave
    __shared__ bf16x8 s_w1[MT * 2 * 64];
    __shared__ bf16x8 s_w2[MT * KB2 * 64];
    __shared__ f32x4 s_b1[MT * 2 * 4];
    __shared__ f32x4 s_b2[MT * 2 * 4];
    __shared__ u32x4 s_w3[MT * 2 * 4];
    const int tid = threadIdx.x;
    {
        const uint4 *g;
        uint4 *d;
        g = reinterpret_cast<const uint4 *>(a.w1_pk);
        d = reinterpret_cast<uint4 *>(s_w1);
        for (int i = tid; i < MT * 2 * 64; i += 256) d[i] = g[i];
        g = reinterpret_cast<const uint4 *>(a.w2_pk);
        d = reinterpret_cast<uint4 *>(s_w2);
        for (int i = tid; i < MT * KB2 * 64; i += 256) d[i] = g[i];
        g = reinterpret_cast<const uint4 *>(a.b1_pk);
        d = reinterpret_cast<uint4 *>(s_b1);
        for (int i = tid; i < MT * 2 * 4; i += 256) d[i] = g[i];
        g = reinterpret_cast<const uint4 *>(a.b2_pk);
        d = reinterpret_cast<uint4 *>(s_b2);
        for (int i = tid; i < MT * 2 * 4; i += 256) d[i] = g[i];
        g = reinterpret_cast<const uint4 *>(a.w3_pk);
        d = reinterpret_cast<uint4 *>(s_w3);
        for (int i = tid; i < MT * 2 * 4; i += 256) d[i] = g[i];
    }
    __syncthreads();

    const int lane = tid & 63, wave = tid >> 6, n = lane & 31, h = lane >> 5;
    const int nq = a.q.nq;
    const int qbase = blockIdx.x * kQPerBlock + wave * kQPerWave;
    int qc[NT];
    bool vq[NT];
    uint32_t xl[NT];
    float nout[NT], slo[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        const int q = qbase + 32 * t + n;
        vq[t] = q < nq;
        qc[t] = vq[t] ? q : 0;
        xl[t] = bf16_bits(len_feature(a.q.input_len[qc[t]]));
        const int32_t no = a.q.nout[qc[t]];
        nout[t] = static_cast<float>(no < 0 ? 0 : no);
        slo[t] = a.q.slo ? a.q.slo[qc[t]] : a.q.default_slo;
    }
    // the input-length slot: k-block, lane half and element holding it
    const int ls_kb = a.len_slot >> 4, ls_h = (a.len_slot >> 3) & 1, ls_e = a.len_slot & 7;
    const bool patch = (h == ls_h);

    const int split = blockIdx.y;
    const int d0 = static_cast<int>(static_cast<long>(a.N) * split / a.nsplit);
    const int d1 = static_cast<int>(static_cast<long>(a.N) * (split + 1) / a.nsplit);

    uint64_t bkey[NT];
    float bu[NT], be[NT], btt[NT], btp[NT];
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        bkey[t] = 0;
        bu[t] = be[t] = btt[t] = btp[t] = 0.0f;
    }

    for (int d = d0; d < d1; ++d) {
        // LDS offsets made opaque per step: the weight fragments are
        // loop-invariant, and hoisting all of them out of the pair loop would
        // need far more registers than a lane has.
        int lo = lane, ho = h;
        asm volatile("" : "+v"(lo), "+v"(ho));
        // ---- features (Eq. 1), B operand of layer 1
        bf16x8 xf[NT][2];
        if constexpr (STAGED) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                const uint16_t *xr = a.X + (static_cast<size_t>(qc[t]) * a.N + d) * kFeatPad + 8 * h;
                xf[t][0] = *reinterpret_cast<const bf16x8 *>(xr);
                xf[t][1] = *reinterpret_cast<const bf16x8 *>(xr + 16);
            }
        } else {
            const bf16x8 *row = reinterpret_cast<const bf16x8 *>(a.dep_bf16 + static_cast<size_t>(d) * kFeatPad);
            const bf16x8 r0 = row[h], r1 = row[2 + h];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                xf[t][0] = (patch && ls_kb == 0) ? put_elem(r0, ls_e, xl[t]) : r0;
                xf[t][1] = (patch && ls_kb == 1) ? put_elem(r1, ls_e, xl[t]) : r1;
            }
        }
        // ---- layer 1
        bf16x8 h1[NT][KB2];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            const f32x16 bi = bias_tile(s_b1 + (mt * 2 + ho) * 4);
            f32x16 acc[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[t] = bi;
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                const bf16x8 w = s_w1[(mt * 2 + kb) * 64 + lo];
#pragma unroll
                for (int t = 0; t < NT; ++t) acc[t] = mfma32(w, xf[t][kb], acc[t]);
            }
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                h1[t][2 * mt] = relu_pack8(acc[t], 0);
                h1[t][2 * mt + 1] = relu_pack8(acc[t], 8);
            }
        }
        // ---- layer 2, folded into the output heads tile by tile
        float z0[NT], z1[NT];
#pragma unroll
        for (int t = 0; t < NT; ++t) z0[t] = z1[t] = 0.0f;
#pragma unroll
        for (int mo = 0; mo < MT; ++mo) {
            const f32x16 bi = bias_tile(s_b2 + (mo * 2 + ho) * 4);
            f32x16 acc[NT];
#pragma unroll
            for (int t = 0; t < NT; ++t) acc[t] = bi;
#pragma unroll
            for (int kb = 0; kb < KB2; ++kb) {
                const bf16x8 w = s_w2[(mo * KB2 + kb) * 64 + lo];
#pragma unroll
                for (int t = 0; t < NT; ++t) acc[t] = mfma32(w, h1[t][kb], acc[t]);
            }
            const u32x4 *w3 = s_w3 + (mo * 2 + ho) * 4;
            const u32x4 wa = w3[0], wb = w3[1], wc = w3[2], wd = w3[3];
#pragma unroll
            for (int t = 0; t < NT; ++t) {
#pragma unroll
                for (int p = 0; p < 8; ++p) {
                    const bf16x2 hp = relu_bf16x2(acc[t][2 * p], acc[t][2 * p + 1]);
                    const uint32_t w0 = p < 4 ? wa[p & 3] : wb[p & 3];
                    const uint32_t w1 = p < 4 ? wc[p & 3] : wd[p & 3];
                    z0[t] = __builtin_amdgcn_fdot2_f32_bf16(hp, __builtin_bit_cast(bf16x2, w0), z0[t], false);
                    z1[t] = __builtin_amdgcn_fdot2_f32_bf16(hp, __builtin_bit_cast(bf16x2, w1), z1[t], false);
                }
            }
        }
        // ---- heads, cost, decision
        const int m = a.dep_model[d];
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const float zz0 = z0[t] + __shfl_xor(z0[t], 32);
            const float zz1 = z1[t] + __shfl_xor(z1[t], 32);
            const float tt = softplus_f32(zz0 + a.b3_0);
            const float tp = softplus_f32(zz1 + a.b3_1);
            const size_t ci = static_cast<size_t>(qc[t]) * a.N + d;
            if constexpr (STAGED) {
                if (h == 0 && vq[t]) {
                    a.cand_ttft[ci] = tt;
                    a.cand_tpot[ci] = tp;
                }
            } else {
                if (a.cand_ttft && h == 0 && vq[t]) {
                    a.cand_ttft[ci] = tt;
                    a.cand_tpot[ci] = tp;
                }
                const float Q = a.qmat[static_cast<size_t>(qc[t]) * a.M + m];
                const Decision r = decide(tt, tp, nout[t], slo[t], Q, a.alpha);
                const uint64_t k = decision_key(r.feasible, r.u, d);
                if (k > bkey[t]) {
                    bkey[t] = k;
                    bu[t] = r.u;
                    be[t] = r.e2e;
                    btt[t] = tt;
                    btp[t] = tp;
                }
            }
        }
    }
    if constexpr (!STAGED) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            if (h != 0 || !vq[t]) continue;
            const int q = qbase + 32 * t + n;
            if (a.nsplit == 1) {
                write_outputs(a.out, q, bkey[t], bu[t], be[t], btt[t], btp[t]);
            } else {
                const size_t pi = static_cast<size_t>(split) * nq + q;
                a.part_key[pi] = bkey[t];
                a.part_val[pi * 4 + 0] = bu[t];
                a.part_val[pi * 4 + 1] = be[t];
                a.part_val[pi * 4 + 2] = btt[t];
                a.part_val[pi * 4 + 3] = btp[t];
            }
        }
    }
}

template <int H>
static hipError_t launch_mlp_h(bool staged, const MlpArgs &a, hipStream_t s) {
    const dim3 grid((a.q.nq + kQPerBlock - 1) / kQPerBlock, staged ? 1 : a.nsplit);
    if (staged) hipLaunchKernelGGL((k_mlp_bf16<H, true>), grid, dim3(256), 0, s, a);
    else hipLaunchKernelGGL((k_mlp_bf16<H, false>), grid, dim3(256), 0, s, a);
    return hipGetLastError();
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
