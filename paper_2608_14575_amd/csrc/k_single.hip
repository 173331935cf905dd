// Single-query routing kernel of libhwr (gfx950): one query against all
// pairs in one workgroup, reading the query and the pairs' current runtime
// signals from pinned host memory and writing the decision there, so that
// one launch (captured once in a graph) is the whole call.  Pairs are the MFMA columns here (32 per tile); the 4 waves
// split the second-layer row tiles and combine their head partials in LDS.
#include "hwr_device.hpp"

namespace hwr {

__device__ __forceinline__ f32x16 mfma32s(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ bf16x8 relu_pack8s(const f32x16 &c, int base) {
    u32x4 u;
    u[0] = __builtin_bit_cast(uint32_t, relu_bf16x2(c[base + 0], c[base + 1]));
    u[1] = __builtin_bit_cast(uint32_t, relu_bf16x2(c[base + 2], c[base + 3]));
    u[2] = __builtin_bit_cast(uint32_t, relu_bf16x2(c[base + 4], c[base + 5]));
    u[3] = __builtin_bit_cast(uint32_t, relu_bf16x2(c[base + 6], c[base + 7]));
    return __builtin_bit_cast(bf16x8, u);
}

template <int H>
__global__ __launch_bounds__(256) void k_single(SingleArgs a) {
    constexpr int MT = H / 32, KB2 = H / 16;
    constexpr int MO = (MT + 3) / 4;          // second-layer row tiles per wave
    __shared__ float s_q[kMaxModels];
    __shared__ float s_z[4][32][2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, n = lane & 31, h = lane >> 5;
    const bf16x8 *w1 = reinterpret_cast<const bf16x8 *>(a.w1_pk);
    const bf16x8 *w2 = reinterpret_cast<const bf16x8 *>(a.w2_pk);
    const u32x4 *w3 = reinterpret_cast<const u32x4 *>(a.w3_pk);
    const f32x4 *b1 = reinterpret_cast<const f32x4 *>(a.b1_pk);
    const f32x4 *b2 = reinterpret_cast<const f32x4 *>(a.b2_pk);

    // Everything that does not depend on the query is loaded first, so that
    // its latency overlaps the read of the query record from host memory:
    // the first-layer fragments and bias tiles, this wave's second-layer
    // fragments, bias tiles and head pairs, and the first tile's pair rows.
    // (at H = 256 the first-layer bias tiles are read where they are used:
    // holding them all would overflow the register file)
    constexpr bool kHoldB1 = H <= 128;
    bf16x8 fw1[MT][2];
    f32x4 fb1[kHoldB1 ? MT : 1][4];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt) {
#pragma unroll
        for (int kb = 0; kb < 2; ++kb) fw1[mt][kb] = w1[(mt * 2 + kb) * 64 + lane];
        if constexpr (kHoldB1) {
#pragma unroll
            for (int i = 0; i < 4; ++i) fb1[mt][i] = b1[(mt * 2 + h) * 4 + i];
        }
    }
    constexpr int MOH = MO == 1 ? 1 : 0;     // second-layer tiles held in registers
    bf16x8 fw2[MO][KB2];
    f32x4 fb2[MO][4];
    u32x4 fw3[MO][4];
#pragma unroll
    for (int i = 0; i < MOH; ++i) {
        const int mo = wave + 4 * i < MT ? wave + 4 * i : 0;
#pragma unroll
        for (int kb = 0; kb < KB2; ++kb) fw2[i][kb] = w2[(mo * KB2 + kb) * 64 + lane];
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            fb2[i][j] = b2[(mo * 2 + h) * 4 + j];
            fw3[i][j] = w3[(mo * 2 + h) * 4 + j];
        }
    }
    // the first tile's pairs: runtime signals (pinned host memory, written
    // by the last state update) and static attributes
    const int d0 = n < a.N ? n : 0;
    hwr_hw_state st0 = a.state[d0];
    int model0 = a.dep_model[d0], gpu0 = a.dep_gpu[d0];

    // query record (pinned host memory): header and embedding
    const uint32_t seq = a.in->seq;
    const int32_t len = a.in->input_len;
    const int32_t no = a.in->nout;
    const float nout = static_cast<float>(no < 0 ? 0 : no);
    const float slo = a.in->slo;
    const uint16_t *emb = reinterpret_cast<const uint16_t *>(a.in + 1);

    // quality of every model (Sec. 3.2 item 3): one wave per model, lanes
    // split D; the embedding slices are read straight from host memory
    for (int m0 = wave; m0 < a.M; m0 += 8) {
        const int m1 = m0 + 4;
        float acc0 = 0.0f, acc1 = 0.0f;
        for (int k = lane * 8; k < a.D; k += 512) {
            const bf16x8 e = *reinterpret_cast<const bf16x8 *>(emb + k);
            const bf16x8 q0 = *reinterpret_cast<const bf16x8 *>(a.wqT + static_cast<size_t>(m0) * a.D + k);
            const bf16x8 q1 = m1 < a.M ? *reinterpret_cast<const bf16x8 *>(a.wqT + static_cast<size_t>(m1) * a.D + k) : q0;
#pragma unroll
            for (int j = 0; j < 8; ++j) {
                acc0 = fmaf(static_cast<float>(e[j]), static_cast<float>(q0[j]), acc0);
                acc1 = fmaf(static_cast<float>(e[j]), static_cast<float>(q1[j]), acc1);
            }
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            acc0 += __shfl_xor(acc0, off);
            acc1 += __shfl_xor(acc1, off);
        }
        if (lane == 0) {
            s_q[m0] = acc0 + a.bq[m0];
            if (m1 < a.M) s_q[m1] = acc1 + a.bq[m1];
        }
    }

    const uint32_t xl = bf16_bits(len_feature(len));
    const int ls_kb = a.len_slot >> 4, ls_h = (a.len_slot >> 3) & 1, ls_e = a.len_slot & 7;

    uint64_t bkey = 0;
    float bu = 0.0f, be = 0.0f, btt = 0.0f, btp = 0.0f;
    const int ntiles = (a.N + 31) / 32;
    for (int ct = 0; ct < ntiles; ++ct) {
        const int d = ct * 32 + n;
        const bool vd = d < a.N;
        // features of pair d (Eq. 1), zero columns past the last pair
        bf16x8 xf[2];
        const int model = model0;
        {
            const PairFeatures pf = pair_features(st0, a.params_b[model], a.model_arch[model], gpu0,
                                                  a.arch_width, a.gpu_width);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) {
                u32x4 u;
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    const int f = 16 * kb + 8 * h + 2 * j;
                    const f32x2 v = {vd ? pf.slot(f) : 0.0f, vd ? pf.slot(f + 1) : 0.0f};
                    u[j] = __builtin_bit_cast(uint32_t, __builtin_convertvector(v, bf16x2));
                }
                xf[kb] = __builtin_bit_cast(bf16x8, u);
            }
            if (vd && h == ls_h) {
                if (ls_kb == 0) xf[0] = put_elem(xf[0], ls_e, xl);
                else xf[1] = put_elem(xf[1], ls_e, xl);
            }
        }
        if (ct + 1 < ntiles) {          // next tile's pairs
            const int dn = (ct + 1) * 32 + n < a.N ? (ct + 1) * 32 + n : 0;
            st0 = a.state[dn];
            model0 = a.dep_model[dn];
            gpu0 = a.dep_gpu[dn];
        }
        // layer 1 (every wave, all row tiles)
        bf16x8 h1[KB2];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            f32x16 acc;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const f32x4 bt = kHoldB1 ? fb1[kHoldB1 ? mt : 0][i] : b1[(mt * 2 + h) * 4 + i];
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[4 * i + j] = bt[j];
            }
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) acc = mfma32s(fw1[mt][kb], xf[kb], acc);
            h1[2 * mt] = relu_pack8s(acc, 0);
            h1[2 * mt + 1] = relu_pack8s(acc, 8);
        }
        // layer 2 row tiles of this wave, folded into the heads
        float z0 = 0.0f, z1 = 0.0f;
#pragma unroll
        for (int i = 0; i < MO; ++i) {
            if (wave + 4 * i >= MT) break;
            if (i >= MOH) {
                const int mo = wave + 4 * i;
#pragma unroll
                for (int kb = 0; kb < KB2; ++kb) fw2[i][kb] = w2[(mo * KB2 + kb) * 64 + lane];
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    fb2[i][j] = b2[(mo * 2 + h) * 4 + j];
                    fw3[i][j] = w3[(mo * 2 + h) * 4 + j];
                }
            }
            f32x16 acc;
#pragma unroll
            for (int p = 0; p < 4; ++p)
#pragma unroll
                for (int j = 0; j < 4; ++j) acc[4 * p + j] = fb2[i][p][j];
#pragma unroll
            for (int kb = 0; kb < KB2; ++kb) acc = mfma32s(fw2[i][kb], h1[kb], acc);
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                const bf16x2 hp = relu_bf16x2(acc[2 * p], acc[2 * p + 1]);
                const uint32_t u0 = p < 4 ? fw3[i][0][p & 3] : fw3[i][1][p & 3];
                const uint32_t u1 = p < 4 ? fw3[i][2][p & 3] : fw3[i][3][p & 3];
                z0 = __builtin_amdgcn_fdot2_f32_bf16(hp, __builtin_bit_cast(bf16x2, u0), z0, false);
                z1 = __builtin_amdgcn_fdot2_f32_bf16(hp, __builtin_bit_cast(bf16x2, u1), z1, false);
            }
        }
        z0 += __shfl_xor(z0, 32);
        z1 += __shfl_xor(z1, 32);
        if (h == 0) {
            s_z[wave][n][0] = z0;
            s_z[wave][n][1] = z1;
        }
        __syncthreads();
        if (wave == 0 && h == 0 && vd) {
            const float zz0 = s_z[0][n][0] + s_z[1][n][0] + s_z[2][n][0] + s_z[3][n][0];
            const float zz1 = s_z[0][n][1] + s_z[1][n][1] + s_z[2][n][1] + s_z[3][n][1];
            const float tt = softplus_fast(zz0 + a.b3_0);
            const float tp = softplus_fast(zz1 + a.b3_1);
            const Decision r = decide(tt, tp, nout, slo, s_q[model], a.alpha);
            const uint64_t k = decision_key(r.feasible, r.u, d);
            if (k > bkey) {
                bkey = k;
                bu = r.u;
                be = r.e2e;
                btt = tt;
                btp = tp;
            }
        }
        __syncthreads();
    }
    if (wave == 0) {
        uint64_t k = bkey;
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) {
            const uint64_t o = shfl_xor_u64(k, off);
            k = o > k ? o : k;
        }
        if (bkey == k && k != 0) {
            SingleOut *o = a.out;
            o->choice = key_pair(k);
            o->feasible = key_feasible(k) ? 1u : 0u;
            o->utility = bu;
            o->e2e = be;
            o->ttft = btt;
            o->tpot = btp;
            __threadfence_system();
            __hip_atomic_store(&o->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
        }
    }
}

hipError_t launch_single(int H, const SingleArgs &a, hipStream_t s) {
    switch (H) {
        case 64: hipLaunchKernelGGL(k_single<64>, dim3(1), dim3(256), 0, s, a); break;
        case 128: hipLaunchKernelGGL(k_single<128>, dim3(1), dim3(256), 0, s, a); break;
        case 256: hipLaunchKernelGGL(k_single<256>, dim3(1), dim3(256), 0, s, a); break;
        default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace hwr
