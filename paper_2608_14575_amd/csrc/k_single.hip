// Single-query routing kernel of libhwr (gfx950): one query against all
// pairs in one workgroup, reading the query from and writing the decision to
// pinned host memory, so that one launch (captured once in a graph) is the
// whole call.  Pairs are the MFMA columns here (32 per tile); the 4 waves
// split the second-layer row tiles and combine their head partials in LDS.
#include "hwr_device.hpp"

namespace hwr {

__device__ __forceinline__ f32x16 mfma32s(bf16x8 a, bf16x8 b, f32x16 c) {
    return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
}

__device__ __forceinline__ f32x16 load_bias_tile(const float *p) {
    const f32x4 *v = reinterpret_cast<const f32x4 *>(p);
    const f32x4 a = v[0], b = v[1], c = v[2], d = v[3];
    return (f32x16){a[0], a[1], a[2], a[3], b[0], b[1], b[2], b[3],
                    c[0], c[1], c[2], c[3], d[0], d[1], d[2], d[3]};
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
    __shared__ __attribute__((aligned(16))) uint16_t s_emb[8192];
    __shared__ float s_q[kMaxModels];
    __shared__ float s_z[4][32][2];
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, n = lane & 31, h = lane >> 5;

    // query record: header, then D bf16 values
    const uint4 *src = reinterpret_cast<const uint4 *>(a.in + 1);
    for (int i = tid; i < a.D / 8; i += 256) reinterpret_cast<uint4 *>(s_emb)[i] = src[i];
    const uint32_t seq = a.in->seq;
    const int32_t len = a.in->input_len;
    const int32_t no = a.in->nout;
    const float nout = static_cast<float>(no < 0 ? 0 : no);
    const float slo = a.in->slo;
    __syncthreads();

    // quality of every model (Sec. 3.2 item 3): one wave per model, lanes split D
    for (int m = wave; m < a.M; m += 4) {
        float acc = 0.0f;
        for (int k = lane * 8; k < a.D; k += 512) {
            const bf16x8 e = *reinterpret_cast<const bf16x8 *>(s_emb + k);
            const bf16x8 w = *reinterpret_cast<const bf16x8 *>(a.wqT + static_cast<size_t>(m) * a.D + k);
#pragma unroll
            for (int j = 0; j < 8; ++j) acc = fmaf(static_cast<float>(e[j]), static_cast<float>(w[j]), acc);
        }
#pragma unroll
        for (int off = 32; off >= 1; off >>= 1) acc += __shfl_xor(acc, off);
        if (lane == 0) s_q[m] = acc + a.bq[m];
    }

    const uint32_t xl = bf16_bits(len_feature(len));
    const int ls_kb = a.len_slot >> 4, ls_h = (a.len_slot >> 3) & 1, ls_e = a.len_slot & 7;
    const bf16x8 *w1 = reinterpret_cast<const bf16x8 *>(a.w1_pk);
    const bf16x8 *w2 = reinterpret_cast<const bf16x8 *>(a.w2_pk);
    const u32x4 *w3 = reinterpret_cast<const u32x4 *>(a.w3_pk);

    uint64_t bkey = 0;
    float bu = 0.0f, be = 0.0f, btt = 0.0f, btp = 0.0f;
    const int ntiles = (a.N + 31) / 32;
    for (int ct = 0; ct < ntiles; ++ct) {
        const int d = ct * 32 + n;
        const bool vd = d < a.N;
        // features of pair d (Eq. 1), zero columns past the last pair
        bf16x8 xf[2];
        {
            const bf16x8 *row = reinterpret_cast<const bf16x8 *>(a.dep_bf16 + static_cast<size_t>(vd ? d : 0) * kFeatPad);
            const bf16x8 zero = {};
            xf[0] = vd ? row[h] : zero;
            xf[1] = vd ? row[2 + h] : zero;
            if (vd && h == ls_h) {
                if (ls_kb == 0) xf[0] = put_elem(xf[0], ls_e, xl);
                else xf[1] = put_elem(xf[1], ls_e, xl);
            }
        }
        // layer 1 (every wave, all row tiles)
        bf16x8 h1[KB2];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            f32x16 acc = load_bias_tile(a.b1_pk + (mt * 2 + h) * 16);
#pragma unroll
            for (int kb = 0; kb < 2; ++kb) acc = mfma32s(w1[(mt * 2 + kb) * 64 + lane], xf[kb], acc);
            h1[2 * mt] = relu_pack8s(acc, 0);
            h1[2 * mt + 1] = relu_pack8s(acc, 8);
        }
        // layer 2 row tiles of this wave, folded into the heads
        float z0 = 0.0f, z1 = 0.0f;
        for (int mo = wave; mo < MT; mo += 4) {
            f32x16 acc = load_bias_tile(a.b2_pk + (mo * 2 + h) * 16);
#pragma unroll
            for (int kb = 0; kb < KB2; ++kb) acc = mfma32s(w2[(mo * KB2 + kb) * 64 + lane], h1[kb], acc);
            const u32x4 *w3t = w3 + (mo * 2 + h) * 4;
            const u32x4 wa = w3t[0], wb = w3t[1], wc = w3t[2], wd = w3t[3];
#pragma unroll
            for (int p = 0; p < 8; ++p) {
                const bf16x2 hp = relu_bf16x2(acc[2 * p], acc[2 * p + 1]);
                const uint32_t u0 = p < 4 ? wa[p & 3] : wb[p & 3];
                const uint32_t u1 = p < 4 ? wc[p & 3] : wd[p & 3];
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
            const Decision r = decide(tt, tp, nout, slo, s_q[a.dep_model[d]], a.alpha);
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
