// Device helpers shared by the libhwr kernels (gfx950).
#pragma once

#include "hwr_internal.hpp"

namespace hwr {

// Query feature of Eq. 1: ln(input_len) / 8, evaluated in fp64 and rounded
// once to fp32 (input_len below 1 is read as 1).
__device__ inline float len_feature(int32_t len) {
    const double v = static_cast<double>(len < 1 ? 1 : len);
    return static_cast<float>(log(v) * 0.125);
}

// The pair's slice of the Eq. 1 feature vector: one-hot architecture id (ia)
// and GPU type (ig), then, from slot b = A + Gw: ln(params_B)/4, the query
// slot (0 here), ln(1+running)/2, ln(1+waiting)/2, kv_util, gpu_util,
// ln(ttft)/4, ln(tpot)/4.  Logs in fp64, each value rounded once to fp32.
struct PairFeatures {
    int ia, ig, b;
    float v[8];
    __device__ float slot(int f) const {
        float x = 0.0f;
        if (f == ia || f == ig) x = 1.0f;
#pragma unroll
        for (int k = 0; k < 8; ++k)
            if (f == b + k) x = v[k];
        return x;
    }
};
__device__ inline PairFeatures pair_features(const hwr_hw_state &s, float params_b, int arch,
                                             int gpu, int arch_width, int gpu_width) {
    PairFeatures p;
    p.ia = arch;
    p.ig = arch_width + gpu;
    p.b = arch_width + gpu_width;
    p.v[0] = static_cast<float>(log(static_cast<double>(params_b)) * 0.25);
    p.v[1] = 0.0f;
    p.v[2] = static_cast<float>(log(1.0 + static_cast<double>(s.running_q)) * 0.5);
    p.v[3] = static_cast<float>(log(1.0 + static_cast<double>(s.waiting_q)) * 0.5);
    p.v[4] = s.kv_util;
    p.v[5] = s.gpu_util;
    p.v[6] = static_cast<float>(log(static_cast<double>(s.ttft_avg_s)) * 0.25);
    p.v[7] = static_cast<float>(log(static_cast<double>(s.tpot_avg_s)) * 0.25);
    return p;
}

__device__ inline uint16_t bf16_bits(float x) {   // nearest, ties to even
    return __builtin_bit_cast(uint16_t, static_cast<__bf16>(x));
}

__device__ inline float softplus_f32(float z) {
    return fmaxf(z, 0.0f) + log1pf(expf(-fabsf(z)));
}

// softplus(z) = max(z, 0) + log1p(e), e = exp(-|z|), on the hardware
// transcendentals: e = 2^(-|z| log2(e)) (v_exp_f32), and log1p by Goldberg's
// correction for the rounding of 1 + e: log1p(e) = ln(u) * e / (u - 1) with
// u = fl(1 + e), exact when u == 1 (D. Goldberg, "What every computer
// scientist should know about floating-point arithmetic", 1991, Thm. 4).
// Relative error a few fp32 ulps over the whole range.
__device__ inline float softplus_fast(float z) {
    constexpr float kLog2E = 1.44269504088896341f;
    constexpr float kLn2 = 0.693147180559945309f;
    const float e = __builtin_amdgcn_exp2f(-fabsf(z) * kLog2E);
    const float u = 1.0f + e;
    const float l = (u == 1.0f) ? e : __builtin_amdgcn_logf(u) * kLn2 * (e / (u - 1.0f));
    return fmaxf(z, 0.0f) + l;
}

// ReLU of two fp32 values, rounded to bf16 and packed (element 0 low).
// Rounding commutes with ReLU, and on bf16 bit patterns ReLU is a signed
// 16-bit max with 0.
__device__ inline bf16x2 relu_bf16x2(float a, float b) {
    const f32x2 v = {a, b};
    i16x2 s = __builtin_bit_cast(i16x2, __builtin_convertvector(v, bf16x2));
    s = __builtin_elementwise_max(s, (i16x2){0, 0});
    return __builtin_bit_cast(bf16x2, s);
}

// Candidate decision values: cost (Eq. 2), bound test (Eq. 3) and utility,
// each fp32 operation rounded once.
struct Decision {
    float e2e, u;
    bool feasible;
};
__device__ inline Decision decide(float ttft, float tpot, float nout, float slo,
                                  float quality, float alpha) {
    Decision r;
    r.e2e = __fmaf_rn(tpot, nout, ttft);
    r.feasible = r.e2e <= slo;
    const float t = __fdiv_rn(r.e2e, slo);
    r.u = __fsub_rn(quality, __fmul_rn(alpha, t));
    return r;
}

// Put the bf16 bits xl into element `elem` (0..7) of v.
__device__ inline bf16x8 put_elem(bf16x8 v, int elem, uint32_t xl) {
    u32x4 u = __builtin_bit_cast(u32x4, v);
    const int w = elem >> 1;
    const uint32_t keep = (elem & 1) ? 0x0000FFFFu : 0xFFFF0000u;
    const uint32_t put = (elem & 1) ? (xl << 16) : xl;
    u[0] = (w == 0) ? ((u[0] & keep) | put) : u[0];
    u[1] = (w == 1) ? ((u[1] & keep) | put) : u[1];
    u[2] = (w == 2) ? ((u[2] & keep) | put) : u[2];
    u[3] = (w == 3) ? ((u[3] & keep) | put) : u[3];
    return __builtin_bit_cast(bf16x8, u);
}

__device__ inline uint64_t shfl_xor_u64(uint64_t v, int m) {
    const uint32_t lo = __shfl_xor(static_cast<uint32_t>(v), m);
    const uint32_t hi = __shfl_xor(static_cast<uint32_t>(v >> 32), m);
    return (static_cast<uint64_t>(hi) << 32) | lo;
}

__device__ inline void write_outputs(const OutArgs &o, int q, uint64_t key, float u,
                                     float e2e, float ttft, float tpot) {
    o.choice[q] = key_pair(key);
    if (o.feasible) o.feasible[q] = key_feasible(key) ? 1 : 0;
    if (o.utility) o.utility[q] = u;
    if (o.e2e) o.e2e[q] = e2e;
    if (o.ttft) o.ttft[q] = ttft;
    if (o.tpot) o.tpot[q] = tpot;
}

}  // namespace hwr
