// Device helpers shared by the libhwr kernels (gfx950).
#pragma once

#include "hwr_internal.hpp"

namespace hwr {

// Natural logarithm in fp64 of a positive, finite, normal x (every argument
// of the features below is one: validated counts plus one, parameter counts
// and latencies above zero).  x = m 2^e with m in [sqrt(1/2), sqrt(2)), and
// ln m = 2 artanh(f) = 2 f (1 + f^2/3 + f^4/5 + ...), f = (m - 1) / (m + 1)
// (the series of Abramowitz & Stegun 4.1.27), taken to f^17: |f| <= 0.172,
// so the first term left out is below 2^-55 relative.  The quotient is the
// hardware reciprocal refined by two Newton steps.  Relative error about
// 2^-50 at most over the features' argument ranges, and every fp32 and bf16
// feature value the same as with an exact log (hwr_probe_feature_log exposes
// this function for that check); about a third of the operations of the
// library's fp64 log.
__device__ inline double ln_pos(double x) {
    double m = __builtin_amdgcn_frexp_mant(x);    // [0.5, 1)
    int e = __builtin_amdgcn_frexp_exp(x);
    if (m < 0.70710678118654752440) {
        m *= 2.0;
        e -= 1;
    }
    const double n = m - 1.0, d = m + 1.0;        // n exact
    double r = __builtin_amdgcn_rcp(d);
    r = fma(r, fma(-d, r, 1.0), r);
    r = fma(r, fma(-d, r, 1.0), r);
    const double f = n * r, s = f * f;
    double p = 1.0 / 17.0;
    p = fma(p, s, 1.0 / 15.0);
    p = fma(p, s, 1.0 / 13.0);
    p = fma(p, s, 1.0 / 11.0);
    p = fma(p, s, 1.0 / 9.0);
    p = fma(p, s, 1.0 / 7.0);
    p = fma(p, s, 1.0 / 5.0);
    p = fma(p, s, 1.0 / 3.0);
    p = fma(p, s, 1.0);
    return fma(static_cast<double>(e), 0.69314718055994530942, (2.0 * f) * p);
}

// Query feature of Eq. 1: ln(input_len) / 8, evaluated in fp64 and rounded
// once to fp32 (input_len below 1 is read as 1).
__device__ inline float len_feature(int32_t len) {
    const double v = static_cast<double>(len < 1 ? 1 : len);
    return static_cast<float>(ln_pos(v) * 0.125);
}

// The pair's slice of the Eq. 1 feature vector: one-hot architecture id (ia)
// and GPU type (ig), then, from slot b = A + Gw: ln(params_B)/4, the query
// slot (0 here), ln(1+running)/2, ln(1+waiting)/2, kv_util, gpu_util,
// ln(ttft)/4, ln(tpot)/4.  Logs in fp64 (ln_pos), each value rounded once to fp32.
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
    p.v[0] = static_cast<float>(ln_pos(static_cast<double>(params_b)) * 0.25);
    p.v[1] = 0.0f;
    p.v[2] = static_cast<float>(ln_pos(1.0 + static_cast<double>(s.running_q)) * 0.5);
    p.v[3] = static_cast<float>(ln_pos(1.0 + static_cast<double>(s.waiting_q)) * 0.5);
    p.v[4] = s.kv_util;
    p.v[5] = s.gpu_util;
    p.v[6] = static_cast<float>(ln_pos(static_cast<double>(s.ttft_avg_s)) * 0.25);
    p.v[7] = static_cast<float>(ln_pos(static_cast<double>(s.tpot_avg_s)) * 0.25);
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
// The quotient e / (u - 1), a factor within an ulp or so of 1, takes the
// hardware reciprocal (v_rcp_f32, about 1 ulp) instead of a full IEEE
// division.  Relative error a few fp32 ulps over the whole range.
__device__ inline float softplus_fast(float z) {
    constexpr float kLog2E = 1.44269504088896341f;
    constexpr float kLn2 = 0.693147180559945309f;
    const float e = __builtin_amdgcn_exp2f(-fabsf(z) * kLog2E);
    const float u = 1.0f + e;
    const float l = (u == 1.0f) ? e : __builtin_amdgcn_logf(u) * kLn2 * (e * __builtin_amdgcn_rcpf(u - 1.0f));
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

// A query's latency bound with its correctly rounded reciprocal, for the
// division C / SLO of the utility (computed once per query).
struct Bound {
    float slo, rcp;
    bool fast;                    // slo in [2^-20, 2^20]: the reciprocal path applies
};
__device__ inline Bound make_bound(float slo) {
    Bound b;
    b.slo = slo;
    b.rcp = __fdiv_rn(1.0f, slo);
    b.fast = slo >= 0x1p-20f && slo <= 0x1p20f;
    return b;
}

// RN(c / slo), the IEEE quotient, from y = RN(1 / slo): q0 = RN(c y), the
// remainder r = c - q0 slo (exact with one FMA), then RN(q0 + r y).  With y
// within half an ulp of 1 / slo and q0 within one ulp of the quotient, this
// correction gives the correctly rounded quotient (P. Markstein, IBM J. Res.
// Dev. 34(1), 1990; Muller et al., Handbook of Floating-Point Arithmetic,
// division by FMA).  The ranges keep every step clear of underflow and
// overflow; outside them the plain IEEE division is used.
__device__ inline float div_bound(float c, const Bound &b) {
    const float q0 = __fmul_rn(c, b.rcp);
    const float r = __fmaf_rn(-q0, b.slo, c);
    float t = __fmaf_rn(r, b.rcp, q0);
    if (!(b.fast && c >= 0x1p-60f && c <= 0x1p60f)) {
        asm volatile("");         // a real branch: keeps the division off the common path
        t = __fdiv_rn(c, b.slo);
    }
    return t;
}

// Per query and cost weight: the bound (when it is the same for every
// candidate, with its reciprocal), the paper bound's a + b * input_len, and
// the weight w with 1 - w (rounded once).
struct QueryRule {
    Bound bound;
    float base, w, w1;
};
__device__ inline QueryRule query_rule(const Rule &R, float slo, int32_t input_len, float nout, float w) {
    QueryRule q;
    q.base = R.bound_paper ? __fmaf_rn(R.b, static_cast<float>(input_len), R.a) : 0.0f;
    q.bound = make_bound(R.bound_paper ? __fmaf_rn(nout, R.tpot_slo, q.base) : slo);
    q.w = w;
    q.w1 = __fsub_rn(1.0f, w);
    return q;
}

// Candidate decision values: cost (Eq. 2), bound test (Eq. 3) and utility,
// each fp32 operation rounded once.
struct Decision {
    float e2e, u;
    bool feasible;
};
__device__ inline Decision decide(float ttft, float tpot, float nout, const Rule &R, const QueryRule &q,
                                  float quality) {
    Decision r;
    r.e2e = __fmaf_rn(tpot, nout, ttft);
    const float B = R.per_cand ? __fmaf_rn(nout, R.tpot_slo, q.base) : q.bound.slo;
    r.feasible = r.e2e <= B;
    if (R.score_paper) {
        r.u = __fsub_rn(__fmul_rn(q.w1, quality), __fmul_rn(q.w, r.e2e));
    } else {
        float t;
        if (R.per_cand) {
            asm volatile("");     // a real branch: the division stays off the other paths
            t = __fdiv_rn(r.e2e, B);
        } else {
            t = div_bound(r.e2e, q.bound);
        }
        r.u = __fsub_rn(quality, __fmul_rn(q.w, t));
    }
    return r;
}

// Running best candidate of one lane (Eq. 3), offered candidates in
// increasing pair order: feasibility first, then utility; a candidate
// replaces the best only when strictly better, so ties keep the lower pair
// index.  A NaN utility ranks as -inf and -0 as +0, exactly as in
// decision_key (the stored utility takes the same canonical value); the key
// is built once, for the reduction across lanes.
struct Best {
    float u, e2e, tt, tp, n;      // n: the candidate's N_out
    int d;                        // -1: no candidate yet
    bool f;
};
__device__ inline Best best_none() {
    Best b;
    b.u = -__builtin_huge_valf();
    b.e2e = b.tt = b.tp = b.n = 0.0f;
    b.d = -1;
    b.f = false;
    return b;
}
// TrackN: keep the candidate's N_out (it varies per candidate only when a
// third head predicts it; otherwise the caller knows it).
template <bool TrackN = true>
__device__ inline void offer(Best &b, const Decision &r, int d, float tt, float tp, float n) {
    const float u = fmaxf(r.u, -__builtin_huge_valf()) + 0.0f;   // NaN -> -inf, -0 -> +0
    // (bitwise, not short-circuit: no branches)
    const bool better = (b.d < 0) | (r.feasible & !b.f) | ((r.feasible == b.f) & (u > b.u));
    // selects, not a branch: one v_cndmask per field
    b.u = better ? u : b.u;
    b.e2e = better ? r.e2e : b.e2e;
    b.tt = better ? tt : b.tt;
    b.tp = better ? tp : b.tp;
    if constexpr (TrackN) b.n = better ? n : b.n;
    b.d = better ? d : b.d;
    b.f = better ? r.feasible : b.f;
}
__device__ inline uint64_t best_key(const Best &b) { return b.d < 0 ? 0 : decision_key(b.f, b.u, b.d); }

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

// Cross-lane steps on DPP (data-parallel primitives inside a 16-lane row):
// quad permutes, half-row and row mirrors; no LDS round trip.
template <int Ctrl>
__device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
    return static_cast<uint32_t>(__builtin_amdgcn_update_dpp(0, static_cast<int>(v), Ctrl, 0xF, 0xF, false));
}
template <int Ctrl>
__device__ __forceinline__ uint64_t max_dpp(uint64_t k) {
    const uint64_t o = (static_cast<uint64_t>(dpp_u32<Ctrl>(static_cast<uint32_t>(k >> 32))) << 32) |
                       dpp_u32<Ctrl>(static_cast<uint32_t>(k));
    return o > k ? o : k;
}
// Cross-lane reductions on DPP (data-parallel primitives within a 16-lane
// row: quad permutes, half-row and row mirrors), then one read of each row's
// lane 0; no LDS round trips.  After the four steps every lane of a row holds
// the row's result.
__device__ __forceinline__ float wave_sum(float v) {
    v += __uint_as_float(dpp_u32<0xB1>(__float_as_uint(v)));    // quad_perm [1,0,3,2]
    v += __uint_as_float(dpp_u32<0x4E>(__float_as_uint(v)));    // quad_perm [2,3,0,1]
    v += __uint_as_float(dpp_u32<0x141>(__float_as_uint(v)));   // row_half_mirror
    v += __uint_as_float(dpp_u32<0x140>(__float_as_uint(v)));   // row_mirror
    const int b = __float_as_int(v);
    return (__int_as_float(__builtin_amdgcn_readlane(b, 0)) + __int_as_float(__builtin_amdgcn_readlane(b, 16))) +
           (__int_as_float(__builtin_amdgcn_readlane(b, 32)) + __int_as_float(__builtin_amdgcn_readlane(b, 48)));
}
// Maximum of a key over aligned groups of G lanes (G a power of two <= 64,
// the same in the whole wave); every lane of a group receives it.  Lanes
// without a candidate hold 0.
__device__ inline uint64_t group_max_u64(uint64_t k, int G) {
    if (G > 1) k = max_dpp<0xB1>(k);     // quad_perm [1,0,3,2]: lane ^ 1
    if (G > 2) k = max_dpp<0x4E>(k);     // quad_perm [2,3,0,1]: lane ^ 2
    if (G > 4) k = max_dpp<0x141>(k);    // row_half_mirror: the other quad of 8
    if (G > 8) k = max_dpp<0x140>(k);    // row_mirror: the other 8 of 16
    for (int off = 16; off < G; off <<= 1) {
        const uint64_t o = shfl_xor_u64(k, off);
        k = o > k ? o : k;
    }
    return k;
}

__device__ inline void write_outputs(const OutArgs &o, int q, uint64_t key, float u,
                                     float e2e, float ttft, float tpot, float nout) {
    if (!o.choice) return;        // decisions taken by a later kernel
    o.choice[q] = key_pair(key);
    if (o.feasible) o.feasible[q] = key_feasible(key) ? 1 : 0;
    if (o.utility) o.utility[q] = u;
    if (o.e2e) o.e2e[q] = e2e;
    if (o.ttft) o.ttft[q] = ttft;
    if (o.tpot) o.tpot[q] = tpot;
    if (o.nout) o.nout[q] = nout;
}

}  // namespace hwr
