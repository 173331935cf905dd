// Single-query routing kernel of libhwr (gfx950): one query against all
// pairs in one workgroup, reading the query and the pairs' current runtime
// signals from pinned host memory and writing the decision there, so that
// one launch (captured once in a graph) is the whole call -- or, in the
// resident form, one launch serves a stream of queries.  Pairs are the MFMA
// columns here (32 per tile); the 4 waves split the second-layer row tiles
// and combine their head partials in LDS.  The quality of every model is
// computed once per query, a 16-lane row per model.
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

// Thread j (0..7) of a pair's group of eight writes feature slots j, j + 8,
// j + 16, j + 24 of its row.  The eight signal slots b .. b + 7 meet each
// residue mod 8 once, so the thread evaluates exactly one signal: number
// (j - b) mod 8 (Eq. 1 layout; the query's input length is signal 1).  Logs
// in fp64 (ln_pos), rounded once to fp32, then to bf16 (as the state kernel does).
__device__ __forceinline__ void pair_row(uint16_t *row, int j, int b0, int ks, int ia, int ig,
                                         uint32_t raw, float params, int32_t len, bool fold) {
    double arg = 1.0, scale = 0.0;
    if (ks == 0) { arg = static_cast<double>(params); scale = 0.25; }
    if (ks == 1) { arg = static_cast<double>(len < 1 ? 1 : len); scale = 0.125; }
    if (ks == 2 || ks == 3) { arg = 1.0 + static_cast<double>(static_cast<int32_t>(raw)); scale = 0.5; }
    if (ks == 6 || ks == 7) { arg = static_cast<double>(__uint_as_float(raw)); scale = 0.25; }
    float v = static_cast<float>(ln_pos(arg) * scale);
    if (ks == 4 || ks == 5) v = __uint_as_float(raw);
    const uint16_t sig = bf16_bits(v);
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const int f = j + 8 * i;
        const uint16_t hot = (f == ia || f == ig || (fold && f >= kFoldSlot)) ? 0x3F80 : 0;
        row[f] = (f >= b0 && f < b0 + 8) ? sig : hot;
    }
}

// Sum over each 16-lane row on DPP: every lane of the row ends with the same
// total (each step adds a lane's value to its partner's, both orders giving
// the same fp32 result).
__device__ __forceinline__ float row_sum16(float v) {
    v += __uint_as_float(dpp_u32<0xB1>(__float_as_uint(v)));    // quad_perm [1,0,3,2]
    v += __uint_as_float(dpp_u32<0x4E>(__float_as_uint(v)));    // quad_perm [2,3,0,1]
    v += __uint_as_float(dpp_u32<0x141>(__float_as_uint(v)));   // row_half_mirror
    v += __uint_as_float(dpp_u32<0x140>(__float_as_uint(v)));   // row_mirror
    return v;
}

// Dot product of eight bf16 pairs, fp32 accumulation.  (Each element goes
// through a named scalar before its bit cast: this compiler reads element 0
// for a bit cast taken of a vector subscript directly.)
__device__ __forceinline__ float dot8_bf16(const bf16x8 &x, const bf16x8 &y) {
    const u32x4 a = __builtin_bit_cast(u32x4, x), b = __builtin_bit_cast(u32x4, y);
    float s = 0.0f;
#pragma unroll
    for (int t = 0; t < 4; ++t) {
        const uint32_t ua = a[t], ub = b[t];
        s = __builtin_amdgcn_fdot2_f32_bf16(__builtin_bit_cast(bf16x2, ua), __builtin_bit_cast(bf16x2, ub), s, false);
    }
    return s;
}

// The same pointer, held in vector registers: loads through it are vector
// loads.  (A load from a pointer every lane shares becomes a scalar load,
// which this compiler schedules after earlier vector loads have been waited
// for; from host memory that is a second round trip.)
template <class T>
__device__ __forceinline__ const __attribute__((address_space(1))) T *per_lane(const T *p) {
    uint64_t v = reinterpret_cast<uint64_t>(p);
    asm volatile("" : "+v"(v));
    return reinterpret_cast<const __attribute__((address_space(1))) T *>(v);
}

// Cross-lane maximum on DPP (see wave_sum), then one read of each row's lane 0.
__device__ __forceinline__ uint64_t wave_max(uint64_t k) {
    k = max_dpp<0xB1>(k);
    k = max_dpp<0x4E>(k);
    k = max_dpp<0x141>(k);
    k = max_dpp<0x140>(k);
    uint64_t best = 0;
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        const uint64_t o = (static_cast<uint64_t>(static_cast<uint32_t>(
                                __builtin_amdgcn_readlane(static_cast<int>(k >> 32), 16 * r))) << 32) |
                           static_cast<uint32_t>(__builtin_amdgcn_readlane(static_cast<int>(k), 16 * r));
        best = o > best ? o : best;
    }
    return best;
}

// RES = false: one launch per query.  RES = true: the resident form, one
// launch serving successive queries.  Thread 0 polls the request record's
// sequence number (pinned host memory, system scope) and the workgroup
// serves each new request in turn.  The weights and the pairs' static
// features are loaded for the first request only; the signals, the query
// and the feature rows are read again for every request, after a
// system-scope acquire.  The workgroup leaves when the host sets `quit`, or
// after max_polls polls without a request: every wait ends.
template <int H, bool RES>
__global__ __launch_bounds__(256) void k_single(SingleArgs a) {
    constexpr int MT = H / 32, KB2 = H / 16;
    constexpr int MO = (MT + 3) / 4;          // second-layer row tiles per wave
    constexpr int kW1 = MT * 128 / 256;       // 16-byte pieces of w1 per thread
    constexpr int kEmb = 4;                   // 16-byte embedding pieces per thread (D <= 8192)
    constexpr int kQP = 8;                    // quality: 16-byte weight pieces held per lane (D <= 1024)
    __shared__ bf16x8 s_w1[MT * 2 * 64];
    __shared__ u32x4 s_bw[2][MT * 8];         // b1 tiles, b2 tiles
    __shared__ u32x4 s_w3p[MT * 4 * kMaxHeads];   // head pairs: [tile][half][head][2]
    __shared__ __attribute__((aligned(16))) uint16_t s_emb[8192];
    __shared__ __attribute__((aligned(16))) uint16_t s_row[kMaxPairs][kFeatPad];   // bf16 rows
    __shared__ int s_model[kMaxPairs];
    __shared__ float s_bq[kMaxModels];
    __shared__ float s_q[kMaxModels];
    __shared__ float s_z[4][32][kMaxHeads];
    __shared__ bf16x8 s_h1[KB2][64];          // first-layer activations of the tile's 32 pairs
    __shared__ uint32_t s_ctl[2];             // resident: request found, its sequence number
    const int NH = a.nheads;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, n = lane & 31, h = lane >> 5;
    // quality: row r of wave w (16 lanes) takes models 4w + r, 4w + r + 16;
    // lane l16 of the row takes the 16-byte pieces l16, l16 + 16, ... of D
    const int l16 = lane & 15, mq = 4 * wave + (lane >> 4), D8 = a.D >> 3;
    const int b0 = a.arch_width + a.gpu_width;
    const int j8 = tid & 7, ks = (j8 - b0) & 7;

    const int p0 = tid >> 3;
    const bool has0 = p0 < a.N;
    const int pc0 = has0 ? p0 : 0;
    // pair p0's static features, and the weights held in registers, live
    // across the requests of the resident form
    float prm0 = 0.0f;
    int ia0 = 0, ig0 = 0, md0 = 0;
    constexpr int MOH = MO == 1 ? 1 : 0;     // second-layer tiles held in registers
    bf16x8 fw2[MO][KB2];
    bf16x8 wqh[kQP];
    uint32_t last = a.last_seq;
    for (int iter = 0;; ++iter) {
        if constexpr (RES) {
            // ---- wait for a request: thread 0 polls, a bounded number of times
            if (tid == 0) {
                uint32_t found = 0, sq = last;
                for (uint32_t it = 0; it < a.max_polls; ++it) {
                    const uint64_t hq = __hip_atomic_load(reinterpret_cast<const uint64_t *>(a.in), __ATOMIC_RELAXED,
                                                          __HIP_MEMORY_SCOPE_SYSTEM);   // seq, quit
                    sq = static_cast<uint32_t>(hq);
                    if (sq != last) {
                        found = 1;
                        break;
                    }
                    if (static_cast<uint32_t>(hq >> 32) != 0) break;
                    __builtin_amdgcn_s_sleep(4);
                }
                s_ctl[0] = found;
                s_ctl[1] = sq;
            }
            __syncthreads();
            if (s_ctl[0] == 0) return;
            last = s_ctl[1];
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "");   // system scope: the request record and the signals
        }
        // ---- phase 1: every independent load is issued before any is waited
        // for -- host memory first (query record, runtime signals), then the
        // device-side weights -- so the phase costs one host round trip.
        // seq, input_len, nout, slo: one dword load each (no unused lanes of a
        // load in flight for the compiler to give to another value)
        const __attribute__((address_space(1))) uint32_t *hp = per_lane(reinterpret_cast<const uint32_t *>(a.in));
        const uint32_t h_seq = hp[0], h_len = hp[2], h_nout = hp[3];
        const float slo = __uint_as_float(hp[4]);
        // (loads are unconditional, indices clamped into range: a load under a
        // branch makes the compiler wait for it, and for all earlier ones, there)
        const uint32_t raw0 = reinterpret_cast<const uint32_t *>(a.state + pc0)[ks >= 2 ? ks - 2 : 0];
        u32x4 re[kEmb];
    #pragma unroll
        for (int i = 0; i < kEmb; ++i) {
            const int idx = tid + 256 * i;
            re[i] = reinterpret_cast<const u32x4 *>(a.in + 1)[idx < a.D / 8 ? idx : 0];
        }
        const bool first = !RES || iter == 0;
        if (first) {
            prm0 = a.pair_params[pc0];
            ia0 = a.pair_arch[pc0];
            ig0 = a.arch_width + a.dep_gpu[pc0];
            md0 = a.dep_model[pc0];
        }
        u32x4 rw1[kW1];
    #pragma unroll
        for (int i = 0; i < kW1; ++i) rw1[i] = first ? reinterpret_cast<const u32x4 *>(a.w1_pk)[tid + 256 * i] : u32x4{};
        // b1 tiles (MT * 8 pieces), b2 tiles (MT * 8), head pairs (MT * 4 * NH)
        const int nbw = MT * 16 + MT * 4 * NH;
        u32x4 rbw;
        {
            const int tb = tid < nbw ? tid : 0;
            const int t = tb < MT * 8 ? 0 : tb < MT * 16 ? 1 : 2;
            const int k = tb - t * (MT * 8);
            const u32x4 *src = reinterpret_cast<const u32x4 *>(t == 0 ? static_cast<const void *>(a.b1_pk)
                                                               : t == 1 ? static_cast<const void *>(a.b2_pk)
                                                                        : static_cast<const void *>(a.w3_pk));
            rbw = first ? src[k] : u32x4{};
        }
        const float rbq = first ? a.bq[tid < a.M ? tid : 0] : 0.0f;
        if (first) {
            const bf16x8 *w2 = reinterpret_cast<const bf16x8 *>(a.w2_pk);
    #pragma unroll
            for (int i = 0; i < MOH; ++i) {
                const int mo = wave + 4 * i < MT ? wave + 4 * i : 0;
    #pragma unroll
                for (int kb = 0; kb < KB2; ++kb) fw2[i][kb] = w2[(mo * KB2 + kb) * 64 + lane];
            }
        }
        if (first) {
            const uint16_t *wm = a.wqT + static_cast<size_t>(mq < a.M ? mq : 0) * a.D;
    #pragma unroll
            for (int i = 0; i < kQP; ++i) {
                const int c = l16 + 16 * i;
                wqh[i] = *reinterpret_cast<const bf16x8 *>(wm + 8 * (c < D8 ? c : 0));
            }
        }
        const uint32_t seq = RES ? last : h_seq;
        const int32_t len = static_cast<int32_t>(h_len);
        const int32_t no = static_cast<int32_t>(h_nout);

        // ---- phase 2: LDS stores, the feature rows, one barrier
    #pragma unroll
        for (int i = 0; i < kEmb; ++i) {
            const int idx = tid + 256 * i;
            if (idx < a.D / 8) reinterpret_cast<u32x4 *>(s_emb)[idx] = re[i];
        }
        if (first) {
    #pragma unroll
            for (int i = 0; i < kW1; ++i) reinterpret_cast<u32x4 *>(s_w1)[tid + 256 * i] = rw1[i];
            if (tid < MT * 16) s_bw[0][tid] = rbw;
            else if (tid < nbw) s_w3p[tid - MT * 16] = rbw;
            if (tid < a.M) s_bq[tid] = rbq;
        }
        if (has0) {
            pair_row(s_row[p0], j8, b0, ks, ia0, ig0, raw0, prm0, len, a.fold_b1 != 0);
            if (j8 == 0) s_model[p0] = md0;
        }
        // more than 32 pairs: eight further pairs per thread per round trip (the
        // signals come from host memory; loads unconditional, indices clamped)
        for (int pb = p0 + 32; pb < a.N; pb += 32 * 8) {
            uint32_t raw[8];
            float prm[8];
            int ia[8], ig[8], md[8];
    #pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int p = pb + 32 * i < a.N ? pb + 32 * i : 0;
                raw[i] = reinterpret_cast<const uint32_t *>(a.state + p)[ks >= 2 ? ks - 2 : 0];
                prm[i] = a.pair_params[p];
                ia[i] = a.pair_arch[p];
                ig[i] = a.arch_width + a.dep_gpu[p];
                md[i] = a.dep_model[p];
            }
    #pragma unroll
            for (int i = 0; i < 8; ++i) {
                const int p = pb + 32 * i;
                if (p < a.N) {
                    pair_row(s_row[p], j8, b0, ks, ia[i], ig[i], ks >= 2 ? raw[i] : 0u, ks == 0 ? prm[i] : 1.0f, len,
                             a.fold_b1 != 0);
                    if (j8 == 0) s_model[p] = md[i];
                }
            }
        }
        __syncthreads();

        const float nout = static_cast<float>(no < 0 ? 0 : no);
        const QueryRule qrule = query_rule(a.rule, slo, len, nout, a.w);
        // ---- quality of every model (Sec. 3.2 item 3), once per request: the
        // held pieces first (all LDS reads issued together, pieces past D
        // masked), further pieces and the second pass of models from memory
        {
            bf16x8 e[kQP];
    #pragma unroll
            for (int i = 0; i < kQP; ++i) {
                const int c = l16 + 16 * i;
                e[i] = reinterpret_cast<const bf16x8 *>(s_emb)[c < D8 ? c : 0];
            }
            float q = 0.0f;
    #pragma unroll
            for (int i = 0; i < kQP; ++i) {
                const float t = dot8_bf16(e[i], wqh[i]);
                q += l16 + 16 * i < D8 ? t : 0.0f;
            }
            const uint16_t *wm = a.wqT + static_cast<size_t>(mq < a.M ? mq : 0) * a.D;
            for (int c = l16 + 16 * kQP; c < D8; c += 16)
                q += dot8_bf16(reinterpret_cast<const bf16x8 *>(s_emb)[c], *reinterpret_cast<const bf16x8 *>(wm + 8 * c));
            q = row_sum16(q);
            if (l16 == 0 && mq < a.M) s_q[mq] = q + s_bq[mq];
            for (int m = mq + 16; m < a.M; m += 16) {     // the same for every lane of a row
                const uint16_t *w = a.wqT + static_cast<size_t>(m) * a.D;
                float q2 = 0.0f;
                for (int c = l16; c < D8; c += 16)
                    q2 += dot8_bf16(reinterpret_cast<const bf16x8 *>(s_emb)[c], *reinterpret_cast<const bf16x8 *>(w + 8 * c));
                q2 = row_sum16(q2);
                if (l16 == 0) s_q[m] = q2 + s_bq[m];
            }
        }
        Best best = best_none();
        const int ntiles = (a.N + 31) / 32;
        for (int ct = 0; ct < ntiles; ++ct) {
            const int d = ct * 32 + n;
            const bool vd = d < a.N;
            const int dc = vd ? d : 0;
            // ---- features of pair d (zero columns past the last pair)
            bf16x8 xf[2];
            {
                const u32x4 *row = reinterpret_cast<const u32x4 *>(s_row[dc]);
                const u32x4 z = {0, 0, 0, 0};
                xf[0] = __builtin_bit_cast(bf16x8, vd ? row[h] : z);
                xf[1] = __builtin_bit_cast(bf16x8, vd ? row[2 + h] : z);
            }
            const int model = s_model[dc];
            // ---- layer 1: wave w computes row tiles w, w + 4, ... (weights
            // from LDS) and shares them through LDS; every wave then takes all
            // of them as its second layer's B operand (a lane holds the same
            // pair and hidden-unit half in every wave)
    #pragma unroll
            for (int i = 0; i < MO; ++i) {
                const int mt = wave + 4 * i;
                if (mt >= MT) break;
                f32x16 acc;
    #pragma unroll
                for (int p = 0; p < 4; ++p) {
                    const f32x4 bt = __builtin_bit_cast(f32x4, s_bw[0][(mt * 2 + h) * 4 + p]);
    #pragma unroll
                    for (int j = 0; j < 4; ++j) acc[4 * p + j] = bt[j];
                }
    #pragma unroll
                for (int kb = 0; kb < 2; ++kb) acc = mfma32s(s_w1[(mt * 2 + kb) * 64 + lane], xf[kb], acc);
                s_h1[2 * mt][lane] = relu_pack8s(acc, 0);
                s_h1[2 * mt + 1][lane] = relu_pack8s(acc, 8);
            }
            __syncthreads();
            bf16x8 h1[KB2];
    #pragma unroll
            for (int kb = 0; kb < KB2; ++kb) h1[kb] = s_h1[kb][lane];
            // ---- layer 2 row tiles of this wave, folded into the heads
            float z0 = 0.0f, z1 = 0.0f, z2 = 0.0f;
    #pragma unroll
            for (int i = 0; i < MO; ++i) {
                if (wave + 4 * i >= MT) break;
                const int mo = wave + 4 * i;
                if (i >= MOH) {
                    const bf16x8 *w2 = reinterpret_cast<const bf16x8 *>(a.w2_pk);
    #pragma unroll
                    for (int kb = 0; kb < KB2; ++kb) fw2[i][kb] = w2[(mo * KB2 + kb) * 64 + lane];
                }
                f32x16 acc;
    #pragma unroll
                for (int p = 0; p < 4; ++p) {
                    const f32x4 bt = __builtin_bit_cast(f32x4, s_bw[1][(mo * 2 + h) * 4 + p]);
    #pragma unroll
                    for (int j = 0; j < 4; ++j) acc[4 * p + j] = bt[j];
                }
    #pragma unroll
                for (int kb = 0; kb < KB2; ++kb) acc = mfma32s(fw2[i][kb], h1[kb], acc);
                const u32x4 *w3 = &s_w3p[(mo * 2 + h) * 2 * NH];
                const u32x4 wa = w3[0], wb = w3[1], wc = w3[2], wd = w3[3];
                const u32x4 we = NH == 3 ? w3[4] : u32x4{0, 0, 0, 0};
                const u32x4 wf = NH == 3 ? w3[5] : u32x4{0, 0, 0, 0};
    #pragma unroll
                for (int p = 0; p < 8; ++p) {
                    const bf16x2 hp = relu_bf16x2(acc[2 * p], acc[2 * p + 1]);
                    const uint32_t u0 = p < 4 ? wa[p & 3] : wb[p & 3];
                    const uint32_t u1 = p < 4 ? wc[p & 3] : wd[p & 3];
                    const uint32_t u2 = p < 4 ? we[p & 3] : wf[p & 3];
                    z0 = __builtin_amdgcn_fdot2_f32_bf16(hp, __builtin_bit_cast(bf16x2, u0), z0, false);
                    z1 = __builtin_amdgcn_fdot2_f32_bf16(hp, __builtin_bit_cast(bf16x2, u1), z1, false);
                    z2 = __builtin_amdgcn_fdot2_f32_bf16(hp, __builtin_bit_cast(bf16x2, u2), z2, false);
                }
            }
            z0 += __shfl_xor(z0, 32);
            z1 += __shfl_xor(z1, 32);
            z2 += __shfl_xor(z2, 32);
            if (h == 0) {
                s_z[wave][n][0] = z0;
                s_z[wave][n][1] = z1;
                s_z[wave][n][2] = z2;
            }
            __syncthreads();
            // ---- heads, cost, decision (Eq. 2, Eq. 3)
            if (wave == 0 && h == 0 && vd) {
                const float zz0 = s_z[0][n][0] + s_z[1][n][0] + s_z[2][n][0] + s_z[3][n][0];
                const float zz1 = s_z[0][n][1] + s_z[1][n][1] + s_z[2][n][1] + s_z[3][n][1];
                const float tt = softplus_fast(zz0 + a.b3_0);
                const float tp = softplus_fast(zz1 + a.b3_1);
                float nc = nout;             // N_out: the query's, or the third head's prediction
                if (NH == 3) {
                    const float zz2 = s_z[0][n][2] + s_z[1][n][2] + s_z[2][n][2] + s_z[3][n][2];
                    nc = softplus_fast(zz2 + a.b3_2);
                }
                offer(best, decide(tt, tp, nc, a.rule, qrule, s_q[model]), d, tt, tp, nc);
            }
            if (ct + 1 < ntiles) __syncthreads();
        }
        if (wave == 0) {
            const uint64_t bkey = best_key(best);
            const uint64_t k = wave_max(bkey);
            if (bkey == k && k != 0) {
                SingleOut *o = a.out;
                o->choice = key_pair(k);
                o->feasible = key_feasible(k) ? 1u : 0u;
                o->utility = best.u;
                o->e2e = best.e2e;
                o->ttft = best.tt;
                o->tpot = best.tp;
                o->nout = best.n;
                // the release store orders this thread's record writes before
                // the sequence number, at system scope
                __hip_atomic_store(&o->seq, seq, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
            }
        }
        if constexpr (!RES) break;
    }   // requests
}

hipError_t launch_single(int H, bool resident, const SingleArgs &a, hipStream_t s) {
    if (resident) {
        switch (H) {
            case 64: return launch_kernel(k_single<64, true>, dim3(1), dim3(256), 0, s, a);
            case 128: return launch_kernel(k_single<128, true>, dim3(1), dim3(256), 0, s, a);
            case 256: return launch_kernel(k_single<256, true>, dim3(1), dim3(256), 0, s, a);
            default: return hipErrorInvalidValue;
        }
    }
    switch (H) {
        case 64: return launch_kernel(k_single<64, false>, dim3(1), dim3(256), 0, s, a);
        case 128: return launch_kernel(k_single<128, false>, dim3(1), dim3(256), 0, s, a);
        case 256: return launch_kernel(k_single<256, false>, dim3(1), dim3(256), 0, s, a);
        default: return hipErrorInvalidValue;
    }
}

}  // namespace hwr
