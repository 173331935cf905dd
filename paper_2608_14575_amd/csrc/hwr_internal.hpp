// Internal definitions shared by the HIP kernels and the host runtime of
// libhwr (gfx950 only).  Nothing here is part of the public C ABI.
#pragma once

#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <cstddef>
#include <cstdint>

#include "hwr.h"

namespace hwr {

constexpr int kFeatPad = 32;     // feature slots padded to two 16-wide MFMA k-blocks
constexpr int kQualTile = 32;    // quality GEMM: models padded to one 32-wide tile
constexpr int kBlock = 256;      // threads per workgroup of the batch kernels
constexpr int kQPerWave = 64;    // fused predictor: queries per wave (two 32-column tiles)
constexpr int kQPerBlock = kQPerWave * 4;   // four query sub-blocks per workgroup
constexpr int kMlpThreads = 512;             // predictor workgroup with two column tiles per wave: 8 waves
constexpr int kGatherQ = 256;    // feature gather: queries per workgroup (one wave per SIMD)
constexpr int kMaxPairs = 1024;
constexpr int kMaxModels = 32;
constexpr int kMaxHeads = 3;     // predictor outputs: TTFT, TPOT and (optionally) N_out
constexpr int kPartVals = 8;     // floats per split partial: u, C, TTFT, TPOT, N_out, pad
constexpr int kMaxWeights = 8;   // cost weights scored in one call (HWR_MAX_WEIGHTS)
// Layer-1 bias folded into the first MFMA layer (bf16 predictor): feature
// slots kFoldSlot .. kFoldSlot + 2 of the bf16 pair rows hold 1.0 and the
// packed W1 rows there hold b1 split into three bf16 parts.  Those slots are
// past every feature (the layout puts zeros after the eight signals), so the
// weights they replace never contribute.
constexpr int kFoldSlot = kFeatPad - 3;
// Pair-major per-candidate buffers ([pair][query]: predictions, staged
// features) space consecutive pairs by the chunk's query count rounded up to
// whole 16-byte groups of fp32 values, so that every pair's row starts
// 16-byte aligned.
constexpr int kPairAlign = 4;
__host__ __device__ constexpr int pair_stride(int nq) { return (nq + kPairAlign - 1) / kPairAlign * kPairAlign; }

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef short i16x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

// Kernel-timing events for the next launch on this thread.  When set (the
// host runtime sets them around each timed launch), the launch hands them to
// the dispatch, which records the kernel's own start and end (not the gap
// before it), and marks them used.
struct LaunchEvents {
    hipEvent_t start = nullptr, stop = nullptr;
    bool used = false;
};
LaunchEvents &launch_events();

// Every kernel of the library is launched through this.
template <typename... Args, typename F = void (*)(Args...)>
inline hipError_t launch_kernel(F kernel, dim3 grid, dim3 block, uint32_t shm, hipStream_t s, Args... args) {
    LaunchEvents &ev = launch_events();
    if (ev.start) {
        hipExtLaunchKernelGGL(kernel, grid, block, shm, s, ev.start, ev.stop, 0u, args...);
        ev.used = true;
    } else {
        hipLaunchKernelGGL(kernel, grid, block, shm, s, args...);
    }
    return hipGetLastError();
}

// Row of output element r (0..15) held by a lane of half h (lane >> 5) in the
// accumulator of a 32x32 MFMA; the column is lane & 31.
__host__ __device__ constexpr int crow(int r, int h) { return 8 * (r >> 2) + 4 * h + (r & 3); }

// Order-preserving map of an fp32 utility onto uint32 (larger u -> larger key).
__host__ __device__ inline uint32_t ord_u32(uint32_t bits) {
    return (bits & 0x80000000u) ? ~bits : (bits | 0x80000000u);
}

// Decision key (Eq. 3): feasibility first, then utility, then the lower pair
// index.  Maximising it as an unsigned integer is exact and associative.
__device__ inline uint64_t decision_key(bool feasible, float u, int d) {
    if (u != u) u = -__builtin_huge_valf();
    if (u == 0.0f) u = 0.0f;
    const uint64_t o = ord_u32(__float_as_uint(u));
    return (static_cast<uint64_t>(feasible) << 63) | (o << 31) |
           static_cast<uint64_t>(0x7FFFFFFF - d);
}
__device__ inline int key_pair(uint64_t k) { return 0x7FFFFFFF - static_cast<int>(k & 0x7FFFFFFFull); }
__device__ inline bool key_feasible(uint64_t k) { return (k >> 63) != 0; }

// ---------------------------------------------------------------- arguments
// Decision rule of a launch (Sec. 3.1 score, Eq. 3 bound).
struct Rule {
    int score_paper;              // 1: u = (1 - w) Q - w C; 0: u = Q - w C / B
    int bound_paper;              // 1: B = a + b * input_len + N_out * tpot_slo; 0: the query's SLO
    int per_cand;                 // bound_paper with N_out predicted per candidate
    float a, b, tpot_slo;
};

struct QueryArgs {
    int nq;                       // queries in this chunk
    const int32_t *input_len;     // [nq]
    const int32_t *nout;          // [nq] given N_out (two-head predictor), else unused
    const float *slo;             // [nq] or nullptr
    float default_slo;
};

struct OutArgs {                  // per query; all but choice may be null
    int32_t *choice;
    uint8_t *feasible;
    float *utility, *e2e, *ttft, *tpot, *nout;
};

struct StateArgs {
    const hwr_hw_state *src;      // [N] (pinned host slot, device-visible)
    int N, arch_width, gpu_width;
    const int32_t *dep_model, *dep_gpu;
    const int32_t *pair_arch;     // [N] architecture id of the pair's model
    const float *pair_params;     // [N] parameter count (B) of the pair's model
    float *dep_f32;               // [N][32]
    uint16_t *dep_bf16;           // [N][32]
    int fold_b1;                  // bf16 rows carry 1.0 in the folded-bias slots
};

struct QualityArgs {
    int nq, D, M;
    const void *emb;              // [nq][D] (bf16 bits or fp32)
    const uint16_t *wq_pk;        // bf16 B-operand fragments
    const float *wq;              // fp32 [D][M]
    const float *bq;              // [M]
    float *qmat;                  // [nq][M]
};

struct MlpArgs {                  // bf16 predictor (fused or staged)
    int N, M, len_slot;
    int nheads;                   // 2, or 3: N_out predicted by the third head
    Rule rule;
    float w;                      // cost weight
    float b3_0, b3_1, b3_2;
    QueryArgs q;
    const uint16_t *dep_bf16;     // [N][32]
    const int32_t *dep_model;     // [N]
    const float *qmat;            // [nq][M]
    const uint16_t *w1_pk, *w2_pk;
    const float *b1_pk, *b2_pk;
    const uint16_t *w3_frag;      // head layer A fragments (compact, see pack_predictor)
    const uint16_t *X;            // staged input [N][ldq][32] (pair-major)
    float *cand_ttft, *cand_tpot; // per-candidate TTFT / TPOT: staged, several weights or debug
    float *cand_nout;             // predicted N_out (three heads), same layout
    int cand_pm;                  // 1: pair-major [N][ldq] (staged always); 0: [nq][N]
    int ldq;                      // pair stride of the pair-major buffers: pair_stride(nq)
    OutArgs out;
    int nsplit;                   // pair ranges (grid.y); >1 writes partials
    int four_tiles;               // the batch fills the device (a workgroup per compute unit or more):
                                  // the four-tile form, where it exists for H
    uint64_t *part_key;           // [nsplit][nq]
    float *part_val;              // [nsplit][nq][kPartVals]
    int fold_b1;                  // b1 is inside W1 (zero accumulator start)
};

struct MlpF32Args {
    int N, F, len_slot, nheads;
    float b3_0, b3_1, b3_2;
    QueryArgs q;
    const float *dep_f32;         // [N][32]
    const float *w1, *b1, *w2, *b2, *w3;   // [F][H], [H], [H][H], [H], [H][nheads]
    float *cand_ttft, *cand_tpot, *cand_nout;   // [N][ldq], pair-major; cand_nout: three heads only
    int ldq;                      // pair_stride(nq)
    int with_quality;             // workgroups past mlp_blocks run `quality`
    int mlp_blocks;               // set by launch_mlp_f32
    QualityArgs quality;
};

struct GatherArgs {
    int N, len_slot;
    QueryArgs q;
    const uint16_t *dep_bf16;     // [N][32]
    uint16_t *X;                  // [N][ldq][32], pair-major
    int ldq;                      // pair_stride(nq)
};

// Decision epilogue over pair-major predictions: candidate (q, d) at d * ldq + q.
struct EpilogueArgs {
    int N, M;
    int ldq;                      // pair_stride(nq)
    Rule rule;
    int nw;                       // cost weights (>= 1); outputs are [nq][nw] when nw > 1
    float w[kMaxWeights];
    QueryArgs q;
    const int32_t *dep_model;
    const float *qmat;            // [nq][M]
    const float *cand_ttft, *cand_tpot;   // [N][ldq], 16-byte aligned
    const float *cand_nout;       // [N][ldq] predicted N_out, or null: the query's given N_out
    float *dbg_ttft, *dbg_tpot, *dbg_nout;   // caller's per-candidate outputs [nq][N], or null
    OutArgs out;
};

struct MergeArgs {
    int nq, nsplit;
    const uint64_t *part_key;
    const float *part_val;
    OutArgs out;
};

// Single query, all pairs: input and output records in pinned host memory.
struct SingleIn {
    uint32_t seq;                 // request number, written last by the host
    uint32_t quit;                // resident kernel: leave (set by the host at teardown)
    int32_t input_len, nout;
    float slo;
    uint32_t pad[3];
    // followed by D bf16 embedding values (16-byte aligned)
};
struct SingleOut {
    uint32_t seq;
    int32_t choice;
    uint32_t feasible;
    float utility, e2e, ttft, tpot;
    float nout;                   // N_out of the chosen pair
};

struct SingleArgs {
    int N, M, D, len_slot, arch_width, gpu_width, nheads;
    Rule rule;
    float w, b3_0, b3_1, b3_2;
    const SingleIn *in;           // device-visible pinned record
    SingleOut *out;               // device-visible pinned record
    const hwr_hw_state *state;    // device-visible pinned copy of the current signals [N]
    const int32_t *dep_model, *dep_gpu;
    const int32_t *pair_arch;     // [N] architecture id of the pair's model
    const float *pair_params;     // [N] parameter count (B) of the pair's model
    const uint16_t *wqT;          // [M][D] bf16
    const float *bq;
    const uint16_t *w1_pk, *w2_pk;
    const float *b1_pk, *b2_pk;
    const uint32_t *w3_pk;
    int fold_b1;                  // feature rows carry 1.0 in the folded-bias slots
    uint32_t last_seq;            // resident: the request answered last (waits for a newer one)
    uint32_t max_polls;           // resident: polls without a request before the kernel leaves
};

// ---------------------------------------------------------------- launchers
// Each returns the launch error (hipSuccess on success).
hipError_t launch_state(const StateArgs &a, hipStream_t s);
// cus: compute units of the device (a grid below it takes the unrolled variant)
hipError_t launch_quality_bf16(const QualityArgs &a, int cus, hipStream_t s);
hipError_t launch_quality_f32(const QualityArgs &a, hipStream_t s);
hipError_t launch_mlp_bf16(int H, bool staged, const MlpArgs &a, hipStream_t s);
int mlp_f32_blocks(long candidates);   // workgroups of launch_mlp_f32's predictor
hipError_t launch_mlp_f32(int H, const MlpF32Args &a, hipStream_t s);
hipError_t launch_gather(const GatherArgs &a, hipStream_t s);
hipError_t launch_epilogue(const EpilogueArgs &a, hipStream_t s);
hipError_t launch_merge(const MergeArgs &a, hipStream_t s);
hipError_t launch_single(int H, bool resident, const SingleArgs &a, hipStream_t s);

}  // namespace hwr
