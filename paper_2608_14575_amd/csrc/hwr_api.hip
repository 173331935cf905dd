// Host runtime of libhwr: the C ABI of include/hwr.h on the HIP runtime.
// Validation, weight re-layout for the MFMA kernels, state ingest, chunked
// batch routing, the graph-launched single-query path, and event timing.
#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cmath>
#include <condition_variable>
#include <cstdio>
#include <cstring>
#include <memory>
#include <mutex>
#include <string>
#include <thread>
#include <vector>

#include "c_boundary.hpp"
#include "hwr_internal.hpp"

using namespace hwr;

namespace hwr {
// Kernel-timing events of the next launch on this thread (see launch_kernel).
LaunchEvents &launch_events() {
    thread_local LaunchEvents ev;
    return ev;
}
}  // namespace hwr

namespace {

thread_local std::string g_init_error;

constexpr int kStateSlots = 64;     // pinned ring of state snapshots
// Resident single-query kernel: polls of the request record before it leaves
// (each one a host-memory round trip plus a short sleep, >= 1 us), and the
// host idle time after which the kernel may have left and is checked for.
constexpr uint32_t kResidentPolls = 1u << 16;
constexpr auto kResidentCheck = std::chrono::milliseconds(20);

struct Pending {
    int kind;
    hipEvent_t a, b;
};

// Work space of one batch route: where the chunk loop keeps the quality
// matrix, the split partials and (staged, fp32 and several-weight routes)
// the per-candidate predictions and features; and how many queries a chunk
// may hold.
struct Workspace {
    float *qmat = nullptr;
    uint64_t *pkey = nullptr;
    float *pval = nullptr;
    size_t part_cap = 0;
    float *ctt = nullptr, *ctp = nullptr, *cno = nullptr;
    uint16_t *X = nullptr;
    int max_chunk = 0;
    bool timing = true;             // kernel timing allowed (it may create events)
};

// Scratch of the entry point that allocates nothing (hwr_route_batch_static):
// one array per device, held until the process ends.  In host code its name
// stands for no device address; its address on each device is taken once,
// with hipGetSymbolAddress, by the first hwr_init on that device.
constexpr size_t kScratchBytes = size_t(64) << 20;
static __device__ __align__(256) unsigned char scratch[kScratchBytes];
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void *g_scratch_ptr[kMaxDevices] = {};

// Host batches in pageable memory: their embeddings pass through a ring of
// pinned slots, each filled by a few host threads while the previous one is
// uploaded (the runtime's own staging of a pageable copy runs on one thread,
// at about half the rate of an upload from pinned memory).
constexpr int kPageSlots = 4;
constexpr size_t kPageSlotBytes = size_t(32) << 20;
constexpr size_t kPageMinBytes = size_t(16) << 20;   // smaller batches keep the runtime's copy

// A few threads that copy one host range into another together with the
// calling thread; one copy at a time (a context is used by one thread).
class CopyPool {
  public:
    explicit CopyPool(int threads) {
        try {
            for (int i = 0; i < threads; ++i) workers_.emplace_back([this] { serve(); });
        } catch (...) {
            stop();                   // a thread could not start: join those that did
            throw;
        }
    }
    ~CopyPool() { stop(); }
    void copy(void *dst, const void *src, size_t bytes) {
        const size_t parts = workers_.size() + 1;
        const size_t piece = std::max<size_t>(size_t(1) << 20, (bytes / parts + 4095) & ~size_t(4095));
        {
            std::lock_guard<std::mutex> l(mu_);
            dst_ = static_cast<char *>(dst);
            src_ = static_cast<const char *>(src);
            bytes_ = bytes;
            piece_ = piece;
            next_ = 0;
            left_ = (bytes + piece - 1) / piece;
            ++gen_;
        }
        wake_.notify_all();
        work();
        std::unique_lock<std::mutex> l(mu_);
        done_.wait(l, [&] { return left_ == 0; });
    }

  private:
    void stop() {
        {
            std::lock_guard<std::mutex> l(mu_);
            stop_ = true;
        }
        wake_.notify_all();
        for (std::thread &t : workers_) t.join();
    }
    void work() {
        for (;;) {
            char *d;
            const char *s;
            size_t n;
            {
                std::lock_guard<std::mutex> l(mu_);
                const size_t off = next_ * piece_;
                if (off >= bytes_) return;
                ++next_;
                d = dst_ + off;
                s = src_ + off;
                n = std::min(piece_, bytes_ - off);
            }
            std::memcpy(d, s, n);
            std::lock_guard<std::mutex> l(mu_);
            if (--left_ == 0) done_.notify_all();
        }
    }
    void serve() {
        uint64_t seen = 0;
        for (;;) {
            {
                std::unique_lock<std::mutex> l(mu_);
                wake_.wait(l, [&] { return stop_ || gen_ != seen; });
                if (stop_) return;
                seen = gen_;
            }
            work();
        }
    }
    std::vector<std::thread> workers_;
    std::mutex mu_;
    std::condition_variable wake_, done_;
    char *dst_ = nullptr;
    const char *src_ = nullptr;
    size_t bytes_ = 0, piece_ = 1, next_ = 0, left_ = 0;
    uint64_t gen_ = 0;
    bool stop_ = false;
};

// What the runtime knows of a host batch's buffer: pinned (page-locked) host
// memory the device reads directly, device memory (not a host buffer at
// all), or anything else (pageable).
enum class HostMem { kPinned, kDevice, kPageable };
HostMem host_mem(const void *p) {
    hipPointerAttribute_t a{};
    const hipError_t e = hipPointerGetAttributes(&a, p);
    (void)hipGetLastError();   // an unregistered pointer may leave its error behind
    if (e != hipSuccess) return HostMem::kPageable;
    if (a.type == hipMemoryTypeHost) return HostMem::kPinned;
    if (a.type == hipMemoryTypeDevice) return HostMem::kDevice;
    return HostMem::kPageable;
}

}  // namespace

struct hwr_ctx {
    // configuration
    int dev = 0;
    hipStream_t stream = nullptr;
    int M = 0, G = 0, N = 0, A = 0, Gw = 0, D = 0, F = 0, H = 0, len_slot = 0;
    int bf16 = 0, pipeline = 0, max_chunk = 0, flags = 0, cus = 0;
    int NH = 2;                   // predictor heads (3: N_out predicted)
    int fold_b1 = 0;              // b1 carried by the first layer's MFMA (bf16)
    float default_slo = 1.0f, b3[kMaxHeads] = {0, 0, 0};
    Rule rule{};                  // score and bound modes
    int nw = 1;                   // cost weights per query (outputs [n][nw] when > 1)
    float w[kMaxWeights] = {};
    // per-pair tables and state
    int32_t *d_dep_model = nullptr, *d_dep_gpu = nullptr, *d_model_arch = nullptr;
    float *d_params = nullptr;
    int32_t *d_pair_arch = nullptr;  // model attributes gathered per pair (single-query path)
    float *d_pair_params = nullptr;
    float *d_dep_f32 = nullptr;
    uint16_t *d_dep_bf16 = nullptr;
    hwr_hw_state *h_ring = nullptr;
    hipEvent_t ring_ev[kStateSlots] = {};
    bool ring_used[kStateSlots] = {};
    int ring_next = 0;
    int state_slot = 0;           // ring slot of the newest snapshot
    bool state_dirty = false;     // newest snapshot not yet turned into pair rows
    bool has_state = false;
    hwr_hw_state *h_cur = nullptr;   // pinned copy of the newest snapshot (single-query path)
    hwr_hw_state *d_cur = nullptr;
    // weights
    float *d_bq = nullptr;
    uint16_t *d_wq_pk = nullptr, *d_wqT = nullptr, *d_w1_pk = nullptr, *d_w2_pk = nullptr;
    float *d_b1_pk = nullptr, *d_b2_pk = nullptr;
    uint32_t *d_w3_pk = nullptr;
    uint16_t *d_w3_frag = nullptr;
    float *d_wq = nullptr, *d_w1 = nullptr, *d_w2 = nullptr, *d_w3 = nullptr, *d_b1 = nullptr,
          *d_b2 = nullptr;
    // work space
    float *d_qmat = nullptr, *d_ctt = nullptr, *d_ctp = nullptr, *d_cno = nullptr;
    uint16_t *d_X = nullptr;
    uint64_t *d_pkey = nullptr;
    float *d_pval = nullptr;
    size_t part_cap = 0;
    void *scratch = nullptr;          // this device's static scratch (hwr_route_batch_static)
    // host-memory batches: device staging.  Inputs are double-buffered (the
    // next chunk's upload overlaps this chunk's kernels); outputs are ordered
    // on the context's stream and need one set.
    size_t hs_cap = 0;
    struct InStage {
        void *emb = nullptr;
        int32_t *len = nullptr, *nout = nullptr;
        float *slo = nullptr;
        hipEvent_t copied = nullptr;   // the upload into this set has finished
        hipEvent_t read = nullptr;     // the kernels that read this set have finished
        bool used = false;
    } hin[2];
    hipStream_t cstream = nullptr;   // upload stream of host-memory batches
    struct PageSlot {
        void *buf = nullptr;           // pinned, kPageSlotBytes
        hipEvent_t done = nullptr;     // its last upload has finished
        bool used = false;
    } pslot[kPageSlots];
    int pslot_next = 0;
    std::unique_ptr<CopyPool> copier;  // set up by the first pageable host batch
    bool page_failed = false;          // the pinned ring could not be set up: the runtime copies
    int32_t *d_hchoice = nullptr;
    float *d_hval = nullptr, *d_hcand = nullptr, *d_hqual = nullptr;
    uint8_t *d_hfeas = nullptr;
    // single-query path
    SingleIn *h_sin = nullptr;
    SingleOut *h_sout = nullptr;
    SingleIn *d_sin = nullptr;
    SingleOut *d_sout = nullptr;
    uint32_t seq = 0;
    hipStream_t sstream = nullptr;   // private stream of the single-query path
    bool res_launched = false;       // resident single-query kernel launched at least once
    bool res_stopping = false;       // asked to leave by a batch (which needs every compute unit)
    std::chrono::steady_clock::time_point res_last{};   // end of the last resident request
    hipGraph_t graph = nullptr;
    hipGraphExec_t gexec = nullptr;
    // timing
    bool prof = false;
    bool no_timing = false;           // set while a route must not create events
    int prof_every = 1;               // time one launch in prof_every of each kind
    int64_t prof_seen[HWR_K_COUNT] = {};
    std::vector<Pending> pending;
    std::vector<hipEvent_t> pool;
    double acc_ms[HWR_K_COUNT] = {};
    int64_t acc_n[HWR_K_COUNT] = {};
    std::string err;
};

namespace {

hwr_status fail(hwr_ctx *c, hwr_status s, const std::string &msg) {
    if (c) c->err = msg;
    else g_init_error = msg;
    return s;
}

hwr_status hip_fail(hwr_ctx *c, hipError_t e, const char *what) {
    std::string m = std::string(what) + ": " + hipGetErrorName(e) + " (" + hipGetErrorString(e) + ")";
    return fail(c, e == hipErrorOutOfMemory ? HWR_ERR_OOM : HWR_ERR_HIP, m);
}

#define HWR_HIP(ctx, call)                                           \
    do {                                                             \
        hipError_t e_ = (call);                                      \
        if (e_ != hipSuccess) return hip_fail((ctx), e_, #call);     \
    } while (0)

template <class T>
hipError_t dev_alloc(T **p, size_t count) {
    *p = nullptr;
    if (count == 0) count = 1;
    return hipMalloc(reinterpret_cast<void **>(p), count * sizeof(T));
}

template <class T>
hipError_t upload(T **p, const T *src, size_t count) {
    hipError_t e = dev_alloc(p, count);
    if (e != hipSuccess) return e;
    return hipMemcpy(*p, src, count * sizeof(T), hipMemcpyHostToDevice);
}

bool finite(float v) { return std::isfinite(v); }

// ---------------------------------------------------------------- weight re-layout
// Quality GEMM B operand: for 64-wide slice s, k-block c and lane (n, h),
// element j holds Wq[64 s + 32 h + 8 c + j][n] (zero for padded models).
std::vector<uint16_t> pack_quality(const uint16_t *wq, int D, int M) {
    std::vector<uint16_t> out(static_cast<size_t>(D) * kQualTile, 0);
    for (int s = 0; s < D / 64; ++s)
        for (int c = 0; c < 4; ++c)
            for (int lane = 0; lane < 64; ++lane) {
                const int n = lane & 31, h = lane >> 5;
                for (int j = 0; j < 8; ++j) {
                    const int k = 64 * s + 32 * h + 8 * c + j;
                    out[((static_cast<size_t>(s) * 4 + c) * 64 + lane) * 8 + j] =
                        n < M ? wq[static_cast<size_t>(k) * M + n] : 0;
                }
            }
    return out;
}

// Predictor A operands.  Layer 1 (W1^T, 32-row tile mt, k-block kb): lane
// (m, h) element j = W1[16 kb + 8 h + j][32 mt + m], zero past F.  Layer 2
// (W2^T, tile mo, k-block kb = 2 t + b): the k order follows the layer-1
// accumulator: element j of lane half h multiplies hidden unit
// 32 t + crow(8 b + j, h).  Bias tiles hold b[32 mt + crow(r, h)] for
// r = 0..15; head pairs hold (W3[row(2p)][o], W3[row(2p+1)][o]) as bf16x2,
// [tile][half][head o][8 pairs].  W3 is [H][NH] (NH = 2 or 3 heads).
struct PackedPredictor {
    std::vector<uint16_t> w1, w2, w3frag;
    std::vector<float> b1, b2;
    std::vector<uint32_t> w3;
};

// bf16 nearest-even bits of a finite fp32 value, and back.
uint16_t bf16_rne(float x) {
    uint32_t u;
    std::memcpy(&u, &x, 4);
    return static_cast<uint16_t>((u + 0x7FFFu + ((u >> 16) & 1u)) >> 16);
}
float bf16_value(uint16_t b) {
    const uint32_t u = static_cast<uint32_t>(b) << 16;
    float x;
    std::memcpy(&x, &u, 4);
    return x;
}

// b = hi + mid + lo exactly, each part a bf16 (8 significant bits apiece; each
// residual is exact in fp32).  False when a part would not be exact (values
// near the bottom of the exponent range), or b is not finite.
bool bf16_split3(float b, uint16_t parts[3]) {
    if (!std::isfinite(b)) return false;
    float r = b;
    for (int i = 0; i < 3; ++i) {
        parts[i] = bf16_rne(r);
        r = r - bf16_value(parts[i]);
    }
    return r == 0.0f &&
           static_cast<double>(bf16_value(parts[0])) + static_cast<double>(bf16_value(parts[1])) +
                   static_cast<double>(bf16_value(parts[2])) == static_cast<double>(b);
}

// Whether the layer-1 bias can ride in the first MFMA layer: bf16 weights,
// three feature slots free after the eight signals, and b1 split exactly.
bool can_fold_b1(const float *b1, int A, int Gw, int H) {
    if (A + Gw + 8 > kFoldSlot) return false;
    uint16_t parts[3];
    for (int i = 0; i < H; ++i)
        if (!bf16_split3(b1[i], parts)) return false;
    return true;
}

PackedPredictor pack_predictor(const uint16_t *w1, const uint16_t *w2, const uint16_t *w3,
                               const float *b1, const float *b2, int F, int H, int NH, bool fold_b1) {
    const int MT = H / 32, KB2 = H / 16;
    PackedPredictor p;
    p.w1.assign(static_cast<size_t>(MT) * 2 * 64 * 8, 0);
    p.w2.assign(static_cast<size_t>(MT) * KB2 * 64 * 8, 0);
    p.b1.assign(static_cast<size_t>(MT) * 2 * 16, 0.0f);
    p.b2.assign(static_cast<size_t>(MT) * 2 * 16, 0.0f);
    p.w3.assign(static_cast<size_t>(MT) * 2 * NH * 8, 0u);
    // Head layer on MFMA (z = W3^T h2^T, 16x16x32 tiles): an A-operand lane
    // holds either the 8 weights of head m over the 8 hidden units that one
    // layer-2 accumulator half h packs into a B operand, or zeros.  Per
    // k-block: [head m][half h][8] for the 2 * NH data fragments, then one zero
    // fragment (k_mlp_bf16 picks the fragment of each lane).
    const int W3S = 2 * NH + 1;
    p.w3frag.assign(static_cast<size_t>(KB2) * W3S * 8, 0);
    for (int kb = 0; kb < KB2; ++kb)
        for (int m = 0; m < NH; ++m)
            for (int h = 0; h < 2; ++h)
                for (int j = 0; j < 8; ++j) {
                    const int hin = 32 * (kb >> 1) + crow(8 * (kb & 1) + j, h);
                    p.w3frag[(static_cast<size_t>(kb) * W3S + m * 2 + h) * 8 + j] =
                        w3[static_cast<size_t>(hin) * NH + m];
                }
    for (int mt = 0; mt < MT; ++mt)
        for (int lane = 0; lane < 64; ++lane) {
            const int m = lane & 31, h = lane >> 5;
            for (int kb = 0; kb < 2; ++kb)
                for (int j = 0; j < 8; ++j) {
                    const int f = 16 * kb + 8 * h + j;
                    uint16_t v = f < F ? w1[static_cast<size_t>(f) * H + 32 * mt + m] : 0;
                    if (fold_b1 && f >= kFoldSlot) {      // feature 1.0 x bias part
                        uint16_t parts[3];
                        bf16_split3(b1[32 * mt + m], parts);
                        v = parts[f - kFoldSlot];
                    }
                    p.w1[((static_cast<size_t>(mt) * 2 + kb) * 64 + lane) * 8 + j] = v;
                }
            for (int kb = 0; kb < KB2; ++kb)
                for (int j = 0; j < 8; ++j) {
                    const int hin = 32 * (kb >> 1) + crow(8 * (kb & 1) + j, h);
                    p.w2[((static_cast<size_t>(mt) * KB2 + kb) * 64 + lane) * 8 + j] =
                        w2[static_cast<size_t>(hin) * H + 32 * mt + m];
                }
        }
    for (int mt = 0; mt < MT; ++mt)
        for (int h = 0; h < 2; ++h) {
            for (int r = 0; r < 16; ++r) {
                p.b1[(mt * 2 + h) * 16 + r] = fold_b1 ? 0.0f : b1[32 * mt + crow(r, h)];
                p.b2[(mt * 2 + h) * 16 + r] = b2[32 * mt + crow(r, h)];
            }
            for (int o = 0; o < NH; ++o)
                for (int pp = 0; pp < 8; ++pp) {
                    const uint32_t lo = w3[static_cast<size_t>(32 * mt + crow(2 * pp, h)) * NH + o];
                    const uint32_t hi = w3[static_cast<size_t>(32 * mt + crow(2 * pp + 1, h)) * NH + o];
                    p.w3[((mt * 2 + h) * NH + o) * 8 + pp] = lo | (hi << 16);
                }
        }
    return p;
}

// ---------------------------------------------------------------- timing
hipEvent_t take_event(hwr_ctx *c) {
    if (!c->pool.empty()) {
        hipEvent_t e = c->pool.back();
        c->pool.pop_back();
        return e;
    }
    hipEvent_t e = nullptr;
    if (hipEventCreate(&e) != hipSuccess) return nullptr;
    return e;
}

// Time one kernel launch of the library: the two events go into its dispatch
// (launch_kernel), so they mark the kernel's own start and end on the stream.
// Whether this launch of `kind` is one of the sampled ones.
bool sampled(hwr_ctx *c, int kind) {
    return c->prof && !c->no_timing && c->prof_seen[kind]++ % c->prof_every == 0;
}

template <class F>
hipError_t timed_on(hwr_ctx *c, hipStream_t s, int kind, F &&launch) {
    if (!sampled(c, kind)) return launch();
    hipEvent_t a = take_event(c), b = take_event(c);
    if (!a || !b) return hipErrorOutOfMemory;
    LaunchEvents &ev = launch_events();
    ev = LaunchEvents{a, b, false};
    const hipError_t e = launch();
    const bool used = ev.used;
    ev = LaunchEvents{};
    if (e != hipSuccess) return e;
    if (!used) return hipErrorInvalidValue;   // every timed launch is one library kernel
    c->pending.push_back({kind, a, b});
    return hipSuccess;
}

// Time a graph launch: events recorded on the stream before and after it.
template <class F>
hipError_t timed_bracket(hwr_ctx *c, hipStream_t s, int kind, F &&launch) {
    if (!sampled(c, kind)) return launch();
    hipEvent_t a = take_event(c), b = take_event(c);
    if (!a || !b) return hipErrorOutOfMemory;
    hipError_t e = hipEventRecord(a, s);
    if (e != hipSuccess) return e;
    e = launch();
    if (e != hipSuccess) return e;
    e = hipEventRecord(b, s);
    if (e != hipSuccess) return e;
    c->pending.push_back({kind, a, b});
    return hipSuccess;
}

template <class F>
hipError_t timed(hwr_ctx *c, int kind, F &&launch) {
    return timed_on(c, c->stream, kind, static_cast<F &&>(launch));
}

hwr_status drain_timing(hwr_ctx *c) {
    for (const Pending &p : c->pending) {
        HWR_HIP(c, hipEventSynchronize(p.b));
        float ms = 0.0f;
        HWR_HIP(c, hipEventElapsedTime(&ms, p.a, p.b));
        c->acc_ms[p.kind] += ms;
        c->acc_n[p.kind] += 1;
        c->pool.push_back(p.a);
        c->pool.push_back(p.b);
    }
    c->pending.clear();
    return HWR_OK;
}

// ---------------------------------------------------------------- validation
hwr_status check_config(const hwr_config *cfg) {
    auto bad = [](const char *m) { return fail(nullptr, HWR_ERR_INVALID_ARG, m); };
    auto uns = [](const char *m) { return fail(nullptr, HWR_ERR_UNSUPPORTED, m); };
    if (!cfg) return bad("config is NULL");
    const int M = cfg->n_models, G = cfg->n_gpu_types, N = cfg->n_deployments;
    if (M < 1 || G < 1 || N < 1) return bad("n_models, n_gpu_types and n_deployments must be >= 1");
    if (cfg->arch_width < 1 || cfg->gpu_width < G) return bad("arch_width >= 1 and gpu_width >= n_gpu_types required");
    if (cfg->arch_width + cfg->gpu_width + 8 > cfg->feat_dim) return bad("feat_dim must hold both one-hots and 8 signal slots");
    if (cfg->feat_dim > kFeatPad) return uns("feat_dim above 32 is not supported");
    if (M > kMaxModels) return uns("more than 32 models is not supported");
    if (N > kMaxPairs) return uns("more than 1024 pairs is not supported");
    if (cfg->embed_dim < 64 || cfg->embed_dim % 64 != 0 || cfg->embed_dim > 8192)
        return uns("embed_dim must be a multiple of 64 in [64, 8192]");
    if (cfg->emb_dtype != cfg->weight_dtype) return uns("emb_dtype must equal weight_dtype");
    if (cfg->weight_dtype != HWR_F32 && cfg->weight_dtype != HWR_BF16) return bad("unknown dtype");
    if (cfg->weight_dtype == HWR_BF16 && cfg->hidden != 64 && cfg->hidden != 128 && cfg->hidden != 256)
        return uns("bf16 hidden width must be 64, 128 or 256");
    if (cfg->weight_dtype == HWR_F32 && cfg->hidden != 64 && cfg->hidden != 128)
        return uns("fp32 hidden width must be 64 or 128");
    if (cfg->pipeline != HWR_PIPE_FUSED && cfg->pipeline != HWR_PIPE_STAGED) return bad("unknown pipeline");
    if (cfg->flags & ~(HWR_FLAG_GRAPH | HWR_FLAG_RESIDENT)) return bad("unknown flags");
    if (cfg->max_chunk < 0 || cfg->max_chunk > (1 << 22)) return bad("max_chunk must be in [0, 2^22]");
    if (cfg->score_mode != HWR_SCORE_NORMALIZED && cfg->score_mode != HWR_SCORE_PAPER) return bad("unknown score_mode");
    if (cfg->bound_mode != HWR_BOUND_GIVEN && cfg->bound_mode != HWR_BOUND_PAPER) return bad("unknown bound_mode");
    if (cfg->bound_mode == HWR_BOUND_PAPER &&
        (!finite(cfg->ttft_slo_a) || !finite(cfg->ttft_slo_b) || !finite(cfg->tpot_slo) ||
         cfg->ttft_slo_a <= 0.0f || cfg->ttft_slo_b < 0.0f || cfg->tpot_slo < 0.0f))
        return bad("paper bound needs ttft_slo_a > 0 and ttft_slo_b, tpot_slo >= 0 (finite)");
    if (cfg->n_weights < 0 || cfg->n_weights > HWR_MAX_WEIGHTS) return bad("n_weights must be in [0, 8]");
    if (cfg->n_weights > 0 && !cfg->cost_weights) return bad("cost_weights is NULL");
    for (int k = 0; k < (cfg->n_weights > 0 ? cfg->n_weights : 1); ++k) {
        const float w = cfg->n_weights > 0 ? cfg->cost_weights[k] : cfg->cost_weight;
        if (!finite(w) || w < 0.0f) return bad("cost weights must be finite and >= 0");
        if (cfg->score_mode == HWR_SCORE_PAPER && w > 1.0f) return bad("paper-score weights (lambda) must be <= 1");
    }
    if (!finite(cfg->default_slo_s) || cfg->default_slo_s <= 0.0f) return bad("default_slo_s must be finite and > 0");
    if (cfg->n_heads != 0 && cfg->n_heads != 2 && cfg->n_heads != 3) return bad("n_heads must be 2 or 3 (0 means 2)");
    if (!cfg->dep_model || !cfg->dep_gpu || !cfg->model_arch || !cfg->model_params_b || !cfg->wq ||
        !cfg->bq || !cfg->w1 || !cfg->b1 || !cfg->w2 || !cfg->b2 || !cfg->w3 || !cfg->b3)
        return bad("a table or weight pointer is NULL");
    for (int d = 0; d < N; ++d) {
        if (cfg->dep_model[d] < 0 || cfg->dep_model[d] >= M) return bad("dep_model out of range");
        if (cfg->dep_gpu[d] < 0 || cfg->dep_gpu[d] >= G) return bad("dep_gpu out of range");
    }
    for (int m = 0; m < M; ++m) {
        if (cfg->model_arch[m] < 0 || cfg->model_arch[m] >= cfg->arch_width) return bad("model_arch out of range");
        if (!finite(cfg->model_params_b[m]) || cfg->model_params_b[m] <= 0.0f) return bad("model_params_b must be > 0");
        if (!finite(cfg->bq[m])) return bad("bq not finite");
    }
    for (int j = 0; j < cfg->hidden; ++j)
        if (!finite(cfg->b1[j]) || !finite(cfg->b2[j])) return bad("b1/b2 not finite");
    for (int k = 0; k < (cfg->n_heads == 3 ? 3 : 2); ++k)
        if (!finite(cfg->b3[k])) return bad("b3 not finite");
    return HWR_OK;
}

// Teardown: every resource is released even if one of the calls fails, so
// their statuses are deliberately ignored.
void release(hwr_ctx *c) {
    if (!c) return;
    (void)hipSetDevice(c->dev);
    (void)hipStreamSynchronize(c->stream);
    for (const Pending &p : c->pending) {
        (void)hipEventDestroy(p.a);
        (void)hipEventDestroy(p.b);
    }
    for (hipEvent_t e : c->pool) (void)hipEventDestroy(e);
    for (int i = 0; i < kStateSlots; ++i)
        if (c->ring_ev[i]) (void)hipEventDestroy(c->ring_ev[i]);
    if (c->h_sin) __atomic_store_n(&c->h_sin->quit, 1u, __ATOMIC_RELEASE);   // a resident kernel leaves
    if (c->sstream) (void)hipStreamSynchronize(c->sstream);
    if (c->gexec) (void)hipGraphExecDestroy(c->gexec);
    if (c->graph) (void)hipGraphDestroy(c->graph);
    void *dev_ptrs[] = {c->d_dep_model, c->d_dep_gpu, c->d_model_arch, c->d_params, c->d_pair_arch,
                        c->d_pair_params, c->d_dep_f32,
                        c->d_dep_bf16, c->d_bq, c->d_wq_pk, c->d_wqT, c->d_w1_pk, c->d_w2_pk,
                        c->d_b1_pk, c->d_b2_pk, c->d_w3_pk, c->d_w3_frag, c->d_wq, c->d_w1, c->d_w2, c->d_w3,
                        c->d_b1, c->d_b2, c->d_qmat, c->d_ctt, c->d_ctp, c->d_cno, c->d_X, c->d_pkey,
                        c->d_pval, c->hin[0].emb, c->hin[0].len, c->hin[0].nout, c->hin[0].slo,
                        c->hin[1].emb, c->hin[1].len, c->hin[1].nout, c->hin[1].slo, c->d_hchoice,
                        c->d_hval, c->d_hcand, c->d_hqual, c->d_hfeas};
    if (c->cstream) (void)hipStreamSynchronize(c->cstream);
    for (void *p : dev_ptrs)
        if (p) (void)hipFree(p);
    for (auto &h : c->hin) {
        if (h.copied) (void)hipEventDestroy(h.copied);
        if (h.read) (void)hipEventDestroy(h.read);
    }
    if (c->cstream) (void)hipStreamDestroy(c->cstream);
    c->copier.reset();
    for (auto &sl : c->pslot) {
        if (sl.buf) (void)hipHostFree(sl.buf);
        if (sl.done) (void)hipEventDestroy(sl.done);
    }
    if (c->h_ring) (void)hipHostFree(c->h_ring);
    if (c->h_cur) (void)hipHostFree(c->h_cur);
    if (c->sstream) (void)hipStreamDestroy(c->sstream);
    if (c->h_sin) (void)hipHostFree(c->h_sin);
    if (c->h_sout) (void)hipHostFree(c->h_sout);
    delete c;
}

hwr_status init_ctx(hwr_ctx *c, const hwr_config *cfg, const hipDeviceProp_t &prop, hwr_ctx **out);

hwr_status init_impl(const hwr_config *cfg, hwr_ctx **out) {
    hwr_status st = check_config(cfg);
    if (st != HWR_OK) return st;
    int ndev = 0;
    hipError_t e = hipGetDeviceCount(&ndev);
    if (e != hipSuccess || ndev < 1) return fail(nullptr, HWR_ERR_HIP, "no HIP device available");
    if (cfg->device < 0 || cfg->device >= ndev) return fail(nullptr, HWR_ERR_INVALID_ARG, "device ordinal out of range");
    hipDeviceProp_t prop;
    if (hipGetDeviceProperties(&prop, cfg->device) != hipSuccess)
        return fail(nullptr, HWR_ERR_HIP, "hipGetDeviceProperties failed");
    if (std::strncmp(prop.gcnArchName, "gfx950", 6) != 0)
        return fail(nullptr, HWR_ERR_UNSUPPORTED, std::string("library is built for gfx950, device is ") + prop.gcnArchName);

    hwr_ctx *c = new hwr_ctx();
    try {
        return init_ctx(c, cfg, prop, out);
    } catch (...) {
        release(c);                   // a host allocation failed part-way: nothing is left behind
        throw;
    }
}

// Fills a new context; on an error it releases it (bail).
hwr_status init_ctx(hwr_ctx *c, const hwr_config *cfg, const hipDeviceProp_t &prop, hwr_ctx **out) {
    c->dev = cfg->device;
    c->stream = static_cast<hipStream_t>(cfg->stream);
    c->M = cfg->n_models;
    c->G = cfg->n_gpu_types;
    c->N = cfg->n_deployments;
    c->A = cfg->arch_width;
    c->Gw = cfg->gpu_width;
    c->D = cfg->embed_dim;
    c->F = cfg->feat_dim;
    c->H = cfg->hidden;
    c->len_slot = c->A + c->Gw + 1;
    c->bf16 = cfg->weight_dtype == HWR_BF16;
    c->pipeline = cfg->pipeline;
    c->max_chunk = cfg->max_chunk > 0 ? cfg->max_chunk : 65536;
    c->flags = cfg->flags;
    c->rule.score_paper = cfg->score_mode == HWR_SCORE_PAPER;
    c->rule.bound_paper = cfg->bound_mode == HWR_BOUND_PAPER;
    c->rule.a = cfg->ttft_slo_a;
    c->rule.b = cfg->ttft_slo_b;
    c->rule.tpot_slo = cfg->tpot_slo;
    c->nw = cfg->n_weights > 0 ? cfg->n_weights : 1;
    for (int k = 0; k < c->nw; ++k) c->w[k] = cfg->n_weights > 0 ? cfg->cost_weights[k] : cfg->cost_weight;
    c->default_slo = cfg->default_slo_s;
    c->NH = cfg->n_heads == 3 ? 3 : 2;
    c->rule.per_cand = c->rule.bound_paper && c->NH == 3;
    for (int k = 0; k < c->NH; ++k) c->b3[k] = cfg->b3[k];
    c->cus = prop.multiProcessorCount;

    auto bail = [&](hipError_t err, const char *what) {
        hwr_status s = hip_fail(nullptr, err, what);
        release(c);
        return s;
    };
#define INIT_HIP(call)                                   \
    do {                                                 \
        hipError_t e_ = (call);                          \
        if (e_ != hipSuccess) return bail(e_, #call);    \
    } while (0)

    INIT_HIP(hipSetDevice(c->dev));
    if (c->dev >= kMaxDevices) return bail(hipErrorInvalidDevice, "device ordinal above the scratch table");
    {
        std::lock_guard<std::mutex> lock(g_scratch_mu);
        if (!g_scratch_ptr[c->dev]) {
            void *ptr = nullptr;
            INIT_HIP(hipGetSymbolAddress(&ptr, HIP_SYMBOL(scratch)));
            if (!ptr) return bail(hipErrorInvalidSymbol, "hipGetSymbolAddress(scratch) gave no address");
            g_scratch_ptr[c->dev] = ptr;
        }
        c->scratch = g_scratch_ptr[c->dev];
    }
    const int M = c->M, N = c->N, D = c->D, F = c->F, H = c->H;
    INIT_HIP(upload(&c->d_dep_model, cfg->dep_model, N));
    INIT_HIP(upload(&c->d_dep_gpu, cfg->dep_gpu, N));
    INIT_HIP(upload(&c->d_model_arch, cfg->model_arch, M));
    INIT_HIP(upload(&c->d_params, cfg->model_params_b, M));
    INIT_HIP(upload(&c->d_bq, cfg->bq, M));
    {
        std::vector<int32_t> pa(N);
        std::vector<float> pp(N);
        for (int d = 0; d < N; ++d) {
            pa[d] = cfg->model_arch[cfg->dep_model[d]];
            pp[d] = cfg->model_params_b[cfg->dep_model[d]];
        }
        INIT_HIP(upload(&c->d_pair_arch, pa.data(), N));
        INIT_HIP(upload(&c->d_pair_params, pp.data(), N));
    }
    INIT_HIP(dev_alloc(&c->d_dep_f32, static_cast<size_t>(N) * kFeatPad));
    INIT_HIP(dev_alloc(&c->d_dep_bf16, static_cast<size_t>(N) * kFeatPad));
    if (c->bf16) {
        const uint16_t *wq = static_cast<const uint16_t *>(cfg->wq);
        std::vector<uint16_t> wqpk = pack_quality(wq, D, M);
        INIT_HIP(upload(&c->d_wq_pk, wqpk.data(), wqpk.size()));
        std::vector<uint16_t> wqT(static_cast<size_t>(M) * D);
        for (int k = 0; k < D; ++k)
            for (int m = 0; m < M; ++m) wqT[static_cast<size_t>(m) * D + k] = wq[static_cast<size_t>(k) * M + m];
        INIT_HIP(upload(&c->d_wqT, wqT.data(), wqT.size()));
        c->fold_b1 = can_fold_b1(cfg->b1, c->A, c->Gw, H) ? 1 : 0;
        PackedPredictor p = pack_predictor(static_cast<const uint16_t *>(cfg->w1),
                                           static_cast<const uint16_t *>(cfg->w2),
                                           static_cast<const uint16_t *>(cfg->w3), cfg->b1, cfg->b2, F, H,
                                           c->NH, c->fold_b1 != 0);
        INIT_HIP(upload(&c->d_w1_pk, p.w1.data(), p.w1.size()));
        INIT_HIP(upload(&c->d_w2_pk, p.w2.data(), p.w2.size()));
        INIT_HIP(upload(&c->d_b1_pk, p.b1.data(), p.b1.size()));
        INIT_HIP(upload(&c->d_b2_pk, p.b2.data(), p.b2.size()));
        INIT_HIP(upload(&c->d_w3_pk, p.w3.data(), p.w3.size()));
        INIT_HIP(upload(&c->d_w3_frag, p.w3frag.data(), p.w3frag.size()));
    } else {
        INIT_HIP(upload(&c->d_wq, static_cast<const float *>(cfg->wq), static_cast<size_t>(D) * M));
        INIT_HIP(upload(&c->d_w1, static_cast<const float *>(cfg->w1), static_cast<size_t>(F) * H));
        INIT_HIP(upload(&c->d_w2, static_cast<const float *>(cfg->w2), static_cast<size_t>(H) * H));
        INIT_HIP(upload(&c->d_w3, static_cast<const float *>(cfg->w3), static_cast<size_t>(H) * c->NH));
        INIT_HIP(upload(&c->d_b1, cfg->b1, H));
        INIT_HIP(upload(&c->d_b2, cfg->b2, H));
    }
    const size_t chunk = static_cast<size_t>(c->max_chunk);
    const size_t ldq = static_cast<size_t>(pair_stride(c->max_chunk));   // pair-major row stride
    INIT_HIP(dev_alloc(&c->d_qmat, chunk * M));
    // per-candidate predictions in HBM: staged and fp32 paths, and several
    // cost weights (the decisions then run after the predictor)
    if (!c->bf16 || c->pipeline == HWR_PIPE_STAGED || c->nw > 1) {
        INIT_HIP(dev_alloc(&c->d_ctt, ldq * N));
        INIT_HIP(dev_alloc(&c->d_ctp, ldq * N));
        if (c->NH == 3) INIT_HIP(dev_alloc(&c->d_cno, ldq * N));
    }
    if (c->bf16 && c->pipeline == HWR_PIPE_STAGED) INIT_HIP(dev_alloc(&c->d_X, ldq * N * kFeatPad));
    if (c->bf16 && c->pipeline == HWR_PIPE_FUSED) {
        c->part_cap = static_cast<size_t>(2 * c->cus) * kQPerBlock;
        INIT_HIP(dev_alloc(&c->d_pkey, c->part_cap));
        INIT_HIP(dev_alloc(&c->d_pval, c->part_cap * kPartVals));
    }
    INIT_HIP(hipHostMalloc(reinterpret_cast<void **>(&c->h_ring),
                           sizeof(hwr_hw_state) * N * kStateSlots, hipHostMallocMapped));
    for (int i = 0; i < kStateSlots; ++i) INIT_HIP(hipEventCreateWithFlags(&c->ring_ev[i], hipEventDisableTiming));
    INIT_HIP(hipHostMalloc(reinterpret_cast<void **>(&c->h_cur), sizeof(hwr_hw_state) * N,
                           hipHostMallocMapped | hipHostMallocCoherent));
    INIT_HIP(hipHostGetDevicePointer(reinterpret_cast<void **>(&c->d_cur), c->h_cur, 0));
    if (c->bf16) {
        const size_t in_bytes = sizeof(SingleIn) + static_cast<size_t>(D) * 2;
        INIT_HIP(hipHostMalloc(reinterpret_cast<void **>(&c->h_sin), in_bytes,
                               hipHostMallocMapped | hipHostMallocCoherent));
        INIT_HIP(hipHostMalloc(reinterpret_cast<void **>(&c->h_sout), sizeof(SingleOut),
                               hipHostMallocMapped | hipHostMallocCoherent));
        std::memset(c->h_sin, 0, in_bytes);
        std::memset(c->h_sout, 0, sizeof(SingleOut));
        INIT_HIP(hipHostGetDevicePointer(reinterpret_cast<void **>(&c->d_sin), c->h_sin, 0));
        INIT_HIP(hipHostGetDevicePointer(reinterpret_cast<void **>(&c->d_sout), c->h_sout, 0));
        INIT_HIP(hipStreamCreateWithFlags(&c->sstream, hipStreamNonBlocking));
    }
#undef INIT_HIP
    *out = c;
    return HWR_OK;
}

// ---------------------------------------------------------------- batch routing
struct DevBatch {
    int n;
    const void *emb;
    const int32_t *len, *nout;
    const float *slo;
    OutArgs out;
    float *cand_ttft, *cand_tpot, *cand_nout, *cand_quality;
};

// Turn the newest state snapshot into the device pair rows, once, ordered on
// the context's stream before the batch that needs them.
hwr_status sync_state(hwr_ctx *c) {
    if (!c->state_dirty) return HWR_OK;
    const int slot = c->state_slot;
    hwr_hw_state *src = c->h_ring + static_cast<size_t>(slot) * c->N;
    hwr_hw_state *dsrc = nullptr;
    HWR_HIP(c, hipHostGetDevicePointer(reinterpret_cast<void **>(&dsrc), src, 0));
    StateArgs a{dsrc, c->N, c->A, c->Gw, c->d_dep_model, c->d_dep_gpu, c->d_pair_arch,
                c->d_pair_params, c->d_dep_f32, c->d_dep_bf16, c->fold_b1};
    HWR_HIP(c, timed(c, HWR_K_STATE, [&] { return launch_state(a, c->stream); }));
    HWR_HIP(c, hipEventRecord(c->ring_ev[slot], c->stream));
    c->ring_used[slot] = true;
    c->state_dirty = false;
    return HWR_OK;
}

MlpF32Args f32_args(const hwr_ctx *c, const QueryArgs &qa) {
    MlpF32Args fa{};
    fa.N = c->N;
    fa.F = c->F;
    fa.len_slot = c->len_slot;
    fa.b3_0 = c->b3[0];
    fa.b3_1 = c->b3[1];
    fa.b3_2 = c->b3[2];
    fa.nheads = c->NH;
    fa.q = qa;
    fa.dep_f32 = c->d_dep_f32;
    fa.w1 = c->d_w1;
    fa.b1 = c->d_b1;
    fa.w2 = c->d_w2;
    fa.b2 = c->d_b2;
    fa.w3 = c->d_w3;
    return fa;
}

// The context's own work space, allocated by hwr_init for max_chunk queries.
Workspace ctx_workspace(const hwr_ctx *c) {
    Workspace w;
    w.qmat = c->d_qmat;
    w.pkey = c->d_pkey;
    w.pval = c->d_pval;
    w.part_cap = c->part_cap;
    w.ctt = c->d_ctt;
    w.ctp = c->d_ctp;
    w.cno = c->d_cno;
    w.X = c->d_X;
    w.max_chunk = c->max_chunk;
    return w;
}

hwr_status route_device(hwr_ctx *c, const DevBatch &b, const Workspace &w) {
    hwr_status st = sync_state(c);
    if (st != HWR_OK) return st;
    if (c->res_launched && !c->res_stopping) {
        // a resident single-query workgroup would hold one compute unit that
        // the batch kernels' last workgroups wait for: ask it to leave
        __atomic_store_n(&c->h_sin->quit, 1u, __ATOMIC_RELEASE);
        c->res_stopping = true;
    }
    const int M = c->M, N = c->N, D = c->D;
    const size_t esz = c->bf16 ? 2 : 4;
    for (int off = 0; off < b.n; off += w.max_chunk) {
        const int cn = std::min(w.max_chunk, b.n - off);
        const int ldq = pair_stride(cn);       // pair-major row stride of this chunk
        QueryArgs qa;
        qa.nq = cn;
        qa.input_len = b.len + off;
        qa.nout = c->NH == 3 ? nullptr : b.nout + off;   // three heads predict N_out
        qa.slo = b.slo ? b.slo + off : nullptr;
        qa.default_slo = c->default_slo;
        OutArgs oa = b.out;
        const size_t oo = static_cast<size_t>(off) * c->nw;   // outputs are [n][nw]
        oa.choice += oo;
        if (oa.feasible) oa.feasible += oo;
        if (oa.utility) oa.utility += oo;
        if (oa.e2e) oa.e2e += oo;
        if (oa.ttft) oa.ttft += oo;
        if (oa.tpot) oa.tpot += oo;
        if (oa.nout) oa.nout += oo;
        float *qmat = b.cand_quality ? b.cand_quality + static_cast<size_t>(off) * M : w.qmat;
        float *ctt = b.cand_ttft ? b.cand_ttft + static_cast<size_t>(off) * N : nullptr;
        float *ctp = b.cand_tpot ? b.cand_tpot + static_cast<size_t>(off) * N : nullptr;
        float *cno = (c->NH == 3 && b.cand_nout) ? b.cand_nout + static_cast<size_t>(off) * N : nullptr;

        QualityArgs qu;
        qu.nq = cn;
        qu.D = D;
        qu.M = M;
        qu.emb = static_cast<const char *>(b.emb) + static_cast<size_t>(off) * D * esz;
        qu.wq_pk = c->d_wq_pk;
        qu.wq = c->d_wq;
        qu.bq = c->d_bq;
        qu.qmat = qmat;
        // fp32: the predictor reads no quality (the epilogue decides), so a
        // chunk small enough for both to share the device runs the quality
        // rows inside the predictor launch, in workgroups of their own.
        const bool quality_inside =
            !c->bf16 && mlp_f32_blocks(static_cast<long>(cn) * N) + (cn + 3) / 4 <= c->cus;
        if (!quality_inside) {
            HWR_HIP(c, timed(c, HWR_K_QUALITY, [&] {
                return c->bf16 ? launch_quality_bf16(qu, c->cus, c->stream) : launch_quality_f32(qu, c->stream);
            }));
        }

        if (c->bf16) {
            MlpArgs ma{};
            ma.N = N;
            ma.M = M;
            ma.len_slot = c->len_slot;
            ma.rule = c->rule;
            ma.w = c->w[0];
            ma.b3_0 = c->b3[0];
            ma.b3_1 = c->b3[1];
            ma.b3_2 = c->b3[2];
            ma.nheads = c->NH;
            ma.q = qa;
            ma.dep_bf16 = c->d_dep_bf16;
            ma.dep_model = c->d_dep_model;
            ma.qmat = qmat;
            ma.w1_pk = c->d_w1_pk;
            ma.w2_pk = c->d_w2_pk;
            ma.b1_pk = c->d_b1_pk;
            ma.b2_pk = c->d_b2_pk;
            ma.fold_b1 = c->fold_b1;
            ma.w3_frag = c->d_w3_frag;
            ma.out = oa;
            ma.nsplit = 1;
            ma.ldq = ldq;
            // one wave per SIMD with four column tiles pays where every
            // compute unit gets a workgroup; smaller batches take the two-tile
            // form (two waves per SIMD), which starts and drains faster
            ma.four_tiles = (cn + kQPerBlock - 1) / kQPerBlock >= c->cus;
            if (c->pipeline == HWR_PIPE_FUSED && c->nw == 1) {
                // per-candidate outputs, if the caller asked for them, go
                // straight to its [query][pair] buffers
                ma.cand_ttft = ctt;
                ma.cand_tpot = ctp;
                ma.cand_nout = cno;
                ma.cand_pm = 0;
                const int blocks = (cn + kQPerBlock - 1) / kQPerBlock;
                int nsplit = 1;
                if (blocks < c->cus) nsplit = std::min(N, (c->cus + blocks - 1) / blocks);
                while (nsplit > 1 && static_cast<size_t>(nsplit) * cn > w.part_cap) --nsplit;
                ma.nsplit = nsplit;
                ma.part_key = w.pkey;
                ma.part_val = w.pval;
                HWR_HIP(c, timed(c, HWR_K_FUSED, [&] { return launch_mlp_bf16(c->H, false, ma, c->stream); }));
                if (nsplit > 1) {
                    MergeArgs mg{cn, nsplit, w.pkey, w.pval, oa};
                    HWR_HIP(c, timed(c, HWR_K_MERGE, [&] { return launch_merge(mg, c->stream); }));
                }
                continue;
            }
            if (c->pipeline == HWR_PIPE_FUSED) {
                // several cost weights: the fused kernel writes every
                // candidate's predictions (pair-major, into the work space)
                // and no decision; the epilogue below takes one decision per
                // weight
                ma.cand_ttft = w.ctt;
                ma.cand_tpot = w.ctp;
                ma.cand_nout = c->NH == 3 ? w.cno : nullptr;
                ma.cand_pm = 1;
                ma.out = OutArgs{};
                ma.nsplit = 1;
                HWR_HIP(c, timed(c, HWR_K_FUSED, [&] { return launch_mlp_bf16(c->H, false, ma, c->stream); }));
            } else {
                GatherArgs ga{N, c->len_slot, qa, c->d_dep_bf16, w.X, ldq};
                HWR_HIP(c, timed(c, HWR_K_GATHER, [&] { return launch_gather(ga, c->stream); }));
                ma.X = w.X;
                ma.cand_ttft = w.ctt;
                ma.cand_tpot = w.ctp;
                ma.cand_nout = w.cno;
                ma.cand_pm = 1;
                HWR_HIP(c, timed(c, HWR_K_MLP, [&] { return launch_mlp_bf16(c->H, true, ma, c->stream); }));
            }
        } else {
            MlpF32Args fa = f32_args(c, qa);
            fa.ldq = ldq;
            fa.cand_ttft = w.ctt;
            fa.cand_tpot = w.ctp;
            fa.cand_nout = w.cno;
            if (quality_inside) {
                fa.with_quality = 1;
                fa.quality = qu;
            }
            HWR_HIP(c, timed(c, HWR_K_MLP, [&] { return launch_mlp_f32(c->H, fa, c->stream); }));
        }
        EpilogueArgs ea{};
        ea.N = N;
        ea.M = M;
        ea.ldq = ldq;
        ea.rule = c->rule;
        ea.nw = c->nw;
        for (int k = 0; k < c->nw; ++k) ea.w[k] = c->w[k];
        ea.q = qa;
        ea.dep_model = c->d_dep_model;
        ea.qmat = qmat;
        // the predictions are pair-major in the work space; the caller's
        // per-candidate buffers ([query][pair]) are written by the epilogue
        ea.cand_ttft = w.ctt;
        ea.cand_tpot = w.ctp;
        ea.cand_nout = c->NH == 3 ? w.cno : nullptr;
        ea.dbg_ttft = ctt;
        ea.dbg_tpot = ctp;
        ea.dbg_nout = c->NH == 3 ? cno : nullptr;
        ea.out = oa;
        HWR_HIP(c, timed(c, HWR_K_EPILOGUE, [&] { return launch_epilogue(ea, c->stream); }));
    }
    return HWR_OK;
}

hwr_status ensure_host_staging(hwr_ctx *c, size_t rows) {
    if (!c->cstream) {
        HWR_HIP(c, hipStreamCreateWithFlags(&c->cstream, hipStreamNonBlocking));
        for (auto &h : c->hin) {
            HWR_HIP(c, hipEventCreateWithFlags(&h.copied, hipEventDisableTiming));
            HWR_HIP(c, hipEventCreateWithFlags(&h.read, hipEventDisableTiming));
        }
    }
    if (rows <= c->hs_cap) return HWR_OK;
    HWR_HIP(c, hipStreamSynchronize(c->stream));
    HWR_HIP(c, hipStreamSynchronize(c->cstream));
    void *ptrs[] = {c->hin[0].emb, c->hin[0].len, c->hin[0].nout, c->hin[0].slo,
                    c->hin[1].emb, c->hin[1].len, c->hin[1].nout, c->hin[1].slo,
                    c->d_hchoice, c->d_hval, c->d_hcand, c->d_hqual, c->d_hfeas};
    for (void *p : ptrs)
        if (p) (void)hipFree(p);          // idle after the synchronisations above
    for (auto &h : c->hin) {
        h.emb = nullptr;
        h.len = h.nout = nullptr;
        h.slo = nullptr;
        h.used = false;
    }
    c->d_hchoice = nullptr;
    c->d_hval = c->d_hcand = c->d_hqual = nullptr;
    c->d_hfeas = nullptr;
    c->hs_cap = 0;
    const size_t esz = c->bf16 ? 2 : 4;
    for (auto &h : c->hin) {
        HWR_HIP(c, hipMalloc(&h.emb, rows * c->D * esz));
        HWR_HIP(c, dev_alloc(&h.len, rows));
        HWR_HIP(c, dev_alloc(&h.nout, rows));
        HWR_HIP(c, dev_alloc(&h.slo, rows));
    }
    HWR_HIP(c, dev_alloc(&c->d_hchoice, rows * c->nw));
    HWR_HIP(c, dev_alloc(&c->d_hval, rows * c->nw * 5));
    HWR_HIP(c, dev_alloc(&c->d_hcand, rows * c->N * 3));
    HWR_HIP(c, dev_alloc(&c->d_hqual, rows * c->M));
    HWR_HIP(c, dev_alloc(&c->d_hfeas, rows * c->nw));
    c->hs_cap = rows;
    return HWR_OK;
}

// Host-memory batches, chunk by chunk.  Chunk i's inputs go up on the upload
// stream into input set i % 2, once the kernels that read that set for chunk
// i - 2 have finished; the context's stream waits for the upload, runs the
// chunk and brings its outputs down.  The next chunk's upload is issued
// before this chunk's download, so with pageable caller memory (whose copies
// the host stages itself) the host stages chunk i + 1 while the device
// computes chunk i.  Returns when every output is in host memory, or, on an
// error, once both streams have drained.
hwr_status route_host_chunks(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r);

// The pinned ring and the copy threads of pageable host batches, set up once.
// When pinned memory cannot be had, pageable batches keep the runtime's copy.
bool page_ring(hwr_ctx *c) {
    if (c->copier) return true;
    if (c->page_failed) return false;
    for (auto &sl : c->pslot) {
        if (hipHostMalloc(&sl.buf, kPageSlotBytes, hipHostMallocDefault) != hipSuccess ||
            hipEventCreateWithFlags(&sl.done, hipEventDisableTiming) != hipSuccess) {
            (void)hipGetLastError();
            for (auto &t : c->pslot) {
                if (t.buf) (void)hipHostFree(t.buf);
                if (t.done) (void)hipEventDestroy(t.done);
                t = hwr_ctx::PageSlot{};
            }
            c->page_failed = true;
            return false;
        }
    }
    const unsigned hw = std::thread::hardware_concurrency();
    try {
        c->copier = std::make_unique<CopyPool>(static_cast<int>(std::min(7u, std::max(1u, hw / 2))));
    } catch (const std::exception &) {
        // no copy threads: pageable batches take the direct copies
        for (auto &t : c->pslot) {
            (void)hipHostFree(t.buf);
            (void)hipEventDestroy(t.done);
            t = hwr_ctx::PageSlot{};
        }
        c->page_failed = true;
        return false;
    }
    return true;
}

// Upload of `bytes` from pageable host memory to device memory on `stream`,
// through the pinned ring: each slot is filled (caller and copy threads) once
// its previous upload has finished, then uploaded.
hwr_status upload_pageable(hwr_ctx *c, void *dst, const void *src, size_t bytes, hipStream_t stream) {
    for (size_t o = 0; o < bytes; o += kPageSlotBytes) {
        const size_t n = std::min(kPageSlotBytes, bytes - o);
        hwr_ctx::PageSlot &sl = c->pslot[c->pslot_next];
        c->pslot_next = (c->pslot_next + 1) % kPageSlots;
        if (sl.used) HWR_HIP(c, hipEventSynchronize(sl.done));
        c->copier->copy(sl.buf, static_cast<const char *>(src) + o, n);
        HWR_HIP(c, hipMemcpyAsync(static_cast<char *>(dst) + o, sl.buf, n, hipMemcpyHostToDevice, stream));
        HWR_HIP(c, hipEventRecord(sl.done, stream));
        sl.used = true;
    }
    return HWR_OK;
}

hwr_status route_host(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r) {
    const hwr_status st = route_host_chunks(c, q, r);
    if (st != HWR_OK) {
        // copies may still read the caller's buffers or write its results:
        // let both streams drain before the caller gets control back
        if (c->cstream) (void)hipStreamSynchronize(c->cstream);
        (void)hipStreamSynchronize(c->stream);
    }
    return st;
}

hwr_status route_host_chunks(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r) {
    const size_t rows = static_cast<size_t>(std::min(q->n, c->max_chunk));
    hwr_status st = ensure_host_staging(c, rows);
    if (st != HWR_OK) return st;
    const size_t esz = c->bf16 ? 2 : 4;
    const int N = c->N, M = c->M, D = c->D;
    hipStream_t s = c->stream, cs = c->cstream;
    const size_t emb_bytes = static_cast<size_t>(q->n) * D * esz;
    const HostMem em = host_mem(q->emb);
    if (em == HostMem::kDevice) return fail(c, HWR_ERR_INVALID_ARG, "HWR_MEM_HOST batch with a device pointer");
    const bool staged_copy = emb_bytes >= kPageMinBytes && em == HostMem::kPageable && page_ring(c);
    auto upload = [&](int off) -> hwr_status {
        const int cn = std::min(c->max_chunk, q->n - off);
        hwr_ctx::InStage &h = c->hin[(off / c->max_chunk) & 1];
        if (h.used) HWR_HIP(c, hipStreamWaitEvent(cs, h.read, 0));
        const char *e = static_cast<const char *>(q->emb) + static_cast<size_t>(off) * D * esz;
        const size_t eb = static_cast<size_t>(cn) * D * esz;
        if (staged_copy) {
            const hwr_status us = upload_pageable(c, h.emb, e, eb, cs);
            if (us != HWR_OK) return us;
        } else {
            HWR_HIP(c, hipMemcpyAsync(h.emb, e, eb, hipMemcpyHostToDevice, cs));
        }
        HWR_HIP(c, hipMemcpyAsync(h.len, q->input_len + off, cn * 4, hipMemcpyHostToDevice, cs));
        if (c->NH == 2)
            HWR_HIP(c, hipMemcpyAsync(h.nout, q->expected_out_len + off, cn * 4, hipMemcpyHostToDevice, cs));
        if (q->slo_s) HWR_HIP(c, hipMemcpyAsync(h.slo, q->slo_s + off, cn * 4, hipMemcpyHostToDevice, cs));
        HWR_HIP(c, hipEventRecord(h.copied, cs));
        return HWR_OK;
    };
    st = upload(0);
    if (st != HWR_OK) return st;
    for (int off = 0; off < q->n; off += c->max_chunk) {
        const int cn = std::min(c->max_chunk, q->n - off);
        hwr_ctx::InStage &h = c->hin[(off / c->max_chunk) & 1];
        HWR_HIP(c, hipStreamWaitEvent(s, h.copied, 0));
        DevBatch b{};
        b.n = cn;
        b.emb = h.emb;
        b.len = h.len;
        b.nout = h.nout;
        b.slo = q->slo_s ? h.slo : nullptr;
        float *v = c->d_hval;
        const size_t vr = rows * c->nw;              // one [rows][nw] block per output
        b.out = OutArgs{c->d_hchoice, c->d_hfeas, v, v + vr, v + 2 * vr, v + 3 * vr, v + 4 * vr};
        b.cand_ttft = r->cand_ttft ? c->d_hcand : nullptr;
        b.cand_tpot = r->cand_tpot ? c->d_hcand + rows * N : nullptr;
        b.cand_nout = r->cand_nout ? c->d_hcand + 2 * rows * N : nullptr;
        b.cand_quality = r->cand_quality ? c->d_hqual : nullptr;
        hwr_status rs = route_device(c, b, ctx_workspace(c));
        if (rs != HWR_OK) return rs;
        HWR_HIP(c, hipEventRecord(h.read, s));
        h.used = true;
        if (off + c->max_chunk < q->n) {
            st = upload(off + c->max_chunk);
            if (st != HWR_OK) return st;
        }
        auto d2h = [&](void *dst, const void *src, size_t bytes) {
            return hipMemcpyAsync(dst, src, bytes, hipMemcpyDeviceToHost, s);
        };
        const size_t oo = static_cast<size_t>(off) * c->nw, on = static_cast<size_t>(cn) * c->nw;
        HWR_HIP(c, d2h(r->choice + oo, c->d_hchoice, on * 4));
        if (r->feasible) HWR_HIP(c, d2h(r->feasible + oo, c->d_hfeas, on));
        if (r->utility) HWR_HIP(c, d2h(r->utility + oo, v, on * 4));
        if (r->e2e_s) HWR_HIP(c, d2h(r->e2e_s + oo, v + vr, on * 4));
        if (r->ttft_s) HWR_HIP(c, d2h(r->ttft_s + oo, v + 2 * vr, on * 4));
        if (r->tpot_s) HWR_HIP(c, d2h(r->tpot_s + oo, v + 3 * vr, on * 4));
        if (r->nout) HWR_HIP(c, d2h(r->nout + oo, v + 4 * vr, on * 4));
        if (r->cand_ttft) HWR_HIP(c, d2h(r->cand_ttft + static_cast<size_t>(off) * N, c->d_hcand, static_cast<size_t>(cn) * N * 4));
        if (r->cand_tpot) HWR_HIP(c, d2h(r->cand_tpot + static_cast<size_t>(off) * N, c->d_hcand + rows * N, static_cast<size_t>(cn) * N * 4));
        if (r->cand_nout && c->NH == 3)
            HWR_HIP(c, d2h(r->cand_nout + static_cast<size_t>(off) * N, c->d_hcand + 2 * rows * N, static_cast<size_t>(cn) * N * 4));
        if (r->cand_quality) HWR_HIP(c, d2h(r->cand_quality + static_cast<size_t>(off) * M, c->d_hqual, static_cast<size_t>(cn) * M * 4));
    }
    HWR_HIP(c, hipStreamSynchronize(s));
    return HWR_OK;
}

// ---------------------------------------------------------------- single query
SingleArgs single_args(const hwr_ctx *c) {
    SingleArgs a{};
    a.N = c->N;
    a.M = c->M;
    a.D = c->D;
    a.len_slot = c->len_slot;
    a.rule = c->rule;
    a.w = c->w[0];
    a.b3_0 = c->b3[0];
    a.b3_1 = c->b3[1];
    a.b3_2 = c->b3[2];
    a.nheads = c->NH;
    a.arch_width = c->A;
    a.gpu_width = c->Gw;
    a.in = c->d_sin;
    a.out = c->d_sout;
    a.state = c->d_cur;
    a.dep_model = c->d_dep_model;
    a.dep_gpu = c->d_dep_gpu;
    a.pair_arch = c->d_pair_arch;
    a.pair_params = c->d_pair_params;
    a.wqT = c->d_wqT;
    a.bq = c->d_bq;
    a.w1_pk = c->d_w1_pk;
    a.w2_pk = c->d_w2_pk;
    a.b1_pk = c->d_b1_pk;
    a.b2_pk = c->d_b2_pk;
    a.w3_pk = c->d_w3_pk;
    a.fold_b1 = c->fold_b1;
    a.last_seq = c->seq;
    a.max_polls = kResidentPolls;
    return a;
}

// Capture the single-query kernel into a graph once; replays read the query
// record and the pair features by address, so state updates need no re-capture.
hwr_status single_graph(hwr_ctx *c) {
    if (c->gexec || !(c->flags & HWR_FLAG_GRAPH)) return HWR_OK;
    const SingleArgs a = single_args(c);
    hipStream_t cs = nullptr;
    HWR_HIP(c, hipStreamCreateWithFlags(&cs, hipStreamNonBlocking));
    hipError_t e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
    if (e == hipSuccess) e = launch_single(c->H, false, a, cs);
    hipGraph_t g = nullptr;
    hipError_t e2 = hipStreamEndCapture(cs, &g);
    (void)hipStreamDestroy(cs);
    if (e != hipSuccess) {
        if (g) (void)hipGraphDestroy(g);
        return hip_fail(c, e, "single-query graph capture");
    }
    if (e2 != hipSuccess) return hip_fail(c, e2, "hipStreamEndCapture");
    c->graph = g;
    HWR_HIP(c, hipGraphInstantiate(&c->gexec, c->graph, nullptr, nullptr, 0));
    return HWR_OK;
}

void read_single_out(const hwr_ctx *c, hwr_route_result *r) {
    const SingleOut *o = c->h_sout;
    r->choice[0] = o->choice;
    if (r->feasible) r->feasible[0] = static_cast<uint8_t>(o->feasible);
    if (r->utility) r->utility[0] = o->utility;
    if (r->e2e_s) r->e2e_s[0] = o->e2e;
    if (r->ttft_s) r->ttft_s[0] = o->ttft;
    if (r->tpot_s) r->tpot_s[0] = o->tpot;
    if (r->nout) r->nout[0] = o->nout;
}

// Resident single-query path (HWR_FLAG_RESIDENT): the kernel stays on the
// device between calls and polls the request record.  It is (re)launched
// when it has never run or may have left after its idle polls; a kernel that
// left while a request was being written is detected and relaunched.
hwr_status route_resident(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r) {
    SingleIn *in = c->h_sin;
    const uint32_t prev = c->seq;
    const uint32_t seq = ++c->seq == 0 ? ++c->seq : c->seq;
    auto launch = [&]() -> hwr_status {
        SingleArgs a = single_args(c);
        a.last_seq = prev;            // the pending request, if already posted, is newer
        __atomic_store_n(&in->quit, 0u, __ATOMIC_RELAXED);
        HWR_HIP(c, launch_single(c->H, true, a, c->sstream));
        c->res_launched = true;
        return HWR_OK;
    };
    if (c->res_stopping) {            // leaves within one poll of the quit flag
        HWR_HIP(c, hipStreamSynchronize(c->sstream));
        c->res_stopping = false;
        hwr_status st = launch();
        if (st != HWR_OK) return st;
    }
    const auto now = std::chrono::steady_clock::now();
    if (!c->res_launched || now - c->res_last > kResidentCheck) {
        const hipError_t qe = hipStreamQuery(c->sstream);
        if (qe == hipSuccess) {
            hwr_status st = launch();
            if (st != HWR_OK) return st;
        } else if (qe != hipErrorNotReady) {
            return hip_fail(c, qe, "resident single-query kernel");
        }
    }
    in->input_len = q->input_len[0];
    in->nout = c->NH == 2 ? q->expected_out_len[0] : 0;
    in->slo = q->slo_s ? q->slo_s[0] : c->default_slo;
    std::memcpy(in + 1, q->emb, static_cast<size_t>(c->D) * 2);
    std::atomic_thread_fence(std::memory_order_release);
    __atomic_store_n(&in->seq, seq, __ATOMIC_RELEASE);
    volatile uint32_t *flag = &c->h_sout->seq;
    const auto t0 = std::chrono::steady_clock::now();
    uint64_t spins = 0;
    while (*flag != seq) {
        if ((++spins & 0xFFF) == 0) {
            const hipError_t qe = hipStreamQuery(c->sstream);
            if (qe != hipSuccess && qe != hipErrorNotReady) return hip_fail(c, qe, "resident single-query kernel");
            if (qe == hipSuccess && *flag != seq) {   // it left before seeing this request
                hwr_status st = launch();
                if (st != HWR_OK) return st;
            }
            if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(10))
                return fail(c, HWR_ERR_HIP, "resident single-query kernel did not answer within 10 s");
        }
    }
    std::atomic_thread_fence(std::memory_order_acquire);
    c->res_last = std::chrono::steady_clock::now();
    read_single_out(c, r);
    return HWR_OK;
}

hwr_status route_single(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r) {
    if (c->flags & HWR_FLAG_RESIDENT) return route_resident(c, q, r);
    hwr_status st = single_graph(c);
    if (st != HWR_OK) return st;
    SingleIn *in = c->h_sin;
    const uint32_t seq = ++c->seq == 0 ? ++c->seq : c->seq;
    in->input_len = q->input_len[0];
    in->nout = c->NH == 2 ? q->expected_out_len[0] : 0;
    in->slo = q->slo_s ? q->slo_s[0] : c->default_slo;
    std::memcpy(in + 1, q->emb, static_cast<size_t>(c->D) * 2);
    in->seq = seq;
    std::atomic_thread_fence(std::memory_order_release);
    if (c->gexec) {
        HWR_HIP(c, timed_bracket(c, c->sstream, HWR_K_SINGLE, [&] { return hipGraphLaunch(c->gexec, c->sstream); }));
    } else {
        const SingleArgs a = single_args(c);
        HWR_HIP(c, timed_on(c, c->sstream, HWR_K_SINGLE, [&] { return launch_single(c->H, false, a, c->sstream); }));
    }
    // wait for the decision record (written last by the kernel, system scope)
    volatile uint32_t *flag = &c->h_sout->seq;
    auto t0 = std::chrono::steady_clock::now();
    uint64_t spins = 0;
    while (*flag != seq) {
        if ((++spins & 0xFFFF) == 0) {
            hipError_t qe = hipStreamQuery(c->sstream);
            if (qe != hipSuccess && qe != hipErrorNotReady) return hip_fail(c, qe, "single-query launch");
            if (qe == hipSuccess && *flag != seq)
                return fail(c, HWR_ERR_HIP, "single-query kernel finished without writing its result");
            if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(10))
                return fail(c, HWR_ERR_HIP, "single-query launch did not complete within 10 s");
        }
    }
    std::atomic_thread_fence(std::memory_order_acquire);
    read_single_out(c, r);
    return HWR_OK;
}

// Arguments common to both route entry points.  HWR_OK with n == 0 means
// there is nothing to do.
hwr_status check_route_args(hwr_ctx *c, const hwr_query_batch *q, const hwr_route_result *r) {
    if (!c) return fail(nullptr, HWR_ERR_INVALID_ARG, "ctx is NULL");
    if (!q || !r) return fail(c, HWR_ERR_INVALID_ARG, "batch or result is NULL");
    if (q->n < 0) return fail(c, HWR_ERR_INVALID_ARG, "n < 0");
    if (q->mem != HWR_MEM_DEVICE && q->mem != HWR_MEM_HOST) return fail(c, HWR_ERR_INVALID_ARG, "unknown mem");
    if (q->n == 0) return HWR_OK;
    if (!q->emb || !q->input_len || !r->choice || (c->NH == 2 && !q->expected_out_len))
        return fail(c, HWR_ERR_INVALID_ARG, "emb, input_len, choice and (two heads) expected_out_len are required");
    if (!c->has_state) return fail(c, HWR_ERR_STATE, "no hardware state yet: call hwr_update_hw_state first");
    return HWR_OK;
}

// Work space carved out of this device's static scratch: the split partials
// (fused, one weight) first, then per chunk row the quality row, the
// per-candidate predictions (staged, fp32 and several-weight routes) and the
// staged features, each block 256-byte aligned.  Chunks hold as many queries
// as fit, at most max_chunk; 0 rows: one query does not fit.
Workspace scratch_workspace(const hwr_ctx *c) {
    Workspace w;
    w.timing = false;
    const size_t M = c->M, N = c->N;
    const bool fused1 = c->bf16 && c->pipeline == HWR_PIPE_FUSED && c->nw == 1;
    const bool per_cand = !c->bf16 || c->pipeline == HWR_PIPE_STAGED || c->nw > 1;
    const bool staged = c->bf16 && c->pipeline == HWR_PIPE_STAGED;
    auto up = [](size_t x) { return (x + 255) & ~size_t(255); };
    const size_t part_cap = fused1 ? static_cast<size_t>(2 * c->cus) * kQPerBlock : 0;
    const size_t fixed = up(part_cap * sizeof(uint64_t)) + up(part_cap * kPartVals * sizeof(float));
    const size_t row = M * 4 + (per_cand ? N * 4 * (c->NH == 3 ? 3 : 2) : 0) + (staged ? N * kFeatPad * 2 : 0);
    // alignment of the per-row blocks, and the pair-major rows padded to
    // pair_stride(rows) (at most kPairAlign - 1 more rows)
    const size_t slack = 5 * 256 + (kPairAlign - 1) * row;
    if (fixed + slack >= kScratchBytes) return w;
    const size_t rows = std::min<size_t>((kScratchBytes - fixed - slack) / row, static_cast<size_t>(c->max_chunk));
    if (rows < 1) return w;
    const size_t ldq = static_cast<size_t>(pair_stride(static_cast<int>(rows)));
    unsigned char *base = static_cast<unsigned char *>(c->scratch);
    size_t off = 0;
    auto take = [&](size_t bytes) {
        unsigned char *p = base + off;
        off += up(bytes);
        return p;
    };
    if (fused1) {
        w.pkey = reinterpret_cast<uint64_t *>(take(part_cap * sizeof(uint64_t)));
        w.pval = reinterpret_cast<float *>(take(part_cap * kPartVals * sizeof(float)));
        w.part_cap = part_cap;
    }
    w.qmat = reinterpret_cast<float *>(take(rows * M * 4));
    if (per_cand) {
        w.ctt = reinterpret_cast<float *>(take(ldq * N * 4));
        w.ctp = reinterpret_cast<float *>(take(ldq * N * 4));
        if (c->NH == 3) w.cno = reinterpret_cast<float *>(take(ldq * N * 4));
    }
    if (staged) w.X = reinterpret_cast<uint16_t *>(take(ldq * N * kFeatPad * 2));
    w.max_chunk = static_cast<int>(rows);
    return off <= kScratchBytes ? w : Workspace{};
}

// Bodies of the exported functions below, which run them through
// c_boundary (no exception reaches the caller).
hwr_status init_entry(const hwr_config *cfg, hwr_ctx **out) {
    if (!out) return fail(nullptr, HWR_ERR_INVALID_ARG, "out is NULL");
    *out = nullptr;
    g_init_error.clear();
    return init_impl(cfg, out);
}

hwr_status update_hw_state(hwr_ctx *c, const hwr_hw_state *state, int32_t n) {
    if (!c) return fail(nullptr, HWR_ERR_INVALID_ARG, "ctx is NULL");
    if (!state) return fail(c, HWR_ERR_INVALID_ARG, "state is NULL");
    if (n != c->N) return fail(c, HWR_ERR_INVALID_ARG, "state count must equal n_deployments");
    for (int d = 0; d < n; ++d) {
        const hwr_hw_state &s = state[d];
        if (s.running_q < 0 || s.waiting_q < 0) return fail(c, HWR_ERR_INVALID_ARG, "queue length < 0");
        if (!finite(s.kv_util) || s.kv_util < 0.0f || s.kv_util > 1.0f)
            return fail(c, HWR_ERR_INVALID_ARG, "kv_util outside [0, 1]");
        if (!finite(s.gpu_util) || s.gpu_util < 0.0f || s.gpu_util > 1.0f)
            return fail(c, HWR_ERR_INVALID_ARG, "gpu_util outside [0, 1]");
        if (!finite(s.ttft_avg_s) || s.ttft_avg_s <= 0.0f || !finite(s.tpot_avg_s) || s.tpot_avg_s <= 0.0f)
            return fail(c, HWR_ERR_INVALID_ARG, "ttft_avg_s / tpot_avg_s must be finite and > 0");
    }
    HWR_HIP(c, hipSetDevice(c->dev));
    // The snapshot goes to the next slot of a pinned ring (turned into device
    // pair rows lazily, before the next batch) and to the pinned current copy
    // the single-query kernel reads.  A slot still awaited by an enqueued
    // state kernel is waited for before it is overwritten.
    const int slot = c->ring_next;
    if (c->ring_used[slot]) {
        HWR_HIP(c, hipEventSynchronize(c->ring_ev[slot]));
        c->ring_used[slot] = false;
    }
    std::memcpy(c->h_ring + static_cast<size_t>(slot) * c->N, state, sizeof(hwr_hw_state) * n);
    std::memcpy(c->h_cur, state, sizeof(hwr_hw_state) * n);
    c->state_slot = slot;
    c->state_dirty = true;
    c->ring_next = (slot + 1) % kStateSlots;
    c->has_state = true;
    return HWR_OK;
}

hwr_status route_batch(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r) {
    hwr_status st = check_route_args(c, q, r);
    if (st != HWR_OK || q->n == 0) return st;
    HWR_HIP(c, hipSetDevice(c->dev));
    if (q->mem == HWR_MEM_DEVICE) {
        DevBatch b{};
        b.n = q->n;
        b.emb = q->emb;
        b.len = q->input_len;
        b.nout = q->expected_out_len;
        b.slo = q->slo_s;
        b.out = OutArgs{r->choice, r->feasible, r->utility, r->e2e_s, r->ttft_s, r->tpot_s, r->nout};
        b.cand_ttft = r->cand_ttft;
        b.cand_tpot = r->cand_tpot;
        b.cand_nout = r->cand_nout;
        b.cand_quality = r->cand_quality;
        return route_device(c, b, ctx_workspace(c));
    }
    for (int i = 0; i < q->n; ++i) {
        if (q->input_len[i] < 1) return fail(c, HWR_ERR_INVALID_ARG, "input_len < 1");
        if (c->NH == 2 && q->expected_out_len[i] < 0) return fail(c, HWR_ERR_INVALID_ARG, "expected_out_len < 0");
        if (q->slo_s && (!finite(q->slo_s[i]) || q->slo_s[i] <= 0.0f))
            return fail(c, HWR_ERR_INVALID_ARG, "slo_s must be finite and > 0");
    }
    if (q->n == 1 && c->bf16 && c->nw == 1 && !r->cand_ttft && !r->cand_tpot && !r->cand_nout &&
        !r->cand_quality)
        return route_single(c, q, r);
    return route_host(c, q, r);
}

hwr_status route_batch_static(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r) {
    hwr_status st = check_route_args(c, q, r);
    if (st != HWR_OK || q->n == 0) return st;
    if (q->mem != HWR_MEM_DEVICE)
        return fail(c, HWR_ERR_INVALID_ARG, "hwr_route_batch_static routes device-memory batches only "
                                            "(host batches stage through buffers allocated on first use)");
    const Workspace w = scratch_workspace(c);
    if (w.max_chunk < 1)
        return fail(c, HWR_ERR_UNSUPPORTED, "one query of this context needs more work space than the " +
                                                std::to_string(kScratchBytes >> 20) + " MiB static scratch holds");
    HWR_HIP(c, hipSetDevice(c->dev));
    DevBatch b{};
    b.n = q->n;
    b.emb = q->emb;
    b.len = q->input_len;
    b.nout = q->expected_out_len;
    b.slo = q->slo_s;
    b.out = OutArgs{r->choice, r->feasible, r->utility, r->e2e_s, r->ttft_s, r->tpot_s, r->nout};
    b.cand_ttft = r->cand_ttft;
    b.cand_tpot = r->cand_tpot;
    b.cand_nout = r->cand_nout;
    b.cand_quality = r->cand_quality;
    c->no_timing = true;              // event timing could create events
    st = route_device(c, b, w);
    c->no_timing = false;
    return st;
}

hwr_status profile_enable(hwr_ctx *c, int32_t enable) {
    if (!c) return fail(nullptr, HWR_ERR_INVALID_ARG, "ctx is NULL");
    if (enable < 0) return fail(c, HWR_ERR_INVALID_ARG, "enable must be >= 0");
    c->prof = enable != 0;
    c->prof_every = enable > 1 ? enable : 1;
    for (int k = 0; k < HWR_K_COUNT; ++k) c->prof_seen[k] = 0;
    return HWR_OK;
}

hwr_status profile_read(hwr_ctx *c, hwr_kernel_times *out, int32_t reset) {
    if (!c || !out) return fail(c, HWR_ERR_INVALID_ARG, "ctx or out is NULL");
    hwr_status st = drain_timing(c);
    if (st != HWR_OK) return st;
    for (int k = 0; k < HWR_K_COUNT; ++k) {
        out->ms[k] = c->acc_ms[k];
        out->launches[k] = c->acc_n[k];
    }
    if (reset) {
        for (int k = 0; k < HWR_K_COUNT; ++k) {
            c->acc_ms[k] = 0.0;
            c->acc_n[k] = 0;
        }
    }
    return HWR_OK;
}
}  // namespace

// ==================================================================== C ABI
extern "C" {

hwr_status hwr_init(const hwr_config *cfg, hwr_ctx **out) {
    return c_boundary([&] { return init_entry(cfg, out); },
                      [](const char *m) { fail(nullptr, HWR_ERR_OOM, m); });
}

hwr_status hwr_update_hw_state(hwr_ctx *c, const hwr_hw_state *state, int32_t n) {
    return c_boundary([&] { return update_hw_state(c, state, n); },
                      [&](const char *m) { fail(c, HWR_ERR_OOM, m); });
}

hwr_status hwr_route_batch(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r) {
    return c_boundary([&] { return route_batch(c, q, r); },
                      [&](const char *m) { fail(c, HWR_ERR_OOM, m); });
}

hwr_status hwr_route_batch_static(hwr_ctx *c, const hwr_query_batch *q, hwr_route_result *r) {
    return c_boundary([&] { return route_batch_static(c, q, r); },
                      [&](const char *m) { fail(c, HWR_ERR_OOM, m); });
}

void hwr_free(hwr_ctx *c) { release(c); }

const char *hwr_last_error(const hwr_ctx *c) {
    if (c) return c->err.c_str();
    return g_init_error.c_str();
}

hwr_status hwr_profile_enable(hwr_ctx *c, int32_t enable) {
    return c_boundary([&] { return profile_enable(c, enable); },
                      [&](const char *m) { fail(c, HWR_ERR_OOM, m); });
}

hwr_status hwr_profile_read(hwr_ctx *c, hwr_kernel_times *out, int32_t reset) {
    return c_boundary([&] { return profile_read(c, out, reset); },
                      [&](const char *m) { fail(c, HWR_ERR_OOM, m); });
}

}  // extern "C"
