// Ceiling probes of the device (gfx950): register-fed bf16 MFMA, a streaming
// HBM read and a streaming HBM write, and the floor of a launch answered
// through pinned host memory.  They give the achievable peaks next to the published
// ones; nothing on the routing path calls them.
#include <hip/hip_ext.h>
#include <hip/hip_runtime.h>

#include <algorithm>
#include <chrono>
#include <cstdint>
#include <vector>

#include "c_boundary.hpp"
#include "hwr_probe.h"

namespace {

typedef __bf16 pbf16x8 __attribute__((ext_vector_type(8)));
typedef float pf32x16 __attribute__((ext_vector_type(16)));

constexpr int kProbeThreads = 256;    // four waves: one per SIMD of a compute unit
constexpr int kChains = 8;            // independent accumulators per wave
constexpr int kFrags = 4;             // distinct A and B operands, cycled

// bf16 of a uniform value in [-1, 1) drawn from a 32-bit LCG state
__device__ inline __bf16 probe_value(uint32_t &s) {
    s = s * 1664525u + 1013904223u;
    const float f = __uint_as_float(0x3F800000u | (s >> 9)) * 2.0f - 3.0f;   // [1,2) -> [-1,1)
    return static_cast<__bf16>(f);
}

// clk (per workgroup): shader-clock cycles and 100 MHz reference ticks
// between the start and the end of its product loop, as seen by its first
// wave (counter reads; written with an ordinary vector store).
__global__ __launch_bounds__(kProbeThreads) void k_probe_mfma(int iters, float *out, uint64_t *clk) {
    uint32_t s = (blockIdx.x * kProbeThreads + threadIdx.x) * 0x9E3779B9u + 0x7F4A7C15u;
    pbf16x8 a[kFrags], b[kFrags];
#pragma unroll
    for (int f = 0; f < kFrags; ++f)
#pragma unroll
        for (int e = 0; e < 8; ++e) {
            a[f][e] = probe_value(s);
            b[f][e] = probe_value(s);
        }
    pf32x16 c[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) c[k] = pf32x16{};
    const uint64_t t0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
    for (int it = 0; it < iters; ++it) {
        // consecutive products take different operands
#pragma unroll
        for (int k = 0; k < kChains; ++k)
            c[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[k % kFrags], b[(k + k / kFrags) % kFrags], c[k], 0, 0, 0);
    }
    // two elements per accumulator: enough to keep every product, and the
    // reads stay few, so that two waves fit on a SIMD
    float sum = 0.0f;
#pragma unroll
    for (int k = 0; k < kChains; ++k) sum += c[k][0] + c[k][15];
    out[blockIdx.x * kProbeThreads + threadIdx.x] = sum;
    const uint64_t t1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
    if (threadIdx.x == 0) {
        clk[2 * blockIdx.x] = t1 - t0;
        clk[2 * blockIdx.x + 1] = r1 - r0;
    }
}

typedef uint32_t pu32x4 __attribute__((ext_vector_type(4)));
constexpr int kReadUnroll = 8;        // loads in flight per lane

// Every lane reads 16 bytes per load, kReadUnroll loads in flight,
// grid-strided, non-temporal (streamed past the caches: measured on this
// part, plain loads of the same pattern reach about 12% less); the single
// store happens only for one XOR value, which keeps the loads.
__global__ __launch_bounds__(kProbeThreads) void k_probe_read(const pu32x4 *__restrict__ p, uint64_t n,
                                                              uint32_t *out) {
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kProbeThreads;
    uint64_t i = static_cast<uint64_t>(blockIdx.x) * kProbeThreads + threadIdx.x;
    uint32_t acc = 0;
    for (; i + (kReadUnroll - 1) * stride < n; i += kReadUnroll * stride) {
        pu32x4 v[kReadUnroll];
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) v[u] = __builtin_nontemporal_load(p + i + u * stride);
#pragma unroll
        for (int u = 0; u < kReadUnroll; ++u) acc += v[u][0] ^ v[u][1] ^ v[u][2] ^ v[u][3];
    }
    for (; i < n; i += stride) {
        const pu32x4 v = __builtin_nontemporal_load(p + i);
        acc ^= v[0] ^ v[1] ^ v[2] ^ v[3];
    }
    if (acc == 0x2545F491u) out[0] = acc;
}

// Every lane writes 16 bytes per store, grid-strided, plain stores (on this
// part non-temporal and unrolled forms measured no faster).
__global__ __launch_bounds__(kProbeThreads) void k_probe_write(pu32x4 *__restrict__ p, uint64_t n) {
    const uint64_t stride = static_cast<uint64_t>(gridDim.x) * kProbeThreads;
    uint64_t i = static_cast<uint64_t>(blockIdx.x) * kProbeThreads + threadIdx.x;
    const pu32x4 v = {static_cast<uint32_t>(i), 1u, 2u, 3u};
    for (; i < n; i += stride) p[i] = v;
}

// Launch floor: one wave copies the request number from a pinned host
// record to the answer record (system scope, the answer written last), as the
// single-query kernel does around its work.
__global__ __launch_bounds__(64) void k_probe_echo(const uint32_t *in, uint32_t *out) {
    if (threadIdx.x == 0) {
        const uint32_t v = __hip_atomic_load(in, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
        __hip_atomic_store(out, v, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
    }
}

hwr_status status_of(hipError_t e) {
    if (e == hipSuccess) return HWR_OK;
    return e == hipErrorOutOfMemory ? HWR_ERR_OOM : HWR_ERR_HIP;
}

// Makes `device` current for the probe and restores the caller's device.
struct DeviceScope {
    int prev = -1;
    hipError_t err = hipSuccess;
    explicit DeviceScope(int device) {
        err = hipGetDevice(&prev);
        if (err == hipSuccess) err = hipSetDevice(device);
    }
    ~DeviceScope() {
        if (prev >= 0) (void)hipSetDevice(prev);
    }
};

// One untimed launch, then `reps` launches each timed on the device from its
// start to its end; the median duration in ms.
template <typename Launch>
hipError_t median_ms(Launch launch, int reps, float *ms) {
    hipStream_t s = nullptr;
    hipEvent_t ev[2 * 64] = {};
    float t[64];
    hipError_t e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    for (int i = 0; e == hipSuccess && i < 2 * reps; ++i) e = hipEventCreate(&ev[i]);
    if (e == hipSuccess) e = launch(s, nullptr, nullptr);
    for (int i = 0; e == hipSuccess && i < reps; ++i) e = launch(s, ev[2 * i], ev[2 * i + 1]);
    if (e == hipSuccess) e = hipStreamSynchronize(s);
    for (int i = 0; e == hipSuccess && i < reps; ++i) e = hipEventElapsedTime(&t[i], ev[2 * i], ev[2 * i + 1]);
    if (e == hipSuccess) {
        std::sort(t, t + reps);
        *ms = reps % 2 ? t[reps / 2] : 0.5f * (t[reps / 2 - 1] + t[reps / 2]);
    }
    for (int i = 0; i < 2 * reps; ++i)
        if (ev[i]) (void)hipEventDestroy(ev[i]);
    if (s) (void)hipStreamDestroy(s);
    return e;
}

hwr_status probe_mfma_bf16(int32_t device, int32_t waves_per_simd, int32_t iters, int32_t reps,
                           double *tflops, double *clock_mhz) {
    if (!tflops || device < 0 || waves_per_simd < 1 || waves_per_simd > 2 || iters < 1 || reps < 1 || reps > 64)
        return HWR_ERR_INVALID_ARG;
    DeviceScope scope(device);
    if (scope.err != hipSuccess) return status_of(scope.err);
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess) return status_of(e);
    const int blocks = prop.multiProcessorCount * waves_per_simd;
    float *out = nullptr;
    uint64_t *clk = nullptr;                   // [reps + 1 launches][blocks][2]
    const size_t nclk = static_cast<size_t>(reps + 1) * blocks * 2;
    e = hipMalloc(&out, static_cast<size_t>(blocks) * kProbeThreads * sizeof(float));
    if (e == hipSuccess) e = hipMalloc(&clk, nclk * sizeof(uint64_t));
    float ms = 0.0f;
    int launch = 0;
    if (e == hipSuccess)
        e = median_ms(
            [&](hipStream_t s, hipEvent_t a, hipEvent_t b) {
                uint64_t *lc = clk + static_cast<size_t>(launch++) * blocks * 2;
                hipExtLaunchKernelGGL(k_probe_mfma, dim3(blocks), dim3(kProbeThreads), 0, s, a, b, 0u, iters, out,
                                      lc);
                return hipGetLastError();
            },
            reps, &ms);
    std::vector<uint64_t> h;
    if (e == hipSuccess && clock_mhz) {
        h.resize(nclk);
        e = hipMemcpy(h.data(), clk, nclk * sizeof(uint64_t), hipMemcpyDeviceToHost);
    }
    (void)hipFree(out);
    (void)hipFree(clk);
    if (e != hipSuccess) return status_of(e);
    if (!(ms > 0.0f)) return HWR_ERR_HIP;
    if (clock_mhz) {
        // per timed launch: all workgroups' cycles over all their reference
        // ticks; the median over the launches
        std::vector<double> mhz;
        for (int l = 1; l <= reps; ++l) {
            double cyc = 0.0, ref = 0.0;
            for (int b = 0; b < blocks; ++b) {
                cyc += static_cast<double>(h[(static_cast<size_t>(l) * blocks + b) * 2]);
                ref += static_cast<double>(h[(static_cast<size_t>(l) * blocks + b) * 2 + 1]);
            }
            mhz.push_back(ref > 0.0 ? cyc / ref * 100.0 : 0.0);
        }
        std::sort(mhz.begin(), mhz.end());
        *clock_mhz = reps % 2 ? mhz[reps / 2] : 0.5 * (mhz[reps / 2 - 1] + mhz[reps / 2]);
    }
    const double flops = 2.0 * 32 * 32 * 16 * kChains * static_cast<double>(iters) * blocks * (kProbeThreads / 64);
    *tflops = flops / (ms * 1e-3) / 1e12;
    return HWR_OK;
}

hwr_status probe_hbm_read(int32_t device, const void *buf, uint64_t bytes, int32_t waves_per_simd,
                          int32_t reps, double *gbps) {
    if (!gbps || !buf || device < 0 || bytes == 0 || bytes % 16 != 0 ||
        reinterpret_cast<uintptr_t>(buf) % 16 != 0 || waves_per_simd < 1 || waves_per_simd > 8 || reps < 1 ||
        reps > 64)
        return HWR_ERR_INVALID_ARG;
    DeviceScope scope(device);
    if (scope.err != hipSuccess) return status_of(scope.err);
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess) return status_of(e);
    const int blocks = prop.multiProcessorCount * waves_per_simd;
    uint32_t *out = nullptr;
    e = hipMalloc(&out, sizeof(uint32_t));
    if (e != hipSuccess) return status_of(e);
    const pu32x4 *p = static_cast<const pu32x4 *>(buf);
    const uint64_t n = bytes / 16;
    float ms = 0.0f;
    e = median_ms(
        [&](hipStream_t s, hipEvent_t a, hipEvent_t b) {
            hipExtLaunchKernelGGL(k_probe_read, dim3(blocks), dim3(kProbeThreads), 0, s, a, b, 0u, p, n, out);
            return hipGetLastError();
        },
        reps, &ms);
    (void)hipFree(out);
    if (e != hipSuccess) return status_of(e);
    if (!(ms > 0.0f)) return HWR_ERR_HIP;
    *gbps = static_cast<double>(bytes) / (ms * 1e-3) / 1e9;
    return HWR_OK;
}

hwr_status probe_hbm_write(int32_t device, void *buf, uint64_t bytes, int32_t waves_per_simd,
                           int32_t reps, double *gbps) {
    if (!gbps || !buf || device < 0 || bytes == 0 || bytes % 16 != 0 ||
        reinterpret_cast<uintptr_t>(buf) % 16 != 0 || waves_per_simd < 1 || waves_per_simd > 8 || reps < 1 ||
        reps > 64)
        return HWR_ERR_INVALID_ARG;
    DeviceScope scope(device);
    if (scope.err != hipSuccess) return status_of(scope.err);
    hipDeviceProp_t prop;
    hipError_t e = hipGetDeviceProperties(&prop, device);
    if (e != hipSuccess) return status_of(e);
    const int blocks = prop.multiProcessorCount * waves_per_simd;
    pu32x4 *p = static_cast<pu32x4 *>(buf);
    const uint64_t n = bytes / 16;
    float ms = 0.0f;
    e = median_ms(
        [&](hipStream_t s, hipEvent_t a, hipEvent_t b) {
            hipExtLaunchKernelGGL(k_probe_write, dim3(blocks), dim3(kProbeThreads), 0, s, a, b, 0u, p, n);
            return hipGetLastError();
        },
        reps, &ms);
    if (e != hipSuccess) return status_of(e);
    if (!(ms > 0.0f)) return HWR_ERR_HIP;
    *gbps = static_cast<double>(bytes) / (ms * 1e-3) / 1e9;
    return HWR_OK;
}

hwr_status probe_launch_floor(int32_t device, int32_t use_graph, int32_t calls, double *p50_us,
                              double *p99_us) {
    if (!p50_us || !p99_us || device < 0 || (use_graph != 0 && use_graph != 1) || calls < 1 || calls > 100000)
        return HWR_ERR_INVALID_ARG;
    DeviceScope scope(device);
    if (scope.err != hipSuccess) return status_of(scope.err);
    uint32_t *h = nullptr, *d = nullptr;         // [0]: request, [16]: answer (separate lines)
    hipStream_t s = nullptr;
    hipGraph_t g = nullptr;
    hipGraphExec_t ge = nullptr;
    hipError_t e = hipHostMalloc(reinterpret_cast<void **>(&h), 256, hipHostMallocMapped | hipHostMallocCoherent);
    if (e == hipSuccess) {
        h[0] = 0;
        h[16] = 0;
        e = hipHostGetDevicePointer(reinterpret_cast<void **>(&d), h, 0);
    }
    if (e == hipSuccess) e = hipStreamCreateWithFlags(&s, hipStreamNonBlocking);
    auto launch = [&]() -> hipError_t {
        if (ge) return hipGraphLaunch(ge, s);
        hipLaunchKernelGGL(k_probe_echo, dim3(1), dim3(64), 0, s, d, d + 16);
        return hipGetLastError();
    };
    if (e == hipSuccess && use_graph) {
        hipStream_t cs = nullptr;
        e = hipStreamCreateWithFlags(&cs, hipStreamNonBlocking);
        if (e == hipSuccess) {
            e = hipStreamBeginCapture(cs, hipStreamCaptureModeThreadLocal);
            if (e == hipSuccess) {
                hipLaunchKernelGGL(k_probe_echo, dim3(1), dim3(64), 0, cs, d, d + 16);
                e = hipGetLastError();
                const hipError_t e2 = hipStreamEndCapture(cs, &g);
                if (e == hipSuccess) e = e2;
            }
            (void)hipStreamDestroy(cs);
        }
        if (e == hipSuccess) e = hipGraphInstantiate(&ge, g, nullptr, nullptr, 0);
    }
    // a few untimed calls, then `calls` timed ones: request number written,
    // launch, spin until the answer carries it
    std::vector<double> us;
    bool late = false;
    for (int i = 0; e == hipSuccess && i < calls + 8; ++i) {
        const uint32_t seq = static_cast<uint32_t>(i + 1);
        const auto t0 = std::chrono::steady_clock::now();
        __atomic_store_n(&h[0], seq, __ATOMIC_RELEASE);
        e = launch();
        uint64_t spins = 0;
        while (e == hipSuccess && __atomic_load_n(&h[16], __ATOMIC_ACQUIRE) != seq) {
            if ((++spins & 0xFFFF) == 0) {
                const hipError_t qe = hipStreamQuery(s);
                if (qe != hipSuccess && qe != hipErrorNotReady) e = qe;
                if (std::chrono::steady_clock::now() - t0 > std::chrono::seconds(10)) {
                    late = true;
                    break;
                }
            }
        }
        if (late) break;
        const auto t1 = std::chrono::steady_clock::now();
        if (i >= 8) us.push_back(std::chrono::duration<double, std::micro>(t1 - t0).count());
    }
    if (s) {
        const hipError_t se = hipStreamSynchronize(s);
        if (e == hipSuccess) e = se;
        (void)hipStreamDestroy(s);
    }
    if (ge) (void)hipGraphExecDestroy(ge);
    if (g) (void)hipGraphDestroy(g);
    if (h) (void)hipHostFree(h);
    if (e != hipSuccess) return status_of(e);
    if (late || us.empty()) return HWR_ERR_HIP;
    std::sort(us.begin(), us.end());
    *p50_us = us[us.size() / 2];
    *p99_us = us[std::min(us.size() - 1, static_cast<size_t>(0.99 * us.size()))];
    return HWR_OK;
}

}  // namespace

extern "C" hwr_status hwr_probe_mfma_bf16(int32_t device, int32_t waves_per_simd, int32_t iters, int32_t reps,
                                          double *tflops, double *clock_mhz) {
    return hwr::c_boundary([&] { return probe_mfma_bf16(device, waves_per_simd, iters, reps, tflops, clock_mhz); },
                           [](const char *) {});
}

extern "C" hwr_status hwr_probe_hbm_read(int32_t device, const void *buf, uint64_t bytes, int32_t waves_per_simd,
                                         int32_t reps, double *gbps) {
    return hwr::c_boundary([&] { return probe_hbm_read(device, buf, bytes, waves_per_simd, reps, gbps); },
                           [](const char *) {});
}

extern "C" hwr_status hwr_probe_hbm_write(int32_t device, void *buf, uint64_t bytes, int32_t waves_per_simd,
                                          int32_t reps, double *gbps) {
    return hwr::c_boundary([&] { return probe_hbm_write(device, buf, bytes, waves_per_simd, reps, gbps); },
                           [](const char *) {});
}

extern "C" hwr_status hwr_probe_launch_floor(int32_t device, int32_t use_graph, int32_t calls, double *p50_us,
                                             double *p99_us) {
    return hwr::c_boundary([&] { return probe_launch_floor(device, use_graph, calls, p50_us, p99_us); },
                           [](const char *) {});
}
