/*
 * hwr_probe.h -- measured ceilings of the device the library runs on.
 *
 * The routing kernels are quoted against two kinds of peak: the part's
 * published one (dense bf16 MFMA 2.5 PFLOP/s, HBM3E 8 TB/s) and the one a
 * plain kernel actually reaches on the same device, in the same thermal and
 * power state.  The first three entry points below measure the second kind;
 * the fourth measures a latency floor:
 *
 *  - hwr_probe_mfma_bf16: bf16 matrix products (32x32x16, fp32 accumulate) fed
 *    from registers only -- no memory traffic, eight independent accumulators
 *    per wave, operands that change from product to product (so the matrix
 *    cores draw the power real data makes them draw).  It bounds what any
 *    MFMA kernel can issue on this part at the clock the power limit allows.
 *  - hwr_probe_hbm_read: a streaming read of a caller buffer much larger than
 *    the last-level cache, non-temporal 16-byte loads by every lane, eight in
 *    flight per lane.  It bounds what a read-dominated kernel can fetch from
 *    HBM.
 *  - hwr_probe_hbm_write: the same for 16-byte stores of every lane into a
 *    caller buffer (its contents are overwritten).  It bounds a
 *    write-dominated kernel.
 *  - hwr_probe_launch_floor: the host-clock time of a launch of one wave
 *    that only answers through pinned host memory, plain or graph-launched:
 *    the floor under a single-query route.
 *
 * One more entry point exposes a device helper for checking rather than a
 * ceiling: hwr_probe_feature_log, the logarithm every feature uses.
 *
 * All are synchronous: they launch on a stream of their own on the given
 * device, wait, and return the median over the timed launches (the rates
 * timed on the device from each launch's own start to its own end).  The MFMA
 * and read probes allocate small device buffers of their own (the products'
 * results and clock readings, one word for the read) and free them before
 * returning.  Not part
 * of routing: nothing in hwr.h calls them.
 */
#ifndef HWR_PROBE_H
#define HWR_PROBE_H

#include <stdint.h>

#include "hwr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* Register-fed bf16 MFMA rate in TFLOP/s (2 * 32 * 32 * 16 flops per
 * product).  waves_per_simd (1..2): waves resident on each SIMD of every
 * compute unit; iters (>= 1): loop trips of eight products per wave and
 * launch; reps (1..64): timed launches after one untimed one.  *tflops is
 * the median over the timed launches.  clock_mhz (may be NULL): the median
 * over the timed launches of the shader clock the product loops ran at
 * (shader-cycle counter over the 100 MHz reference counter, summed over the
 * workgroups).  Errors: HWR_ERR_INVALID_ARG for a NULL tflops or an argument
 * out of range (no device touched), HWR_ERR_HIP, HWR_ERR_OOM. */
hwr_status hwr_probe_mfma_bf16(int32_t device, int32_t waves_per_simd, int32_t iters, int32_t reps,
                               double *tflops, double *clock_mhz);

/* Streaming read rate in GB/s (1e9 bytes per second) of `bytes` bytes at
 * `buf`, device memory of `device` owned by the caller and only read.  buf
 * 16-byte aligned, bytes a non-zero multiple of 16; waves_per_simd (1..8)
 * as above; reps (1..64) timed launches after one untimed one.  *gbps is the
 * median.  Errors: HWR_ERR_INVALID_ARG (NULL pointer, misaligned buffer,
 * size or count out of range; no device touched), HWR_ERR_HIP, HWR_ERR_OOM. */
hwr_status hwr_probe_hbm_read(int32_t device, const void *buf, uint64_t bytes, int32_t waves_per_simd,
                              int32_t reps, double *gbps);

/* Launch floor in microseconds, host clock: the host writes a request number
 * into a pinned host record, launches one wave (use_graph 0: a plain kernel
 * launch; 1: a graph holding that launch, captured once), and spins until the
 * wave has copied the number into a pinned answer record with a system-scope
 * store.  The single-query route does the same around its work, so this is
 * the part of its latency no kernel can remove.  calls (1..100000) timed calls
 * after 8 untimed ones; *p50_us and *p99_us are their median and 99th
 * percentile.  Errors: HWR_ERR_INVALID_ARG (NULL output, use_graph not 0 or 1,
 * calls out of range; no device touched), HWR_ERR_HIP (including no answer
 * within 10 s), HWR_ERR_OOM. */
hwr_status hwr_probe_launch_floor(int32_t device, int32_t use_graph, int32_t calls, double *p50_us,
                                  double *p99_us);

/* Streaming write rate in GB/s of `bytes` bytes at `buf`, device memory of
 * `device` owned by the caller, whose contents the probe overwrites.
 * Arguments and errors as hwr_probe_hbm_read. */
hwr_status hwr_probe_hbm_write(int32_t device, void *buf, uint64_t bytes, int32_t waves_per_simd,
                               int32_t reps, double *gbps);

/* The device's feature logarithm, for checking: y[i] = ln(x[i]) as every
 * Eq. 1 feature log of the library computes it (fp64; the features then
 * round ln(x) times their scale once to fp32, then to bf16).  x and y are
 * host arrays of n (1..2^26) doubles owned by the caller; every x[i] must be
 * positive, finite and normal, the arguments the features have (counts plus
 * one, parameter counts, latencies).  Synchronous: it allocates two device
 * buffers of n doubles, runs one kernel on the device's null stream and
 * frees them.  Errors: HWR_ERR_INVALID_ARG (NULL pointer, n out of range, an
 * x[i] outside the domain; no device touched), HWR_ERR_HIP, HWR_ERR_OOM. */
hwr_status hwr_probe_feature_log(int32_t device, const double *x, int64_t n, double *y);

#ifdef __cplusplus
}
#endif

#endif /* HWR_PROBE_H */
