/*
 * stlite_probe.h -- throughput probes of the MI355X matrix cores and of its
 * HBM read path, used by the benchmark as measured second denominators beside
 * the published bf16 and bandwidth peaks.  Not part of the compression method.
 *
 * Each probe keeps every SIMD busy with independent MFMA chains whose
 * operands come from caller-supplied data and rotate among eight A and
 * eight B fragments per lane, so that the matrix cores switch data as they
 * do in the compression kernels (a loop on constant operands draws less
 * power and would overstate the sustained rate).
 */
#ifndef STLITE_PROBE_H
#define STLITE_PROBE_H

#include <stddef.h>
#include <stdint.h>

#include "stlite.h"

#ifdef __cplusplus
extern "C" {
#endif

/* MFMA shape of a probe. */
typedef enum stlite_probe_shape {
  STLITE_PROBE_MFMA_16X16X32_BF16 = 0, /* v_mfma_f32_16x16x32_bf16: 16384 flops per instruction */
  STLITE_PROBE_MFMA_32X32X16_BF16 = 1, /* v_mfma_f32_32x32x16_bf16: 32768 flops per instruction */
  /* v_mfma_f32_32x32x16_bf16 with the window score's vector work: after every
   * MFMA, fma + exp2 + add on two finished fp32 results of the other of two
   * accumulators (one exponential per logit, the mix of the score passes);
   * 32768 flops per instruction */
  STLITE_PROBE_MFMA_32X32X16_BF16_EXP2 = 2,
  /* v_mfma_f32_16x16x32_bf16 with the same vector work per matrix-core cycle
   * (fma + exp2 + add on two results per two MFMAs); 16384 flops per
   * instruction */
  STLITE_PROBE_MFMA_16X16X32_BF16_EXP2 = 3
} stlite_probe_shape;

/*
 * Runs n_groups work-groups of 256 threads, each lane issuing 8 MFMAs per
 * iteration (16 for STLITE_PROBE_MFMA_16X16X32_BF16_EXP2) for `iters` iterations: 8 * iters * 4 * n_groups waves' worth of
 * instructions, i.e. flops = 8 * iters * (4 * n_groups) * flops_per_instruction
 * (16 * ... for the 16x16x32 exp2 probe).
 *   operands  device, bf16 bits, >= n_groups * 256 * 128 elements (read once)
 *   sink      device, fp32, >= n_groups * 256 elements (written: keeps the
 *             results live)
 * n_groups >= 1, iters >= 1; an unknown shape or a non-positive count is
 * STLITE_ERR_INVALID_ARG.  Enqueues on `stream` only.
 */
stlite_status stlite_probe_mfma(stlite_probe_shape shape, const uint16_t* operands, float* sink,
                                int32_t n_groups, int32_t iters, void* stream);

/*
 * Streaming read of `bytes` bytes at `src` (device), once, in 16-byte loads:
 * n_groups work-groups of 256 threads, each lane reading every
 * (n_groups * 256)-th 16-byte word, four loads in flight per lane; with
 * `nontemporal` != 0 the loads carry the non-temporal cache policy.
 *   src   device, 16-byte aligned, bytes a positive multiple of 16
 *   sink  device, fp32, >= n_groups * 256 elements (written: keeps the loads)
 * A NULL pointer, a misaligned or empty source, or n_groups < 1 is
 * STLITE_ERR_INVALID_ARG.  Enqueues on `stream` only.
 */
stlite_status stlite_probe_read(const void* src, size_t bytes, float* sink, int32_t n_groups,
                                int32_t nontemporal, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* STLITE_PROBE_H */
