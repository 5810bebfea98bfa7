/*
 * apb_probe.h -- measurement probe of the MI355X matrix cores (libapb_probe.so).
 *
 * Not part of the attention path: a ceiling for it.  The published dense
 * bf16 MFMA peak assumes the nominal 2.4 GHz shader clock; under a sustained
 * matrix-core load the clock settles lower, by an amount that depends on the
 * data being multiplied.  This probe runs nothing but back-to-back
 * v_mfma_f32_32x32x16_bf16 instructions on operands read from caller memory
 * (random bf16 values give a realistic switching load), so its rate is what a
 * bf16 kernel could reach on this chip if it did no other work.
 */
#ifndef APB_PROBE_H_
#define APB_PROBE_H_

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

/*
 * apb_probe_mfma_bf16 -- launch `n_workgroups` workgroups of 8 waves; every
 * wave keeps four independent 32x32 fp32 accumulators and issues
 * 4 * iters MFMAs of 32x32x16 bf16 (32768 flops each), rotating through
 * eight operand pairs it loaded from `operands`.
 *
 *   operands  device bf16 bits, at least 8192 elements (16 KiB), 16-byte
 *             aligned; read only.
 *   sink      device fp32 [n_workgroups * 512]; receives one sum of the
 *             accumulators per lane (keeps the work observable).
 *   iters     1 <= iters <= 1<<20, a multiple of 8.
 * Returns 0 on success, 1 for a bad argument (nothing launched), 2 for a HIP
 * launch error.  Asynchronous on `stream` (a hipStream_t, NULL = default).
 */
int32_t apb_probe_mfma_bf16(const uint16_t* operands, float* sink, int32_t n_workgroups,
                            int32_t iters, void* stream);

/* Flops one call performs: n_workgroups * 8 * 4 * iters * 32768 (host only). */
double apb_probe_mfma_flops(int32_t n_workgroups, int32_t iters);

#ifdef __cplusplus
}
#endif

#endif  // APB_PROBE_H_
