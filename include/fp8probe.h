/*
 * fp8probe.h -- measurement aid shipped beside libfp8lin.so (libfp8probe.so);
 * not part of the FP8 linear layer.
 *
 * fp8probe_mfma_loop -- launches `blocks` workgroups of 8 waves, each wave
 * issuing iters x 8 FP8 matrix instructions (v_mfma_f32_16x16x128_f8f6f4) on
 * register operands with no memory traffic, then writing one float per wave to
 * out (device, blocks * 8 floats, 4-byte aligned).  Asynchronous on stream.
 * Returns 0, 1 for a bad argument (nothing launched) or 3 for a launch error.
 * fp8probe_mfma_loop_flops -- the FLOPs of one such launch (2 * 16 * 16 * 128
 * per instruction).
 */
#ifndef FP8PROBE_H
#define FP8PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int64_t fp8probe_mfma_loop_flops(int32_t blocks, int32_t iters);
int32_t fp8probe_mfma_loop(int32_t blocks, int32_t iters, float *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FP8PROBE_H */
