/*
 * fp8probe.h -- measurement aid shipped beside libfp8lin.so (libfp8probe.so);
 * not part of the FP8 linear layer.
 *
 * fp8probe_mfma_loop -- launches `blocks` workgroups of 8 waves, each wave
 * issuing iters x 8 FP8 matrix instructions (v_mfma_f32_16x16x128_f8f6f4) on
 * register operands with no memory traffic, then writing one float per wave to
 * out (device, blocks * 8 floats, 4-byte aligned).  vary != 0: consecutive
 * instructions take different pseudo-random operands (finite E4M3 codes), as
 * in a matmul; vary == 0: every instruction the same operands.  Asynchronous
 * on stream.
 * Returns 0, 1 for a bad argument (nothing launched) or 3 for a launch error.
 * fp8probe_mfma_loop_flops -- the FLOPs of one such launch (2 * 16 * 16 * 128
 * per instruction).
 *
 * fp8probe_stream -- the memory traffic of a cast with no arithmetic: reads n
 * bf16 elements of src (device, 16-byte aligned, n a multiple of 16) and
 * writes one byte per element to dst1 and, if dst2 is not NULL, one more to
 * dst2 (device, 16-byte aligned): 3 or 4 bytes per element, each workgroup a
 * contiguous range, 16-byte non-temporal loads and stores.  Returns as above.
 *
 * fp8probe_lds -- LDS traffic of the matmul's main loop in isolation: 256
 * workgroups of 8 waves, each wave iters x 8 ds_read_b128 of 1 KiB and/or
 * iters x 8 global_load_lds_dwordx4 copies of 1 KiB into its own 8 KiB of LDS
 * (mode 0: 8 waves read; 1: 8 waves copy; 2: 4 copy while 4 read; 3: 4 read).
 * src: device, 16-byte aligned, fp8probe_lds_src_bytes() readable bytes (each
 * workgroup copies from its own 1 MiB window); out: device, 256 uint32,
 * written only by a practically impossible data pattern.  Returns as above.
 */
#ifndef FP8PROBE_H
#define FP8PROBE_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

int64_t fp8probe_mfma_loop_flops(int32_t blocks, int32_t iters);
int32_t fp8probe_mfma_loop(int32_t blocks, int32_t iters, int32_t vary, float *out, void *stream);
int32_t fp8probe_stream(const void *src, int64_t n, void *dst1, void *dst2, void *stream);
int64_t fp8probe_lds_src_bytes(void);
int32_t fp8probe_lds(int32_t mode, int32_t iters, const void *src, uint32_t *out, void *stream);

#ifdef __cplusplus
}
#endif

#endif /* FP8PROBE_H */
