// Measurement aid, not part of the method: the sustained rate of the FP8
// matrix cores of gfx950 with no memory traffic at all.  Every wave issues
// v_mfma_f32_16x16x128_f8f6f4 on register operands in a loop (eight
// independent accumulators, so the instructions never wait for each other);
// the accumulators are summed into one word per wave at the end so that the
// loop is not removed.  bench.py --mfma-ceiling launches it and reports
// 2 * 16 * 16 * 128 FLOP per instruction over the launch time, the ceiling the
// matmul kernels are compared with under the chip's sustained clock.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp8probe.h"

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kAcc = 8;

__global__ __launch_bounds__(512) void mfma_loop_kernel(int iters, uint32_t seed, float* __restrict__ out) {
    // finite E4M3 codes of moderate size: bytes 0x30..0x3F (0.5 .. 0.94)
    const uint32_t t = (seed + threadIdx.x * 2654435761u + blockIdx.x * 40503u) | 0x30303030u;
    const uint32_t code = t & 0x3F3F3F3Fu;
    v8i a, b;
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        a[i] = (int)(code ^ (uint32_t)(i * 0x01010101u & 0x07070707u));
        b[i] = (int)(code ^ (uint32_t)((i + 3) * 0x01010101u & 0x07070707u));
    }
    v4f acc[kAcc];
#pragma unroll
    for (int j = 0; j < kAcc; ++j) acc[j] = v4f{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < kAcc; ++j)
            acc[j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, b, acc[j], 0, 0, 0, 0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < kAcc; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
    if ((threadIdx.x & 63) == 0) out[blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)] = s;
}

}  // namespace

extern "C" {

int64_t fp8probe_mfma_loop_flops(int32_t blocks, int32_t iters) {
    return (int64_t)blocks * 8 * iters * kAcc * 2 * 16 * 16 * 128;
}

int32_t fp8probe_mfma_loop(int32_t blocks, int32_t iters, float* out, void* stream) {
    if (blocks < 1 || blocks > 65536 || iters < 1 || !out || ((uintptr_t)out % 4)) return 1;
    hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(512), 0, (hipStream_t)stream, iters, 12345u, out);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

}  // extern "C"
