// Measurement aid, not part of the method: the sustained rate of the FP8
// matrix cores of gfx950 with no memory traffic at all.  Every wave issues
// v_mfma_f32_16x16x128_f8f6f4 on register operands in a loop (eight
// independent accumulators, so the instructions never wait for each other);
// the accumulators are summed into one word per wave at the end so that the
// loop is not removed.  bench.py --mfma-ceiling launches it and reports
// 2 * 16 * 16 * 128 FLOP per instruction over the launch time, the ceiling the
// matmul kernels are compared with under the chip's sustained clock.
// Operands: with `vary` the eight instructions of an iteration take four
// different pseudo-random A and B fragments (every byte a finite E4M3 code),
// so the multiplier inputs change from one instruction to the next as in a
// matmul; without it every instruction reads the same fragments.  The power a
// matrix core draws, and so the clock it sustains, depends on that.
#include <hip/hip_runtime.h>
#include <stdint.h>

#include "fp8probe.h"

namespace {

typedef int v8i __attribute__((ext_vector_type(8)));
typedef float v4f __attribute__((ext_vector_type(4)));

constexpr int kAcc = 8;

// xorshift32 step (a pseudo-random word per call)
__device__ __forceinline__ uint32_t next_word(uint32_t& s) {
    s ^= s << 13;
    s ^= s >> 17;
    s ^= s << 5;
    return s;
}

__global__ __launch_bounds__(512) void mfma_loop_kernel(int iters, uint32_t seed, int vary, float* __restrict__ out) {
    uint32_t st = seed ^ (threadIdx.x * 2654435761u) ^ (blockIdx.x * 40503u + 1u);
    // random finite E4M3 codes: clearing bit 0x08 of each byte's exponent
    // field keeps every byte below the NaN pattern S.1111.111
    v8i a[4], b[4];
#pragma unroll
    for (int f = 0; f < 4; ++f)
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            a[f][i] = (int)(next_word(st) & 0xF7F7F7F7u);
            b[f][i] = (int)(next_word(st) & 0xF7F7F7F7u);
        }
    if (!vary) {
#pragma unroll
        for (int f = 1; f < 4; ++f) {
            a[f] = a[0];
            b[f] = b[0];
        }
    }
    v4f acc[kAcc];
#pragma unroll
    for (int j = 0; j < kAcc; ++j) acc[j] = v4f{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < kAcc; ++j)
            acc[j] = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a[j & 3], b[(j >> 1) & 3], acc[j], 0, 0, 0,
                                                                      0, 0, 0);
    }
    float s = 0.f;
#pragma unroll
    for (int j = 0; j < kAcc; ++j) s += acc[j][0] + acc[j][1] + acc[j][2] + acc[j][3];
    if ((threadIdx.x & 63) == 0) out[blockIdx.x * (blockDim.x >> 6) + (threadIdx.x >> 6)] = s;
}

// Cast-shaped stream: each workgroup reads one contiguous range of bf16
// elements, sixteen per lane and step (two 16-byte non-temporal loads), with
// four such groups (eight loads) in flight per lane, and writes one byte per
// element (the high byte of each bf16: no conversion arithmetic) as one
// 16-byte non-temporal store per group to dst1 and, if given, to dst2.
constexpr int kStreamThreads = 256, kStreamG = 4;
typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ uint32_t high_bytes(uint32_t a, uint32_t b) {
    return ((a >> 8) & 0xFFu) | ((a >> 16) & 0xFF00u) | ((b << 8) & 0xFF0000u) | (b & 0xFF000000u);
}

__global__ __launch_bounds__(kStreamThreads) void stream_kernel(const u32x4* __restrict__ src, int64_t ng,
                                                                 u32x4* __restrict__ dst1, u32x4* __restrict__ dst2) {
    // ng groups of 16 elements = 2 source vectors and 1 destination vector each
    const int64_t chunk = ((ng + gridDim.x - 1) / gridDim.x + 255) & ~(int64_t)255;
    const int64_t b0 = min(ng, (int64_t)blockIdx.x * chunk), b1 = min(ng, b0 + chunk);
    for (int64_t i = b0 + threadIdx.x; i < b1; i += kStreamG * kStreamThreads) {
        u32x4 v[2 * kStreamG];
#pragma unroll
        for (int l = 0; l < kStreamG; ++l) {
            const int64_t j = min(i + l * kStreamThreads, b1 - 1);
            v[2 * l] = __builtin_nontemporal_load(src + 2 * j);
            v[2 * l + 1] = __builtin_nontemporal_load(src + 2 * j + 1);
        }
        __builtin_amdgcn_sched_barrier(0);
#pragma unroll
        for (int l = 0; l < kStreamG; ++l) {
            const int64_t j = i + l * kStreamThreads;
            if (j < b1) {
                const u32x4 a = v[2 * l], b = v[2 * l + 1];
                const u32x4 c = {high_bytes(a.x, a.y), high_bytes(a.z, a.w), high_bytes(b.x, b.y), high_bytes(b.z, b.w)};
                __builtin_nontemporal_store(c, dst1 + j);
                if (dst2) __builtin_nontemporal_store(u32x4{c.y, c.x, c.w, c.z}, dst2 + j);
            }
        }
    }
}

// LDS traffic of the matmul's main loop in isolation: one workgroup of 8
// waves per compute unit, each wave owning an 8 KiB region of LDS laid out as
// eight 1 KiB rows of 16-byte chunks.  Readers issue ds_read_b128 over their
// region (every lane a different chunk, every bank once per phase); copiers
// fill their region from global memory with global_load_lds_dwordx4 (1 KiB
// per instruction, up to 16 in flight per wave), reading a 1 MiB window of src
// per workgroup so that the data comes from L2.  mode 0: all 8 waves read;
// 1: all 8 copy; 2: waves 0-3 copy while 4-7 read; 3: waves 0-3 read, 4-7 idle.
constexpr int kLdsRegion = 8192, kLdsWindow = 1 << 20;

__device__ __forceinline__ uint32_t lds_addr(const void* p) {
    return (uint32_t)(uintptr_t)(__attribute__((address_space(3))) const void*)p;
}

__global__ __launch_bounds__(512) void lds_probe_kernel(int mode, int iters, const uint8_t* __restrict__ src,
                                                        uint32_t* __restrict__ out) {
    // 128 KiB (half unused) so that one workgroup fills a compute unit's LDS
    // and every compute unit runs exactly one
    __shared__ __attribute__((aligned(1024))) uint8_t smem[16 * kLdsRegion];
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    for (int i = threadIdx.x; i < 8 * kLdsRegion / 4; i += 512) ((uint32_t*)smem)[i] = (uint32_t)i;
    __syncthreads();
    const bool copy = mode == 1 || (mode == 2 && w < 4);
    const bool read = mode == 0 || (mode == 2 && w >= 4) || (mode == 3 && w < 4);
    const uint8_t* region = smem + w * kLdsRegion;
    const uint8_t* window = src + (size_t)(blockIdx.x % 64) * kLdsWindow;
    const uint32_t dst = __builtin_amdgcn_readfirstlane(lds_addr(region));
    u32x4 x = {0u, 0u, 0u, 0u};
    for (int it = 0; it < iters; ++it) {
        if (read) {
#pragma unroll
            for (int q = 0; q < 8; ++q) x ^= *(const u32x4*)(region + q * 1024 + lane * 16);
        }
        if (copy) {
#pragma unroll
            for (int q = 0; q < 8; ++q) {
                const uint32_t off = (uint32_t)((((it * 8 + q) & (kLdsWindow / 1024 - 1)) * 1024) + lane * 16);
                asm volatile("s_mov_b32 m0, %0\n\ts_nop 0\n\tglobal_load_lds_dwordx4 %1, %2"
                             :
                             : "s"(dst + q * 1024), "v"(off), "s"(window)
                             : "memory");
            }
            asm volatile("s_waitcnt vmcnt(8)" ::: "memory");
        }
        asm volatile("" ::: "memory");
    }
    asm volatile("s_waitcnt vmcnt(0)" ::: "memory");
    if (x.x == 0x9E3779B9u) out[blockIdx.x] = x.y;  // keeps the reads; practically never taken
}

}  // namespace

extern "C" {

int64_t fp8probe_lds_src_bytes(void) { return (int64_t)64 * kLdsWindow; }

int32_t fp8probe_lds(int32_t mode, int32_t iters, const void* src, uint32_t* out, void* stream) {
    if (mode < 0 || mode > 3 || iters < 1 || !src || !out || ((uintptr_t)src % 16) || ((uintptr_t)out % 4))
        return 1;
    hipLaunchKernelGGL(lds_probe_kernel, dim3(256), dim3(512), 0, (hipStream_t)stream, (int)mode, (int)iters,
                       (const uint8_t*)src, out);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

int32_t fp8probe_stream(const void* src, int64_t n, void* dst1, void* dst2, void* stream) {
    if (n < 16 || n % 16 || !src || !dst1 || ((uintptr_t)src % 16) || ((uintptr_t)dst1 % 16) ||
        (dst2 && ((uintptr_t)dst2 % 16)))
        return 1;
    hipLaunchKernelGGL(stream_kernel, dim3(2048), dim3(kStreamThreads), 0, (hipStream_t)stream, (const u32x4*)src,
                       n / 16, (u32x4*)dst1, (u32x4*)dst2);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

int64_t fp8probe_mfma_loop_flops(int32_t blocks, int32_t iters) {
    return (int64_t)blocks * 8 * iters * kAcc * 2 * 16 * 16 * 128;
}

int32_t fp8probe_mfma_loop(int32_t blocks, int32_t iters, int32_t vary, float* out, void* stream) {
    if (blocks < 1 || blocks > 65536 || iters < 1 || !out || ((uintptr_t)out % 4)) return 1;
    hipLaunchKernelGGL(mfma_loop_kernel, dim3(blocks), dim3(512), 0, (hipStream_t)stream, iters, 12345u,
                       vary ? 1 : 0, out);
    return hipGetLastError() == hipSuccess ? 0 : 3;
}

}  // extern "C"
