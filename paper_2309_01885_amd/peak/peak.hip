// Peak-check kernels for the roofline denominators: what this chip's matrix
// cores and HBM sustain outside the method's kernels.  Built into
// libqe_peak.so, apart from libqe.so: these are measurement probes, not part
// of the quantizer's C ABI.
//
//   qpk_mfma_bf16 / qpk_mfma_f16 / qpk_mfma_f32: register-only loops of the
//     matrix-core instruction the split products (v_mfma_f32_32x32x16_bf16,
//     v_mfma_f32_32x32x16_f16) and the fp32 products (v_mfma_f32_32x32x2f32)
//     use, four independent accumulators per wave, two waves per SIMD; the
//     caller times the launch.  Flops per launch: blocks * 4 waves * iters *
//     16 MFMAs * (2 * 32 * 32 * K), K = 16, 16 or 2.
//   qpk_copy: dst = src over n 16-byte elements, grid-stride or one contiguous
//     range per workgroup (HBM stream).
//   qpk_clock: per-wave shader-clock and constant-rate (100 MHz) counter
//     deltas across the bf16 loop, from which the engine clock under matrix
//     load follows.
//
// All return 0 on success, 1 on bad arguments, 5 on a HIP launch error.
#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;

// Operands are finite bf16 values in [2^-7, 2) from a per-thread LCG, so the
// accumulators stay finite; their sum is stored so that nothing is removed.
__device__ inline void seed_bf16(unsigned x, u32x4& ua, u32x4& ub)
{
    for (int i = 0; i < 4; ++i) {
        x = x * 1664525u + 1013904223u;
        ua[i] = (x & 0x3f7f3f7fu) | 0x3c003c00u;
        x = x * 1664525u + 1013904223u;
        ub[i] = (x & 0x3f7f3f7fu) | 0x3c003c00u;
    }
}

__device__ inline void bf16_loop(int iters, const u32x4& ua, const u32x4& ub, f32x16 (&acc)[4])
{
    const bf16x8 a = __builtin_bit_cast(bf16x8, ua), b = __builtin_bit_cast(bf16x8, ub);
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int k = 0; k < 4; ++k)
                acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, acc[k], 0, 0, 0);
    }
}

// fp16 operands in [2^-2, 1) (exponent field 13 or 14) from the same LCG.
__device__ inline void seed_f16(unsigned x, u32x4& ua, u32x4& ub)
{
    for (int i = 0; i < 4; ++i) {
        x = x * 1664525u + 1013904223u;
        ua[i] = (x & 0x07ff07ffu) | 0x34003400u;
        x = x * 1664525u + 1013904223u;
        ub[i] = (x & 0x07ff07ffu) | 0x34003400u;
    }
}

__device__ inline float acc_sum(const f32x16 (&acc)[4])
{
    float s = 0.f;
    for (int k = 0; k < 4; ++k)
        for (int v = 0; v < 16; ++v) s += acc[k][v];
    return s;
}

__global__ __launch_bounds__(kThreads, 2) void mfma_bf16_kernel(float* out, int iters)
{
    u32x4 ua, ub;
    seed_bf16(threadIdx.x * 2654435761u ^ blockIdx.x * 40503u ^ 7u, ua, ub);
    f32x16 acc[4] = {};
    bf16_loop(iters, ua, ub, acc);
    out[(size_t)blockIdx.x * kThreads + threadIdx.x] = acc_sum(acc);
}

__global__ __launch_bounds__(kThreads, 2) void mfma_f16_kernel(float* out, int iters)
{
    u32x4 ua, ub;
    seed_f16(threadIdx.x * 2654435761u ^ blockIdx.x * 40503u ^ 7u, ua, ub);
    const f16x8 a = __builtin_bit_cast(f16x8, ua), b = __builtin_bit_cast(f16x8, ub);
    f32x16 acc[4] = {};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int k = 0; k < 4; ++k)
                acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_f16(a, b, acc[k], 0, 0, 0);
    }
    out[(size_t)blockIdx.x * kThreads + threadIdx.x] = acc_sum(acc);
}

__global__ __launch_bounds__(kThreads, 2) void mfma_f32_kernel(float* out, int iters)
{
    float a = 1.f + (float)(threadIdx.x & 63) * 0x1p-10f;
    float b = 1.f - (float)(blockIdx.x & 63) * 0x1p-10f;
    f32x16 acc[4] = {};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int r = 0; r < 4; ++r)
#pragma unroll
            for (int k = 0; k < 4; ++k)
                acc[k] = __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, acc[k], 0, 0, 0);
    }
    out[(size_t)blockIdx.x * kThreads + threadIdx.x] = acc_sum(acc);
}

__global__ __launch_bounds__(kThreads, 2) void clock_kernel(float* out, uint64_t* clk, int iters)
{
    u32x4 ua, ub;
    seed_bf16(threadIdx.x * 2654435761u ^ blockIdx.x * 40503u ^ 7u, ua, ub);
    f32x16 acc[4] = {};
    const uint64_t c0 = __builtin_amdgcn_s_memtime(), r0 = __builtin_amdgcn_s_memrealtime();
    bf16_loop(iters, ua, ub, acc);
    const float s = acc_sum(acc);
    const uint64_t c1 = __builtin_amdgcn_s_memtime(), r1 = __builtin_amdgcn_s_memrealtime();
    out[(size_t)blockIdx.x * kThreads + threadIdx.x] = s;
    if ((threadIdx.x & 63) == 0) {
        const size_t w = (size_t)blockIdx.x * (kThreads / 64) + threadIdx.x / 64;
        clk[2 * w] = c1 - c0;        // vector stores of the per-wave deltas
        clk[2 * w + 1] = r1 - r0;
    }
}

// Grid-stride copy, one 16-byte element per thread per pass.
__global__ __launch_bounds__(kThreads) void copy_kernel(const f32x4* __restrict__ src,
                                                        f32x4* __restrict__ dst, size_t n)
{
    const size_t stride = (size_t)gridDim.x * kThreads;
    for (size_t i = (size_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) dst[i] = src[i];
}

// Each workgroup copies one contiguous range of `per` elements, four 16-byte
// loads in flight per thread.
__global__ __launch_bounds__(kThreads) void copy_chunk_kernel(const f32x4* __restrict__ src,
                                                              f32x4* __restrict__ dst, size_t n,
                                                              size_t per)
{
    const size_t b0 = (size_t)blockIdx.x * per;
    const size_t b1 = b0 + per < n ? b0 + per : n;
    for (size_t i = b0 + threadIdx.x; i < b1; i += 4 * kThreads) {
        f32x4 v[4];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (i + u * kThreads < b1) v[u] = src[i + u * kThreads];
#pragma unroll
        for (int u = 0; u < 4; ++u)
            if (i + u * kThreads < b1) dst[i + u * kThreads] = v[u];
    }
}

int launched() { return hipGetLastError() == hipSuccess ? 0 : 5; }

}  // namespace

extern "C" {

// out: blocks * 256 floats.
int qpk_mfma_bf16(float* out, int blocks, int iters, void* stream)
{
    if (!out || blocks <= 0 || iters <= 0) return 1;
    hipLaunchKernelGGL(mfma_bf16_kernel, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream,
                       out, iters);
    return launched();
}

int qpk_mfma_f16(float* out, int blocks, int iters, void* stream)
{
    if (!out || blocks <= 0 || iters <= 0) return 1;
    hipLaunchKernelGGL(mfma_f16_kernel, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream,
                       out, iters);
    return launched();
}

int qpk_mfma_f32(float* out, int blocks, int iters, void* stream)
{
    if (!out || blocks <= 0 || iters <= 0) return 1;
    hipLaunchKernelGGL(mfma_f32_kernel, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream, out,
                       iters);
    return launched();
}

// out: blocks * 256 floats; clk: blocks * 4 waves * 2 uint64 (shader clocks,
// 100 MHz ticks).
int qpk_clock(float* out, uint64_t* clk, int blocks, int iters, void* stream)
{
    if (!out || !clk || blocks <= 0 || iters <= 0) return 1;
    hipLaunchKernelGGL(clock_kernel, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream, out,
                       clk, iters);
    return launched();
}

// src, dst: n16 16-byte elements each, 16-byte aligned, not overlapping;
// chunked = 0: grid-stride, else one contiguous range per workgroup.
int qpk_copy(const void* src, void* dst, size_t n16, int blocks, int chunked, void* stream)
{
    if (!src || !dst || n16 == 0 || blocks <= 0) return 1;
    if (((uintptr_t)src | (uintptr_t)dst) & 15) return 1;
    if (chunked)
        hipLaunchKernelGGL(copy_chunk_kernel, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream,
                           (const f32x4*)src, (f32x4*)dst, n16, (n16 + blocks - 1) / blocks);
    else
        hipLaunchKernelGGL(copy_kernel, dim3(blocks), dim3(kThreads), 0, (hipStream_t)stream,
                           (const f32x4*)src, (f32x4*)dst, n16);
    return launched();
}

}  // extern "C"
