// Peak microbenchmarks for the bench's measured denominators (measurement only; the half-sweep
// does not use them): FP32 MFMA issue rate, FP32 VALU FMA rate (unpacked: packed FP32 is not
// generated anywhere in this project) and a streaming HBM copy.  Each launch runs on the
// caller's stream; the caller times it and counts the work from the documented formulas.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;   // independent accumulators per wave (covers the MFMA latency)

// Each wave: iters x kChains v_mfma_f32_16x16x4f32 (2048 flops each), chains independent.
__global__ __launch_bounds__(64) void k_peak_mfma(const float* __restrict__ in, int iters,
                                                  float* __restrict__ out) {
    const int lane = threadIdx.x;
    const float a = in[lane] * 1e-3f, b = in[64 + lane] * 1e-3f;
    f4 acc[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) acc[k] = f4{0.f, 0.f, 0.f, 0.f};
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < kChains; ++k)
            acc[k] = __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, acc[k], 0, 0, 0);
    }
    f4 s = acc[0];
#pragma unroll
    for (int k = 1; k < kChains; ++k) s += acc[k];
    out[blockIdx.x * 64 + lane] = s[0] + s[1] + s[2] + s[3];
}

// Each lane: iters x kChains fmaf (2 flops each), chains independent.
__global__ __launch_bounds__(256) void k_peak_fma(const float* __restrict__ in, int iters,
                                                  float* __restrict__ out) {
    const int t = threadIdx.x;
    const float a = 1.f + in[t & 63] * 1e-7f, b = in[64 + (t & 63)] * 1e-7f;
    float acc[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) acc[k] = (float)k * 1e-3f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int k = 0; k < kChains; ++k) acc[k] = __builtin_fmaf(acc[k], a, b);
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kChains; ++k) s += acc[k];
    out[blockIdx.x * 256 + t] = s;
}

// dst[i] = src[i] over n4 float4 elements, grid-stride.
__global__ __launch_bounds__(256) void k_copy(const f4* __restrict__ src, f4* __restrict__ dst,
                                              int64_t n4) {
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < n4; i += stride)
        dst[i] = src[i];
}

}  // namespace

extern "C" {

// in: >= 128 floats; out: >= blocks * 64 floats.  Work: blocks * iters * kChains * 2048 flops.
int peaks_mfma(const float* in, float* out, int blocks, int iters, void* stream) {
    if (!in || !out || blocks <= 0 || iters <= 0) return -1;
    hipLaunchKernelGGL(k_peak_mfma, dim3(blocks), dim3(64), 0, (hipStream_t)stream, in, iters,
                       out);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

// in: >= 128 floats; out: >= blocks * 256 floats.  Work: blocks * 256 * iters * kChains * 2.
int peaks_fma(const float* in, float* out, int blocks, int iters, void* stream) {
    if (!in || !out || blocks <= 0 || iters <= 0) return -1;
    hipLaunchKernelGGL(k_peak_fma, dim3(blocks), dim3(256), 0, (hipStream_t)stream, in, iters,
                       out);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

// src, dst: n4 float4 each, 16-byte aligned.  Traffic: 32 * n4 bytes (read + write).
int peaks_copy(const void* src, void* dst, int64_t n4, int blocks, void* stream) {
    if (!src || !dst || n4 <= 0 || blocks <= 0) return -1;
    if (((uintptr_t)src | (uintptr_t)dst) & 15) return -1;
    hipLaunchKernelGGL(k_copy, dim3(blocks), dim3(256), 0, (hipStream_t)stream, (const f4*)src,
                       (f4*)dst, n4);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

int peaks_chains(void) { return kChains; }

}  // extern "C"
