// Peak microbenchmarks for the bench's measured denominators (measurement only; the half-sweep
// does not use them): FP32 MFMA issue rate, FP32 VALU FMA rate (unpacked: packed FP32 is not
// generated anywhere in this project), a streaming HBM copy, and a pairing of an MFMA stream
// with a VALU stream on every SIMD (whether the two kinds of work overlap).  Each launch runs on
// the caller's stream; the caller times it and counts the work from the documented formulas.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef float f4 __attribute__((ext_vector_type(4)));

constexpr int kChains = 8;        // independent accumulators per wave (covers the latencies)
constexpr int kFmaPerIter = 64;   // VALU FMAs per loop iteration and lane (the chains in turn)

// The MFMA stream of one wave: iters x kChains v_mfma_f32_16x16x4f32 (2048 flops each), chains
// independent; returns the lane's share of their sum.
__device__ __forceinline__ float mfma_stream(float a, float b, int iters) {
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
    return s[0] + s[1] + s[2] + s[3];
}

// The VALU stream of one lane: iters x kFmaPerIter fmaf (2 flops each) over kChains independent
// chains (64 per iteration, so the loop's own scalar instructions stay few); returns their sum.
__device__ __forceinline__ float valu_stream(float a, float b, int iters) {
    float acc[kChains];
#pragma unroll
    for (int k = 0; k < kChains; ++k) acc[k] = (float)k * 1e-3f;
    for (int it = 0; it < iters; ++it) {
#pragma unroll
        for (int j = 0; j < kFmaPerIter; ++j)
            acc[j % kChains] = __builtin_fmaf(acc[j % kChains], a, b);
    }
    float s = 0.f;
#pragma unroll
    for (int k = 0; k < kChains; ++k) s += acc[k];
    return s;
}

__global__ __launch_bounds__(64) void k_peak_mfma(const float* __restrict__ in, int iters,
                                                  float* __restrict__ out) {
    const int lane = threadIdx.x;
    out[blockIdx.x * 64 + lane] = mfma_stream(in[lane] * 1e-3f, in[64 + lane] * 1e-3f, iters);
}

__global__ __launch_bounds__(256) void k_peak_fma(const float* __restrict__ in, int iters,
                                                  float* __restrict__ out) {
    const int t = threadIdx.x;
    out[blockIdx.x * 256 + t] =
        valu_stream(1.f + in[t & 63] * 1e-7f, in[64 + (t & 63)] * 1e-7f, iters);
}

// Eight waves: waves 0-3 run the MFMA stream (iters_m iterations) when mode & 1, waves 4-7 the
// VALU stream (iters_v iterations) when mode & 2; the others exit at once.  Wave w of a
// workgroup runs on SIMD w mod 4 (the MFMA stream on waves 0, 2, 4, 6 takes twice as long as on
// waves 0-3), so with one workgroup per CU every SIMD holds one wave of each kind: if the two
// kinds of work overlapped, mode 3 would take the longer of modes 1 and 2, not their sum.
__global__ __launch_bounds__(512) void k_peak_pair(const float* __restrict__ in, int iters_m,
                                                   int iters_v, int mode,
                                                   float* __restrict__ out) {
    const int t = threadIdx.x, lane = t & 63, w = t >> 6;
    float v = 0.f;
    if (w < 4 && (mode & 1)) v = mfma_stream(in[lane] * 1e-3f, in[64 + lane] * 1e-3f, iters_m);
    if (w >= 4 && (mode & 2))
        v = valu_stream(1.f + in[lane] * 1e-7f, in[64 + lane] * 1e-7f, iters_v);
    out[blockIdx.x * 512 + t] = v;
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

// in: >= 128 floats; out: >= blocks * 256 floats.
// Work: blocks * 256 * iters * kFmaPerIter * 2 flops.
int peaks_fma(const float* in, float* out, int blocks, int iters, void* stream) {
    if (!in || !out || blocks <= 0 || iters <= 0) return -1;
    hipLaunchKernelGGL(k_peak_fma, dim3(blocks), dim3(256), 0, (hipStream_t)stream, in, iters,
                       out);
    return hipGetLastError() == hipSuccess ? 0 : -2;
}

// in: >= 128 floats; out: >= blocks * 512 floats.  mode 1: the MFMA waves only (blocks * 4 *
// iters_m * kChains * 2048 flops), 2: the VALU waves only (blocks * 256 * iters_v * kFmaPerIter
// * 2 flops), 3: both.  blocks = the CU count pairs the two kinds on every SIMD.
int peaks_pair(const float* in, float* out, int blocks, int iters_m, int iters_v, int mode,
               void* stream) {
    if (!in || !out || blocks <= 0 || iters_m <= 0 || iters_v <= 0 || mode < 1 || mode > 3)
        return -1;
    hipLaunchKernelGGL(k_peak_pair, dim3(blocks), dim3(512), 0, (hipStream_t)stream, in, iters_m,
                       iters_v, mode, out);
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
int peaks_fma_per_iter(void) { return kFmaPerIter; }

}  // extern "C"
