// Measured peaks of the device, the second denominator of the roofline
// fractions next to the published ones: a dense bf16 MFMA loop and a plain
// 16-byte copy. Not part of the PVConv path; the benchmark loads this library
// on its own.
#include <hip/hip_runtime.h>
#include <stdint.h>

namespace {

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float f32x16;

constexpr int kSets = 4;  // operand sets, so consecutive MFMAs see different bits

__device__ __forceinline__ uint32_t mix(uint32_t h) {
    h ^= h >> 16;
    h *= 0x7feb352du;
    h ^= h >> 15;
    h *= 0x846ca68bu;
    h ^= h >> 16;
    return h;
}

// Every wave runs `iters` rounds of kSets independent
// v_mfma_f32_32x32x16_bf16 (32*32*16*2 flop each) on random bf16 operands
// of magnitude [1, 2) with random signs, so the matrix cores switch about as
// many bits as on real data.
__global__ __launch_bounds__(256) void pv_peak_mfma_kernel(int iters, float* __restrict__ out) {
    const uint32_t tid = blockIdx.x * 256u + threadIdx.x;
    bf16x8 a[kSets], b[kSets];
    uint32_t h = mix(tid + 1u);
#pragma unroll
    for (int s = 0; s < kSets; s++)
#pragma unroll
        for (int i = 0; i < 8; i++) {
            h = mix(h + 0x9e3779b9u);
            a[s][i] = (short)(0x3f80u | (h & 0x807fu));
            b[s][i] = (short)(0x3f80u | ((h >> 16) & 0x807fu));
        }
    f32x16 acc[kSets];
#pragma unroll
    for (int s = 0; s < kSets; s++)
#pragma unroll
        for (int e = 0; e < 16; e++) acc[s][e] = 0.f;
    for (int it = 0; it < iters; it++) {
#pragma unroll
        for (int s = 0; s < kSets; s++)
            acc[s] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[s], b[(s + 1) % kSets], acc[s], 0,
                                                             0, 0);
    }
    float sum = 0.f;
#pragma unroll
    for (int s = 0; s < kSets; s++)
#pragma unroll
        for (int e = 0; e < 16; e++) sum += acc[s][e];
    out[tid] = sum;
}

// dst[i] = src[i] over n 16-byte elements: each workgroup copies 1024
// consecutive elements, four per thread, with non-temporal (streaming) loads
// and stores, the fastest of the plain copies tried on this device.
typedef unsigned u32x4 __attribute__((ext_vector_type(4)));
constexpr int kCopyPer = 4;
__global__ __launch_bounds__(256) void pv_peak_copy_kernel(const u32x4* __restrict__ src,
                                                           u32x4* __restrict__ dst, size_t n) {
    const size_t base = (size_t)blockIdx.x * 256 * kCopyPer + threadIdx.x;
    u32x4 v[kCopyPer];
#pragma unroll
    for (int u = 0; u < kCopyPer; u++)
        if (base + u * 256 < n) v[u] = __builtin_nontemporal_load(src + base + u * 256);
#pragma unroll
    for (int u = 0; u < kCopyPer; u++)
        if (base + u * 256 < n) __builtin_nontemporal_store(v[u], dst + base + u * 256);
}

}  // namespace

extern "C" {

// Threads the MFMA probe writes one float each to (its `out` size).
int pv_peak_mfma_threads(int blocks) { return blocks * 256; }

// Flop of one MFMA probe launch.
double pv_peak_mfma_flop(int blocks, int iters) {
    return (double)blocks * 4 * iters * kSets * (32.0 * 32 * 16 * 2);
}

// Launches the MFMA probe: `blocks` workgroups of four waves, `out` holds
// blocks * 256 floats (device). Returns 0 or the HIP error code.
int pv_peak_mfma(int blocks, int iters, float* out, hipStream_t s) {
    if (blocks <= 0 || iters <= 0 || !out) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(pv_peak_mfma_kernel, dim3(blocks), dim3(256), 0, s, iters, out);
    return (int)hipGetLastError();
}

// Copies n16 16-byte elements (device pointers, 16-byte aligned, not
// overlapping). Returns 0 or the HIP error code.
int pv_peak_copy(const void* src, void* dst, size_t n16, hipStream_t s) {
    if (!src || !dst || ((uintptr_t)src | (uintptr_t)dst) % 16) return (int)hipErrorInvalidValue;
    if (n16 == 0) return 0;
    const size_t blocks = (n16 + 256 * kCopyPer - 1) / (256 * kCopyPer);
    if (blocks > 0x7fffffffu) return (int)hipErrorInvalidValue;
    hipLaunchKernelGGL(pv_peak_copy_kernel, dim3((unsigned)blocks), dim3(256), 0, s,
                       (const u32x4*)src, (u32x4*)dst, n16);
    return (int)hipGetLastError();
}

}  // extern "C"
