// Shared per-point MLP layer (Section 4.2) with the fusion by addition of
// Section 4.3 folded into the GEMM epilogue, and the per-cloud max-pool of the
// PointNet backbone (Section 5.1 "Models").
//
// bf16 path: each wave computes 32 points x (32*NB) output channels with
// v_mfma_f32_32x32x16_bf16. A fragments are read straight from the point rows
// (fp32 inputs are rounded to bf16 in registers), B fragments straight from
// the [C_out][C_in] weight rows, which stay resident in L2. The epilogue adds
// bias and the per-cloud row, applies folded batch norm and the activation,
// adds the residual (the devoxelised voxel branch) and stores.
#include "pv_common.h"

namespace {

constexpr int kWaves = 4;

template <typename XT>
__device__ __forceinline__ pv_bf16x8 load_a8(const XT* p, bool full, int valid);

template <>
__device__ __forceinline__ pv_bf16x8 load_a8<float>(const float* p, bool full, int valid) {
    float v[8];
    if (full) {
        const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
        v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
        v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
    } else {
        for (int t = 0; t < 8; t++) v[t] = t < valid ? p[t] : 0.f;
    }
    pv_bf16x8 r;
    for (int t = 0; t < 8; t++) r[t] = (short)pv_f32_to_bf16(v[t]);
    return r;
}

template <>
__device__ __forceinline__ pv_bf16x8 load_a8<uint16_t>(const uint16_t* p, bool full, int valid) {
    pv_bf16x8 r;
    if (full) {
        const uint4 a = *(const uint4*)p;
        const uint32_t w[4] = {a.x, a.y, a.z, a.w};
        for (int i = 0; i < 4; i++) {
            r[2 * i] = (short)(w[i] & 0xffffu);
            r[2 * i + 1] = (short)(w[i] >> 16);
        }
    } else {
        for (int t = 0; t < 8; t++) r[t] = t < valid ? (short)p[t] : (short)0;
    }
    return r;
}

template <int NB, bool VEC, typename XT>
__global__ __launch_bounds__(kWaves * 64) void pv_point_mlp_bf16_kernel(
    const XT* __restrict__ x, int x_ld, int M, int Cin, int Cout, const uint16_t* __restrict__ w,
    PvBnFold bn, int act, float slope, const float* __restrict__ cloud_bias, int ppc,
    const float* __restrict__ residual, int res_ld, void* __restrict__ out, int out_bf16,
    int out_ld) {
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int m0 = (blockIdx.x * kWaves + wave) * 32;
    const int n0 = blockIdx.y * (NB * 32);
    if (m0 >= M) return;
    const int r32 = lane & 31, khalf = (lane >> 5) * 8;
    const int m = m0 + r32;
    const bool mrow = m < M;
    const XT* xr = x + (size_t)(mrow ? m : 0) * x_ld;

    pv_f32x16 acc[NB];
    for (int j = 0; j < NB; j++)
        for (int e = 0; e < 16; e++) acc[j][e] = 0.f;

    for (int k0 = 0; k0 < Cin; k0 += 16) {
        const int k = k0 + khalf;
        const int valid = mrow ? max(0, min(8, Cin - k)) : 0;
        const pv_bf16x8 a = load_a8<XT>(xr + k, VEC && valid == 8, valid);
        for (int nb = 0; nb < NB; nb++) {
            const int n = n0 + nb * 32 + r32;
            const int wv = n < Cout ? max(0, min(8, Cin - k)) : 0;
            const pv_bf16x8 bfr =
                load_a8<uint16_t>(w + (size_t)(n < Cout ? n : 0) * Cin + k, VEC && wv == 8, wv);
            acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, bfr, acc[nb], 0, 0, 0);
        }
    }

    for (int nb = 0; nb < NB; nb++) {
        const int n = n0 + nb * 32 + r32;
        if (n >= Cout) continue;
        float scale, shift;
        pv_bn_coeffs(bn, n, scale, shift);
        for (int e = 0; e < 16; e++) {
            const int mm = m0 + 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
            if (mm >= M) continue;
            float v = acc[nb][e];
            if (cloud_bias) v += cloud_bias[(size_t)(mm / ppc) * Cout + n];
            v = pv_activate(v * scale + shift, act, slope);
            if (residual) v += residual[(size_t)mm * res_ld + n];
            if (out_bf16)
                ((uint16_t*)out)[(size_t)mm * out_ld + n] = pv_f32_to_bf16(v);
            else
                ((float*)out)[(size_t)mm * out_ld + n] = v;
        }
    }
}

template <typename XT>
__device__ __forceinline__ float ld1(const XT* p);
template <>
__device__ __forceinline__ float ld1<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ld1<uint16_t>(const uint16_t* p) { return pv_bf16_to_f32(*p); }

template <typename XT>
__global__ __launch_bounds__(256) void pv_point_mlp_f32_kernel(
    const XT* __restrict__ x, int x_ld, int M, int Cin, int Cout, const float* __restrict__ w,
    PvBnFold bn, int act, float slope, const float* __restrict__ cloud_bias, int ppc,
    const float* __restrict__ residual, int res_ld, void* __restrict__ out, int out_bf16,
    int out_ld) {
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (size_t)M * Cout) return;
    const int n = (int)(i % Cout);
    const size_t m = i / Cout;
    const XT* xr = x + m * x_ld;
    const float* wr = w + (size_t)n * Cin;
    float s = 0.f;
    for (int k = 0; k < Cin; k++) s += wr[k] * ld1<XT>(xr + k);
    if (cloud_bias) s += cloud_bias[(m / ppc) * Cout + n];
    float scale, shift;
    pv_bn_coeffs(bn, n, scale, shift);
    float v = pv_activate(s * scale + shift, act, slope);
    if (residual) v += residual[m * res_ld + n];
    if (out_bf16)
        ((uint16_t*)out)[m * out_ld + n] = pv_f32_to_bf16(v);
    else
        ((float*)out)[m * out_ld + n] = v;
}

template <int NB, typename XT>
void launch_mfma(const void* x, int x_ld, int M, int Cin, int Cout, const void* w, bool vec,
                 const PvBnFold& bn, int act, float slope, const float* cb, int ppc,
                 const float* res, int res_ld, void* out, bool out_bf16, int out_ld,
                 hipStream_t s) {
    dim3 g((M + kWaves * 32 - 1) / (kWaves * 32), (Cout + NB * 32 - 1) / (NB * 32));
    if (vec)
        hipLaunchKernelGGL((pv_point_mlp_bf16_kernel<NB, true, XT>), g, dim3(kWaves * 64), 0, s,
                           (const XT*)x, x_ld, M, Cin, Cout, (const uint16_t*)w, bn, act, slope,
                           cb, ppc, res, res_ld, out, (int)out_bf16, out_ld);
    else
        hipLaunchKernelGGL((pv_point_mlp_bf16_kernel<NB, false, XT>), g, dim3(kWaves * 64), 0, s,
                           (const XT*)x, x_ld, M, Cin, Cout, (const uint16_t*)w, bn, act, slope,
                           cb, ppc, res, res_ld, out, (int)out_bf16, out_ld);
}

template <typename XT>
__global__ __launch_bounds__(256) void pv_maxpool_kernel(const XT* __restrict__ x, int x_ld,
                                                         int N, int C, float* __restrict__ out) {
    __shared__ float part[4][64];
    const int c = blockIdx.x * 64 + (threadIdx.x & 63);
    const int slice = threadIdx.x >> 6;
    const int b = blockIdx.y;
    float m = -INFINITY;
    if (c < C)
        for (int k = slice; k < N; k += 4) m = fmaxf(m, ld1<XT>(x + ((size_t)b * N + k) * x_ld + c));
    part[slice][threadIdx.x & 63] = m;
    __syncthreads();
    if (slice == 0 && c < C) {
        for (int i = 1; i < 4; i++) m = fmaxf(m, part[i][threadIdx.x]);
        out[(size_t)b * C + c] = m;
    }
}

}  // namespace

pvconv_status pv_launch_point_mlp(const void* x, bool x_bf16, int x_ld, int M, int Cin,
                                  int Cout, const void* w, bool bf16, const PvBnFold& bn,
                                  int act, float slope, const float* cb, int ppc,
                                  const float* res, int res_ld, void* out, bool out_bf16,
                                  int out_ld, hipStream_t s) {
    if (M == 0) return PVCONV_OK;
    if (bf16) {
        const size_t esz = x_bf16 ? 2 : 4;
        const bool vec = Cin % 8 == 0 && pv_aligned16(x) && pv_aligned16(w) &&
                         ((size_t)x_ld * esz) % 16 == 0;
        if (x_bf16) {
            if (Cout > 64)
                launch_mfma<4, uint16_t>(x, x_ld, M, Cin, Cout, w, vec, bn, act, slope, cb, ppc,
                                         res, res_ld, out, out_bf16, out_ld, s);
            else
                launch_mfma<2, uint16_t>(x, x_ld, M, Cin, Cout, w, vec, bn, act, slope, cb, ppc,
                                         res, res_ld, out, out_bf16, out_ld, s);
        } else {
            if (Cout > 64)
                launch_mfma<4, float>(x, x_ld, M, Cin, Cout, w, vec, bn, act, slope, cb, ppc, res,
                                      res_ld, out, out_bf16, out_ld, s);
            else
                launch_mfma<2, float>(x, x_ld, M, Cin, Cout, w, vec, bn, act, slope, cb, ppc, res,
                                      res_ld, out, out_bf16, out_ld, s);
        }
    } else {
        const size_t total = (size_t)M * Cout;
        const unsigned blocks = (unsigned)((total + 255) / 256);
        if (x_bf16)
            hipLaunchKernelGGL(pv_point_mlp_f32_kernel<uint16_t>, dim3(blocks), dim3(256), 0, s,
                               (const uint16_t*)x, x_ld, M, Cin, Cout, (const float*)w, bn, act,
                               slope, cb, ppc, res, res_ld, out, (int)out_bf16, out_ld);
        else
            hipLaunchKernelGGL(pv_point_mlp_f32_kernel<float>, dim3(blocks), dim3(256), 0, s,
                               (const float*)x, x_ld, M, Cin, Cout, (const float*)w, bn, act,
                               slope, cb, ppc, res, res_ld, out, (int)out_bf16, out_ld);
    }
    return pv_launch_status();
}

pvconv_status pv_launch_maxpool(const void* x, bool bf16, int x_ld, int B, int N, int C,
                                float* out, hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    dim3 g((C + 63) / 64, B);
    if (bf16)
        hipLaunchKernelGGL(pv_maxpool_kernel<uint16_t>, g, dim3(256), 0, s, (const uint16_t*)x,
                           x_ld, N, C, out);
    else
        hipLaunchKernelGGL(pv_maxpool_kernel<float>, g, dim3(256), 0, s, (const float*)x, x_ld,
                           N, C, out);
    return pv_launch_status();
}
