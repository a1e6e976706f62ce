// Shared per-point MLP layer (Section 4.2) with the fusion by addition of
// Section 4.3 folded into the GEMM epilogue, and the per-cloud max-pool of the
// PointNet backbone (Section 5.1 "Models").
//
// bf16 path (pv_point_mlp_tile_kernel): the layer is a [M x Cin] x [Cin x Cout]
// product whose bytes, not flops, set its time, so each wave owns 32 points x
// (32*NB) output channels and puts every global load of its tile in flight
// before it touches the first one: the residual rows (the devoxelised voxel
// branch), the point rows and the weight rows. v_mfma_f32_32x32x16_bf16 runs
// with the weights as the A operand and the points as B, so each lane ends up
// holding four consecutive output channels of one point; the epilogue adds
// bias and the per-cloud row, applies the folded batch norm (from a table in
// LDS) and the activation, adds the residual and writes 16-byte (8-byte for
// bf16) vectors. Shapes that rule out vector access take the scalar kernel.
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

// Raw 8-value operand fragments: fp32 rows stay as two float4 until the MFMA
// needs them, so no conversion sits between the loads.
struct Frag32 {
    float4 lo, hi;
};
__device__ __forceinline__ Frag32 raw_load(const float* p) {
    return Frag32{*(const float4*)p, *(const float4*)(p + 4)};
}
__device__ __forceinline__ uint4 raw_load(const uint16_t* p) { return *(const uint4*)p; }
__device__ __forceinline__ pv_bf16x8 to_frag(const Frag32& f, bool keep) {
    const uint32_t u0 = pv_pack_bf16x2(f.lo.x, f.lo.y), u1 = pv_pack_bf16x2(f.lo.z, f.lo.w);
    const uint32_t u2 = pv_pack_bf16x2(f.hi.x, f.hi.y), u3 = pv_pack_bf16x2(f.hi.z, f.hi.w);
    const uint4 u = keep ? uint4{u0, u1, u2, u3} : uint4{0u, 0u, 0u, 0u};
    pv_bf16x8 r;
    __builtin_memcpy(&r, &u, 16);
    return r;
}
__device__ __forceinline__ pv_bf16x8 to_frag(const uint4& f, bool keep) {
    const uint4 u = keep ? f : uint4{0u, 0u, 0u, 0u};
    pv_bf16x8 r;
    __builtin_memcpy(&r, &u, 16);
    return r;
}

template <typename XT>
struct RawOf;
template <>
struct RawOf<float> {
    typedef Frag32 T;
};
template <>
struct RawOf<uint16_t> {
    typedef uint4 T;
};

// Requirements (checked by the launcher): Cin % 8 == 0, Cout % 4 == 0, x rows
// and weight rows 16-byte aligned, residual / cloud rows 16-byte aligned,
// output rows 16-byte (fp32) or 8-byte (bf16) aligned.
template <int NB, typename XT>
__global__ __launch_bounds__(kWaves * 64) void pv_point_mlp_tile_kernel(
    const XT* __restrict__ x, int x_ld, int M, int Cin, int Cout, const uint16_t* __restrict__ w,
    PvBnFold bn, int act, float slope, const float* __restrict__ cloud_bias, int ppc,
    const float* __restrict__ residual, int res_ld, void* __restrict__ out, int out_bf16,
    int out_ld) {
    __shared__ float4 tab[2][NB * 8];  // folded scale / shift, 4 channels per entry
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int n0 = blockIdx.y * (NB * 32);
    const int ncols = min(NB * 32, Cout - n0);
    if (threadIdx.x < NB * 32) {
        const int c = min(n0 + (int)threadIdx.x, Cout - 1);
        float sc, sh;
        pv_bn_coeffs(bn, c, sc, sh);
        ((float*)tab[0])[threadIdx.x] = sc;
        ((float*)tab[1])[threadIdx.x] = sh;
    }
    __syncthreads();
    const int m0 = (blockIdx.x * kWaves + wave) * 32;
    if (m0 >= M) return;
    const int r32 = lane & 31, h = lane >> 5;
    // Rows past M are clamped onto the last row: they compute values that are
    // never stored, and every load stays inside the caller's buffers.
    const int m = min(m0 + r32, M - 1);
    const bool mrow = m0 + r32 < M;
    const XT* xr = x + (size_t)m * x_ld + 8 * h;
    const uint16_t* wr[NB];
#pragma unroll
    for (int nb = 0; nb < NB; nb++)
        wr[nb] = w + (size_t)min(n0 + nb * 32 + r32, Cout - 1) * Cin + 8 * h;

    // Column offsets of this lane's four-channel groups, clamped into the
    // valid columns so that every load below is unconditional (one batch,
    // no branches between loads); clamped groups are never stored.
    int coff[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; nb++)
#pragma unroll
        for (int g = 0; g < 4; g++) coff[nb][g] = n0 + min(nb * 32 + g * 8 + 4 * h, ncols - 4);

    // The residual rows go in flight first: they are consumed last.
    float4 res[NB][4];
    if (residual) {
        const float* rr = residual + (size_t)m * res_ld;
#pragma unroll
        for (int nb = 0; nb < NB; nb++)
#pragma unroll
            for (int g = 0; g < 4; g++) res[nb][g] = *(const float4*)(rr + coff[nb][g]);
    } else {
#pragma unroll
        for (int nb = 0; nb < NB; nb++)
#pragma unroll
            for (int g = 0; g < 4; g++) res[nb][g] = float4{0.f, 0.f, 0.f, 0.f};
    }

    pv_f32x16 acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; nb++)
#pragma unroll
        for (int e = 0; e < 16; e++) acc[nb][e] = 0.f;

    typedef typename RawOf<XT>::T XRaw;
    for (int k0 = 0; k0 < Cin; k0 += 64) {
        XRaw xf[4];
        uint4 wf[4][NB];
        bool kv[4];
#pragma unroll
        for (int ks = 0; ks < 4; ks++) {
            // xr and wr already point at this lane's half (8 * h) of each step
            const int k = k0 + ks * 16;
            kv[ks] = k + 8 * h < Cin;
            const int kk = kv[ks] ? k : 0;
            xf[ks] = raw_load(xr + kk);
#pragma unroll
            for (int nb = 0; nb < NB; nb++) wf[ks][nb] = raw_load(wr[nb] + kk);
        }
#pragma unroll
        for (int ks = 0; ks < 4; ks++) {
            const pv_bf16x8 bfr = to_frag(xf[ks], kv[ks]);
#pragma unroll
            for (int nb = 0; nb < NB; nb++)
                acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(to_frag(wf[ks][nb], kv[ks]),
                                                                  bfr, acc[nb], 0, 0, 0);
        }
    }

    // Every value of the tile is finished before the first store: on this
    // architecture one counter tracks loads and stores alike, so a load after
    // a store would have to wait for that store.
    if (cloud_bias) {
        const float* cbr = cloud_bias + (size_t)(m / ppc) * Cout;
        float4 cb[NB][4];
#pragma unroll
        for (int nb = 0; nb < NB; nb++)
#pragma unroll
            for (int g = 0; g < 4; g++) cb[nb][g] = *(const float4*)(cbr + coff[nb][g]);
#pragma unroll
        for (int nb = 0; nb < NB; nb++)
#pragma unroll
            for (int g = 0; g < 4; g++) {
                acc[nb][4 * g] += cb[nb][g].x;
                acc[nb][4 * g + 1] += cb[nb][g].y;
                acc[nb][4 * g + 2] += cb[nb][g].z;
                acc[nb][4 * g + 3] += cb[nb][g].w;
            }
    }
    const float neg = act == PVCONV_ACT_LEAKY ? slope : (act == PVCONV_ACT_RELU ? 0.f : 1.f);
#pragma unroll
    for (int nb = 0; nb < NB; nb++)
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const int t = (coff[nb][g] - n0) >> 2;
            const float4 sc = tab[0][t], sh = tab[1][t];
            float v[4] = {acc[nb][4 * g] * sc.x + sh.x, acc[nb][4 * g + 1] * sc.y + sh.y,
                          acc[nb][4 * g + 2] * sc.z + sh.z, acc[nb][4 * g + 3] * sc.w + sh.w};
#pragma unroll
            for (int j = 0; j < 4; j++) v[j] = v[j] >= 0.f ? v[j] : v[j] * neg;
            res[nb][g].x += v[0];
            res[nb][g].y += v[1];
            res[nb][g].z += v[2];
            res[nb][g].w += v[3];
        }
    if (!mrow) return;
    const size_t orow = (size_t)(m0 + r32) * out_ld;
#pragma unroll
    for (int nb = 0; nb < NB; nb++)
#pragma unroll
        for (int g = 0; g < 4; g++) {
            if (nb * 32 + g * 8 + 4 * h >= ncols) continue;
            const float4 v = res[nb][g];
            if (out_bf16)
                *(uint2*)((uint16_t*)out + orow + coff[nb][g]) =
                    uint2{pv_pack_bf16x2(v.x, v.y), pv_pack_bf16x2(v.z, v.w)};
            else
                *(float4*)((float*)out + orow + coff[nb][g]) = v;
        }
}

// Scalar-epilogue kernel for shapes the tile kernel cannot take (odd channel
// counts or unaligned rows): one wave per 32 points x (32*NB) channels with
// the points as the A operand.
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
                 bool tile, const PvBnFold& bn, int act, float slope, const float* cb, int ppc,
                 const float* res, int res_ld, void* out, bool out_bf16, int out_ld,
                 hipStream_t s) {
    dim3 g((M + kWaves * 32 - 1) / (kWaves * 32), (Cout + NB * 32 - 1) / (NB * 32));
    if (tile)
        hipLaunchKernelGGL((pv_point_mlp_tile_kernel<NB, XT>), g, dim3(kWaves * 64), 0, s,
                           (const XT*)x, x_ld, M, Cin, Cout, (const uint16_t*)w, bn, act, slope,
                           cb, ppc, res, res_ld, out, (int)out_bf16, out_ld);
    else if (vec)
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
        const bool tile =
            vec && Cout % 4 == 0 && (!res || (pv_aligned16(res) && res_ld % 4 == 0)) &&
            (!cb || pv_aligned16(cb)) && out_ld % 4 == 0 &&
            ((uintptr_t)out & (out_bf16 ? 7u : 15u)) == 0;
        if (x_bf16) {
            if (Cout > 64)
                launch_mfma<4, uint16_t>(x, x_ld, M, Cin, Cout, w, vec, tile, bn, act, slope, cb,
                                         ppc, res, res_ld, out, out_bf16, out_ld, s);
            else
                launch_mfma<2, uint16_t>(x, x_ld, M, Cin, Cout, w, vec, tile, bn, act, slope, cb,
                                         ppc, res, res_ld, out, out_bf16, out_ld, s);
        } else {
            if (Cout > 64)
                launch_mfma<4, float>(x, x_ld, M, Cin, Cout, w, vec, tile, bn, act, slope, cb,
                                      ppc, res, res_ld, out, out_bf16, out_ld, s);
            else
                launch_mfma<2, float>(x, x_ld, M, Cin, Cout, w, vec, tile, bn, act, slope, cb,
                                      ppc, res, res_ld, out, out_bf16, out_ld, s);
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
