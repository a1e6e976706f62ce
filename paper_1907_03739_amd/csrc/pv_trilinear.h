// Trilinear devoxelisation arithmetic (Section 4.1 "Devoxelization"), shared
// by the devoxelisation kernel and the point-MLP kernel that gathers the
// voxel branch itself, so that both give the same bits.
#pragma once
#include "pv_common.h"

// Cell indices and weights along one axis: cell centres at (i + 1/2) / R,
// border cells replicated. The cell coordinate and the weights are formed in
// fp64 (the gather is bound by memory, not ALU), so the only fp32 rounding
// left is the weighted sum itself.
struct PvAxis {
    int i0, i1;
    double w0, w1;
};

__device__ __forceinline__ PvAxis pv_trilinear_axis(float x, int R) {
    double t = (double)x * (double)R - 0.5;
    t = fmin(fmax(t, 0.0), (double)(R - 1));  // also maps NaN to 0
    const double f = floor(t);
    PvAxis a;
    a.i0 = (int)f;
    a.i1 = min(a.i0 + 1, R - 1);
    a.w1 = t - f;
    a.w0 = 1.0 - a.w1;
    return a;
}

template <typename GT>
__device__ __forceinline__ void pv_fma8(const GT* src, float wt, float* acc);
template <>
__device__ __forceinline__ void pv_fma8<float>(const float* src, float wt, float* acc) {
    const float4 a = *(const float4*)src, b = *(const float4*)(src + 4);
    acc[0] += wt * a.x; acc[1] += wt * a.y; acc[2] += wt * a.z; acc[3] += wt * a.w;
    acc[4] += wt * b.x; acc[5] += wt * b.y; acc[6] += wt * b.z; acc[7] += wt * b.w;
}
template <>
__device__ __forceinline__ void pv_fma8<uint16_t>(const uint16_t* src, float wt, float* acc) {
    const uint4 a = *(const uint4*)src;
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
    for (int i = 0; i < 4; i++) {
        acc[2 * i] += wt * pv_bf16_to_f32((uint16_t)(w[i] & 0xffffu));
        acc[2 * i + 1] += wt * pv_bf16_to_f32((uint16_t)(w[i] >> 16));
    }
}

// Eight consecutive channels of one point: the weighted sum over its 8 corner
// cells (u, then v, then w, lower corner first), base = channel 0 of cell 0
// of the point's cloud, C = grid row length. acc is zeroed here.
template <typename GT>
__device__ __forceinline__ void pv_trilinear8(const GT* base, int C, int R, const PvAxis& ax,
                                              const PvAxis& ay, const PvAxis& az, float* acc) {
#pragma unroll
    for (int j = 0; j < 8; j++) acc[j] = 0.f;
#pragma unroll
    for (int a = 0; a < 2; a++) {
        const int iu = a ? ax.i1 : ax.i0;
        const double wu = a ? ax.w1 : ax.w0;
#pragma unroll
        for (int e = 0; e < 2; e++) {
            const int iv = e ? ay.i1 : ay.i0;
            const double wv = e ? ay.w1 : ay.w0;
#pragma unroll
            for (int f = 0; f < 2; f++) {
                const int iw = f ? az.i1 : az.i0;
                const float wt = (float)((wu * wv) * (f ? az.w1 : az.w0));
                pv_fma8<GT>(base + (((size_t)iu * R + iv) * R + iw) * C, wt, acc);
            }
        }
    }
}
