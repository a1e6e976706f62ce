// Backward pass of the layer's steps, with respect to their inputs: the
// adjoints of the linear maps of Eq. 2 (Section 4.1 "Voxelization"), of the
// trilinear and nearest-neighbour devoxelisations (Section 4.1
// "Devoxelization") and of the 3x3x3 convolution (Section 4.1 "Feature
// Aggregation"), and the elementwise batch norm + activation.
//
//  * voxelise backward is a gather: each point reads its voxel's gradient row
//    and divides by the voxel's count (one item per point and 8 channels, as
//    in the devoxelise gather);
//  * devoxelise backward is a scatter-add onto the grid: the gradient grid is
//    cleared by a fill kernel, then every (point, corner, channel) adds its
//    weighted gradient with a hardware fp32 atomic (global_atomic_add_f32),
//    one channel per lane. The order of the adds, and so the last bits of the
//    sums, vary between runs;
//  * the convolution's input gradient is the forward convolution of the
//    output gradient with the kernel mirrored through its centre and its
//    channel axes swapped, W'[i][t][o] = W[o][26 - t][i]: a transform kernel
//    writes W' into the workspace and the forward MFMA kernel does the rest.
#include "pv_common.h"

namespace {

template <typename T>
__device__ __forceinline__ void load8(const T* src, float* v);
template <>
__device__ __forceinline__ void load8<float>(const float* src, float* v) {
    const float4 a = *(const float4*)src, b = *(const float4*)(src + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* src, float* v) {
    const uint4 a = *(const uint4*)src;
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int i = 0; i < 4; i++) {
        v[2 * i] = pv_bf16_to_f32((uint16_t)(w[i] & 0xffffu));
        v[2 * i + 1] = pv_bf16_to_f32((uint16_t)(w[i] >> 16));
    }
}

template <typename T>
__device__ __forceinline__ float load1(const T* p);
template <>
__device__ __forceinline__ float load1<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load1<uint16_t>(const uint16_t* p) { return pv_bf16_to_f32(*p); }

__device__ __forceinline__ void store8(float* dst, const float* v) {
    *(float4*)dst = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

// Items: (point, 8-channel group) when VEC, else (point, channel); each XCD
// takes a contiguous range of workgroups.
__device__ __forceinline__ size_t xcd_item(unsigned nblocks) {
    size_t bid = blockIdx.x;
    if ((nblocks & 7) == 0) bid = (bid & 7) * (nblocks >> 3) + (bid >> 3);
    return bid * 256 + threadIdx.x;
}

// dF[k] = dV[id_k] / N[id_k]. An index outside the grid, or a count below
// one, is invalid input: the index is clamped and the count taken as one.
template <typename GT, bool VEC>
__global__ __launch_bounds__(256) void pv_voxelize_backward_kernel(
    const GT* __restrict__ dgrid, const int32_t* __restrict__ ids,
    const int32_t* __restrict__ counts, float* __restrict__ dfeats, int N, int R, int C,
    size_t items) {
    const size_t item = xcd_item(gridDim.x);
    if (item >= items) return;
    const int per_point = VEC ? C / 8 : C;
    const size_t point = item / per_point;
    const int g = (int)(item - point * per_point);
    const size_t b = point / N;
    const int V = R * R * R;
    const int id = min(max(ids[point], 0), V - 1);
    const float n = (float)max(counts[b * V + id], 1);
    const GT* row = dgrid + (b * V + id) * C;
    if (VEC) {
        float v[8];
        load8<GT>(row + g * 8, v);
#pragma unroll
        for (int i = 0; i < 8; i++) v[i] = v[i] / n;
        store8(dfeats + point * C + g * 8, v);
    } else {
        dfeats[point * C + g] = load1<GT>(row + g) / n;
    }
}

// Zero fill of n floats (grid-stride, 16-byte stores where aligned).
__global__ __launch_bounds__(256) void pv_fill_zero_kernel(float* __restrict__ p, size_t n) {
    const size_t stride = (size_t)gridDim.x * 256;
    if (((uintptr_t)p & 15) == 0) {
        float4* p4 = (float4*)p;
        const size_t n4 = n / 4;
        for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n4; i += stride)
            p4[i] = make_float4(0.f, 0.f, 0.f, 0.f);
        for (size_t i = n4 * 4 + (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride)
            p[i] = 0.f;
    } else {
        for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += stride) p[i] = 0.f;
    }
}

// The trilinear cells and weights of a normalised coordinate along one axis,
// as the forward devoxelisation forms them (fp64, rounded once per product).
struct Axis {
    int i0, i1;
    double w0, w1;
};

__device__ __forceinline__ Axis trilinear_axis(float x, int R) {
    double t = (double)x * (double)R - 0.5;
    t = fmin(fmax(t, 0.0), (double)(R - 1));  // also maps NaN to 0
    const double f = floor(t);
    Axis a;
    a.i0 = (int)f;
    a.i1 = min(a.i0 + 1, R - 1);
    a.w1 = t - f;
    a.w0 = 1.0 - a.w1;
    return a;
}

// Scatter kernels: one (point, channel) item per lane, consecutive lanes on
// consecutive channels of a point, so that every atomic instruction adds to
// 64 consecutive floats of a cell row (6.5x faster than 8 channels per lane,
// whose atomics touch 8 floats 32 bytes apart).

// dG[cell] += w(point, cell) * dout[point] over the point's 8 cells.
__global__ __launch_bounds__(256) void pv_devoxelize_backward_kernel(
    const float* __restrict__ dout, const float* __restrict__ pn, float* __restrict__ dgrid,
    int N, int R, int C, size_t items) {
    const size_t item = xcd_item(gridDim.x);
    if (item >= items) return;
    const size_t point = item / C;
    const int c = (int)(item - point * C);
    const size_t b = point / N;
    const size_t V = (size_t)R * R * R;
    const float* p = pn + point * 3;
    const Axis ax = trilinear_axis(p[0], R), ay = trilinear_axis(p[1], R),
               az = trilinear_axis(p[2], R);
    const float v = dout[point * C + c];
    float* base = dgrid + b * V * C + c;
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
                unsafeAtomicAdd(base + (((size_t)iu * R + iv) * R + iw) * C, wt * v);
            }
        }
    }
}

// dG[id_k] += dout[k]. An index outside the grid is clamped (invalid input).
__global__ __launch_bounds__(256) void pv_devoxelize_nearest_backward_kernel(
    const float* __restrict__ dout, const int32_t* __restrict__ ids, float* __restrict__ dgrid,
    int N, int R, int C, size_t items) {
    const size_t item = xcd_item(gridDim.x);
    if (item >= items) return;
    const size_t point = item / C;
    const int c = (int)(item - point * C);
    const size_t b = point / N;
    const int V = R * R * R;
    const int id = min(max(ids[point], 0), V - 1);
    unsafeAtomicAdd(dgrid + (b * V + id) * C + c, dout[point * C + c]);
}

// W'[i][t][o] = W[o][26 - t][i]: the kernel mirrored through its centre
// (offset d -> -d) with input and output channels swapped.
template <typename T>
__global__ __launch_bounds__(256) void pv_conv_weight_flip_kernel(const T* __restrict__ w,
                                                                  T* __restrict__ wf, int Cin,
                                                                  int Cout) {
    const size_t n = (size_t)Cout * 27 * Cin;
    for (size_t j = (size_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (size_t)gridDim.x * 256) {
        // j indexes W' = [Cin][27][Cout]
        const int o = (int)(j % Cout);
        const int t = (int)((j / Cout) % 27);
        const int i = (int)(j / ((size_t)Cout * 27));
        wf[j] = w[((size_t)o * 27 + (26 - t)) * Cin + i];
    }
}

// dz = dy * act'(y) * gamma / sqrt(var + eps), act' read from the sign of y:
// 1 where y > 0, else the negative-side slope (leaky: slope, ReLU: 0,
// none: 1). V4: four consecutive elements of one row per thread (C % 4 == 0,
// 16-byte aligned dy and dz).
template <typename YT>
__device__ __forceinline__ void load4(const YT* p, float* v);
template <>
__device__ __forceinline__ void load4<float>(const float* p, float* v) {
    const float4 a = *(const float4*)p;
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
}
template <>
__device__ __forceinline__ void load4<uint16_t>(const uint16_t* p, float* v) {
    const uint2 a = *(const uint2*)p;
    v[0] = pv_bf16_to_f32((uint16_t)(a.x & 0xffffu));
    v[1] = pv_bf16_to_f32((uint16_t)(a.x >> 16));
    v[2] = pv_bf16_to_f32((uint16_t)(a.y & 0xffffu));
    v[3] = pv_bf16_to_f32((uint16_t)(a.y >> 16));
}

// dz may alias dy (each element is read, then written, by one thread).
template <typename YT, bool V4>
__global__ __launch_bounds__(256) void pv_act_bn_backward_kernel(
    const float* dy, const YT* __restrict__ y, PvBnFold bn, float neg, float* dz, int C,
    size_t n) {
    const size_t stride = (size_t)gridDim.x * 256;
    constexpr int E = V4 ? 4 : 1;
    for (size_t j = ((size_t)blockIdx.x * 256 + threadIdx.x) * E; j < n; j += stride * E) {
        const int c = (int)(j % C);
        float yv[E], g[E];
        if (V4) {
            load4<YT>(y + j, yv);
            load4<float>(dy + j, g);
        } else {
            yv[0] = load1<YT>(y + j);
            g[0] = dy[j];
        }
#pragma unroll
        for (int e = 0; e < E; e++) {
            float scale, shift;
            pv_bn_coeffs(bn, c + e, scale, shift);
            g[e] = g[e] * (yv[e] > 0.f ? 1.f : neg) * scale;
        }
        if (V4)
            *(float4*)(dz + j) = make_float4(g[0], g[1], g[2], g[3]);
        else
            dz[j] = g[0];
    }
}

unsigned blocks_for(size_t items) { return (unsigned)((items + 255) / 256); }

unsigned fill_blocks(size_t n) {
    const size_t b = (n / 4 + 255) / 256;
    return (unsigned)std::max<size_t>(1, std::min<size_t>(b, 4096));
}

}  // namespace

size_t pv_conv3d_bwd_data_ws_bytes(int Cin, int Cout, bool bf16) {
    return pv_align256((size_t)Cout * 27 * Cin * (bf16 ? 2 : 4)) +
           pv_conv3d_ws_bytes(Cout, Cin, bf16);
}

pvconv_status pv_launch_voxelize_backward(const void* dgrid, bool bf16, int B, int N, int C,
                                          int R, const int32_t* ids, const int32_t* counts,
                                          float* dfeats, hipStream_t s) {
    if (B == 0 || N == 0) return PVCONV_OK;
    const bool vec = (C % 8 == 0) && pv_aligned16(dgrid) && pv_aligned16(dfeats);
    const size_t items = (size_t)B * N * (vec ? C / 8 : C);
    auto go = [&](auto t) {
        typedef decltype(t) GT;
        if (vec)
            hipLaunchKernelGGL((pv_voxelize_backward_kernel<GT, true>), dim3(blocks_for(items)),
                               dim3(256), 0, s, (const GT*)dgrid, ids, counts, dfeats, N, R, C,
                               items);
        else
            hipLaunchKernelGGL((pv_voxelize_backward_kernel<GT, false>), dim3(blocks_for(items)),
                               dim3(256), 0, s, (const GT*)dgrid, ids, counts, dfeats, N, R, C,
                               items);
    };
    if (bf16)
        go(uint16_t{});
    else
        go(float{});
    return pv_launch_status();
}

pvconv_status pv_launch_devoxelize_backward(const float* dout, int B, int N, int C, int R,
                                            const float* pn, const int32_t* ids, float* dgrid,
                                            hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    const size_t gn = (size_t)B * R * R * R * C;
    hipLaunchKernelGGL(pv_fill_zero_kernel, dim3(fill_blocks(gn)), dim3(256), 0, s, dgrid, gn);
    if (N == 0) return pv_launch_status();
    const size_t items = (size_t)B * N * C;
    if (ids)
        hipLaunchKernelGGL(pv_devoxelize_nearest_backward_kernel, dim3(blocks_for(items)),
                           dim3(256), 0, s, dout, ids, dgrid, N, R, C, items);
    else
        hipLaunchKernelGGL(pv_devoxelize_backward_kernel, dim3(blocks_for(items)), dim3(256), 0,
                           s, dout, pn, dgrid, N, R, C, items);
    return pv_launch_status();
}

pvconv_status pv_launch_conv3d_backward_data(const void* dy, int B, int R, int Cin, int Cout,
                                             const void* w, bool bf16, void* dx, bool dx_bf16,
                                             void* ws, hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    const size_t nw = (size_t)Cout * 27 * Cin;
    void* wf = ws;
    void* conv_ws = (char*)ws + pv_align256(nw * (bf16 ? 2 : 4));
    const unsigned blocks = (unsigned)std::min<size_t>((nw + 255) / 256, 2048);
    if (bf16)
        hipLaunchKernelGGL((pv_conv_weight_flip_kernel<uint16_t>), dim3(blocks), dim3(256), 0, s,
                           (const uint16_t*)w, (uint16_t*)wf, Cin, Cout);
    else
        hipLaunchKernelGGL((pv_conv_weight_flip_kernel<float>), dim3(blocks), dim3(256), 0, s,
                           (const float*)w, (float*)wf, Cin, Cout);
    pvconv_status st = pv_launch_status();
    if (st != PVCONV_OK) return st;
    // dx = conv(dy, W'): Cout input channels, Cin output channels, no BN or
    // activation
    return pv_launch_conv3d(dy, B, R, Cout, Cin, wf, pv_make_fold(nullptr, nullptr),
                            PVCONV_ACT_NONE, 0.f, bf16, dx, dx_bf16, conv_ws, s);
}

pvconv_status pv_launch_act_bn_backward(const float* dy, const void* y, bool y_bf16, size_t M,
                                        int C, const PvBnFold& bn, int act, float slope,
                                        float* dz, hipStream_t s) {
    const size_t n = M * (size_t)C;
    if (n == 0) return PVCONV_OK;
    const float neg = act == PVCONV_ACT_LEAKY ? slope : (act == PVCONV_ACT_RELU ? 0.f : 1.f);
    const bool v4 = C % 4 == 0 && pv_aligned16(dy) && pv_aligned16(dz) &&
                    ((uintptr_t)y & (y_bf16 ? 7 : 15)) == 0;
    const size_t per = v4 ? 4 : 1;
    const unsigned blocks = (unsigned)std::min<size_t>((n / per + 255) / 256, 8192);
    auto go = [&](auto yt, auto v4t) {
        typedef decltype(yt) YT;
        hipLaunchKernelGGL((pv_act_bn_backward_kernel<YT, decltype(v4t)::value>), dim3(blocks),
                           dim3(256), 0, s, dy, (const YT*)y, bn, neg, dz, C, n);
    };
    if (y_bf16) {
        if (v4) go(uint16_t{}, std::true_type{}); else go(uint16_t{}, std::false_type{});
    } else {
        if (v4) go(float{}, std::true_type{}); else go(float{}, std::false_type{});
    }
    return pv_launch_status();
}
