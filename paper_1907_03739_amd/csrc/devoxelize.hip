// Trilinear devoxelisation (Section 4.1 "Devoxelization"), and the
// nearest-neighbour mapping the same section sets against it (each point takes
// the row of the voxel it falls into).
//
// Wavefront-cooperative gather: consecutive lanes take consecutive 8-channel
// groups of the same point, so each of the point's 8 corner cells is read as
// one contiguous C-channel row (16 B per lane for bf16, 32 B for fp32) and the
// point's output row is written contiguously. Corner indices and weights are
// recomputed per lane from the normalised coordinates (cell centres at
// (i + 1/2) / R, border cells replicated). Each XCD takes a contiguous range
// of points (a few clouds), so that its L2 holds the rows those clouds touch.
#include "pv_common.h"
#include "pv_trilinear.h"

namespace {

template <typename GT>
__device__ __forceinline__ float load1(const GT* p);
template <>
__device__ __forceinline__ float load1<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load1<uint16_t>(const uint16_t* p) { return pv_bf16_to_f32(*p); }

template <typename GT, bool VEC>
__global__ __launch_bounds__(256) void pv_devoxelize_kernel(const GT* __restrict__ grid,
                                                            const float* __restrict__ pn,
                                                            float* __restrict__ out, int N, int R,
                                                            int C, size_t items) {
    // Workgroups are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous range of them (a few clouds), so that the corner rows
    // neighbouring points share are fetched once into that XCD's L2 instead
    // of into all eight.
    size_t bid = blockIdx.x;
    if ((gridDim.x & 7) == 0) bid = (bid & 7) * (gridDim.x >> 3) + (bid >> 3);
    const size_t item = bid * 256 + threadIdx.x;
    if (item >= items) return;
    const int per_point = VEC ? C / 8 : C;
    const size_t point = item / per_point;
    const int g = (int)(item - point * per_point);
    const size_t b = point / N;
    const size_t V = (size_t)R * R * R;
    const float* p = pn + point * 3;
    const PvAxis ax = pv_trilinear_axis(p[0], R), ay = pv_trilinear_axis(p[1], R),
                 az = pv_trilinear_axis(p[2], R);
    const GT* base = grid + b * V * C;
    if (VEC) {
        float acc[8];
        pv_trilinear8<GT>(base + g * 8, C, R, ax, ay, az, acc);
        float* o = out + point * C + g * 8;
        *(float4*)o = make_float4(acc[0], acc[1], acc[2], acc[3]);
        *(float4*)(o + 4) = make_float4(acc[4], acc[5], acc[6], acc[7]);
    } else {
        float acc = 0.f;
        for (int a = 0; a < 2; a++)
            for (int e = 0; e < 2; e++)
                for (int f = 0; f < 2; f++) {
                    const float wt = (float)(((a ? ax.w1 : ax.w0) * (e ? ay.w1 : ay.w0)) *
                                             (f ? az.w1 : az.w0));
                    const size_t cell = ((size_t)(a ? ax.i1 : ax.i0) * R + (e ? ay.i1 : ay.i0)) * R +
                                        (f ? az.i1 : az.i0);
                    acc += wt * load1<GT>(base + cell * C + g);
                }
        out[point * C + g] = acc;
    }
}

template <typename GT>
__device__ __forceinline__ void copy8(const GT* src, float* dst);
template <>
__device__ __forceinline__ void copy8<float>(const float* src, float* dst) {
    *(float4*)dst = *(const float4*)src;
    *(float4*)(dst + 4) = *(const float4*)(src + 4);
}
template <>
__device__ __forceinline__ void copy8<uint16_t>(const uint16_t* src, float* dst) {
    const uint4 a = *(const uint4*)src;
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
    float v[8];
    for (int i = 0; i < 4; i++) {
        v[2 * i] = pv_bf16_to_f32((uint16_t)(w[i] & 0xffffu));
        v[2 * i + 1] = pv_bf16_to_f32((uint16_t)(w[i] >> 16));
    }
    *(float4*)dst = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
}

// Nearest neighbour: out row k = grid row ids[k] of its cloud, in fp32. The
// same item layout and XCD mapping as the trilinear kernel; one 16-byte (bf16)
// or 32-byte (fp32) read and one 32-byte write per item. An index outside the
// grid (invalid input) is clamped, so every read stays inside the cloud's grid.
template <typename GT, bool VEC>
__global__ __launch_bounds__(256) void pv_devoxelize_nearest_kernel(
    const GT* __restrict__ grid, const int32_t* __restrict__ ids, float* __restrict__ out, int N,
    int R, int C, size_t items) {
    size_t bid = blockIdx.x;
    if ((gridDim.x & 7) == 0) bid = (bid & 7) * (gridDim.x >> 3) + (bid >> 3);
    const size_t item = bid * 256 + threadIdx.x;
    if (item >= items) return;
    const int per_point = VEC ? C / 8 : C;
    const size_t point = item / per_point;
    const int g = (int)(item - point * per_point);
    const size_t b = point / N;
    const int V = R * R * R;
    const int id = min(max(ids[point], 0), V - 1);
    const GT* row = grid + (b * V + id) * C;
    if (VEC)
        copy8<GT>(row + g * 8, out + point * C + g * 8);
    else
        out[point * C + g] = load1<GT>(row + g);
}

template <typename GT>
void launch_nearest(const void* grid, int B, int R, int C, const int32_t* ids, int N, float* out,
                    hipStream_t s) {
    const bool vec = (C % 8 == 0) && pv_aligned16(grid) && pv_aligned16(out);
    const size_t items = (size_t)B * N * (vec ? C / 8 : C);
    const unsigned blocks = (unsigned)((items + 255) / 256);
    if (vec)
        hipLaunchKernelGGL((pv_devoxelize_nearest_kernel<GT, true>), dim3(blocks), dim3(256), 0,
                           s, (const GT*)grid, ids, out, N, R, C, items);
    else
        hipLaunchKernelGGL((pv_devoxelize_nearest_kernel<GT, false>), dim3(blocks), dim3(256), 0,
                           s, (const GT*)grid, ids, out, N, R, C, items);
}

template <typename GT>
void launch(const void* grid, int B, int R, int C, const float* pn, int N, float* out,
            hipStream_t s) {
    const bool vec = (C % 8 == 0) && pv_aligned16(grid) && pv_aligned16(out);
    const size_t items = (size_t)B * N * (vec ? C / 8 : C);
    const unsigned blocks = (unsigned)((items + 255) / 256);
    if (vec)
        hipLaunchKernelGGL((pv_devoxelize_kernel<GT, true>), dim3(blocks), dim3(256), 0, s,
                           (const GT*)grid, pn, out, N, R, C, items);
    else
        hipLaunchKernelGGL((pv_devoxelize_kernel<GT, false>), dim3(blocks), dim3(256), 0, s,
                           (const GT*)grid, pn, out, N, R, C, items);
}

}  // namespace

pvconv_status pv_launch_devoxelize(const void* grid, int B, int R, int C, bool grid_bf16,
                                   const float* pn, int N, float* out, hipStream_t s) {
    if (B == 0 || N == 0) return PVCONV_OK;
    if (grid_bf16)
        launch<uint16_t>(grid, B, R, C, pn, N, out, s);
    else
        launch<float>(grid, B, R, C, pn, N, out, s);
    return pv_launch_status();
}

pvconv_status pv_launch_devoxelize_nearest(const void* grid, int B, int R, int C, bool grid_bf16,
                                           const int32_t* ids, int N, float* out,
                                           hipStream_t s) {
    if (B == 0 || N == 0) return PVCONV_OK;
    if (grid_bf16)
        launch_nearest<uint16_t>(grid, B, R, C, ids, N, out, s);
    else
        launch_nearest<float>(grid, B, R, C, ids, N, out, s);
    return pv_launch_status();
}
