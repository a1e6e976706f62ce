// Backward pass of the layer's steps, with respect to their inputs: the
// adjoints of the linear maps of Eq. 2 (Section 4.1 "Voxelization"), of the
// trilinear and nearest-neighbour devoxelisations (Section 4.1
// "Devoxelization") and of the 3x3x3 convolution (Section 4.1 "Feature
// Aggregation"), and the elementwise batch norm + activation.
//
//  * voxelise backward is a gather: each point reads its voxel's gradient row
//    and divides by the voxel's count (one item per point and 8 channels, as
//    in the devoxelise gather);
//  * devoxelise backward, the adjoint of a gather, is computed as a gather
//    too, so that every grid row is written once and its sum is taken in a
//    fixed order: the points are sorted stably by the cell of their base
//    corner (the lower of the two trilinear cells on every axis; nearest:
//    their voxel) with a radix sort, each cell's range of the sorted list is
//    recorded, and each cell then sums the weighted gradients of the points
//    whose base corner is the cell or its lower neighbour on some axes;
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

// ---------------------------------------------------------------------------
// Devoxelisation backward as a gather. A point's trilinear cells are, on
// every axis, its base cell i0 and i1 = min(i0 + 1, R - 1), so the points
// that reach cell (u, v, w) have base cells in {u-1, u} x {v-1, v} x
// {w-1, w}. The points are sorted stably by (cloud, base cell) with an LSD
// radix sort on 8-bit digits (one pass per digit of the cell index; the
// clouds' entries stay in their own ranges); each cell's range in the
// sorted list is recorded with, per sorted point, its eight corner weights
// (as pv_devoxelize forms them: fp64 products rounded once) and its
// gradient row (copied into sorted order), and the cells that some point
// reaches are marked (a byte per cell). One workgroup per 64 consecutive
// cells then writes their rows: zeros for unmarked cells, and for marked
// ones the sum, over the cell's eight candidate base cells in a fixed order
// and their points in index order, of the point's weight at this cell times
// its gradient. The sum's order is fixed by the data, so the grid is the
// same bits on every run. Nearest neighbour: the key is the voxel, one range
// per cell, weight one.
// ---------------------------------------------------------------------------
constexpr int kSortChunk = 256;  // entries per sort workgroup (one wave)

// Sort keys: the point's base cell (or voxel, clamped: an index outside the
// grid is invalid input) and its entry index b*N + i; the cell ranges and
// the reached-cell marks cleared.
__global__ __launch_bounds__(256) void pv_devox_bwd_keys_kernel(
    const float* __restrict__ pn, const int32_t* __restrict__ ids, int R, size_t E,
    size_t ncells, uint32_t* __restrict__ key, int32_t* __restrict__ val,
    int2* __restrict__ bounds, uint32_t* __restrict__ act) {
    const size_t stride = (size_t)gridDim.x * 256;
    const size_t t0 = (size_t)blockIdx.x * 256 + threadIdx.x;
    for (size_t i = t0; i < E; i += stride) {
        int cell;
        if (ids) {
            cell = min(max(ids[i], 0), R * R * R - 1);
        } else {
            const float* p = pn + i * 3;
            cell = (trilinear_axis(p[0], R).i0 * R + trilinear_axis(p[1], R).i0) * R +
                   trilinear_axis(p[2], R).i0;
        }
        key[i] = (uint32_t)cell;
        val[i] = (int32_t)i;
    }
    for (size_t k = t0; k < ncells; k += stride) bounds[k] = make_int2(0, 0);
    for (size_t k = t0; k < (ncells + 3) / 4; k += stride) act[k] = 0u;
}

// Radix pass, 1/3: each chunk's histogram of the digit (key >> shift) & 255,
// stored digit-major per cloud: hist[b][digit][chunk]. Workgroup b*nch + j
// takes chunk j of cloud b (so do the scatter's).
__global__ __launch_bounds__(64) void pv_radix_hist_kernel(const uint32_t* __restrict__ key,
                                                           int N, int nch, int shift,
                                                           uint32_t* __restrict__ hist) {
    __shared__ uint32_t h[256];
    const int j = (int)(blockIdx.x % nch), b = (int)(blockIdx.x / nch), lane = threadIdx.x;
    for (int d = lane; d < 256; d += 64) h[d] = 0u;
    __syncthreads();
    const uint32_t* kb = key + (size_t)b * N;
    const int i1 = min(N, (j + 1) * kSortChunk);
    for (int i = j * kSortChunk + lane; i < i1; i += 64) atomicAdd(&h[(kb[i] >> shift) & 255u], 1u);
    __syncthreads();
    for (int d = lane; d < 256; d += 64) hist[((size_t)b * 256 + d) * nch + j] = h[d];
}

// Radix pass, 2/3: per cloud, the exclusive prefix of hist in (digit,
// chunk) order, plus the cloud's first entry: where each chunk's entries of
// each digit start in the output.
__global__ __launch_bounds__(256) void pv_radix_scan_kernel(uint32_t* __restrict__ hist, int N,
                                                            int nch) {
    __shared__ uint32_t s[256];
    const int b = blockIdx.x, d = threadIdx.x;
    uint32_t* row = hist + ((size_t)b * 256 + d) * nch;
    uint32_t t = 0;
    for (int j = 0; j < nch; j++) t += row[j];
    s[d] = t;
    __syncthreads();
    for (int off = 1; off < 256; off <<= 1) {  // inclusive prefix over the digits
        const uint32_t v = d >= off ? s[d - off] : 0u;
        __syncthreads();
        s[d] += v;
        __syncthreads();
    }
    uint32_t run = s[d] - t + (uint32_t)((size_t)b * N);
    for (int j = 0; j < nch; j++) {
        const uint32_t c = row[j];
        row[j] = run;
        run += c;
    }
}

// Radix pass, 3/3: each chunk moves its entries, in order, to their digit's
// place: the lanes of a round that share a digit (found with one ballot per
// digit bit) take consecutive places in lane order after the chunk's earlier
// entries of that digit. Stable, so after the last pass the entries of a
// cell are in index order.
__global__ __launch_bounds__(64) void pv_radix_scatter_kernel(
    const uint32_t* __restrict__ kin, const int32_t* __restrict__ vin,
    uint32_t* __restrict__ kout, int32_t* __restrict__ vout, const uint32_t* __restrict__ hist,
    int N, int nch, int shift) {
    __shared__ uint32_t run[256];
    const int j = (int)(blockIdx.x % nch), b = (int)(blockIdx.x / nch), lane = threadIdx.x;
    for (int d = lane; d < 256; d += 64) run[d] = hist[((size_t)b * 256 + d) * nch + j];
    __syncthreads();
    const size_t cb = (size_t)b * N;
    const uint64_t below = (1ull << lane) - 1ull;
    const int i1 = min(N, (j + 1) * kSortChunk);
    for (int r = j * kSortChunk; r < i1; r += 64) {
        const int i = r + lane;
        const bool ok = i < i1;
        const uint32_t k = ok ? kin[cb + i] : 0u;
        const int32_t v = ok ? vin[cb + i] : 0;
        const uint32_t d = (k >> shift) & 255u;
        uint64_t peers = __ballot(ok);
#pragma unroll
        for (int bit = 0; bit < 8; bit++) {
            const uint64_t m = __ballot((d >> bit) & 1u);
            peers &= ((d >> bit) & 1u) ? m : ~m;
        }
        if (ok) {
            const uint32_t pos = run[d] + (uint32_t)__popcll(peers & below);
            kout[pos] = k;
            vout[pos] = v;
        }
        __syncthreads();  // every lane has read its digit's place
        if (ok && (peers & below) == 0ull) run[d] += (uint32_t)__popcll(peers);
        __syncthreads();
    }
}

// Each cell's range [first, last + 1) in the sorted list (cells without
// points keep the cleared [0, 0)), the cells the points reach, marked, and
// (trilinear) per sorted entry its eight corner weights as pv_devoxelize
// forms them, corner (a, b, c) = offsets (0/1) from the base cell at
// 4a + 2b + c: fp64 products, rounded once. Where both corners of an axis are the grid's last
// cell, the upper one's weight is 0.
__global__ __launch_bounds__(256) void pv_devox_bwd_bounds_kernel(
    const uint32_t* __restrict__ key, const int32_t* __restrict__ val,
    const float* __restrict__ pn, int N, size_t E, int R, int2* __restrict__ bounds,
    float4* __restrict__ rec_w, uint8_t* __restrict__ act) {
    const size_t stride = (size_t)gridDim.x * 256;
    const int V = R * R * R;
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < E; i += stride) {
        const size_t b = i / N;
        const int in = (int)(i - b * N);
        const uint32_t k = key[i];
        int2* bd = bounds + b * V + k;
        if (in == 0 || key[i - 1] != k) bd->x = (int)i;
        if (in == N - 1 || key[i + 1] != k) bd->y = (int)(i + 1);
        const int e = val[i];
        // the cells this point reaches, marked (every writer stores 1)
        const int ku = (int)(k / (uint32_t)(R * R)), kv = (int)(k / (uint32_t)R) % R,
                  kw = (int)(k % (uint32_t)R);
        for (int c = 0; c < (pn ? 8 : 1); c++) {
            const int cu = min(ku + (c >> 2), R - 1), cv = min(kv + ((c >> 1) & 1), R - 1),
                      cw = min(kw + (c & 1), R - 1);
            act[b * V + ((size_t)cu * R + cv) * R + cw] = 1;
        }
        if (pn) {
            const float* p = pn + (size_t)e * 3;
            const Axis ax = trilinear_axis(p[0], R), ay = trilinear_axis(p[1], R),
                       az = trilinear_axis(p[2], R);
            float wt[8];
#pragma unroll
            for (int c = 0; c < 8; c++)
                wt[c] = (float)(((c & 4 ? ax.w1 : ax.w0) * (c & 2 ? ay.w1 : ay.w0)) *
                                (c & 1 ? az.w1 : az.w0));
            rec_w[2 * i] = make_float4(wt[0], wt[1], wt[2], wt[3]);
            rec_w[2 * i + 1] = make_float4(wt[4], wt[5], wt[6], wt[7]);
        }
    }
}

// The gradient rows in sorted order: srow[i] = dout[val[i]], VW floats per
// item.
template <int VW>
__global__ __launch_bounds__(256) void pv_devox_bwd_rows_kernel(const float* __restrict__ dout,
                                                                const int32_t* __restrict__ val,
                                                                int C, size_t items,
                                                                float* __restrict__ srow) {
    const int per = C / VW;
    const size_t stride = (size_t)gridDim.x * 256;
    for (size_t it = (size_t)blockIdx.x * 256 + threadIdx.x; it < items; it += stride) {
        const size_t i = it / per;
        const int q = (int)(it - i * per);
        const float* src = dout + (size_t)val[i] * C + q * VW;
        float* dst = srow + i * C + q * VW;
        if constexpr (VW == 4)
            *(float4*)dst = *(const float4*)src;
        else
            *dst = *src;
    }
}

// x / d for 0 <= x < 2^24 and d >= 1, with inv = 1/d in fp32: the product's
// floor is the quotient or one off it, corrected with the remainder.
__device__ __forceinline__ int pv_div_small(int x, int d, float inv, int* rem) {
    int q = (int)((float)x * inv);
    int r = x - q * d;
    if (r < 0) {
        q--;
        r += d;
    } else if (r >= d) {
        q++;
        r -= d;
    }
    *rem = r;
    return q;
}

// dG rows: workgroup x takes cells x*64 .. x*64 + 63 (of all clouds' cells
// in order); every wave reads their marks, so all know which are reached.
// Items (cell j, channel group q) = threadIdx.x, + 256, ... (walked by
// constant steps, no divisions): unmarked cells' rows are written as
// zeros, marked ones as their sums.
template <int VW, bool NEAREST>
__global__ __launch_bounds__(256) void pv_devox_bwd_gather_kernel(
    const float* __restrict__ srow, const float* __restrict__ rec_w,
    const int2* __restrict__ bounds, const uint8_t* __restrict__ act, size_t ncells, int R,
    int C, float* __restrict__ dgrid) {
    const int per = C / VW;
    const int V = R * R * R, RR = R * R;
    const float invR = 1.f / (float)R, invRR = 1.f / (float)RR;
    const int lane = threadIdx.x & 63;
    const int j0 = (int)threadIdx.x / per, q0 = (int)threadIdx.x - j0 * per;
    const int dj = 256 / per, dq = 256 - dj * per;
    for (size_t c0 = (size_t)blockIdx.x * 64; c0 < ncells; c0 += (size_t)gridDim.x * 64) {
        const uint64_t marked = __ballot(c0 + lane < ncells && act[c0 + lane] != 0);
        const int nc = (int)std::min<size_t>(64, ncells - c0);
        const size_t b0 = c0 / (size_t)V;  // the chunk's first cell: cloud and index
        const int cell0 = (int)(c0 - b0 * V);
        int j = j0, q = q0;
        while (j < nc) {
            const size_t cg = c0 + j;
            float acc[VW];
#pragma unroll
            for (int k = 0; k < VW; k++) acc[k] = 0.f;
            if ((marked >> j) & 1ull) {
                int cell = cell0 + j;
                size_t b = b0;
                while (cell >= V) {  // the chunk runs into the next cloud
                    cell -= V;
                    b++;
                }
                if (NEAREST) {
                    const int2 rg = bounds[cg];
#pragma unroll 2
                    for (int sidx = rg.x; sidx < rg.y; sidx++) {
                        const float* src = srow + (size_t)sidx * C + q * VW;
                        if constexpr (VW == 4) {
                            const float4 x = *(const float4*)src;
                            acc[0] += x.x; acc[1] += x.y; acc[2] += x.z; acc[3] += x.w;
                        } else {
                            acc[0] += *src;
                        }
                    }
                } else {
                    int rr, w;
                    const int u = pv_div_small(cell, RR, invRR, &rr);
                    const int v = pv_div_small(rr, R, invR, &w);
                    // the base cells (u - 1 .. u, v - 1 .. v, w - 1 .. w) in
                    // index order, whose points reach this cell through their
                    // corner 7 - t; their ranges loaded together
                    const int2* bc = bounds + b * V + ((u - 1) * R + (v - 1)) * R + (w - 1);
                    int2 rgs[8];
#pragma unroll
                    for (int t = 0; t < 8; t++) {
                        const bool in =
                            ((t & 4) || u > 0) && ((t & 2) || v > 0) && ((t & 1) || w > 0);
                        rgs[t] = in ? bc[(t >> 2) * RR + ((t >> 1) & 1) * R + (t & 1)]
                                    : make_int2(0, 0);
                    }
#pragma unroll
                    for (int t = 0; t < 8; t++) {
#pragma unroll 2
                        for (int sidx = rgs[t].x; sidx < rgs[t].y; sidx++) {
                            const float wt = rec_w[(size_t)sidx * 8 + (7 - t)];
                            const float* src = srow + (size_t)sidx * C + q * VW;
                            if constexpr (VW == 4) {
                                const float4 x = *(const float4*)src;
                                acc[0] += wt * x.x; acc[1] += wt * x.y;
                                acc[2] += wt * x.z; acc[3] += wt * x.w;
                            } else {
                                acc[0] += wt * *src;
                            }
                        }
                    }
                }
            }
            float* dst = dgrid + cg * C + q * VW;
            if constexpr (VW == 4)
                *(float4*)dst = make_float4(acc[0], acc[1], acc[2], acc[3]);
            else
                dst[0] = acc[0];
            j += dj;
            q += dq;
            if (q >= per) {
                q -= per;
                j++;
            }
        }
    }
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
// TAB: the folded BN scale of each channel is formed once per workgroup into
// LDS (pv_bn_coeffs, so the same bits as forming it per element); each
// thread keeps U groups of E elements in flight.
template <typename YT, bool V4, bool TAB>
__global__ __launch_bounds__(256) void pv_act_bn_backward_kernel(
    const float* dy, const YT* __restrict__ y, PvBnFold bn, float neg, float* dz, int C,
    size_t n) {
    extern __shared__ float s_scale[];  // TAB: [C]
    if constexpr (TAB) {
        for (int c = threadIdx.x; c < C; c += 256) {
            float scale, shift;
            pv_bn_coeffs(bn, c, scale, shift);
            s_scale[c] = scale;
        }
        __syncthreads();
    }
    constexpr int E = V4 ? 4 : 1, U = 4;
    const size_t step = (size_t)gridDim.x * 256 * E;
    for (size_t j0 = ((size_t)blockIdx.x * 256 + threadIdx.x) * E; j0 < n; j0 += step * U) {
        float yv[U][E], g[U][E];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const size_t j = j0 + u * step;
            if (j >= n) continue;
            if (V4) {
                load4<YT>(y + j, yv[u]);
                load4<float>(dy + j, g[u]);
            } else {
                yv[u][0] = load1<YT>(y + j);
                g[u][0] = dy[j];
            }
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            const size_t j = j0 + u * step;
            if (j >= n) continue;
            const int c = (int)(j % C);
#pragma unroll
            for (int e = 0; e < E; e++) {
                float scale, shift;
                if (TAB)
                    scale = s_scale[c + e];
                else
                    pv_bn_coeffs(bn, c + e, scale, shift);
                g[u][e] = g[u][e] * (yv[u][e] > 0.f ? 1.f : neg) * scale;
            }
            if (V4)
                *(float4*)(dz + j) = make_float4(g[u][0], g[u][1], g[u][2], g[u][3]);
            else
                dz[j] = g[u][0];
        }
    }
}

// ---------------------------------------------------------------------------
// Convolution weight gradient on the MFMA units:
//   dW[o][t][i] = sum over clouds b and output voxels p of dy[b][p][o] * x[b][p + d_t][i]
// an implicit GEMM with M = output channels, N = (tap, input channel) and
// K = voxels. A workgroup (four waves) owns 64 output channels x one chunk of
// CI (32, else 16) input channels x all 27 taps for a contiguous range of
// 8x8x8 bricks (a split of the voxel sum); each split writes its partial
// sums, and a second kernel adds the splits in split order. Per brick, both
// operands sit in LDS as they lie in memory, voxel-major with channels
// fastest:
//  * dy of the brick, [512 p][64 o] (128-byte rows; 64-byte halves swapped
//    where bit 1 of p is set, so that the four consecutive rows one
//    fragment read touches fall in distinct banks);
//  * x of the brick's 10x10x10 halo for the CI channels, [1000][CI i].
// The MFMA fragments need the transposes (8 consecutive voxels of one
// channel per lane). gfx950's transposing LDS read does that: each group of
// 16 lanes names 16 pieces of 4 channels (4 voxels x 4 pieces), and lane
// 4a + c receives channel 4a + c of the 4 voxels. Two such reads (voxels
// k0 .. k0+3, k0+4 .. k0+7) make one 8-voxel fragment, for A (dy) and for B
// (the halo shifted by the tap). A brick's global loads are issued together
// into registers while the previous brick's MFMAs run, then written to LDS
// with 16-byte stores.
// The GEMM's columns come in blocks of 32: block q holds TPB = 32 / CI taps,
// column n tap TPB q + n / CI, input channel n % CI (taps past 26 are
// padding: computed, never written). Every wave owns both 32-channel blocks
// of the 64 output channels and column blocks w, w + 4, w + 8, ... (CI 32:
// 7 blocks a wave, one padding tap in all; CI 16: 4 tap pairs, five).
// Voxels outside the grid (ragged bricks, the halo's border) read as zero.
constexpr int kWgO = 64;                              // output channels per workgroup
constexpr int kDyBytes = 512 * kWgO * 2;              // 65536
template <int CI>
struct WgShape {
    static constexpr int kXtBytes = 1000 * CI * 2;                // 32000 or 64000
    static constexpr int kLds = kDyBytes + kXtBytes;
    static constexpr int kPieces = 1000 * CI / 8;                 // 16-byte halo pieces
    static constexpr int kXtPer = (kPieces + 255) / 256;          // per thread: 8 or 16
    static constexpr int kTpb = 32 / CI;                          // taps per column block
    static constexpr int kBlocks = (27 + kTpb - 1) / kTpb;        // 14 or 27
    static constexpr int kQb = (kBlocks + 3) / 4;                 // per wave: 4 or 7
};

typedef short pv_i16x4 __attribute__((ext_vector_type(4)));

// byte offset of channels [c, c + 8) of voxel p in the dy tile (c % 8 == 0,
// or any channel offset within such a piece)
__device__ __forceinline__ int wg_dy_off(int p, int cbyte) { return p * 128 + (cbyte ^ ((p & 2) << 5)); }

// A brick's operands in registers, between their global loads and their LDS
// stores: dy of voxels tid and tid + 256 (64 channels each: consecutive
// lanes store consecutive rows), and halo pieces tid + 256 k (piece = voxel
// * CI / 8 + which 8 of its CI channels).
template <int CI>
struct WgradRegs {
    uint4 d0[8], d1[8];
    uint4 x[WgShape<CI>::kXtPer];
};

template <int CI>
__device__ __forceinline__ void wgrad_load(WgradRegs<CI>& g, const uint16_t* __restrict__ dy,
                                           const uint16_t* __restrict__ x, int brick, int nbr,
                                           int R, int Cin, int Cout, int o0, int i0) {
    const int tid = threadIdx.x;
    int rest = brick;
    const int bw = rest % nbr;
    rest /= nbr;
    const int bv = rest % nbr;
    rest /= nbr;
    const int bu = rest % nbr;
    const int b = rest / nbr;
    const int u0 = bu * 8, v0 = bv * 8, w0 = bw * 8;
    const size_t V = (size_t)R * R * R;
    const uint4 z = make_uint4(0, 0, 0, 0);
    // every load reads a voxel clamped into the grid; outside voxels are then
    // replaced by zero (no branches around the loads)
    auto cl = [R](int a) { return min(max(a, 0), R - 1); };
    auto sel = [&z](bool in, uint4 v) { return in ? v : z; };
    {
        // voxels p = tid and p + 256 = the same (v, w), u + 4
        const int p = tid, u = u0 + (p >> 6), v = v0 + ((p >> 3) & 7), w = w0 + (p & 7);
        const bool in0 = u < R && v < R && w < R, in1 = v < R && w < R && u + 4 < R;
        const uint16_t* dyb = dy + (size_t)b * V * Cout + o0;
        const uint16_t* r0 = dyb + (((size_t)cl(u) * R + cl(v)) * R + cl(w)) * Cout;
        const uint16_t* r1 = dyb + (((size_t)cl(u + 4) * R + cl(v)) * R + cl(w)) * Cout;
#pragma unroll
        for (int q = 0; q < 8; q++) {
            g.d0[q] = sel(in0, *(const uint4*)(r0 + 8 * q));
            g.d1[q] = sel(in1, *(const uint4*)(r1 + 8 * q));
        }
    }
    const uint16_t* xb = x + (size_t)b * V * Cin + i0;
    constexpr int PPV = CI / 8;  // pieces per halo voxel
#pragma unroll
    for (int k = 0; k < WgShape<CI>::kXtPer; k++) {
        const int piece = tid + 256 * k, h = piece / PPV, part = piece % PPV;
        const int hw = h % 10, hv = (h / 10) % 10, hu = h / 100;
        const int u = u0 + hu - 1, v = v0 + hv - 1, w = w0 + hw - 1;
        const bool in = piece < WgShape<CI>::kPieces && u >= 0 && u < R && v >= 0 && v < R &&
                        w >= 0 && w < R;
        g.x[k] = sel(in, *(const uint4*)(xb + (((size_t)cl(u) * R + cl(v)) * R + cl(w)) * Cin +
                                         8 * part));
    }
}

template <int CI>
__device__ __forceinline__ void wgrad_store(const WgradRegs<CI>& g, char* ldy, char* lxt) {
    const int tid = threadIdx.x;
#pragma unroll
    for (int q = 0; q < 8; q++) {
        *(uint4*)(ldy + wg_dy_off(tid, 16 * q)) = g.d0[q];
        *(uint4*)(ldy + wg_dy_off(tid + 256, 16 * q)) = g.d1[q];
    }
#pragma unroll
    for (int k = 0; k < WgShape<CI>::kXtPer; k++) {
        const int piece = tid + 256 * k;
        if (piece < WgShape<CI>::kPieces) *(uint4*)(lxt + piece * 16) = g.x[k];
    }
}

__device__ __forceinline__ pv_bf16x8 wg_frag(const char* lo, const char* hi) {
    const pv_i16x4 a = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (pv_i16x4 __attribute__((address_space(3)))*)lo);
    const pv_i16x4 c = __builtin_amdgcn_ds_read_tr16_b64_v4i16(
        (pv_i16x4 __attribute__((address_space(3)))*)hi);
    pv_bf16x8 r;
    r[0] = a[0]; r[1] = a[1]; r[2] = a[2]; r[3] = a[3];
    r[4] = c[0]; r[5] = c[1]; r[6] = c[2]; r[7] = c[3];
    return r;
}

template <int CI>
__global__ __launch_bounds__(256, 1) void pv_conv3d_wgrad_kernel(
    const uint16_t* __restrict__ dy, const uint16_t* __restrict__ x, float* __restrict__ part,
    int R, int Cin, int Cout, int nbr, int nbricks, int per_split) {
    using S = WgShape<CI>;
    constexpr int QB = S::kQb, TPB = S::kTpb;
    __shared__ __attribute__((aligned(16))) char lds[S::kLds];
    char* ldy = lds;
    char* lxt = lds + kDyBytes;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int r32 = lane & 31, khalf = lane >> 5;
    const int split = blockIdx.x, o0 = blockIdx.y * kWgO, i0 = blockIdx.z * CI;
    const int b0 = split * per_split, b1 = min(nbricks, b0 + per_split);

    pv_f32x16 acc[2][QB];
#pragma unroll
    for (int ob = 0; ob < 2; ob++)
#pragma unroll
        for (int qi = 0; qi < QB; qi++)
#pragma unroll
            for (int j = 0; j < 16; j++) acc[ob][qi][j] = 0.f;
    // As a source of the transposing reads, lane l names piece a = l % 4 of
    // voxel j = (l % 16) / 4 of its group g = l / 16: group g serves k-half
    // g / 2 and columns 16 (g % 2) .. +15 of its block (A: output channels;
    // B: CI 16, tap TPB q + g % 2, CI 32, channels 16 (g % 2) ..).
    const int grp = lane >> 4, sj = (lane >> 2) & 3, sa = lane & 3;
    const int gh = grp >> 1;  // k-half this lane serves as a source
    constexpr int XROW = CI * 2;  // bytes per halo voxel
    // B: the halo offset of this lane's source piece at (pu, pv, pw) =
    // (0, 0, sj), per column block: the tap's (du + 1, dv + 1, dw + 1)
    // shift; padding columns (tap >= 27) read tap 26
    int boff[QB];
#pragma unroll
    for (int qi = 0; qi < QB; qi++) {
        const int tap = min(26, TPB * (wave + 4 * qi) + (CI == 16 ? (grp & 1) : 0));
        const int du = tap / 9 - 1, dv = (tap / 3) % 3 - 1, dw = tap % 3 - 1;
        boff[qi] = (((du + 1) * 10 + (dv + 1)) * 10 + (dw + 1 + sj)) * XROW +
                   (CI == 16 ? 0 : (grp & 1) * 32) + sa * 8;
    }
    const int acol = (grp & 1) * 32 + sa * 8;  // A: byte offset of its 4 channels in a dy row

    // the next brick's operands load during the current brick's MFMAs
    WgradRegs<CI> g;
    if (b0 < b1) wgrad_load<CI>(g, dy, x, b0, nbr, R, Cin, Cout, o0, i0);
    for (int brick = b0; brick < b1; brick++) {
        wgrad_store<CI>(g, ldy, lxt);
        __syncthreads();
        if (brick + 1 < b1) wgrad_load<CI>(g, dy, x, brick + 1, nbr, R, Cin, Cout, o0, i0);
        // 32 k-steps of 16 voxels (two w-rows): k-half h is row r = 2 ks + h
        // (pu, pv) = (r >> 3, r & 7); the fragments of step ks + 1 are read
        // during the MFMAs of step ks
        pv_bf16x8 a[2][2], bfr[2][QB];
        auto frags = [&](int ks, int buf) {
            const int r = 2 * ks + gh, pu = r >> 3, pv = r & 7;
            const int p0 = r * 8 + sj;  // voxel of the first read (pw = sj), then + 4
#pragma unroll
            for (int ob = 0; ob < 2; ob++)
                a[buf][ob] = wg_frag(ldy + wg_dy_off(p0, ob * 64 + acol),
                                     ldy + wg_dy_off(p0 + 4, ob * 64 + acol));
            const int hoff = (pu * 10 + pv) * 10 * XROW;
#pragma unroll
            for (int qi = 0; qi < QB; qi++)
                bfr[buf][qi] = wg_frag(lxt + boff[qi] + hoff, lxt + boff[qi] + hoff + 4 * XROW);
        };
        frags(0, 0);
#pragma unroll
        for (int ks = 0; ks < 32; ks++) {
            const int cur = ks & 1;
            if (ks + 1 < 32) frags(ks + 1, cur ^ 1);
#pragma unroll
            for (int ob = 0; ob < 2; ob++)
#pragma unroll
                for (int qi = 0; qi < QB; qi++)
                    acc[ob][qi] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                        a[cur][ob], bfr[cur][qi], acc[ob][qi], 0, 0, 0);
        }
        __syncthreads();
    }
    // partial sums: rows o = 8 j + 4 khalf + e of each 32-channel block, column r32
    float* dst = part + (size_t)split * Cout * 27 * Cin;
#pragma unroll
    for (int qi = 0; qi < QB; qi++) {
        const int tap = TPB * (wave + 4 * qi) + r32 / CI, i = i0 + r32 % CI;
        if (tap >= 27) continue;
#pragma unroll
        for (int ob = 0; ob < 2; ob++)
#pragma unroll
            for (int j = 0; j < 16; j++) {
                const int o = o0 + ob * 32 + 8 * (j >> 2) + 4 * khalf + (j & 3);
                dst[((size_t)o * 27 + tap) * Cin + i] = acc[ob][qi][j];
            }
    }
}

// dW[j] = the sum of the splits' partials for element j, in split order.
__global__ __launch_bounds__(256) void pv_wgrad_reduce_kernel(const float* __restrict__ part,
                                                              float* __restrict__ dw, size_t n,
                                                              int nsplit) {
    for (size_t j = (size_t)blockIdx.x * 256 + threadIdx.x; j < n; j += (size_t)gridDim.x * 256) {
        float sum = 0.f;
        for (int s = 0; s < nsplit; s++) sum += part[(size_t)s * n + j];
        dw[j] = sum;
    }
}

// Splits of the voxel sum: enough workgroups for every CU, whole bricks each.
int wgrad_splits(int B, int R, int Cin, int Cout) {
    const int nbr = (R + 7) / 8;
    const int nbricks = B * nbr * nbr * nbr;
    const int tiles = (Cout / kWgO) * (Cin % 32 == 0 ? Cin / 32 : Cin / 16);
    const int want = (256 + tiles - 1) / tiles;
    return std::max(1, std::min(nbricks, want));
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

namespace {
struct DevoxBwdWs {
    uint32_t* key[2];
    int32_t* val[2];
    uint32_t* hist;  // [B][256][chunks per cloud]
    int2* bounds;    // [B * R^3]
    float4* rec_w;   // [B * N][2] their corner weights (trilinear)
    uint8_t* act;    // [B * R^3] cells some point reaches (rounded up to 4 bytes)
    float* srow;     // [B * N][C] gradient rows in sorted order
};

size_t devox_bwd_layout(int B, int N, int C, int R, char* base, DevoxBwdWs* ws) {
    const size_t E = (size_t)B * N, V = (size_t)R * R * R;
    const size_t nch = ((size_t)N + kSortChunk - 1) / kSortChunk;
    size_t off = 0;
    auto take = [&](size_t bytes) {
        char* p = base ? base + off : nullptr;
        off += pv_align256(bytes);
        return p;
    };
    for (int i = 0; i < 2; i++) {
        ws->key[i] = (uint32_t*)take(E * 4);
        ws->val[i] = (int32_t*)take(E * 4);
    }
    ws->hist = (uint32_t*)take((size_t)B * 256 * nch * 4);
    ws->bounds = (int2*)take((size_t)B * V * sizeof(int2));
    ws->rec_w = (float4*)take(E * 2 * sizeof(float4));
    ws->act = (uint8_t*)take(((size_t)B * V + 3) / 4 * 4);
    ws->srow = (float*)take(E * (size_t)C * 4);

    return off;
}
}  // namespace

size_t pv_devox_bwd_ws_bytes(int B, int N, int C, int R) {
    DevoxBwdWs ws;
    return devox_bwd_layout(B, N, C, R, nullptr, &ws);
}

pvconv_status pv_launch_devoxelize_backward(const float* dout, int B, int N, int C, int R,
                                            const float* pn, const int32_t* ids, float* dgrid,
                                            void* workspace, hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    const size_t V = (size_t)R * R * R;
    const size_t gn = (size_t)B * V * C;
    if (N == 0) {
        hipLaunchKernelGGL(pv_fill_zero_kernel, dim3(fill_blocks(gn)), dim3(256), 0, s, dgrid, gn);
        return pv_launch_status();
    }
    DevoxBwdWs ws;
    devox_bwd_layout(B, N, C, R, (char*)workspace, &ws);
    const size_t E = (size_t)B * N;
    const int nch = (N + kSortChunk - 1) / kSortChunk;
    const size_t ncells = (size_t)B * V;
    const unsigned kb = (unsigned)std::min<size_t>((std::max(E, ncells) + 255) / 256, 4096);
    hipLaunchKernelGGL(pv_devox_bwd_keys_kernel, dim3(kb), dim3(256), 0, s, pn, ids, R, E, ncells,
                       ws.key[0], ws.val[0], ws.bounds, (uint32_t*)ws.act);
    // one pass per 8-bit digit of the largest cell index
    int cur = 0;
    for (int shift = 0; shift == 0 || ((V - 1) >> shift) != 0; shift += 8) {
        hipLaunchKernelGGL(pv_radix_hist_kernel, dim3(B * nch), dim3(64), 0, s, ws.key[cur], N, nch,
                           shift, ws.hist);
        hipLaunchKernelGGL(pv_radix_scan_kernel, dim3(B), dim3(256), 0, s, ws.hist, N, nch);
        hipLaunchKernelGGL(pv_radix_scatter_kernel, dim3(B * nch), dim3(64), 0, s, ws.key[cur],
                           ws.val[cur], ws.key[cur ^ 1], ws.val[cur ^ 1], ws.hist, N, nch, shift);
        cur ^= 1;
    }
    hipLaunchKernelGGL(pv_devox_bwd_bounds_kernel, dim3(std::min<size_t>(blocks_for(E), 4096)),
                       dim3(256), 0, s, ws.key[cur], ws.val[cur], ids ? nullptr : pn, N, E, R,
                       ws.bounds, ws.rec_w, ws.act);
    const bool vec = C % 4 == 0 && ((uintptr_t)dout & 15) == 0 && ((uintptr_t)dgrid & 15) == 0;
    const size_t rows = E * (size_t)(vec ? C / 4 : C);
    const unsigned rb = (unsigned)std::min<size_t>((rows + 255) / 256, 8192);
    if (vec)
        hipLaunchKernelGGL(pv_devox_bwd_rows_kernel<4>, dim3(rb), dim3(256), 0, s, dout,
                           ws.val[cur], C, rows, ws.srow);
    else
        hipLaunchKernelGGL(pv_devox_bwd_rows_kernel<1>, dim3(rb), dim3(256), 0, s, dout,
                           ws.val[cur], C, rows, ws.srow);
    const unsigned gb = (unsigned)std::min<size_t>((ncells + 63) / 64, (size_t)1 << 20);
#define PV_DEVOX_BWD(VW, NEAR)                                                                   \
    hipLaunchKernelGGL((pv_devox_bwd_gather_kernel<VW, NEAR>), dim3(gb), dim3(256), 0, s, ws.srow, \
                       (const float*)ws.rec_w, ws.bounds, ws.act, ncells, R, C, dgrid)
    if (vec) {
        if (ids) PV_DEVOX_BWD(4, true);
        else PV_DEVOX_BWD(4, false);
    } else {
        if (ids) PV_DEVOX_BWD(1, true);
        else PV_DEVOX_BWD(1, false);
    }
#undef PV_DEVOX_BWD
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
    // the scale table takes C floats of LDS (up to 64 KB)
    const bool tab = C <= 16384;
    auto go = [&](auto yt, auto v4t) {
        typedef decltype(yt) YT;
        if (tab)
            hipLaunchKernelGGL((pv_act_bn_backward_kernel<YT, decltype(v4t)::value, true>),
                               dim3(blocks), dim3(256), (size_t)C * sizeof(float), s, dy,
                               (const YT*)y, bn, neg, dz, C, n);
        else
            hipLaunchKernelGGL((pv_act_bn_backward_kernel<YT, decltype(v4t)::value, false>),
                               dim3(blocks), dim3(256), 0, s, dy, (const YT*)y, bn, neg, dz, C, n);
    };
    if (y_bf16) {
        if (v4) go(uint16_t{}, std::true_type{}); else go(uint16_t{}, std::false_type{});
    } else {
        if (v4) go(float{}, std::true_type{}); else go(float{}, std::false_type{});
    }
    return pv_launch_status();
}

size_t pv_conv3d_wgrad_ws_bytes(int B, int R, int Cin, int Cout) {
    return (size_t)wgrad_splits(B, R, Cin, Cout) * Cout * 27 * Cin * sizeof(float);
}

pvconv_status pv_launch_conv3d_backward_weight(const void* dy, const void* x, int B, int R,
                                               int Cin, int Cout, float* dw, void* ws,
                                               hipStream_t s) {
    const size_t n = (size_t)Cout * 27 * Cin;
    if (B == 0) {
        hipLaunchKernelGGL(pv_fill_zero_kernel, dim3(fill_blocks(n)), dim3(256), 0, s, dw, n);
        return pv_launch_status();
    }
    const int nbr = (R + 7) / 8, nbricks = B * nbr * nbr * nbr;
    const int nsplit = wgrad_splits(B, R, Cin, Cout);
    const int per = (nbricks + nsplit - 1) / nsplit;
    const int used = (nbricks + per - 1) / per;  // splits that hold at least one brick
    float* part = (float*)ws;
    if (Cin % 32 == 0)
        hipLaunchKernelGGL(pv_conv3d_wgrad_kernel<32>, dim3(used, Cout / kWgO, Cin / 32), dim3(256),
                           0, s, (const uint16_t*)dy, (const uint16_t*)x, part, R, Cin, Cout, nbr,
                           nbricks, per);
    else
        hipLaunchKernelGGL(pv_conv3d_wgrad_kernel<16>, dim3(used, Cout / kWgO, Cin / 16), dim3(256),
                           0, s, (const uint16_t*)dy, (const uint16_t*)x, part, R, Cin, Cout, nbr,
                           nbricks, per);
    const unsigned blocks = (unsigned)std::min<size_t>((n + 255) / 256, 2048);
    hipLaunchKernelGGL(pv_wgrad_reduce_kernel, dim3(blocks), dim3(256), 0, s, part, dw, n, used);
    return pv_launch_status();
}
