// Normalisation and voxelisation (Section 4.1 "Normalization", "Voxelization",
// Eq. 2) for gfx950.
//
// Data flow for one call (B clouds, N points, grid R^3, C channels):
//   1. normalise: per-cloud centroid (int64 fixed point, order-free), largest
//      centred norm, normalised coordinates and voxel ids.
//   2. bucket: per cloud, an LDS histogram over (a partition of) the voxels,
//      written out as `counts`, scanned, and used to scatter point indices
//      into a list sorted by voxel; each 256-voxel tile records its slice.
//   3. fill: one workgroup per 256-voxel tile writes the tile's whole slice
//      of the dense grid once, coalesced: the mean of the voxel's features
//      (fp64 sums) or zeros.
// Small problems (R^3 <= 32768 and N <= 16384) fuse 1 and 2 into a single
// workgroup per cloud; larger ones split normalisation over many workgroups
// (four short launches that pass partial results through the workspace) and
// bucket one 32768-voxel partition per workgroup.
#include "pv_common.h"

namespace {

constexpr int kPart = 32768;        // voxels per LDS histogram (128 KiB of int32)
constexpr int kTile = 256;          // voxels per fill workgroup
constexpr int kSmallMaxN = 16384;   // largest N for the fused per-cloud path
constexpr int kNormPts = 2048;      // points per workgroup, split normalisation
constexpr int kNormThreads = 256;

// ---------------------------------------------------------------------------
// Normalisation arithmetic. IEEE fp64, round to nearest even, no contraction,
// so that voxel ids are reproducible bit for bit.
// ---------------------------------------------------------------------------
__device__ __forceinline__ int ceil_log2_i(int n) { return n <= 1 ? 0 : 32 - __clz(n - 1); }

// Fixed-point scale for one axis from the largest |coordinate| A > 0:
// with A = f * 2^e, f in [1/2, 1), S = 62 - ceil(log2 N) - e keeps every
// partial sum of llrint(x * 2^S) below 2^62 in magnitude.
__device__ __forceinline__ int fixed_scale(float A, int N) {
    if (!(A > 0.f)) return 0;
    unsigned long long bits = (unsigned long long)__double_as_longlong((double)A);
    int e = (int)((bits >> 52) & 0x7ffull) - 1022;
    return 62 - ceil_log2_i(N) - e;
}

__device__ __forceinline__ long long fixed_term(float x, int S) {
    return (long long)rint(ldexp((double)x, S));
}

__device__ __forceinline__ double centroid_from_sum(long long q, int S, float A, int N) {
#pragma clang fp contract(off)
    if (!(A > 0.f)) return 0.0;
    return ldexp((double)q / (double)N, -S);
}

__device__ __forceinline__ double sq_dist(const float* p, const double* c) {
#pragma clang fp contract(off)
    double dx = (double)p[0] - c[0];
    double dy = (double)p[1] - c[1];
    double dz = (double)p[2] - c[2];
    return (dx * dx + dy * dy) + dz * dz;
}

__device__ __forceinline__ int voxel_axis(double x, int R) {
#pragma clang fp contract(off)
    double f = floor(x * (double)R);
    f = fmin(fmax(f, 0.0), (double)(R - 1));  // also maps NaN to 0
    return (int)f;
}

// Normalised coordinates of one point and its voxel id.
__device__ __forceinline__ int normalise_point(const float* p, const double* c, double M2,
                                               double m, int R, float* pn_out) {
#pragma clang fp contract(off)
    int uvw[3];
    for (int a = 0; a < 3; a++) {
        double d = (double)p[a] - c[a];
        double unit = (M2 == 0.0) ? 0.0 : d / m;
        double x = unit * 0.5 + 0.5;
        if (pn_out) pn_out[a] = (float)x;
        uvw[a] = voxel_axis(x, R);
    }
    return (uvw[0] * R + uvw[1]) * R + uvw[2];
}

// ---------------------------------------------------------------------------
// Workgroup reductions and scans (wave64).
// ---------------------------------------------------------------------------
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
    for (int o = 32; o > 0; o >>= 1) v = op(v, __shfl_xor(v, o, 64));
    return v;
}

template <int NT, typename T, typename Op>
__device__ T block_reduce(T v, Op op, T* lds /* NT/64 entries */) {
    v = wave_reduce(v, op);
    const int w = threadIdx.x >> 6;
    __syncthreads();
    if ((threadIdx.x & 63) == 0) lds[w] = v;
    __syncthreads();
    T r = lds[0];
    for (int i = 1; i < NT / 64; i++) r = op(r, lds[i]);
    return r;
}

struct MaxF { __device__ float operator()(float a, float b) const { return fmaxf(a, b); } };
struct MaxD { __device__ double operator()(double a, double b) const { return fmax(a, b); } };
struct AddL {
    __device__ long long operator()(long long a, long long b) const { return a + b; }
};

// Exclusive scan of one int per thread over the workgroup; also returns the total.
template <int NT>
__device__ int block_exclusive_scan(int v, int* lds /* NT/64 */, int& total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int incl = v;
    for (int o = 1; o < 64; o <<= 1) {
        int t = __shfl_up(incl, o, 64);
        if (lane >= o) incl += t;
    }
    __syncthreads();
    if (lane == 63) lds[w] = incl;
    __syncthreads();
    int before = 0;
    total = 0;
    for (int i = 0; i < NT / 64; i++) {
        int s = lds[i];
        if (i < w) before += s;
        total += s;
    }
    return before + incl - v;
}

// Per-cloud normalisation parameters, computed by one workgroup of NT threads
// over all N points of the cloud.
template <int NT>
__device__ void cloud_params(const float* p, int N, double* c, double& M2, double& m,
                             float* redf, long long* redl, double* redd) {
    float A[3] = {0.f, 0.f, 0.f};
    for (int k = threadIdx.x; k < N; k += NT)
        for (int a = 0; a < 3; a++) A[a] = fmaxf(A[a], fabsf(p[3 * k + a]));
    int S[3];
    for (int a = 0; a < 3; a++) {
        A[a] = block_reduce<NT>(A[a], MaxF(), redf);
        S[a] = fixed_scale(A[a], N);
    }
    long long q[3] = {0, 0, 0};
    for (int k = threadIdx.x; k < N; k += NT)
        for (int a = 0; a < 3; a++)
            if (A[a] > 0.f) q[a] += fixed_term(p[3 * k + a], S[a]);
    for (int a = 0; a < 3; a++) {
        q[a] = block_reduce<NT>(q[a], AddL(), redl);
        c[a] = centroid_from_sum(q[a], S[a], A[a], N);
    }
    double mx = 0.0;
    for (int k = threadIdx.x; k < N; k += NT) mx = fmax(mx, sq_dist(p + 3 * k, c));
    M2 = block_reduce<NT>(mx, MaxD(), redd);
    m = sqrt(M2);
}

// Histogram scan + tile ranges + scatter, shared by the two bucket kernels.
// hist[0..nv) holds the counts of voxels [v_begin, v_begin + nv) on entry.
template <int NT>
__device__ void scan_and_ranges(int* hist, int nv, int v_begin, int* scan_lds, int2* tile_range,
                                int tile_first) {
    const int seg = (nv + NT - 1) / NT;
    const int s0 = min(nv, (int)threadIdx.x * seg), s1 = min(nv, s0 + seg);
    int local = 0;
    for (int i = s0; i < s1; i++) local += hist[i];
    int total;
    int run = block_exclusive_scan<NT>(local, scan_lds, total);
    for (int i = s0; i < s1; i++) {
        int h = hist[i];
        hist[i] = run;
        run += h;
    }
    __syncthreads();
    const int ntiles = (nv + kTile - 1) / kTile;
    for (int t = threadIdx.x; t < ntiles; t += NT) {
        int lo = hist[t * kTile];
        int hi = (t + 1) * kTile < nv ? hist[(t + 1) * kTile] : total;
        tile_range[tile_first + t] = make_int2(lo, hi);
    }
    __syncthreads();
    (void)v_begin;
}

// ---------------------------------------------------------------------------
// Fused path: one workgroup per cloud does normalisation and bucketing.
// ---------------------------------------------------------------------------
__global__ __launch_bounds__(1024) void pv_voxelize_bucket_small_kernel(
    const float* __restrict__ coords, int N, int R, int32_t* __restrict__ vox_id,
    float* __restrict__ norm_coords, int32_t* __restrict__ counts, int32_t* __restrict__ list,
    int2* __restrict__ tile_range) {
    constexpr int NT = 1024;
    __shared__ int hist[kPart];
    __shared__ float redf[NT / 64];
    __shared__ long long redl[NT / 64];
    __shared__ double redd[NT / 64];
    __shared__ int scan_lds[NT / 64];

    const int b = blockIdx.x;
    const int V = R * R * R;
    const int tiles = (V + kTile - 1) / kTile;
    const float* p = coords + (size_t)b * N * 3;
    for (int i = threadIdx.x; i < V; i += NT) hist[i] = 0;

    double c[3], M2, m;
    cloud_params<NT>(p, N, c, M2, m, redf, redl, redd);

    int32_t* ids = vox_id + (size_t)b * N;
    for (int k = threadIdx.x; k < N; k += NT) {
        float pn[3];
        int id = normalise_point(p + 3 * k, c, M2, m, R, pn);
        if (norm_coords) {
            float* o = norm_coords + ((size_t)b * N + k) * 3;
            o[0] = pn[0];
            o[1] = pn[1];
            o[2] = pn[2];
        }
        ids[k] = id;
        atomicAdd(&hist[id], 1);
    }
    __syncthreads();
    int32_t* cnt = counts + (size_t)b * V;
    for (int i = threadIdx.x; i < V; i += NT) cnt[i] = hist[i];
    __syncthreads();
    scan_and_ranges<NT>(hist, V, 0, scan_lds, tile_range, b * tiles);
    int32_t* lst = list + (size_t)b * N;
    for (int k = threadIdx.x; k < N; k += NT) {  // same points as above: own writes
        int pos = atomicAdd(&hist[ids[k]], 1);
        lst[pos] = k;
    }
}

// ---------------------------------------------------------------------------
// Split path. Partial results per (cloud, workgroup g) pass between launches:
//   pA [B][G][3] float, pQ [B][G][3] int64, pM [B][G] double.
// ---------------------------------------------------------------------------
struct SplitWs {
    float* pA;
    long long* pQ;
    double* pM;
    int G;
};

__global__ __launch_bounds__(kNormThreads) void pv_norm_absmax_kernel(const float* coords, int N,
                                                                      SplitWs ws) {
    __shared__ float redf[kNormThreads / 64];
    const int g = blockIdx.x, b = blockIdx.y;
    const float* p = coords + (size_t)b * N * 3;
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    float A[3] = {0.f, 0.f, 0.f};
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads)
        for (int a = 0; a < 3; a++) A[a] = fmaxf(A[a], fabsf(p[3 * k + a]));
    for (int a = 0; a < 3; a++) {
        float r = block_reduce<kNormThreads>(A[a], MaxF(), redf);
        if (threadIdx.x == 0) ws.pA[((size_t)b * ws.G + g) * 3 + a] = r;
    }
}

// Reduce the G partials of cloud b (every workgroup does it; G is small).
__device__ void split_absmax(const SplitWs& ws, int b, float* A) {
    for (int a = 0; a < 3; a++) {
        float r = 0.f;
        for (int g = 0; g < ws.G; g++) r = fmaxf(r, ws.pA[((size_t)b * ws.G + g) * 3 + a]);
        A[a] = r;
    }
}

__device__ void split_centroid(const SplitWs& ws, int b, int N, double* c) {
    float A[3];
    split_absmax(ws, b, A);
    for (int a = 0; a < 3; a++) {
        long long q = 0;
        for (int g = 0; g < ws.G; g++) q += ws.pQ[((size_t)b * ws.G + g) * 3 + a];
        c[a] = centroid_from_sum(q, fixed_scale(A[a], N), A[a], N);
    }
}

__global__ __launch_bounds__(kNormThreads) void pv_norm_sum_kernel(const float* coords, int N,
                                                                   SplitWs ws) {
    __shared__ long long redl[kNormThreads / 64];
    const int g = blockIdx.x, b = blockIdx.y;
    const float* p = coords + (size_t)b * N * 3;
    float A[3];
    split_absmax(ws, b, A);
    int S[3];
    for (int a = 0; a < 3; a++) S[a] = fixed_scale(A[a], N);
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    long long q[3] = {0, 0, 0};
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads)
        for (int a = 0; a < 3; a++)
            if (A[a] > 0.f) q[a] += fixed_term(p[3 * k + a], S[a]);
    for (int a = 0; a < 3; a++) {
        long long r = block_reduce<kNormThreads>(q[a], AddL(), redl);
        if (threadIdx.x == 0) ws.pQ[((size_t)b * ws.G + g) * 3 + a] = r;
    }
}

__global__ __launch_bounds__(kNormThreads) void pv_norm_radius_kernel(const float* coords, int N,
                                                                      SplitWs ws) {
    __shared__ double redd[kNormThreads / 64];
    const int g = blockIdx.x, b = blockIdx.y;
    const float* p = coords + (size_t)b * N * 3;
    double c[3];
    split_centroid(ws, b, N, c);
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    double mx = 0.0;
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads) mx = fmax(mx, sq_dist(p + 3 * k, c));
    double r = block_reduce<kNormThreads>(mx, MaxD(), redd);
    if (threadIdx.x == 0) ws.pM[(size_t)b * ws.G + g] = r;
}

__global__ __launch_bounds__(kNormThreads) void pv_norm_points_kernel(
    const float* coords, int N, int R, SplitWs ws, int32_t* __restrict__ vox_id,
    float* __restrict__ norm_coords) {
    const int g = blockIdx.x, b = blockIdx.y;
    const float* p = coords + (size_t)b * N * 3;
    double c[3];
    split_centroid(ws, b, N, c);
    double M2 = 0.0;
    for (int i = 0; i < ws.G; i++) M2 = fmax(M2, ws.pM[(size_t)b * ws.G + i]);
    const double m = sqrt(M2);
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads) {
        float pn[3];
        int id = normalise_point(p + 3 * k, c, M2, m, R, pn);
        if (norm_coords) {
            float* o = norm_coords + ((size_t)b * N + k) * 3;
            o[0] = pn[0];
            o[1] = pn[1];
            o[2] = pn[2];
        }
        vox_id[(size_t)b * N + k] = id;
    }
}

// One workgroup per (partition p, cloud b): histogram of the points whose voxel
// lies in [p*kPart, p*kPart + nv), counts out, scan, tile ranges, scatter into
// the partition's own list region list[(b*P + p)*N ...].
__global__ __launch_bounds__(1024) void pv_bucket_partition_kernel(
    const int32_t* __restrict__ vox_id, int N, int R, int P, int32_t* __restrict__ counts,
    int32_t* __restrict__ list, int2* __restrict__ tile_range) {
    constexpr int NT = 1024;
    __shared__ int hist[kPart];
    __shared__ int scan_lds[NT / 64];
    const int p = blockIdx.x, b = blockIdx.y;
    const int V = R * R * R;
    const int tiles = (V + kTile - 1) / kTile;
    const int v0 = p * kPart, nv = min(kPart, V - v0);
    for (int i = threadIdx.x; i < nv; i += NT) hist[i] = 0;
    __syncthreads();
    const int32_t* ids = vox_id + (size_t)b * N;
    for (int k = threadIdx.x; k < N; k += NT) {
        int r = ids[k] - v0;
        if (r >= 0 && r < nv) atomicAdd(&hist[r], 1);
    }
    __syncthreads();
    int32_t* cnt = counts + (size_t)b * V + v0;
    for (int i = threadIdx.x; i < nv; i += NT) cnt[i] = hist[i];
    __syncthreads();
    scan_and_ranges<NT>(hist, nv, v0, scan_lds, tile_range, b * tiles + v0 / kTile);
    int32_t* lst = list + ((size_t)b * P + p) * N;
    for (int k = threadIdx.x; k < N; k += NT) {
        int r = ids[k] - v0;
        if (r >= 0 && r < nv) lst[atomicAdd(&hist[r], 1)] = k;
    }
}

// ---------------------------------------------------------------------------
// Fill: one workgroup per 256-voxel tile writes the tile's grid rows once.
// ---------------------------------------------------------------------------
template <typename FT>
__device__ __forceinline__ void load8(const FT* src, double* acc);
template <>
__device__ __forceinline__ void load8<float>(const float* src, double* acc) {
    float4 a = *(const float4*)src, b = *(const float4*)(src + 4);
    acc[0] += a.x; acc[1] += a.y; acc[2] += a.z; acc[3] += a.w;
    acc[4] += b.x; acc[5] += b.y; acc[6] += b.z; acc[7] += b.w;
}
template <>
__device__ __forceinline__ void load8<uint16_t>(const uint16_t* src, double* acc) {
    uint4 a = *(const uint4*)src;
    uint32_t w[4] = {a.x, a.y, a.z, a.w};
    for (int i = 0; i < 4; i++) {
        acc[2 * i] += pv_bf16_to_f32((uint16_t)(w[i] & 0xffffu));
        acc[2 * i + 1] += pv_bf16_to_f32((uint16_t)(w[i] >> 16));
    }
}
template <typename GT>
__device__ __forceinline__ void store8(GT* dst, const float* v);
template <>
__device__ __forceinline__ void store8<float>(float* dst, const float* v) {
    *(float4*)dst = make_float4(v[0], v[1], v[2], v[3]);
    *(float4*)(dst + 4) = make_float4(v[4], v[5], v[6], v[7]);
}
template <>
__device__ __forceinline__ void store8<uint16_t>(uint16_t* dst, const float* v) {
    *(uint4*)dst = make_uint4(pv_pack_bf16x2(v[0], v[1]), pv_pack_bf16x2(v[2], v[3]),
                              pv_pack_bf16x2(v[4], v[5]), pv_pack_bf16x2(v[6], v[7]));
}

template <typename FT>
__device__ __forceinline__ float load1(const FT* p);
template <>
__device__ __forceinline__ float load1<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float load1<uint16_t>(const uint16_t* p) { return pv_bf16_to_f32(*p); }
template <typename GT>
__device__ __forceinline__ void store1(GT* p, float v);
template <>
__device__ __forceinline__ void store1<float>(float* p, float v) { *p = v; }
template <>
__device__ __forceinline__ void store1<uint16_t>(uint16_t* p, float v) { *p = pv_f32_to_bf16(v); }

template <typename FT, typename GT, bool VEC>
__global__ __launch_bounds__(256) void pv_voxel_fill_kernel(
    const FT* __restrict__ feats, int feat_ld, int N, int C, int R, int P,
    const int32_t* __restrict__ counts, const int32_t* __restrict__ list,
    const int2* __restrict__ tile_range, GT* __restrict__ grid) {
    constexpr int NT = 256;
    __shared__ int cnt[kTile];
    __shared__ int off[kTile];
    __shared__ int scan_lds[NT / 64];
    const int t = blockIdx.x, b = blockIdx.y;
    const int V = R * R * R;
    const int tiles = (V + kTile - 1) / kTile;
    const int v0 = t * kTile, nv = min(kTile, V - v0);
    const int2 rg = tile_range[(size_t)b * tiles + t];
    GT* out = grid + ((size_t)b * V + v0) * C;

    if (rg.x == rg.y) {  // no point in this tile: zeros only
        if (VEC) {
            const int chunks = nv * C * (int)sizeof(GT) / 16;
            uint4* o = (uint4*)out;
            for (int i = threadIdx.x; i < chunks; i += NT) o[i] = make_uint4(0, 0, 0, 0);
        } else {
            for (int i = threadIdx.x; i < nv * C; i += NT) out[i] = (GT)0;
        }
        return;
    }
    int n = threadIdx.x < nv ? counts[(size_t)b * V + v0 + threadIdx.x] : 0;
    int total;
    int ex = block_exclusive_scan<NT>(n, scan_lds, total);
    cnt[threadIdx.x] = n;
    off[threadIdx.x] = rg.x + ex;
    __syncthreads();

    const int p = v0 / kPart;
    const int32_t* lst = list + ((size_t)b * P + p) * N;
    const FT* fb = feats + (size_t)b * N * feat_ld;
    if (VEC) {
        const int gpv = C / 8;  // 8-channel groups per voxel
        for (int item = threadIdx.x; item < nv * gpv; item += NT) {
            const int vi = item / gpv, cg = item - vi * gpv;
            const int nk = cnt[vi];
            float mean[8];
            if (nk == 0) {
                for (int i = 0; i < 8; i++) mean[i] = 0.f;
            } else {
                double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                const int j0 = off[vi];
                for (int j = j0; j < j0 + nk; j++)
                    load8<FT>(fb + (size_t)lst[j] * feat_ld + cg * 8, acc);
                for (int i = 0; i < 8; i++) mean[i] = (float)(acc[i] / (double)nk);
            }
            store8<GT>(out + (size_t)vi * C + cg * 8, mean);
        }
    } else {
        for (int item = threadIdx.x; item < nv * C; item += NT) {
            const int vi = item / C, c = item - vi * C;
            const int nk = cnt[vi];
            float mean = 0.f;
            if (nk > 0) {
                double acc = 0.0;
                const int j0 = off[vi];
                for (int j = j0; j < j0 + nk; j++)
                    acc += (double)load1<FT>(fb + (size_t)lst[j] * feat_ld + c);
                mean = (float)(acc / (double)nk);
            }
            store1<GT>(out + (size_t)vi * C + c, mean);
        }
    }
}

template <typename FT, typename GT>
void launch_fill(const void* feats, int feat_ld, int B, int N, int C, int R, int P,
                 const int32_t* counts, const int32_t* list, const int2* tr, void* grid,
                 bool vec, hipStream_t s) {
    const int V = R * R * R;
    dim3 g((V + kTile - 1) / kTile, B);
    if (vec)
        hipLaunchKernelGGL((pv_voxel_fill_kernel<FT, GT, true>), g, dim3(256), 0, s,
                           (const FT*)feats, feat_ld, N, C, R, P, counts, list, tr, (GT*)grid);
    else
        hipLaunchKernelGGL((pv_voxel_fill_kernel<FT, GT, false>), g, dim3(256), 0, s,
                           (const FT*)feats, feat_ld, N, C, R, P, counts, list, tr, (GT*)grid);
}

struct VoxWs {
    int32_t* list;
    int2* tile_range;
    int32_t* ids;
    SplitWs split;
};

VoxWs carve_ws(void* ws, int B, int N, int R) {
    const int V = R * R * R;
    const int P = (V + kPart - 1) / kPart;
    const int tiles = (V + kTile - 1) / kTile;
    const int G = (N + kNormPts - 1) / kNormPts;
    char* p = (char*)ws;
    VoxWs w;
    w.list = (int32_t*)p;
    p += pv_align256((size_t)B * P * N * sizeof(int32_t));
    w.tile_range = (int2*)p;
    p += pv_align256((size_t)B * tiles * sizeof(int2));
    w.ids = (int32_t*)p;
    p += pv_align256((size_t)B * N * sizeof(int32_t));
    w.split.G = G;
    w.split.pA = (float*)p;
    p += pv_align256((size_t)B * G * 3 * sizeof(float));
    w.split.pQ = (long long*)p;
    p += pv_align256((size_t)B * G * 3 * sizeof(long long));
    w.split.pM = (double*)p;
    return w;
}

}  // namespace

size_t pv_voxelize_ws_bytes(int B, int N, int R) {
    const int V = R * R * R;
    const int P = (V + kPart - 1) / kPart;
    const int tiles = (V + kTile - 1) / kTile;
    const int G = (N + kNormPts - 1) / kNormPts;
    return pv_align256((size_t)B * P * N * sizeof(int32_t)) +
           pv_align256((size_t)B * tiles * sizeof(int2)) +
           pv_align256((size_t)B * N * sizeof(int32_t)) +
           pv_align256((size_t)B * G * 3 * sizeof(float)) +
           pv_align256((size_t)B * G * 3 * sizeof(long long)) +
           pv_align256((size_t)B * G * sizeof(double));
}

pvconv_status pv_launch_voxelize(const float* coords, const void* feats, bool feat_bf16,
                                 int feat_ld, int B, int N, int C, int R, void* grid,
                                 bool grid_bf16, int32_t* counts, int32_t* vox_id,
                                 float* norm_coords, void* ws, hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    const int V = R * R * R;
    const int P = (V + kPart - 1) / kPart;
    VoxWs w = carve_ws(ws, B, N, R);
    int32_t* ids = vox_id ? vox_id : w.ids;
    if (N > 0) {
        if (V <= kPart && N <= kSmallMaxN) {
            hipLaunchKernelGGL(pv_voxelize_bucket_small_kernel, dim3(B), dim3(1024), 0, s, coords,
                               N, R, ids, norm_coords, counts, w.list, w.tile_range);
        } else {
            dim3 g(w.split.G, B);
            hipLaunchKernelGGL(pv_norm_absmax_kernel, g, dim3(kNormThreads), 0, s, coords, N,
                               w.split);
            hipLaunchKernelGGL(pv_norm_sum_kernel, g, dim3(kNormThreads), 0, s, coords, N,
                               w.split);
            hipLaunchKernelGGL(pv_norm_radius_kernel, g, dim3(kNormThreads), 0, s, coords, N,
                               w.split);
            hipLaunchKernelGGL(pv_norm_points_kernel, g, dim3(kNormThreads), 0, s, coords, N, R,
                               w.split, ids, norm_coords);
            hipLaunchKernelGGL(pv_bucket_partition_kernel, dim3(P, B), dim3(1024), 0, s, ids, N,
                               R, P, counts, w.list, w.tile_range);
        }
    } else {
        // No points: every tile is empty. The fill kernel writes zeros; counts
        // are zeroed here with the same kind of plain store kernel.
        hipLaunchKernelGGL(pv_bucket_partition_kernel, dim3(P, B), dim3(1024), 0, s, ids, 0, R,
                           P, counts, w.list, w.tile_range);
    }
    const size_t esz_f = feat_bf16 ? 2 : 4, esz_g = grid_bf16 ? 2 : 4;
    const bool vec = (C % 8 == 0) && pv_aligned16(feats) && pv_aligned16(grid) &&
                     ((size_t)feat_ld * esz_f) % 16 == 0 && ((size_t)C * esz_g) % 16 == 0;
    if (feat_bf16) {
        if (grid_bf16)
            launch_fill<uint16_t, uint16_t>(feats, feat_ld, B, N, C, R, P, counts, w.list,
                                            w.tile_range, grid, vec, s);
        else
            launch_fill<uint16_t, float>(feats, feat_ld, B, N, C, R, P, counts, w.list,
                                         w.tile_range, grid, vec, s);
    } else {
        if (grid_bf16)
            launch_fill<float, uint16_t>(feats, feat_ld, B, N, C, R, P, counts, w.list,
                                         w.tile_range, grid, vec, s);
        else
            launch_fill<float, float>(feats, feat_ld, B, N, C, R, P, counts, w.list,
                                      w.tile_range, grid, vec, s);
    }
    return pv_launch_status();
}
