// Normalisation and voxelisation (Section 4.1 "Normalization", "Voxelization",
// Eq. 2) for gfx950.
//
// Data flow for one call (B clouds, N points, grid R^3, C channels):
//   1. normalise: per-cloud centroid (int64 fixed point, order-free), largest
//      centred norm, then every point's normalised coordinates and voxel id.
//      Clouds of up to 4096 points: one kernel, whose 256-point slices each
//      recompute the cloud's parameters from registers. Larger clouds: four
//      short kernels (abs-max, fixed-point sum, radius, points) that pass
//      per-workgroup partial results through the workspace.
//   2. tile fill: one workgroup per (cloud, tile of TV voxels) collects the
//      points that fall in its tile, counting-sorts them by voxel in LDS,
//      writes the tile's counts, zero rows for its empty voxels and, for the
//      occupied ones, the mean of their features (fp64 sums). Voxels holding
//      many points are summed by a whole wave with the points split across
//      lanes, so a heavily collided cloud costs a few extra rounds of loads.
//      Barriers order LDS only, so the grid rows stream out while the
//      workgroup works on.
// No global atomics; with 16-byte grid rows every grid element is written
// once. Otherwise the normalisation launch first zeroes the grid (extra
// workgroups) and the tile fill overwrites the occupied rows.
#include <algorithm>
#include <mutex>
#include <unordered_map>

#include "pv_common.h"

namespace {

constexpr int kNormPts = 1024;      // points per workgroup, large-cloud normalisation
constexpr int kNormThreads = 256;
constexpr int kSmallMaxN = 4096;    // largest cloud normalised by one kernel
constexpr int kHeavy = 32;          // voxels with more points are summed by a whole wave
constexpr int kExport = 32;         // large clouds: voxels with more points go to the heavy-voxel kernel
constexpr int kChunk = 256;         // points per work item of the heavy-voxel kernel
constexpr int kHeavyMaxC = 128;     // ... for up to this many channels (its sums' workspace)
constexpr int kMaxCap = 4096;       // tile points kept in LDS at once
constexpr int kCUs = 256;           // compute units of an MI355X

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
        pn_out[a] = (float)x;
        uvw[a] = voxel_axis(x, R);
    }
    return (uvw[0] * R + uvw[1]) * R + uvw[2];
}

__device__ __forceinline__ void write_point(int32_t* vox_id, float* norm_coords, size_t k, int id,
                                            const float* pn) {
    vox_id[k] = id;
    float* o = norm_coords + k * 3;
    o[0] = pn[0];
    o[1] = pn[1];
    o[2] = pn[2];
}

// ---------------------------------------------------------------------------
// Workgroup barrier for LDS data only. Every barrier in this file hands LDS
// data between threads; no thread reads global memory another thread of the
// workgroup wrote. So the barrier orders LDS accesses alone and does not wait
// for outstanding global stores (which __syncthreads() would), letting grid
// rows stream out while the workgroup carries on.
// ---------------------------------------------------------------------------
__device__ __forceinline__ void lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

// ---------------------------------------------------------------------------
// Workgroup reductions and scans (wave64).
// ---------------------------------------------------------------------------
template <typename T, typename Op>
__device__ __forceinline__ T wave_reduce(T v, Op op) {
    for (int o = 32; o > 0; o >>= 1) v = op(v, __shfl_xor(v, o, 64));
    return v;
}

struct MaxF { __device__ float operator()(float a, float b) const { return fmaxf(a, b); } };
struct MaxD { __device__ double operator()(double a, double b) const { return fmax(a, b); } };
struct AddL {
    __device__ long long operator()(long long a, long long b) const { return a + b; }
};

// K values reduced together over an NT-thread workgroup; every thread gets
// the results. lds holds K * NT/64 entries.
template <int NT, int K, typename T, typename Op>
__device__ void block_reduce_k(T (&v)[K], Op op, T* lds) {
#pragma unroll
    for (int i = 0; i < K; i++) v[i] = wave_reduce(v[i], op);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0)
#pragma unroll
        for (int i = 0; i < K; i++) lds[i * (NT / 64) + w] = v[i];
    lds_barrier();
#pragma unroll
    for (int i = 0; i < K; i++) {
        T r = lds[i * (NT / 64)];
        for (int j = 1; j < NT / 64; j++) r = op(r, lds[i * (NT / 64) + j]);
        v[i] = r;
    }
    lds_barrier();
}

// Exclusive scan of one int per thread over the workgroup; also returns the total.
template <int NT>
__device__ int block_exclusive_scan(int v, int* lds /* NT/64 */, int& total) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    int incl = v;
    for (int o = 1; o < 64; o <<= 1) {
        int t = __shfl_up(incl, o, 64);
        if (lane >= o) incl += t;
    }
    lds_barrier();
    if (lane == 63) lds[w] = incl;
    lds_barrier();
    int before = 0;
    total = 0;
    for (int i = 0; i < NT / 64; i++) {
        int s = lds[i];
        if (i < w) before += s;
        total += s;
    }
    lds_barrier();
    return before + incl - v;
}

// ---------------------------------------------------------------------------
// Normalisation, clouds of up to kSmallMaxN points: grid (slices, clouds) of
// 256-thread workgroups. Every workgroup holds its cloud's points in
// registers (PPT per thread), computes the normalisation parameters with
// three workgroup reductions (the three axes reduced together) and writes
// the voxel id and normalised coordinates of its own slice of 256 points.
// The parameters are order-free, so all slices of a cloud agree bit for bit.
// ---------------------------------------------------------------------------
// Zero fill of the whole grid (16-byte stores, grid-stride over `zero_blocks`
// workgroups). The tile kernel then writes the rows of occupied voxels.
__device__ __forceinline__ void zero_fill_role(uint4* grid16, size_t n16, int zb, int zero_blocks) {
    for (size_t i = (size_t)zb * 256 + threadIdx.x; i < n16; i += (size_t)zero_blocks * 256)
        grid16[i] = make_uint4(0, 0, 0, 0);
}

// A cloud's normalisation parameters (centroid c, largest squared centred
// norm M2, m = sqrt(M2)) from its N points, held PPT per thread (point
// threadIdx.x + i*NT in x[i]) by an NT-thread workgroup. Every reduction is
// order-free, so every workgroup that calls this for a cloud gets the same
// bits.
template <int PPT, int NT>
__device__ void cloud_params(const float (&x)[PPT][3], int N, double (&c)[3], double& M2,
                             double& m) {
    __shared__ float redf[3 * NT / 64];
    __shared__ long long redl[3 * NT / 64];
    __shared__ double redd[NT / 64];
    float A[3] = {0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < PPT; i++)
#pragma unroll
        for (int a = 0; a < 3; a++) A[a] = fmaxf(A[a], fabsf(x[i][a]));
    block_reduce_k<NT>(A, MaxF(), redf);
    int S[3];
    long long q[3] = {0, 0, 0};
#pragma unroll
    for (int a = 0; a < 3; a++) {
        S[a] = fixed_scale(A[a], N);
#pragma unroll
        for (int i = 0; i < PPT; i++)
            if (A[a] > 0.f && threadIdx.x + i * NT < N) q[a] += fixed_term(x[i][a], S[a]);
    }
    block_reduce_k<NT>(q, AddL(), redl);
#pragma unroll
    for (int a = 0; a < 3; a++) c[a] = centroid_from_sum(q[a], S[a], A[a], N);
    double mx[1] = {0.0};
#pragma unroll
    for (int i = 0; i < PPT; i++)
        if (threadIdx.x + i * NT < N) mx[0] = fmax(mx[0], sq_dist(x[i], c));
    block_reduce_k<NT>(mx, MaxD(), redd);
    M2 = mx[0];
    m = sqrt(M2);
}

// The cloud's N points into registers, PPT per thread (zero past N).
template <int PPT, int NT>
__device__ __forceinline__ void load_cloud(const float* __restrict__ p, int N,
                                           float (&x)[PPT][3]) {
#pragma unroll
    for (int i = 0; i < PPT; i++) {
        const int k = threadIdx.x + i * NT;
#pragma unroll
        for (int a = 0; a < 3; a++) x[i][a] = k < N ? p[3 * k + a] : 0.f;
    }
}

template <int PPT>
__device__ void ids_role(const float* __restrict__ coords, int N, int R, int slice, int b,
                         int32_t* __restrict__ vox_id, float* __restrict__ norm_coords) {
    constexpr int NT = 256;
    float x[PPT][3];
    load_cloud<PPT, NT>(coords + (size_t)b * N * 3, N, x);
    double c[3], M2, m;
    cloud_params<PPT, NT>(x, N, c, M2, m);
    // this workgroup's slice: points slice*256 + tid, i.e. register row `slice`
#pragma unroll
    for (int i = 0; i < PPT; i++) {
        const int k = threadIdx.x + i * NT;
        if (i != slice || k >= N) continue;
        float pn[3];
        const int id = normalise_point(x[i], c, M2, m, R, pn);
        write_point(vox_id, norm_coords, (size_t)b * N + k, id, pn);
    }
}

// One launch, three roles: the first B * slices workgroups normalise (slice
// blockIdx % slices of cloud blockIdx / slices), the next npack repack conv
// weights (a layer's convolutions, independent work that fills CUs the
// normalisation leaves idle), the rest zero the grid.
template <int PPT>
__global__ __launch_bounds__(256) void pv_voxel_ids_kernel(const float* __restrict__ coords,
                                                           int N, int R, int slices, int nid,
                                                           int32_t* __restrict__ vox_id,
                                                           float* __restrict__ norm_coords,
                                                           uint4* __restrict__ grid16, size_t n16,
                                                           PvPackJobs pack, int npack) {
    const int bid = blockIdx.x;
    if (bid >= nid + npack) {
        zero_fill_role(grid16, n16, bid - nid - npack, gridDim.x - nid - npack);
        return;
    }
    if (bid >= nid) {
        pv_pack_role(pack, bid - nid);
        return;
    }
    ids_role<PPT>(coords, N, R, bid % slices, bid / slices, vox_id, norm_coords);
}

// ---------------------------------------------------------------------------
// Normalisation, larger clouds: four kernels over G = ceil(N / kNormPts)
// workgroups per cloud, each step combining the previous step's G partials
// (read in parallel, one per thread) before working on its own points.
// Partials: pA [B][G][3] abs-max, pQ [B][G][3] fixed-point sums, pM [B][G]
// largest squared distance.
// ---------------------------------------------------------------------------
struct SplitWs {
    float* pA;
    long long* pQ;
    double* pM;
    int G;
    // points bucketed by tile: tcount [B][T] points per tile, tcursor [B][T]
    // fill cursors, tstart [B][T] bucket offsets, bk / br [B][N] point index
    // and voxel within the tile, in tile order (within a tile in no
    // particular order)
    int* tcount;
    int* tcursor;
    int* tstart;
    int* bk;
    int* br;
    int T;
    int TV;
    // heavy-voxel queue: hq[0] entries, then (cloud, voxel, bucket offset,
    // points) per voxel; room for hmax voxels. hpart [chunks][C] fp64 sums of
    // each chunk of kChunk points (room for C <= kHeavyMaxC).
    int* hq;
    int hmax;
    double* hpart;
};

__device__ void combine_absmax(const SplitWs& ws, int b, float* redf, float (&A)[3]) {
    A[0] = A[1] = A[2] = 0.f;
    for (int g = threadIdx.x; g < ws.G; g += kNormThreads)
        for (int a = 0; a < 3; a++) A[a] = fmaxf(A[a], ws.pA[((size_t)b * ws.G + g) * 3 + a]);
    block_reduce_k<kNormThreads>(A, MaxF(), redf);
}

__device__ void combine_centroid(const SplitWs& ws, int b, int N, float* redf, long long* redl,
                                 double (&c)[3]) {
    float A[3];
    combine_absmax(ws, b, redf, A);
    long long q[3] = {0, 0, 0};
    for (int g = threadIdx.x; g < ws.G; g += kNormThreads)
        for (int a = 0; a < 3; a++) q[a] += ws.pQ[((size_t)b * ws.G + g) * 3 + a];
    block_reduce_k<kNormThreads>(q, AddL(), redl);
    for (int a = 0; a < 3; a++) c[a] = centroid_from_sum(q[a], fixed_scale(A[a], N), A[a], N);
}

// Grid (G * B + npack + zero workgroups): the first G * B compute abs-max
// partials, the next npack repack conv weights, the rest zero the grid.
__global__ __launch_bounds__(kNormThreads) void pv_norm_absmax_kernel(const float* coords, int N,
                                                                      SplitWs ws, int B,
                                                                      uint4* grid16, size_t n16,
                                                                      PvPackJobs pack, int npack) {
    __shared__ float redf[3 * kNormThreads / 64];
    const int nid = ws.G * B;
    if ((int)blockIdx.x >= nid + npack) {
        zero_fill_role(grid16, n16, blockIdx.x - nid - npack, gridDim.x - nid - npack);
        return;
    }
    if ((int)blockIdx.x >= nid) {
        pv_pack_role(pack, blockIdx.x - nid);
        return;
    }
    if (blockIdx.x == 0) {  // the tile counters start at zero (used two launches later)
        for (int i = threadIdx.x; i < 2 * B * ws.T; i += kNormThreads)
            (i < B * ws.T ? ws.tcount : ws.tcursor)[i % (B * ws.T)] = 0;
        if (threadIdx.x == 0 && ws.hq) ws.hq[0] = 0;
    }
    const int g = blockIdx.x % ws.G, b = blockIdx.x / ws.G;
    const float* p = coords + (size_t)b * N * 3;
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    float A[3] = {0.f, 0.f, 0.f};
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads)
        for (int a = 0; a < 3; a++) A[a] = fmaxf(A[a], fabsf(p[3 * k + a]));
    block_reduce_k<kNormThreads>(A, MaxF(), redf);
    if (threadIdx.x < 3) ws.pA[((size_t)b * ws.G + g) * 3 + threadIdx.x] = A[threadIdx.x];
}

__global__ __launch_bounds__(kNormThreads) void pv_norm_sum_kernel(const float* coords, int N,
                                                                   SplitWs ws) {
    __shared__ float redf[3 * kNormThreads / 64];
    __shared__ long long redl[3 * kNormThreads / 64];
    const int g = blockIdx.x, b = blockIdx.y;
    const float* p = coords + (size_t)b * N * 3;
    float A[3];
    combine_absmax(ws, b, redf, A);
    int S[3];
    for (int a = 0; a < 3; a++) S[a] = fixed_scale(A[a], N);
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    long long q[3] = {0, 0, 0};
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads)
        for (int a = 0; a < 3; a++)
            if (A[a] > 0.f) q[a] += fixed_term(p[3 * k + a], S[a]);
    block_reduce_k<kNormThreads>(q, AddL(), redl);
    if (threadIdx.x < 3) ws.pQ[((size_t)b * ws.G + g) * 3 + threadIdx.x] = q[threadIdx.x];
}

__global__ __launch_bounds__(kNormThreads) void pv_norm_radius_kernel(const float* coords, int N,
                                                                      SplitWs ws) {
    __shared__ float redf[3 * kNormThreads / 64];
    __shared__ long long redl[3 * kNormThreads / 64];
    __shared__ double redd[kNormThreads / 64];
    const int g = blockIdx.x, b = blockIdx.y;
    const float* p = coords + (size_t)b * N * 3;
    double c[3];
    combine_centroid(ws, b, N, redf, redl, c);
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    double mx[1] = {0.0};
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads)
        mx[0] = fmax(mx[0], sq_dist(p + 3 * k, c));
    block_reduce_k<kNormThreads>(mx, MaxD(), redd);
    if (threadIdx.x == 0) ws.pM[(size_t)b * ws.G + g] = mx[0];
}

__global__ __launch_bounds__(kNormThreads) void pv_norm_points_kernel(
    const float* coords, int N, int R, SplitWs ws, int32_t* __restrict__ vox_id,
    float* __restrict__ norm_coords) {
    __shared__ float redf[3 * kNormThreads / 64];
    __shared__ long long redl[3 * kNormThreads / 64];
    __shared__ double redd[kNormThreads / 64];
    const int g = blockIdx.x, b = blockIdx.y;
    const float* p = coords + (size_t)b * N * 3;
    double c[3];
    combine_centroid(ws, b, N, redf, redl, c);
    double mx[1] = {0.0};
    for (int i = threadIdx.x; i < ws.G; i += kNormThreads)
        mx[0] = fmax(mx[0], ws.pM[(size_t)b * ws.G + i]);
    block_reduce_k<kNormThreads>(mx, MaxD(), redd);
    const double M2 = mx[0];
    const double m = sqrt(M2);
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    // points per tile of this slice, LDS first, then one global add per tile
    extern __shared__ int thist[];  // [T]
    for (int t = threadIdx.x; t < ws.T; t += kNormThreads) thist[t] = 0;
    lds_barrier();
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads) {
        float pn[3];
        const int id = normalise_point(p + 3 * k, c, M2, m, R, pn);
        write_point(vox_id, norm_coords, (size_t)b * N + k, id, pn);
        atomicAdd(&thist[id / ws.TV], 1);
    }
    lds_barrier();
    for (int t = threadIdx.x; t < ws.T; t += kNormThreads)
        if (thist[t]) atomicAdd(&ws.tcount[(size_t)b * ws.T + t], thist[t]);
}

// Given voxel indices: the tile counters and the heavy-voxel queue of large
// clouds start at zero (workgroup 0 of the first launch, for B > 0; the other
// workgroups zero the grid when the tile kernel writes only occupied rows),
// then points per tile, LDS first, one global add per tile (second launch,
// grid (G, B)). Indices outside the grid are dropped here and in the bucket
// scatter alike.
__global__ __launch_bounds__(kNormThreads) void pv_tile_reset_kernel(SplitWs ws, int B,
                                                                     uint4* grid16, size_t n16) {
    if (blockIdx.x > 0) {
        zero_fill_role(grid16, n16, blockIdx.x - 1, gridDim.x - 1);
        return;
    }
    if (B == 0) return;  // small clouds: nothing is bucketed, only the grid is zeroed
    for (int i = threadIdx.x; i < 2 * B * ws.T; i += kNormThreads)
        (i < B * ws.T ? ws.tcount : ws.tcursor)[i % (B * ws.T)] = 0;
    if (threadIdx.x == 0 && ws.hq) ws.hq[0] = 0;
}

__global__ __launch_bounds__(kNormThreads) void pv_tile_count_kernel(
    const int32_t* __restrict__ ids, int N, SplitWs ws) {
    extern __shared__ int thist[];  // [T]
    const int g = blockIdx.x, b = blockIdx.y;
    for (int t = threadIdx.x; t < ws.T; t += kNormThreads) thist[t] = 0;
    lds_barrier();
    const int k0 = g * kNormPts, k1 = min(N, k0 + kNormPts);
    for (int k = k0 + threadIdx.x; k < k1; k += kNormThreads) {
        const int id = ids[(size_t)b * N + k];
        if (id >= 0 && id / ws.TV < ws.T) atomicAdd(&thist[id / ws.TV], 1);
    }
    lds_barrier();
    for (int t = threadIdx.x; t < ws.T; t += kNormThreads)
        if (thist[t]) atomicAdd(&ws.tcount[(size_t)b * ws.T + t], thist[t]);
}

// Scatter of each point into its tile's bucket: grid (G, B), the same slices
// as pv_norm_points_kernel. Each workgroup takes the exclusive prefix of the
// cloud's tile counts, ranks its points per tile in LDS, reserves a range of
// every tile's bucket with one global add and writes (point, voxel in tile).
__global__ __launch_bounds__(kNormThreads) void pv_bucket_kernel(const int32_t* __restrict__ ids,
                                                                 int N, SplitWs ws) {
    constexpr int NT = kNormThreads;
    constexpr int PPT = kNormPts / NT;
    extern __shared__ int bl[];  // pre[T], hist[T]
    __shared__ int scan_lds[NT / 64];
    int* pre = bl;
    int* hist = bl + ws.T;
    const int g = blockIdx.x, b = blockIdx.y;
    const int* tc = ws.tcount + (size_t)b * ws.T;
    {
        const int seg = (ws.T + NT - 1) / NT;
        const int s0 = min(ws.T, (int)threadIdx.x * seg), s1 = min(ws.T, s0 + seg);
        int local = 0;
        for (int t = s0; t < s1; t++) local += tc[t];
        int total;
        int run = block_exclusive_scan<NT>(local, scan_lds, total);
        for (int t = s0; t < s1; t++) {
            pre[t] = run;
            if (g == 0) ws.tstart[(size_t)b * ws.T + t] = run;
            run += tc[t];
        }
        for (int t = threadIdx.x; t < ws.T; t += NT) hist[t] = 0;
    }
    lds_barrier();
    const int k0 = g * kNormPts;
    int tile[PPT], rank[PPT], vid[PPT];
#pragma unroll
    for (int i = 0; i < PPT; i++) {
        const int k = k0 + i * NT + threadIdx.x;
        tile[i] = -1;
        if (k < N) {
            vid[i] = ids[(size_t)b * N + k];
            // an index outside the grid (given indices: invalid input) is dropped
            if (vid[i] >= 0 && vid[i] / ws.TV < ws.T) {
                tile[i] = vid[i] / ws.TV;
                rank[i] = atomicAdd(&hist[tile[i]], 1);
            }
        }
    }
    lds_barrier();
    for (int t = threadIdx.x; t < ws.T; t += NT)
        if (hist[t]) pre[t] += atomicAdd(&ws.tcursor[(size_t)b * ws.T + t], hist[t]);
    lds_barrier();
#pragma unroll
    for (int i = 0; i < PPT; i++) {
        if (tile[i] < 0) continue;
        const size_t pos = (size_t)b * N + pre[tile[i]] + rank[i];
        ws.bk[pos] = k0 + i * NT + threadIdx.x;
        ws.br[pos] = vid[i] - tile[i] * ws.TV;
    }
}

// ---------------------------------------------------------------------------
// Feature rows: 8 channels at a time (16 or 32 bytes) or one channel.
// ---------------------------------------------------------------------------
template <typename FT>
__device__ __forceinline__ void load8f(const FT* src, float* v);
template <>
__device__ __forceinline__ void load8f<float>(const float* src, float* v) {
    const float4 a = *(const float4*)src, b = *(const float4*)(src + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
template <>
__device__ __forceinline__ void load8f<uint16_t>(const uint16_t* src, float* v) {
    const uint4 a = *(const uint4*)src;
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
    for (int i = 0; i < 4; i++) {
        v[2 * i] = pv_bf16_to_f32((uint16_t)(w[i] & 0xffffu));
        v[2 * i + 1] = pv_bf16_to_f32((uint16_t)(w[i] >> 16));
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

// Sum of 8 channels over the points list[j0], list[j0 + step], ... (< j1) in
// that order, fp64, with U points' loads in flight at a time.
template <typename FT, int U = 8>
__device__ __forceinline__ void sum8(const FT* fb, int feat_ld, int col, const int* list, int j0,
                                     int j1, int step, double* acc) {
    int j = j0;
    for (; j + (U - 1) * step < j1; j += U * step) {
        float f[U][8];
#pragma unroll
        for (int u = 0; u < U; u++) load8f<FT>(fb + (size_t)list[j + u * step] * feat_ld + col, f[u]);
#pragma unroll
        for (int u = 0; u < U; u++)
#pragma unroll
            for (int i = 0; i < 8; i++) acc[i] += (double)f[u][i];
    }
    for (; j < j1; j += step) {
        float f[8];
        load8f<FT>(fb + (size_t)list[j] * feat_ld + col, f);
#pragma unroll
        for (int i = 0; i < 8; i++) acc[i] += (double)f[i];
    }
}

// ---------------------------------------------------------------------------
// Tile fill: one workgroup per (tile t of TV voxels, cloud b).
//
// Dynamic LDS: hist[TV] points per voxel, start[TV+1] exclusive prefix,
// cur[TV] scatter cursors, heavy[TV] heavy-voxel list, kbuf[CAP] and
// rbuf[CAP] the tile's points (index, voxel) as found, list[CAP] the points
// sorted by voxel, then a region used either as the fp32 feature stage (the
// tile's points' features, when they fit) or as red[256][8] doubles for the
// heavy-voxel reduction (also the fp64 accumulators of a voxel holding more
// than CAP points).
// ---------------------------------------------------------------------------
// heavy-voxel reduction buffer: 8 doubles per thread
constexpr int red_bytes(int NT) { return NT * 8 * (int)sizeof(double); }

struct TileLds {
    int* hist;
    int* start;
    int* cur;
    int* heavy;
    int* kbuf;
    int* rbuf;
    int* list;
    double* red;
    float* stage;
};

size_t tile_lds_bytes(int NT, int TV, int CAP, int stage_bytes) {
    return (size_t)(4 * TV + 1) * 4 + (size_t)3 * CAP * 4 + 16 /* align */ +
           (size_t)(stage_bytes > red_bytes(NT) ? stage_bytes : red_bytes(NT));
}

__device__ inline TileLds tile_lds(char* smem, int TV, int CAP) {
    TileLds L;
    int* p = (int*)smem;
    L.hist = p;
    L.start = p + TV;
    L.cur = L.start + TV + 1;
    L.heavy = L.cur + TV;
    L.kbuf = L.heavy + TV;
    L.rbuf = L.kbuf + CAP;
    L.list = L.rbuf + CAP;
    uintptr_t r = (uintptr_t)(L.list + CAP);
    L.red = (double*)((r + 15) & ~(uintptr_t)15);
    L.stage = (float*)L.red;
    return L;
}

// Where a tile hands its heaviest voxels (more than kExport points) to the
// heavy-voxel kernel instead of summing them itself: their sorted point
// lists go back to the tile's bucket (global, from bstart), one queue entry
// each. hq == nullptr: no export.
struct HeavyOut {
    int* hq;
    int* bucket;   // the tile's bucket: point indices, from the tile's first
    int b, vox0;   // cloud, first voxel of the tile
    int bstart;    // bucket offset of the tile within the cloud
};

// Means of voxels [lo, hi) of the tile from list (voxel vi's points at
// list[start[vi] - base .. start[vi+1] - base)), written to out (the tile's
// grid rows).
//  * staged (VEC, the segment's features fit the stage): every point's
//    features are first copied to LDS with independent loads, then each
//    (voxel, 8-channel group) item sums from LDS and the grid rows stream out;
//  * otherwise (VEC): voxels of up to kHeavy points are summed straight from
//    global memory; heavier voxels are then taken one at a time by the whole
//    workgroup, the points split across threads;
//  * not VEC: one (voxel, channel) item per thread, straight from memory.
// last: no LDS reuse follows, so the closing barriers are skipped.
// side(): other stores of the workgroup (the empty rows), issued once this
// range's first feature loads are in flight so that they queue behind them.
template <int NT, typename FT, typename GT, bool VEC, typename Side>
__device__ void tile_fill_range(const TileLds& L, int lo, int hi, int base, const FT* fb,
                                int feat_ld, int C, GT* out, int* s_nheavy, int stage_bytes,
                                bool last, Side side, const HeavyOut& ho) {
    if (threadIdx.x == 0) *s_nheavy = 0;
    lds_barrier();
    if (VEC) {
        const int gpv = C / 8;  // 8-channel groups per voxel
        const int items = (hi - lo) * gpv;
        const int npts = L.start[hi] - L.start[lo];
        if ((size_t)npts * C * 4 <= (size_t)stage_bytes) {
            // stage: row j (list order) = the features of point list[j]
            const int pieces = npts * gpv;
            bool sided = false;
            for (int i0 = threadIdx.x; i0 < pieces; i0 += 4 * NT) {
                float f[4][8];
#pragma unroll
                for (int u = 0; u < 4; u++) {
                    const int i = i0 + u * NT;
                    if (i < pieces) {
                        const int j = i / gpv, cg = i - j * gpv;
                        load8f<FT>(fb + (size_t)L.list[j] * feat_ld + cg * 8, f[u]);
                    }
                }
                if (!sided) {
                    side();
                    sided = true;
                }
#pragma unroll
                for (int u = 0; u < 4; u++) {
                    const int i = i0 + u * NT;
                    if (i < pieces) {
                        float* d = L.stage + (size_t)i * 8;
                        *(float4*)d = make_float4(f[u][0], f[u][1], f[u][2], f[u][3]);
                        *(float4*)(d + 4) = make_float4(f[u][4], f[u][5], f[u][6], f[u][7]);
                    }
                }
            }
            if (!sided) side();
            lds_barrier();
            for (int item = threadIdx.x; item < items; item += NT) {
                const int vi = lo + item / gpv, cg = item % gpv;
                const int nk = L.hist[vi];
                if (nk == 0) continue;  // empty voxel: its row is already zero
                float mean[8];
                {
                    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                    const int j0 = L.start[vi] - base;
                    for (int j = j0; j < j0 + nk; j++) {
                        const float* src = L.stage + ((size_t)j * gpv + cg) * 8;
                        const float4 x0 = *(const float4*)src, x1 = *(const float4*)(src + 4);
                        acc[0] += x0.x; acc[1] += x0.y; acc[2] += x0.z; acc[3] += x0.w;
                        acc[4] += x1.x; acc[5] += x1.y; acc[6] += x1.z; acc[7] += x1.w;
                    }
#pragma unroll
                    for (int i = 0; i < 8; i++) mean[i] = (float)(acc[i] / (double)nk);
                }
                store8<GT>(out + (size_t)vi * C + cg * 8, mean);
            }
            if (!last) lds_barrier();
            return;
        }
        // Occupied voxels: light ones listed in occ (L.cur, free once the
        // points are sorted) so that the (voxel, channel group) items are
        // spread evenly over the threads, heavy ones for the wave loop.
        // exported voxels are listed from heavy[hi - lo - 1] down
        __shared__ int s_nocc, s_nexp;
        int* occ = L.cur;
        if (threadIdx.x == 0) s_nocc = s_nexp = 0;
        lds_barrier();
        for (int vi = lo + threadIdx.x; vi < hi; vi += NT) {
            const int nk = L.hist[vi];
            if (nk == 0) continue;  // empty voxel: a zero row
            if (ho.hq && nk > kExport)
                L.heavy[hi - lo - 1 - atomicAdd(&s_nexp, 1)] = vi;
            else if (nk > kHeavy)
                L.heavy[atomicAdd(s_nheavy, 1)] = vi;
            else
                occ[atomicAdd(&s_nocc, 1)] = vi;
        }
        lds_barrier();
        // Exported voxels: the sorted point list back to the bucket (at the
        // voxel's offset in the tile) and a queue entry.
        const int nexp = s_nexp;
        if (nexp > 0) {
            __shared__ int s_slot0;
            if (threadIdx.x == 0) s_slot0 = atomicAdd(ho.hq, nexp);
            lds_barrier();
            for (int e = 0; e < nexp; e++) {
                const int vi = L.heavy[hi - lo - 1 - e], q = s_slot0 + e;
                const int nk = L.hist[vi], j0 = L.start[vi] - base;
                for (int j = threadIdx.x; j < nk; j += NT)
                    ho.bucket[L.start[vi] + j] = L.list[j0 + j];
                if (threadIdx.x == 0) {
                    int* ent = ho.hq + 1 + 4 * q;
                    ent[0] = ho.b;
                    ent[1] = ho.vox0 + vi;
                    ent[2] = ho.bstart + L.start[vi];
                    ent[3] = nk;
                }
            }
        }
        // Items go in batches of IB per thread: the first two points of every
        // item of a batch are loaded at once (most occupied voxels hold one or
        // two points), then the zero rows go out (side()), then each item adds
        // its remaining points. One counter tracks loads and stores in issue
        // order, so loads issued after side()'s stores would wait for them.
        constexpr int IB = 2;
        const int nocc = s_nocc, nitems = nocc * gpv;
        bool sided = false;
        for (int i0 = threadIdx.x; i0 < nitems; i0 += IB * NT) {
            float f0[IB][8], f1[IB][8];
            int vis[IB], cgs[IB], nks[IB], j0s[IB];
#pragma unroll
            for (int q = 0; q < IB; q++) {
                const int item = i0 + q * NT;
                nks[q] = 0;
                if (item < nitems) {
                    vis[q] = occ[item / gpv];
                    cgs[q] = item % gpv;
                    nks[q] = L.hist[vis[q]];
                    j0s[q] = L.start[vis[q]] - base;
                    load8f<FT>(fb + (size_t)L.list[j0s[q]] * feat_ld + cgs[q] * 8, f0[q]);
                    if (nks[q] > 1)
                        load8f<FT>(fb + (size_t)L.list[j0s[q] + 1] * feat_ld + cgs[q] * 8, f1[q]);
                }
            }
            if (!sided) {
                side();
                sided = true;
            }
#pragma unroll
            for (int q = 0; q < IB; q++) {
                if (nks[q] == 0) continue;
                double acc[8];
#pragma unroll
                for (int i = 0; i < 8; i++) acc[i] = (double)f0[q][i];
                if (nks[q] > 1)
#pragma unroll
                    for (int i = 0; i < 8; i++) acc[i] += (double)f1[q][i];
                sum8<FT, 4>(fb, feat_ld, cgs[q] * 8, L.list, j0s[q] + 2, j0s[q] + nks[q], 1, acc);

                float mean[8];
#pragma unroll
                for (int i = 0; i < 8; i++) mean[i] = (float)(acc[i] / (double)nks[q]);
                store8<GT>(out + (size_t)vis[q] * C + cgs[q] * 8, mean);
            }
        }
        if (!sided) side();
        lds_barrier();
        // Heavy voxels: one per wave, four at a time. For channel groups cg0 ..
        // cg0+ng-1, lane = sub * ng + (cg - cg0) sums points j = sub, sub+S,
        // ... (S = 64 / ng subsets); the S partial sums are then combined in
        // subset order through LDS.
        const int nheavy = *s_nheavy;
        const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
        double* red = L.red + (size_t)wave * 64 * 8;
        for (int r0 = 0; r0 < nheavy; r0 += NT / 64) {
            const int hidx = r0 + wave;
            const bool active = hidx < nheavy;
            const int vi = active ? L.heavy[hidx] : 0;
            const int nk = active ? L.hist[vi] : 0;
            const int j0 = active ? L.start[vi] - base : 0;
            for (int cg0 = 0; cg0 < gpv; cg0 += 64) {
                const int ng = min(64, gpv - cg0);
                const int S = 64 / ng;
                const int sub = lane / ng, cl = lane % ng;
                double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                if (active && sub < S)
                    sum8<FT>(fb, feat_ld, (cg0 + cl) * 8, L.list, j0 + sub, j0 + nk, S, acc);
                if (sub < S)
#pragma unroll
                    for (int i = 0; i < 8; i++) red[(sub * ng + cl) * 8 + i] = acc[i];
                lds_barrier();
                if (active && lane < ng) {
                    double tot[8];
#pragma unroll
                    for (int i = 0; i < 8; i++) tot[i] = red[lane * 8 + i];
                    for (int s2 = 1; s2 < S; s2++)
#pragma unroll
                        for (int i = 0; i < 8; i++) tot[i] += red[(s2 * ng + lane) * 8 + i];
                    float mean[8];
#pragma unroll
                    for (int i = 0; i < 8; i++) mean[i] = (float)(tot[i] / (double)nk);
                    store8<GT>(out + (size_t)vi * C + (cg0 + lane) * 8, mean);
                }
                lds_barrier();
            }
        }
    } else {
        side();
        const int items = (hi - lo) * C;
        for (int item = threadIdx.x; item < items; item += NT) {
            const int vi = lo + item / C, ch = item % C;
            const int nk = L.hist[vi];
            if (nk == 0) continue;  // empty voxel: its row is already zero
            double acc = 0.0;
            const int j0 = L.start[vi] - base;
            for (int j = j0; j < j0 + nk; j++)
                acc += (double)load1<FT>(fb + (size_t)L.list[j] * feat_ld + ch);
            store1<GT>(out + (size_t)vi * C + ch, (float)(acc / (double)nk));
        }
    }
    if (!last) lds_barrier();
}

// The tile's points among ids[0 .. N): count per voxel and keep (index,
// voxel) while they fit. Reads 16 ids per thread per round when the array
// is 16-byte aligned.
__device__ __forceinline__ void tile_collect_one(const TileLds& L, int k, int r, int nv, int CAP,
                                                 int* s_ntile) {
    if (r >= 0 && r < nv) {
        atomicAdd(&L.hist[r], 1);
        const int slot = atomicAdd(s_ntile, 1);
        if (slot < CAP) {
            L.kbuf[slot] = k;
            L.rbuf[slot] = r;
        }
    }
}

// The rest of a tile once its points are collected (L.hist, L.kbuf/rbuf):
// counts out, prefix over the voxels, counting sort, zero rows (zero_rows),
// means. each_point(fn) calls fn(point, voxel - v0) for every point of the
// cloud that may lie in the tile (for the segmented passes, when the tile
// holds more than CAP points).
template <int NT, typename FT, typename GT, bool VEC, typename EachPoint>
__device__ void tile_finish(const TileLds& L, int TV, int nv, int CAP, int32_t* cnt, GT* out,
                            const FT* fb, int feat_ld, int C, bool zero_rows, int stage_bytes,
                            int* scan_lds, int* s_nheavy, EachPoint each_point,
                            const HeavyOut& ho) {
    // 2. counts out; exclusive prefix over the tile's voxels
    for (int i = threadIdx.x; i < nv; i += NT) cnt[i] = L.hist[i];
    // The tile's empty voxels: zero rows (16-byte stores), streaming out
    // while the occupied voxels are gathered.
    auto zero_empty_rows = [&]() {
        if (!VEC || !zero_rows) return;
        const int pr = C * (int)sizeof(GT) / 16;  // 16-byte pieces per row
        uint4* o16 = (uint4*)out;
        for (int i = threadIdx.x; i < nv * pr; i += NT)
            if (L.hist[i / pr] == 0) o16[i] = make_uint4(0u, 0u, 0u, 0u);
    };
    auto nothing = []() {};
    {
        const int seg = (TV + NT - 1) / NT;
        const int s0 = min(TV, (int)threadIdx.x * seg), s1 = min(TV, s0 + seg);
        int local = 0;
        for (int i = s0; i < s1; i++) local += L.hist[i];
        int total;
        int run = block_exclusive_scan<NT>(local, scan_lds, total);
        for (int i = s0; i < s1; i++) {
            L.start[i] = run;
            run += L.hist[i];
        }
        if (threadIdx.x == 0) L.start[TV] = total;
    }
    lds_barrier();
    const int total = L.start[TV];
    if (total <= CAP) {
        // 3. counting sort of the kept points by voxel, then the fill
        for (int i = threadIdx.x; i < nv; i += NT) L.cur[i] = L.start[i];
        lds_barrier();
        for (int s = threadIdx.x; s < total; s += NT)
            L.list[atomicAdd(&L.cur[L.rbuf[s]], 1)] = L.kbuf[s];
        lds_barrier();
        tile_fill_range<NT, FT, GT, VEC>(L, 0, nv, 0, fb, feat_ld, C, out, s_nheavy, stage_bytes,
                                         true, zero_empty_rows, ho);
        return;
    }
    zero_empty_rows();
    // More points than fit: voxel segments of at most CAP points, each
    // gathered by scanning the ids again. A single voxel beyond CAP points is
    // summed by the whole workgroup with LDS fp64 atomics.
    int lo = 0;
    while (lo < nv) {
        if (L.start[lo + 1] - L.start[lo] > CAP) {
            const int nk = L.start[lo + 1] - L.start[lo];
            double* hacc = L.red;  // C <= 1024 doubles fit in red[] (16 KB)
            for (int ch = threadIdx.x; ch < C; ch += NT) hacc[ch] = 0.0;
            lds_barrier();
            each_point([&](int k, int r) {
                if (r == lo)
                    for (int ch = 0; ch < C; ch++)
                        atomicAdd(&hacc[ch], (double)load1<FT>(fb + (size_t)k * feat_ld + ch));
            });
            lds_barrier();
            for (int ch = threadIdx.x; ch < C; ch += NT)
                store1<GT>(out + (size_t)lo * C + ch, (float)(hacc[ch] / (double)nk));
            lds_barrier();
            lo++;
            continue;
        }
        // largest hi with start[hi] - start[lo] <= CAP (binary search)
        int a = lo + 1, z = nv;
        while (a < z) {
            const int mid = (a + z + 1) >> 1;
            if (L.start[mid] - L.start[lo] <= CAP)
                a = mid;
            else
                z = mid - 1;
        }
        const int hi = a, base = L.start[lo];
        for (int i = lo + threadIdx.x; i < hi; i += NT) L.cur[i] = L.start[i] - base;
        lds_barrier();
        each_point([&](int k, int r) {
            if (r >= lo && r < hi) L.list[atomicAdd(&L.cur[r], 1)] = k;
        });
        lds_barrier();
        // (the later segments scan the bucket again: nothing is exported)
        tile_fill_range<NT, FT, GT, VEC>(L, lo, hi, base, fb, feat_ld, C, out, s_nheavy, stage_bytes,
                                         false, nothing,
                                         HeavyOut{nullptr, nullptr, 0, 0, 0});
        lo = hi;
    }
}

template <int NT, typename FT, typename GT, bool VEC>
__global__ __launch_bounds__(NT) void pv_voxel_tile_kernel(
    const int32_t* __restrict__ vox_id, const FT* __restrict__ feats, int feat_ld, int N, int C,
    int R, int TV, int CAP, int stage_bytes, int zero_rows, GT* __restrict__ grid,
    int32_t* __restrict__ counts, int* bk, const int* __restrict__ br,
    const int* __restrict__ tcount, const int* __restrict__ tstart, int T, int* hq) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ int scan_lds[NT / 64];
    __shared__ int s_ntile, s_nheavy;
    const TileLds L = tile_lds(smem, TV, CAP);

    const int t = blockIdx.x, b = blockIdx.y;
    const bool bucketed = bk != nullptr;
    const int bstart = bucketed ? tstart[(size_t)b * T + t] : 0;
    const int btotal = bucketed ? tcount[(size_t)b * T + t] : 0;
    const int V = R * R * R;
    const int v0 = t * TV, nv = min(TV, V - v0);
    const int32_t* ids = vox_id + (size_t)b * N;
    const FT* fb = feats + (size_t)b * N * feat_ld;
    GT* out = grid + ((size_t)b * V + v0) * C;

    for (int i = threadIdx.x; i < TV; i += NT) L.hist[i] = 0;
    if (threadIdx.x == 0) s_ntile = 0;
    lds_barrier();
    // 1. the tile's points: its bucket when the points were bucketed by tile
    // (large clouds), else a scan of all the cloud's ids
    const int* kb = bucketed ? bk + (size_t)b * N + bstart : nullptr;
    const int* rb = bucketed ? br + (size_t)b * N + bstart : nullptr;
    // every point of the tile (bucketed) or of the cloud, as (index, voxel - v0)
    auto each_point = [&](auto fn) {
        if (bucketed)
            for (int j = threadIdx.x; j < btotal; j += NT) fn(kb[j], rb[j]);
        else
            for (int k = threadIdx.x; k < N; k += NT) fn(k, ids[k] - v0);
    };
    if (bucketed) {
        for (int j0 = threadIdx.x; j0 < btotal; j0 += 4 * NT) {
            int kk[4], rr[4];
#pragma unroll
            for (int u = 0; u < 4; u++) {
                const int j = j0 + u * NT;
                kk[u] = j < btotal ? kb[j] : 0;
                rr[u] = j < btotal ? rb[j] : -1;
            }
#pragma unroll
            for (int u = 0; u < 4; u++) tile_collect_one(L, kk[u], rr[u], nv, CAP, &s_ntile);
        }
    } else {
        int k0 = 0;
        if (((uintptr_t)ids & 15) == 0) {
            const int n16 = N / 16 * 16;  // rounds of 4 int4 loads per thread
            for (int kq = threadIdx.x * 4; kq < n16; kq += NT * 16) {
                int4 q[4];
#pragma unroll
                for (int u = 0; u < 4; u++) {
                    const int k = kq + u * NT * 4;
                    q[u] = k < n16 ? *(const int4*)(ids + k) : make_int4(-1 - v0, 0, 0, 0);
                }
#pragma unroll
                for (int u = 0; u < 4; u++) {
                    const int k = kq + u * NT * 4;
                    if (k < n16) {
                        tile_collect_one(L, k, q[u].x - v0, nv, CAP, &s_ntile);
                        tile_collect_one(L, k + 1, q[u].y - v0, nv, CAP, &s_ntile);
                        tile_collect_one(L, k + 2, q[u].z - v0, nv, CAP, &s_ntile);
                        tile_collect_one(L, k + 3, q[u].w - v0, nv, CAP, &s_ntile);
                    }
                }
            }
            k0 = n16;
        }
        for (int k = k0 + threadIdx.x; k < N; k += NT)
            tile_collect_one(L, k, ids[k] - v0, nv, CAP, &s_ntile);
    }
    lds_barrier();
    const HeavyOut ho{bucketed ? hq : nullptr, bucketed ? bk + (size_t)b * N + bstart : nullptr, b,
                      v0, bstart};
    tile_finish<NT, FT, GT, VEC>(L, TV, nv, CAP, counts + (size_t)b * V + v0, out, fb, feat_ld, C,
                                 zero_rows != 0, stage_bytes, scan_lds, &s_nheavy, each_point, ho);
}

// Tile shape. Small clouds (every tile scans all N ids, cheap): about 2048
// tiles of 128 threads, about 18 KB of LDS, so that eight workgroups fit per
// CU and every tile is resident at once; coarse grids go down to 32 voxels
// per tile to get there. Large clouds (points bucketed by tile beforehand):
// about 1024 tiles of 256 threads, so that a dense cluster spreads over
// several workgroups.
struct TileShape {
    int nt, tv;
};
TileShape tile_shape(int B, int V, int N) {
    const bool small_cloud = N <= kSmallMaxN;
    const long long want = small_cloud ? 2048 : 1024;
    int tv = 1024;
    while (tv > 32 && (long long)B * ((V + tv - 1) / tv) < want) tv >>= 1;
    return TileShape{small_cloud ? 128 : 256, tv};
}


// LDS budget of the tile kernel: no feature stage (each (voxel, channel
// group) sums straight from memory) and room for the tile's points, tiles
// with more points taking the segmented path. Large clouds: kMaxCap points.
// Small clouds: as many as keep every tile of the grid resident at once (the
// 160 KB of a CU shared by its tiles, less 2 KB of slack), at least 256, at
// most kMaxCap (coarse grids, with many points per tile, have few tiles).
// Dynamic LDS beyond 64 KB has to be granted per kernel; when that fails the
// capacity shrinks to what 64 KB holds.
template <typename K>
void tile_budget(K kernel, int NT, int TV, int N, long tiles, int& cap, int& stage) {
    const bool small_cloud = N <= kSmallMaxN;
    int want = kMaxCap;
    if (small_cloud) {
        const long per_cu = std::max(1L, (tiles + kCUs - 1) / kCUs);
        const long budget = std::min<long>(65536, 160 * 1024 / per_cu - 2048);
        const long fit = (budget - (long)tile_lds_bytes(NT, TV, 0, 0)) / 12;
        want = (int)std::max(256L, std::min<long>(kMaxCap, fit));
    }
    cap = N < want ? (N > 0 ? N : 1) : want;
    stage = 0;
    const size_t small = 65536;
    const size_t want_bytes = tile_lds_bytes(NT, TV, cap, stage);
    if (want_bytes <= small) return;
    // the grant is per kernel and lasts for the process: ask once per kernel
    // and size (a launch being captured into a graph then makes no other call)
    static std::mutex mu;
    static std::unordered_map<const void*, size_t> granted;
    {
        std::lock_guard<std::mutex> lock(mu);
        auto it = granted.find((const void*)kernel);
        if (it != granted.end() && want_bytes <= it->second) return;
    }
    if (hipFuncSetAttribute((const void*)kernel, hipFuncAttributeMaxDynamicSharedMemorySize,
                            (int)want_bytes) == hipSuccess) {
        std::lock_guard<std::mutex> lock(mu);
        size_t& g = granted[(const void*)kernel];
        g = std::max(g, want_bytes);
        return;
    }
    (void)hipGetLastError();
    stage = 0;
    while (cap > 1 && tile_lds_bytes(NT, TV, cap, stage) > small) cap >>= 1;
}

// Tiles' point sources: the points bucketed by tile (large clouds) or none
// (each tile scans all ids).
struct Buckets {
    int* bk;
    const int* br;
    const int* tcount;
    const int* tstart;
    int T;
    int* hq;  // heavy-voxel queue (nullptr: none)
};

template <int NT, typename FT, typename GT>
void launch_tiles_nt(const int32_t* ids, const void* feats, int feat_ld, int B, int N, int C,
                     int R, int TV, void* grid, int32_t* counts, bool vec, bool zero_rows,
                     const Buckets& bu, hipStream_t s) {
    const int V = R * R * R;
    dim3 g((V + TV - 1) / TV, B);
    int cap, stage;
    if (vec) {
        auto k = pv_voxel_tile_kernel<NT, FT, GT, true>;
        tile_budget(k, NT, TV, N, (long)g.x * g.y, cap, stage);
        hipLaunchKernelGGL(k, g, dim3(NT), tile_lds_bytes(NT, TV, cap, stage), s, ids,
                           (const FT*)feats, feat_ld, N, C, R, TV, cap, stage, (int)zero_rows,
                           (GT*)grid, counts, bu.bk, bu.br, bu.tcount, bu.tstart, bu.T, bu.hq);
    } else {
        auto k = pv_voxel_tile_kernel<NT, FT, GT, false>;
        tile_budget(k, NT, TV, N, (long)g.x * g.y, cap, stage);
        hipLaunchKernelGGL(k, g, dim3(NT), tile_lds_bytes(NT, TV, cap, stage), s, ids,
                           (const FT*)feats, feat_ld, N, C, R, TV, cap, 0, 0, (GT*)grid, counts,
                           bu.bk, bu.br, bu.tcount, bu.tstart, bu.T, bu.hq);
    }
}

// Heavy voxels handed over by the tiles (large clouds, more than kExport
// points each), cut into chunks of kChunk points, chunk c of the queue order
// taken by workgroup c % gridDim.x. The queue is read in windows of 256
// entries: an exclusive scan of the entries' chunk counts gives each chunk
// its voxel. In a chunk, thread sub * ng + (cg - cg0) sums points sub,
// sub + S, ... (S = 256 / ng subsets of the voxel's ng channel groups); the
// partials are combined in subset order through LDS and written as the
// chunk's fp64 sums. No workgroup waits for another: the next kernel
// combines each voxel's chunks.
__device__ __forceinline__ int heavy_window(const int* hq, int nq, int w0, int* s_pre, int* s_scan) {
    const int ent = w0 + (int)threadIdx.x;
    const int nch = ent < nq ? (hq[1 + 4 * ent + 3] + kChunk - 1) / kChunk : 0;
    int total;
    const int pre = block_exclusive_scan<256>(nch, s_scan, total);
    s_pre[threadIdx.x] = pre;
    lds_barrier();
    return total;
}

template <typename FT>
__global__ __launch_bounds__(256) void pv_voxel_heavy_kernel(
    const FT* __restrict__ feats, int feat_ld, int N, int C, const int* __restrict__ bk,
    const int* __restrict__ hq, double* __restrict__ hpart) {
    __shared__ double red[256 * 8];
    __shared__ int s_pre[256], s_scan[4];
    const int nq = hq[0];
    const int gpv = C / 8, t = threadIdx.x, G = gridDim.x;
    int chunk_base = 0;
    for (int w0 = 0; w0 < nq; w0 += 256) {
        const int total = heavy_window(hq, nq, w0, s_pre, s_scan);
        int local = (int)(((long)blockIdx.x - chunk_base) % G);
        if (local < 0) local += G;
        for (; local < total; local += G) {
            // the window entry holding chunk `local`: last e with s_pre[e] <= local
            int lo = 0, hi = min(256, nq - w0) - 1;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (s_pre[mid] <= local) lo = mid; else hi = mid - 1;
            }
            const int* e = hq + 1 + 4 * (w0 + lo);
            const int b = e[0], off = e[2], nk = e[3];
            const int p0 = (local - s_pre[lo]) * kChunk, p1 = min(nk, p0 + kChunk);
            const FT* fb = feats + (size_t)b * N * feat_ld;
            const int* list = bk + (size_t)b * N + off;
            double* dst = hpart + (size_t)(chunk_base + local) * C;
            for (int cg0 = 0; cg0 < gpv; cg0 += 256) {
                const int ng = min(256, gpv - cg0);
                const int S = 256 / ng;
                const int sub = t / ng, cl = t % ng;
                if (sub < S) {
                    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                    sum8<FT>(fb, feat_ld, (cg0 + cl) * 8, list, p0 + sub, p1, S, acc);
#pragma unroll
                    for (int i = 0; i < 8; i++) red[(sub * ng + cl) * 8 + i] = acc[i];
                }
                lds_barrier();
                if (t < ng) {
                    double tot[8];
#pragma unroll
                    for (int i = 0; i < 8; i++) tot[i] = red[t * 8 + i];
                    for (int s2 = 1; s2 < S; s2++)
#pragma unroll
                        for (int i = 0; i < 8; i++) tot[i] += red[(s2 * ng + t) * 8 + i];
#pragma unroll
                    for (int i = 0; i < 8; i++) dst[(cg0 + t) * 8 + i] = tot[i];
                }
                lds_barrier();
            }
        }
        chunk_base += total;
    }
}

// The queued voxels' means: voxel q of the queue (workgroup q % gridDim.x)
// adds its chunks' sums in chunk order and writes its grid row.
template <typename GT>
__global__ __launch_bounds__(256) void pv_voxel_heavy_mean_kernel(int C, int R,
                                                                 const int* __restrict__ hq,
                                                                 const double* __restrict__ hpart,
                                                                 GT* __restrict__ grid) {
    __shared__ int s_pre[256], s_scan[4];
    const int nq = hq[0];
    const int V = R * R * R, gpv = C / 8, G = gridDim.x;
    int chunk_base = 0;
    for (int w0 = 0; w0 < nq; w0 += 256) {
        const int total = heavy_window(hq, nq, w0, s_pre, s_scan);
        for (int e = (int)blockIdx.x - w0 % G; e < min(256, nq - w0); e += G) {
            if (e < 0) continue;
            const int* ent = hq + 1 + 4 * (w0 + e);
            const int b = ent[0], vox = ent[1], nk = ent[3];
            const int nch = (nk + kChunk - 1) / kChunk;
            const double* src = hpart + (size_t)(chunk_base + s_pre[e]) * C;
            GT* out = grid + ((size_t)b * V + vox) * C;
            for (int cg = threadIdx.x; cg < gpv; cg += 256) {
                double tot[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                for (int k = 0; k < nch; k++)
#pragma unroll
                    for (int i = 0; i < 8; i++) tot[i] += src[(size_t)k * C + cg * 8 + i];
                float mean[8];
#pragma unroll
                for (int i = 0; i < 8; i++) mean[i] = (float)(tot[i] / (double)nk);
                store8<GT>(out + cg * 8, mean);
            }
        }
        chunk_base += total;
        lds_barrier();
    }
}

template <typename FT, typename GT>
void launch_tiles(const int32_t* ids, const void* feats, int feat_ld, int B, int N, int C, int R,
                  void* grid, int32_t* counts, bool vec, bool zero_rows, const Buckets& bu,
                  hipStream_t s) {
    const TileShape t = tile_shape(B, R * R * R, N);
    if (t.nt == 128)
        launch_tiles_nt<128, FT, GT>(ids, feats, feat_ld, B, N, C, R, t.tv, grid, counts, vec,
                                     zero_rows, bu, s);
    else
        launch_tiles_nt<256, FT, GT>(ids, feats, feat_ld, B, N, C, R, t.tv, grid, counts, vec,
                                     zero_rows, bu, s);
}

// Zero fill byte by byte, for grids the 16-byte path cannot cover.
__global__ __launch_bounds__(256) void pv_zero_elems_kernel(char* __restrict__ p, size_t n) {
    for (size_t i = (size_t)blockIdx.x * 256 + threadIdx.x; i < n; i += (size_t)gridDim.x * 256)
        p[i] = 0;
}

struct VoxWs {
    int32_t* ids;
    float* pnorm;
    SplitWs split;
};

// Workspace: ids [B][N], normalised coordinates [B][N][3], the split
// normalisation's partials and, for large clouds, the tile buckets.
VoxWs carve_ws(void* ws, int B, int N, int R, size_t* bytes) {
    const int G = (N + kNormPts - 1) / kNormPts;
    const int V = R * R * R;
    const TileShape ts = tile_shape(B, V, N);
    const bool large = N > kSmallMaxN;
    size_t off = 0;
    VoxWs w;
    auto take = [&](size_t n) {
        void* q = ws ? (void*)((char*)ws + off) : nullptr;
        off += pv_align256(n);
        return q;
    };
    w.ids = (int32_t*)take((size_t)B * N * sizeof(int32_t));
    w.pnorm = (float*)take((size_t)B * N * 3 * sizeof(float));
    w.split.G = G;
    w.split.pA = (float*)take((size_t)B * G * 3 * sizeof(float));
    w.split.pQ = (long long*)take((size_t)B * G * 3 * sizeof(long long));
    w.split.pM = (double*)take((size_t)B * G * sizeof(double));
    w.split.TV = ts.tv;
    w.split.T = large ? (V + ts.tv - 1) / ts.tv : 0;
    const size_t nt = (size_t)B * w.split.T;
    w.split.tcount = (int*)take(nt * sizeof(int));
    w.split.tcursor = (int*)take(nt * sizeof(int));
    w.split.tstart = (int*)take(nt * sizeof(int));
    w.split.bk = (int*)take(large ? (size_t)B * N * sizeof(int) : 0);
    w.split.br = (int*)take(large ? (size_t)B * N * sizeof(int) : 0);
    // a voxel goes to the queue with more than kExport points
    w.split.hmax = large ? B * (N / (kExport + 1)) : 0;
    w.split.hq = (int*)take(large ? (1 + 4 * (size_t)w.split.hmax) * sizeof(int) : 0);
    // chunks: at most one per kChunk queued points plus one per voxel
    const size_t hchunks = large ? (size_t)w.split.hmax + (size_t)B * N / kChunk : 0;
    w.split.hpart = (double*)take(hchunks * kHeavyMaxC * sizeof(double));
    if (bytes) *bytes = off;
    return w;
}

}  // namespace

size_t pv_voxelize_ws_bytes(int B, int N, int R) {
    size_t bytes = 0;
    carve_ws(nullptr, B, N, R, &bytes);
    return bytes;
}

namespace {

// How a voxelisation call writes the grid: 16-byte rows (vec: the tile kernel
// writes every row, zero rows for empty voxels) or not (the grid is zeroed
// first, by zb workgroups of the first launch, or element by element when
// 16-byte stores cannot cover it).
struct GridPlan {
    bool vec, grid_ok;
    size_t gbytes, n16;
    int zb;
};

GridPlan grid_plan(const void* feats, bool feat_bf16, int feat_ld, int B, int C, int R,
                   const void* grid, bool grid_bf16) {
    GridPlan g;
    const size_t esz_f = feat_bf16 ? 2 : 4, esz_g = grid_bf16 ? 2 : 4;
    g.vec = (C % 8 == 0) && pv_aligned16(feats) && pv_aligned16(grid) &&
            ((size_t)feat_ld * esz_f) % 16 == 0 && ((size_t)C * esz_g) % 16 == 0;
    g.gbytes = (size_t)B * R * R * R * C * esz_g;
    g.n16 = g.gbytes / 16;
    g.grid_ok = pv_aligned16(grid) && g.gbytes % 16 == 0;
    g.zb = (g.grid_ok && !g.vec) ? (int)std::min<size_t>(2048, (g.n16 + 4095) / 4096) : 0;
    return g;
}

// Everything after the voxel indices (and, for large clouds, the tile
// buckets) are known: the tile kernel, then the heavy-voxel kernels.
pvconv_status voxelize_fill(const int32_t* ids, const void* feats, bool feat_bf16, int feat_ld,
                            int B, int N, int C, int R, void* grid, bool grid_bf16,
                            int32_t* counts, const VoxWs& w, const GridPlan& gp,
                            hipStream_t s) {
    const bool vec = gp.vec;
    const Buckets bu = N > kSmallMaxN
                           ? Buckets{w.split.bk, w.split.br, w.split.tcount, w.split.tstart,
                                     w.split.T, vec && C <= kHeavyMaxC ? w.split.hq : nullptr}
                           : Buckets{nullptr, nullptr, nullptr, nullptr, 0, nullptr};
    if (!gp.grid_ok) {
        // a grid that 16-byte stores cannot cover: the plain element kernel
        hipLaunchKernelGGL(pv_zero_elems_kernel, dim3(1024), dim3(256), 0, s, (char*)grid,
                           gp.gbytes);
    }
    // heavy voxels queued by the tiles (large clouds, 16-byte rows)
    const int hgrid = std::min(256, w.split.hmax);
    auto heavy = [&](auto ft, auto gt) {
        typedef decltype(ft) FT;
        typedef decltype(gt) GT;
        if (bu.hq && hgrid > 0) {
            hipLaunchKernelGGL((pv_voxel_heavy_kernel<FT>), dim3(hgrid), dim3(256), 0, s,
                               (const FT*)feats, feat_ld, N, C, w.split.bk, w.split.hq,
                               w.split.hpart);
            hipLaunchKernelGGL((pv_voxel_heavy_mean_kernel<GT>), dim3(hgrid), dim3(256), 0, s, C,
                               R, w.split.hq, w.split.hpart, (GT*)grid);
        }
    };
    if (feat_bf16) {
        if (grid_bf16)
            launch_tiles<uint16_t, uint16_t>(ids, feats, feat_ld, B, N, C, R, grid, counts, vec,
                                             vec, bu, s);
        else
            launch_tiles<uint16_t, float>(ids, feats, feat_ld, B, N, C, R, grid, counts, vec, vec,
                                          bu, s);
    } else {
        if (grid_bf16)
            launch_tiles<float, uint16_t>(ids, feats, feat_ld, B, N, C, R, grid, counts, vec, vec,
                                          bu, s);
        else
            launch_tiles<float, float>(ids, feats, feat_ld, B, N, C, R, grid, counts, vec, vec, bu,
                                       s);
    }
    if (feat_bf16) {
        if (grid_bf16) heavy(uint16_t{}, uint16_t{}); else heavy(uint16_t{}, float{});
    } else {
        if (grid_bf16) heavy(float{}, uint16_t{}); else heavy(float{}, float{});
    }
    return pv_launch_status();
}

}  // namespace

pvconv_status pv_launch_voxelize(const float* coords, const void* feats, bool feat_bf16,
                                 int feat_ld, int B, int N, int C, int R, void* grid,
                                 bool grid_bf16, int32_t* counts, int32_t* vox_id,
                                 float* norm_coords, void* ws, hipStream_t s,
                                 const PvPackJobs* pack) {
    const PvPackJobs jobs = pack ? *pack : PvPackJobs{};
    const int npack = pv_pack_blocks(jobs);
    if (B == 0) {
        pv_launch_pack_conv_weights(jobs, s);
        return pv_launch_status();
    }
    VoxWs w = carve_ws(ws, B, N, R, nullptr);
    int32_t* ids = vox_id ? vox_id : w.ids;
    float* pn = norm_coords ? norm_coords : w.pnorm;
    // Rows of empty voxels are zero. With 16-byte rows the tile kernel writes
    // them itself (each grid row is then written exactly once); otherwise the
    // grid is zeroed first, alongside the normalisation, and the tile kernel
    // overwrites the occupied rows.
    const GridPlan gp = grid_plan(feats, feat_bf16, feat_ld, B, C, R, grid, grid_bf16);
    const int zb = gp.zb;
    const size_t n16 = gp.n16;
    uint4* grid16 = (uint4*)grid;
    if (N <= kSmallMaxN) {
        const int slices = (N + 255) / 256;
        const int nid = slices * B;
        if (nid + npack + zb > 0) {
            const dim3 gi(nid + npack + zb);
            if (N <= 1024)
                hipLaunchKernelGGL(pv_voxel_ids_kernel<4>, gi, dim3(256), 0, s, coords, N, R,
                                   slices, nid, ids, pn, grid16, n16, jobs, npack);
            else if (N <= 2048)
                hipLaunchKernelGGL(pv_voxel_ids_kernel<8>, gi, dim3(256), 0, s, coords, N, R,
                                   slices, nid, ids, pn, grid16, n16, jobs, npack);
            else
                hipLaunchKernelGGL(pv_voxel_ids_kernel<16>, gi, dim3(256), 0, s, coords, N, R,
                                   slices, nid, ids, pn, grid16, n16, jobs, npack);
        }
    } else {
        const int nid = w.split.G * B;
        dim3 g(w.split.G, B);
        hipLaunchKernelGGL(pv_norm_absmax_kernel, dim3(nid + npack + zb), dim3(kNormThreads), 0,
                           s, coords, N, w.split, B, grid16, n16, jobs, npack);
        hipLaunchKernelGGL(pv_norm_sum_kernel, g, dim3(kNormThreads), 0, s, coords, N, w.split);
        hipLaunchKernelGGL(pv_norm_radius_kernel, g, dim3(kNormThreads), 0, s, coords, N, w.split);
        hipLaunchKernelGGL(pv_norm_points_kernel, g, dim3(kNormThreads),
                           (size_t)w.split.T * sizeof(int), s, coords, N, R, w.split, ids, pn);
        hipLaunchKernelGGL(pv_bucket_kernel, g, dim3(kNormThreads),
                           (size_t)2 * w.split.T * sizeof(int), s, ids, N, w.split);
    }
    return voxelize_fill(ids, feats, feat_bf16, feat_ld, B, N, C, R, grid, grid_bf16, counts, w,
                         gp, s);
}

pvconv_status pv_launch_voxelize_from_ids(const int32_t* ids, const void* feats, bool feat_bf16,
                                          int feat_ld, int B, int N, int C, int R, void* grid,
                                          bool grid_bf16, int32_t* counts, void* ws,
                                          hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    VoxWs w = carve_ws(ws, B, N, R, nullptr);
    const GridPlan gp = grid_plan(feats, feat_bf16, feat_ld, B, C, R, grid, grid_bf16);
    uint4* grid16 = (uint4*)grid;
    if (N <= kSmallMaxN) {
        // the tiles scan the indices themselves; only a grid without 16-byte
        // rows needs zeroing first
        if (gp.zb > 0)
            hipLaunchKernelGGL(pv_tile_reset_kernel, dim3(1 + gp.zb), dim3(kNormThreads), 0, s,
                               w.split, 0, grid16, gp.n16);
    } else {
        dim3 g(w.split.G, B);
        hipLaunchKernelGGL(pv_tile_reset_kernel, dim3(1 + gp.zb), dim3(kNormThreads), 0, s,
                           w.split, B, grid16, gp.n16);
        hipLaunchKernelGGL(pv_tile_count_kernel, g, dim3(kNormThreads),
                           (size_t)w.split.T * sizeof(int), s, ids, N, w.split);
        hipLaunchKernelGGL(pv_bucket_kernel, g, dim3(kNormThreads),
                           (size_t)2 * w.split.T * sizeof(int), s, ids, N, w.split);
    }
    return voxelize_fill(ids, feats, feat_bf16, feat_ld, B, N, C, R, grid, grid_bf16, counts, w,
                         gp, s);
}
