// Normalisation and voxelisation (Section 4.1 "Normalization", "Voxelization",
// Eq. 2) for gfx950.
//
// Clouds of up to 4096 points (kSmallMaxN): one launch, pv_voxel_slab_kernel
// (described where it is defined). Each workgroup owns a slab of one cloud's
// grid: it recomputes the cloud's normalisation (order-free, so every
// workgroup gets the same bits), sorts the slab's points by voxel stably and
// averages them in point order, while its writer waves stream the zero rows
// of the empty voxels. Within a voxel the features are summed in point order
// from zero (voxels of up to 16 points, as the oracle sums them; heavier
// ones in a fixed order of subsets), so the grid is the same bits on every
// run.
//
// Larger clouds: the normalisation in four short kernels (abs-max,
// fixed-point sum, radius, points) that pass per-workgroup partial results
// through the workspace, the points bucketed by tile, then one workgroup per
// (cloud, tile of TV voxels) that counting-sorts its bucket by voxel in LDS,
// writes the tile's counts, zero rows for its empty voxels and, for the
// occupied ones, the mean of their features (fp64 sums); voxels of more than
// kExport points go to the heavy-voxel kernels, which spread them over the
// chip in chunks.
// No global float atomics.
#include <algorithm>
#include <mutex>
#include <unordered_map>

#include "pv_common.h"
#include "pv_wave.h"

namespace {

constexpr int kNormPts = 1024;      // points per workgroup, large-cloud normalisation
constexpr int kNormThreads = 256;
constexpr int kSmallMaxN = 4096;    // largest cloud normalised by one kernel
constexpr int kHeavy = 32;          // voxels with more points are summed by a whole wave
constexpr int kExport = 32;         // large clouds: voxels with more points go to the heavy-voxel kernel
constexpr int kChunk = 256;         // points per work item of the heavy-voxel kernel
constexpr int kHeavyMaxC = 128;     // ... for up to this many channels (its sums' workspace)
constexpr int kMaxCap = 4096;       // tile points kept in LDS at once

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

// One axis of a point's normalised coordinates, and its voxel coordinate.
__device__ __forceinline__ int normalise_axis(float p, double c, double M2, double m, int R,
                                              float& pn) {
#pragma clang fp contract(off)
    const double d = (double)p - c;
    const double unit = (M2 == 0.0) ? 0.0 : d / m;
    const double x = unit * 0.5 + 0.5;
    pn = (float)x;
    return voxel_axis(x, R);
}

// Normalised coordinates of one point and its voxel id.
__device__ __forceinline__ int normalise_point(const float* p, const double* c, double M2,
                                               double m, int R, float* pn_out) {
    int uvw[3];
    for (int a = 0; a < 3; a++) uvw[a] = normalise_axis(p[a], c[a], M2, m, R, pn_out[a]);
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
struct MaxF { __device__ float operator()(float a, float b) const { return fmaxf(a, b); } };
struct MaxD { __device__ double operator()(double a, double b) const { return fmax(a, b); } };
struct AddL {
    __device__ long long operator()(long long a, long long b) const { return a + b; }
};

// K values reduced together over an NT-thread workgroup; every thread gets
// the results. lds holds K * NT/64 entries.
// The workgroup's barrier (LDS data only), as a functor.
struct HwSync {
    __device__ void operator()() const { lds_barrier(); }
};

// A barrier among the first NW waves of the workgroup only, on a counter in
// LDS, so that the workgroup's other waves never have to reach it (they may
// be stalled issuing stores). Each arrival adds one; the g-th barrier opens
// when the counter reaches g * NW. The wait is bounded (well under a
// second): a wave that never arrives would be a bug, and the others then go
// on rather than hang.
template <int NW>
struct WaveGroupSync {
    int* ctr;
    int gen;
    __device__ void operator()() {
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
        gen++;
        if ((threadIdx.x & 63) == 0) atomicAdd(ctr, 1);
        for (int spin = 0; spin < (1 << 24); spin++)
            if (__hip_atomic_load(ctr, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) >= gen * NW)
                break;
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    }
};

// trailing: a barrier after the reads too, so that lds may be reused at
// once (not needed when each reduction has LDS of its own)
template <int NT, int K, typename T, typename Op, typename Sync = HwSync>
__device__ void block_reduce_k(T (&v)[K], Op op, T* lds, Sync&& sync = Sync{},
                               bool trailing = true) {
#pragma unroll
    for (int i = 0; i < K; i++) v[i] = wave_reduce(v[i], op);
    const int w = threadIdx.x >> 6;
    if ((threadIdx.x & 63) == 0)
#pragma unroll
        for (int i = 0; i < K; i++) lds[i * (NT / 64) + w] = v[i];
    sync();
#pragma unroll
    for (int i = 0; i < K; i++) {
        T r = lds[i * (NT / 64)];
        for (int j = 1; j < NT / 64; j++) r = op(r, lds[i * (NT / 64) + j]);
        v[i] = r;
    }
    if (trailing) sync();
}

// Inclusive prefix sum over the wave by DPP moves (shifts within rows of 16
// lanes, then the row broadcasts), without cross-lane LDS instructions.
__device__ __forceinline__ int wave_inclusive_scan(int v) {
    v += (int)dpp_u32<0x111, 0xf>((uint32_t)v);  // row_shr:1
    v += (int)dpp_u32<0x112, 0xf>((uint32_t)v);  // row_shr:2
    v += (int)dpp_u32<0x114, 0xf>((uint32_t)v);  // row_shr:4
    v += (int)dpp_u32<0x118, 0xf>((uint32_t)v);  // row_shr:8
    v += (int)dpp_u32<0x142, 0xa>((uint32_t)v);  // row_bcast:15 into rows 1 and 3
    v += (int)dpp_u32<0x143, 0xc>((uint32_t)v);  // row_bcast:31 into rows 2 and 3
    return v;
}

// Exclusive scan of one int per thread over the workgroup; also returns the total.
template <int NT, typename Sync = HwSync>
__device__ int block_exclusive_scan(int v, int* lds /* NT/64 */, int& total, Sync&& sync = Sync{}) {
    const int lane = threadIdx.x & 63, w = threadIdx.x >> 6;
    const int incl = wave_inclusive_scan(v);
    sync();
    if (lane == 63) lds[w] = incl;
    sync();
    int before = 0;
    total = 0;
    for (int i = 0; i < NT / 64; i++) {
        int s = lds[i];
        if (i < w) before += s;
        total += s;
    }
    sync();
    return before + incl - v;
}

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
// bits. Each reduction has LDS of its own, so no barrier follows its reads.
template <int PPT, int NT, typename Sync = HwSync>
__device__ void cloud_params(const float (&x)[PPT][3], int N, double (&c)[3], double& M2,
                             double& m, Sync&& sync = Sync{}) {
    __shared__ float redf[3 * NT / 64];
    __shared__ long long redl[3 * NT / 64];
    __shared__ double redd[NT / 64];
    float A[3] = {0.f, 0.f, 0.f};
#pragma unroll
    for (int i = 0; i < PPT; i++)
#pragma unroll
        for (int a = 0; a < 3; a++) A[a] = fmaxf(A[a], fabsf(x[i][a]));
    block_reduce_k<NT>(A, MaxF(), redf, sync, false);
    int S[3];
    long long q[3] = {0, 0, 0};
#pragma unroll
    for (int a = 0; a < 3; a++) {
        S[a] = fixed_scale(A[a], N);
#pragma unroll
        for (int i = 0; i < PPT; i++)
            if (A[a] > 0.f && threadIdx.x + i * NT < N) q[a] += fixed_term(x[i][a], S[a]);
    }
    block_reduce_k<NT>(q, AddL(), redl, sync, false);
#pragma unroll
    for (int a = 0; a < 3; a++) c[a] = centroid_from_sum(q[a], S[a], A[a], N);
    double mx[1] = {0.0};
#pragma unroll
    for (int i = 0; i < PPT; i++)
        if (threadIdx.x + i * NT < N) mx[0] = fmax(mx[0], sq_dist(x[i], c));
    block_reduce_k<NT>(mx, MaxD(), redd, sync, false);
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
// Slab fill, clouds of up to kSmallMaxN points: the whole voxelisation in one
// launch. Workgroup (s, b) owns the contiguous voxel range [v0, v0 + nv) of
// cloud b (a slab of the grid, v0 = s * nvs). Its waves take two roles.
//  * Compute waves (threads 0 .. kSlabNC-1) recompute the cloud's
//    normalisation from the coordinates (order-free, so every workgroup of
//    the cloud gets the same bits) or read given voxel indices, count the
//    slab's points per voxel and list them in point-index order (ballots
//    and per-wave counts), counting-sort them by voxel stably (one wave, 64
//    points per step), then gather the features of the sorted points into
//    LDS in segments (one round of loads per segment, all in flight) and
//    average each occupied voxel's rows in sorted order in fp64: within a
//    voxel the points are summed in point order from zero, as Eq. 2's
//    oracle sums them, and the grid is the same bits on every run. A voxel
//    with more points than the stage holds is summed from global memory by
//    a whole wave, its points split into subsets whose sums are added in
//    subset order.
//  * A loader wave (threads kSlabLoader ..) streams the slab's feature rows
//    into the LDS stage (global_load_lds, no registers) as soon as the
//    points are listed, while the compute waves sort them, and raises a
//    flag in LDS when they have landed.
//  * Writer waves (the others) store zeros over the rows of the slab's empty
//    voxels and write the slab's counts. Rows that no point can reach go
//    out from the first cycle: a normalised point lies within 1/2 of the
//    cube's centre, so a voxel whose cell is further away stays empty. The
//    other empty rows follow once the counts are known. Compute and writer
//    waves never write the same bytes.
// While the writes stream, issuing a store can stall for microseconds (the
// memory system pushes back), so the two roles share no barrier after the
// first: the compute waves synchronise among themselves on a counter in LDS
// (WaveGroupSync) and the writers wait for the counts on a flag in LDS.
// ---------------------------------------------------------------------------
constexpr int kSlabNC = 512;             // compute threads (eight waves)
constexpr int kSortWaves = 4;            // compute waves that rank the points
constexpr int kSlabLoader = kSlabNC;     // first thread of the loader waves
constexpr int kLoaders = 2;              // loader waves
constexpr int kSplit = 16;               // staged voxels with more points: summed by a whole wave
// threads: kSlabLoader + 64 * kLoaders .. NT-1 write zeros. 1024 (six writer
// waves) for clouds of up to 2048 points, whose compute waves fit in 128
// registers, else 768 (two writer waves)
constexpr int kSlabNT = 1024;
constexpr int kSlabNTSmall = 768;
constexpr int kSlabWGs = 256;            // slabs per launch (one workgroup per CU)
constexpr int kSlabMinVox = 64;          // fewest voxels per slab
constexpr int kSlabMaxVox = 2048;        // most voxels per slab (bounds its LDS)

struct SlabShape {
    int S, nvs;  // slabs per cloud, voxels per slab
};
// The kernel's dynamic LDS is about 17 bytes per slab voxel and 10 per point
// of the cloud; with the static stage it has to fit a CU's 160 KB.
constexpr int kSlabDynBudget = 62 * 1024;
SlabShape slab_shape(int B, int V, int N) {
    const int max_vox =
        std::max(kSlabMinVox, std::min(kSlabMaxVox, (kSlabDynBudget - 10 * std::max(N, 1)) / 17));
    int S = std::max(1, kSlabWGs / std::max(B, 1));
    S = std::min(S, std::max(1, V / kSlabMinVox));
    S = std::max(S, (V + max_vox - 1) / max_vox);
    const int nvs = (V + S - 1) / S;
    return SlabShape{(V + nvs - 1) / nvs, nvs};
}

// LDS of a slab workgroup (byte offsets; 16-bit entries where the values
// fit: N <= 4096 points, nvs <= 2048 voxels):
//  hist[nvs] int, start[nvs + 1], occ[nvs] (occupied voxels in voxel order),
//  sortj[N], sortk[N] (the slab's points sorted by voxel: their position in
//  kbuf, their index), far[nvs] bytes (no point can reach the voxel);
//  then the sort's working set: kbuf[N] (the slab's points in point order),
//  rbuf[N] int (their voxel in the slab, later with their rank),
//  wc[kSortWaves][nvs] (per-wave cursors). All of this is the kernel's
//  dynamic LDS. The feature stage is a static array of its own (kStageBytes, plus 1 KB of slack: the
//  last load of a wave may run past the rows), so that the compiler sees
//  that the loads streaming into it touch none of the tables: raw feature
//  rows go into it straight from global memory, in kbuf order during the
//  sort when the whole slab fits ("pre"), else in segments of the sorted
//  order after it.
struct SlabLayout {
    int hist, start, occ, sortj, sortk, far, kbuf, rbuf, wc, pre;
};
__host__ __device__ inline SlabLayout slab_layout(int nvs, int N) {
    const int N1 = N > 1 ? N : 1;
    auto al = [](int x) { return (x + 15) & ~15; };
    SlabLayout L;
    int o = 0;
    L.hist = o;
    o += 4 * nvs;
    L.start = o;
    o += 2 * (nvs + 1);
    L.occ = o;
    o += 2 * nvs;
    L.sortj = o;
    o += 2 * N1;
    L.sortk = o;
    o += 2 * N1;
    L.far = o;
    o = al(o + nvs);
    L.kbuf = o;
    o += al(2 * N1);
    L.rbuf = o;
    o += al(4 * N1);
    L.wc = o;
    o += al(2 * kSortWaves * nvs);
    L.pre = o;
    return L;
}
constexpr int kStageSlack = 1024;
constexpr int kStageBytes = 96 * 1024;
// A slab with more points than the stage holds, but no more than this many
// beyond it, stages the rest after the sort in the sort's dead tables.
constexpr int kExtRows = 128;

// No normalised point reaches voxel `vox`: its cell lies further than 1/2
// from the cube's centre. Exact integer test in units of 1/(2R): the cell
// spans [2u, 2u + 2] per axis, the centre is at R, the radius R.
__device__ __forceinline__ bool outside_ball(int vox, int R) {
    const int w = vox % R, v = (vox / R) % R, u = vox / (R * R);
    auto gap = [R](int i) { return max(max(2 * i - R, R - 2 * i - 2), 0); };
    const long long du = gap(u), dv = gap(v), dw = gap(w);
    return du * du + dv * dv + dw * dw > (long long)R * R;
}

__device__ __forceinline__ unsigned long long lanes_below() {
    const int lane = threadIdx.x & 63;
    return lane ? (~0ull >> (64 - lane)) : 0ull;
}

// Sum of 8 channels over the points list[j], list[j + step], ... (< j1) in
// that order, fp64, in rounds of U points whose loads are all in flight
// (indices past the end repeat the round's last point and are not added).
template <typename FT, int U, typename IT>
__device__ __forceinline__ void round_sum8(const FT* fb, int feat_ld, int col, const IT* list,
                                           int j, int j1, int step, double* acc) {
    for (; j < j1; j += U * step) {
        const int n = min(U, (j1 - j + step - 1) / step);
        float f[U][8];
#pragma unroll
        for (int u = 0; u < U; u++)
            load8f<FT>(fb + (size_t)list[j + min(u, n - 1) * step] * feat_ld + col, f[u]);
#pragma unroll
        for (int u = 0; u < U; u++)
            if (u < n)
#pragma unroll
                for (int i = 0; i < 8; i++) acc[i] += (double)f[u][i];
    }
}

// A voxel too heavy for the feature stage, by one wave, channel groups cg0 ..
// cg0+ng-1: lane = sub * ng + (cg - cg0) sums points j0 + sub, j0 + sub + S,
// ... (S = 64 / ng subsets); lane cl < ng gets the total of its channel
// group, the S partial sums added in subset order.
template <typename FT, typename IT>
__device__ __forceinline__ void wave_sum8(const FT* fb, int feat_ld, const IT* list, int j0,
                                          int nk, int cg0, int ng, double* tot) {
    const int lane = threadIdx.x & 63;
    const int S = 64 / ng, sub = lane / ng, cl = lane % ng;
    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
    if (sub < S) round_sum8<FT, 4>(fb, feat_ld, (cg0 + cl) * 8, list, j0 + sub, j0 + nk, S, acc);
#pragma unroll
    for (int i = 0; i < 8; i++) tot[i] = __shfl(acc[i], cl, 64);
    for (int s2 = 1; s2 < S; s2++)
#pragma unroll
        for (int i = 0; i < 8; i++) tot[i] += __shfl(acc[i], s2 * ng + cl, 64);
}

// Raw feature rows of FT into the LDS stage at dst, straight from global
// memory (global_load_lds, 16 bytes a lane, the lane's bytes at dst + 16 *
// lane): rows [0, nrows), row r holding the features of point pt(r). Wave
// `wave` of the NC/64 taking part issues every (NC/64)-th 64-piece block;
// the last block's lanes past the end re-load the last piece into the slack.
template <int NC, typename FT, typename PointOf>
__device__ __forceinline__ void dma_rows(char* dst, int nrows, int C, const FT* fb, int feat_ld,
                                         PointOf pt, int wave) {
    const int lane = threadIdx.x & 63;
    const int ppr = C * (int)sizeof(FT) / 16;  // 16-byte pieces per row
    const int npiece = nrows * ppr;
    const bool pow2 = (ppr & (ppr - 1)) == 0;
    const int sh = __ffs(ppr) - 1;
    // U wave-steps at a time: their row indices (LDS reads) first, then the
    // DMAs, so that the index reads' latency is paid once per U steps
    constexpr int U = 8;
    for (int p00 = wave * 64; p00 < npiece; p00 += U * NC) {
        const FT* src[U];
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int pc = min(p00 + u * NC + lane, npiece - 1);
            const int r = pow2 ? pc >> sh : pc / ppr, q = pc - r * ppr;
            src[u] = fb + (size_t)pt(r) * feat_ld + q * (16 / (int)sizeof(FT));
        }
#pragma unroll
        for (int u = 0; u < U; u++) {
            const int p0 = p00 + u * NC;
            if (p0 < npiece)
                __builtin_amdgcn_global_load_lds(
                    (const void __attribute__((address_space(1)))*)src[u],
                    (void __attribute__((address_space(3)))*)(dst + p0 * 16), 16, 0, 0);
        }
    }
}

// 8 channels of a raw feature row in LDS as fp32.
__device__ __forceinline__ void stage8(const float* p, float* v) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void stage8(const uint16_t* p, float* v) {
    const uint4 a = *(const uint4*)p;
    const uint32_t w[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int i = 0; i < 4; i++) {
        v[2 * i] = pv_bf16_to_f32((uint16_t)(w[i] & 0xffffu));
        v[2 * i + 1] = pv_bf16_to_f32((uint16_t)(w[i] >> 16));
    }
}
__device__ __forceinline__ float stage1(const float* p) { return *p; }
__device__ __forceinline__ float stage1(const uint16_t* p) { return pv_bf16_to_f32(*p); }

// VEC: C % 8 == 0 and 16-byte feature rows and grid rows (8 channels at a
// time); else channel by channel. GVEC: grid rows are whole 16-byte pieces
// (the writers' zero stores), else element stores.
template <int PPT, int NT, typename FT, typename GT, bool VEC, bool GVEC>
__global__ __launch_bounds__(NT) void pv_voxel_slab_kernel(
    const float* __restrict__ coords, const int32_t* __restrict__ ids_in,
    const FT* __restrict__ feats, int feat_ld, int N, int C, int R, int nvs, int nslab,
    int cap_pre, GT* __restrict__ grid, int32_t* __restrict__ counts,
    int32_t* __restrict__ vox_id, float* __restrict__ norm_coords, PvPackJobs pack, int npack,
    int sparse) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ __attribute__((aligned(16))) char s_stage[kStageBytes + kStageSlack];
    // compute waves' barrier counter; counts complete; the slab's point count
    // + 1 once listed; loader waves whose rows have landed
    __shared__ int s_ctr, s_counted, s_listed, s_rows_in;
    __shared__ int wcnt[PPT][kSlabNC / 64];
    __shared__ uint16_t s_extk[kExtRows];  // points of list positions cap_pre, cap_pre + 1, ...
    const int bid = blockIdx.x;
    if (bid >= (int)gridDim.x - npack) {  // extra workgroups: conv weight packing
        const int pb = bid - ((int)gridDim.x - npack);
        if (threadIdx.x < 512) pv_pack_role(pack, 2 * pb + (threadIdx.x >= 256), threadIdx.x & 255);
        return;
    }
    constexpr int NC = kSlabNC, NW = NT - kSlabLoader - 64 * kLoaders;
    const int s = bid % nslab, b = bid / nslab;
    const int V = R * R * R;
    const int v0 = s * nvs, nv = min(nvs, V - v0);
    GT* out = grid + ((size_t)b * V + v0) * C;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const SlabLayout LY = slab_layout(nvs, N);
    int* hist = (int*)(smem + LY.hist);
    uint16_t* start = (uint16_t*)(smem + LY.start);
    uint16_t* occ = (uint16_t*)(smem + LY.occ);
    uint16_t* sortj = (uint16_t*)(smem + LY.sortj);
    uint16_t* sortk = (uint16_t*)(smem + LY.sortk);
    unsigned char* far = (unsigned char*)(smem + LY.far);
    uint16_t* kbuf = (uint16_t*)(smem + LY.kbuf);
    int* rbuf = (int*)(smem + LY.rbuf);
    uint16_t* wc = (uint16_t*)(smem + LY.wc);
    // Rows past the stage (slabs of cap_pre < ns <= cap_pre + cap_ext points)
    // go to kbuf .. the end of the dynamic LDS once the sort is done with it,
    // less the slack a wave's last DMA may write past its rows.
    const int cap_ext =
        VEC ? min(kExtRows, max(0, (LY.pre - LY.kbuf - kStageSlack) / (C * (int)sizeof(FT)))) : 0;
    for (int i = tid; i < nvs; i += NT) {
        hist[i] = 0;
        far[i] = !ids_in && i < nv && outside_ball(v0 + i, R);
    }
    if (tid == 0) {
        s_ctr = 0;
        s_counted = 0;
        s_listed = 0;
        s_rows_in = 0;
    }
    lds_barrier();  // the only barrier of the whole workgroup

    // zero stores of the writer waves over the rows of voxels vi with
    // want(vi): 16-byte pieces when the rows are made of them, else elements.
    // Each thread keeps one piece (or element) column q of rows r0, r0 + rs,
    // ..., so that the loop divides nothing, four rows a round (their table
    // reads together); consecutive threads still write consecutive bytes.
    constexpr int W0 = kSlabLoader + 64 * kLoaders;  // first writer thread
    auto zero_rows = [&](auto want) {
        const int wt = tid - W0;
        const int pr = GVEC ? C * (int)sizeof(GT) / 16 : C;  // pieces per row
        const int rs = NW / pr;                              // rows per round
        if (rs > 0) {
            const int q = wt % pr, r0 = wt / pr;
            if (r0 >= rs) return;
            for (int r = r0; r < nv; r += 4 * rs) {
                bool z[4];
#pragma unroll
                for (int u = 0; u < 4; u++) z[u] = r + u * rs < nv && want(r + u * rs);
#pragma unroll
                for (int u = 0; u < 4; u++) {
                    if (!z[u]) continue;
                    const size_t i = (size_t)(r + u * rs) * pr + q;
                    if (GVEC)
                        ((uint4*)out)[i] = make_uint4(0u, 0u, 0u, 0u);
                    else
                        out[i] = (GT)0;
                }
            }
            return;
        }
        for (int i = wt; i < nv * pr; i += NW) {  // rows wider than NW pieces
            if (!want(i / pr)) continue;
            if (GVEC)
                ((uint4*)out)[i] = make_uint4(0u, 0u, 0u, 0u);
            else
                out[i] = (GT)0;
        }
    };
    if (tid >= W0) {
        // writers, before the counts exist: the rows no point can reach
        // (normalised points only; given indices may name any voxel)
        if (!ids_in && !sparse) zero_rows([&](int vi) { return far[vi] != 0; });
        // wait (bounded, well under a second) until the compute waves have counted
        for (int spin = 0; spin < (1 << 23); spin++) {
            if (__hip_atomic_load(&s_counted, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP))
                break;
            __builtin_amdgcn_s_sleep(2);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
        // the other empty rows (sparse: none), then the counts
        if (!sparse) zero_rows([&](int vi) { return hist[vi] == 0 && !far[vi]; });
        for (int v = tid - W0; v < nv; v += NW) counts[(size_t)b * V + v0 + v] = hist[v];
        return;
    }
    // bounded wait (well under a second) for a flag in LDS
    auto wait_flag = [](int* f) {
        for (int spin = 0; spin < (1 << 23); spin++) {
            if (__hip_atomic_load(f, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP)) break;
            __builtin_amdgcn_s_sleep(1);
        }
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    };
    const FT* fb = feats + (size_t)b * N * feat_ld;
    if (tid >= kSlabLoader) {
        // the loader: once the points are listed, the whole slab's rows
        // (when they fit the stage) in point order
        wait_flag(&s_listed);
        const int ns = s_listed - 1;
        if (VEC && ns <= cap_pre + cap_ext)
            dma_rows<64 * kLoaders, FT>(s_stage, min(ns, cap_pre), C, fb, feat_ld,
                                        [&](int r) { return (int)kbuf[r]; }, wave - NC / 64);
        __builtin_amdgcn_s_waitcnt(0);  // this wave's rows have landed
        if (lane == 0) atomicAdd(&s_rows_in, 1);
        return;
    }

    // ---- compute waves ----------------------------------------------------
    WaveGroupSync<NC / 64> sync{&s_ctr, 0};
    // 1. the cloud's points and the voxel ids of those in the slab
    float x[PPT][3];
    int id[PPT];
    if (ids_in) {
#pragma unroll
        for (int i = 0; i < PPT; i++) {
            const int k = tid + i * NC;
            id[i] = k < N ? ids_in[(size_t)b * N + k] : -1;
        }
    } else {
        load_cloud<PPT, NC>(coords + (size_t)b * N * 3, N, x);
        double c[3], M2, m;
        cloud_params<PPT, NC>(x, N, c, M2, m, sync);
        // The slab spans voxel coordinates u in [ulo, uhi]. A point's u is
        // first estimated with d * (1/m) for d / m (within a few units in the
        // last place of the exact quotient, so the estimate's cell is the
        // exact one unless it lies within 1e-9 of a cell face, where the
        // exact division decides). The candidates, the points in the u range,
        // are packed per wave into LDS (the stage, unused until the points
        // are listed) and get their exact normalised coordinates and voxel id
        // there, a full wave at a time; each lane then reads back its own.
        const int ulo = v0 / (R * R), uhi = (v0 + nv - 1) / (R * R);
        const double minv = M2 == 0.0 ? 0.0 : 1.0 / m;
        float4* cbuf = (float4*)s_stage + wave * (PPT * 64);
        const unsigned long long lt = lanes_below();
        int ncand = 0, cpos[PPT];
#pragma unroll
        for (int i = 0; i < PPT; i++) {
            id[i] = -1;
            bool cand = false;
            if (tid + i * NC < N) {
#pragma clang fp contract(off)
                const double xs = (((double)x[i][0] - c[0]) * minv * 0.5 + 0.5) * (double)R;
                const double f = floor(xs);
                int u;
                float pnx;
                if (xs - f < 1e-9 || f + 1.0 - xs < 1e-9)
                    u = normalise_axis(x[i][0], c[0], M2, m, R, pnx);
                else
                    u = (int)fmin(fmax(f, 0.0), (double)(R - 1));
                cand = u >= ulo && u <= uhi;
            }
            const unsigned long long cm = __ballot(cand);
            cpos[i] = cand ? ncand + __popcll(cm & lt) : -1;
            if (cand) cbuf[cpos[i]] = make_float4(x[i][0], x[i][1], x[i][2], 0.f);
            ncand += __popcll(cm);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
        for (int j = lane; j < ((ncand + 63) & ~63); j += 64) {
            if (j >= ncand) continue;
            const float4 p = cbuf[j];
            float pn[3];
            const int u = normalise_axis(p.x, c[0], M2, m, R, pn[0]);
            const int v = normalise_axis(p.y, c[1], M2, m, R, pn[1]);
            const int w = normalise_axis(p.z, c[2], M2, m, R, pn[2]);
            cbuf[j] = make_float4(pn[0], pn[1], pn[2], __int_as_float((u * R + v) * R + w));
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
        // each lane's own candidates; the slab's points get their index and
        // normalised coordinates written now (the compute waves issue no
        // global loads that these stores could hold up)
#pragma unroll
        for (int i = 0; i < PPT; i++) {
            if (cpos[i] < 0) continue;
            const float4 r = cbuf[cpos[i]];
            id[i] = __float_as_int(r.w);
            if (id[i] >= v0 && id[i] < v0 + nv) {
                const float pn[3] = {r.x, r.y, r.z};
                write_point(vox_id, norm_coords, (size_t)b * N + tid + i * NC, id[i], pn);
            }
        }
    }
    // the slab's points in point-index order: register row i of the threads
    // is points [i * NC, (i + 1) * NC); counts per (row, wave), per voxel
    unsigned long long bal[PPT];
#pragma unroll
    for (int i = 0; i < PPT; i++) {
        const int k = tid + i * NC;
        const bool in = k < N && id[i] >= v0 && id[i] < v0 + nv;
        bal[i] = __ballot(in);
        if (lane == 0) wcnt[i][wave] = __popcll(bal[i]);
        if (in) atomicAdd(&hist[id[i] - v0], 1);
    }
    sync();
    if (tid == 0) __hip_atomic_store(&s_counted, 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    int ns = 0;
    {
        const unsigned long long lt = lanes_below();
#pragma unroll
        for (int i = 0; i < PPT; i++) {
            int before = ns;
            for (int w = 0; w < NC / 64; w++) {
                const int cw = wcnt[i][w];
                if (w < wave) before += cw;
                ns += cw;
            }
            if ((bal[i] >> lane) & 1ull) {
                const int pos = before + __popcll(bal[i] & lt);
                kbuf[pos] = (uint16_t)(tid + i * NC);
                rbuf[pos] = id[i] - v0;
                if (pos >= cap_pre && pos < cap_pre + kExtRows)
                    s_extk[pos - cap_pre] = (uint16_t)(tid + i * NC);
            }
        }
        for (int i = tid; i < kSortWaves * nvs; i += NC) wc[i] = 0;
    }
    sync();
    // 2. the loader streams the slab's feature rows into LDS while the
    // points are sorted (when they fit the stage)
    if (tid == 0)
        __hip_atomic_store(&s_listed, ns + 1, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_WORKGROUP);
    const bool pre = VEC && ns <= cap_pre;
    const bool ext = VEC && !pre && ns <= cap_pre + cap_ext;

    // 3. exclusive prefix over the slab's voxels of (points, occupied): hi
    // 16 bits count points (ns <= 4096), lo 16 bits voxels
    int n_occ;
    {
        const int seg = (nv + NC - 1) / NC;
        const int s0 = min(nv, tid * seg), s1 = min(nv, s0 + seg);
        int local = 0;
        for (int i = s0; i < s1; i++) local += (hist[i] << 16) + (hist[i] > 0);
        int total;
        int run = block_exclusive_scan<NC>(local, (int*)wcnt, total, sync);
        for (int i = s0; i < s1; i++) {
            const int h = hist[i];
            start[i] = (uint16_t)(run >> 16);
            if (h > 0) occ[run & 0xffff] = (uint16_t)i;
            run += (h << 16) + (h > 0);
        }
        n_occ = total & 0xffff;
    }
    sync();
    // 4. stable counting sort by voxel. Sort wave w (of kSortWaves) takes the
    // w-th part of the point-ordered list, 64 entries at a time, and ranks
    // each entry among the equal voxels before it in its part (within 64
    // entries: lanes with the same voxel, found by ballots over the voxel's
    // bits; across steps: a cursor per voxel, wc[w]); the rank goes into
    // rbuf's upper bits. Then position = start + the equal voxels of the
    // earlier parts + rank.
    {
        const int quarter = (ns + kSortWaves - 1) / kSortWaves;
        const int j0w = wave < kSortWaves ? wave * quarter : ns;
        const int j1w = min(ns, j0w + quarter);
        int nbits = 0;
        while ((1 << nbits) < nv) nbits++;
        const unsigned long long lt = lanes_below();
        uint16_t* cw = wc + wave * nvs;
        for (int j0 = j0w; j0 < j1w; j0 += 64) {
            const int j = j0 + lane;
            const bool valid = j < j1w;
            const int r = valid ? rbuf[j] : 0;
            unsigned long long same = __ballot(valid);
            for (int bit = 0; bit < nbits; bit++) {
                const unsigned long long ones = __ballot((r >> bit) & 1);
                same &= ((r >> bit) & 1) ? ones : ~ones;
            }
            const int rank = __popcll(same & lt), cnt = __popcll(same);
            const int at = valid ? cw[r] : 0;
            if (valid) rbuf[j] = ((at + rank) << 12) | r;
            __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront", "local");
            if (valid && rank == cnt - 1) cw[r] = (uint16_t)(at + cnt);
            __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront", "local");
        }
        sync();
        for (int j = tid; j < ns; j += NC) {
            const int e = rbuf[j], r = e & 0xfff;
            int pos = start[r] + (e >> 12);
            for (int w2 = 0; (w2 + 1) * quarter <= j; w2++) pos += wc[w2 * nvs + r];
            sortj[pos] = (uint16_t)j;
            sortk[pos] = kbuf[j];
        }
    }
    sync();
    if (pre || ext)  // both loader waves' rows have landed (bounded wait)
        for (int spin = 0; spin < (1 << 23); spin++) {
            if (__hip_atomic_load(&s_rows_in, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP) >=
                kLoaders)
                break;
            __builtin_amdgcn_s_sleep(1);
        }
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
    // ext: the loaders (which read kbuf for their addresses) are done and
    // the sort's tables are dead, so the rest of the slab's rows go there
    const FT* xstage = (const FT*)(smem + LY.kbuf);
    if (ext) {
        dma_rows<NC, FT>(smem + LY.kbuf, ns - cap_pre, C, fb, feat_ld,
                         [&](int r) { return (int)s_extk[r]; }, wave);
        __builtin_amdgcn_s_waitcnt(0);
        sync();
    }

    // 5. means, over the occupied voxels in voxel order. pre: one pass over
    // the prefetched rows (a voxel's rows through sortj). Else in segments
    // whose points (a contiguous run of the sorted list) fit the stage; a
    // voxel with more points than that is summed from global memory by
    // wave 0.
    const int gpv = VEC ? C / 8 : C;  // columns: 8-channel groups, or channels
    // items (o, q): thread tid keeps column q = tid % gpv of voxels o0 + r0,
    // o0 + r0 + rs, ... (rs = NC / gpv; when a row has more columns than
    // there are threads, columns are strided instead)
    const int rs = max(1, NC / gpv);
    const int q0 = gpv <= NC ? tid % gpv : tid, r0 = gpv <= NC ? tid / gpv : 0;
    const bool col_ok = gpv <= NC ? r0 < rs : true;
    const int qstep = gpv <= NC ? gpv : NC;
    // the mean of voxel occ[o] over column q, its rows in the stage at
    // row_of(sorted position): the rows in sorted order (point order), fp64
    auto mean_item = [&](int o, int q, auto rowp) {
        const int v = occ[o], nk = hist[v], p0 = start[v];
        if (VEC) {
            double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
            for (int j = 0; j < nk; j++) {
                float f[8];
                stage8(rowp(p0 + j) + q * 8, f);
#pragma unroll
                for (int i = 0; i < 8; i++) acc[i] += (double)f[i];
            }
            float mean[8];
#pragma unroll
            for (int i = 0; i < 8; i++) mean[i] = (float)(acc[i] / (double)nk);
            store8<GT>(out + (size_t)v * C + q * 8, mean);
        } else {
            double acc = 0.0;
            for (int j = 0; j < nk; j++) acc += (double)stage1(rowp(p0 + j) + q);
            store1<GT>(out + (size_t)v * C + q, (float)(acc / (double)nk));
        }
    };
    // The staged voxels of occ[oa .. ob): those of up to kSplit points one
    // item (o, q) a thread; heavier ones (VEC) one voxel a wave, taken in
    // turn, lane sub * ng + cl summing rows sub, sub + S, ... of column group
    // cg0 + cl (S = 64 / ng subsets), the S sums added in subset order.
    auto staged_means = [&](int oa, int ob, auto rowp) {
        for (int q = q0; col_ok && q < gpv; q += qstep)
            for (int o = oa + r0; o < ob; o += rs)
                if (!VEC || hist[occ[o]] <= kSplit) mean_item(o, q, rowp);
        if (!VEC) return;
        int nheavy = 0;
        for (int o0 = oa; o0 < ob; o0 += 64) {
            const int o = o0 + lane;
            unsigned long long hm = __ballot(o < ob && hist[occ[min(o, ob - 1)]] > kSplit);
            while (hm) {
                const int oh = o0 + __ffsll((long long)hm) - 1;
                hm &= hm - 1;
                if (nheavy++ % (NC / 64) != wave) continue;
                const int v = occ[oh], nk = hist[v], p0 = start[v];
                for (int cg0 = 0; cg0 < gpv; cg0 += 64) {
                    const int ng = min(64, gpv - cg0);
                    const int S = 64 / ng, sub = lane / ng, cl = lane % ng;
                    double acc[8] = {0, 0, 0, 0, 0, 0, 0, 0};
                    if (sub < S)
                        for (int j = sub; j < nk; j += S) {
                            float f[8];
                            stage8(rowp(p0 + j) + (cg0 + cl) * 8, f);
#pragma unroll
                            for (int i = 0; i < 8; i++) acc[i] += (double)f[i];
                        }
                    double tot[8];
#pragma unroll
                    for (int i = 0; i < 8; i++) tot[i] = __shfl(acc[i], cl, 64);
                    for (int s2 = 1; s2 < S; s2++)
#pragma unroll
                        for (int i = 0; i < 8; i++) tot[i] += __shfl(acc[i], s2 * ng + cl, 64);
                    if (lane < ng) {
                        float mean[8];
#pragma unroll
                        for (int i = 0; i < 8; i++) mean[i] = (float)(tot[i] / (double)nk);
                        store8<GT>(out + (size_t)v * C + (cg0 + lane) * 8, mean);
                    }
                }
            }
        }
    };
    const FT* stage = (const FT*)s_stage;
    if (pre) {
        staged_means(0, n_occ, [&](int p) { return stage + (size_t)sortj[p] * C; });
    } else if (ext) {
        staged_means(0, n_occ, [&](int p) {
            const int j = sortj[p];
            return j < cap_pre ? stage + (size_t)j * C : xstage + (size_t)(j - cap_pre) * C;
        });
    } else {
        auto seg_end = [&](int o) { return o < n_occ ? (int)start[occ[o]] : ns; };
        int oa = 0;
        while (oa < n_occ) {
            const int pa = start[occ[oa]];
            // the last ob with seg_end(ob) - pa <= cap_pre (binary search)
            int lo = oa, hi = n_occ;
            while (lo < hi) {
                const int mid = (lo + hi + 1) >> 1;
                if (seg_end(mid) - pa <= cap_pre) lo = mid; else hi = mid - 1;
            }
            const int ob = lo;
            if (ob == oa) {
                // one voxel beyond the stage: wave 0 sums it from global memory
                const int v = occ[oa], nk = hist[v];
                if (wave == 0) {
                    for (int cg0 = 0; cg0 < gpv; cg0 += 64) {
                        const int ng = min(64, gpv - cg0);
                        if (VEC) {
                            double tot[8];
                            wave_sum8<FT>(fb, feat_ld, sortk, pa, nk, cg0, ng, tot);
                            if (lane < ng) {
                                float mean[8];
#pragma unroll
                                for (int i = 0; i < 8; i++) mean[i] = (float)(tot[i] / (double)nk);
                                store8<GT>(out + (size_t)v * C + (cg0 + lane) * 8, mean);
                            }
                        } else if (lane < ng) {
                            double acc = 0.0;
                            for (int j = pa; j < pa + nk; j++)
                                acc += (double)load1<FT>(fb + (size_t)sortk[j] * feat_ld + cg0 + lane);
                            store1<GT>(out + (size_t)v * C + cg0 + lane, (float)(acc / (double)nk));
                        }
                    }
                }
                oa++;
                continue;
            }
            const int np = seg_end(ob) - pa;
            if (VEC) {
                dma_rows<NC, FT>(s_stage, np, C, fb, feat_ld,
                                 [&](int r) { return (int)sortk[pa + r]; }, wave);
                __builtin_amdgcn_s_waitcnt(0);
            } else {
                // channel by channel: column q of rows r0, r0 + rs, ...
                FT* st = (FT*)s_stage;
                for (int q = q0; col_ok && q < gpv; q += qstep)
                    for (int r = r0; r < np; r += rs)
                        st[(size_t)r * C + q] = fb[(size_t)sortk[pa + r] * feat_ld + q];
            }
            sync();
            staged_means(oa, ob, [&](int p) { return stage + (size_t)(p - pa) * C; });
            sync();  // the stage is free again
            oa = ob;
        }
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

// One of the tile's points (index k, voxel r in the tile): count it per
// voxel and keep (index, voxel) while they fit.
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
// tile's bucket (for the segmented passes, when the tile holds more than
// CAP points).
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

// Tile fill of a large cloud whose points are bucketed by tile: one
// workgroup per (tile t, cloud b) reads its bucket.
template <int NT, typename FT, typename GT, bool VEC>
__global__ __launch_bounds__(NT) void pv_voxel_tile_kernel(
    const FT* __restrict__ feats, int feat_ld, int N, int C, int R, int TV, int CAP,
    int stage_bytes, int zero_rows, GT* __restrict__ grid, int32_t* __restrict__ counts,
    int* bk, const int* __restrict__ br, const int* __restrict__ tcount,
    const int* __restrict__ tstart, int T, int* hq) {
    extern __shared__ __attribute__((aligned(16))) char smem[];
    __shared__ int scan_lds[NT / 64];
    __shared__ int s_ntile, s_nheavy;
    const TileLds L = tile_lds(smem, TV, CAP);

    const int t = blockIdx.x, b = blockIdx.y;
    const int bstart = tstart[(size_t)b * T + t];
    const int btotal = tcount[(size_t)b * T + t];
    const int V = R * R * R;
    const int v0 = t * TV, nv = min(TV, V - v0);
    const FT* fb = feats + (size_t)b * N * feat_ld;
    GT* out = grid + ((size_t)b * V + v0) * C;

    for (int i = threadIdx.x; i < TV; i += NT) L.hist[i] = 0;
    if (threadIdx.x == 0) s_ntile = 0;
    lds_barrier();
    // 1. the tile's points: its bucket, as (index, voxel - v0)
    const int* kb = bk + (size_t)b * N + bstart;
    const int* rb = br + (size_t)b * N + bstart;
    auto each_point = [&](auto fn) {
        for (int j = threadIdx.x; j < btotal; j += NT) fn(kb[j], rb[j]);
    };
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
    lds_barrier();
    const HeavyOut ho{hq, bk + (size_t)b * N + bstart, b, v0, bstart};
    tile_finish<NT, FT, GT, VEC>(L, TV, nv, CAP, counts + (size_t)b * V + v0, out, fb, feat_ld, C,
                                 zero_rows != 0, stage_bytes, scan_lds, &s_nheavy, each_point, ho);
}

// Dynamic LDS beyond 64 KB is granted per kernel (once per kernel and size:
// a launch being captured into a graph then makes no other call).
bool grant_lds(const void* kernel, size_t bytes) {
    if (bytes <= 65536) return true;
    static std::mutex mu;
    static std::unordered_map<const void*, size_t> granted;
    std::lock_guard<std::mutex> lock(mu);
    auto it = granted.find(kernel);
    if (it != granted.end() && bytes <= it->second) return true;
    if (hipFuncSetAttribute(kernel, hipFuncAttributeMaxDynamicSharedMemorySize, (int)bytes) !=
        hipSuccess) {
        (void)hipGetLastError();
        return false;
    }
    granted[kernel] = std::max(granted[kernel], bytes);
    return true;
}

// Tile shape of a large cloud (points bucketed by tile beforehand): about
// 1024 tiles of 256 threads, so that a dense cluster spreads over several
// workgroups.
constexpr int kTileNT = 256;
int tile_voxels(int B, int V) {
    int tv = 1024;
    while (tv > 32 && (long long)B * ((V + tv - 1) / tv) < 1024) tv >>= 1;
    return tv;
}

// LDS of the tile kernel: no feature stage (each (voxel, channel group) sums
// straight from memory) and room for kMaxCap of the tile's points, tiles
// with more points taking the segmented path. Dynamic LDS beyond 64 KB is
// granted per kernel; when that fails the capacity shrinks to what 64 KB
// holds.
template <typename K>
void tile_budget(K kernel, int NT, int TV, int N, int& cap) {
    cap = N < kMaxCap ? (N > 0 ? N : 1) : kMaxCap;
    if (grant_lds((const void*)kernel, tile_lds_bytes(NT, TV, cap, 0))) return;
    while (cap > 1 && tile_lds_bytes(NT, TV, cap, 0) > 65536) cap >>= 1;
}

// The points bucketed by tile.
struct Buckets {
    int* bk;
    const int* br;
    const int* tcount;
    const int* tstart;
    int T;
    int* hq;  // heavy-voxel queue (nullptr: none)
};

template <typename FT, typename GT>
void launch_tiles(const void* feats, int feat_ld, int B, int N, int C, int R, void* grid,
                  int32_t* counts, bool vec, const Buckets& bu, hipStream_t s) {
    const int V = R * R * R, TV = tile_voxels(B, V);
    dim3 g((V + TV - 1) / TV, B);
    int cap;
    if (vec) {
        auto k = pv_voxel_tile_kernel<kTileNT, FT, GT, true>;
        tile_budget(k, kTileNT, TV, N, cap);
        hipLaunchKernelGGL(k, g, dim3(kTileNT), tile_lds_bytes(kTileNT, TV, cap, 0), s,
                           (const FT*)feats, feat_ld, N, C, R, TV, cap, 0, 1, (GT*)grid, counts,
                           bu.bk, bu.br, bu.tcount, bu.tstart, bu.T, bu.hq);
    } else {
        auto k = pv_voxel_tile_kernel<kTileNT, FT, GT, false>;
        tile_budget(k, kTileNT, TV, N, cap);
        hipLaunchKernelGGL(k, g, dim3(kTileNT), tile_lds_bytes(kTileNT, TV, cap, 0), s,
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
    const bool large = N > kSmallMaxN;
    const int TV = tile_voxels(B, V);
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
    w.split.TV = TV;
    w.split.T = large ? (V + TV - 1) / TV : 0;
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

// A large cloud once its voxel indices and tile buckets are known: the tile
// kernel, then the heavy-voxel kernels.
pvconv_status voxelize_fill(const void* feats, bool feat_bf16, int feat_ld, int B, int N, int C,
                            int R, void* grid, bool grid_bf16, int32_t* counts, const VoxWs& w,
                            const GridPlan& gp, hipStream_t s) {
    const bool vec = gp.vec;
    const Buckets bu{w.split.bk, w.split.br, w.split.tcount, w.split.tstart, w.split.T,
                     vec && C <= kHeavyMaxC ? w.split.hq : nullptr};
    if (!gp.grid_ok) {
        // a grid that 16-byte stores cannot cover: the plain element kernel
        hipLaunchKernelGGL(pv_zero_elems_kernel, dim3(1024), dim3(256), 0, s, (char*)grid,
                           gp.gbytes);
    }
    // heavy voxels queued by the tiles (16-byte rows)
    const int hgrid = std::min(256, w.split.hmax);
    auto run = [&](auto ft, auto gt) {
        typedef decltype(ft) FT;
        typedef decltype(gt) GT;
        launch_tiles<FT, GT>(feats, feat_ld, B, N, C, R, grid, counts, vec, bu, s);
        if (bu.hq && hgrid > 0) {
            hipLaunchKernelGGL((pv_voxel_heavy_kernel<FT>), dim3(hgrid), dim3(256), 0, s,
                               (const FT*)feats, feat_ld, N, C, w.split.bk, w.split.hq,
                               w.split.hpart);
            hipLaunchKernelGGL((pv_voxel_heavy_mean_kernel<GT>), dim3(hgrid), dim3(256), 0, s, C,
                               R, w.split.hq, w.split.hpart, (GT*)grid);
        }
    };
    if (feat_bf16) {
        if (grid_bf16) run(uint16_t{}, uint16_t{}); else run(uint16_t{}, float{});
    } else {
        if (grid_bf16) run(float{}, uint16_t{}); else run(float{}, float{});
    }
    return pv_launch_status();
}

}  // namespace

namespace {


// Clouds of up to kSmallMaxN points: the slab kernel does the whole
// voxelisation (ids_in given: from those voxel indices, no normalisation).
// Its LDS holds the slab's points and per-voxel tables, then as many staged
// mean rows as fit in a CU's 160 KB.
template <typename FT, typename GT, bool VEC, bool GVEC>
pvconv_status launch_slab_t(const float* coords, const int32_t* ids_in, const void* feats,
                            int feat_ld, int B, int N, int C, int R, void* grid, int32_t* counts,
                            int32_t* vox_id, float* pn, const PvPackJobs& jobs, bool sparse,
                            hipStream_t s) {
    const int V = R * R * R;
    const SlabShape sh = slab_shape(B, V, N);
    const int npack = (pv_pack_blocks(jobs) + 1) / 2;
    // dynamic LDS: the tables and the sort's working set (at most ~57 KB for
    // nvs <= 2048, N <= 4096, next to the kernel's 97 KB static stage); the
    // stage holds cap_pre raw feature rows
    const SlabLayout LY = slab_layout(sh.nvs, N);
    const size_t row = (size_t)C * sizeof(FT);
    const int cap_pre = (int)std::min((size_t)kStageBytes / row, (size_t)std::max(N, 1));
    const size_t bytes = (size_t)LY.pre;
    const dim3 g((unsigned)((size_t)B * sh.S + npack));
    auto go = [&](auto kernel, int nt) {
        if (!grant_lds((const void*)kernel, bytes)) return PVCONV_EHIP;
        hipLaunchKernelGGL(kernel, g, dim3(nt), bytes, s, coords, ids_in, (const FT*)feats,
                           feat_ld, N, C, R, sh.nvs, sh.S, cap_pre, (GT*)grid, counts, vox_id,
                           pn, jobs, npack, (int)sparse);
        return pv_launch_status();
    };
    // points per compute thread: the cloud over kSlabNC threads
    static_assert(kSlabNC == 512, "points per compute thread below assume 512 threads");
    if (N <= 1024) return go(pv_voxel_slab_kernel<2, kSlabNT, FT, GT, VEC, GVEC>, kSlabNT);
    if (N <= 2048) return go(pv_voxel_slab_kernel<4, kSlabNT, FT, GT, VEC, GVEC>, kSlabNT);
    return go(pv_voxel_slab_kernel<8, kSlabNTSmall, FT, GT, VEC, GVEC>, kSlabNTSmall);
}

pvconv_status launch_slab(const float* coords, const int32_t* ids_in, const void* feats,
                          bool feat_bf16, int feat_ld, int B, int N, int C, int R, void* grid,
                          bool grid_bf16, int32_t* counts, int32_t* vox_id, float* pn, bool vec,
                          const PvPackJobs& jobs, bool sparse, hipStream_t s) {
    // zero stores of whole 16-byte pieces need 16-byte grid rows
    const bool gvec = pv_aligned16(grid) && (C * (grid_bf16 ? 2 : 4)) % 16 == 0;
    // (vec implies 16-byte grid rows)
#define PV_SLAB(FT, GT)                                                                        \
    if (vec)                                                                                   \
        return launch_slab_t<FT, GT, true, true>(coords, ids_in, feats, feat_ld, B, N, C, R,   \
                                                 grid, counts, vox_id, pn, jobs, sparse, s);   \
    if (gvec)                                                                                  \
        return launch_slab_t<FT, GT, false, true>(coords, ids_in, feats, feat_ld, B, N, C, R,  \
                                                  grid, counts, vox_id, pn, jobs, sparse, s);  \
    return launch_slab_t<FT, GT, false, false>(coords, ids_in, feats, feat_ld, B, N, C, R,     \
                                               grid, counts, vox_id, pn, jobs, sparse, s)
    if (feat_bf16) {
        if (grid_bf16) {
            PV_SLAB(uint16_t, uint16_t);
        }
        PV_SLAB(uint16_t, float);
    }
    if (grid_bf16) {
        PV_SLAB(float, uint16_t);
    }
    PV_SLAB(float, float);
#undef PV_SLAB
}

}  // namespace

pvconv_status pv_launch_voxelize(const float* coords, const void* feats, bool feat_bf16,
                                 int feat_ld, int B, int N, int C, int R, void* grid,
                                 bool grid_bf16, int32_t* counts, int32_t* vox_id,
                                 float* norm_coords, void* ws, hipStream_t s,
                                 const PvPackJobs* pack, bool sparse) {
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
    if (N <= kSmallMaxN)
        return launch_slab(coords, nullptr, feats, feat_bf16, feat_ld, B, N, C, R, grid,
                           grid_bf16, counts, ids, pn, gp.vec, jobs, sparse, s);
    const int zb = gp.zb;
    const size_t n16 = gp.n16;
    uint4* grid16 = (uint4*)grid;
    {
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
    return voxelize_fill(feats, feat_bf16, feat_ld, B, N, C, R, grid, grid_bf16, counts, w, gp, s);
}

pvconv_status pv_launch_voxelize_from_ids(const int32_t* ids, const void* feats, bool feat_bf16,
                                          int feat_ld, int B, int N, int C, int R, void* grid,
                                          bool grid_bf16, int32_t* counts, void* ws,
                                          hipStream_t s, bool sparse) {
    if (B == 0) return PVCONV_OK;
    VoxWs w = carve_ws(ws, B, N, R, nullptr);
    const GridPlan gp = grid_plan(feats, feat_bf16, feat_ld, B, C, R, grid, grid_bf16);
    uint4* grid16 = (uint4*)grid;
    if (N <= kSmallMaxN)
        return launch_slab(nullptr, ids, feats, feat_bf16, feat_ld, B, N, C, R, grid, grid_bf16,
                           counts, nullptr, nullptr, gp.vec, PvPackJobs{}, sparse, s);
    {
        dim3 g(w.split.G, B);
        hipLaunchKernelGGL(pv_tile_reset_kernel, dim3(1 + gp.zb), dim3(kNormThreads), 0, s,
                           w.split, B, grid16, gp.n16);
        hipLaunchKernelGGL(pv_tile_count_kernel, g, dim3(kNormThreads),
                           (size_t)w.split.T * sizeof(int), s, ids, N, w.split);
        hipLaunchKernelGGL(pv_bucket_kernel, g, dim3(kNormThreads),
                           (size_t)2 * w.split.T * sizeof(int), s, ids, N, w.split);
    }
    return voxelize_fill(feats, feat_bf16, feat_ld, B, N, C, R, grid, grid_bf16, counts, w, gp, s);
}

bool pv_voxelize_sparse_ok(int N) { return N <= kSmallMaxN; }
