// The PointNet++ primitives that PVCNN++ keeps around its PVConv layers
// (Section 5.2 "Models": PointNet++ extended with PVConv), as PointNet++
// defines them: iterative farthest point sampling and ball-query grouping
// (set abstraction), and inverse-distance interpolation over the three
// nearest neighbours (feature propagation). gfx950, wave64.
//
// Every choice of an index (the farthest point, ball membership, the three
// nearest neighbours) compares fp32 squared distances formed as
// fma(dz, dz, fma(dy, dy, dx * dx)), dx = x_j - x_c, with ties going to the
// lower index: the same choices on every run and in every launch
// configuration.
#include "pv_common.h"
#include "pv_wave.h"

namespace {

__device__ __forceinline__ float sqdist(float ax, float ay, float az, float bx, float by,
                                        float bz) {
#pragma clang fp contract(off)
    const float dx = ax - bx, dy = ay - by, dz = az - bz;
    return __builtin_fmaf(dz, dz, __builtin_fmaf(dy, dy, dx * dx));
}

struct MaxU32 {
    __device__ uint32_t operator()(uint32_t a, uint32_t b) const { return a > b ? a : b; }
};

// ---------------------------------------------------------------------------
// Farthest point sampling, one workgroup of NT threads per cloud. Thread t
// keeps points t, t + NT, ... (PPT of them) and their distance to the samples
// taken so far in registers. Each step: update those distances with the last
// sample and take the thread's farthest point (the lowest index among equals:
// the thread's points come in index order and only a strictly larger distance
// replaces); then the wave's: the maximum distance over the wave, the lanes
// holding it by ballot, and among several such lanes the lowest index (rare:
// a second reduction over the indices); then the workgroup's through one LDS
// slot per wave. TAB (clouds of up to kFpsTab points): the cloud's
// coordinates sit in an LDS table, and the winner's are read from it by
// index; otherwise each thread also carries its farthest point's coordinates
// and the winning lane writes them to its slot. The slots alternate between
// two buffers so that one barrier per step suffices: step s+2 writes the
// buffer step s read only after every wave has passed the barrier of step
// s+1, which follows those reads.
// ---------------------------------------------------------------------------
constexpr int kFpsTab = 8192;

template <int PPT, int NT, bool TAB>
__global__ __launch_bounds__(NT) void pv_fps_kernel(const float* __restrict__ xyz, int N,
                                                    int npoint, int32_t* __restrict__ idx,
                                                    float* __restrict__ new_xyz) {
    constexpr int NW = NT / 64;
    __shared__ float s_d[2][NW];
    __shared__ int s_j[2][NW];
    __shared__ float s_pt[2][NW][4];
    __shared__ float s_tab[TAB ? 3 * kFpsTab : 1];
    const int b = blockIdx.x, tid = threadIdx.x, lane = tid & 63, w = tid >> 6;
    const float* p = xyz + (size_t)b * N * 3;
    float px[PPT], py[PPT], pz[PPT], dmin[PPT];
#pragma unroll
    for (int k = 0; k < PPT; k++) {
        const int j = tid + k * NT;
        const bool ok = j < N;
        const float* q = p + (size_t)(ok ? j : 0) * 3;
        px[k] = q[0];
        py[k] = q[1];
        pz[k] = q[2];
        dmin[k] = ok ? INFINITY : -1.f;  // -1: never the farthest
        if (TAB && ok) {  // the table is only read for TAB
            s_tab[j] = px[k];
            s_tab[kFpsTab + j] = py[k];
            s_tab[2 * kFpsTab + j] = pz[k];
        }
    }
    float lx = p[0], ly = p[1], lz = p[2];
    int32_t* out = idx + (size_t)b * npoint;
    float* oxyz = new_xyz ? new_xyz + (size_t)b * npoint * 3 : nullptr;
    if (tid == 0) {
        out[0] = 0;
        if (oxyz) {
            oxyz[0] = lx;
            oxyz[1] = ly;
            oxyz[2] = lz;
        }
    }
    if (TAB) pv_lds_barrier();
    for (int s = 1; s < npoint; s++) {
        float bestd = -1.f, bx = 0.f, by = 0.f, bz = 0.f;
        int bestj = 0;
#pragma unroll
        for (int k = 0; k < PPT; k++) {
            dmin[k] = fminf(dmin[k], sqdist(px[k], py[k], pz[k], lx, ly, lz));
            const bool better = dmin[k] > bestd;  // strict: the lower index stays
            bestd = better ? dmin[k] : bestd;
            bestj = better ? tid + k * NT : bestj;
            if constexpr (!TAB) {
                bx = better ? px[k] : bx;
                by = better ? py[k] : by;
                bz = better ? pz[k] : bz;
            }
        }
        // the wave's farthest point: a maximum over the distances' bits
        // (distances are >= 0, so their bits order as their values), offset
        // by one so that 0 means "no point" (the reduction fills lanes it
        // leaves out with 0); then the lanes holding it by ballot
        const uint32_t key = bestd >= 0.f ? __float_as_uint(bestd) + 1u : 0u;
        const uint32_t wkey = wave_reduce(key, MaxU32{});
        const uint64_t hold = __ballot(key != 0u && key == wkey);
        int wj = 0x7fffffff;
        float wd = -1.f;
        if (hold != 0ull) {
            wd = __uint_as_float(wkey - 1u);
            if ((hold & (hold - 1ull)) == 0ull) {  // one lane
                wj = __builtin_amdgcn_readlane(bestj, __ffsll((long long)hold) - 1);
            } else {  // equal distances in several lanes: the lowest index
                const uint32_t jk = (hold >> lane) & 1ull ? 0xffffffffu - (uint32_t)bestj : 0u;
                wj = (int)(0xffffffffu - wave_reduce(jk, MaxU32{}));
            }
        }
        const int buf = s & 1;
        if (lane == 0) {
            s_d[buf][w] = wd;
            s_j[buf][w] = wj;
        }
        if constexpr (!TAB) {
            if (bestj == wj && wd >= 0.f) {  // the one lane that holds it
                s_pt[buf][w][0] = bx;
                s_pt[buf][w][1] = by;
                s_pt[buf][w][2] = bz;
            }
        }
        pv_lds_barrier();
        float best = s_d[buf][0];
        int bj = s_j[buf][0], bw = 0;
#pragma unroll
        for (int i = 1; i < NW; i++) {
            const float d = s_d[buf][i];
            const int j = s_j[buf][i];
            if (d > best || (d == best && j < bj)) {
                best = d;
                bj = j;
                bw = i;
            }
        }
        if constexpr (TAB) {
            lx = s_tab[bj];
            ly = s_tab[kFpsTab + bj];
            lz = s_tab[2 * kFpsTab + bj];
        } else {
            lx = s_pt[buf][bw][0];
            ly = s_pt[buf][bw][1];
            lz = s_pt[buf][bw][2];
        }
        if (tid == 0) {
            out[s] = bj;
            if (oxyz) {
                oxyz[(size_t)s * 3] = lx;
                oxyz[(size_t)s * 3 + 1] = ly;
                oxyz[(size_t)s * 3 + 2] = lz;
            }
        }
    }
}

// ---------------------------------------------------------------------------
// Ball query, one wave per centre: the wave scans the cloud in index order,
// kU chunks of 64 points per round (their loads in flight together), and
// keeps the first nsample points inside the ball in that order (ballot, then
// each lane's rank among the lanes below it). All control is wave-uniform.
// ---------------------------------------------------------------------------
constexpr int kBallWaves = 4;
constexpr int kBallU = 4;

__global__ __launch_bounds__(kBallWaves * 64) void pv_ball_query_kernel(
    const float* __restrict__ xyz, int N, const float* __restrict__ centers, int M,
    int total, float r2, int nsample, int32_t* __restrict__ idx) {
    const int lane = threadIdx.x & 63;
    const int q = blockIdx.x * kBallWaves + (threadIdx.x >> 6);
    if (q >= total) return;  // the whole wave
    const int b = q / M;
    const float* p = xyz + (size_t)b * N * 3;
    const float cx = centers[(size_t)q * 3], cy = centers[(size_t)q * 3 + 1],
                cz = centers[(size_t)q * 3 + 2];
    int32_t* out = idx + (size_t)q * nsample;
    const uint64_t below = (1ull << lane) - 1ull;
    int cnt = 0, first = -1;
    for (int base = 0; base < N && cnt < nsample; base += 64 * kBallU) {
        float x[kBallU], y[kBallU], z[kBallU];
#pragma unroll
        for (int u = 0; u < kBallU; u++) {
            const int j = min(base + u * 64 + lane, N - 1);
            x[u] = p[(size_t)j * 3];
            y[u] = p[(size_t)j * 3 + 1];
            z[u] = p[(size_t)j * 3 + 2];
        }
#pragma unroll
        for (int u = 0; u < kBallU; u++) {
            const int j = base + u * 64 + lane;
            const bool in = j < N && sqdist(x[u], y[u], z[u], cx, cy, cz) < r2;
            const uint64_t m = __ballot(in);
            if (m != 0ull) {
                const int pos = cnt + __popcll(m & below);
                if (in && pos < nsample) out[pos] = j;
                if (first < 0) first = base + u * 64 + __ffsll((long long)m) - 1;
                cnt += __popcll(m);
            }
        }
    }
    const int fill = first >= 0 ? first : 0;
    for (int k = min(cnt, nsample) + lane; k < nsample; k += 64) out[k] = fill;
}

// ---------------------------------------------------------------------------
// Grouping: row (q, k) of the output holds the neighbour j = idx[q][k]'s
// coordinates relative to centre q, then its C features. One thread per
// output element, channels fastest (coalesced stores).
// ---------------------------------------------------------------------------
template <typename FT, typename OT>
__global__ __launch_bounds__(256) void pv_group_kernel(
    const float* __restrict__ xyz, const FT* __restrict__ feats, int feat_ld, int N, int C,
    const float* __restrict__ centers, int M, const int32_t* __restrict__ idx, int nsample,
    OT* __restrict__ out, int out_ld, size_t total) {
    const int W = 3 + C;
    for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total;
         e += (size_t)gridDim.x * 256) {
        const size_t row = e / W;
        const int c = (int)(e - row * W);
        const size_t q = row / nsample;
        const int b = (int)(q / M);
        const int j = min(max(idx[row], 0), N - 1);
        float v;
        if (c < 3)
            v = xyz[((size_t)b * N + j) * 3 + c] - centers[q * 3 + c];
        else if constexpr (sizeof(FT) == 2)
            v = pv_bf16_to_f32(feats[((size_t)b * N + j) * feat_ld + (c - 3)]);
        else
            v = feats[((size_t)b * N + j) * feat_ld + (c - 3)];
        if constexpr (sizeof(OT) == 2)
            out[row * out_ld + c] = pv_f32_to_bf16(v);
        else
            out[row * out_ld + c] = v;
    }
}

// ---------------------------------------------------------------------------
// Three nearest neighbours: kNnLanes lanes per unknown point, each scanning
// every kNnLanes-th known point (the cloud's known points pass through LDS
// in tiles) and keeping its three nearest in (distance, index) order: a
// strictly smaller distance moves ahead, and the lane's candidates come in
// index order, so among equals the lower index stays in front. The lanes'
// lists are then merged pairwise by shuffles in the same (distance, index)
// order. Then the normalised inverse-distance weights, in fp32.
// ---------------------------------------------------------------------------
constexpr int kNnThreads = 256;
constexpr int kNnLanes = 4;
constexpr int kNnPoints = kNnThreads / kNnLanes;  // unknown points per workgroup
constexpr int kNnTile = 1024;

struct Near3 {
    float d[3];
    int i[3];
};
// (d, i) lexicographic order
__device__ __forceinline__ bool nn_less(float da, int ia, float db, int ib) {
    return da < db || (da == db && ia < ib);
}
__device__ __forceinline__ void nn_insert(Near3& n, float d, int i) {
    if (nn_less(d, i, n.d[2], n.i[2])) {
        if (nn_less(d, i, n.d[1], n.i[1])) {
            n.d[2] = n.d[1];
            n.i[2] = n.i[1];
            if (nn_less(d, i, n.d[0], n.i[0])) {
                n.d[1] = n.d[0];
                n.i[1] = n.i[0];
                n.d[0] = d;
                n.i[0] = i;
            } else {
                n.d[1] = d;
                n.i[1] = i;
            }
        } else {
            n.d[2] = d;
            n.i[2] = i;
        }
    }
}

__global__ __launch_bounds__(kNnThreads) void pv_three_nn_kernel(
    const float* __restrict__ unknown, int n, const float* __restrict__ known, int m,
    int32_t* __restrict__ idx, float* __restrict__ weight) {
    __shared__ float s_k[kNnTile * 3];
    const int b = blockIdx.y;
    const int q = threadIdx.x % kNnLanes;  // this lane's share of the candidates
    const int i = blockIdx.x * kNnPoints + threadIdx.x / kNnLanes;
    const bool active = i < n;
    const float* u = unknown + ((size_t)b * n + (active ? i : 0)) * 3;
    const float ux = u[0], uy = u[1], uz = u[2];
    const float* kp = known + (size_t)b * m * 3;
    Near3 nn{{INFINITY, INFINITY, INFINITY}, {0x7fffffff, 0x7fffffff, 0x7fffffff}};
    for (int t0 = 0; t0 < m; t0 += kNnTile) {
        const int cnt = min(kNnTile, m - t0);
        pv_lds_barrier();  // the previous tile's reads are done
        for (int e = threadIdx.x; e < cnt * 3; e += kNnThreads) s_k[e] = kp[(size_t)t0 * 3 + e];
        pv_lds_barrier();
        for (int j = q; j < cnt; j += kNnLanes) {
            const float d = sqdist(s_k[j * 3], s_k[j * 3 + 1], s_k[j * 3 + 2], ux, uy, uz);
            if (d < nn.d[2]) nn_insert(nn, d, t0 + j);  // a strict < keeps the earlier index
        }
    }
    // merge with the other lanes of this point (xor 1, then xor 2)
#pragma unroll
    for (int off = 1; off < kNnLanes; off <<= 1) {
        float od[3];
        int oi[3];
#pragma unroll
        for (int k = 0; k < 3; k++) {
            od[k] = __shfl_xor(nn.d[k], off, 64);
            oi[k] = __shfl_xor(nn.i[k], off, 64);
        }
#pragma unroll
        for (int k = 0; k < 3; k++) nn_insert(nn, od[k], oi[k]);
    }
    if (!active || q != 0) return;
    const float a0 = 1.f / (sqrtf(nn.d[0]) + 1e-8f), a1 = 1.f / (sqrtf(nn.d[1]) + 1e-8f),
                a2 = 1.f / (sqrtf(nn.d[2]) + 1e-8f);
    const float sum = (a0 + a1) + a2;
    const size_t o = ((size_t)b * n + i) * 3;
    idx[o] = nn.i[0];
    idx[o + 1] = nn.i[1];
    idx[o + 2] = nn.i[2];
    weight[o] = a0 / sum;
    weight[o + 1] = a1 / sum;
    weight[o + 2] = a2 / sum;
}

// ---------------------------------------------------------------------------
// Inverse-distance interpolation: out[b][i][c] = sum_k w[b][i][k] *
// feats[b][idx[b][i][k]][c], one thread per output element, channels fastest.
// ---------------------------------------------------------------------------
template <typename FT, typename OT>
__global__ __launch_bounds__(256) void pv_three_interpolate_kernel(
    const FT* __restrict__ feats, int feat_ld, int m, int C, const int32_t* __restrict__ idx,
    const float* __restrict__ weight, int n, OT* __restrict__ out, int out_ld, size_t total) {
    for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total;
         e += (size_t)gridDim.x * 256) {
        const size_t row = e / C;  // (b, i)
        const int c = (int)(e - row * C);
        const int b = (int)(row / n);
        float acc = 0.f;
#pragma unroll
        for (int k = 0; k < 3; k++) {
            const int j = min(max(idx[row * 3 + k], 0), m - 1);
            const size_t off = ((size_t)b * m + j) * feat_ld + c;
            float f;
            if constexpr (sizeof(FT) == 2)
                f = pv_bf16_to_f32(feats[off]);
            else
                f = feats[off];
            acc += weight[row * 3 + k] * f;
        }
        if constexpr (sizeof(OT) == 2)
            out[row * out_ld + c] = pv_f32_to_bf16(acc);
        else
            out[row * out_ld + c] = acc;
    }
}

// ---------------------------------------------------------------------------
// Maximum over each group's S rows (a centre's neighbours after the shared
// MLP): out[g][c] = max_k x[g*S + k][c]. One thread per output element,
// channels fastest; exact, so the order of the comparisons does not matter.
// ---------------------------------------------------------------------------
template <typename XT, typename OT>
__global__ __launch_bounds__(256) void pv_group_max_kernel(const XT* __restrict__ x, int x_ld,
                                                           int S, int C, OT* __restrict__ out,
                                                           int out_ld, size_t total) {
    for (size_t e = (size_t)blockIdx.x * 256 + threadIdx.x; e < total;
         e += (size_t)gridDim.x * 256) {
        const size_t g = e / C;
        const int c = (int)(e - g * C);
        const XT* r = x + g * S * (size_t)x_ld + c;
        float m = -INFINITY;
        for (int k = 0; k < S; k++) {
            float v;
            if constexpr (sizeof(XT) == 2)
                v = pv_bf16_to_f32(r[(size_t)k * x_ld]);
            else
                v = r[(size_t)k * x_ld];
            m = fmaxf(m, v);
        }
        if constexpr (sizeof(OT) == 2)
            out[g * out_ld + c] = pv_f32_to_bf16(m);
        else
            out[g * out_ld + c] = m;
    }
}

unsigned grid_for(size_t total) {
    const size_t blocks = (total + 255) / 256;
    return (unsigned)(blocks < 65536 ? blocks : 65536);
}

}  // namespace

pvconv_status pv_launch_fps(const float* xyz, int B, int N, int npoint, int32_t* idx,
                            float* new_xyz, hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    // four waves (one per SIMD), so that each step's wave reductions are
    // paid four times, not sixteen; the clouds' points in registers
#define PV_FPS(PPT, NT, TAB)                                                              \
    hipLaunchKernelGGL((pv_fps_kernel<PPT, NT, TAB>), dim3(B), dim3(NT), 0, s, xyz, N, npoint, \
                       idx, new_xyz)
    if (N <= 256) PV_FPS(4, 64, true);
    else if (N <= 1024) PV_FPS(4, 256, true);
    else if (N <= 2048) PV_FPS(8, 256, true);
    else if (N <= 4096) PV_FPS(16, 256, true);
    else if (N <= kFpsTab) PV_FPS(32, 256, true);
    else if (N <= kPvFpsMaxN) PV_FPS(16, 1024, false);
    else return PVCONV_ENOTSUP;
#undef PV_FPS
    return pv_launch_status();
}

pvconv_status pv_launch_ball_query(const float* xyz, int B, int N, const float* centers, int M,
                                   float radius, int nsample, int32_t* idx, hipStream_t s) {
    const int total = B * M;
    if (total == 0) return PVCONV_OK;
    const float r2 = radius * radius;
    hipLaunchKernelGGL(pv_ball_query_kernel, dim3((total + kBallWaves - 1) / kBallWaves),
                       dim3(kBallWaves * 64), 0, s, xyz, N, centers, M, total, r2, nsample, idx);
    return pv_launch_status();
}

pvconv_status pv_launch_group(const float* xyz, const void* feats, bool feat_bf16, int feat_ld,
                              int B, int N, int C, const float* centers, int M,
                              const int32_t* idx, int nsample, void* out, bool out_bf16,
                              int out_ld, hipStream_t s) {
    const size_t total = (size_t)B * M * nsample * (3 + C);
    if (total == 0) return PVCONV_OK;
#define PV_GROUP(FT, OT)                                                                     \
    hipLaunchKernelGGL((pv_group_kernel<FT, OT>), dim3(grid_for(total)), dim3(256), 0, s, xyz, \
                       (const FT*)feats, feat_ld, N, C, centers, M, idx, nsample, (OT*)out,    \
                       out_ld, total)
    if (feat_bf16 && out_bf16) PV_GROUP(uint16_t, uint16_t);
    else if (feat_bf16) PV_GROUP(uint16_t, float);
    else if (out_bf16) PV_GROUP(float, uint16_t);
    else PV_GROUP(float, float);
#undef PV_GROUP
    return pv_launch_status();
}

pvconv_status pv_launch_three_nn(const float* unknown, int B, int n, const float* known, int m,
                                 int32_t* idx, float* weight, hipStream_t s) {
    if (B == 0 || n == 0) return PVCONV_OK;
    hipLaunchKernelGGL(pv_three_nn_kernel, dim3((n + kNnPoints - 1) / kNnPoints, B),
                       dim3(kNnThreads), 0, s, unknown, n, known, m, idx, weight);
    return pv_launch_status();
}

pvconv_status pv_launch_three_interpolate(const void* feats, bool feat_bf16, int feat_ld, int B,
                                          int m, int C, const int32_t* idx, const float* weight,
                                          int n, void* out, bool out_bf16, int out_ld,
                                          hipStream_t s) {
    const size_t total = (size_t)B * n * C;
    if (total == 0) return PVCONV_OK;
#define PV_INTERP(FT, OT)                                                                   \
    hipLaunchKernelGGL((pv_three_interpolate_kernel<FT, OT>), dim3(grid_for(total)),         \
                       dim3(256), 0, s, (const FT*)feats, feat_ld, m, C, idx, weight, n,     \
                       (OT*)out, out_ld, total)
    if (feat_bf16 && out_bf16) PV_INTERP(uint16_t, uint16_t);
    else if (feat_bf16) PV_INTERP(uint16_t, float);
    else if (out_bf16) PV_INTERP(float, uint16_t);
    else PV_INTERP(float, float);
#undef PV_INTERP
    return pv_launch_status();
}

pvconv_status pv_launch_group_max(const void* x, bool x_bf16, int x_ld, int G, int S, int C,
                                  void* out, bool out_bf16, int out_ld, hipStream_t s) {
    const size_t total = (size_t)G * C;
    if (total == 0) return PVCONV_OK;
#define PV_GMAX(XT, OT)                                                                     \
    hipLaunchKernelGGL((pv_group_max_kernel<XT, OT>), dim3(grid_for(total)), dim3(256), 0, s, \
                       (const XT*)x, x_ld, S, C, (OT*)out, out_ld, total)
    if (x_bf16 && out_bf16) PV_GMAX(uint16_t, uint16_t);
    else if (x_bf16) PV_GMAX(uint16_t, float);
    else if (out_bf16) PV_GMAX(float, uint16_t);
    else PV_GMAX(float, float);
#undef PV_GMAX
    return pv_launch_status();
}
