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
// bf16) vectors. Shapes that rule out vector access load value by value
// (ragged or unaligned C_in) or read and write channel by channel (ragged
// C_out or unaligned rows). Inside a whole PVConv layer the residual is the
// trilinear devoxelisation of the bf16 grid, which the kernel's DV variant
// gathers itself (pv_launch_devox_point_mlp): one launch fewer and no fp32
// intermediate rows in HBM.
#include <type_traits>

#include "pv_common.h"
#include "pv_trilinear.h"

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

// VEC (checked by the launcher): Cin % 8 == 0, x rows and weight rows
// 16-byte aligned; else every operand value is loaded on its own, with zero
// past Cin. C4 (checked by the launcher): Cout % 4 == 0, residual / cloud
// rows 16-byte aligned, output rows 16-byte (fp32) or 8-byte (bf16) aligned;
// else the epilogue reads and writes channel by channel.
//
// DV: the residual is the trilinear devoxelisation of a bf16 grid (Section
// 4.1), gathered by this kernel instead of read as rows of a separate
// launch's output: the workgroup's 128 points x (32*NB) channels are summed
// into LDS (fp32, the same arithmetic and order as the devoxelisation kernel,
// so the result is the same bits) by all four waves before the GEMM. (Four
// more waves gathering while the GEMM waves load and multiply measured
// slower: two waves per SIMD leave room for only two items' loads in flight.)
// Requires C4, Cout % 8 == 0 and a 16-byte aligned grid.
template <int NB, typename XT, bool VEC, bool C4, bool DV = false>
__global__ __launch_bounds__(kWaves * 64) void pv_point_mlp_tile_kernel(
    const XT* __restrict__ x, int x_ld, int M, int Cin, int Cout, const uint16_t* __restrict__ w,
    PvBnFold bn, int act, float slope, const float* __restrict__ cloud_bias, int ppc,
    const float* __restrict__ residual, int res_ld, void* __restrict__ out, int out_bf16,
    int out_ld, PvDevoxIn dvin) {
    __shared__ float4 tab[2][NB * 8];  // folded scale / shift, 4 channels per entry
    // DV: the devoxelised rows of the workgroup's points, padded by 4 floats
    // so that the 32 rows read by one instruction start in different banks
    constexpr int kDvLd = NB * 32 + 4;
    __shared__ __attribute__((aligned(16))) float dvrow[DV ? kWaves * 32 : 1][DV ? kDvLd : 1];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    // DV: each XCD takes a contiguous range of points (a few clouds), so that
    // the corner rows nearby points share are fetched into one L2
    int bx = blockIdx.x;
    if (DV && (gridDim.x & 7) == 0) bx = (bx & 7) * (gridDim.x >> 3) + (bx >> 3);
    const int n0 = blockIdx.y * (NB * 32);
    const int ncols = min(NB * 32, Cout - n0);
    if (threadIdx.x < NB * 32) {
        const int c = min(n0 + (int)threadIdx.x, Cout - 1);
        float sc, sh;
        pv_bn_coeffs(bn, c, sc, sh);
        ((float*)tab[0])[threadIdx.x] = sc;
        ((float*)tab[1])[threadIdx.x] = sh;
    }
    if constexpr (DV) {
        // Items (point, 8-channel group): consecutive lanes take consecutive
        // groups of one point, so each corner row is read contiguously. NB*2
        // items per thread (fewer valid ones in a ragged last channel block),
        // in rounds of up to four whose 32 corner loads are all in flight
        // together. The launcher takes NB = 2 (64-channel column blocks):
        // one round of four items, and at the part-segmentation layer 512
        // workgroups, two per CU, all resident at once. The kernel reads
        // nothing from HBM twice, so the latency of this gather and of the
        // feature loads that follow it is what bounds it.
        const int tid = threadIdx.x;
        const int G = ncols >> 3, items = kWaves * 32 * G;
        const size_t V = (size_t)dvin.R * dvin.R * dvin.R;
        constexpr int kIPT = NB * 2, kRound = kIPT < 4 ? kIPT : 4;
#pragma unroll
        for (int r = 0; r < kIPT; r += kRound) {
            float a[kRound][8];
#pragma unroll
            for (int u = 0; u < kRound; u++) {
                const int i = min(tid + (r + u) * kWaves * 64, items - 1);
                const int pl = i / G, g = i - pl * G;
                const int m = min(bx * kWaves * 32 + pl, M - 1);
                const float* p = dvin.pn + (size_t)m * 3;
                const PvAxis ax = pv_trilinear_axis(p[0], dvin.R),
                             ay = pv_trilinear_axis(p[1], dvin.R),
                             az = pv_trilinear_axis(p[2], dvin.R);
                pv_trilinear8<uint16_t>(dvin.grid + (size_t)(m / dvin.N) * V * Cout + n0 + g * 8,
                                        Cout, dvin.R, ax, ay, az, a[u]);
            }
#pragma unroll
            for (int u = 0; u < kRound; u++) {
                const int i = tid + (r + u) * kWaves * 64;
                if (i >= items) continue;
                const int pl = i / G, g = i - pl * G;
                *(float4*)&dvrow[pl][g * 8] = make_float4(a[u][0], a[u][1], a[u][2], a[u][3]);
                *(float4*)&dvrow[pl][g * 8 + 4] = make_float4(a[u][4], a[u][5], a[u][6], a[u][7]);
            }
        }
    }
    __syncthreads();
    const int m0 = (bx * kWaves + wave) * 32;
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

    // Column offsets of this lane's four-channel groups. C4: clamped into the
    // valid columns so that every load below is unconditional (one batch,
    // no branches between loads); clamped groups are never stored. Else
    // unclamped, each channel checked against Cout.
    int coff[NB][4];
#pragma unroll
    for (int nb = 0; nb < NB; nb++)
#pragma unroll
        for (int g = 0; g < 4; g++)
            coff[nb][g] = n0 + (C4 ? min(nb * 32 + g * 8 + 4 * h, ncols - 4) : nb * 32 + g * 8 + 4 * h);
    // four channels from row p at column c (C4: one 16-byte load)
    auto row4 = [&](const float* p, int c) -> float4 {
        if constexpr (C4) return *(const float4*)(p + c);
        return float4{c < Cout ? p[c] : 0.f, c + 1 < Cout ? p[c + 1] : 0.f,
                      c + 2 < Cout ? p[c + 2] : 0.f, c + 3 < Cout ? p[c + 3] : 0.f};
    };

    // The residual rows go in flight first: they are consumed last.
    float4 res[NB][4];
    if constexpr (DV) {
#pragma unroll
        for (int nb = 0; nb < NB; nb++)
#pragma unroll
            for (int g = 0; g < 4; g++)
                res[nb][g] = *(const float4*)&dvrow[wave * 32 + r32][coff[nb][g] - n0];
    } else if (residual) {
        const float* rr = residual + (size_t)m * res_ld;
#pragma unroll
        for (int nb = 0; nb < NB; nb++)
#pragma unroll
            for (int g = 0; g < 4; g++) res[nb][g] = row4(rr, coff[nb][g]);
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
    if constexpr (!VEC) {
        for (int k0 = 0; k0 < Cin; k0 += 64) {
            pv_bf16x8 xg[4], wg[4][NB];
#pragma unroll
            for (int ks = 0; ks < 4; ks++) {
                const int k = k0 + ks * 16 + 8 * h;   // this lane's 8 values of the step
                const int valid = max(0, min(8, Cin - k));
                xg[ks] = load_a8<XT>(x + (size_t)m * x_ld + k, false, valid);
#pragma unroll
                for (int nb = 0; nb < NB; nb++)
                    wg[ks][nb] = load_a8<uint16_t>(
                        w + (size_t)min(n0 + nb * 32 + r32, Cout - 1) * Cin + k, false, valid);
            }
#pragma unroll
            for (int ks = 0; ks < 4; ks++)
#pragma unroll
                for (int nb = 0; nb < NB; nb++)
                    acc[nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(wg[ks][nb], xg[ks], acc[nb],
                                                                      0, 0, 0);
        }
    }
    for (int k0 = 0; VEC && k0 < Cin; k0 += 64) {
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
            for (int g = 0; g < 4; g++) cb[nb][g] = row4(cbr, coff[nb][g]);
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
            if constexpr (!C4) {
                const float e[4] = {v.x, v.y, v.z, v.w};
                for (int j = 0; j < 4 && coff[nb][g] + j < Cout; j++) {
                    if (out_bf16)
                        ((uint16_t*)out)[orow + coff[nb][g] + j] = pv_f32_to_bf16(e[j]);
                    else
                        ((float*)out)[orow + coff[nb][g] + j] = e[j];
                }
            } else if (out_bf16) {
                *(uint2*)((uint16_t*)out + orow + coff[nb][g]) =
                    uint2{pv_pack_bf16x2(v.x, v.y), pv_pack_bf16x2(v.z, v.w)};
            } else {
                *(float4*)((float*)out + orow + coff[nb][g]) = v;
            }
        }
}

// ---- wide layers: LDS-tiled MFMA GEMM ------------------------------------
// For K >= 128 and C_out >= 128 the layer is MFMA-bound, so operands are
// shared through LDS: a 256-thread workgroup owns a TN x TM (channels x
// points) output tile, stages K in chunks of kGK = 64 (weights and point rows
// as bf16, 128 bytes of data per row padded to kGPitch = 144 so that the
// 16-byte fragment reads of 16 consecutive rows hit distinct banks), double
// buffered: the next chunk's global loads are in flight while the current
// chunk feeds the MFMAs, one barrier per chunk. Each wave computes
// (NB*32) x (MB*32) of the tile with the weights as the A operand, so the
// epilogue holds 4 consecutive channels of one point per lane.
constexpr int kGK = 64;
constexpr int kGPitch = 144;

template <int NB, int MB, int WN, int WM>
struct GemmShape {
    static constexpr int TN = WN * NB * 32;   // output channels per workgroup
    static constexpr int TM = WM * MB * 32;   // points per workgroup
    static constexpr int ROWS = TN + TM;      // staged rows per chunk
    static constexpr int NTHR = 64 * WN * WM; // threads (four or eight waves)
    static constexpr int RSET = NTHR / 8;     // rows per piece set (8 threads per row)
    static constexpr int PIECES = ROWS * 8 / NTHR;  // 16-byte pieces per thread per chunk
    static constexpr int LDS = 2 * ROWS * kGPitch;
    static_assert(WN * WM == 4 || WN * WM == 8, "four or eight waves");
    static_assert(ROWS % RSET == 0 && TN % RSET == 0, "whole piece sets, weights apart");
};

__device__ __forceinline__ uint4 piece_bf16(const uint16_t* p) { return *(const uint4*)p; }
__device__ __forceinline__ uint4 piece_bf16(const float* p) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    return uint4{pv_pack_bf16x2(a.x, a.y), pv_pack_bf16x2(a.z, a.w), pv_pack_bf16x2(b.x, b.y),
                 pv_pack_bf16x2(b.z, b.w)};
}

// Requirements (checked by the launcher): Cin % 8 == 0, Cout % 4 == 0, x and
// weight rows 16-byte aligned, residual / cloud rows 16-byte aligned, output
// rows 16-byte (fp32) or 8-byte (bf16) aligned.
// EXT: a per-cloud row or a residual is given (else neither is read, and
// the registers that prefetch them are not needed).
template <int NB, int MB, int WN, int WM, typename XT, bool EXT>
__global__ __launch_bounds__(64 * WN * WM, 1) void pv_point_mlp_lds_kernel(
    const XT* __restrict__ x, int x_ld, int M, int Cin, int Cout, const uint16_t* __restrict__ w,
    PvBnFold bn, int act, float slope, const float* __restrict__ cloud_bias, int ppc,
    const float* __restrict__ residual, int res_ld, void* __restrict__ out, int out_bf16,
    int out_ld, int ntn, int nblocks) {
    typedef GemmShape<NB, MB, WN, WM> S;
    __shared__ __attribute__((aligned(16))) char lds[S::LDS];
    __shared__ float4 tab[2][S::TN / 4];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // Consecutive tiles (same point rows, neighbouring channel tiles) go to
    // the same XCD, so the point rows are fetched into one L2.
    int bid = blockIdx.x;
    if ((nblocks & 7) == 0) bid = (bid & 7) * (nblocks >> 3) + (bid >> 3);
    const int n0 = (bid % ntn) * S::TN, m0 = (bid / ntn) * S::TM;

    if (tid < S::TN) {
        const int c = min(n0 + tid, Cout - 1);
        float sc, sh;
        pv_bn_coeffs(bn, c, sc, sh);
        ((float*)tab[0])[tid] = sc;
        ((float*)tab[1])[tid] = sh;
    }

    // Staging: piece i*NTHR + tid is row i*RSET + tid/8 of the chunk (weight
    // rows first, then point rows), bytes (tid%8)*16 .. +15 of its 128.
    // Rows past M or C_out are clamped onto the last valid row (their results
    // are never stored); columns past C_in stage as zero.
    const int part = tid & 7;
    const uint16_t* wsrc = w + part * 8;
    const XT* xsrc = x + part * 8;
    // The columns past C_in are zeroed when the chunk is stored to LDS, not
    // when it is loaded: a select right after the load would make the wave
    // wait for the load there, before the MFMAs it is meant to overlap.
    // Two register sets (see kD below); past the last chunk the loads re-read
    // column 0 (stored as zeros, never used), so that every load is
    // unconditional and the wait counts stay exact.
    uint4 stage[2][S::PIECES];
    auto stage_load = [&](int set, int k0) {
        const bool ok = k0 + part * 8 < Cin;
        const int k = ok ? k0 : 0;
#pragma unroll
        for (int i = 0; i < S::PIECES; i++) {
            const int row = i * S::RSET + (tid >> 3);
            uint4 v;
            if (i * S::RSET < S::TN)   // resolved at compile time (TN: whole piece sets)
                v = piece_bf16(wsrc + (size_t)min(n0 + row, Cout - 1) * Cin + k);
            else
                v = piece_bf16(xsrc + (size_t)min(m0 + row - S::TN, M - 1) * x_ld + k);
            stage[set][i] = v;
        }
    };
    auto stage_store = [&](int buf, int set, int k0) {
        const bool ok = k0 + part * 8 < Cin;
        char* base = lds + buf * (S::ROWS * kGPitch) + (tid >> 3) * kGPitch + part * 16;
#pragma unroll
        for (int i = 0; i < S::PIECES; i++)
            *(uint4*)(base + i * S::RSET * kGPitch) = ok ? stage[set][i] : uint4{0u, 0u, 0u, 0u};
    };

    const int wn = wave % WN, wm = wave / WN;
    const int r32 = lane & 31, khalf = lane >> 5;
    const int a_off = (wn * NB * 32 + r32) * kGPitch + khalf * 16;
    const int b_off = (S::TN + wm * MB * 32 + r32) * kGPitch + khalf * 16;

    pv_f32x16 acc[MB][NB];
#pragma unroll
    for (int i = 0; i < MB; i++)
#pragma unroll
        for (int j = 0; j < NB; j++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[i][j][e] = 0.f;

    const int nch = (Cin + kGK - 1) / kGK;
    // Chunk j is staged through register set j % 2 and LDS buffer j % 2.
    // Loads run kD chunks ahead: two, unless fp32 rows of eight pieces a
    // thread make two sets too many registers.
    constexpr int kD = std::is_same<XT, float>::value && S::PIECES >= 8 ? 1 : 2;
    stage_load(0, 0);
    if (kD == 2) stage_load(1, kGK);
    stage_store(0, 0, 0);
    __syncthreads();
    // chunk c (parity P = c % 2, a compile-time index into the register
    // sets): chunk c + kD loads, the MFMAs read LDS buffer P, then chunk c + 1
    // is stored from its set to buffer 1 - P
    auto chunk = [&](int c, auto parity) {
        constexpr int P = decltype(parity)::value;
        stage_load(kD == 2 ? P : 1 - P, (c + kD) * kGK);
        const char* buf = lds + P * (S::ROWS * kGPitch);
#pragma unroll
        for (int ks = 0; ks < kGK / 16; ks++) {
            pv_bf16x8 a[NB], b[MB];
#pragma unroll
            for (int nb = 0; nb < NB; nb++)
                a[nb] = *(const pv_bf16x8*)(buf + a_off + nb * 32 * kGPitch + ks * 32);
#pragma unroll
            for (int mb = 0; mb < MB; mb++)
                b[mb] = *(const pv_bf16x8*)(buf + b_off + mb * 32 * kGPitch + ks * 32);
#pragma unroll
            for (int mb = 0; mb < MB; mb++)
#pragma unroll
                for (int nb = 0; nb < NB; nb++)
                    acc[mb][nb] =
                        __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[nb], b[mb], acc[mb][nb], 0, 0, 0);
        }
        if (c + 1 < nch) stage_store(1 - P, 1 - P, (c + 1) * kGK);
        __syncthreads();
    };
    for (int c = 0; c < nch; c += 2) {
        chunk(c, std::integral_constant<int, 0>{});
        if (c + 1 < nch) chunk(c + 1, std::integral_constant<int, 1>{});
    }

    // Epilogue, one (32-point block mb, 32-channel block nb) at a time.
    // acc[mb][nb][4g + j] is channel wn*NB*32 + nb*32 + 8g + 4*khalf + j of
    // the tile at point wm*MB*32 + mb*32 + r32. A block's values are finished
    // first, then the per-cloud and residual rows of the next block are
    // loaded into the same registers, then the block is stored: one counter
    // tracks loads and stores alike, so a load issued after a store would
    // wait for it.
    const float neg = act == PVCONV_ACT_LEAKY ? slope : (act == PVCONV_ACT_RELU ? 0.f : 1.f);
    float4 ext[2][4];   // [cloud row, residual][g] of the block being finished
    auto load_ext = [&](int mb, int nb) {
        const int m = min(m0 + wm * MB * 32 + mb * 32 + r32, M - 1);
        const float* cbr = EXT && cloud_bias ? cloud_bias + (size_t)(m / ppc) * Cout : nullptr;
        const float* rr = EXT && residual ? residual + (size_t)m * res_ld : nullptr;
#pragma unroll
        for (int g = 0; g < 4; g++) {
            const int n = min(n0 + wn * NB * 32 + nb * 32 + g * 8 + 4 * khalf, Cout - 4);
            ext[0][g] = cbr ? *(const float4*)(cbr + n) : float4{0.f, 0.f, 0.f, 0.f};
            ext[1][g] = rr ? *(const float4*)(rr + n) : float4{0.f, 0.f, 0.f, 0.f};
        }
    };
    load_ext(0, 0);
#pragma unroll
    for (int mb = 0; mb < MB; mb++) {
        const int m = m0 + wm * MB * 32 + mb * 32 + r32;
        const size_t orow = (size_t)min(m, M - 1) * out_ld;
#pragma unroll
        for (int nb = 0; nb < NB; nb++) {
            const int blk = mb * NB + nb;
            float4 val[4];
#pragma unroll
            for (int g = 0; g < 4; g++) {
                const int nl = wn * NB * 32 + nb * 32 + g * 8 + 4 * khalf;
                const float4 sc = tab[0][nl >> 2], sh = tab[1][nl >> 2];
                const float4 cb = ext[0][g], rs = ext[1][g];
                float v[4] = {(acc[mb][nb][4 * g] + cb.x) * sc.x + sh.x,
                              (acc[mb][nb][4 * g + 1] + cb.y) * sc.y + sh.y,
                              (acc[mb][nb][4 * g + 2] + cb.z) * sc.z + sh.z,
                              (acc[mb][nb][4 * g + 3] + cb.w) * sc.w + sh.w};
#pragma unroll
                for (int j = 0; j < 4; j++) v[j] = v[j] >= 0.f ? v[j] : v[j] * neg;
                val[g] = float4{v[0] + rs.x, v[1] + rs.y, v[2] + rs.z, v[3] + rs.w};
            }
            if (blk + 1 < MB * NB) load_ext((blk + 1) / NB, (blk + 1) % NB);
#pragma unroll
            for (int g = 0; g < 4; g++) {
                const int nl = wn * NB * 32 + nb * 32 + g * 8 + 4 * khalf;
                if (m >= M || n0 + nl >= Cout) continue;
                if (out_bf16)
                    *(uint2*)((uint16_t*)out + orow + n0 + nl) =
                        uint2{pv_pack_bf16x2(val[g].x, val[g].y), pv_pack_bf16x2(val[g].z, val[g].w)};
                else
                    *(float4*)((float*)out + orow + n0 + nl) = val[g];
            }
        }
    }
}

template <typename XT>
__device__ __forceinline__ float ld1(const XT* p);
template <>
__device__ __forceinline__ float ld1<float>(const float* p) { return *p; }
template <>
__device__ __forceinline__ float ld1<uint16_t>(const uint16_t* p) { return pv_bf16_to_f32(*p); }

// 8 consecutive values as fp32 (no rounding): the max-pool's loads.
__device__ __forceinline__ void load8_raw(const float* p, float (&v)[8]) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}
__device__ __forceinline__ void load8_raw(const uint16_t* p, float (&v)[8]) {
    const uint4 a = *(const uint4*)p;
    const uint32_t u[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int i = 0; i < 4; i++) {
        v[2 * i] = __uint_as_float(u[i] << 16);
        v[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
    }
}

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
                 bool c4, const PvBnFold& bn, int act, float slope, const float* cb, int ppc,
                 const float* res, int res_ld, void* out, bool out_bf16, int out_ld,
                 hipStream_t s) {
    dim3 g((M + kWaves * 32 - 1) / (kWaves * 32), (Cout + NB * 32 - 1) / (NB * 32));
#define PV_TILE(V, C)                                                                         \
    hipLaunchKernelGGL((pv_point_mlp_tile_kernel<NB, XT, V, C>), g, dim3(kWaves * 64), 0, s, \
                       (const XT*)x, x_ld, M, Cin, Cout, (const uint16_t*)w, bn, act, slope,   \
                       cb, ppc, res, res_ld, out, (int)out_bf16, out_ld, PvDevoxIn{})
    if (vec) {
        if (c4) PV_TILE(true, true); else PV_TILE(true, false);
    } else {
        if (c4) PV_TILE(false, true); else PV_TILE(false, false);
    }
#undef PV_TILE
}

template <int NB, int MB, int WN, int WM, typename XT>
void launch_lds(const void* x, int x_ld, int M, int Cin, int Cout, const void* w,
                const PvBnFold& bn, int act, float slope, const float* cb, int ppc,
                const float* res, int res_ld, void* out, bool out_bf16, int out_ld,
                hipStream_t s) {
    typedef GemmShape<NB, MB, WN, WM> S;
    const int ntn = (Cout + S::TN - 1) / S::TN;
    const int nblocks = ntn * ((M + S::TM - 1) / S::TM);
    if (cb || res)
        hipLaunchKernelGGL((pv_point_mlp_lds_kernel<NB, MB, WN, WM, XT, true>), dim3(nblocks),
                           dim3(S::NTHR), 0, s, (const XT*)x, x_ld, M, Cin, Cout, (const uint16_t*)w,
                           bn, act, slope, cb, ppc, res, res_ld, out, (int)out_bf16, out_ld, ntn,
                           nblocks);
    else
        hipLaunchKernelGGL((pv_point_mlp_lds_kernel<NB, MB, WN, WM, XT, false>), dim3(nblocks),
                           dim3(S::NTHR), 0, s, (const XT*)x, x_ld, M, Cin, Cout, (const uint16_t*)w,
                           bn, act, slope, cb, ppc, res, res_ld, out, (int)out_bf16, out_ld, ntn,
                           nblocks);
}

// ---- small-M path --------------------------------------------------------
// Fewer rows than one tile workgroup covers (e.g. one row per cloud): one wave
// per output element, the lanes splitting K, then a wave-wide sum. bf16
// operands (fp32 rows rounded to bf16) with fp32 accumulation, like the MFMA
// path.
template <typename XT>
__device__ __forceinline__ void load8_f32(const XT* p, float (&v)[8]);
template <>
__device__ __forceinline__ void load8_f32<float>(const float* p, float (&v)[8]) {
    const float4 a = *(const float4*)p, b = *(const float4*)(p + 4);
    v[0] = pv_bf16_to_f32(pv_f32_to_bf16(a.x)); v[1] = pv_bf16_to_f32(pv_f32_to_bf16(a.y));
    v[2] = pv_bf16_to_f32(pv_f32_to_bf16(a.z)); v[3] = pv_bf16_to_f32(pv_f32_to_bf16(a.w));
    v[4] = pv_bf16_to_f32(pv_f32_to_bf16(b.x)); v[5] = pv_bf16_to_f32(pv_f32_to_bf16(b.y));
    v[6] = pv_bf16_to_f32(pv_f32_to_bf16(b.z)); v[7] = pv_bf16_to_f32(pv_f32_to_bf16(b.w));
}
template <>
__device__ __forceinline__ void load8_f32<uint16_t>(const uint16_t* p, float (&v)[8]) {
    const uint4 a = *(const uint4*)p;
    const uint32_t u[4] = {a.x, a.y, a.z, a.w};
#pragma unroll
    for (int i = 0; i < 4; i++) {
        v[2 * i] = __uint_as_float(u[i] << 16);
        v[2 * i + 1] = __uint_as_float(u[i] & 0xffff0000u);
    }
}
template <typename XT>
__device__ __forceinline__ float ldb(const XT* p);
template <>
__device__ __forceinline__ float ldb<float>(const float* p) {
    return pv_bf16_to_f32(pv_f32_to_bf16(*p));
}
template <>
__device__ __forceinline__ float ldb<uint16_t>(const uint16_t* p) { return pv_bf16_to_f32(*p); }

template <typename XT, bool VEC>
__global__ __launch_bounds__(256) void pv_point_mlp_rows_kernel(
    const XT* __restrict__ x, int x_ld, int M, int Cin, int Cout, const uint16_t* __restrict__ w,
    PvBnFold bn, int act, float slope, const float* __restrict__ cloud_bias, int ppc,
    const float* __restrict__ residual, int res_ld, void* __restrict__ out, int out_bf16,
    int out_ld) {
    const int lane = threadIdx.x & 63;
    const long e = (long)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (e >= (long)M * Cout) return;
    const int m = (int)(e / Cout), n = (int)(e % Cout);
    const XT* xr = x + (size_t)m * x_ld;
    const uint16_t* wr = w + (size_t)n * Cin;
    float s = 0.f;
    if (VEC) {
#pragma unroll 2
        for (int k = lane * 8; k < Cin; k += 512) {
            float a[8], b[8];
            load8_f32<XT>(xr + k, a);
            load8_f32<uint16_t>(wr + k, b);
#pragma unroll
            for (int j = 0; j < 8; j++) s += a[j] * b[j];
        }
    } else {
#pragma unroll 4
        for (int k = lane; k < Cin; k += 64) s += ldb<XT>(xr + k) * pv_bf16_to_f32(wr[k]);
    }
#pragma unroll
    for (int off = 32; off > 0; off >>= 1) s += __shfl_xor(s, off, 64);
    if (lane != 0) return;
    if (cloud_bias) s += cloud_bias[(size_t)(m / ppc) * Cout + n];
    float sc, sh;
    pv_bn_coeffs(bn, n, sc, sh);
    float v = pv_activate(s * sc + sh, act, slope);
    if (residual) v += residual[(size_t)m * res_ld + n];
    if (out_bf16)
        ((uint16_t*)out)[(size_t)m * out_ld + n] = pv_f32_to_bf16(v);
    else
        ((float*)out)[(size_t)m * out_ld + n] = v;
}

// ---- per-cloud max-pool -------------------------------------------------
// out starts at -inf (fill kernel); each block takes a slice of kPoolPts
// points of one cloud and a range of channels, reduces in registers (and
// across its four waves in LDS), then merges into out with integer atomics:
// for a non-negative float the int ordering is the float ordering, for a
// negative one the unsigned ordering is reversed, so atomicMax on int and
// atomicMin on unsigned give the float max in any order, bit-exactly.
constexpr int kPoolPts = 128;

__device__ __forceinline__ void atomic_max_f32(float* a, float v) {
    if (__float_as_int(v) >= 0)
        atomicMax((int*)a, __float_as_int(v));
    else
        atomicMin((unsigned int*)a, __float_as_uint(v));
}

__global__ __launch_bounds__(256) void pv_fill_f32_kernel(float* __restrict__ p, int n, float v) {
    const int i = blockIdx.x * 256 + threadIdx.x;
    if (i < n) p[i] = v;
}

// VEC: C % 8 == 0 and 16-byte rows; a lane owns 8 consecutive channels, a
// wave 512, and the block's four waves split the slice's points.
template <typename XT>
__global__ __launch_bounds__(256) void pv_maxpool_vec_kernel(const XT* __restrict__ x, int x_ld,
                                                             int N, int C,
                                                             float* __restrict__ out) {
    __shared__ float part[4][512];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int b = blockIdx.y;
    const int p0 = blockIdx.z * kPoolPts, p1 = min(p0 + kPoolPts, N);
    const int cb = blockIdx.x * 512, c0 = cb + lane * 8;
    float m[8];
#pragma unroll
    for (int j = 0; j < 8; j++) m[j] = -INFINITY;
    if (c0 < C) {
        const XT* base = x + (size_t)b * N * x_ld + c0;
        for (int p = p0 + wave; p < p1; p += 16) {
            // four rows in flight; past the slice, a row repeats (max is idempotent)
            float v[4][8];
#pragma unroll
            for (int u = 0; u < 4; u++) {
                const int row = p + 4 * u < p1 ? p + 4 * u : p;
                load8_raw(base + (size_t)row * x_ld, v[u]);
            }
#pragma unroll
            for (int u = 0; u < 4; u++)
#pragma unroll
                for (int j = 0; j < 8; j++) m[j] = fmaxf(m[j], v[u][j]);
        }
    }
#pragma unroll
    for (int j = 0; j < 8; j++) part[wave][lane * 8 + j] = m[j];
    __syncthreads();
    for (int i = threadIdx.x; i < 512; i += 256) {
        const int c = cb + i;
        if (c >= C) continue;
        const float r = fmaxf(fmaxf(part[0][i], part[1][i]), fmaxf(part[2][i], part[3][i]));
        atomic_max_f32(out + (size_t)b * C + c, r);
    }
}

template <typename XT>
__global__ __launch_bounds__(256) void pv_maxpool_scalar_kernel(const XT* __restrict__ x,
                                                                int x_ld, int N, int C,
                                                                float* __restrict__ out) {
    const int c = blockIdx.x * 256 + threadIdx.x;
    const int b = blockIdx.y;
    const int p0 = blockIdx.z * kPoolPts, p1 = min(p0 + kPoolPts, N);
    if (c >= C) return;
    const XT* base = x + (size_t)b * N * x_ld + c;
    float m = -INFINITY;
#pragma unroll 4
    for (int p = p0; p < p1; p++) m = fmaxf(m, ld1<XT>(base + (size_t)p * x_ld));
    atomic_max_f32(out + (size_t)b * C + c, m);
}

}  // namespace

pvconv_status pv_launch_point_mlp(const void* x, bool x_bf16, int x_ld, int M, int Cin,
                                  int Cout, const void* w, bool bf16, const PvBnFold& bn,
                                  int act, float slope, const float* cb, int ppc,
                                  const float* res, int res_ld, void* out, bool out_bf16,
                                  int out_ld, hipStream_t s) {
    if (M == 0) return PVCONV_OK;
    if (bf16 && M < kWaves * 32) {
        const size_t esz = x_bf16 ? 2 : 4;
        const bool vec = Cin % 8 == 0 && pv_aligned16(x) && pv_aligned16(w) &&
                         ((size_t)x_ld * esz) % 16 == 0;
        const unsigned blocks = (unsigned)(((long)M * Cout + 3) / 4);
#define PV_ROWS(XT, V)                                                                         \
    hipLaunchKernelGGL((pv_point_mlp_rows_kernel<XT, V>), dim3(blocks), dim3(256), 0, s,       \
                       (const XT*)x, x_ld, M, Cin, Cout, (const uint16_t*)w, bn, act, slope, cb, \
                       ppc, res, res_ld, out, (int)out_bf16, out_ld)
        if (x_bf16) {
            if (vec) PV_ROWS(uint16_t, true); else PV_ROWS(uint16_t, false);
        } else {
            if (vec) PV_ROWS(float, true); else PV_ROWS(float, false);
        }
#undef PV_ROWS
        return pv_launch_status();
    }
    if (bf16) {
        const size_t esz = x_bf16 ? 2 : 4;
        const bool vec = Cin % 8 == 0 && pv_aligned16(x) && pv_aligned16(w) &&
                         ((size_t)x_ld * esz) % 16 == 0;
        // c4: four-channel groups of the residual, cloud and output rows are
        // whole aligned vectors
        const bool c4 = Cout % 4 == 0 && (!res || (pv_aligned16(res) && res_ld % 4 == 0)) &&
                        (!cb || pv_aligned16(cb)) && out_ld % 4 == 0 &&
                        ((uintptr_t)out & (out_bf16 ? 7u : 15u)) == 0;
        const bool tile = vec && c4;
        // wide layers: LDS-tiled GEMM, 256 x 256 (channels x points) tiles of
        // eight waves (two per SIMD, 128 x 64 each) when they still give a
        // workgroup per CU, else eight-wave 128 x 256 (128 x 32 each) or
        // 128 x 128 tiles (eight waves of 64 x 32)
        const long big_tiles = (long)((Cout + 255) / 256) * ((M + 255) / 256);
        if (tile && Cin >= 128 && Cout >= 256 && big_tiles >= 256) {
            if (x_bf16)
                launch_lds<4, 2, 2, 4, uint16_t>(x, x_ld, M, Cin, Cout, w, bn, act, slope, cb, ppc,
                                                 res, res_ld, out, out_bf16, out_ld, s);
            else
                launch_lds<4, 2, 2, 4, float>(x, x_ld, M, Cin, Cout, w, bn, act, slope, cb, ppc,
                                              res, res_ld, out, out_bf16, out_ld, s);
            return pv_launch_status();
        }
        // 128 x 128 tiles where 128 x 256 would leave CUs idle (e.g. the head's
        // 256-wide first layer: 34 % faster), of eight waves so that two share
        // each SIMD (2 % on the part-segmentation network against four)
        const long mid_tiles = (long)((Cout + 127) / 128) * ((M + 255) / 256);
        if (tile && Cin >= 128 && Cout >= 128 && mid_tiles < 256) {
            if (x_bf16)
                launch_lds<2, 1, 2, 4, uint16_t>(x, x_ld, M, Cin, Cout, w, bn, act, slope, cb, ppc,
                                                 res, res_ld, out, out_bf16, out_ld, s);
            else
                launch_lds<2, 1, 2, 4, float>(x, x_ld, M, Cin, Cout, w, bn, act, slope, cb, ppc,
                                              res, res_ld, out, out_bf16, out_ld, s);
            return pv_launch_status();
        }
        if (tile && Cin >= 128 && Cout >= 128) {
            if (x_bf16)

                launch_lds<4, 1, 1, 8, uint16_t>(x, x_ld, M, Cin, Cout, w, bn, act, slope, cb, ppc,
                                                 res, res_ld, out, out_bf16, out_ld, s);
            else
                launch_lds<4, 1, 1, 8, float>(x, x_ld, M, Cin, Cout, w, bn, act, slope, cb, ppc,
                                              res, res_ld, out, out_bf16, out_ld, s);
            return pv_launch_status();
        }
        if (x_bf16) {
            if (Cout > 64)
                launch_mfma<4, uint16_t>(x, x_ld, M, Cin, Cout, w, vec, c4, bn, act, slope, cb,
                                         ppc, res, res_ld, out, out_bf16, out_ld, s);
            else
                launch_mfma<2, uint16_t>(x, x_ld, M, Cin, Cout, w, vec, c4, bn, act, slope, cb,
                                         ppc, res, res_ld, out, out_bf16, out_ld, s);
        } else {
            if (Cout > 64)
                launch_mfma<4, float>(x, x_ld, M, Cin, Cout, w, vec, c4, bn, act, slope, cb,
                                      ppc, res, res_ld, out, out_bf16, out_ld, s);
            else
                launch_mfma<2, float>(x, x_ld, M, Cin, Cout, w, vec, c4, bn, act, slope, cb,
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

pvconv_status pv_launch_devox_point_mlp(const PvDevoxIn& dv, const void* x, bool x_bf16,
                                        int x_ld, int M, int Cin, int Cout, const void* w,
                                        const PvBnFold& bn, int act, float slope, void* out,
                                        bool out_bf16, int out_ld, hipStream_t s) {
    const size_t esz = x_bf16 ? 2 : 4;
    // the shapes the unfused path runs on the tile kernel with vector access
    const bool ok = M >= kWaves * 32 && Cin % 8 == 0 && pv_aligned16(x) && pv_aligned16(w) &&
                    ((size_t)x_ld * esz) % 16 == 0 && Cout % 8 == 0 && out_ld % 4 == 0 &&
                    ((uintptr_t)out & (out_bf16 ? 7u : 15u)) == 0 && pv_aligned16(dv.grid) &&
                    !(Cin >= 128 && Cout >= 128) && dv.N > 0 && M % dv.N == 0;
    if (!ok) return PVCONV_ENOTSUP;
    // 64-channel tiles also for wider layers: twice the workgroups (two per
    // CU at the part-seg shape) to cover the gather's latency, 1 % faster on
    // that layer than 128-channel tiles, though the point rows are read twice
#define PV_DV(NB, XT)                                                                         \
    hipLaunchKernelGGL((pv_point_mlp_tile_kernel<NB, XT, true, true, true>),                  \
                       dim3((M + kWaves * 32 - 1) / (kWaves * 32), (Cout + NB * 32 - 1) / (NB * 32)), \
                       dim3(kWaves * 64), 0, s, (const XT*)x, x_ld, M, Cin, Cout,              \
                       (const uint16_t*)w, bn, act, slope, nullptr, 1, nullptr, 0, out,         \
                       (int)out_bf16, out_ld, dv)
    if (x_bf16) PV_DV(2, uint16_t); else PV_DV(2, float);
#undef PV_DV
    return pv_launch_status();
}

pvconv_status pv_launch_maxpool(const void* x, bool bf16, int x_ld, int B, int N, int C,
                                float* out, hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    const int n = B * C;
    hipLaunchKernelGGL(pv_fill_f32_kernel, dim3((n + 255) / 256), dim3(256), 0, s, out, n,
                       -INFINITY);
    const unsigned slices = (unsigned)((N + kPoolPts - 1) / kPoolPts);
    const size_t esz = bf16 ? 2 : 4;
    const bool vec = C % 8 == 0 && pv_aligned16(x) && ((size_t)x_ld * esz) % 16 == 0;
    if (vec) {
        dim3 g((C + 511) / 512, B, slices);
        if (bf16)
            hipLaunchKernelGGL(pv_maxpool_vec_kernel<uint16_t>, g, dim3(256), 0, s,
                               (const uint16_t*)x, x_ld, N, C, out);
        else
            hipLaunchKernelGGL(pv_maxpool_vec_kernel<float>, g, dim3(256), 0, s, (const float*)x,
                               x_ld, N, C, out);
    } else {
        dim3 g((C + 255) / 256, B, slices);
        if (bf16)
            hipLaunchKernelGGL(pv_maxpool_scalar_kernel<uint16_t>, g, dim3(256), 0, s,
                               (const uint16_t*)x, x_ld, N, C, out);
        else
            hipLaunchKernelGGL(pv_maxpool_scalar_kernel<float>, g, dim3(256), 0, s,
                               (const float*)x, x_ld, N, C, out);
    }
    return pv_launch_status();
}
