// 3x3x3 volumetric convolution + folded batch norm + activation
// (Section 4.1 "Feature Aggregation"; fixed-offset kernel of Section 3, Eq. 1).
//
// bf16 path: implicit GEMM on the MFMA units. M = output voxels, N = output
// channels, K = 27 taps x input channels. A workgroup owns a 4x8x8 brick of
// output voxels and NT output channels. For each chunk of 32 input channels it
// stages the brick's 6x10x10 halo in LDS once (zero-filled outside the grid),
// then walks the 27 taps: each tap's A operand is the halo shifted by the tap
// offset, read straight from LDS, and the tap's NT x 32 weight slice is
// double-buffered through LDS. Each of the 4 waves computes one u-slice of the
// brick (64 voxels = two 32-row MFMA blocks) against all NT channels with
// v_mfma_f32_32x32x16_bf16, so every A fragment feeds NT/32 MFMAs and every B
// fragment two. The epilogue folds bias + batch norm into one scale/shift per
// channel, applies the activation and stores bf16 or fp32.
//
// fp32 path: one thread per (voxel, output channel), plain FMA loop.
#include "pv_common.h"

namespace {

constexpr int kBU = 4, kBV = 8, kBW = 8;     // output brick (u, v, w)
constexpr int kHU = kBU + 2, kHV = kBV + 2, kHW = kBW + 2;
constexpr int kHaloVox = kHU * kHV * kHW;    // 600
constexpr int kKC = 32;                      // input channels per K chunk
constexpr int kRow = kKC + 8;                // LDS row pitch in bf16 (80 B: conflict-free b128 reads)
constexpr int kThreads = 256;

__device__ __forceinline__ uint4 pack8(const uint16_t* e) {
    return make_uint4((uint32_t)e[0] | ((uint32_t)e[1] << 16), (uint32_t)e[2] | ((uint32_t)e[3] << 16),
                      (uint32_t)e[4] | ((uint32_t)e[5] << 16), (uint32_t)e[6] | ((uint32_t)e[7] << 16));
}

template <int NT, bool VEC>
__global__ __launch_bounds__(kThreads, 2) void pv_conv3d_bf16_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ w, PvBnFold bn, int act,
    float slope, void* __restrict__ y, int out_bf16, int R, int Cin, int Cout, int nbu, int nbv,
    int nbw) {
    __shared__ __attribute__((aligned(16))) uint16_t halo[kHaloVox * kRow];
    __shared__ __attribute__((aligned(16))) uint16_t wbuf[2][NT * kRow];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    int bid = blockIdx.x;
    const int nblk_n = Cout / NT;
    const int nt = bid % nblk_n;
    bid /= nblk_n;
    const int bw = bid % nbw;
    bid /= nbw;
    const int bv = bid % nbv;
    bid /= nbv;
    const int bu = bid % nbu;
    const int b = bid / nbu;
    const int u0 = bu * kBU, v0 = bv * kBV, w0 = bw * kBW, n0 = nt * NT;
    const size_t cloud = (size_t)b * R * R * R;

    constexpr int NB = NT / 32;
    pv_f32x16 acc[2][NB];
    for (int i = 0; i < 2; i++)
        for (int j = 0; j < NB; j++)
            for (int e = 0; e < 16; e++) acc[i][j][e] = 0.f;

    // Weight slice (tap, cc) -> registers: NT rows x 32 channels = NT*4 chunks
    // of 16 B; each thread owns NT*4/256 chunks.
    constexpr int WCHUNKS = NT * 4;
    constexpr int WCH = (WCHUNKS + kThreads - 1) / kThreads;
    uint4 wreg[WCH];
    auto load_w = [&](int tap, int cc) {
        for (int i = 0; i < WCH; i++) {
            const int ch = tid + i * kThreads;
            if (ch >= WCHUNKS) break;
            const int n = ch >> 2, q = ch & 3;
            const int c = cc + q * 8;
            const uint16_t* src = w + ((size_t)(n0 + n) * 27 + tap) * Cin + c;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (VEC) {
                if (c < Cin) v = *(const uint4*)src;
            } else {
                uint16_t e[8];
                for (int t = 0; t < 8; t++) e[t] = (c + t < Cin) ? src[t] : (uint16_t)0;
                v = pack8(e);
            }
            wreg[i] = v;
        }
    };
    auto store_w = [&](int buf) {
        for (int i = 0; i < WCH; i++) {
            const int ch = tid + i * kThreads;
            if (ch >= WCHUNKS) break;
            const int n = ch >> 2, q = ch & 3;
            *(uint4*)&wbuf[buf][n * kRow + q * 8] = wreg[i];
        }
    };

    // A-fragment row of this lane: voxel (lv, lw) inside the wave's u-slice.
    const int r32 = lane & 31, khalf = (lane >> 5) * 8;

    for (int cc = 0; cc < Cin; cc += kKC) {
        __syncthreads();  // previous chunk's readers are done with halo / wbuf
        for (int idx = tid; idx < kHaloVox * 4; idx += kThreads) {
            const int hv = idx >> 2, q = idx & 3;
            const int hu = hv / (kHV * kHW), rem = hv - hu * (kHV * kHW);
            const int hvv = rem / kHW, hw = rem - hvv * kHW;
            const int gu = u0 + hu - 1, gv = v0 + hvv - 1, gw = w0 + hw - 1;
            const int c = cc + q * 8;
            uint4 v = make_uint4(0, 0, 0, 0);
            if (gu >= 0 && gu < R && gv >= 0 && gv < R && gw >= 0 && gw < R && c < Cin) {
                const uint16_t* src = x + (cloud + ((size_t)gu * R + gv) * R + gw) * Cin + c;
                if (VEC) {
                    v = *(const uint4*)src;
                } else {
                    uint16_t e[8];
                    for (int t = 0; t < 8; t++) e[t] = (c + t < Cin) ? src[t] : (uint16_t)0;
                    v = pack8(e);
                }
            }
            *(uint4*)&halo[hv * kRow + q * 8] = v;
        }
        load_w(0, cc);
        store_w(0);
        __syncthreads();
        const int ksteps = (Cin - cc) >= kKC ? 2 : ((Cin - cc) + 15) / 16;
        for (int tap = 0; tap < 27; ++tap) {
            if (tap + 1 < 27) load_w(tap + 1, cc);
            const int du = tap / 9, dv = (tap / 3) % 3, dw = tap % 3;  // offset + 1
            const uint16_t* wb = wbuf[tap & 1];
            for (int ks = 0; ks < ksteps; ++ks) {
                pv_bf16x8 a[2], bb[NB];
                for (int mb = 0; mb < 2; mb++) {
                    const int lv = mb * 4 + (r32 >> 3), lw = r32 & 7;
                    const int h = ((wave + du) * kHV + (lv + dv)) * kHW + (lw + dw);
                    a[mb] = *(const pv_bf16x8*)&halo[h * kRow + ks * 16 + khalf];
                }
                for (int nb = 0; nb < NB; nb++)
                    bb[nb] = *(const pv_bf16x8*)&wb[(nb * 32 + r32) * kRow + ks * 16 + khalf];
                for (int mb = 0; mb < 2; mb++)
                    for (int nb = 0; nb < NB; nb++)
                        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(a[mb], bb[nb],
                                                                             acc[mb][nb], 0, 0, 0);
            }
            if (tap + 1 < 27) store_w((tap + 1) & 1);
            __syncthreads();
        }
    }

    // Epilogue. Lane holds column n = r32 of each 32x32 block and rows
    // 8*(e/4) + 4*(lane/32) + e%4 for e = 0..15.
    const int u = u0 + wave;
    for (int nb = 0; nb < NB; nb++) {
        const int n = n0 + nb * 32 + r32;
        float scale, shift;
        pv_bn_coeffs(bn, n, scale, shift);
        for (int mb = 0; mb < 2; mb++) {
            for (int e = 0; e < 16; e++) {
                const int row = 8 * (e >> 2) + 4 * (lane >> 5) + (e & 3);
                const int v = v0 + mb * 4 + (row >> 3), ww = w0 + (row & 7);
                if (u >= R || v >= R || ww >= R) continue;
                const float val = pv_activate(acc[mb][nb][e] * scale + shift, act, slope);
                const size_t o = (cloud + ((size_t)u * R + v) * R + ww) * Cout + n;
                if (out_bf16)
                    ((uint16_t*)y)[o] = pv_f32_to_bf16(val);
                else
                    ((float*)y)[o] = val;
            }
        }
    }
}

__global__ __launch_bounds__(256) void pv_conv3d_f32_kernel(const float* __restrict__ x,
                                                            const float* __restrict__ w,
                                                            PvBnFold bn, int act, float slope,
                                                            void* __restrict__ y, int out_bf16,
                                                            int B, int R, int Cin, int Cout) {
    const size_t V = (size_t)R * R * R;
    const size_t i = (size_t)blockIdx.x * 256 + threadIdx.x;
    if (i >= (size_t)B * V * Cout) return;
    const int o = (int)(i % Cout);
    const size_t vox = i / Cout;
    const size_t b = vox / V;
    const int r = (int)(vox % V);
    const int u = r / (R * R), v = (r / R) % R, ww = r % R;
    float s = 0.f;
    for (int tap = 0; tap < 27; tap++) {
        const int nu = u + tap / 9 - 1, nv = v + (tap / 3) % 3 - 1, nw = ww + tap % 3 - 1;
        if (nu < 0 || nu >= R || nv < 0 || nv >= R || nw < 0 || nw >= R) continue;
        const float* xi = x + (b * V + ((size_t)nu * R + nv) * R + nw) * Cin;
        const float* wk = w + ((size_t)o * 27 + tap) * Cin;
        for (int c = 0; c < Cin; c++) s += wk[c] * xi[c];
    }
    float scale, shift;
    pv_bn_coeffs(bn, o, scale, shift);
    const float val = pv_activate(s * scale + shift, act, slope);
    if (out_bf16)
        ((uint16_t*)y)[i] = pv_f32_to_bf16(val);
    else
        ((float*)y)[i] = val;
}

template <int NT>
void launch_bf16(const void* x, int B, int R, int Cin, int Cout, const void* w,
                 const PvBnFold& bn, int act, float slope, void* y, bool out_bf16, bool vec,
                 hipStream_t s) {
    const int nbu = (R + kBU - 1) / kBU, nbv = (R + kBV - 1) / kBV, nbw = (R + kBW - 1) / kBW;
    const size_t blocks = (size_t)B * nbu * nbv * nbw * (Cout / NT);
    if (vec)
        hipLaunchKernelGGL((pv_conv3d_bf16_kernel<NT, true>), dim3((unsigned)blocks),
                           dim3(kThreads), 0, s, (const uint16_t*)x, (const uint16_t*)w, bn, act,
                           slope, y, (int)out_bf16, R, Cin, Cout, nbu, nbv, nbw);
    else
        hipLaunchKernelGGL((pv_conv3d_bf16_kernel<NT, false>), dim3((unsigned)blocks),
                           dim3(kThreads), 0, s, (const uint16_t*)x, (const uint16_t*)w, bn, act,
                           slope, y, (int)out_bf16, R, Cin, Cout, nbu, nbv, nbw);
}

}  // namespace

pvconv_status pv_launch_conv3d(const void* x, int B, int R, int Cin, int Cout, const void* w,
                               const PvBnFold& bn, int act, float slope, bool bf16, void* y,
                               bool out_bf16, hipStream_t s) {
    if (B == 0) return PVCONV_OK;
    if (bf16) {
        const bool vec = (Cin % 8 == 0) && pv_aligned16(x) && pv_aligned16(w);
        if (Cout % 128 == 0)
            launch_bf16<128>(x, B, R, Cin, Cout, w, bn, act, slope, y, out_bf16, vec, s);
        else if (Cout % 64 == 0)
            launch_bf16<64>(x, B, R, Cin, Cout, w, bn, act, slope, y, out_bf16, vec, s);
        else
            launch_bf16<32>(x, B, R, Cin, Cout, w, bn, act, slope, y, out_bf16, vec, s);
    } else {
        const size_t total = (size_t)B * R * R * R * Cout;
        hipLaunchKernelGGL(pv_conv3d_f32_kernel, dim3((unsigned)((total + 255) / 256)), dim3(256),
                           0, s, (const float*)x, (const float*)w, bn, act, slope, y,
                           (int)out_bf16, B, R, Cin, Cout);
    }
    return pv_launch_status();
}
