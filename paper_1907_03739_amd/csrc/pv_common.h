// Internal helpers shared by the gfx950 kernels of libpvconv.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "pvconv.h"

typedef __attribute__((__vector_size__(8 * sizeof(short)))) short pv_bf16x8;
typedef __attribute__((__vector_size__(16 * sizeof(float)))) float pv_f32x16;
typedef __attribute__((__vector_size__(4 * sizeof(float)))) float pv_f32x4;

// bfloat16 <-> float on raw bits. float -> bf16 uses gfx950's conversion
// instruction (round to nearest, ties to even; NaN stays NaN), no branches.
// Workgroup barrier for LDS data only: orders the LDS accesses around it
// and, unlike __syncthreads(), does not wait for outstanding global loads
// and stores, so loads issued for later work stay in flight across it. Only
// for barriers that hand LDS data between threads.
__device__ __forceinline__ void pv_lds_barrier() {
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "workgroup", "local");
    __builtin_amdgcn_s_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "workgroup", "local");
}

__device__ __forceinline__ float pv_bf16_to_f32(uint16_t h) {
    return __uint_as_float(((uint32_t)h) << 16);
}
__device__ __forceinline__ uint16_t pv_f32_to_bf16(float f) {
    const __bf16 h = (__bf16)f;
    uint16_t u;
    __builtin_memcpy(&u, &h, 2);
    return u;
}
__device__ __forceinline__ uint32_t pv_pack_bf16x2(float lo, float hi) {
    typedef float pv_f2 __attribute__((ext_vector_type(2)));
    typedef __bf16 pv_b2 __attribute__((ext_vector_type(2)));
    const pv_b2 v = __builtin_convertvector((pv_f2){lo, hi}, pv_b2);
    uint32_t u;
    __builtin_memcpy(&u, &v, 4);
    return u;
}

// Folded inference batch norm for one channel: y = x * scale + shift.
struct PvBnFold {
    const float* gamma;
    const float* beta;
    const float* mean;
    const float* var;
    const float* bias;  // linear/conv bias folded in, may be NULL
    float eps;
};

__device__ __forceinline__ void pv_bn_coeffs(const PvBnFold& bn, int c, float& scale,
                                             float& shift) {
    float b = bn.bias ? bn.bias[c] : 0.f;
    if (bn.gamma) {
        scale = bn.gamma[c] / sqrtf(bn.var[c] + bn.eps);
        shift = bn.beta[c] + (b - bn.mean[c]) * scale;
    } else {
        scale = 1.f;
        shift = b;
    }
}

// Activation as x >= 0 ? x : x * neg, with neg = 1 (none), 0 (ReLU) or the
// leaky slope: one compare, one multiply, one select, no branches.
__device__ __forceinline__ float pv_activate(float v, int act, float slope) {
    const float neg = act == PVCONV_ACT_LEAKY ? slope : (act == PVCONV_ACT_RELU ? 0.f : 1.f);
    return v >= 0.f ? v : v * neg;
}

static inline PvBnFold pv_make_fold(const pvconv_bn* bn, const float* bias) {
    PvBnFold f;
    f.gamma = (bn && bn->gamma) ? bn->gamma : nullptr;
    f.beta = f.gamma ? bn->beta : nullptr;
    f.mean = f.gamma ? bn->mean : nullptr;
    f.var = f.gamma ? bn->var : nullptr;
    f.eps = f.gamma ? bn->eps : 0.f;
    f.bias = bias;
    return f;
}

static inline pvconv_status pv_launch_status() {
    return hipGetLastError() == hipSuccess ? PVCONV_OK : PVCONV_EHIP;
}

static inline bool pv_aligned16(const void* p) { return ((uintptr_t)p & 15u) == 0; }

static inline size_t pv_align256(size_t x) { return (x + 255) & ~(size_t)255; }

// bf16 conv weights [Cout][27][Cin] repacked into the MFMA fragment order;
// up to PVCONV_MAX_CONVS jobs per launch
struct PvPackJob {
    const uint16_t* w;
    uint4* packed;
    int Cin, Cout, total, vec, blocks;
};
struct PvPackJobs {
    PvPackJob job[PVCONV_MAX_CONVS];
    int n;
};

// ---- internal launchers (arguments already validated) ---------------------
size_t pv_voxelize_ws_bytes(int B, int N, int R);
// pack (optional): weight-packing jobs run by extra workgroups of the
// voxelisation launch (nullptr: none). sparse: the caller reads the grid only
// at voxels whose count is positive, so the rows of empty voxels are not
// written (honoured where pv_voxelize_sparse_ok(N), else the grid is whole).
pvconv_status pv_launch_voxelize(const float* coords, const void* feats, bool feat_bf16,
                                 int feat_ld, int B, int N, int C, int R, void* grid,
                                 bool grid_bf16, int32_t* counts, int32_t* vox_id,
                                 float* norm_coords, void* ws, hipStream_t s,
                                 const PvPackJobs* pack = nullptr, bool sparse = false);
// the same with the voxel indices given (no normalisation)
pvconv_status pv_launch_voxelize_from_ids(const int32_t* ids, const void* feats, bool feat_bf16,
                                          int feat_ld, int B, int N, int C, int R, void* grid,
                                          bool grid_bf16, int32_t* counts, void* ws,
                                          hipStream_t s, bool sparse = false);
bool pv_voxelize_sparse_ok(int N);
size_t pv_conv3d_ws_bytes(int Cin, int Cout, bool bf16);
// bf16 conv weights [Cout][27][Cin] repacked into the MFMA fragment order
// (into a workspace of pv_conv3d_ws_bytes), the convolutions of a layer in one
// launch
void pv_pack_job(PvPackJobs& jobs, const void* w, int Cin, int Cout, void* packed);
void pv_launch_pack_conv_weights(const PvPackJobs& jobs, hipStream_t s);
static inline int pv_pack_blocks(const PvPackJobs& jobs) {
    int blocks = 0;
    for (int q = 0; q < jobs.n; q++) blocks += jobs.job[q].blocks;
    return blocks;
}
// The packed layout: the convolution's MFMA A fragments in load order, for
// input-channel chunks of kPvPackKC and the 27 taps. Workgroup blk (of
// pv_pack_blocks) of a packing launch, 256 threads, one 16-byte piece each.
constexpr int kPvPackKC = 16;
constexpr int kPvPackTaps = 27;
// tid: the thread's index within its 256-thread share of the workgroup.
__device__ __forceinline__ void pv_pack_role(const PvPackJobs& jobs, int blk,
                                             int tid = threadIdx.x) {
    int q = 0;
    while (q + 1 < jobs.n && blk >= jobs.job[q].blocks) blk -= jobs.job[q++].blocks;
    const PvPackJob& J = jobs.job[q];
    const int i = blk * 256 + tid;
    if (i >= J.total) return;
    const int G = (J.Cout + 31) / 32;  // output channels padded to 32 with zeros
    const int lane = i & 63;
    int r = i >> 6;
    const int g = r % G;
    r /= G;
    const int t = r % kPvPackTaps;
    const int c = r / kPvPackTaps;
    const int n = g * 32 + (lane & 31);
    const int k = c * kPvPackKC + (lane >> 5) * 8;
    if (n >= J.Cout) {
        J.packed[i] = make_uint4(0u, 0u, 0u, 0u);
        return;
    }
    const uint16_t* src = J.w + ((size_t)n * kPvPackTaps + t) * J.Cin;
    if (J.vec) {  // Cin % 8 == 0 and 16-byte aligned rows: one load
        J.packed[i] = k < J.Cin ? *(const uint4*)(src + k) : make_uint4(0u, 0u, 0u, 0u);
        return;
    }
    uint16_t e[8];
#pragma unroll
    for (int j = 0; j < 8; j++) e[j] = k + j < J.Cin ? src[k + j] : (uint16_t)0;
    J.packed[i] = make_uint4((uint32_t)e[0] | ((uint32_t)e[1] << 16),
                             (uint32_t)e[2] | ((uint32_t)e[3] << 16),
                             (uint32_t)e[4] | ((uint32_t)e[5] << 16),
                             (uint32_t)e[6] | ((uint32_t)e[7] << 16));
}
// packed: the bf16 weights are already repacked in ws (w is then unused).
// split_ws: fp32 room for pv_conv3d_split_ws_bytes, or nullptr: grids too
// small to fill the chip then split the input channels across workgroups
// (fixed-order sum of the partials), else they run unsplit. occ: per-voxel
// counts of the input grid [B][R^3] or nullptr; with it, input voxels of
// count 0 read as zero and their rows are never read (a sparse grid). need:
// per-voxel counts of the layer's points [B][R^3] or nullptr; with it only
// the outputs within one voxel of an occupied voxel are computed (those a
// devoxelisation of the points reads), the others left unspecified (where
// given together, occ and need are the same counts).
pvconv_status pv_launch_conv3d(const void* x, int B, int R, int Cin, int Cout, const void* w,
                               const PvBnFold& bn, int act, float slope, bool bf16, void* y,
                               bool out_bf16, void* ws, hipStream_t s, bool packed = false,
                               float* split_ws = nullptr, const int32_t* occ = nullptr,
                               const int32_t* need = nullptr);
int pv_conv3d_splits(int B, int R, int Cin, int Cout);
size_t pv_conv3d_split_ws_bytes(int B, int R, int Cin, int Cout);
pvconv_status pv_launch_devoxelize(const void* grid, int B, int R, int C, bool grid_bf16,
                                   const float* pn, int N, float* out, hipStream_t s);
pvconv_status pv_launch_devoxelize_nearest(const void* grid, int B, int R, int C, bool grid_bf16,
                                           const int32_t* ids, int N, float* out,
                                           hipStream_t s);
// The voxel branch of a PVConv layer as the point MLP's residual: a bf16 grid
// [B][R^3][Cout] devoxelised trilinearly at the normalised coordinates pn
// [B*N][3] (N points per cloud).
struct PvDevoxIn {
    const uint16_t* grid;
    const float* pn;
    int N, R;
};
// Point MLP whose residual is that devoxelisation, gathered inside the GEMM
// kernel (one launch instead of two, no fp32 intermediate). Returns
// PVCONV_ENOTSUP for shapes it does not take; the caller then runs the
// devoxelisation and the point MLP separately.
pvconv_status pv_launch_devox_point_mlp(const PvDevoxIn& dv, const void* x, bool x_bf16,
                                        int x_ld, int M, int Cin, int Cout, const void* w,
                                        const PvBnFold& bn, int act, float slope, void* out,
                                        bool out_bf16, int out_ld, hipStream_t s);
pvconv_status pv_launch_point_mlp(const void* x, bool x_bf16, int x_ld, int M, int Cin,
                                  int Cout, const void* w, bool bf16, const PvBnFold& bn,
                                  int act, float slope, const float* cloud_bias, int ppc,
                                  const float* residual, int res_ld, void* out, bool out_bf16,
                                  int out_ld, hipStream_t s);
pvconv_status pv_launch_maxpool(const void* x, bool bf16, int x_ld, int B, int N, int C,
                                float* out, hipStream_t s);
// PointNet++ primitives of PVCNN++ (pointnet2.hip)
constexpr int kPvFpsMaxN = 16384;  // points per cloud farthest point sampling takes
pvconv_status pv_launch_fps(const float* xyz, int B, int N, int npoint, int32_t* idx,
                            float* new_xyz, hipStream_t s);
pvconv_status pv_launch_ball_query(const float* xyz, int B, int N, const float* centers, int M,
                                   float radius, int nsample, int32_t* idx, hipStream_t s);
pvconv_status pv_launch_group(const float* xyz, const void* feats, bool feat_bf16, int feat_ld,
                              int B, int N, int C, const float* centers, int M,
                              const int32_t* idx, int nsample, void* out, bool out_bf16,
                              int out_ld, hipStream_t s);
pvconv_status pv_launch_three_nn(const float* unknown, int B, int n, const float* known, int m,
                                 int32_t* idx, float* weight, hipStream_t s);
pvconv_status pv_launch_three_interpolate(const void* feats, bool feat_bf16, int feat_ld, int B,
                                          int m, int C, const int32_t* idx, const float* weight,
                                          int n, void* out, bool out_bf16, int out_ld,
                                          hipStream_t s);
pvconv_status pv_launch_group_max(const void* x, bool x_bf16, int x_ld, int G, int S, int C,
                                  void* out, bool out_bf16, int out_ld, hipStream_t s);
// backward (backward.hip)
size_t pv_conv3d_bwd_data_ws_bytes(int Cin, int Cout, bool bf16);
pvconv_status pv_launch_voxelize_backward(const void* dgrid, bool bf16, int B, int N, int C,
                                          int R, const int32_t* ids, const int32_t* counts,
                                          float* dfeats, hipStream_t s);
// ids != NULL: nearest neighbour (pn unused), else trilinear; workspace of
// pv_devox_bwd_ws_bytes (256-byte aligned; unused when N == 0)
size_t pv_devox_bwd_ws_bytes(int B, int N, int C, int R);
pvconv_status pv_launch_devoxelize_backward(const float* dout, int B, int N, int C, int R,
                                            const float* pn, const int32_t* ids, float* dgrid,
                                            void* workspace, hipStream_t s);
pvconv_status pv_launch_conv3d_backward_data(const void* dy, int B, int R, int Cin, int Cout,
                                             const void* w, bool bf16, void* dx, bool dx_bf16,
                                             void* ws, hipStream_t s);
size_t pv_conv3d_wgrad_ws_bytes(int B, int R, int Cin, int Cout);
pvconv_status pv_launch_conv3d_backward_weight(const void* dy, const void* x, int B, int R,
                                               int Cin, int Cout, float* dw, void* ws,
                                               hipStream_t s);
pvconv_status pv_launch_act_bn_backward(const float* dy, const void* y, bool y_bf16, size_t M,
                                        int C, const PvBnFold& bn, int act, float slope,
                                        float* dz, hipStream_t s);
