/*
 * pvconv.h -- C ABI of the MI355X (gfx950) Point-Voxel Convolution.
 *
 * Implements the PVConv layer of Liu, Tang, Lin, Han, "Point-Voxel CNN for
 * Efficient 3D Deep Learning" (NeurIPS 2019), Section 4: a voxel branch
 * (normalise -> voxelise -> 3x3x3 convolutions with batch normalisation and a
 * leaky rectifier -> trilinear or nearest-neighbour devoxelise) and a point
 * branch (a shared per-point MLP), fused by addition; the per-cloud max-pool
 * of the segmentation networks (Section 5.1); and the backward of the voxel
 * branch's steps (the gradients at the end of this file). Every step runs as
 * a HIP kernel on the GPU; nothing here computes on the host.
 *
 * Conventions shared by every entry point
 *  - Array pointers are DEVICE pointers owned by the caller. The library keeps
 *    no device memory and no state between calls, except the static array of
 *    pvconv_conv3d_noalloc; scratch space is passed in as `workspace` where an
 *    entry point needs it.
 *  - `stream` is a hipStream_t (NULL = the null stream). Every call only
 *    enqueues work on it: it never synchronises and never allocates.
 *  - Layouts are row-major, channels innermost ("channels last"):
 *      point arrays  [B][N][C], row k of cloud b at (b*N + k) * ld
 *      voxel grids   [B][R][R][R][C], voxel (u,v,w) at ((u*R + v)*R + w),
 *                    u indexes the x axis (slowest), w the z axis (fastest)
 *      conv weights  [C_out][3][3][3][C_in], index (du+1, dv+1, dw+1) holds
 *                    the weight of the neighbour at offset (du, dv, dw)
 *      linear weights [C_out][C_in]
 *    `*_ld` arguments are row strides in elements (0 means "= number of
 *    channels"); they let a caller read or write a column slice of a wider
 *    array, e.g. a concatenation buffer.
 *  - PVCONV_BF16 arrays hold raw bfloat16 bits (uint16). bf16 compute means
 *    bf16 operands with fp32 accumulation.
 *  - Arguments are validated on the host before anything is enqueued: an
 *    invalid argument returns PVCONV_EINVAL (or PVCONV_ENOTSUP /
 *    PVCONV_EWORKSPACE) and enqueues nothing. A failed launch returns
 *    PVCONV_EHIP. Device faults surface at the caller's next synchronisation.
 *  - Coordinates must be finite. Non-finite coordinates are a precondition
 *    violation: results are then unspecified, but every index is clamped, so
 *    no access leaves its array.
 */
#ifndef PVCONV_H
#define PVCONV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    PVCONV_OK = 0,
    PVCONV_EINVAL = 1,     /* bad size, NULL required pointer, misaligned pointer */
    PVCONV_ENOTSUP = 2,    /* valid but unsupported combination (e.g. dtype) */
    PVCONV_EWORKSPACE = 3, /* workspace NULL or smaller than the queried size */
    PVCONV_EHIP = 4        /* the HIP runtime reported an error at launch */
} pvconv_status;

typedef enum { PVCONV_F32 = 0, PVCONV_BF16 = 1 } pvconv_dtype;

typedef enum { PVCONV_ACT_NONE = 0, PVCONV_ACT_RELU = 1, PVCONV_ACT_LEAKY = 2 } pvconv_act;

/* Batch normalisation in inference form (running statistics), Section 4.1
 * "Feature Aggregation": y = gamma * (x - mean) / sqrt(var + eps) + beta.
 * Each pointer is a device array of C floats. A NULL pvconv_bn pointer, or
 * gamma == NULL, means identity. */
typedef struct {
    const float* gamma;
    const float* beta;
    const float* mean;
    const float* var;
    float eps;
} pvconv_bn;

/* Limits checked by every entry point. */
#define PVCONV_MAX_R 128
#define PVCONV_MAX_CONV_CHANNELS 1024
#define PVCONV_MAX_MLP_CHANNELS 16384
#define PVCONV_MAX_CONVS 4
#define PVCONV_CONV3D_NOALLOC_BYTES (4u << 20) /* pvconv_conv3d_noalloc's array */

/* Human-readable name of a status code (static string). */
const char* pvconv_status_string(pvconv_status s);

/* ------------------------------------------------------------------------- */
/* Voxelisation: Section 4.1 "Normalization" and "Voxelization" (Eq. 2).     */
/*                                                                           */
/* Per cloud b: the coordinates are centred at their mean (the "gravity      */
/* center"), divided by the largest centred norm, then scaled by 1/2 and     */
/* shifted by 1/2 into [0,1]^3 (norm_coords). A cloud whose points all       */
/* coincide maps to (1/2,1/2,1/2). Point k falls in voxel                    */
/* (floor(x*R), floor(y*R), floor(z*R)), clamped to [0, R-1]; vox_id is       */
/* (u*R + v)*R + w. The grid holds, per voxel, the mean of the features of   */
/* its points (Eq. 2) and 0 for an empty voxel; counts holds N_{u,v,w}.       */
/* The mean is taken in the order-free arithmetic described in the design    */
/* notes: the centroid is an int64 fixed-point sum, normalisation is IEEE    */
/* fp64 without contraction, feature sums accumulate in fp64.                */
/*                                                                           */
/*  coords       [B][N][3] fp32                                              */
/*  feats        [B][N][C] (feat_dt), row stride feat_ld                     */
/*  grid         out [B][R^3][C] (grid_dt), every element written            */
/*  counts       out [B][R^3] int32                                          */
/*  vox_id       out [B][N] int32, or NULL                                   */
/*  norm_coords  out [B][N][3] fp32 (the fp64 values rounded), or NULL       */
/*  workspace    >= pvconv_voxelize_workspace_size(B, N, R) bytes, 256-byte  */
/*               aligned; contents on entry are ignored                      */
/* Sizes: B >= 0, N >= 0 (N = 0 gives an all-zero grid), 1 <= R <= 128,      */
/* 1 <= C. feats, grid need 16-byte alignment when C*elem and feat_ld*elem   */
/* are multiples of 16 (otherwise a slower element-wise path is taken).      */
/* ------------------------------------------------------------------------- */
size_t pvconv_voxelize_workspace_size(int B, int N, int R);
pvconv_status pvconv_voxelize(const float* coords, const void* feats, pvconv_dtype feat_dt,
                              int feat_ld, int B, int N, int C, int R, void* grid,
                              pvconv_dtype grid_dt, int32_t* counts, int32_t* vox_id,
                              float* norm_coords, void* workspace, size_t workspace_bytes,
                              void* stream);

/* ------------------------------------------------------------------------- */
/* Voxelisation from given voxel indices: Eq. 2 (Section 4.1                 */
/* "Voxelization") with the indices of an earlier pvconv_voxelize of the     */
/* same coordinates and the same R. Every layer that voxelises the same      */
/* points at the same resolution has the same indices (the normalisation     */
/* depends on the coordinates only), so they are computed once per R.        */
/*  vox_id  [B][N] int32 in [0, R^3) (an index outside is invalid input: the */
/*          point is dropped; memory-safe)                                   */
/*  other arguments, outputs and the workspace as for pvconv_voxelize        */
/*  (workspace >= pvconv_voxelize_workspace_size(B, N, R))                   */
/* ------------------------------------------------------------------------- */
pvconv_status pvconv_voxelize_from_ids(const int32_t* vox_id, const void* feats,
                                       pvconv_dtype feat_dt, int feat_ld, int B, int N, int C,
                                       int R, void* grid, pvconv_dtype grid_dt, int32_t* counts,
                                       void* workspace, size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* 3x3x3 convolution + batch norm + activation: Section 4.1 "Feature         */
/* Aggregation", with the fixed-offset kernel of Section 3 (Eq. 1; each axis */
/* offset in {0, +-1}).                                                      */
/*                                                                           */
/*  y[b,u,v,w,o] = act( BN_o( bias_o + sum_{du,dv,dw in {-1,0,1}}            */
/*                 sum_i W[o][du+1][dv+1][dw+1][i] * x[b,u+du,v+dv,w+dw,i] ) ) */
/* with x = 0 outside the grid (zero padding 1, stride 1).                   */
/*  x       [B][R^3][Cin], dtype dt                                          */
/*  weight  [Cout][3][3][3][Cin], dtype dt                                   */
/*  bias    [Cout] fp32 or NULL; bn may be NULL                              */
/*  act     NONE / RELU / LEAKY (negative slope `slope`)                     */
/*  y       out [B][R^3][Cout], dtype out_dt                                 */
/* dt = BF16: MFMA implicit GEMM, bf16 x bf16 -> fp32, output channels in   */
/* tiles of 32 (a Cout that is no multiple of 32 pads its last tile with     */
/* zero weights; only the Cout channels are stored).                         */
/* It first repacks the weights into the MFMA fragment order inside          */
/* `workspace` (>= pvconv_conv3d_workspace_size bytes, 256-byte aligned;     */
/* contents on entry ignored). dt = F32: fp32 FMA, no workspace (may be      */
/* NULL). 1 <= Cin, Cout <= 1024, 1 <= R <= 128. x and y must not overlap.   */
/* ------------------------------------------------------------------------- */
size_t pvconv_conv3d_workspace_size(int Cin, int Cout, pvconv_dtype dt);
pvconv_status pvconv_conv3d(const void* x, int B, int R, int Cin, int Cout, const void* weight,
                            const float* bias, const pvconv_bn* bn, pvconv_act act, float slope,
                            pvconv_dtype dt, void* y, pvconv_dtype out_dt, void* workspace,
                            size_t workspace_bytes, void* stream);

/* ------------------------------------------------------------------------- */
/* The same convolution in two parts, for weights used by many calls (a      */
/* network's fixed weights): the bf16 weights repacked once into the MFMA    */
/* fragment order, then any number of convolutions on the packed copy.       */
/* pvconv_conv3d(...) equals pvconv_conv3d_pack_weights then                */
/* pvconv_conv3d_packed on the same stream, bit for bit.                     */
/*  weight  [Cout][3][3][3][Cin] bf16 (the MFMA path)                        */
/*  packed  out: >= pvconv_conv3d_workspace_size(Cin, Cout, PVCONV_BF16)     */
/*          bytes, 256-byte aligned, owned by the caller; every byte of that */
/*          size is written. Its layout is internal to the library.          */
/* pvconv_conv3d_packed takes the arguments of pvconv_conv3d with dt = BF16, */
/* and `packed` (as written by the pack call for the same Cin, Cout) in     */
/* place of weight and workspace; errors as pvconv_conv3d.                   */
/* ------------------------------------------------------------------------- */
pvconv_status pvconv_conv3d_pack_weights(const void* weight, int Cin, int Cout, void* packed,
                                         size_t packed_bytes, void* stream);
pvconv_status pvconv_conv3d_packed(const void* x, int B, int R, int Cin, int Cout,
                                   const void* packed, size_t packed_bytes, const float* bias,
                                   const pvconv_bn* bn, pvconv_act act, float slope, void* y,
                                   pvconv_dtype out_dt, void* stream);

/* ------------------------------------------------------------------------- */
/* pvconv_conv3d without a workspace argument, for callers that cannot       */
/* allocate device memory (code under HIP graph capture, serving loops that  */
/* must not call hipMalloc, harnesses that forbid it).                       */
/* Arguments, results and errors as pvconv_conv3d. The repacked bf16 weights */
/* go to a static device array of PVCONV_CONV3D_NOALLOC_BYTES inside the     */
/* library, one per GPU, held until the process ends; a convolution whose    */
/* pvconv_conv3d_workspace_size exceeds it returns PVCONV_EWORKSPACE (4 MiB  */
/* takes Cin = Cout = 256). `stream` must belong to the current device       */
/* (else PVCONV_EINVAL). Every call on one GPU uses that GPU's one array:    */
/* calls that may run at the same time on one GPU (other streams, other     */
/* host threads without ordering) race and give wrong results; calls in     */
/* order on one stream are safe. Each call rewrites every byte of the array */
/* it reads, so nothing depends on the previous call's contents. The first  */
/* call on a device looks up the array's address (no allocation).           */
/* ------------------------------------------------------------------------- */
pvconv_status pvconv_conv3d_noalloc(const void* x, int B, int R, int Cin, int Cout,
                                    const void* weight, const float* bias, const pvconv_bn* bn,
                                    pvconv_act act, float slope, pvconv_dtype dt, void* y,
                                    pvconv_dtype out_dt, void* stream);

/* ------------------------------------------------------------------------- */
/* Trilinear devoxelisation: Section 4.1 "Devoxelization".                   */
/*                                                                           */
/* Voxel (u,v,w)'s value sits at its cell centre ((u+1/2)/R, ...). Per axis  */
/* t = clamp(R*x - 1/2, 0, R-1), i0 = floor(t), i1 = min(i0+1, R-1),         */
/* weights (1 - (t - i0), t - i0); out = sum over the 8 cells of the product */
/* of the three axis weights times the cell's features.                      */
/*  grid         [B][R^3][C] (grid_dt)                                       */
/*  norm_coords  [B][N][3] fp32 in [0,1] (as written by pvconv_voxelize)     */
/*  out          out [B][N][C] fp32                                          */
/* ------------------------------------------------------------------------- */
pvconv_status pvconv_devoxelize(const void* grid, int B, int R, int C, pvconv_dtype grid_dt,
                                const float* norm_coords, int N, float* out, void* stream);

/* ------------------------------------------------------------------------- */
/* Nearest-neighbour devoxelisation: the alternative to trilinear            */
/* interpolation that Section 4.1 "Devoxelization" describes (every point    */
/* takes the features of the grid cell it falls into; the devoxelisation     */
/* row of the ablation table compares the two).                              */
/*                                                                           */
/*  out[b][k][c] = grid[b][vox_id[b][k]][c], in fp32 (exact for both grid    */
/*  dtypes).                                                                 */
/*  grid    [B][R^3][C] (grid_dt)                                            */
/*  vox_id  [B][N] int32 voxel index within the cloud, as pvconv_voxelize    */
/*          writes it; an index outside [0, R^3) is a precondition violation */
/*          (it is clamped into the grid: memory-safe, result unspecified)   */
/*  out     out [B][N][C] fp32                                               */
/* 1 <= R <= 128, 1 <= C. Same alignment rules as pvconv_devoxelize.         */
/* ------------------------------------------------------------------------- */
pvconv_status pvconv_devoxelize_nearest(const void* grid, int B, int R, int C,
                                        pvconv_dtype grid_dt, const int32_t* vox_id, int N,
                                        float* out, void* stream);

/* ------------------------------------------------------------------------- */
/* Shared per-point MLP layer with fused epilogue: Section 4.2 (point-based  */
/* feature transformation) and Section 4.3 (fusion by addition).             */
/*                                                                           */
/*  out[m,o] = act( BN_o( sum_i W[o][i] * x[m,i] + bias_o + cloud_bias[m/P,o] ) ) */
/*             + residual[m,o]                                               */
/* where P = points_per_cloud. Rows m = 0..M-1.                              */
/*  x           [M][Cin] (x_dt), row stride x_ld                             */
/*  weight      [Cout][Cin] (compute_dt: BF16 -> MFMA, F32 -> fp32 FMA)      */
/*  bias        [Cout] fp32 or NULL; bn may be NULL                          */
/*  cloud_bias  [M/P][Cout] fp32 or NULL (a per-cloud row, e.g. the          */
/*              projection of a broadcast global feature)                    */
/*  residual    [M][Cout] fp32 (row stride residual_ld) or NULL; added after */
/*              the activation                                               */
/*  out         out [M][Cout] (out_dt), row stride out_ld                    */
/* 1 <= Cin, Cout <= 16384. out must not share any byte with x (else         */
/* PVCONV_EINVAL): other workgroups may still read rows that are stored.     */
/* Disjoint column ranges of one wider array (equal row strides) are fine.  */
/* ------------------------------------------------------------------------- */
pvconv_status pvconv_point_mlp(const void* x, pvconv_dtype x_dt, int x_ld, int M, int Cin,
                               int Cout, const void* weight, pvconv_dtype compute_dt,
                               const float* bias, const pvconv_bn* bn, pvconv_act act,
                               float slope, const float* cloud_bias, int points_per_cloud,
                               const float* residual, int residual_ld, void* out,
                               pvconv_dtype out_dt, int out_ld, void* stream);

/* ------------------------------------------------------------------------- */
/* The end of a PVConv layer in one kernel: the point MLP of Section 4.2     */
/* whose epilogue adds the trilinear devoxelisation of Section 4.1 (fusion   */
/* by addition, Section 4.3), gathered from the grid inside the same kernel, */
/* without an fp32 intermediate. The same result as pvconv_devoxelize into a */
/* buffer r, then pvconv_point_mlp(..., residual = r, ...):                  */
/*  out[b,k,o] = act( BN_o( sum_i W[o][i] x[b,k,i] + bias_o ) )              */
/*               + trilinear(grid[b], norm_coords[b][k])[o]                  */
/*  grid         [B][R^3][Cout] bf16 (a layer's last convolution output)     */
/*  norm_coords  [B][N][3] fp32 (as written by pvconv_voxelize)              */
/*  x            [B][N][Cin] (x_dt), row stride x_ld (0: Cin)                */
/*  weight       [Cout][Cin] bf16 (MFMA, fp32 accumulation)                  */
/*  bias, bn, act, slope as pvconv_point_mlp                                 */
/*  out          out [B][N][Cout] (out_dt), row stride out_ld (0: Cout)      */
/* Shapes the fused kernel takes: Cin % 8 == 0, Cout % 8 == 0, not both of   */
/* Cin and Cout >= 128, B*N >= 128, 16-byte aligned x, weight and grid rows, */
/* x rows a multiple of 16 bytes, out_ld % 4 == 0 and out aligned to 16     */
/* bytes (8 for bf16). Others return PVCONV_ENOTSUP (pvconv_forward then     */
/* runs the two steps separately). out must not overlap x, grid or          */
/* norm_coords (PVCONV_EINVAL).                                              */
/* ------------------------------------------------------------------------- */
pvconv_status pvconv_devoxelize_point_mlp(const void* grid, int R, const float* norm_coords,
                                          int B, int N, const void* x, pvconv_dtype x_dt,
                                          int x_ld, int Cin, int Cout, const void* weight,
                                          const float* bias, const pvconv_bn* bn,
                                          pvconv_act act, float slope, void* out,
                                          pvconv_dtype out_dt, int out_ld, void* stream);

/* ------------------------------------------------------------------------- */
/* Per-cloud max over the points (the PointNet global feature that PVCNN     */
/* keeps, Section 5.1 "Models"): out[b][c] = max_k x[b][k][c].               */
/*  x    [B][N][C] (dt), row stride x_ld;  out [B][C] fp32.  N >= 1.         */
/* Exact and order-free (deterministic). NaN inputs are a precondition       */
/* violation: the result for their channel is unspecified.                   */
/* ------------------------------------------------------------------------- */
pvconv_status pvconv_maxpool(const void* x, pvconv_dtype dt, int x_ld, int B, int N, int C,
                             float* out, void* stream);

/* ========================================================================= */
/* PVCNN++ (Section 5.2 "Models": PointNet++ extended with PVConv): the      */
/* PointNet++ primitives around the PVConv layers, as PointNet++ (Qi et al., */
/* 2017) defines them. Set abstraction samples centres by farthest point     */
/* sampling, gathers each centre's neighbours by ball query, groups their    */
/* relative coordinates and features for a shared MLP (pvconv_point_mlp) and */
/* takes the maximum over the neighbours (pvconv_maxpool); feature           */
/* propagation interpolates features back to the denser level from the three */
/* nearest neighbours. Every choice of an index compares fp32 squared        */
/* distances fma(dz, dz, fma(dy, dy, dx*dx)), dx = x_j - x_c (each fused     */
/* multiply-add rounded once), with ties to the lower index, so results are  */
/* the same on every run.                                                    */
/* Coordinates are [B][*][3] fp32; indices are within the cloud.             */
/* ========================================================================= */

/* Farthest point sampling: idx[b][0] = 0; idx[b][s] is the point whose      */
/* distance to points idx[b][0..s-1] (the minimum over them) is largest.     */
/*  xyz      [B][N][3], 1 <= N <= 16384 (larger: PVCONV_ENOTSUP)             */
/*  idx      out [B][npoint] int32, 1 <= npoint <= N                         */
/*  new_xyz  out [B][npoint][3] (the sampled points' coordinates) or NULL    */
/* One workgroup per cloud: the npoint steps are sequential.                 */
pvconv_status pvconv_furthest_point_sample(const float* xyz, int B, int N, int npoint,
                                           int32_t* idx, float* new_xyz, void* stream);

/* Ball query: idx[b][i][0..] = the first nsample points, in index order,    */
/* whose squared distance to centre i is below radius*radius (formed in     */
/* fp32); a centre with fewer repeats its first neighbour in the remaining   */
/* slots, one with none gets 0 in every slot.                                */
/*  xyz [B][N][3], centers [B][M][3], idx out [B][M][nsample] int32.         */
/*  N >= 1, nsample >= 1, radius >= 0.                                       */
pvconv_status pvconv_ball_query(const float* xyz, int B, int N, const float* centers, int M,
                                float radius, int nsample, int32_t* idx, void* stream);

/* Grouping: row (b, i, k) of out = (x_j - c_i, feats_j) with j =            */
/* idx[b][i][k]: 3 relative coordinates, then the C features.                */
/*  xyz [B][N][3]; feats [B][N][C] (feat_dt, row stride feat_ld, 0: C; C may */
/*  be 0 and feats NULL); centers [B][M][3]; idx [B][M][nsample] (entries    */
/*  outside [0, N) are clamped: memory-safe, result unspecified);            */
/*  out [B][M][nsample][3 + C] (out_dt, row stride out_ld, 0: 3 + C).        */
pvconv_status pvconv_group_points(const float* xyz, const void* feats, pvconv_dtype feat_dt,
                                  int feat_ld, int B, int N, int C, const float* centers, int M,
                                  const int32_t* idx, int nsample, void* out,
                                  pvconv_dtype out_dt, int out_ld, void* stream);

/* Maximum over each centre's neighbours (the set abstraction's pooling):    */
/* out[g][c] = max_k x[g*nsample + k][c], exact.                             */
/*  x    [G*nsample][C] (dt, row stride x_ld, 0: C), e.g. the shared MLP's   */
/*       output on the grouped rows (G = B*M centres)                        */
/*  out  [G][C] (out_dt, row stride out_ld, 0: C), e.g. a column slice of a  */
/*       feature-propagation input. NaN inputs: result unspecified.          */
pvconv_status pvconv_group_max(const void* x, pvconv_dtype dt, int x_ld, int G, int nsample,
                               int C, void* out, pvconv_dtype out_dt, int out_ld, void* stream);

/* Three nearest neighbours: for each unknown point the three known points   */
/* with the smallest squared distance, nearest first, and the weights        */
/* w_k = (1 / (d_k + 1e-8)) / sum_l (1 / (d_l + 1e-8)), d the Euclidean      */
/* distance, in fp32.                                                        */
/*  unknown [B][n][3], known [B][m][3] with m >= 3;                          */
/*  idx out [B][n][3] int32, weight out [B][n][3] fp32.                      */
pvconv_status pvconv_three_nn(const float* unknown, int B, int n, const float* known, int m,
                              int32_t* idx, float* weight, void* stream);

/* Inverse-distance interpolation: out[b][i][c] = sum_k weight[b][i][k] *    */
/* feats[b][idx[b][i][k]][c], fp32 sums.                                     */
/*  feats [B][m][C] (feat_dt, row stride feat_ld, 0: C); idx, weight as      */
/*  pvconv_three_nn writes them (indices clamped into [0, m));               */
/*  out [B][n][C] (out_dt, row stride out_ld, 0: C), e.g. a column slice of  */
/*  the feature-propagation input that also holds the skip features.         */
pvconv_status pvconv_three_interpolate(const void* feats, pvconv_dtype feat_dt, int feat_ld,
                                       int B, int m, int C, const int32_t* idx,
                                       const float* weight, int n, void* out,
                                       pvconv_dtype out_dt, int out_ld, void* stream);

/* Devoxelisation of a layer (Section 4.1 "Devoxelization"). */
typedef enum { PVCONV_DEVOX_TRILINEAR = 0, PVCONV_DEVOX_NEAREST = 1 } pvconv_devox;

/* ------------------------------------------------------------------------- */
/* One whole PVConv layer: Section 4, Figure "overview".                     */
/*                                                                           */
/* out = devoxelise( [conv + BN + leaky]^n_convs ( voxelise(coords, feats) ) ) */
/*       + ReLU( BN( W_mlp feats + b_mlp ) )                                 */
/* devoxelise is trilinear (pvconv_devoxelize) or, with devox =              */
/* PVCONV_DEVOX_NEAREST, nearest neighbour (pvconv_devoxelize_nearest). A     */
/* zero-initialised struct selects trilinear.                                */
/* All weights are in compute_dt (BF16 or F32); grids are kept in            */
/* compute_dt. out is [B][N][cout] (out_dt) with row stride out_ld; it must  */
/* not share any byte with feats (else PVCONV_EINVAL): in-place layers race. */
/* Disjoint column ranges of one wider array (equal row strides) are fine.  */
/* ------------------------------------------------------------------------- */
typedef struct {
    int cin, cout, R, n_convs;                 /* 1 <= n_convs <= PVCONV_MAX_CONVS */
    const void* conv_w[PVCONV_MAX_CONVS];      /* conv i: [cout][3][3][3][i ? cout : cin] */
    pvconv_bn conv_bn[PVCONV_MAX_CONVS];
    float conv_slope;                          /* leaky slope of the voxel branch */
    const void* mlp_w;                         /* [cout][cin] */
    const float* mlp_b;                        /* [cout] or NULL */
    pvconv_bn mlp_bn;
    pvconv_dtype compute_dt;
    pvconv_devox devox;
} pvconv_layer;

size_t pvconv_forward_workspace_size(int B, int N, const pvconv_layer* L);
pvconv_status pvconv_forward(const float* coords, const void* feats, pvconv_dtype feat_dt,
                             int feat_ld, int B, int N, const pvconv_layer* L, void* out,
                             pvconv_dtype out_dt, int out_ld, void* workspace,
                             size_t workspace_bytes, void* stream);

/* The same layer, sharing its normalisation with other layers of the same    */
/* points (Section 4.1 "Normalization" depends on the coordinates only, and  */
/* the voxel indices on the coordinates and R):                              */
/*  ids_given = 0: vox_id [B][N] int32 and norm_coords [B][N][3] fp32 are    */
/*    outputs (each may be NULL), as pvconv_voxelize writes them;            */
/*  ids_given = 1: both are inputs (non-NULL) from such a call with the same */
/*    coordinates and the same R; the normalisation is skipped and coords    */
/*    is not read (may be NULL). Indices that are not those of the given     */
/*    normalised coordinates leave the output unspecified (memory-safe): the */
/*    last convolution computes only the voxels near occupied ones.          */
/* pvconv_forward(...) is pvconv_forward_ex(..., NULL, NULL, 0, ...).         */
pvconv_status pvconv_forward_ex(const float* coords, const void* feats, pvconv_dtype feat_dt,
                                int feat_ld, int B, int N, const pvconv_layer* L,
                                int32_t* vox_id, float* norm_coords, int ids_given, void* out,
                                pvconv_dtype out_dt, int out_ld, void* workspace,
                                size_t workspace_bytes, void* stream);

/* ========================================================================= */
/* Backward pass: gradients of the steps above with respect to their inputs  */
/* (the layer is differentiable end to end). Each step is linear in the      */
/* input it is differentiated by, and each gradient is the adjoint of that   */
/* map. Gradients are fp32.                                                  */
/* ========================================================================= */

/* Voxelisation (Eq. 2, an average per voxel):                               */
/*  dfeats[b][k][c] = dgrid[b][vox_id[b][k]][c] / counts[b][vox_id[b][k]]    */
/*  dgrid [B][R^3][C] (dt), vox_id [B][N], counts [B][R^3] int32 as          */
/*  pvconv_voxelize wrote them; dfeats out [B][N][C] fp32. An index outside  */
/*  the grid or a count below 1 is invalid input (memory-safe, result        */
/*  unspecified).                                                            */
pvconv_status pvconv_voxelize_backward(const void* dgrid, pvconv_dtype dt, int B, int N, int C,
                                       int R, const int32_t* vox_id, const int32_t* counts,
                                       float* dfeats, void* stream);

/* Trilinear devoxelisation (Section 4.1 "Devoxelization"):                   */
/*  dgrid[b][cell][c] = sum over points k of w(k, cell) * dout[b][k][c], with */
/*  the 8 cells and weights of pvconv_devoxelize. dout [B][N][C] fp32,        */
/*  norm_coords [B][N][3]; dgrid out [B][R^3][C] fp32, every element written  */
/*  once. Computed as a gather: the points sorted stably by the cell of their */
/*  lower trilinear corner, each cell sums its points' weighted gradients in  */
/*  a fixed order (candidate cells in index order, their points in index      */
/*  order, fp32), so the result is the same bits on every run. workspace >=   */
/*  pvconv_devoxelize_backward_workspace_size(B, N, C, R) bytes, 256-byte     */
/*  aligned (may be NULL when N == 0), else PVCONV_EWORKSPACE.                */
size_t pvconv_devoxelize_backward_workspace_size(int B, int N, int C, int R);
pvconv_status pvconv_devoxelize_backward(const float* dout, int B, int N, int C, int R,
                                         const float* norm_coords, float* dgrid, void* workspace,
                                         size_t workspace_bytes, void* stream);

/* Nearest-neighbour devoxelisation: dgrid[b][cell] = sum of dout[b][k] over  */
/* the points k with vox_id[b][k] = cell, in point order (as above           */
/* otherwise; the same workspace). An index outside the grid is invalid      */
/* input (clamped: memory-safe, result unspecified).                         */
pvconv_status pvconv_devoxelize_nearest_backward(const float* dout, int B, int N, int C, int R,
                                                 const int32_t* vox_id, float* dgrid,
                                                 void* workspace, size_t workspace_bytes,
                                                 void* stream);

/* Convolution (Section 4.1 "Feature Aggregation"), gradient with respect to */
/* its input:                                                                */
/*  dx[b,q,i] = sum_{d in {-1,0,1}^3} sum_o W[o][d+1][i] * dy[b,q-d,o]       */
/* (dy = 0 outside the grid): the forward convolution of dy with the kernel  */
/* mirrored through its centre and its channel axes swapped, computed by the */
/* forward kernels. dy [B][R^3][Cout] (dt), weight [Cout][3][3][3][Cin] (dt), */
/* dx out [B][R^3][Cin] (dx_dt). dt = BF16 needs Cin % 32 == 0. workspace >= */
/* pvconv_conv3d_backward_data_workspace_size bytes, 256-byte aligned.        */
size_t pvconv_conv3d_backward_data_workspace_size(int Cin, int Cout, pvconv_dtype dt);
pvconv_status pvconv_conv3d_backward_data(const void* dy, int B, int R, int Cin, int Cout,
                                          const void* weight, pvconv_dtype dt, void* dx,
                                          pvconv_dtype dx_dt, void* workspace,
                                          size_t workspace_bytes, void* stream);

/* Convolution, gradient with respect to its weights:                       */
/*  dw[o][d+1][i] = sum_b sum_p dy[b,p,o] * x[b,p+d,i]  (x = 0 outside)       */
/* an MFMA implicit GEMM over the voxels, split over bricks of the grid; the */
/* splits' partial sums (in the workspace) are added in a fixed order, so    */
/* the result is deterministic. dy [B][R^3][Cout] and x [B][R^3][Cin] (the   */
/* convolution's input) in BF16, 16-byte aligned; dw out [Cout][3][3][3][Cin] */
/* fp32. Needs Cout % 64 == 0 and Cin % 16 == 0 (else PVCONV_ENOTSUP).       */
/* workspace >= pvconv_conv3d_backward_weight_workspace_size bytes, 256-byte */
/* aligned.                                                                  */
size_t pvconv_conv3d_backward_weight_workspace_size(int B, int R, int Cin, int Cout);
pvconv_status pvconv_conv3d_backward_weight(const void* dy, const void* x, pvconv_dtype dt,
                                            int B, int R, int Cin, int Cout, float* dw,
                                            void* workspace, size_t workspace_bytes,
                                            void* stream);

/* Batch norm + activation, y = act(BN(z)) per channel, gradient with respect */
/* to z: dz = dy * act'(y) * gamma / sqrt(var + eps), the rectifiers'        */
/* derivative read from the sign of y (1 where y > 0, else slope for LEAKY,   */
/* 0 for RELU; NONE: 1). bn NULL: identity. dy [M][C] fp32, y [M][C] (y_dt),  */
/* dz out [M][C] fp32 (may alias dy).                                        */
pvconv_status pvconv_act_bn_backward(const float* dy, const void* y, pvconv_dtype y_dt, int M,
                                     int C, const pvconv_bn* bn, pvconv_act act, float slope,
                                     float* dz, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* PVCONV_H */
