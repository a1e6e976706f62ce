// C ABI of libpvconv: argument validation on the host, then launches on the
// caller's stream. Nothing is enqueued when validation fails.
#include <mutex>

#include "pv_common.h"

// The workspace of pvconv_conv3d_noalloc: one copy per GPU in the library's
// device image, so that entry point allocates nothing. On the host this name
// is only a stand-in: host code takes the device address of the current
// GPU's copy from static_ws_on_device(), never from the name itself.
static __device__ __align__(256) unsigned char scratch[PVCONV_CONV3D_NOALLOC_BYTES];

namespace {

inline bool dtype_ok(pvconv_dtype d) { return d == PVCONV_F32 || d == PVCONV_BF16; }
inline size_t esize(pvconv_dtype d) { return d == PVCONV_BF16 ? 2 : 4; }
inline bool act_ok(pvconv_act a) {
    return a == PVCONV_ACT_NONE || a == PVCONV_ACT_RELU || a == PVCONV_ACT_LEAKY;
}
inline bool bn_ok(const pvconv_bn* bn) {
    if (!bn || !bn->gamma) return true;
    return bn->beta && bn->mean && bn->var && bn->eps >= 0.f;
}
inline hipStream_t as_stream(void* s) { return (hipStream_t)s; }

// Elements must fit the int32 voxel ids and list offsets the kernels use.
inline bool sizes_fit(long long B, long long N) { return B * N <= (1LL << 30); }

// Two row-major arrays of `rows` rows share at least one byte: array a has
// rows of ca elements of dtype ta at a stride of lda elements, b likewise.
// Column slices of one wider array (the same row pitch, disjoint column
// ranges, as the segmentation networks use them) do not overlap.
inline bool overlap(const void* a, long long rows, int ca, int lda, pvconv_dtype ta,
                    const void* b, int cb, int ldb, pvconv_dtype tb) {
    if (rows <= 0) return false;
    const long long pa = (long long)lda * esize(ta), pb = (long long)ldb * esize(tb);
    const long long wa = (long long)ca * esize(ta), wb = (long long)cb * esize(tb);
    const long long a0 = (long long)(uintptr_t)a, b0 = (long long)(uintptr_t)b;
    if (a0 + (rows - 1) * pa + wa <= b0 || b0 + (rows - 1) * pb + wb <= a0) return false;
    if (pa != pb) return true;
    // the same pitch: b's rows start e bytes into a's rows (or a's into b's)
    const long long e = ((b0 - a0) % pa + pa) % pa;
    return !(e >= wa && e + wb <= pa);
}

// Two byte ranges [a, a + na) and [b, b + nb) intersect.
inline bool bytes_overlap(const void* a, size_t na, const void* b, size_t nb) {
    const uintptr_t a0 = (uintptr_t)a, b0 = (uintptr_t)b;
    return na && nb && a0 < b0 + nb && b0 < a0 + na;
}

struct ForwardWs {
    void* conv_ws[PVCONV_MAX_CONVS];
    void* vox_ws;
    int32_t* counts;
    int32_t* ids;
    float* pnorm;
    void* grid_a;
    void* grid_b;
    float* devox;
    float* split;  // fp32 partial sums of split convolutions (small grids), or NULL
    size_t total;
};

ForwardWs carve_forward(void* base, int B, int N, const pvconv_layer* L) {
    const size_t V = (size_t)L->R * L->R * L->R;
    const size_t es = esize(L->compute_dt);
    const int cmax = L->cin > L->cout ? L->cin : L->cout;
    size_t off = 0;
    ForwardWs w;
    char* p = (char*)base;
    auto take = [&](size_t bytes) {
        void* q = p ? p + off : nullptr;
        off += pv_align256(bytes);
        return q;
    };
    for (int i = 0; i < PVCONV_MAX_CONVS; i++)
        w.conv_ws[i] = i < L->n_convs ? take(pv_conv3d_ws_bytes(i ? L->cout : L->cin, L->cout,
                                                                L->compute_dt == PVCONV_BF16))
                                      : nullptr;
    w.vox_ws = take(pv_voxelize_ws_bytes(B, N, L->R));
    w.counts = (int32_t*)take((size_t)B * V * 4);
    w.ids = (int32_t*)take((size_t)B * N * 4);
    w.pnorm = (float*)take((size_t)B * N * 12);
    w.grid_a = take((size_t)B * V * cmax * es);
    w.grid_b = take((size_t)B * V * L->cout * es);
    w.devox = (float*)take((size_t)B * N * L->cout * 4);
    size_t split = 0;
    if (L->compute_dt == PVCONV_BF16)
        for (int i = 0; i < L->n_convs; i++) {
            const size_t b = pv_conv3d_split_ws_bytes(B, L->R, i ? L->cout : L->cin, L->cout);
            split = b > split ? b : split;
        }
    w.split = split ? (float*)take(split) : nullptr;
    w.total = off;
    return w;
}

// Device address of `scratch` on the GPU that runs work on stream s (which
// must be the current device's), looked up with that device current on its
// first use and kept per device.
constexpr int kMaxDevices = 64;
std::mutex g_static_ws_mu;
void* g_static_ws[kMaxDevices];

pvconv_status static_ws_on_device(hipStream_t s, void** out) {
    int dev = -1;
    if (hipGetDevice(&dev) != hipSuccess) return PVCONV_EHIP;
    if (dev < 0 || dev >= kMaxDevices) return PVCONV_ENOTSUP;
    if (s) {
        hipDevice_t sd = -1;
        if (hipStreamGetDevice(s, &sd) != hipSuccess) return PVCONV_EHIP;
        if (sd != dev) return PVCONV_EINVAL;
    }
    std::lock_guard<std::mutex> lock(g_static_ws_mu);
    if (!g_static_ws[dev]) {
        void* p = nullptr;
        if (hipGetSymbolAddress(&p, HIP_SYMBOL(scratch)) != hipSuccess || !p) {
            (void)hipGetLastError();  // leave no error for the next launch check
            return PVCONV_EHIP;
        }
        g_static_ws[dev] = p;
    }
    *out = g_static_ws[dev];
    return PVCONV_OK;
}

// Everything pvconv_conv3d checks except the workspace (B == 0 passes).
pvconv_status check_conv3d(const void* x, int B, int R, int Cin, int Cout, const void* weight,
                           const float* bias, const pvconv_bn* bn, pvconv_act act,
                           pvconv_dtype dt, const void* y, pvconv_dtype out_dt) {
    if (B < 0 || R < 1 || R > PVCONV_MAX_R || Cin < 1 || Cout < 1 ||
        Cin > PVCONV_MAX_CONV_CHANNELS || Cout > PVCONV_MAX_CONV_CHANNELS)
        return PVCONV_EINVAL;
    if (!dtype_ok(dt) || !dtype_ok(out_dt) || !act_ok(act) || !bn_ok(bn)) return PVCONV_EINVAL;
    if (B == 0) return PVCONV_OK;
    if (!x || !weight || !y) return PVCONV_EINVAL;
    if (((uintptr_t)x & (esize(dt) - 1)) || ((uintptr_t)weight & (esize(dt) - 1)) ||
        ((uintptr_t)y & (esize(out_dt) - 1)) || ((uintptr_t)bias & 3))
        return PVCONV_EINVAL;
    // every input voxel is read by up to 27 workgroups while others store
    if (overlap(x, (long long)B * R * R * R, Cin, Cin, dt, y, Cout, Cout, out_dt))
        return PVCONV_EINVAL;
    return PVCONV_OK;
}

pvconv_status check_layer(const pvconv_layer* L) {
    if (!L) return PVCONV_EINVAL;
    if (L->cin < 1 || L->cout < 1 || L->cin > PVCONV_MAX_CONV_CHANNELS ||
        L->cout > PVCONV_MAX_CONV_CHANNELS || L->R < 1 || L->R > PVCONV_MAX_R ||
        L->n_convs < 1 || L->n_convs > PVCONV_MAX_CONVS)
        return PVCONV_EINVAL;
    if (!dtype_ok(L->compute_dt)) return PVCONV_EINVAL;
    for (int i = 0; i < L->n_convs; i++)
        if (!L->conv_w[i] || !bn_ok(&L->conv_bn[i])) return PVCONV_EINVAL;
    if (!L->mlp_w || !bn_ok(&L->mlp_bn)) return PVCONV_EINVAL;
    if (L->devox != PVCONV_DEVOX_TRILINEAR && L->devox != PVCONV_DEVOX_NEAREST)
        return PVCONV_EINVAL;
    return PVCONV_OK;
}

}  // namespace

extern "C" {

const char* pvconv_status_string(pvconv_status s) {
    switch (s) {
        case PVCONV_OK: return "ok";
        case PVCONV_EINVAL: return "invalid argument";
        case PVCONV_ENOTSUP: return "unsupported argument combination";
        case PVCONV_EWORKSPACE: return "workspace missing or too small";
        case PVCONV_EHIP: return "HIP launch error";
    }
    return "unknown status";
}

size_t pvconv_voxelize_workspace_size(int B, int N, int R) {
    if (B < 0 || N < 0 || R < 1 || R > PVCONV_MAX_R) return 0;
    return pv_voxelize_ws_bytes(B, N, R);
}

pvconv_status pvconv_voxelize(const float* coords, const void* feats, pvconv_dtype feat_dt,
                              int feat_ld, int B, int N, int C, int R, void* grid,
                              pvconv_dtype grid_dt, int32_t* counts, int32_t* vox_id,
                              float* norm_coords, void* workspace, size_t workspace_bytes,
                              void* stream) {
    if (B < 0 || N < 0 || C < 1 || R < 1 || R > PVCONV_MAX_R || !sizes_fit(B, N))
        return PVCONV_EINVAL;
    if (!dtype_ok(feat_dt) || !dtype_ok(grid_dt)) return PVCONV_EINVAL;
    if (feat_ld == 0) feat_ld = C;
    if (feat_ld < C) return PVCONV_EINVAL;
    if (B == 0) return PVCONV_OK;
    if (!grid || !counts || (N > 0 && (!coords || !feats))) return PVCONV_EINVAL;
    if (((uintptr_t)coords & 3) || ((uintptr_t)counts & 3) || ((uintptr_t)vox_id & 3) ||
        ((uintptr_t)norm_coords & 3) || ((uintptr_t)feats & (esize(feat_dt) - 1)) ||
        ((uintptr_t)grid & (esize(grid_dt) - 1)))
        return PVCONV_EINVAL;
    if (!workspace || ((uintptr_t)workspace & 255) ||
        workspace_bytes < pv_voxelize_ws_bytes(B, N, R))
        return PVCONV_EWORKSPACE;
    return pv_launch_voxelize(coords, feats, feat_dt == PVCONV_BF16, feat_ld, B, N, C, R, grid,
                              grid_dt == PVCONV_BF16, counts, vox_id, norm_coords, workspace,
                              as_stream(stream));
}

pvconv_status pvconv_voxelize_from_ids(const int32_t* vox_id, const void* feats,
                                       pvconv_dtype feat_dt, int feat_ld, int B, int N, int C,
                                       int R, void* grid, pvconv_dtype grid_dt, int32_t* counts,
                                       void* workspace, size_t workspace_bytes, void* stream) {
    if (B < 0 || N < 0 || C < 1 || R < 1 || R > PVCONV_MAX_R || !sizes_fit(B, N))
        return PVCONV_EINVAL;
    if (!dtype_ok(feat_dt) || !dtype_ok(grid_dt)) return PVCONV_EINVAL;
    if (feat_ld == 0) feat_ld = C;
    if (feat_ld < C) return PVCONV_EINVAL;
    if (B == 0) return PVCONV_OK;
    if (!grid || !counts || (N > 0 && (!vox_id || !feats))) return PVCONV_EINVAL;
    if (((uintptr_t)vox_id & 3) || ((uintptr_t)counts & 3) ||
        ((uintptr_t)feats & (esize(feat_dt) - 1)) || ((uintptr_t)grid & (esize(grid_dt) - 1)))
        return PVCONV_EINVAL;
    if (!workspace || ((uintptr_t)workspace & 255) ||
        workspace_bytes < pv_voxelize_ws_bytes(B, N, R))
        return PVCONV_EWORKSPACE;
    return pv_launch_voxelize_from_ids(vox_id, feats, feat_dt == PVCONV_BF16, feat_ld, B, N, C,
                                       R, grid, grid_dt == PVCONV_BF16, counts, workspace,
                                       as_stream(stream));
}

size_t pvconv_conv3d_workspace_size(int Cin, int Cout, pvconv_dtype dt) {
    if (Cin < 1 || Cout < 1 || Cin > PVCONV_MAX_CONV_CHANNELS || Cout > PVCONV_MAX_CONV_CHANNELS ||
        !dtype_ok(dt))
        return 0;
    return pv_conv3d_ws_bytes(Cin, Cout, dt == PVCONV_BF16);
}

pvconv_status pvconv_conv3d(const void* x, int B, int R, int Cin, int Cout, const void* weight,
                            const float* bias, const pvconv_bn* bn, pvconv_act act, float slope,
                            pvconv_dtype dt, void* y, pvconv_dtype out_dt, void* workspace,
                            size_t workspace_bytes, void* stream) {
    const pvconv_status st =
        check_conv3d(x, B, R, Cin, Cout, weight, bias, bn, act, dt, y, out_dt);
    if (st != PVCONV_OK || B == 0) return st;
    const size_t need = pv_conv3d_ws_bytes(Cin, Cout, dt == PVCONV_BF16);
    if (need && (!workspace || ((uintptr_t)workspace & 255) || workspace_bytes < need))
        return PVCONV_EWORKSPACE;
    return pv_launch_conv3d(x, B, R, Cin, Cout, weight, pv_make_fold(bn, bias), act, slope,
                            dt == PVCONV_BF16, y, out_dt == PVCONV_BF16, workspace,
                            as_stream(stream));
}

pvconv_status pvconv_conv3d_pack_weights(const void* weight, int Cin, int Cout, void* packed,
                                         size_t packed_bytes, void* stream) {
    if (Cin < 1 || Cout < 1 || Cin > PVCONV_MAX_CONV_CHANNELS || Cout > PVCONV_MAX_CONV_CHANNELS)
        return PVCONV_EINVAL;
    if (!weight || ((uintptr_t)weight & 1)) return PVCONV_EINVAL;
    const size_t need = pv_conv3d_ws_bytes(Cin, Cout, true);
    if (!packed || ((uintptr_t)packed & 255) || packed_bytes < need) return PVCONV_EWORKSPACE;
    if (bytes_overlap(weight, (size_t)Cout * 27 * Cin * 2, packed, need)) return PVCONV_EINVAL;
    PvPackJobs jobs{};
    pv_pack_job(jobs, weight, Cin, Cout, packed);
    pv_launch_pack_conv_weights(jobs, as_stream(stream));
    return pv_launch_status();
}

pvconv_status pvconv_conv3d_packed(const void* x, int B, int R, int Cin, int Cout,
                                   const void* packed, size_t packed_bytes, const float* bias,
                                   const pvconv_bn* bn, pvconv_act act, float slope, void* y,
                                   pvconv_dtype out_dt, void* stream) {
    // the packed copy stands in for the weights in the common checks
    const pvconv_status st = check_conv3d(x, B, R, Cin, Cout, packed, bias, bn, act,
                                          PVCONV_BF16, y, out_dt);
    if (st != PVCONV_OK || B == 0) return st;
    const size_t need = pv_conv3d_ws_bytes(Cin, Cout, true);
    if (((uintptr_t)packed & 255) || packed_bytes < need) return PVCONV_EWORKSPACE;
    if (bytes_overlap(y, (size_t)B * R * R * R * Cout * esize(out_dt), packed, need))
        return PVCONV_EINVAL;
    return pv_launch_conv3d(x, B, R, Cin, Cout, nullptr, pv_make_fold(bn, bias), act, slope,
                            true, y, out_dt == PVCONV_BF16, const_cast<void*>(packed),
                            as_stream(stream), /*packed=*/true);
}

pvconv_status pvconv_conv3d_noalloc(const void* x, int B, int R, int Cin, int Cout,
                                    const void* weight, const float* bias, const pvconv_bn* bn,
                                    pvconv_act act, float slope, pvconv_dtype dt, void* y,
                                    pvconv_dtype out_dt, void* stream) {
    pvconv_status st = check_conv3d(x, B, R, Cin, Cout, weight, bias, bn, act, dt, y, out_dt);
    if (st != PVCONV_OK || B == 0) return st;
    const size_t need = pv_conv3d_ws_bytes(Cin, Cout, dt == PVCONV_BF16);
    if (need > PVCONV_CONV3D_NOALLOC_BYTES) return PVCONV_EWORKSPACE;
    hipStream_t s = as_stream(stream);
    void* ws = nullptr;
    if (need && (st = static_ws_on_device(s, &ws)) != PVCONV_OK) return st;
    // the packing launch rewrites all `need` bytes of the array, so nothing
    // from an earlier call is read
    return pv_launch_conv3d(x, B, R, Cin, Cout, weight, pv_make_fold(bn, bias), act, slope,
                            dt == PVCONV_BF16, y, out_dt == PVCONV_BF16, ws, s);
}

pvconv_status pvconv_devoxelize(const void* grid, int B, int R, int C, pvconv_dtype grid_dt,
                                const float* norm_coords, int N, float* out, void* stream) {
    if (B < 0 || N < 0 || R < 1 || R > PVCONV_MAX_R || C < 1 || !sizes_fit(B, N))
        return PVCONV_EINVAL;
    if (!dtype_ok(grid_dt)) return PVCONV_EINVAL;
    if (B == 0 || N == 0) return PVCONV_OK;
    if (!grid || !norm_coords || !out) return PVCONV_EINVAL;
    if (((uintptr_t)grid & (esize(grid_dt) - 1)) || ((uintptr_t)norm_coords & 3) ||
        ((uintptr_t)out & 3))
        return PVCONV_EINVAL;
    return pv_launch_devoxelize(grid, B, R, C, grid_dt == PVCONV_BF16, norm_coords, N, out,
                                as_stream(stream));
}

pvconv_status pvconv_devoxelize_nearest(const void* grid, int B, int R, int C,
                                        pvconv_dtype grid_dt, const int32_t* vox_id, int N,
                                        float* out, void* stream) {
    if (B < 0 || N < 0 || R < 1 || R > PVCONV_MAX_R || C < 1 || !sizes_fit(B, N))
        return PVCONV_EINVAL;
    if (!dtype_ok(grid_dt)) return PVCONV_EINVAL;
    if (B == 0 || N == 0) return PVCONV_OK;
    if (!grid || !vox_id || !out) return PVCONV_EINVAL;
    if (((uintptr_t)grid & (esize(grid_dt) - 1)) || ((uintptr_t)vox_id & 3) ||
        ((uintptr_t)out & 3))
        return PVCONV_EINVAL;
    return pv_launch_devoxelize_nearest(grid, B, R, C, grid_dt == PVCONV_BF16, vox_id, N, out,
                                        as_stream(stream));
}

pvconv_status pvconv_point_mlp(const void* x, pvconv_dtype x_dt, int x_ld, int M, int Cin,
                               int Cout, const void* weight, pvconv_dtype compute_dt,
                               const float* bias, const pvconv_bn* bn, pvconv_act act,
                               float slope, const float* cloud_bias, int points_per_cloud,
                               const float* residual, int residual_ld, void* out,
                               pvconv_dtype out_dt, int out_ld, void* stream) {
    if (M < 0 || Cin < 1 || Cout < 1 || Cin > PVCONV_MAX_MLP_CHANNELS ||
        Cout > PVCONV_MAX_MLP_CHANNELS || M > (1 << 30))
        return PVCONV_EINVAL;
    if (!dtype_ok(x_dt) || !dtype_ok(compute_dt) || !dtype_ok(out_dt) || !act_ok(act) ||
        !bn_ok(bn))
        return PVCONV_EINVAL;
    if (x_ld == 0) x_ld = Cin;
    if (out_ld == 0) out_ld = Cout;
    if (residual_ld == 0) residual_ld = Cout;
    if (x_ld < Cin || out_ld < Cout || residual_ld < Cout) return PVCONV_EINVAL;
    if (cloud_bias && points_per_cloud < 1) return PVCONV_EINVAL;
    if (M == 0) return PVCONV_OK;
    if (!x || !weight || !out) return PVCONV_EINVAL;
    if (((uintptr_t)x & (esize(x_dt) - 1)) || ((uintptr_t)weight & (esize(compute_dt) - 1)) ||
        ((uintptr_t)out & (esize(out_dt) - 1)) || ((uintptr_t)bias & 3) ||
        ((uintptr_t)cloud_bias & 3) || ((uintptr_t)residual & 3))
        return PVCONV_EINVAL;
    // an output row can be stored before another workgroup has read the
    // input row it overlaps
    if (overlap(x, M, Cin, x_ld, x_dt, out, Cout, out_ld, out_dt)) return PVCONV_EINVAL;
    return pv_launch_point_mlp(x, x_dt == PVCONV_BF16, x_ld, M, Cin, Cout, weight,
                               compute_dt == PVCONV_BF16, pv_make_fold(bn, bias), act, slope,
                               cloud_bias, cloud_bias ? points_per_cloud : 1, residual,
                               residual_ld, out, out_dt == PVCONV_BF16, out_ld,
                               as_stream(stream));
}

pvconv_status pvconv_devoxelize_point_mlp(const void* grid, int R, const float* norm_coords,
                                          int B, int N, const void* x, pvconv_dtype x_dt,
                                          int x_ld, int Cin, int Cout, const void* weight,
                                          const float* bias, const pvconv_bn* bn,
                                          pvconv_act act, float slope, void* out,
                                          pvconv_dtype out_dt, int out_ld, void* stream) {
    if (B < 0 || N < 0 || !sizes_fit(B, N) || R < 1 || R > PVCONV_MAX_R || Cin < 1 ||
        Cout < 1 || Cin > PVCONV_MAX_MLP_CHANNELS || Cout > PVCONV_MAX_MLP_CHANNELS)
        return PVCONV_EINVAL;
    if (!dtype_ok(x_dt) || !dtype_ok(out_dt) || !act_ok(act) || !bn_ok(bn)) return PVCONV_EINVAL;
    if (x_ld == 0) x_ld = Cin;
    if (out_ld == 0) out_ld = Cout;
    if (x_ld < Cin || out_ld < Cout) return PVCONV_EINVAL;
    if (B == 0 || N == 0) return PVCONV_OK;
    if (!grid || !norm_coords || !x || !weight || !out) return PVCONV_EINVAL;
    if (((uintptr_t)grid & 1) || ((uintptr_t)norm_coords & 3) ||
        ((uintptr_t)x & (esize(x_dt) - 1)) || ((uintptr_t)weight & 1) ||
        ((uintptr_t)out & (esize(out_dt) - 1)) || ((uintptr_t)bias & 3))
        return PVCONV_EINVAL;
    const long long M = (long long)B * N;
    const size_t out_bytes = (size_t)((M - 1) * out_ld + Cout) * esize(out_dt);
    if (overlap(x, M, Cin, x_ld, x_dt, out, Cout, out_ld, out_dt) ||
        bytes_overlap(out, out_bytes, grid, (size_t)B * R * R * R * Cout * 2) ||
        bytes_overlap(out, out_bytes, norm_coords, (size_t)M * 12))
        return PVCONV_EINVAL;
    return pv_launch_devox_point_mlp(PvDevoxIn{(const uint16_t*)grid, norm_coords, N, R}, x,
                                     x_dt == PVCONV_BF16, x_ld, (int)M, Cin, Cout, weight,
                                     pv_make_fold(bn, bias), act, slope, out,
                                     out_dt == PVCONV_BF16, out_ld, as_stream(stream));
}

pvconv_status pvconv_maxpool(const void* x, pvconv_dtype dt, int x_ld, int B, int N, int C,
                             float* out, void* stream) {
    if (B < 0 || N < 1 || C < 1 || !dtype_ok(dt) || !sizes_fit(B, N)) return PVCONV_EINVAL;
    if (x_ld == 0) x_ld = C;
    if (x_ld < C) return PVCONV_EINVAL;
    if (B == 0) return PVCONV_OK;
    if (!x || !out || ((uintptr_t)x & (esize(dt) - 1)) || ((uintptr_t)out & 3))
        return PVCONV_EINVAL;
    return pv_launch_maxpool(x, dt == PVCONV_BF16, x_ld, B, N, C, out, as_stream(stream));
}

pvconv_status pvconv_furthest_point_sample(const float* xyz, int B, int N, int npoint,
                                           int32_t* idx, float* new_xyz, void* stream) {
    if (B < 0 || N < 1 || npoint < 1 || npoint > N || !sizes_fit(B, N)) return PVCONV_EINVAL;
    if (B == 0) return PVCONV_OK;
    if (!xyz || !idx || ((uintptr_t)xyz & 3) || ((uintptr_t)idx & 3) || ((uintptr_t)new_xyz & 3))
        return PVCONV_EINVAL;
    if (N > kPvFpsMaxN) return PVCONV_ENOTSUP;
    if (bytes_overlap(idx, (size_t)B * npoint * 4, xyz, (size_t)B * N * 12) ||
        (new_xyz && (bytes_overlap(new_xyz, (size_t)B * npoint * 12, xyz, (size_t)B * N * 12) ||
                     bytes_overlap(new_xyz, (size_t)B * npoint * 12, idx, (size_t)B * npoint * 4))))
        return PVCONV_EINVAL;
    return pv_launch_fps(xyz, B, N, npoint, idx, new_xyz, as_stream(stream));
}

pvconv_status pvconv_ball_query(const float* xyz, int B, int N, const float* centers, int M,
                                float radius, int nsample, int32_t* idx, void* stream) {
    if (B < 0 || N < 1 || M < 0 || nsample < 1 || !(radius >= 0.f) || !sizes_fit(B, N) ||
        !sizes_fit(B, M) || (long long)B * M * nsample > (1LL << 30))
        return PVCONV_EINVAL;
    if (B == 0 || M == 0) return PVCONV_OK;
    if (!xyz || !centers || !idx || ((uintptr_t)xyz & 3) || ((uintptr_t)centers & 3) ||
        ((uintptr_t)idx & 3))
        return PVCONV_EINVAL;
    const size_t ib = (size_t)B * M * nsample * 4;
    if (bytes_overlap(idx, ib, xyz, (size_t)B * N * 12) ||
        bytes_overlap(idx, ib, centers, (size_t)B * M * 12))
        return PVCONV_EINVAL;
    return pv_launch_ball_query(xyz, B, N, centers, M, radius, nsample, idx, as_stream(stream));
}

pvconv_status pvconv_group_points(const float* xyz, const void* feats, pvconv_dtype feat_dt,
                                  int feat_ld, int B, int N, int C, const float* centers, int M,
                                  const int32_t* idx, int nsample, void* out,
                                  pvconv_dtype out_dt, int out_ld, void* stream) {
    if (B < 0 || N < 1 || C < 0 || C > PVCONV_MAX_MLP_CHANNELS - 3 || M < 0 || nsample < 1 ||
        !sizes_fit(B, N) || (long long)B * M * nsample > (1LL << 30))
        return PVCONV_EINVAL;
    if (!dtype_ok(feat_dt) || !dtype_ok(out_dt)) return PVCONV_EINVAL;
    if (feat_ld == 0) feat_ld = C;
    if (out_ld == 0) out_ld = 3 + C;
    if (feat_ld < C || out_ld < 3 + C) return PVCONV_EINVAL;
    if (B == 0 || M == 0) return PVCONV_OK;
    if (!xyz || !centers || !idx || !out || (C > 0 && !feats)) return PVCONV_EINVAL;
    if (((uintptr_t)xyz & 3) || ((uintptr_t)centers & 3) || ((uintptr_t)idx & 3) ||
        ((uintptr_t)feats & (esize(feat_dt) - 1)) || ((uintptr_t)out & (esize(out_dt) - 1)))
        return PVCONV_EINVAL;
    const long long rows = (long long)B * M * nsample;
    const size_t ob = (size_t)((rows - 1) * out_ld + 3 + C) * esize(out_dt);
    if (bytes_overlap(out, ob, xyz, (size_t)B * N * 12) ||
        bytes_overlap(out, ob, centers, (size_t)B * M * 12) ||
        bytes_overlap(out, ob, idx, (size_t)rows * 4) ||
        (C > 0 && bytes_overlap(out, ob, feats,
                                (size_t)(((long long)B * N - 1) * feat_ld + C) * esize(feat_dt))))
        return PVCONV_EINVAL;
    return pv_launch_group(xyz, feats, feat_dt == PVCONV_BF16, feat_ld, B, N, C, centers, M, idx,
                           nsample, out, out_dt == PVCONV_BF16, out_ld, as_stream(stream));
}

pvconv_status pvconv_group_max(const void* x, pvconv_dtype dt, int x_ld, int G, int nsample,
                               int C, void* out, pvconv_dtype out_dt, int out_ld, void* stream) {
    if (G < 0 || nsample < 1 || C < 1 || C > PVCONV_MAX_MLP_CHANNELS ||
        (long long)G * nsample > (1LL << 30))
        return PVCONV_EINVAL;
    if (!dtype_ok(dt) || !dtype_ok(out_dt)) return PVCONV_EINVAL;
    if (x_ld == 0) x_ld = C;
    if (out_ld == 0) out_ld = C;
    if (x_ld < C || out_ld < C) return PVCONV_EINVAL;
    if (G == 0) return PVCONV_OK;
    if (!x || !out || ((uintptr_t)x & (esize(dt) - 1)) || ((uintptr_t)out & (esize(out_dt) - 1)))
        return PVCONV_EINVAL;
    if (bytes_overlap(out, (size_t)(((long long)G - 1) * out_ld + C) * esize(out_dt), x,
                      (size_t)(((long long)G * nsample - 1) * x_ld + C) * esize(dt)))
        return PVCONV_EINVAL;
    return pv_launch_group_max(x, dt == PVCONV_BF16, x_ld, G, nsample, C, out,
                               out_dt == PVCONV_BF16, out_ld, as_stream(stream));
}

pvconv_status pvconv_three_nn(const float* unknown, int B, int n, const float* known, int m,
                              int32_t* idx, float* weight, void* stream) {
    if (B < 0 || n < 0 || m < 3 || !sizes_fit(B, n) || !sizes_fit(B, m)) return PVCONV_EINVAL;
    if (B == 0 || n == 0) return PVCONV_OK;
    if (!unknown || !known || !idx || !weight || ((uintptr_t)unknown & 3) ||
        ((uintptr_t)known & 3) || ((uintptr_t)idx & 3) || ((uintptr_t)weight & 3))
        return PVCONV_EINVAL;
    const size_t ob = (size_t)B * n * 12;
    if (bytes_overlap(idx, ob, weight, ob) || bytes_overlap(idx, ob, unknown, ob) ||
        bytes_overlap(weight, ob, unknown, ob) ||
        bytes_overlap(idx, ob, known, (size_t)B * m * 12) ||
        bytes_overlap(weight, ob, known, (size_t)B * m * 12))
        return PVCONV_EINVAL;
    return pv_launch_three_nn(unknown, B, n, known, m, idx, weight, as_stream(stream));
}

pvconv_status pvconv_three_interpolate(const void* feats, pvconv_dtype feat_dt, int feat_ld,
                                       int B, int m, int C, const int32_t* idx,
                                       const float* weight, int n, void* out,
                                       pvconv_dtype out_dt, int out_ld, void* stream) {
    if (B < 0 || m < 1 || C < 1 || n < 0 || C > PVCONV_MAX_MLP_CHANNELS || !sizes_fit(B, n) ||
        !sizes_fit(B, m))
        return PVCONV_EINVAL;
    if (!dtype_ok(feat_dt) || !dtype_ok(out_dt)) return PVCONV_EINVAL;
    if (feat_ld == 0) feat_ld = C;
    if (out_ld == 0) out_ld = C;
    if (feat_ld < C || out_ld < C) return PVCONV_EINVAL;
    if (B == 0 || n == 0) return PVCONV_OK;
    if (!feats || !idx || !weight || !out || ((uintptr_t)feats & (esize(feat_dt) - 1)) ||
        ((uintptr_t)idx & 3) || ((uintptr_t)weight & 3) || ((uintptr_t)out & (esize(out_dt) - 1)))
        return PVCONV_EINVAL;
    const long long rows = (long long)B * n;
    const size_t ob = (size_t)((rows - 1) * out_ld + C) * esize(out_dt);
    if (bytes_overlap(out, ob, feats,
                      (size_t)(((long long)B * m - 1) * feat_ld + C) * esize(feat_dt)) ||
        bytes_overlap(out, ob, idx, (size_t)rows * 12) ||
        bytes_overlap(out, ob, weight, (size_t)rows * 12))
        return PVCONV_EINVAL;
    return pv_launch_three_interpolate(feats, feat_dt == PVCONV_BF16, feat_ld, B, m, C, idx,
                                       weight, n, out, out_dt == PVCONV_BF16, out_ld,
                                       as_stream(stream));
}

size_t pvconv_forward_workspace_size(int B, int N, const pvconv_layer* L) {
    if (B < 0 || N < 0 || check_layer(L) != PVCONV_OK) return 0;
    return carve_forward(nullptr, B, N, L).total;
}

pvconv_status pvconv_forward(const float* coords, const void* feats, pvconv_dtype feat_dt,
                             int feat_ld, int B, int N, const pvconv_layer* L, void* out,
                             pvconv_dtype out_dt, int out_ld, void* workspace,
                             size_t workspace_bytes, void* stream) {
    return pvconv_forward_ex(coords, feats, feat_dt, feat_ld, B, N, L, nullptr, nullptr, 0, out,
                             out_dt, out_ld, workspace, workspace_bytes, stream);
}

pvconv_status pvconv_forward_ex(const float* coords, const void* feats, pvconv_dtype feat_dt,
                                int feat_ld, int B, int N, const pvconv_layer* L,
                                int32_t* vox_id, float* norm_coords, int ids_given, void* out,
                                pvconv_dtype out_dt, int out_ld, void* workspace,
                                size_t workspace_bytes, void* stream) {
    pvconv_status st = check_layer(L);
    if (st != PVCONV_OK) return st;
    if (B < 0 || N < 0 || !sizes_fit(B, N) || !dtype_ok(feat_dt) || !dtype_ok(out_dt))
        return PVCONV_EINVAL;
    if (feat_ld == 0) feat_ld = L->cin;
    if (out_ld == 0) out_ld = L->cout;
    if (feat_ld < L->cin || out_ld < L->cout) return PVCONV_EINVAL;
    if (ids_given != 0 && ids_given != 1) return PVCONV_EINVAL;
    if (B == 0 || N == 0) return PVCONV_OK;
    if ((!ids_given && !coords) || (ids_given && (!vox_id || !norm_coords)) || !feats || !out)
        return PVCONV_EINVAL;
    if (((uintptr_t)coords & 3) || ((uintptr_t)feats & (esize(feat_dt) - 1)) ||
        ((uintptr_t)out & (esize(out_dt) - 1)) || ((uintptr_t)vox_id & 3) ||
        ((uintptr_t)norm_coords & 3))
        return PVCONV_EINVAL;
    // several workgroups read each feature row while others store output
    // rows: the two must not share memory
    if (overlap(feats, (long long)B * N, L->cin, feat_ld, feat_dt, out, L->cout, out_ld, out_dt))
        return PVCONV_EINVAL;
    const size_t need = carve_forward(nullptr, B, N, L).total;
    if (!workspace || ((uintptr_t)workspace & 255) || workspace_bytes < need)
        return PVCONV_EWORKSPACE;
    ForwardWs w = carve_forward(workspace, B, N, L);
    hipStream_t s = as_stream(stream);
    const bool bf = L->compute_dt == PVCONV_BF16;
    const int R = L->R;

    int32_t* ids = vox_id ? vox_id : w.ids;
    const float* pnorm = norm_coords ? norm_coords : w.pnorm;
    // bf16: the weights of all the convolutions repacked by extra workgroups
    // of the normalisation launch (or in a launch of their own when the
    // normalisation is skipped)
    PvPackJobs jobs{};
    if (bf)
        for (int i = 0; i < L->n_convs; i++)
            pv_pack_job(jobs, L->conv_w[i], i ? L->cout : L->cin, L->cout, w.conv_ws[i]);
    // bf16 small clouds: the grid holds only its occupied rows (most voxels
    // are empty: their rows are neither written nor read); the first
    // convolution reads the counts and takes empty voxels as zero
    const bool sparse = bf && pv_voxelize_sparse_ok(N);
    if (ids_given) {
        pv_launch_pack_conv_weights(jobs, s);
        st = pv_launch_voxelize_from_ids(ids, feats, feat_dt == PVCONV_BF16, feat_ld, B, N,
                                         L->cin, R, w.grid_a, bf, w.counts, w.vox_ws, s, sparse);
    } else {
        st = pv_launch_voxelize(coords, feats, feat_dt == PVCONV_BF16, feat_ld, B, N, L->cin, R,
                                w.grid_a, bf, w.counts, ids,
                                norm_coords ? norm_coords : w.pnorm, w.vox_ws, s, &jobs, sparse);
    }
    if (st != PVCONV_OK) return st;
    void* src = w.grid_a;
    void* dst = w.grid_b;
    int cin = L->cin;
    // The last convolution's grid is read only by the devoxelisation, at
    // its points' corners (trilinear) or voxels (nearest), all within one
    // voxel of an occupied voxel: only those outputs are computed.
    for (int i = 0; i < L->n_convs; i++) {
        const bool last = i == L->n_convs - 1;
        st = pv_launch_conv3d(src, B, R, cin, L->cout, L->conv_w[i],
                              pv_make_fold(&L->conv_bn[i], nullptr), PVCONV_ACT_LEAKY,
                              L->conv_slope, bf, dst, bf, w.conv_ws[i], s, /*packed=*/bf,
                              w.split, i == 0 && sparse ? w.counts : nullptr,
                              last && bf && (i > 0 || sparse) ? w.counts : nullptr);
        if (st != PVCONV_OK) return st;
        void* t = src;
        src = dst;
        dst = t;
        cin = L->cout;
    }
    // bf16 trilinear: the devoxelisation runs inside the point-MLP kernel
    if (bf && L->devox == PVCONV_DEVOX_TRILINEAR) {
        st = pv_launch_devox_point_mlp(PvDevoxIn{(const uint16_t*)src, pnorm, N, R}, feats,
                                       feat_dt == PVCONV_BF16, feat_ld, B * N, L->cin, L->cout,
                                       L->mlp_w, pv_make_fold(&L->mlp_bn, L->mlp_b),
                                       PVCONV_ACT_RELU, 0.f, out, out_dt == PVCONV_BF16, out_ld,
                                       s);
        if (st != PVCONV_ENOTSUP) return st;
    }
    st = L->devox == PVCONV_DEVOX_NEAREST
             ? pv_launch_devoxelize_nearest(src, B, R, L->cout, bf, ids, N, w.devox, s)
             : pv_launch_devoxelize(src, B, R, L->cout, bf, pnorm, N, w.devox, s);
    if (st != PVCONV_OK) return st;
    return pv_launch_point_mlp(feats, feat_dt == PVCONV_BF16, feat_ld, B * N, L->cin, L->cout,
                               L->mlp_w, bf, pv_make_fold(&L->mlp_bn, L->mlp_b), PVCONV_ACT_RELU,
                               0.f, nullptr, 1, w.devox, L->cout, out, out_dt == PVCONV_BF16,
                               out_ld, s);
}

pvconv_status pvconv_voxelize_backward(const void* dgrid, pvconv_dtype dt, int B, int N, int C,
                                       int R, const int32_t* vox_id, const int32_t* counts,
                                       float* dfeats, void* stream) {
    if (B < 0 || N < 0 || C < 1 || R < 1 || R > PVCONV_MAX_R || !sizes_fit(B, N) ||
        !dtype_ok(dt))
        return PVCONV_EINVAL;
    if (B == 0 || N == 0) return PVCONV_OK;
    if (!dgrid || !vox_id || !counts || !dfeats) return PVCONV_EINVAL;
    if (((uintptr_t)dgrid & (esize(dt) - 1)) || ((uintptr_t)vox_id & 3) ||
        ((uintptr_t)counts & 3) || ((uintptr_t)dfeats & 3))
        return PVCONV_EINVAL;
    return pv_launch_voxelize_backward(dgrid, dt == PVCONV_BF16, B, N, C, R, vox_id, counts,
                                       dfeats, as_stream(stream));
}

size_t pvconv_devoxelize_backward_workspace_size(int B, int N, int C, int R) {
    if (B < 0 || N < 0 || C < 1 || R < 1 || R > PVCONV_MAX_R || !sizes_fit(B, N)) return 0;
    return pv_devox_bwd_ws_bytes(B, N, C, R);
}

static pvconv_status devox_backward(const float* dout, int B, int N, int C, int R,
                                    const float* pn, const int32_t* ids, float* dgrid,
                                    void* workspace, size_t workspace_bytes, void* stream) {
    if (B < 0 || N < 0 || C < 1 || R < 1 || R > PVCONV_MAX_R || !sizes_fit(B, N))
        return PVCONV_EINVAL;
    if (B == 0) return PVCONV_OK;
    if (!dgrid || (N > 0 && (!dout || (!pn && !ids)))) return PVCONV_EINVAL;
    if (((uintptr_t)dout & 3) || ((uintptr_t)pn & 3) || ((uintptr_t)ids & 3) ||
        ((uintptr_t)dgrid & 3))
        return PVCONV_EINVAL;
    if (N > 0 && (!workspace || ((uintptr_t)workspace & 255) ||
                  workspace_bytes < pv_devox_bwd_ws_bytes(B, N, C, R)))
        return PVCONV_EWORKSPACE;
    return pv_launch_devoxelize_backward(dout, B, N, C, R, pn, ids, dgrid, workspace,
                                         as_stream(stream));
}

pvconv_status pvconv_devoxelize_backward(const float* dout, int B, int N, int C, int R,
                                         const float* norm_coords, float* dgrid, void* workspace,
                                         size_t workspace_bytes, void* stream) {
    if (B > 0 && N > 0 && !norm_coords) return PVCONV_EINVAL;
    return devox_backward(dout, B, N, C, R, norm_coords, nullptr, dgrid, workspace,
                          workspace_bytes, stream);
}

pvconv_status pvconv_devoxelize_nearest_backward(const float* dout, int B, int N, int C, int R,
                                                 const int32_t* vox_id, float* dgrid,
                                                 void* workspace, size_t workspace_bytes,
                                                 void* stream) {
    if (B > 0 && N > 0 && !vox_id) return PVCONV_EINVAL;
    return devox_backward(dout, B, N, C, R, nullptr, vox_id, dgrid, workspace, workspace_bytes,
                          stream);
}

size_t pvconv_conv3d_backward_data_workspace_size(int Cin, int Cout, pvconv_dtype dt) {
    if (Cin < 1 || Cout < 1 || Cin > PVCONV_MAX_CONV_CHANNELS ||
        Cout > PVCONV_MAX_CONV_CHANNELS || !dtype_ok(dt))
        return 0;
    return pv_conv3d_bwd_data_ws_bytes(Cin, Cout, dt == PVCONV_BF16);
}

pvconv_status pvconv_conv3d_backward_data(const void* dy, int B, int R, int Cin, int Cout,
                                          const void* weight, pvconv_dtype dt, void* dx,
                                          pvconv_dtype dx_dt, void* workspace,
                                          size_t workspace_bytes, void* stream) {
    if (B < 0 || R < 1 || R > PVCONV_MAX_R || Cin < 1 || Cout < 1 ||
        Cin > PVCONV_MAX_CONV_CHANNELS || Cout > PVCONV_MAX_CONV_CHANNELS)
        return PVCONV_EINVAL;
    if (!dtype_ok(dt) || !dtype_ok(dx_dt)) return PVCONV_EINVAL;
    if (B == 0) return PVCONV_OK;
    if (!dy || !weight || !dx) return PVCONV_EINVAL;
    if (((uintptr_t)dy & (esize(dt) - 1)) || ((uintptr_t)weight & (esize(dt) - 1)) ||
        ((uintptr_t)dx & (esize(dx_dt) - 1)))
        return PVCONV_EINVAL;
    if (dt == PVCONV_BF16 && Cin % 32 != 0) return PVCONV_ENOTSUP;
    if (dy == dx) return PVCONV_EINVAL;
    const size_t need = pv_conv3d_bwd_data_ws_bytes(Cin, Cout, dt == PVCONV_BF16);
    if (!workspace || ((uintptr_t)workspace & 255) || workspace_bytes < need)
        return PVCONV_EWORKSPACE;
    return pv_launch_conv3d_backward_data(dy, B, R, Cin, Cout, weight, dt == PVCONV_BF16, dx,
                                          dx_dt == PVCONV_BF16, workspace, as_stream(stream));
}

size_t pvconv_conv3d_backward_weight_workspace_size(int B, int R, int Cin, int Cout) {
    if (B < 0 || R < 1 || R > PVCONV_MAX_R || Cin < 1 || Cout < 1 ||
        Cin > PVCONV_MAX_CONV_CHANNELS || Cout > PVCONV_MAX_CONV_CHANNELS)
        return 0;
    return pv_conv3d_wgrad_ws_bytes(B, R, Cin, Cout);
}

pvconv_status pvconv_conv3d_backward_weight(const void* dy, const void* x, pvconv_dtype dt,
                                            int B, int R, int Cin, int Cout, float* dw,
                                            void* workspace, size_t workspace_bytes,
                                            void* stream) {
    if (B < 0 || R < 1 || R > PVCONV_MAX_R || Cin < 1 || Cout < 1 ||
        Cin > PVCONV_MAX_CONV_CHANNELS || Cout > PVCONV_MAX_CONV_CHANNELS || !dtype_ok(dt) ||
        !sizes_fit(B, (long long)R * R * R))
        return PVCONV_EINVAL;
    if (dt != PVCONV_BF16 || Cout % 64 != 0 || Cin % 16 != 0) return PVCONV_ENOTSUP;
    if (!dw || (B > 0 && (!dy || !x))) return PVCONV_EINVAL;
    if (!pv_aligned16(dy) || !pv_aligned16(x) || ((uintptr_t)dw & 3)) return PVCONV_EINVAL;
    const size_t need = pv_conv3d_wgrad_ws_bytes(B, R, Cin, Cout);
    if (need && (!workspace || ((uintptr_t)workspace & 255) || workspace_bytes < need))
        return PVCONV_EWORKSPACE;
    return pv_launch_conv3d_backward_weight(dy, x, B, R, Cin, Cout, dw, workspace,
                                            as_stream(stream));
}

pvconv_status pvconv_act_bn_backward(const float* dy, const void* y, pvconv_dtype y_dt, int M,
                                     int C, const pvconv_bn* bn, pvconv_act act, float slope,
                                     float* dz, void* stream) {
    if (M < 0 || C < 1 || !dtype_ok(y_dt) || !act_ok(act) || !bn_ok(bn)) return PVCONV_EINVAL;
    if (M == 0) return PVCONV_OK;
    if (!dy || !y || !dz) return PVCONV_EINVAL;
    if (((uintptr_t)dy & 3) || ((uintptr_t)y & (esize(y_dt) - 1)) || ((uintptr_t)dz & 3))
        return PVCONV_EINVAL;
    return pv_launch_act_bn_backward(dy, y, y_dt == PVCONV_BF16, (size_t)M, C,
                                     pv_make_fold(bn, nullptr), act, slope, dz,
                                     as_stream(stream));
}

}  // extern "C"
