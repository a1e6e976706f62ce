// Wave64 cross-lane helpers shared by the gfx950 kernels of libpvconv: DPP
// moves, the read of lane 63, and a reduction over the wave.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

// Moves of a 32- or 64-bit value across lanes by DPP (row_mask ROWS; rows
// left out keep 0).
template <int CTRL, int ROWS>
static __device__ __forceinline__ uint32_t dpp_u32(uint32_t v) {
    return (uint32_t)__builtin_amdgcn_update_dpp(0, (int)v, CTRL, ROWS, 0xf, false);
}
template <int CTRL, int ROWS, typename T>
static __device__ __forceinline__ T dpp_move(T v) {
    static_assert(sizeof(T) == 4 || sizeof(T) == 8, "32- or 64-bit lanes");
    T r;
    if constexpr (sizeof(T) == 4) {
        uint32_t u;
        __builtin_memcpy(&u, &v, 4);
        u = dpp_u32<CTRL, ROWS>(u);
        __builtin_memcpy(&r, &u, 4);
    } else {
        uint64_t u;
        __builtin_memcpy(&u, &v, 8);
        const uint64_t lo = dpp_u32<CTRL, ROWS>((uint32_t)u);
        const uint64_t hi = dpp_u32<CTRL, ROWS>((uint32_t)(u >> 32));
        u = lo | (hi << 32);
        __builtin_memcpy(&r, &u, 8);
    }
    return r;
}
template <typename T>
static __device__ __forceinline__ T read_lane63(T v) {
    T r;
    if constexpr (sizeof(T) == 4) {
        int u;
        __builtin_memcpy(&u, &v, 4);
        u = __builtin_amdgcn_readlane(u, 63);
        __builtin_memcpy(&r, &u, 4);
    } else {
        int u[2];
        __builtin_memcpy(u, &v, 8);
        u[0] = __builtin_amdgcn_readlane(u[0], 63);
        u[1] = __builtin_amdgcn_readlane(u[1], 63);
        __builtin_memcpy(&r, u, 8);
    }
    return r;
}

// Reduction over the wave (every lane gets the result) by DPP moves: quad
// swaps, half-row and row mirrors, then the row broadcasts into lane 63.
// The moves fill lanes they leave out with 0, so op must have 0 as its
// identity: sums, or maxima of non-negative values (every use here).
template <typename T, typename Op>
static __device__ __forceinline__ T wave_reduce(T v, Op op) {
    v = op(v, dpp_move<0xB1, 0xf>(v));   // quad_perm [1,0,3,2]
    v = op(v, dpp_move<0x4E, 0xf>(v));   // quad_perm [2,3,0,1]
    v = op(v, dpp_move<0x141, 0xf>(v));  // row_half_mirror
    v = op(v, dpp_move<0x140, 0xf>(v));  // row_mirror
    v = op(v, dpp_move<0x142, 0xa>(v));  // row_bcast:15 into rows 1 and 3
    v = op(v, dpp_move<0x143, 0xc>(v));  // row_bcast:31 into rows 2 and 3
    return read_lane63(v);
}
