// 3x3x3 volumetric convolution + folded batch norm + activation
// (Section 4.1 "Feature Aggregation"; fixed-offset kernel of Section 3, Eq. 1).
//
// bf16 path: implicit GEMM on the MFMA units. M = output voxels, N = output
// channels, K = 27 taps x input channels.
//
//  * One workgroup per CU owns an 8x8x8 brick of output voxels and 32*NB
//    output channels. Its waves form 4 voxel groups x WCH channel groups:
//    each wave computes two u-slices of the brick (128 voxels) against
//    32*NB/WCH channels with v_mfma_f32_32x32x16_bf16: A = weights (rows =
//    output channels), B = voxels (columns), 4 x NB/WCH accumulator blocks,
//    so every voxel fragment feeds NB/WCH MFMAs and every weight fragment
//    four. WCH = 1: four waves, one per SIMD; WCH = 2 (eight waves, two per
//    SIMD, so that one wave's waits overlap the other's MFMAs) for
//    64-channel tiles of narrow inputs on small grids. Inputs of up to 128 channels on grids with enough tiles
//    take 64-channel tiles with compact halos (SB): 72 KB of LDS and at
//    most 128 accumulator registers per wave, so two workgroups share a CU
//    and one's prologue and epilogue overlap the other's MFMAs.
//  * The input is consumed in chunks of 16 channels (one MFMA k step). A
//    chunk's 10x10x10 halo (zero outside the grid) sits in LDS at 48 bytes per
//    voxel (32 bytes of data) and 640 bytes per 10-voxel row: with that
//    padding the 16-byte fragment reads of every tap hit distinct banks (SB:
//    32 bytes per voxel, the two halves swapped where bit 2 of w is set, the
//    same effect). The next chunk's halo is fetched into the other of two
//    buffers during the first taps of the current chunk.
//  * The 27 taps of a chunk are unrolled, so every LDS fragment address is a
//    per-lane base plus an immediate. Weights come pre-packed in fragment
//    order (pv_pack_conv_weights_kernel): each fragment load is one coalesced
//    1 KB buffer load, issued two taps ahead into registers. The only barrier
//    is one per chunk.
//  * The epilogue folds bias + batch norm into one scale/shift per channel
//    (a table in LDS), applies the activation and stages the tile through
//    LDS so that every store instruction writes whole contiguous rows.
//
// fp32 path: four lanes per (voxel, output channel), plain FMA loops.
#include <algorithm>

#include "pv_common.h"

namespace {

constexpr int kBrick = 8;                          // output brick edge (u, v, w)
constexpr int kHalo = kBrick + 2;                  // halo edge
constexpr int kHaloVox = kHalo * kHalo * kHalo;    // 1000
constexpr int kKC = 16;                            // input channels per chunk
constexpr int kVoxPitch = 48;                      // LDS bytes per halo voxel
constexpr int kRowPitch = 640;                     // LDS bytes per 10-voxel row
constexpr int kHaloBytes = kHalo * kHalo * kRowPitch;  // 64000 per buffer
constexpr int kPieces = kHaloVox * 2;              // 16-byte pieces per chunk halo
constexpr int kTaps = 27;
constexpr int kOOB = 0x40000000;                   // byte offset always out of range
// Epilogue staging: the output tile goes through LDS as [512 voxels][PW
// channels] rows of up to 256 bytes, padded by 16 bytes, then out with
// coalesced 16-byte stores.
constexpr int kStageRow = 256 + 16;
constexpr int kStageBytes = kBrick * kBrick * kBrick * kStageRow;  // 139264
constexpr int kLdsBytes = kStageBytes > 2 * kHaloBytes ? kStageBytes : 2 * kHaloBytes;
// Two-workgroups-per-CU variant (SB): the epilogue stages the 64-channel
// tile through LDS in one pass (bf16: whole 128-byte halves of the output
// rows) or two (fp32). Its two halo buffers are compact: 32 bytes per
// voxel, 384 per 10-voxel row (64 bytes of padding: consecutive rows start
// half a 256-byte bank window apart), and the two 16-byte halves of a voxel
// swap places where bit 2 of its w is set, so that the 16 lanes of a
// fragment read that are served together (8 consecutive voxels of two
// consecutive rows) hit distinct banks.
constexpr int kStageRowSB = 128 + 16;
constexpr int kVoxPitchSB = 32;
constexpr int kRowPitchSB = kHalo * kVoxPitchSB + 64;            // 384
constexpr int kHaloBytesSB = kHalo * kHalo * kRowPitchSB;        // 38400 per buffer
constexpr int kLdsBytesSB =
    512 * kStageRowSB > 2 * kHaloBytesSB ? 512 * kStageRowSB : 2 * kHaloBytesSB;

__device__ __forceinline__ uint4 pack8(const uint16_t* e) {
    return make_uint4((uint32_t)e[0] | ((uint32_t)e[1] << 16), (uint32_t)e[2] | ((uint32_t)e[3] << 16),
                      (uint32_t)e[4] | ((uint32_t)e[5] << 16), (uint32_t)e[6] | ((uint32_t)e[7] << 16));
}

__device__ __forceinline__ pv_bf16x8 as_frag(uint4 v) {
    pv_bf16x8 r;
    __builtin_memcpy(&r, &v, 16);
    return r;
}

// Raw buffer loads: an offset at or past the resource's size reads as zero,
// which provides the conv's zero padding (and zero channels past C_in)
// without branches or selects on the loaded value.
__device__ __forceinline__ __amdgpu_buffer_rsrc_t make_rsrc(const void* base, uint32_t bytes) {
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(base), (short)0, (int)bytes,
                                             0x00020000);
}

__device__ __forceinline__ uint4 bload16(__amdgpu_buffer_rsrc_t r, int voff, int soff) {
    const auto v = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    uint4 u;
    __builtin_memcpy(&u, &v, 16);
    return u;
}

// 8 bf16 channels one by one: channel i at voff + 2i if i < valid, else zero.
__device__ __forceinline__ uint4 bload8_elems(__amdgpu_buffer_rsrc_t r, int voff, int soff,
                                              int valid) {
    uint16_t e[8];
#pragma unroll
    for (int i = 0; i < 8; i++)
        e[i] = __builtin_amdgcn_raw_buffer_load_b16(r, i < valid ? voff + 2 * i : kOOB, soff, 0);
    return pack8(e);
}

// WCH channel groups of waves: 1 (four waves, 256 threads) or 2 (eight
// waves, two per SIMD). SB: compact halo buffers and at most 128
// accumulator registers, so that two workgroups share a CU and one's
// prologue and epilogue overlap the other's MFMAs.
// SP (with occ, the forward's first convolution on its sparse grid): an
// MFMA whose 32 input voxels are all empty adds only zeros to accumulators
// that started at +0, so it is skipped (same bits). A bitmap of the halo's
// occupied voxels (one word per halo row) gives each wave, once per brick,
// which of its blocks have an occupied input voxel at each tap.
// OS (with need, the forward's last convolution, whose grid the
// devoxelisation samples only at its points' trilinear corners, all within
// one voxel of an occupied voxel): only the blocks of 32 output voxels with
// an occupied voxel within one voxel run their MFMAs, dealt evenly to the
// waves; a wave with none skips its fragment reads too, and a workgroup with
// none returns before loading anything; the outputs they leave are not needed (their values are
// unspecified, those of needed voxels the same bits as the full loop's).
// Split-K (ksplit > 1): the input channels' chunks are divided among ksplit
// groups of workgroups (cps chunks each); split s reads channels from
// s*cps*16 (rows of x_ld elements), and writes its fp32 partial sums, without
// batch norm or activation, to y + s*B*R^3*Cout (the caller passes an
// identity fold and no activation); pv_conv_split_reduce_kernel adds them.
template <int NB, int WCH, bool VEC, bool SB = false, bool SP = false, bool OS = false>
__global__ __launch_bounds__(256 * WCH, SB ? 2 : 1) void pv_conv3d_bf16_kernel(
    const uint16_t* __restrict__ x, const uint16_t* __restrict__ wpk, PvBnFold bn, int act,
    float slope, void* __restrict__ y, int out_bf16, int vec_out, int R, int Cin, int Cout,
    int nbr, int nblocks, int x_ld, int ksplit, int cps, int B, const int32_t* __restrict__ occ,
    const int32_t* __restrict__ need) {
    __shared__ __attribute__((aligned(16))) char lds[SB ? kLdsBytesSB : kLdsBytes];
    __shared__ float bn_tab[2][NB * 32];  // folded scale and shift per output channel
    // SP, OS: occupied w of each halo row
    __shared__ uint32_t occ_row[SP || OS ? kHalo * kHalo : 1];

    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    // Blocks are dispatched round-robin over the 8 XCDs; give each XCD a
    // contiguous range of bricks so that neighbouring halos share its L2.
    // With SP or OS a brick's work depends on its cloud's occupancy: there
    // each XCD takes an eighth of every cloud (whole clouds per XCD left the
    // XCDs that drew the denser clouds running long after the others).
    int bid = blockIdx.x;
    const int per = nblocks / max(B, 1);  // workgroups per cloud
    if ((SP || OS) && (per & 7) == 0 && per * B == nblocks) {
        // every XCD takes one contiguous eighth of every cloud, rotated by
        // the cloud, so that clouds of different occupancy share the XCDs
        const int x = bid & 7, k = bid >> 3, c = k / (per >> 3), j = k % (per >> 3);
        bid = c * per + ((x + c) & 7) * (per >> 3) + j;
    } else if ((nblocks & 7) == 0) {
        bid = (bid & 7) * (nblocks >> 3) + (bid >> 3);
    }
    if (ksplit > 1) {  // this workgroup's share of the input channels
        const int split = bid % ksplit;
        bid /= ksplit;
        const int c_lo = split * cps * kKC;
        x += c_lo;
        wpk += (size_t)split * cps * kTaps * ((Cout + 31) / 32) * 512;
        Cin = min(Cin - c_lo, cps * kKC);
        y = (float*)y + (size_t)split * B * R * R * R * Cout;
    }
    constexpr int NT = NB * 32;
    // Waves = 4 voxel groups x WCH channel groups: each wave owns two u-slices
    // of the brick (4 blocks of 32 voxels) and NBW blocks of 32 channels.
    static_assert(NB % WCH == 0, "channel groups split the tile evenly");
    constexpr int NTH = 256 * WCH, NBW = NB / WCH;
    constexpr int kSets = (kPieces + NTH - 1) / NTH;  // halo pieces per thread
    const int wv = wave / WCH, wc = wave % WCH;
    const int ntiles = (Cout + NT - 1) / NT;  // the last tile may be partly past Cout
    const int nt = bid % ntiles;
    bid /= ntiles;
    const int bw = bid % nbr;
    bid /= nbr;
    const int bv = bid % nbr;
    bid /= nbr;
    const int bu = bid % nbr;
    const int b = bid / nbr;
    const int u0 = bu * kBrick, v0 = bv * kBrick, w0 = bw * kBrick, n0 = nt * NT;
    const size_t cloud = (size_t)b * R * R * R;
    const int nch = (Cin + kKC - 1) / kKC;

    const int r32 = lane & 31, khalf = lane >> 5;
    // LDS byte address of this lane's B fragment (voxel column r32 of block
    // mb, channels khalf*8 .. +7) at tap offset (0,0,0) in buffer 0: block mb
    // covers u = 2*wave + mb/2 and v rows (mb&1)*4 .. +3, eight w each.
    // SB: one base per w shift of the taps (the half swap depends on w).
    constexpr int RP = SB ? kRowPitchSB : kRowPitch, HB = SB ? kHaloBytesSB : kHaloBytes;
    auto half_off = [](int hw, int h) { return SB ? (h ^ ((hw >> 2) & 1)) * 16 : h * 16; };
    // Slot mb of the wave computes the block at u-slice blk_u(mb), v rows
    // blk_v(mb)*4 .. +3: 2*wave + mb/2 and mb&1, unless OS deals the blocks
    // out (then slot mb holds block g = bits 4mb .. 4mb+3 of gpack, u-slice
    // g/2, v half g&1).
    uint32_t gpack = 0u;
    auto blk_u = [&](int mb) -> int {
        if constexpr (OS) return (int)((gpack >> (4 * mb + 1)) & 7u);
        return 2 * wv + (mb >> 1);
    };
    auto blk_v = [&](int mb) -> int {
        if constexpr (OS) return (int)((gpack >> (4 * mb)) & 1u);
        return mb & 1;
    };
    int bbase[4], bsw[4][3];
    auto place = [&](int mb, int ul, int vh) {
        const int vl = vh * 4 + (r32 >> 3), wl = r32 & 7;
        bbase[mb] = (ul * kHalo + vl) * kRowPitch + wl * kVoxPitch + khalf * 16;
#pragma unroll
        for (int tw = 0; tw < 3; tw++)
            bsw[mb][tw] = (ul * kHalo + vl) * kRowPitchSB + (wl + tw) * kVoxPitchSB +
                          half_off(wl + tw, khalf);
    };
#pragma unroll
    for (int mb = 0; mb < 4; mb++) place(mb, 2 * wv + (mb >> 1), mb & 1);
    // LDS byte address (in buffer 0) of block mb's B fragment at tap tn
    auto frag_addr = [&](int mb, int tn) {
        const int tu = tn / 9, tv = (tn / 3) % 3, tw = tn % 3;
        if constexpr (SB) return bsw[mb][tw] + (tu * kHalo + tv) * RP;
        return bbase[mb] + (tu * kHalo + tv) * kRowPitch + tw * kVoxPitch;
    };

    // Halo pieces of this thread: piece p = set*NTH + tid is voxel p/2 (as
    // (hu,hv,hw) of the 10x10x10 halo), channels (p%2)*8 .. +7 of the chunk.
    // Threads past the last piece repeat voxel 999 (same value, same slot).
    // goff: byte offset into the input resource (kOOB outside the grid);
    // loff: LDS byte offset in buffer 0.
    const int ulo = max(u0 - 1, 0), uhi = min(u0 + kBrick + 1, R);
    // rows of x_ld elements, of which the first Cin are this conv's (or this
    // split's) channels; the range ends with the last row's channels
    const size_t slab = (size_t)R * R * x_ld;  // elements per u-slab
    const __amdgpu_buffer_rsrc_t xr = make_rsrc(
        x + cloud * x_ld + ulo * slab, (uint32_t)(((uhi - ulo) * slab - (x_ld - Cin)) * 2));
    const int pq = tid & 1;
    int goff[kSets], loff[kSets];
    if constexpr (SP || OS) {
        if (tid < kHalo * kHalo) occ_row[tid] = 0u;
        __syncthreads();
    }
#pragma unroll
    for (int set = 0; set < kSets; set++) {
        const int h = min(set * (NTH / 2) + (tid >> 1), kHaloVox - 1);
        const int hu = h / (kHalo * kHalo), hv = (h / kHalo) % kHalo, hw = h % kHalo;
        const int gu = u0 + hu - 1, gv = v0 + hv - 1, gw = w0 + hw - 1;
        bool in = gu >= 0 && gu < R && gv >= 0 && gv < R && gw >= 0 && gw < R;
        // a sparse input grid: empty voxels read as zero (their rows were
        // never written), through the out-of-range offset
        if (occ && in) in = occ[cloud + ((size_t)gu * R + gv) * R + gw] > 0;
        if constexpr (SP)
            if (in && pq == 0) atomicOr(&occ_row[hu * kHalo + hv], 1u << hw);
        if constexpr (OS && !SP)
            if (in && pq == 0 && need[cloud + ((size_t)gu * R + gv) * R + gw] > 0)
                atomicOr(&occ_row[hu * kHalo + hv], 1u << hw);
        goff[set] = in ? ((((gu - ulo) * R + gv) * R + gw) * x_ld + pq * 8) * 2 : kOOB;
        loff[set] = SB ? (hu * kHalo + hv) * kRowPitchSB + hw * kVoxPitchSB + half_off(hw, pq)
                       : (hu * kHalo + hv) * kRowPitch + hw * kVoxPitch + pq * 16;
    }
    // Piece of set `set` for the chunk starting at channel cc: pieces whose
    // channels lie past Cin read as zero.
    auto halo_load = [&](int set, int cc) -> uint4 {
        if (VEC) return bload16(xr, cc + pq * 8 < Cin ? goff[set] : kOOB, cc * 2);
        return bload8_elems(xr, goff[set], cc * 2, Cin - cc - pq * 8);
    };

    // Packed weights: for chunk c, tap t and 32-channel output group g the 64
    // lanes' fragments are 1 KB at ((c*27 + t)*G + g)*1024 (output channels
    // past Cout packed as zeros).
    const int G = (Cout + 31) / 32;
    const __amdgpu_buffer_rsrc_t wr = make_rsrc(wpk, (uint32_t)((size_t)nch * kTaps * G * 1024));
    const int wlane = lane * 16;
    auto load_w = [&](int c, int tap, pv_bf16x8 (&wf)[NBW]) {
        const int cc = c < nch ? c : nch - 1;  // past the end: reload, never used
#pragma unroll
        for (int nb = 0; nb < NBW; nb++)
            wf[nb] = as_frag(bload16(wr, wlane,
                                     ((cc * kTaps + tap) * G + nt * NB + wc * NBW + nb) * 1024));
    };

    pv_f32x16 acc[4][NBW];
#pragma unroll
    for (int i = 0; i < 4; i++)
#pragma unroll
        for (int j = 0; j < NBW; j++)
#pragma unroll
            for (int e = 0; e < 16; e++) acc[i][j][e] = 0.f;

    if (tid < NT) {  // channels past Cout take the last one's (never stored)
        float sc, sh;
        pv_bn_coeffs(bn, min(n0 + tid, Cout - 1), sc, sh);
        bn_tab[0][tid] = sc;
        bn_tab[1][tid] = sh;
    }
    // A sparse input (occ) whose halo holds no occupied voxel: every product
    // is zero, so the accumulators stay zero and the epilogue writes
    // act(BN(0)), the same bits as the full loop would. The reduction is also
    // the barrier before the epilogue reads bn_tab.
    bool live = true;
    if (occ) {
        bool any = false;
#pragma unroll
        for (int set = 0; set < kSets; set++) any |= goff[set] != kOOB;
        live = __syncthreads_or(any);
    }
    // OS: block g's outputs (u-slice g/2, v rows (g&1)*4 .. +3) and their
    // neighbours are halo rows g/2 .. +2 by (g&1)*4 .. +5, all ten w; the
    // block is live when one of them holds an occupied voxel. A brick with no
    // live block has nothing to compute or store. The live blocks are dealt
    // to the waves in turn (slot k of wave w takes the (4k + w)-th), so that
    // the brick's busiest wave has ceil(live / 4) of them; bit k of blive
    // marks a slot that holds one.
    bool wave_live = true;
    uint32_t blive = 15u;
    if constexpr (OS) {
        if constexpr (!SP) __syncthreads();  // the bitmap is complete
        bool lv = false;
        if (lane < 16) {  // lane g tests block g
            uint32_t m = 0u;
#pragma unroll
            for (int du = 0; du < 3; du++)
#pragma unroll
                for (int dv = 0; dv < 6; dv++)
                    m |= occ_row[((lane >> 1) + du) * kHalo + (lane & 1) * 4 + dv];
            lv = m != 0u;
        }
        const uint32_t bl = (uint32_t)__builtin_amdgcn_ballot_w64(lv);
        if (bl == 0u) return;  // every wave reads the same bitmap
        uint32_t m = bl;
        const int ws = __builtin_amdgcn_readfirstlane(wv);
        for (int i = 0; i < ws; i++) m &= m - 1u;
        uint32_t gp = 0u, bv = 0u;
#pragma unroll
        for (int k = 0; k < 4; k++) {
            const uint32_t g = m ? (uint32_t)__builtin_ctz(m) : 0u;  // idle: valid addresses
            bv |= (m ? 1u : 0u) << k;
            gp |= g << (4 * k);
#pragma unroll
            for (int i = 0; i < 4; i++) m &= m - 1u;  // past the next four live blocks
        }
        gpack = __builtin_amdgcn_readfirstlane(gp);
        blive = __builtin_amdgcn_readfirstlane(bv);
#pragma unroll
        for (int k = 0; k < 4; k++) place(k, blk_u(k), blk_v(k));
        wave_live = blive != 0u;
    }
    // SP: bit 10*tv + w of msk[mb][tu] is set when block mb's input row
    // (tu, tv) holds an occupied voxel at halo w; the block's fragment at tap
    // (tu, tv, tw) covers w = tw .. tw + 7 of four such rows.
    uint32_t msk[4][3];
    if constexpr (SP) {
#pragma unroll
        for (int mb = 0; mb < 4; mb++)
#pragma unroll
            for (int tu = 0; tu < 3; tu++) {
                uint32_t m = 0u;
#pragma unroll
                for (int tv = 0; tv < 3; tv++) {
                    uint32_t r = 0u;
#pragma unroll
                    for (int k = 0; k < 4; k++)
                        r |= occ_row[(blk_u(mb) + tu) * kHalo + blk_v(mb) * 4 + tv + k];
                    m |= r << (10 * tv);
                }
                msk[mb][tu] = __builtin_amdgcn_readfirstlane(m);
            }
    }
    if (live) {
        // Chunk 0's halo, the weights of the first kWD taps.
#pragma unroll
        for (int set = 0; set < kSets; set++) *(uint4*)(lds + loff[set]) = halo_load(set, 0);
        // Weights load kWD taps ahead through a ring of kWD + 1 sets (a
        // divisor of 27, so the ring realigns at every chunk). The 32-channel
        // tiles (one wave per SIMD, four MFMAs per tap) look further ahead,
        // and store each halo piece eight taps after its load (1.5-2 % on
        // the small grids' convolutions).
        constexpr int kWD = (!SB && NB == 1) ? 8 : 2, kWR = kWD + 1;
        static_assert(kTaps % kWR == 0, "the weight ring realigns at every chunk");
        pv_bf16x8 wf[kWR][NBW];
#pragma unroll
        for (int k = 0; k < kWD; k++) load_w(0, k, wf[k]);
        __syncthreads();

        // Chunk c sits in LDS buffer c%2: 27 taps, unrolled. Tap t computes with
        // weight set t%kWR while tap t+kWD's weights load, and with B fragments
        // bf[t%2] while tap t+1's are read from LDS into the other set. Piece
        // set s of the next chunk's halo is loaded at tap s into
        // hr[s%kHaloLag] and stored to the other LDS buffer at tap
        // s+kHaloLag. One loop body for every chunk keeps the accumulators in
        // the same registers throughout.
        constexpr int kHaloLag = (!SB && NB == 1) ? 8 : 4;
        for (int c = 0; c < nch; c++) {
            const int cur_off = (c & 1) * HB, nxt_off = HB - cur_off;
            // Next chunk's halo. Past the last chunk the double-buffered
            // variant reloads the last chunk into the idle buffer, and SB
            // loads out of range (zeros, no memory access) into it: with
            // unconditional loads the compiler's wait counts stay exact (with
            // a branch around them it must assume they were skipped, and each
            // tap's weight wait then also waits for the next tap's weights).
            // Element-wise loads (!VEC) keep the branch: unconditional, they
            // spill registers.
            const bool fetch = VEC || !SB || c + 1 < nch;
            const int cn = c + 1 < nch ? (c + 1) * kKC : (SB ? Cin : c * kKC);
            pv_bf16x8 bf[2][4];
            uint4 hr[kHaloLag];
#pragma unroll
            for (int mb = 0; mb < 4; mb++)
                bf[0][mb] = *(const pv_bf16x8*)(lds + frag_addr(mb, 0) + cur_off);
#pragma unroll
            for (int t = 0; t < kTaps; t++) {
                const int cur = t & 1, nxt = cur ^ 1;
                if (t + kWD < kTaps)
                    load_w(c, t + kWD, wf[(t + kWD) % kWR]);
                else
                    load_w(c + 1, t + kWD - kTaps, wf[(t + kWD) % kWR]);
                if (fetch && t >= kHaloLag && t < kSets + kHaloLag)
                    *(uint4*)(lds + loff[t - kHaloLag] + nxt_off) = hr[(t - kHaloLag) % kHaloLag];
                if (fetch && t < kSets) hr[t % kHaloLag] = halo_load(t, cn);
                if (t + 1 < kTaps && (!OS || wave_live)) {
#pragma unroll
                    for (int mb = 0; mb < 4; mb++)
                        bf[nxt][mb] = *(const pv_bf16x8*)(lds + frag_addr(mb, t + 1) + cur_off);
                }
#pragma unroll
                for (int mb = 0; mb < 4 && (!OS || wave_live); mb++) {
                    if constexpr (OS) {
                        uint32_t bb = blive;
                        asm volatile("" : "+s"(bb));
                        if (((bb >> mb) & 1u) == 0u) continue;
                    }
                    if constexpr (SP) {
                        // opaque here, so that the test stays a scalar shift,
                        // mask and branch inside the loop (hoisted, the 108
                        // tests of a chunk would not fit in scalar registers)
                        uint32_t mm = msk[mb][t / 9];
                        asm volatile("" : "+s"(mm));
                        if (((mm >> (10 * ((t / 3) % 3) + t % 3)) & 0xffu) == 0u) continue;
                    }
#pragma unroll
                    for (int nb = 0; nb < NBW; nb++)
                        acc[mb][nb] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(
                            wf[t % kWR][nb], bf[cur][mb], acc[mb][nb], 0, 0, 0);
                }
                __builtin_amdgcn_sched_barrier(0);
            }
            // chunk done: the next halo is complete and this buffer is free
            if constexpr (SB)
                pv_lds_barrier();  // LDS only: the weight prefetch stays in flight
            else
                __syncthreads();
        }
    }

    // Epilogue. Block (mb, nb) holds D[n][voxel]: lane has voxel column r32
    // of the block and output channels 8*j + 4*khalf + i (e = 4*j + i). The
    // tile is staged in LDS in passes of PW channels (256 bytes per voxel),
    // then each thread copies 16-byte pieces out, so every store instruction
    // writes whole contiguous rows.
    // The output type is a compile-time branch of the epilogue (one straight
    // copy per type), so that the per-element code carries no type tests.
    const float neg = act == PVCONV_ACT_LEAKY ? slope : (act == PVCONV_ACT_RELU ? 0.f : 1.f);
    auto epilogue = [&](auto out_type) {
        constexpr bool OBF = decltype(out_type)::value;
        constexpr int esz = OBF ? 2 : 4;
        constexpr int PW = SB ? (OBF ? (NT < 64 ? NT : 64) : (NT < 32 ? NT : 32))
                              : (OBF ? (NT < 128 ? NT : 128) : (NT < 64 ? NT : 64));
        constexpr int kRow = SB ? kStageRowSB : kStageRow;  // LDS bytes per staged voxel
        constexpr int pieces = PW * esz / 16;  // 16-byte pieces per voxel row
        const size_t yrow = (size_t)Cout * esz;
#pragma unroll
        for (int pass = 0; pass * PW < NT; pass++) {
#pragma unroll
            for (int nb = 0; nb < NBW; nb++) {
#pragma unroll
                for (int j = 0; j < 4; j++) {
                    const int nl = (wc * NBW + nb) * 32 + 8 * j + 4 * khalf;  // channel in the tile
                    if (nl < pass * PW || nl >= (pass + 1) * PW) continue;
                    const float4 sc = *(const float4*)&bn_tab[0][nl];
                    const float4 sh = *(const float4*)&bn_tab[1][nl];
                    const int cb = (nl - pass * PW) * esz;  // byte offset in the row
#pragma unroll
                    for (int mb = 0; mb < 4; mb++) {
                        if (OS && ((blive >> mb) & 1u) == 0u) continue;  // an idle slot
                        const int vox = blk_u(mb) * 64 + (blk_v(mb) * 4 + (r32 >> 3)) * 8 +
                                        (r32 & 7);
                        float r[4] = {acc[mb][nb][4 * j + 0] * sc.x + sh.x,
                                      acc[mb][nb][4 * j + 1] * sc.y + sh.y,
                                      acc[mb][nb][4 * j + 2] * sc.z + sh.z,
                                      acc[mb][nb][4 * j + 3] * sc.w + sh.w};
#pragma unroll
                        for (int e = 0; e < 4; e++) r[e] = r[e] >= 0.f ? r[e] : r[e] * neg;
                        char* d = lds + vox * kRow + cb;
                        if constexpr (OBF)
                            *(uint2*)d = make_uint2(pv_pack_bf16x2(r[0], r[1]),
                                                    pv_pack_bf16x2(r[2], r[3]));
                        else
                            *(float4*)d = make_float4(r[0], r[1], r[2], r[3]);
                    }
                    __builtin_amdgcn_sched_barrier(0);
                }
            }
            pv_lds_barrier();
            // copy out: piece k of voxel vox (k < pieces); a pass partly past
            // Cout copies its first ncols channels (whole pieces, then the
            // elements of a last partial one)
            const size_t col = ((size_t)n0 + pass * PW) * esz;
            const int ncols = min(PW, Cout - n0 - pass * PW);
            if (ncols <= 0) continue;  // uniform: the whole pass lies past Cout
            const int vbytes = ncols * esz;
            if (ncols == PW && vec_out && u0 + kBrick <= R && v0 + kBrick <= R &&
                w0 + kBrick <= R) {
                // the whole brick inside the grid: batches of UC pieces per
                // thread, every LDS read of a batch issued before its stores
                constexpr int kIt = 512 * pieces / NTH, UC = kIt < 4 ? kIt : 4;
                static_assert(kIt % UC == 0, "copy-out batches divide the pieces");
#pragma unroll 1
                for (int i0 = 0; i0 < kIt; i0 += UC) {
                    uint4 val[UC];
#pragma unroll
                    for (int q = 0; q < UC; q++) {
                        const int i = tid + (i0 + q) * NTH, vox = i / pieces, k = i % pieces;
                        val[q] = *(const uint4*)(lds + vox * kRow + k * 16);
                    }
#pragma unroll
                    for (int q = 0; q < UC; q++) {
                        const int i = tid + (i0 + q) * NTH, vox = i / pieces, k = i % pieces;
                        const int u = u0 + (vox >> 6), v = v0 + ((vox >> 3) & 7),
                                  ww = w0 + (vox & 7);
                        *(uint4*)((char*)y + (cloud + ((size_t)u * R + v) * R + ww) * yrow + col +
                                  k * 16) = val[q];
                    }
                }
                pv_lds_barrier();
                continue;
            }
            for (int i = tid; i < 512 * pieces; i += NTH) {
                const int vox = i / pieces, k = i % pieces;
                const int u = u0 + (vox >> 6), v = v0 + ((vox >> 3) & 7), ww = w0 + (vox & 7);
                if (u >= R || v >= R || ww >= R || k * 16 >= vbytes) continue;
                const uint4 val = *(const uint4*)(lds + vox * kRow + k * 16);
                char* dst = (char*)y + (cloud + ((size_t)u * R + v) * R + ww) * yrow + col + k * 16;
                const int nel = min(16, vbytes - k * 16) / esz;  // elements of this piece
                if (vec_out && nel * esz == 16) {
                    *(uint4*)dst = val;
                } else {
                    const uint32_t q[4] = {val.x, val.y, val.z, val.w};
                    for (int e = 0; e < nel; e++) {
                        if constexpr (OBF)
                            ((uint16_t*)dst)[e] = (uint16_t)(q[e >> 1] >> ((e & 1) * 16));
                        else
                            ((uint32_t*)dst)[e] = q[e];
                    }
                }
            }
            pv_lds_barrier();
        }
    };
    if (out_bf16)
        epilogue(std::integral_constant<bool, true>{});
    else
        epilogue(std::integral_constant<bool, false>{});
}

// Repack bf16 weights [Cout][27][Cin] into the fragment order the MFMA conv
// reads: 16-byte element ((c*27 + t)*G + g)*64 + lane holds the 8 channels
// k = c*16 + (lane/32)*8 .. +7 of output channel g*32 + lane%32 at tap t
// (zero past Cin and past Cout), G = ceil(Cout/32). One thread per element;
// one launch packs the
// weights of all the convolutions of a layer (the blocks of job q follow those of
// jobs 0 .. q-1).
static_assert(kKC == kPvPackKC && kTaps == kPvPackTaps, "the packing matches the kernel");

__global__ __launch_bounds__(256) void pv_pack_conv_weights_kernel(PvPackJobs jobs) {
    pv_pack_role(jobs, blockIdx.x);
}

// fp32 path: four consecutive lanes per output (voxel, channel), each
// summing the taps tap = part, part + 4, ... over all input channels (16
// bytes at a time when the rows allow), then a 4-lane sum.
template <bool V4>
__global__ __launch_bounds__(256) void pv_conv3d_f32_kernel(const float* __restrict__ x,
                                                            const float* __restrict__ w,
                                                            PvBnFold bn, int act, float slope,
                                                            void* __restrict__ y, int out_bf16,
                                                            int B, int R, int Cin, int Cout) {
    const size_t V = (size_t)R * R * R;
    const size_t t = (size_t)blockIdx.x * 256 + threadIdx.x;
    const size_t i = t >> 2;  // output element
    const int part = (int)(t & 3);
    const bool live = i < (size_t)B * V * Cout;
    const size_t ic = live ? i : 0;  // dead lanes still join the 4-lane sum
    const int o = (int)(ic % Cout);
    const size_t vox = ic / Cout;
    const size_t b = vox / V;
    const int r = (int)(vox % V);
    const int u = r / (R * R), v = (r / R) % R, ww = r % R;
    float s = 0.f;
    if (live) {
        for (int tap = part; tap < 27; tap += 4) {
            const int nu = u + tap / 9 - 1, nv = v + (tap / 3) % 3 - 1, nw = ww + tap % 3 - 1;
            if (nu < 0 || nu >= R || nv < 0 || nv >= R || nw < 0 || nw >= R) continue;
            const float* xi = x + (b * V + ((size_t)nu * R + nv) * R + nw) * Cin;
            const float* wk = w + ((size_t)o * 27 + tap) * Cin;
            if (V4) {
                for (int c = 0; c < Cin; c += 4) {
                    const float4 a = *(const float4*)(xi + c), q = *(const float4*)(wk + c);
                    s += q.x * a.x;
                    s += q.y * a.y;
                    s += q.z * a.z;
                    s += q.w * a.w;
                }
            } else {
                for (int c = 0; c < Cin; c++) s += wk[c] * xi[c];
            }
        }
    }
    s += __shfl_xor(s, 1, 64);
    s += __shfl_xor(s, 2, 64);
    if (!live || part != 0) return;
    float scale, shift;
    pv_bn_coeffs(bn, o, scale, shift);
    const float val = pv_activate(s * scale + shift, act, slope);
    if (out_bf16)
        ((uint16_t*)y)[i] = pv_f32_to_bf16(val);
    else
        ((float*)y)[i] = val;
}

// y = act(BN(sum of the ksplit partial sums)), the partials added in split
// order. Four channels per thread (C_out % 4 == 0 and 16-byte aligned rows),
// else one.
template <bool V4>
__global__ __launch_bounds__(256) void pv_conv_split_reduce_kernel(
    const float* __restrict__ part, int ksplit, size_t n, int Cout, PvBnFold bn, int act,
    float slope, void* __restrict__ y, int out_bf16) {
    const size_t i0 = ((size_t)blockIdx.x * 256 + threadIdx.x) * (V4 ? 4 : 1);
    if (i0 >= n) return;
    const int c0 = (int)(i0 % Cout);
    float v[V4 ? 4 : 1];
    if constexpr (V4) {
        float4 a = *(const float4*)(part + i0);
        for (int s = 1; s < ksplit; s++) {
            const float4 b = *(const float4*)(part + (size_t)s * n + i0);
            a.x += b.x;
            a.y += b.y;
            a.z += b.z;
            a.w += b.w;
        }
        v[0] = a.x;
        v[1] = a.y;
        v[2] = a.z;
        v[3] = a.w;
    } else {
        float a = part[i0];
        for (int s = 1; s < ksplit; s++) a += part[(size_t)s * n + i0];
        v[0] = a;
    }
#pragma unroll
    for (int e = 0; e < (V4 ? 4 : 1); e++) {
        float sc, sh;
        pv_bn_coeffs(bn, c0 + e, sc, sh);
        v[e] = pv_activate(v[e] * sc + sh, act, slope);
    }
    if (out_bf16) {
        uint16_t* o = (uint16_t*)y + i0;
        if constexpr (V4)
            *(uint2*)o = make_uint2(pv_pack_bf16x2(v[0], v[1]), pv_pack_bf16x2(v[2], v[3]));
        else
            o[0] = pv_f32_to_bf16(v[0]);
    } else {
        float* o = (float*)y + i0;
        if constexpr (V4)
            *(float4*)o = make_float4(v[0], v[1], v[2], v[3]);
        else
            o[0] = v[0];
    }
}

template <int NB, int WCH, bool SB = false>
void launch_bf16(const void* x, int B, int R, int Cin, int Cout, const void* w,
                 const PvBnFold& bn, int act, float slope, void* y, bool out_bf16, bool vec,
                 hipStream_t s, int ksplit = 1, int cps = 0, const int32_t* occ = nullptr,
                 const int32_t* need = nullptr) {
    const int nbr = (R + kBrick - 1) / kBrick;
    const size_t blocks =
        (size_t)B * nbr * nbr * nbr * ((Cout + NB * 32 - 1) / (NB * 32)) * ksplit;
    // 16-byte stores: aligned output with rows of whole 16-byte pieces
    const bool vec_out = pv_aligned16(y) && ((size_t)Cout * (out_bf16 ? 2 : 4)) % 16 == 0;
#define PV_CONV(V, SPX, OSX)                                                                \
    hipLaunchKernelGGL((pv_conv3d_bf16_kernel<NB, WCH, V, SB, SPX, OSX>),                   \
                       dim3((unsigned)blocks),                                                 \
                       dim3(256 * WCH), 0, s, (const uint16_t*)x, (const uint16_t*)w, bn, act, \
                       slope, y, (int)out_bf16, (int)vec_out, R, Cin, Cout, nbr, (int)blocks, \
                       Cin, ksplit, cps, B, occ, need)
    // a sparse input on the two-per-CU form skips its empty fragments' MFMAs,
    // a needed-output mask its unneeded blocks, waves and bricks (given
    // together, the two are the same counts)
    if (vec && SB && occ && need)
        PV_CONV(true, SB, SB);
    else if (vec && SB && occ)
        PV_CONV(true, SB, false);
    else if (vec && SB && need)
        PV_CONV(true, false, SB);
    else if (vec)
        PV_CONV(true, false, false);
    else
        PV_CONV(false, false, false);
#undef PV_CONV
}

}  // namespace

size_t pv_conv3d_ws_bytes(int Cin, int Cout, bool bf16) {
    if (!bf16) return 0;
    const size_t nch = (size_t)(Cin + kKC - 1) / kKC;
    return nch * kKC * kTaps * (size_t)((Cout + 31) / 32 * 32) * 2;  // Cout padded to 32
}

void pv_pack_job(PvPackJobs& jobs, const void* w, int Cin, int Cout, void* packed) {
    PvPackJob& J = jobs.job[jobs.n++];
    J.w = (const uint16_t*)w;
    J.packed = (uint4*)packed;
    J.Cin = Cin;
    J.Cout = Cout;
    J.total = (int)(pv_conv3d_ws_bytes(Cin, Cout, true) / 16);
    J.vec = (int)(Cin % 8 == 0 && pv_aligned16(w));
    J.blocks = (J.total + 255) / 256;
}

void pv_launch_pack_conv_weights(const PvPackJobs& jobs, hipStream_t s) {
    const int blocks = pv_pack_blocks(jobs);
    if (blocks > 0)
        hipLaunchKernelGGL(pv_pack_conv_weights_kernel, dim3(blocks), dim3(256), 0, s, jobs);
}

int pv_conv3d_splits(int B, int R, int Cin, int Cout) {
    // Grids so small that the unsplit launch (32-channel tiles) leaves most
    // CUs idle, fewer than 64 workgroups (PVCNN++'s R = 8 level: 16), divide
    // the input channels among more workgroups of the two-per-CU variant.
    // At 64 and more (the R = 16 blocks) the split's extra prologues, fp32
    // partials and reduction cost more than the occupancy gains (measured).
    const int nbr = (R + kBrick - 1) / kBrick;
    const long bricks = (long)B * nbr * nbr * nbr;
    const long tiles = bricks * (Cout / 64);
    const int nch = (Cin + kKC - 1) / kKC;
    if (Cout % 64 != 0 || Cin % kKC != 0 || bricks * ((Cout + 31) / 32) >= 64 || nch < 2 ||
        tiles == 0)
        return 1;
    const int want = (int)((512 + tiles - 1) / tiles);
    const int cps = (nch + std::min(want, nch) - 1) / std::min(want, nch);
    return (nch + cps - 1) / cps;
}

size_t pv_conv3d_split_ws_bytes(int B, int R, int Cin, int Cout) {
    const int S = pv_conv3d_splits(B, R, Cin, Cout);
    return S > 1 ? (size_t)S * B * R * R * R * Cout * 4 : 0;
}

pvconv_status pv_launch_conv3d(const void* x, int B, int R, int Cin, int Cout, const void* w,
                               const PvBnFold& bn, int act, float slope, bool bf16, void* y,
                               bool out_bf16, void* ws, hipStream_t s, bool packed,
                               float* split_ws, const int32_t* occ, const int32_t* need) {
    if (B == 0) return PVCONV_OK;
    if (bf16) {
        if (!packed) {
            PvPackJobs jobs{};
            pv_pack_job(jobs, w, Cin, Cout, ws);
            pv_launch_pack_conv_weights(jobs, s);
        }
        w = ws;
        const bool vec = (Cin % 8 == 0) && pv_aligned16(x);
        const int S = split_ws ? pv_conv3d_splits(B, R, Cin, Cout) : 1;
        if (S > 1) {
            // fp32 partial sums per split (identity fold, no activation),
            // then their fixed-order sum with the batch norm and activation
            const int nch = (Cin + kKC - 1) / kKC, cps = (nch + S - 1) / S;
            launch_bf16<2, 1, true>(x, B, R, Cin, Cout, w, PvBnFold{}, PVCONV_ACT_NONE, 0.f,
                                    split_ws, false, vec, s, S, cps, occ);
            const size_t n = (size_t)B * R * R * R * Cout;
            const bool v4 = Cout % 4 == 0 && pv_aligned16(y) && pv_aligned16(split_ws);
            const size_t threads = v4 ? n / 4 : n;
            const unsigned blocks = (unsigned)((threads + 255) / 256);
            if (v4)
                hipLaunchKernelGGL(pv_conv_split_reduce_kernel<true>, dim3(blocks), dim3(256), 0,
                                   s, split_ws, S, n, Cout, bn, act, slope, y, (int)out_bf16);
            else
                hipLaunchKernelGGL(pv_conv_split_reduce_kernel<false>, dim3(blocks), dim3(256),
                                   0, s, split_ws, S, n, Cout, bn, act, slope, y, (int)out_bf16);
            return pv_launch_status();
        }
        // Channel tile: the widest (most reuse of each halo) that still gives
        // about one workgroup per CU; small grids (R = 16) take narrow tiles.
        const int nbr = (R + kBrick - 1) / kBrick;
        const long bricks = (long)B * nbr * nbr * nbr;
        // Inputs of up to 128 channels with enough tiles for two workgroups
        // per CU: 64-channel tiles with compact halos, two per CU (one's
        // prologue and epilogue overlap the other's MFMAs: 11 % faster at
        // 64->128 and 64->64, 2.5 % at 128->128, than one 128-channel
        // workgroup per CU). Otherwise 64-channel tiles, one workgroup per
        // CU: eight waves (two channel groups) for narrow inputs, four for
        // wide ones (a 128-channel tile of four waves would hold all 256
        // accumulator registers and spill in its epilogue).
        const bool two = Cin <= 64;
        if (Cin <= 128 && Cout % 64 == 0 && bricks * (Cout / 64) >= 512) {
            launch_bf16<2, 1, true>(x, B, R, Cin, Cout, w, bn, act, slope, y, out_bf16, vec, s, 1, 0, occ,
                                    need);
        } else if (Cout % 64 == 0 && bricks * (Cout / 64) >= 256) {
            if (two)
                launch_bf16<2, 2>(x, B, R, Cin, Cout, w, bn, act, slope, y, out_bf16, vec, s, 1, 0, occ);
            else
                launch_bf16<2, 1>(x, B, R, Cin, Cout, w, bn, act, slope, y, out_bf16, vec, s, 1, 0, occ);
        } else {
            launch_bf16<1, 1>(x, B, R, Cin, Cout, w, bn, act, slope, y, out_bf16, vec, s, 1, 0, occ);
        }
    } else {
        const size_t total = (size_t)B * R * R * R * Cout;
        const unsigned blocks = (unsigned)((4 * total + 255) / 256);
        if (Cin % 4 == 0 && pv_aligned16(x) && pv_aligned16(w))
            hipLaunchKernelGGL(pv_conv3d_f32_kernel<true>, dim3(blocks), dim3(256), 0, s,
                               (const float*)x, (const float*)w, bn, act, slope, y, (int)out_bf16,
                               B, R, Cin, Cout);
        else
            hipLaunchKernelGGL(pv_conv3d_f32_kernel<false>, dim3(blocks), dim3(256), 0, s,
                               (const float*)x, (const float*)w, bn, act, slope, y, (int)out_bf16,
                               B, R, Cin, Cout);
    }
    return pv_launch_status();
}
