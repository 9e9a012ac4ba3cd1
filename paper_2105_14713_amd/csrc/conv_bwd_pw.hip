// Input gradient of 1x1 (any stride, no padding; N in {2, 4, 8, 16, 32}) and
// 3x3 (stride 1 or 2; N in {8, 16, 32}) 1xN-pruned convolutions on matrix
// cores: fp32, NCHW.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4 (Eq. 7 with Omega-bar, stored as Eq. 8's BSR)
// and Sec. 4.1 (fine-tuning with the pattern fixed).  For a 1x1 layer the
// adjoint of Eq. 7 is
//     dX[c][pixel] = sum_g sum_{i < N} Wt_g[c][i] * dY[gN + i][pixel],
//     Wt_g[c][i] = D[z][i] if col-group g keeps input channel c at block z,
//                  else 0,
// a dense contraction over the output channels with Omega-bar's transpose
// as the left operand (a strided layer's dY pixel feeds input (oh*sh, ow*sw)
// only).
//
// Work.  A workgroup of eight waves computes 32 input channels x 256 pixels
// (each wave one 32-pixel column block) with v_mfma_f32_32x32x2f32: row =
// input channel, column = pixel, one col-group (N output channels, N / 2
// steps) after another.  Col-groups that keep none of the 32 channels are
// skipped.
//  - Index.  I ascends within a col-group, so the blocks of a col-group whose
//    channel falls in [c0, c0 + 32) are one run.  In a prologue each thread
//    finds one col-group's run by narrowing with 32 samples at a time (one
//    round of independent loads per 32x narrowing) and records its first
//    block and a mask of the channels it keeps: channel c0 + k is block
//    first + popcount(mask below bit k).
//  - A.  The 32 x N tiles Wt_g of 8 col-groups at a time (N = 16, 32) or
//    256 / N (N <= 8) are copied from D straight into one LDS buffer between
//    two barriers (rows of channels a col-group does not keep read zeros
//    through an out-of-range offset), so no registers hold tiles in flight
//    and a wave multiplies 4N (N >= 16) or 128 MFMA steps per barrier pair
//    (a version with one col-group's tile per barrier, built in LDS one
//    col-group ahead through registers, was 2-16 % slower per layer).
//  - B.  dY rows gN .. gN+N-1 at the wave's pixels, loaded into registers
//    one col-group ahead.
// Every output element is written once, by one lane, after a fixed-order
// accumulation: the result does not depend on timing.

#include <utility>

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kBpWaves = 8;
constexpr int kBpThreads = 64 * kBpWaves;
constexpr int kBpPix = kBpWaves * 32;                   // pixels per workgroup (a 32-pixel block per wave)
constexpr int kBpMaxG = kBpThreads;                     // col-groups (one prologue thread each)

// First entry in [zb, ze) of a col-group whose input channel is >= c0 (ze if
// none).  I ascends within a col-group, so the entries below c0 form a
// prefix; [lo, hi) is narrowed 32 samples at a time (one round of independent
// loads per 32x narrowing; entries before lo are < c0, and I[hi] >= c0 or
// hi = ze).
__device__ __forceinline__ int32_t run_first(__amdgpu_buffer_rsrc_t rI, int32_t zb, int32_t ze, int32_t c0) {
    auto ld_i = [&](int32_t e) { return int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, e * 4, 0, 0)); };
    int32_t lo = zb, hi = ze;
    while (hi - lo > 32) {
        const int32_t step = (hi - lo + 31) / 32;
        int32_t below = 0;   // samples k (I[lo + k*step] < c0) form a prefix
#pragma unroll
        for (int k = 0; k < 32; ++k) {
            const int32_t e = lo + k * step;
            below += (e < hi && ld_i(e) < c0) ? 1 : 0;
        }
        const int32_t nlo = below == 0 ? lo : lo + (below - 1) * step + 1;
        hi = below == 0 ? lo : min(hi, lo + below * step);
        lo = nlo;
    }
    int32_t below = 0;   // the entries [lo, hi): those below c0
#pragma unroll
    for (int k = 0; k < 32; ++k) {
        const int32_t e = lo + k;
        below += (e < hi && ld_i(e) < c0) ? 1 : 0;
    }
    return lo + below;
}

// ---------------------------------------------------------------------------
// Input gradient of a 3x3 layer, stride 1 or 2, any padding: for every tap
// (q, r) the contraction above with dY read at the positions the tap maps the
// input pixel to,
//     dX[c][ih][iw] = sum_g sum_{i < N} sum_{q, r} Wt_g[c][i][q][r] * dY[gN + i][oh][ow],
//     oh = (ih + ph - q) / s, ow = (iw + pw - r) / s,
// the term absent where a division is inexact or (oh, ow) lies outside the
// output.  Same workgroup shape as the 1x1 kernel (32 input channels x 256
// input pixels, a wave per 32-pixel block, rows = channels); each col-group
// is multiplied for its nine taps in turn.  Its 32 x (N x 9) tile of
// Omega-bar's transpose (row c: the kept block's D row, taps innermost) is
// copied from D straight into LDS between two barriers (rows of channels the
// col-group does not keep read zeros); the dY values of the next tap are
// loaded while this tap multiplies.  At stride 2 an input pixel takes 1, 2 or
// 4 of the nine taps; the others read zeros.  Each output element is stored
// once: deterministic.
// ---------------------------------------------------------------------------

// Workgroup -> (32-channel tile, pixel tile) of the input-gradient kernels: a
// one-dimensional grid in which the channel tiles of one pixel tile are
// consecutive logical ids, and consecutive logical ids run on one XCD, so
// the dY values of a pixel tile are fetched into one L2 (with the pixel
// tile as the grid's x and the channel tile as its y they were spread over
// all eight).
__device__ __forceinline__ void dx_tile(const ConvArgs& a, int32_t& c0, int32_t& p0) {
    const int32_t ct = (a.m + 31) / 32;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), int32_t(gridDim.x));
    c0 = (L % ct) * 32;
    p0 = (L / ct) * kBpPix;
}

template <typename F, int... Is>
__device__ __forceinline__ void static_for_impl(F&& f, std::integer_sequence<int, Is...>) {
    (f(std::integral_constant<int, Is>{}), ...);
}
template <int Count, typename F>
__device__ __forceinline__ void static_for(F&& f) {
    static_for_impl(f, std::make_integer_sequence<int, Count>{});
}

template <int N, int SD>
__global__ void __launch_bounds__(kBpThreads) __attribute__((amdgpu_waves_per_eu(4))) bwd_data_k3(ConvArgs a, const float* __restrict__ dy,
                                                           float* __restrict__ dx) {
    typedef PwMfma<32> M;
    typedef typename M::acc_t acc_t;
    constexpr int KK = 9;
    constexpr int S = N / 2;                            // MFMA steps per tap
    constexpr int RW = N * KK;                          // floats of a D row
    constexpr int AP = RW + 1;                          // LDS pitch of a tile row
    static_assert(32 % kBpWaves == 0 && RW >= 64, "tile rows split over waves, pieces of 64 floats");
    __shared__ int32_t sFirst[kBpMaxG];                 // first block of col-group g in the tile
    __shared__ uint32_t sMask[kBpMaxG];                 // bit k: g keeps channel c0 + k
    __shared__ int32_t sGl[kBpMaxG];                    // col-groups with a kept block in the tile
    __shared__ int32_t sCnt[kBpWaves];
    __shared__ float sA[32 * AP];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int32_t c0, p0;                                     // first input channel and input pixel
    dx_tile(a, c0, p0);

    // ---- Index prologue: thread g < G finds col-group g's run of blocks in
    // [c0, c0 + 32): entries first, first + 1, ... in ascending channel order,
    // so channel c0 + k is block first + popcount(mask below bit k).
    const int32_t g = tid;
    bool any = false;
    const __amdgpu_buffer_rsrc_t rI = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(a.I), 0, __builtin_amdgcn_readfirstlane(a.t * 4), kRawBufferFlags);
    if (g < a.G) {
        int32_t zb, ze;
        group_range(a, g, zb, ze);
        const int32_t first = run_first(rI, zb, ze, c0);
        uint32_t mask = 0;
#pragma unroll
        for (int k = 0; k < 32; ++k) {
            const int32_t e = first + k;
            const int32_t c = e < ze ? int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, e * 4, 0, 0)) : INT32_MAX;
            if (c < c0 + 32 && c < a.m) mask |= 1u << (c - c0);
        }
        sFirst[g] = first;
        sMask[g] = mask;
        any = mask != 0;
    }
    const uint64_t bal = __ballot(any);
    if (lane == 0) sCnt[wave] = __builtin_popcountll(bal);
    __syncthreads();
    int32_t base = 0, ng = 0;
#pragma unroll
    for (int w = 0; w < kBpWaves; ++w) {
        base += w < wave ? sCnt[w] : 0;
        ng += sCnt[w];
    }
    if (any) sGl[base + __builtin_popcountll(bal & ((uint64_t(1) << lane) - 1))] = g;
    __syncthreads();

    // ---- Lane roles.  A: row (input channel c0 + lane % 32), entry parity
    // kk.  B: input pixel lane % 32 of the wave's block, output channel 2s + kk.
    const int col = lane & 31, kk = lane >> 5;
    const int32_t HWo = a.HWo, HWi = a.H * a.W;
    const int32_t batch = a.npix / HWo;
    const int32_t ybytes = int32_t(int64_t(batch) * a.n * HWo * 4);
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(dy), 0, __builtin_amdgcn_readfirstlane(ybytes), kRawBufferFlags);
    const uint32_t chb = uint32_t(HWo) * 4;   // bytes between dY channels
    const int32_t p = p0 + wave * 32 + col;
    int64_t xo = -1;                          // dX element offset at channel 0 (or -1)
    uint32_t yk[KK];                          // per tap: byte offset of dY at channel kk (or out of range)
    {
        const bool in = p < batch * HWi;
        const int32_t b = in ? p / HWi : 0, hw = p - b * HWi;
        const int32_t ih = hw / a.W, iw = hw - ih * a.W;
        if (in) xo = int64_t(b) * a.m * HWi + hw;
        const int64_t ybase = int64_t(b) * a.n * HWo;
        int32_t orow[3], ocol[3];
        bool vrow[3], vcol[3];
#pragma unroll
        for (int q = 0; q < 3; ++q) {
            const int32_t th = ih + a.ph - q, tw = iw + a.pw - q;
            vrow[q] = th >= 0 && (SD == 1 || (th & 1) == 0) && th / SD < a.Ho;
            vcol[q] = tw >= 0 && (SD == 1 || (tw & 1) == 0) && tw / SD < a.Wo;
            orow[q] = (th / SD) * a.Wo;
            ocol[q] = tw / SD;
        }
#pragma unroll
        for (int q = 0; q < 3; ++q)
#pragma unroll
            for (int r = 0; r < 3; ++r)
                yk[q * 3 + r] = in && vrow[q] && vcol[r]
                                    ? uint32_t((ybase + orow[q] + ocol[r]) * 4) + uint32_t(kk) * chb
                                    : kBufferOutOfRange;
    }
    // The step's output channel pair in the scalar offset (uniform, in range
    // for every row below n); a row past n (ragged last col-group) takes an
    // out-of-range vector offset instead.  One path, no branch: the loads of
    // consecutive taps stay in one counted sequence.
    auto load_b = [&](float (&bv)[S], int32_t gg, int tap) __attribute__((always_inline)) {
        const int32_t ob = __builtin_amdgcn_readfirstlane(gg * N);
        if (ob + N <= a.n) {   // (uniform) every row exists: no per-step mask
#pragma unroll
            for (int s = 0; s < S; ++s)
                bv[s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rY, int32_t(yk[tap]), int32_t(uint32_t(ob + 2 * s) * chb), 0));
        } else {
            const int32_t lim = a.n - ob - kk;   // this lane's rows 2s + kk < n - ob
#pragma unroll
            for (int s = 0; s < S; ++s)
                bv[s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rY, int32_t(2 * s < lim ? yk[tap] : kBufferOutOfRange), int32_t(uint32_t(ob + 2 * s) * chb), 0));
        }
    };
    // Tile of col-group gg: row c (channel c0 + c) is D row z (RW floats) if
    // the col-group keeps the channel at block z, else zeros (an out-of-range
    // offset).  Copied in 64-float pieces, the last one of a row overlapping
    // the one before; wave w copies rows 4w .. 4w + 3.
    constexpr int C = (RW + 63) / 64;                   // pieces per row
    const v4i32 rD = buffer_rsrc(a.D, int32_t(int64_t(a.t) * RW * 4));
    auto copy_a = [&](int32_t gg) __attribute__((always_inline)) {
        const int32_t first = __builtin_amdgcn_readfirstlane(sFirst[gg]);
        const uint32_t mask = __builtin_amdgcn_readfirstlane(sMask[gg]);
#pragma unroll
        for (int rr = 0; rr < 32 / kBpWaves; ++rr) {
            const int32_t row = wave * (32 / kBpWaves) + rr;
            const bool kept = (mask >> row) & 1;
            const int32_t z = first + __builtin_popcount(mask & ((1u << row) - 1));
#pragma unroll
            for (int u = 0; u < C; ++u) {
                const int j0 = u * 64 < RW - 64 ? u * 64 : RW - 64;
                copy4_to_lds(rD, (const lds_char*)(sA + row * AP + j0),
                             kept ? (z * RW + j0 + lane) * 4 : int32_t(kBufferOutOfRange), 0);
            }
        }
    };

    acc_t acc;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) acc[r] = 0.f;
    auto multiply = [&](int tap, const float (&bv)[S]) __attribute__((always_inline)) {
        const float* ar = &sA[col * AP + kk * KK + tap];
#pragma unroll
        for (int s = 0; s < S; ++s) acc = M::step(ar[2 * s * KK], bv[s], acc);
    };

    if (ng > 0) {
        float b0[S], b1[S];
        copy_a(sGl[0]);
        load_b(b0, sGl[0], 0);
        vm_wait<0>();
        __syncthreads();
        // Step (col-group j, tap T) multiplies register set (j * 9 + T) % 2
        // and loads the next step's dY values into the other one.
        auto group = [&](int32_t j, auto par) __attribute__((always_inline)) {
            const int32_t gg = sGl[j];
            const bool more = j + 1 < ng;
            const int32_t gn = more ? sGl[j + 1] : gg;
            static_for<KK>([&](auto T) {
                constexpr bool odd = ((decltype(par)::value + decltype(T)::value) & 1) != 0;
                float (&cur)[S] = odd ? b1 : b0;
                float (&nxt)[S] = odd ? b0 : b1;
                if (T + 1 < KK)
                    load_b(nxt, gg, T + 1 < KK ? T + 1 : 0);
                else if (more)
                    load_b(nxt, gn, 0);
                multiply(T, cur);
            });
            if (more) {
                __syncthreads();   // every wave is done with the tile
                copy_a(gn);
                vm_wait<0>();
                __syncthreads();
            }
        };
        for (int32_t j = 0; j < ng; j += 2) {
            group(j, std::integral_constant<int, 0>{});
            if (j + 1 >= ng) break;
            group(j + 1, std::integral_constant<int, KK & 1>{});
        }
    }

    // ---- Store: MFMA (row, col) -> dX channel c0 + row at the lane's pixel
    // (zero for pixels no tap reaches).
    if (xo >= 0) {
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) {
            const int32_t c = c0 + M::row(lane, r);
            if (c < a.m) store_out(&dx[xo + int64_t(c) * HWi], acc[r]);
        }
    }
}


// ---------------------------------------------------------------------------
// The 1x1 kernel (see the top of the file).
// ---------------------------------------------------------------------------

template <int N>
__global__ void __launch_bounds__(kBpThreads) __attribute__((amdgpu_waves_per_eu(4))) bwd_data_pw(ConvArgs a, const float* __restrict__ dy,
                                                            float* __restrict__ dx) {
    typedef PwMfma<32> M;
    typedef typename M::acc_t acc_t;
    constexpr int CG = N >= 16 ? 8 : 256 / N;           // col-groups per stage (a 32 x 8N or 32 x 256 tile)
    constexpr int S = N / 2;                            // MFMA steps per col-group
    constexpr int RW = CG * N;                          // floats of a staged row
    constexpr int AP = RW + 1;                          // LDS pitch of a staged row
    constexpr int CPR = RW / 64;                        // 64-float copies per row
    static_assert(RW % 64 == 0 && 32 % kBpWaves == 0, "whole copies, rows split over waves");
    static_assert(N >= 2 && 64 % N == 0, "an MFMA step takes two output channels of one col-group");
    __shared__ int32_t sFirst[kBpMaxG];                 // first block of col-group g in the tile
    __shared__ uint32_t sMask[kBpMaxG];                 // bit k: g keeps channel c0 + k
    __shared__ int32_t sGl[kBpMaxG];                    // col-groups with a kept block in the tile
    __shared__ int32_t sCnt[kBpWaves];
    __shared__ float sA[32 * AP];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int32_t c0, p0;                                     // first input channel and output pixel
    dx_tile(a, c0, p0);

    // ---- Index prologue (as in the 3x3 kernel).
    const int32_t g = tid;
    bool any = false;
    const __amdgpu_buffer_rsrc_t rI = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(a.I), 0, __builtin_amdgcn_readfirstlane(a.t * 4), kRawBufferFlags);
    if (g < a.G) {
        int32_t zb, ze;
        group_range(a, g, zb, ze);
        const int32_t first = run_first(rI, zb, ze, c0);
        uint32_t mask = 0;
#pragma unroll
        for (int k = 0; k < 32; ++k) {
            const int32_t e = first + k;
            const int32_t c = e < ze ? int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, e * 4, 0, 0)) : INT32_MAX;
            if (c < c0 + 32 && c < a.m) mask |= 1u << (c - c0);
        }
        sFirst[g] = first;
        sMask[g] = mask;
        any = mask != 0;
    }
    const uint64_t bal = __ballot(any);
    if (lane == 0) sCnt[wave] = __builtin_popcountll(bal);
    __syncthreads();
    int32_t base = 0, ng = 0;
#pragma unroll
    for (int w = 0; w < kBpWaves; ++w) {
        base += w < wave ? sCnt[w] : 0;
        ng += sCnt[w];
    }
    if (any) sGl[base + __builtin_popcountll(bal & ((uint64_t(1) << lane) - 1))] = g;
    __syncthreads();

    // ---- Lane roles.  A: row (input channel c0 + lane % 32), entry parity
    // kk.  B: output pixel lane % 32 of the wave's block, output channel 2s + kk.
    const int col = lane & 31, kk = lane >> 5;
    const int32_t HWo = a.HWo, HWi = a.H * a.W;
    const int32_t ybytes = int32_t(int64_t(a.npix / HWo) * a.n * HWo * 4);
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(dy), 0, __builtin_amdgcn_readfirstlane(ybytes), kRawBufferFlags);
    const uint32_t chb = uint32_t(HWo) * 4;   // bytes between dY channels
    const int32_t p = p0 + wave * 32 + col;
    uint32_t yk = kBufferOutOfRange;          // byte offset of the pixel's dY value at channel kk
    int64_t xo = -1;                          // element offset of its dX value at channel 0
    int32_t ih0 = 0, iw0 = 0;                 // the input position it reads (oh * sh, ow * sw)
    if (p < a.npix) {
        const int32_t b = p / HWo, hw = p - b * HWo;
        const int32_t oh = hw / a.Wo, ow = hw - oh * a.Wo;
        ih0 = oh * a.sh;
        iw0 = ow * a.sw;
        yk = uint32_t((int64_t(b) * a.n * HWo + hw) * 4) + uint32_t(kk) * chb;
        xo = int64_t(b) * a.m * HWi + int64_t(ih0) * a.W + iw0;
    }
    auto load_b = [&](float (&bv)[S], int32_t gg) __attribute__((always_inline)) {
        const int32_t ob = __builtin_amdgcn_readfirstlane(gg * N);
        if (ob + N <= a.n) {   // (uniform) every row exists: no per-step mask
#pragma unroll
            for (int s = 0; s < S; ++s)
                bv[s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rY, int32_t(yk), int32_t(uint32_t(ob + 2 * s) * chb), 0));
        } else {
            const int32_t lim = a.n - ob - kk;   // this lane's rows 2s + kk < n - ob
#pragma unroll
            for (int s = 0; s < S; ++s)
                bv[s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rY, int32_t(2 * s < lim ? yk : kBufferOutOfRange), int32_t(uint32_t(ob + 2 * s) * chb), 0));
        }
    };
    // Stage of col-groups sGl[j0 .. j0 + CG): row c holds, for slot j, the
    // D row of the block where col-group sGl[j0 + j] keeps channel c0 + c
    // (zeros if it does not, or past the last col-group).  Copy u of a row
    // covers floats 64u .. 64u + 63: slot (64u + lane) / N, entry lane % N.
    const v4i32 rD = buffer_rsrc(a.D, int32_t(int64_t(a.t) * N * 4));
    auto copy_a = [&](int32_t j0) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < CPR; ++u) {
            const int32_t j = j0 + (64 * u + lane) / N;
            const int32_t gg = j < ng ? sGl[j] : 0;
            const int32_t first = sFirst[gg];
            const uint32_t mask = j < ng ? sMask[gg] : 0u;
#pragma unroll
            for (int rr = 0; rr < 32 / kBpWaves; ++rr) {
                const int32_t row = wave * (32 / kBpWaves) + rr;
                const bool kept = (mask >> row) & 1;
                const int32_t z = first + __builtin_popcount(mask & ((1u << row) - 1));
                copy4_to_lds(rD, (const lds_char*)(sA + row * AP + 64 * u),
                             kept ? (z * N + (lane % N)) * 4 : int32_t(kBufferOutOfRange), 0);
            }
        }
    };

    acc_t acc;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) acc[r] = 0.f;
    auto multiply = [&](int slot, const float (&bv)[S]) __attribute__((always_inline)) {
        const float* ar = &sA[col * AP + slot * N + kk];
#pragma unroll
        for (int s = 0; s < S; ++s) acc = M::step(ar[2 * s], bv[s], acc);
    };

    if (ng > 0) {
        float b0[S], b1[S];
        copy_a(0);
        load_b(b0, sGl[0]);
        vm_wait<0>();
        __syncthreads();
        // Col-group j multiplies register set j % 2 (CG is even) and loads
        // col-group j + 1's dY values into the other one.
        for (int32_t j0 = 0; j0 < ng; j0 += CG) {
            static_for<CG>([&](auto J) {
                constexpr int jj = decltype(J)::value;
                float (&cur)[S] = (jj & 1) ? b1 : b0;
                float (&nxt)[S] = (jj & 1) ? b0 : b1;
                if (j0 + jj < ng) {
                    if (j0 + jj + 1 < ng) load_b(nxt, sGl[j0 + jj + 1]);
                    multiply(jj, cur);
                }
            });
            if (j0 + CG < ng) {
                __syncthreads();   // every wave is done with the stage
                copy_a(j0 + CG);
                vm_wait<0>();
                __syncthreads();
            }
        }
    }

    // ---- Store: MFMA (row, col) -> dX channel c0 + row at the lane's input
    // position; a strided layer's other positions of the sh x sw block get 0
    // (the blocks of all output pixels cover the input once: Ho * sh >= H).
    if (xo >= 0) {
        const int32_t dhe = min(a.sh, a.H - ih0), dwe = min(a.sw, a.W - iw0);
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) {
            const int32_t c = c0 + M::row(lane, r);
            if (c >= a.m) continue;
            float* q = &dx[xo + int64_t(c) * HWi];
            store_out(q, acc[r]);
            if (a.sh * a.sw > 1)
                for (int32_t dh = 0; dh < dhe; ++dh)
                    for (int32_t dw = 0; dw < dwe; ++dw)
                        if (dh != 0 || dw != 0) store_out(q + int64_t(dh) * a.W + dw, 0.f);
        }
    }
}


// ---------------------------------------------------------------------------
// Input gradient of a stride-2 3x3 layer by parity class.  An input pixel
// (ih, iw) receives tap (q, r) only where ih + ph - q and iw + pw - r are
// even, so the pixels with one parity of (ih + ph, iw + pw) share their taps:
// (even, even) taps q, r in {0, 2} (four), mixed ones two, (odd, odd) the
// centre tap only.  One launch per class (QA, RB = the parities of the taps
// it takes) walks that class's pixels densely (iw = 2j + bb for consecutive
// j: consecutive lanes read consecutive dY columns) and multiplies only its
// taps, where the single 3x3 kernel multiplies all nine and reads zeros for
// the rest.  Steps are (col-group, tap) pairs, eight per stage: the stage's
// 32 x N tiles (D rows of the kept channels at the tap, gathered from D's
// [block][row][tap] order) are copied into LDS between two barriers as in
// the 1x1 kernel; dY values are loaded one step ahead.
// ---------------------------------------------------------------------------

template <int N, int QA, int RB>
__global__ void __launch_bounds__(kBpThreads) __attribute__((amdgpu_waves_per_eu(4))) bwd_data_s2(ConvArgs a, const float* __restrict__ dy,
                                                           float* __restrict__ dx, int32_t ca, int32_t cb) {
    typedef PwMfma<32> M;
    typedef typename M::acc_t acc_t;
    constexpr int NQ = QA == 0 ? 2 : 1, NR = RB == 0 ? 2 : 1;
    constexpr int NT = NQ * NR;                         // taps of the class
    constexpr int CG = 8 / NT;                          // col-groups per stage
    constexpr int STEPS = CG * NT;                      // (col-group, tap) steps per stage: 8
    constexpr int S = N / 2;                            // MFMA steps per (col-group, tap)
    constexpr int RW = STEPS * N;                       // floats of a staged row
    constexpr int AP = RW + 1;                          // LDS pitch of a staged row
    constexpr int CPR = RW / 64;                        // 64-float copies per row
    static_assert(RW % 64 == 0 && 32 % kBpWaves == 0, "whole copies, rows split over waves");
    __shared__ int32_t sFirst[kBpMaxG];
    __shared__ uint32_t sMask[kBpMaxG];
    __shared__ int32_t sGl[kBpMaxG];
    __shared__ int32_t sCnt[kBpWaves];
    __shared__ float sA[32 * AP];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    int32_t c0, p0;                                     // first input channel and pixel of the class
    dx_tile(a, c0, p0);

    // ---- Index prologue (as in the 3x3 kernel).
    const int32_t g = tid;
    bool any = false;
    const __amdgpu_buffer_rsrc_t rI = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(a.I), 0, __builtin_amdgcn_readfirstlane(a.t * 4), kRawBufferFlags);
    if (g < a.G) {
        int32_t zb, ze;
        group_range(a, g, zb, ze);
        const int32_t first = run_first(rI, zb, ze, c0);
        uint32_t mask = 0;
#pragma unroll
        for (int k = 0; k < 32; ++k) {
            const int32_t e = first + k;
            const int32_t c = e < ze ? int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, e * 4, 0, 0)) : INT32_MAX;
            if (c < c0 + 32 && c < a.m) mask |= 1u << (c - c0);
        }
        sFirst[g] = first;
        sMask[g] = mask;
        any = mask != 0;
    }
    const uint64_t bal = __ballot(any);
    if (lane == 0) sCnt[wave] = __builtin_popcountll(bal);
    __syncthreads();
    int32_t base = 0, ng = 0;
#pragma unroll
    for (int w = 0; w < kBpWaves; ++w) {
        base += w < wave ? sCnt[w] : 0;
        ng += sCnt[w];
    }
    if (any) sGl[base + __builtin_popcountll(bal & ((uint64_t(1) << lane) - 1))] = g;
    __syncthreads();

    // ---- Lane roles as in the 3x3 kernel; the lane's pixel is pixel p of
    // the class: (b, i, j) -> (ih, iw) = (2i + ca, 2j + cb).
    const int col = lane & 31, kk = lane >> 5;
    const int32_t HWo = a.HWo, HWi = a.H * a.W;
    const int32_t batch = a.npix / HWo;
    const int32_t hc = (a.H - ca + 1) / 2, wc = (a.W - cb + 1) / 2;   // the class's rows and columns
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(dy), 0, __builtin_amdgcn_readfirstlane(int32_t(int64_t(batch) * a.n * HWo * 4)),
        kRawBufferFlags);
    const uint32_t chb = uint32_t(HWo) * 4;
    const int32_t p = p0 + wave * 32 + col;
    int64_t xo = -1;
    uint32_t yk[NT];                          // per class tap: byte offset of dY at channel kk (or out of range)
    {
        const bool in = p < batch * hc * wc;
        const int32_t b = in ? p / (hc * wc) : 0, rem = p - b * hc * wc;
        const int32_t i = rem / wc, j = rem - i * wc;
        const int32_t ih = 2 * i + ca, iw = 2 * j + cb;
        if (in) xo = int64_t(b) * a.m * HWi + int64_t(ih) * a.W + iw;
        const int64_t ybase = int64_t(b) * a.n * HWo;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const int32_t q = QA + 2 * (t / NR), r = RB + 2 * (t % NR);
            const int32_t oh = (ih + a.ph - q) >> 1, ow = (iw + a.pw - r) >> 1;   // exact: the class's parity
            const bool ok = in && ih + a.ph - q >= 0 && iw + a.pw - r >= 0 && oh < a.Ho && ow < a.Wo;
            yk[t] = ok ? uint32_t((ybase + int64_t(oh) * a.Wo + ow) * 4) + uint32_t(kk) * chb : kBufferOutOfRange;
        }
    }
    auto load_b = [&](float (&bv)[S], int32_t gg, int t) __attribute__((always_inline)) {
        const int32_t ob = __builtin_amdgcn_readfirstlane(gg * N);
        if (ob + N <= a.n) {   // (uniform) every row exists: no per-step mask
#pragma unroll
            for (int s = 0; s < S; ++s)
                bv[s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rY, int32_t(yk[t]), int32_t(uint32_t(ob + 2 * s) * chb), 0));
        } else {
            const int32_t lim = a.n - ob - kk;
#pragma unroll
            for (int s = 0; s < S; ++s)
                bv[s] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rY, int32_t(2 * s < lim ? yk[t] : kBufferOutOfRange), int32_t(uint32_t(ob + 2 * s) * chb), 0));
        }
    };
    // Stage of col-groups sGl[j0 .. j0 + CG): row c, step k = slot * NT + t,
    // entry i holds D[z][i][tap t] for the block z where col-group
    // sGl[j0 + slot] keeps channel c0 + c (zero if none).  Copy u of a row
    // covers floats 64u .. 64u + 63.
    const v4i32 rD = buffer_rsrc(a.D, int32_t(int64_t(a.t) * N * 9 * 4));
    auto copy_a = [&](int32_t j0) __attribute__((always_inline)) {
#pragma unroll
        for (int u = 0; u < CPR; ++u) {
            const int32_t f = 64 * u + lane, step = f / N, i = f % N;
            const int32_t slot = step / NT, t = step % NT;
            const int32_t tap = (QA + 2 * (t / NR)) * 3 + RB + 2 * (t % NR);
            const int32_t jj = j0 + slot;
            const int32_t gg = jj < ng ? sGl[jj] : 0;
            const int32_t first = sFirst[gg];
            const uint32_t mask = jj < ng ? sMask[gg] : 0u;
#pragma unroll
            for (int rr = 0; rr < 32 / kBpWaves; ++rr) {
                const int32_t row = wave * (32 / kBpWaves) + rr;
                const bool kept = (mask >> row) & 1;
                const int32_t z = first + __builtin_popcount(mask & ((1u << row) - 1));
                copy4_to_lds(rD, (const lds_char*)(sA + row * AP + 64 * u),
                             kept ? ((z * N + i) * 9 + tap) * 4 : int32_t(kBufferOutOfRange), 0);
            }
        }
    };

    acc_t acc;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) acc[r] = 0.f;
    auto multiply = [&](int step, const float (&bv)[S]) __attribute__((always_inline)) {
        const float* ar = &sA[col * AP + step * N + kk];
#pragma unroll
        for (int s = 0; s < S; ++s) acc = M::step(ar[2 * s], bv[s], acc);
    };

    if (ng > 0) {
        float b0[S], b1[S];
        copy_a(0);
        load_b(b0, sGl[0], 0);
        vm_wait<0>();
        __syncthreads();
        // Step k of a stage (slot k / NT, tap k % NT) multiplies register set
        // k % 2 (eight steps per stage) and loads step k + 1's dY values.
        for (int32_t j0 = 0; j0 < ng; j0 += CG) {
            static_for<STEPS>([&](auto K) {
                constexpr int k = decltype(K)::value;
                constexpr int slot = k / NT, t = k % NT;
                float (&cur)[S] = (k & 1) ? b1 : b0;
                float (&nxt)[S] = (k & 1) ? b0 : b1;
                if (j0 + slot < ng) {
                    if (t + 1 < NT)
                        load_b(nxt, sGl[j0 + slot], t + 1 < NT ? t + 1 : 0);
                    else if (j0 + slot + 1 < ng)
                        load_b(nxt, sGl[j0 + slot + 1], 0);
                    multiply(k, cur);
                }
            });
            if (j0 + CG < ng) {
                __syncthreads();
                copy_a(j0 + CG);
                vm_wait<0>();
                __syncthreads();
            }
        }
    }

    if (xo >= 0) {
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) {
            const int32_t c = c0 + M::row(lane, r);
            if (c < a.m) store_out(&dx[xo + int64_t(c) * HWi], acc[r]);
        }
    }
}

}  // namespace

bool bwd_data_pw_applies(const ConvArgs& a, onexn_dtype wdt, onexn_dtype dxdt, int32_t batch) {
    if (wdt != ONEXN_F32 || dxdt != ONEXN_F32) return false;
    const bool pw = a.kh == 1 && a.kw == 1 && a.ph == 0 && a.pw == 0 &&                     // any stride,
                    (a.N == 2 || a.N == 4 || a.N == 8 || a.N == 16 || a.N == 32);        // N >= 2
    const bool k3 = a.kh == 3 && a.kw == 3 && a.sh == a.sw && (a.sh == 1 || a.sh == 2) &&   // any padding
                    (a.N == 8 || a.N == 16 || a.N == 32);
    if (!pw && !k3) return false;
    if (int64_t(a.t) * a.N * a.KK * 4 >= (int64_t(1) << 31)) return false;   // D through a buffer
    if (a.G > kBpMaxG) return false;
    if (int64_t(batch) * a.n * a.HWo * 4 >= (int64_t(1) << 31)) return false;   // 32-bit buffer offsets
    return true;
}

onexn_status launch_bwd_data_pw(const ConvArgs& a, const void* dy, void* dx, hipStream_t s) {
    // The 1x1 kernel walks the output pixels, the 3x3 one the input pixels.
    const bool k3 = a.kh == 3;
    const int64_t pix = k3 ? int64_t(a.npix / a.HWo) * a.H * a.W : int64_t(a.npix);
    const int64_t ptiles = (pix + kBpPix - 1) / kBpPix;
    const int64_t ctiles = (int64_t(a.m) + 31) / 32;
    if (ptiles * ctiles > INT32_MAX)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_bwd_data: grid out of range");
    const dim3 grid{uint32_t(ptiles * ctiles), 1, 1};
    const float* y = static_cast<const float*>(dy);
    float* x = static_cast<float*>(dx);
    if (!k3) {
        switch (a.N) {
            case 32: hipLaunchKernelGGL(bwd_data_pw<32>, grid, dim3(kBpThreads), 0, s, a, y, x); break;
            case 16: hipLaunchKernelGGL(bwd_data_pw<16>, grid, dim3(kBpThreads), 0, s, a, y, x); break;
            case 8: hipLaunchKernelGGL(bwd_data_pw<8>, grid, dim3(kBpThreads), 0, s, a, y, x); break;
            case 4: hipLaunchKernelGGL(bwd_data_pw<4>, grid, dim3(kBpThreads), 0, s, a, y, x); break;
            default: hipLaunchKernelGGL(bwd_data_pw<2>, grid, dim3(kBpThreads), 0, s, a, y, x); break;
        }
    } else if (a.sh == 1 || tuning(kTuneBwdKernel) == 2) {   // stride 2 here: all nine taps per pixel
        auto go = [&](auto k32, auto k16, auto k8) {
            if (a.N == 32) hipLaunchKernelGGL(k32, grid, dim3(kBpThreads), 0, s, a, y, x);
            else if (a.N == 16) hipLaunchKernelGGL(k16, grid, dim3(kBpThreads), 0, s, a, y, x);
            else hipLaunchKernelGGL(k8, grid, dim3(kBpThreads), 0, s, a, y, x);
        };
        if (a.sh == 1) go(bwd_data_k3<32, 1>, bwd_data_k3<16, 1>, bwd_data_k3<8, 1>);
        else go(bwd_data_k3<32, 2>, bwd_data_k3<16, 2>, bwd_data_k3<8, 2>);
    } else {
        // One launch per parity class: pixels (2i + ca, 2j + cb) take the taps
        // of parities ((ca + ph) % 2, (cb + pw) % 2).
        const int32_t batch = a.npix / a.HWo;
        for (int32_t ca = 0; ca < 2 && ca < a.H; ++ca)
            for (int32_t cb = 0; cb < 2 && cb < a.W; ++cb) {
                const int64_t cpix = int64_t(batch) * ((a.H - ca + 1) / 2) * ((a.W - cb + 1) / 2);
                const dim3 cgrid{uint32_t((cpix + kBpPix - 1) / kBpPix * ctiles), 1, 1};
                const int cls = ((ca + a.ph) & 1) << 1 | ((cb + a.pw) & 1);
                auto go = [&](auto k32, auto k16, auto k8) {
                    if (a.N == 32) hipLaunchKernelGGL(k32, cgrid, dim3(kBpThreads), 0, s, a, y, x, ca, cb);
                    else if (a.N == 16) hipLaunchKernelGGL(k16, cgrid, dim3(kBpThreads), 0, s, a, y, x, ca, cb);
                    else hipLaunchKernelGGL(k8, cgrid, dim3(kBpThreads), 0, s, a, y, x, ca, cb);
                };
                switch (cls) {
                    case 0: go(bwd_data_s2<32, 0, 0>, bwd_data_s2<16, 0, 0>, bwd_data_s2<8, 0, 0>); break;
                    case 1: go(bwd_data_s2<32, 0, 1>, bwd_data_s2<16, 0, 1>, bwd_data_s2<8, 0, 1>); break;
                    case 2: go(bwd_data_s2<32, 1, 0>, bwd_data_s2<16, 1, 0>, bwd_data_s2<8, 1, 0>); break;
                    default: go(bwd_data_s2<32, 1, 1>, bwd_data_s2<16, 1, 1>, bwd_data_s2<8, 1, 1>); break;
                }
                const hipError_t cerr = hipGetLastError();
                if (cerr != hipSuccess)
                    return fail(ONEXN_ERR_HIP, "conv2d_bwd_data: launch failed: %s", hipGetErrorString(cerr));
            }
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(ONEXN_ERR_HIP, "conv2d_bwd_data: launch failed: %s", hipGetErrorString(err));
    return ONEXN_OK;
}

}  // namespace onexn

// ---------------------------------------------------------------------------
// Weight gradient of the kept blocks on matrix cores: fp32, NCHW, N in
// {16, 32}, kernels of up to 63 taps, any stride and padding.
//
//     dD[z][i][q][r] = sum over output pixels of
//                      X[I[z]][oh*sh - ph + q][ow*sw - pw + r] * dY[gN + i][oh][ow]
//
// (Sec. 3.4's BSR layout, z a kept block of col-group g).  For a tile of N
// consecutive kept blocks of one col-group and one tap (q, r) this is an
// N x N contraction over the output pixels: rows = blocks, columns = block
// rows i, with v_mfma_f32_32x32x2f32 (N = 32) or v_mfma_f32_16x16x4f32
// (N = 16).  A workgroup of four waves stages 128-pixel chunks of the tile's
// N gathered input rows (at the tap's shifted positions, zero in the padding)
// and the col-group's N dY rows in LDS (coalesced along pixels, each thread
// one pixel; the next chunk's values are loaded into registers while this
// chunk is multiplied); each wave multiplies 32 of the chunk's pixels, and
// the four partial sums are added through LDS in wave order at the end.
// Layers with few (tile, tap) items split their pixels over several
// workgroups, whose sums are added into dD (zeroed first) with atomic adds:
// those layers' results can differ in the last bits from run to run; with
// one range per item (the default where items suffice) every element is
// stored once after a fixed-order accumulation.
// ---------------------------------------------------------------------------

namespace onexn {
namespace {

constexpr int kBwWaves = 4;
constexpr int kBwThreads = 64 * kBwWaves;
constexpr int kBwCh = 128;                     // pixels per staged chunk (one per thread and row pair)
constexpr int kBwPitch = kBwCh + 1;            // LDS row pitch (floats)

__global__ void __launch_bounds__(256) bw_zero(float* __restrict__ p, int64_t n) {
    for (int64_t i = int64_t(blockIdx.x) * 256 + threadIdx.x; i < n; i += int64_t(gridDim.x) * 256) p[i] = 0.f;
}

template <int N, bool KT>
__global__ void __launch_bounds__(kBwThreads) bwd_weight_pw(ConvArgs a, const float* __restrict__ x,
                                                             const float* __restrict__ dy,
                                                             float* __restrict__ dD, int32_t tiles_per_g,
                                                             int32_t nsplit) {
    typedef PwMfma<N> M;
    typedef typename M::acc_t acc_t;
    constexpr int KS = M::KS;                  // pixels per MFMA step
    constexpr int RPT = N * kBwCh / kBwThreads;   // rows per thread and operand (one pixel each)
    static_assert(kBwThreads % kBwCh == 0, "a thread keeps one pixel of every chunk");
    __shared__ float sX[N * kBwPitch];
    __shared__ float sY[N * kBwPitch];
    __shared__ float sR[kBwWaves][64 * M::ACC];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    // Work item: (col-group, tile of N (block, tap) pairs, pixel range).  The
    // col-group's pairs are numbered tap-major, pair = tap * cnt + k for its
    // k-th kept block, so a tile is N blocks of one tap where the col-group
    // keeps many, and several taps of its few blocks where it keeps few.
    const int32_t item = blockIdx.x;
    const int32_t split = item % nsplit;
    const int32_t gt = item / nsplit;
    const int32_t g = gt / tiles_per_g, tile = gt - g * tiles_per_g;
    int32_t zb, ze;
    group_range(a, g, zb, ze);
    const int32_t cnt = ze - zb, npairs = cnt * a.KK;
    const int32_t pr0 = tile * N;              // first pair of the tile
    if (pr0 >= npairs) return;                 // (uniform: the col-group has fewer tiles)
    const int32_t pb = int32_t(int64_t(a.npix) * split / nsplit);
    const int32_t pe = int32_t(int64_t(a.npix) * (split + 1) / nsplit);

    // This thread's pixel of each chunk and its rows (r0 + 2 j for N = 32, ...).
    const int px = tid % kBwCh, r0 = tid / kBwCh;
    constexpr int RS = kBwThreads / kBwCh;     // row stride between a thread's rows
    const int32_t HWo = a.HWo, HW = a.H * a.W;
    const int32_t batch = a.npix / HWo;
    const uint32_t chb = uint32_t(HWo) * 4, xchb = uint32_t(HW) * 4;   // channel strides of dY and X
    const __amdgpu_buffer_rsrc_t rX = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(x), 0, __builtin_amdgcn_readfirstlane(int32_t(int64_t(batch) * a.m * HW * 4)),
        kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(dy), 0, __builtin_amdgcn_readfirstlane(int32_t(int64_t(batch) * a.n * HWo * 4)),
        kRawBufferFlags);
    // Per row of the thread: the pair's input channel (bytes) and tap, and
    // the col-group's output channel (bytes); a pair past the col-group's, a
    // channel outside [0, m) or a row past n reads zeros.
    uint32_t xr[RPT], yr[RPT];
    int32_t tq[RPT];                           // row's tap index (KT), 63 for no pair
    uint32_t valid = 0;                        // bit j: row j is a pair with a channel in [0, m)
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
        const int32_t r = r0 + RS * j;
        const int32_t pr = pr0 + r;
        const int32_t tap = pr < npairs ? pr / cnt : 0;
        const int32_t c = pr < npairs ? a.I[zb + pr - tap * cnt] : -1;
        const bool ok = uint32_t(c) < uint32_t(a.m);
        // (KT: the channel's byte offset plus the tap's shift (q*W + r)*4.)
        const int32_t q = tap / a.kw;
        xr[j] = ok ? uint32_t(c) * xchb + (KT ? uint32_t(q * a.W + tap - q * a.kw) * 4 : 0u) : 0u;
        tq[j] = ok ? tap : 63;
        valid |= uint32_t(ok) << j;
        const int32_t o = g * N + r;
        yr[j] = o < a.n ? uint32_t(o) * chb : kBufferOutOfRange;
    }
    // A 1x1 layer (KT false) has the one tap (0, 0): one bounds check per
    // pixel.  Otherwise the pixel's taps that land inside the image form a
    // bit mask (kh + kw compares), and a row tests its tap's bit.
    float vx[RPT], vy[RPT];
    auto load = [&](int32_t p0) __attribute__((always_inline)) {
        const int32_t p = p0 + px;
        const bool in = p < pe;
        // Output pixel p; under row j's tap (q, r) it reads input pixel
        // (oh*sh - ph + q, ow*sw - pw + r), zero outside the image (padding).
        const int32_t b = in ? p / HWo : 0, hw = p - b * HWo;
        const int32_t oh = hw / a.Wo, ow = hw - oh * a.Wo;
        const int32_t ih0 = oh * a.sh - a.ph, iw0 = ow * a.sw - a.pw;
        const uint32_t bx = uint32_t((int64_t(b) * a.m * HW + int64_t(ih0) * a.W + iw0) * 4);
        const uint32_t by = in ? uint32_t((int64_t(b) * a.n * HWo + hw) * 4) : kBufferOutOfRange;
        if (!KT) {
            const bool okp = in && uint32_t(ih0) < uint32_t(a.H) && uint32_t(iw0) < uint32_t(a.W);
#pragma unroll
            for (int j = 0; j < RPT; ++j) {
                const bool ok = okp && ((valid >> j) & 1);
                vx[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rX, int32_t(ok ? bx + xr[j] : kBufferOutOfRange), 0, 0));
                vy[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rY, int32_t(by + yr[j]), 0, 0));
            }
        } else {
            // Bit q*kw + r: tap (q, r) reads inside the image (kh * kw <= 63).
            uint64_t cm = 0, mask = 0;
            for (int32_t r = 0; r < a.kw; ++r) cm |= uint64_t(uint32_t(iw0 + r) < uint32_t(a.W)) << r;
            for (int32_t q = 0; q < a.kh; ++q)
                mask |= uint32_t(ih0 + q) < uint32_t(a.H) ? cm << (q * a.kw) : 0;
            mask = in ? mask : 0;
#pragma unroll
            for (int j = 0; j < RPT; ++j) {
                const bool ok = (mask >> tq[j]) & 1;
                vx[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rX, int32_t(ok ? bx + xr[j] : kBufferOutOfRange), 0, 0));
                vy[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rY, int32_t(by + yr[j]), 0, 0));
            }
        }
    };
    auto put = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            sX[(r0 + RS * j) * kBwPitch + px] = vx[j];
            sY[(r0 + RS * j) * kBwPitch + px] = vy[j];
        }
    };

    acc_t acc;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) acc[r] = 0.f;
    // Lane roles: A (block row lane % N, pixel k = lane / N of a step), B
    // (column lane % N, same k).
    const int rc = lane % N, k = lane / N;
    const float* ax = sX + rc * kBwPitch + wave * 32 + k;
    const float* by = sY + rc * kBwPitch + wave * 32 + k;

    if (pb < pe) {
        load(pb);
        for (int32_t p0 = pb; p0 < pe; p0 += kBwCh) {
            __syncthreads();   // the previous chunk's reads are done
            put();
            __syncthreads();
            if (p0 + kBwCh < pe) load(p0 + kBwCh);
#pragma unroll
            for (int st = 0; st < 32 / KS; ++st) acc = M::step(ax[st * KS], by[st * KS], acc);
        }
    }

    // The four waves' partial sums, added in wave order by wave 0.
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) sR[wave][r * 64 + lane] = acc[r];
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r)
        acc[r] = ((sR[0][r * 64 + lane] + sR[1][r * 64 + lane]) + sR[2][r * 64 + lane]) + sR[3][r * 64 + lane];
    // MFMA (row, col): pair pr0 + row (block zb + k, tap), block row col.
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) {
        const int32_t pr = pr0 + M::row(lane, r);
        if (pr >= npairs) continue;
        const int32_t tap = pr / cnt;
        float* dst = dD + (int64_t(zb + pr - tap * cnt) * N + rc) * a.KK + tap;
        if (nsplit > 1) unsafeAtomicAdd(dst, acc[r]);
        else *dst = acc[r];
    }
}


// 1x1 stride-1 unpadded layers whose images hold a multiple of 4 pixels: the
// same work items, with the chunk staged four pixels at a time.  A thread
// loads a 16-byte quad of pixels of RPT rows of each operand (one
// buffer_load_dwordx4 per row, a quad never crossing an image) and writes it
// with one 16-byte LDS store; rows sit at a 16-byte-aligned pitch.  An MFMA
// step's pixel k of lane group k is pixel k * 32/KS + s of the wave's 32, so
// a lane reads its row's 32/KS consecutive pixels with 16-byte LDS reads.
// Against one pixel per thread and access: a quarter of the loads, LDS
// stores and LDS reads per MFMA.
constexpr int kBqPitch = kBwCh + 4;            // LDS row pitch (floats): rows 16-byte aligned

template <int N>
__global__ void __launch_bounds__(kBwThreads) bwd_weight_q4(ConvArgs a, const float* __restrict__ x,
                                                             const float* __restrict__ dy,
                                                             float* __restrict__ dD, int32_t tiles_per_g,
                                                             int32_t nsplit) {
    typedef PwMfma<N> M;
    typedef typename M::acc_t acc_t;
    constexpr int KS = M::KS;                  // lane groups = pixels per MFMA step
    constexpr int P = kBqPitch;
    constexpr int QPR = kBwCh / 4;             // pixel quads per chunk row
    constexpr int RG = kBwThreads / QPR;       // row groups
    constexpr int RPT = N / RG;                // rows per thread and operand
    constexpr int PPL = 32 / KS;               // consecutive pixels a lane reads per chunk
    static_assert(kBwThreads % QPR == 0 && N % RG == 0 && PPL % 4 == 0, "quad staging");
    __shared__ __attribute__((aligned(16))) float sX[N * P];
    __shared__ __attribute__((aligned(16))) float sY[N * P];
    __shared__ float sR[kBwWaves][64 * M::ACC];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t item = blockIdx.x;
    const int32_t split = item % nsplit;
    const int32_t gt = item / nsplit;
    const int32_t g = gt / tiles_per_g, tile = gt - g * tiles_per_g;
    int32_t zb, ze;
    group_range(a, g, zb, ze);
    const int32_t e0 = zb + tile * N;          // first block of the tile (one tap)
    if (e0 >= ze) return;
    // Pixel range, cut at multiples of 4 (npix is one).
    const int32_t pb = int32_t(int64_t(a.npix) * split / nsplit) & ~3;
    const int32_t pe = split + 1 == nsplit ? a.npix : int32_t(int64_t(a.npix) * (split + 1) / nsplit) & ~3;

    const int pq = tid % QPR, rg = tid / QPR;  // this thread's quad and row group
    const int32_t HWo = a.HWo;
    const int32_t batch = a.npix / HWo;
    const uint32_t chb = uint32_t(HWo) * 4;    // channel stride of both X and dY (stride 1, no padding)
    const __amdgpu_buffer_rsrc_t rX = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(x), 0, __builtin_amdgcn_readfirstlane(int32_t(int64_t(batch) * a.m * HWo * 4)),
        kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(dy), 0, __builtin_amdgcn_readfirstlane(int32_t(int64_t(batch) * a.n * HWo * 4)),
        kRawBufferFlags);
    uint32_t xr[RPT], yr[RPT];                 // row offsets (bytes), or out of range
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
        const int32_t r = rg + RG * j;
        const int32_t e = e0 + r;
        const int32_t c = e < ze ? a.I[e] : -1;
        xr[j] = uint32_t(c) < uint32_t(a.m) ? uint32_t(c) * chb : kBufferOutOfRange;
        const int32_t o = g * N + r;
        yr[j] = o < a.n ? uint32_t(o) * chb : kBufferOutOfRange;
    }
    f32x4 vx[RPT], vy[RPT];
    auto load = [&](int32_t p0) __attribute__((always_inline)) {
        const int32_t p = p0 + 4 * pq;
        const bool in = p < pe;
        const int32_t b = in ? p / HWo : 0, hw = p - b * HWo;
        const uint32_t bx = uint32_t((int64_t(b) * a.m * HWo + hw) * 4);
        const uint32_t by = uint32_t((int64_t(b) * a.n * HWo + hw) * 4);
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            const bool okx = in && xr[j] != kBufferOutOfRange, oky = in && yr[j] != kBufferOutOfRange;
            vx[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                rX, int32_t(okx ? bx + xr[j] : kBufferOutOfRange), 0, 0));
            vy[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(
                rY, int32_t(oky ? by + yr[j] : kBufferOutOfRange), 0, 0));
        }
    };
    auto put = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            *reinterpret_cast<f32x4*>(&sX[(rg + RG * j) * P + 4 * pq]) = vx[j];
            *reinterpret_cast<f32x4*>(&sY[(rg + RG * j) * P + 4 * pq]) = vy[j];
        }
    };

    acc_t acc;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) acc[r] = 0.f;
    const int rc = lane % N, k = lane / N;
    const float* ax = sX + rc * P + wave * 32 + k * PPL;
    const float* ay = sY + rc * P + wave * 32 + k * PPL;

    if (pb < pe) {
        load(pb);
        for (int32_t p0 = pb; p0 < pe; p0 += kBwCh) {
            __syncthreads();   // the previous chunk's reads are done
            put();
            __syncthreads();
            if (p0 + kBwCh < pe) load(p0 + kBwCh);
#pragma unroll
            for (int v = 0; v < PPL / 4; ++v) {
                const f32x4 av = *reinterpret_cast<const f32x4*>(ax + 4 * v);
                const f32x4 bv = *reinterpret_cast<const f32x4*>(ay + 4 * v);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc = M::step(av[e], bv[e], acc);
            }
        }
    }

#pragma unroll
    for (int r = 0; r < M::ACC; ++r) sR[wave][r * 64 + lane] = acc[r];
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r)
        acc[r] = ((sR[0][r * 64 + lane] + sR[1][r * 64 + lane]) + sR[2][r * 64 + lane]) + sR[3][r * 64 + lane];
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) {
        const int32_t e = e0 + M::row(lane, r);
        if (e >= ze) continue;
        float* dst = dD + int64_t(e) * N + rc;
        if (nsplit > 1) unsafeAtomicAdd(dst, acc[r]);
        else *dst = acc[r];
    }
}


// Weight gradient at N <= 8, where an N x N tile would leave the matrix
// cores mostly idle: for each tap (q, r) the dense product
//     G[c][o] = sum over output pixels of X[c][oh*sh - ph + q][ow*sw - pw + r] * dY[o][oh][ow]
// of a tile of 32 input channels and 32 output channels (32/N col-groups)
// on v_mfma_f32_32x32x2f32, of which only the entries of kept blocks are
// stored: dD[z][i][q][r] = G[I[z]][gN + i] (at p = 0.5 half the tile's work
// is for pruned blocks).  Items are (channel tile, tap, output-channel tile,
// pixel range); a prologue finds each of the tile's col-groups' kept blocks among
// the 32 channels (first block and channel mask, as in the input
// gradient), and a tile that holds none returns.  Chunks of 128 pixels are
// staged as in bwd_weight_q4 (Q = 4: 16-byte pixel quads, 1x1 stride-1
// unpadded layers with images of a multiple of 4 pixels) or one pixel per
// access (Q = 1, any kernel, stride and padding); four waves split a
// chunk's pixels and add their sums in wave order.  Each dD entry belongs to
// one tile: stored once, or added with atomics when pixel ranges split.
template <int N, int Q>
__global__ void __launch_bounds__(kBwThreads) bwd_weight_dense(ConvArgs a, const float* __restrict__ x,
                                                                const float* __restrict__ dy,
                                                                float* __restrict__ dD, int32_t otiles,
                                                                int32_t nsplit) {
    typedef PwMfma<32> M;
    typedef typename M::acc_t acc_t;
    constexpr int GPT = 32 / N;                // col-groups per output-channel tile
    constexpr int P = kBqPitch;
    constexpr int QPR = kBwCh / Q;             // pixel groups per chunk row
    constexpr int RG = kBwThreads / QPR;       // row groups
    constexpr int RPT = 32 / RG;               // rows per thread and operand
    constexpr int PPL = 16;                    // consecutive pixels a lane reads per chunk
    typedef typename std::conditional<Q == 4, f32x4, float>::type vq_t;
    static_assert(N <= 8 && 32 % N == 0 && kBwThreads % QPR == 0 && 32 % RG == 0, "tile shape");
    __shared__ __attribute__((aligned(16))) float sX[32 * P];
    __shared__ __attribute__((aligned(16))) float sY[32 * P];
    __shared__ float sR[kBwWaves][64 * M::ACC];
    __shared__ int32_t sFirst[GPT];
    __shared__ uint32_t sMask[GPT];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t item = blockIdx.x;
    const int32_t split = item % nsplit, tt = item / nsplit;
    const int32_t ot = tt % otiles, ctap = tt / otiles;
    const int32_t tap = ctap % a.KK, ct = ctap / a.KK;
    const int32_t tq = tap / a.kw, tr = tap - tq * a.kw;   // the tile's tap (q, r)
    const int32_t c0 = ct * 32, o0 = ot * 32, g0 = o0 / N;

    // ---- The tile's col-groups' kept blocks among channels [c0, c0 + 32).
    if (tid < GPT) {
        const int32_t g = g0 + tid;
        uint32_t mask = 0;
        int32_t first = 0;
        if (g < a.G) {
            const __amdgpu_buffer_rsrc_t rI = __builtin_amdgcn_make_buffer_rsrc(
                const_cast<int32_t*>(a.I), 0, a.t * 4, kRawBufferFlags);
            int32_t zb, ze;
            group_range(a, g, zb, ze);
            first = run_first(rI, zb, ze, c0);
            for (int k = 0; k < 32; ++k) {
                const int32_t e = first + k;
                const int32_t c = e < ze ? int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, e * 4, 0, 0)) : INT32_MAX;
                if (c < c0 + 32 && c < a.m) mask |= 1u << (c - c0);
            }
        }
        sFirst[tid] = first;
        sMask[tid] = mask;
    }
    __syncthreads();
    uint32_t anyk = 0;
#pragma unroll
    for (int j = 0; j < GPT; ++j) anyk |= sMask[j];
    if (anyk == 0) return;                     // (uniform) no kept block in the tile

    const int32_t pb = int32_t(int64_t(a.npix) * split / nsplit) & ~(Q - 1);
    const int32_t pe = split + 1 == nsplit ? a.npix : int32_t(int64_t(a.npix) * (split + 1) / nsplit) & ~(Q - 1);
    const int pq = tid % QPR, rg = tid / QPR;
    const int32_t HWo = a.HWo, HW = a.H * a.W;
    const int32_t batch = a.npix / HWo;
    const uint32_t chb = uint32_t(HWo) * 4, xchb = uint32_t(HW) * 4;   // channel strides of dY and X
    const __amdgpu_buffer_rsrc_t rX = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(x), 0, __builtin_amdgcn_readfirstlane(int32_t(int64_t(batch) * a.m * HW * 4)),
        kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(dy), 0, __builtin_amdgcn_readfirstlane(int32_t(int64_t(batch) * a.n * HWo * 4)),
        kRawBufferFlags);
    uint32_t xr[RPT], yr[RPT];                 // row offsets (bytes), or out of range
#pragma unroll
    for (int j = 0; j < RPT; ++j) {
        const int32_t r = rg + RG * j;
        xr[j] = c0 + r < a.m ? uint32_t(c0 + r) * xchb : kBufferOutOfRange;
        yr[j] = o0 + r < a.n ? uint32_t(o0 + r) * chb : kBufferOutOfRange;
    }
    vq_t vx[RPT], vy[RPT];
    auto load = [&](int32_t p0) __attribute__((always_inline)) {
        const int32_t p = p0 + Q * pq;
        const bool pin = p < pe;
        const int32_t b = pin ? p / HWo : 0, hw = p - b * HWo;
        // Output pixel p reads input pixel (oh*sh - ph + q, ow*sw - pw + r)
        // under the tile's tap, zero outside the image (pixel quads: 1x1
        // stride 1 unpadded only, where that is pixel hw itself).
        const int32_t oh = hw / a.Wo, ow = hw - oh * a.Wo;
        const int32_t ih = oh * a.sh - a.ph + tq, iw = ow * a.sw - a.pw + tr;
        const bool in = pin && uint32_t(ih) < uint32_t(a.H) && uint32_t(iw) < uint32_t(a.W);
        const uint32_t bx = uint32_t((int64_t(b) * a.m * HW + int64_t(ih) * a.W + iw) * 4);
        const uint32_t by = uint32_t((int64_t(b) * a.n * HWo + hw) * 4);
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            const bool okx = in && xr[j] != kBufferOutOfRange, oky = pin && yr[j] != kBufferOutOfRange;
            const int32_t ox = int32_t(okx ? bx + xr[j] : kBufferOutOfRange);
            const int32_t oy = int32_t(oky ? by + yr[j] : kBufferOutOfRange);
            if constexpr (Q == 4) {
                vx[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rX, ox, 0, 0));
                vy[j] = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rY, oy, 0, 0));
            } else {
                vx[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rX, ox, 0, 0));
                vy[j] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rY, oy, 0, 0));
            }
        }
    };
    auto put = [&]() __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < RPT; ++j) {
            *reinterpret_cast<vq_t*>(&sX[(rg + RG * j) * P + Q * pq]) = vx[j];
            *reinterpret_cast<vq_t*>(&sY[(rg + RG * j) * P + Q * pq]) = vy[j];
        }
    };

    acc_t acc;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) acc[r] = 0.f;
    // Lane (row rc, group k): step s takes pixel k * 16 + s of the wave's 32.
    const int rc = lane & 31, k = lane >> 5;
    const float* ax = sX + rc * P + wave * 32 + k * PPL;
    const float* ay = sY + rc * P + wave * 32 + k * PPL;
    if (pb < pe) {
        load(pb);
        for (int32_t p0 = pb; p0 < pe; p0 += kBwCh) {
            __syncthreads();   // the previous chunk's reads are done
            put();
            __syncthreads();
            if (p0 + kBwCh < pe) load(p0 + kBwCh);
#pragma unroll
            for (int v = 0; v < PPL / 4; ++v) {
                const f32x4 av = *reinterpret_cast<const f32x4*>(ax + 4 * v);
                const f32x4 bv = *reinterpret_cast<const f32x4*>(ay + 4 * v);
#pragma unroll
                for (int e = 0; e < 4; ++e) acc = M::step(av[e], bv[e], acc);
            }
        }
    }

#pragma unroll
    for (int r = 0; r < M::ACC; ++r) sR[wave][r * 64 + lane] = acc[r];
    __syncthreads();
    if (wave != 0) return;
#pragma unroll
    for (int r = 0; r < M::ACC; ++r)
        acc[r] = ((sR[0][r * 64 + lane] + sR[1][r * 64 + lane]) + sR[2][r * 64 + lane]) + sR[3][r * 64 + lane];
    // MFMA (row, col) = (input channel c0 + row, output channel o0 + col):
    // stored where col-group (o0 + col) / N keeps the channel.
    const int32_t oc = rc;                     // column within the tile
    const int gs = oc / N, i = oc % N;         // col-group slot and block row
    const uint32_t mask = sMask[gs];
    const int32_t first = sFirst[gs];
#pragma unroll
    for (int r = 0; r < M::ACC; ++r) {
        const int row = M::row(lane, r);
        if (!((mask >> row) & 1)) continue;
        const int32_t z = first + __builtin_popcount(mask & ((1u << row) - 1));
        float* dst = dD + (int64_t(z) * N + i) * a.KK + tap;
        if (nsplit > 1) unsafeAtomicAdd(dst, acc[r]);
        else *dst = acc[r];
    }
}

}  // namespace

// Layers at N = 2, 4, 8: the dense-product kernel.
static bool dense_dd(const ConvArgs& a) { return a.N == 2 || a.N == 4 || a.N == 8; }

bool bwd_weight_pw_applies(const ConvArgs& a, onexn_dtype xdt, int32_t batch) {
    if (xdt != ONEXN_F32) return false;
    if (a.N != 16 && a.N != 32 && !dense_dd(a)) return false;
    if (a.KK > 63) return false;   // one bit per tap, 63 meaning "no pair"
    if (int64_t(batch) * a.n * a.HWo * 4 >= (int64_t(1) << 31) ||
        int64_t(batch) * a.m * a.H * a.W * 4 >= (int64_t(1) << 31))
        return false;   // 32-bit buffer offsets
    return true;
}

static onexn_status launch_bwd_weight_dense(const ConvArgs& a, const void* x, const void* dy, float* dD,
                                           hipStream_t s) {
    const int64_t ctiles = (int64_t(a.m) + 31) / 32, otiles = (int64_t(a.n) + 31) / 32;
    const int64_t tiles = ctiles * a.KK * otiles;
    int64_t nsplit = (4 * int64_t(device_cu_count()) + tiles - 1) / tiles;
    nsplit = std::max<int64_t>(1, std::min<int64_t>(nsplit, a.npix / 1024));
    if (tuning(kTuneBwdSplit) >= 1) nsplit = tuning(kTuneBwdSplit);
    const int64_t grid = tiles * nsplit;
    if (grid < 1 || grid > INT32_MAX) return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_bwd_weight: grid out of range");
    if (nsplit > 1) {
        const int64_t n = int64_t(a.t) * a.N * a.KK;
        hipLaunchKernelGGL(bw_zero, dim3(uint32_t(std::min<int64_t>((n + 255) / 256, 4096))), dim3(256), 0, s, dD, n);
        const hipError_t zerr = hipGetLastError();
        if (zerr != hipSuccess)
            return fail(ONEXN_ERR_HIP, "conv2d_bwd_weight: launch failed: %s", hipGetErrorString(zerr));
    }
    const bool quads = a.KK == 1 && a.sh == 1 && a.sw == 1 && a.ph == 0 && a.pw == 0 && a.HWo % 4 == 0 &&
                       tuning(kTuneBwdKernel) != 3 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 &&
                       (reinterpret_cast<uintptr_t>(dy) & 15) == 0;
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(uint32_t(grid)), dim3(kBwThreads), 0, s, a, static_cast<const float*>(x),
                           static_cast<const float*>(dy), dD, int32_t(otiles), int32_t(nsplit));
    };
    switch (a.N) {
        case 8: quads ? go(bwd_weight_dense<8, 4>) : go(bwd_weight_dense<8, 1>); break;
        case 4: quads ? go(bwd_weight_dense<4, 4>) : go(bwd_weight_dense<4, 1>); break;
        default: quads ? go(bwd_weight_dense<2, 4>) : go(bwd_weight_dense<2, 1>); break;
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(ONEXN_ERR_HIP, "conv2d_bwd_weight: launch failed: %s", hipGetErrorString(err));
    return ONEXN_OK;
}

onexn_status launch_bwd_weight_pw(const ConvArgs& a, const void* x, const void* dy, float* dD, hipStream_t s) {
    if (dense_dd(a)) return launch_bwd_weight_dense(a, x, dy, dD, s);
    // A col-group keeps at most m blocks: m * KK pairs.
    const int64_t tiles_per_g = (int64_t(a.m) * a.KK + a.N - 1) / a.N;
    const int64_t tiles = (int64_t(a.t) * a.KK + a.N - 1) / a.N + a.G;   // tiles with pairs, at most
    // Pixel ranges per tile: enough workgroups for four per CU, each range
    // at least 1024 pixels; one range where the tiles suffice (stored, not added).
    int64_t nsplit = (4 * int64_t(device_cu_count()) + tiles - 1) / tiles;
    nsplit = std::max<int64_t>(1, std::min<int64_t>(nsplit, a.npix / 1024));
    if (tuning(kTuneBwdSplit) >= 1) nsplit = tuning(kTuneBwdSplit);
    const int64_t grid = int64_t(a.G) * tiles_per_g * nsplit;
    if (grid < 1 || grid > INT32_MAX)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_bwd_weight: grid out of range");
    if (nsplit > 1) {
        const int64_t n = int64_t(a.t) * a.N * a.KK;
        hipLaunchKernelGGL(bw_zero, dim3(uint32_t(std::min<int64_t>((n + 255) / 256, 4096))), dim3(256), 0, s, dD, n);
        const hipError_t zerr = hipGetLastError();
        if (zerr != hipSuccess)
            return fail(ONEXN_ERR_HIP, "conv2d_bwd_weight: launch failed: %s", hipGetErrorString(zerr));
    }
    // (A 1x1 layer's tiles all lie within its one tap: no per-row shifts.)
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(uint32_t(grid)), dim3(kBwThreads), 0, s, a, static_cast<const float*>(x),
                           static_cast<const float*>(dy), dD, int32_t(tiles_per_g), int32_t(nsplit));
    };
    // 1x1 stride-1 unpadded layers with whole pixel quads per image: quads.
    const bool quads = a.KK == 1 && a.sh == 1 && a.sw == 1 && a.ph == 0 && a.pw == 0 && a.HWo % 4 == 0 &&
                       tuning(kTuneBwdKernel) != 3 && (reinterpret_cast<uintptr_t>(x) & 15) == 0 && (reinterpret_cast<uintptr_t>(dy) & 15) == 0 &&
                       tuning(kTuneBwdKernel) != 3;
    if (a.N == 32) {
        if (quads) go(bwd_weight_q4<32>);
        else if (a.KK > 1) go(bwd_weight_pw<32, true>);
        else go(bwd_weight_pw<32, false>);
    } else {
        if (quads) go(bwd_weight_q4<16>);
        else if (a.KK > 1) go(bwd_weight_pw<16, true>);
        else go(bwd_weight_pw<16, false>);
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(ONEXN_ERR_HIP, "conv2d_bwd_weight: launch failed: %s", hipGetErrorString(err));
    return ONEXN_OK;
}

}  // namespace onexn
