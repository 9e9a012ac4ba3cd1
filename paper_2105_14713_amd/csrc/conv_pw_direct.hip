// 1x1 1xN-pruned convolution (any stride and padding), fp32, NCHW,
// N in {16, 32}, with both matrix-core operands loaded straight from global
// memory into registers.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the contraction
//     Y_g[N][pixels] = D_g^T[N][kept_g] * X[I_g][pixels].
//
// Operand layout.  An fp32 MFMA lane holds one contraction entry of one row
// (A) or one column (B):
//   N = 32, v_mfma_f32_32x32x2f32: lane l holds A[row l % 32][entry l / 32],
//     i.e. D[z + l / 32][l % 32] -- the two kept blocks' 64 weights are one
//     contiguous 256-byte run of D -- and B[entry l / 32][pixel l % 32], i.e.
//     input channel I[z + l / 32] at the lane's pixel: 32 consecutive pixels
//     of one gathered input row per half-wave.
//   N = 16, v_mfma_f32_16x16x4f32: the same with four blocks and 16 pixels.
// So neither operand needs a transposition or an LDS staging buffer: each
// step is one weight load and one input load per column block, all
// coalesced, and the input offset of a pixel (stride and padding included)
// is computed once.
//
// Work split.  A unit is (col-group, NB column blocks of pixels).  A
// workgroup of four waves takes 4 / KSPLIT units; KSPLIT waves share a unit's
// kept blocks (contiguous ranges) and add their partial sums through LDS at
// the end, for layers with few pixels and long col-groups.
//
// Pipelining.  Steps are taken in batches of kDB: channel indices come in
// lane-parallel windows of 64 entries loaded a window ahead, a batch's
// weight and input loads are all issued before the previous batch's MFMAs,
// so a wave keeps two batches of loads in flight.  Entries past the wave's
// range and channels outside [0, m) read zeros (out-of-range buffer offsets),
// so they add nothing.

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kDThreads = 256;
// kDB: MFMA steps per batch (8 for long contractions, 2 for short ones,
// whose waves would otherwise multiply mostly zero padding).
template <int N, int NB, int KSPLIT, int kDB, bool kEp>
__global__ void __launch_bounds__(kDThreads) pw_direct(ConvArgs a) {
    typedef PwMfma<N> M;
    typedef typename M::acc_t acc_t;
    constexpr int KS = M::KS, COLS = M::COLS;
    constexpr int UPW = 4 / KSPLIT;                 // units per workgroup
    constexpr int RED = KSPLIT > 1 ? 4 * NB * M::ACC * 64 : 1;
    __shared__ float sR[RED];
    // Fused epilogue: scale and bias of each unit's N channels, staged when
    // the unit starts and read back run by run at the store.
    __shared__ __attribute__((aligned(16))) float sEp[kEp ? 4 * 2 * N : 4];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int uw = wave / KSPLIT, kq = wave % KSPLIT;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    // Units are numbered pixel-block-major, col-group-minor, so the
    // workgroups sharing a pixel range run on one XCD (and its L2).
    const int32_t unit = L * UPW + uw;
    const int32_t pblocks = (a.npix + NB * COLS - 1) / (NB * COLS);
    const int32_t g = unit % a.G, pb = unit / a.G;
    const bool live = pb < pblocks;
    int32_t zb = 0, ze = 0;
    if (live) group_range(a, g, zb, ze);
    if constexpr (kEp) {
        if (kq == 0 && lane < N) {
            const int32_t o = g * N + lane;
            sEp[uw * 2 * N + lane] = o < a.n && a.ep_scale ? a.ep_scale[o] : 1.f;
            sEp[uw * 2 * N + N + lane] = o < a.n && a.ep_bias ? a.ep_bias[o] : 0.f;
        }
    }
    const int32_t per = (ze - zb + KSPLIT - 1) / KSPLIT;
    const int32_t z0 = min(ze, zb + kq * per), z1 = min(ze, z0 + per);

    const int32_t batch = a.npix / a.HWo;
    const uint32_t xbytes = uint32_t(int64_t(batch) * a.x_img * 4);
    const int col = lane % COLS, kk = lane / COLS;   // lane's pixel column and entry within a step

    // Byte offset of the lane's input pixel (channel 0) in each column block,
    // or xbytes where there is none (past the last pixel, or in the padding).
    uint32_t xo[NB];
    int64_t yo[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int32_t p = (pb * NB + nb) * COLS + col;
        xo[nb] = kBufferOutOfRange;
        yo[nb] = -1;
        if (live && p < a.npix) {
            const int32_t b = p / a.HWo, hw = p - b * a.HWo;
            const int32_t oh = hw / a.Wo, ow = hw - oh * a.Wo;
            const int32_t ih = oh * a.sh - a.ph, iw = ow * a.sw - a.pw;
            if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
                xo[nb] = uint32_t((int64_t(b) * a.x_img + int64_t(ih) * a.W + iw) * 4);
            yo[nb] = int64_t(b) * a.y_img + hw;
        }
    }

    // The sizes are wave-uniform; saying so (readfirstlane) keeps the buffer
    // resources in scalar registers -- a resource the compiler must treat as
    // divergent turns every load into a loop over the distinct values.
    const __amdgpu_buffer_rsrc_t rX = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.x), 0, __builtin_amdgcn_readfirstlane(int32_t(xbytes)), kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rD = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.D), 0, __builtin_amdgcn_readfirstlane(z1 * N * 4), kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rI = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(a.I), 0, __builtin_amdgcn_readfirstlane(z1 * 4), kRawBufferFlags);
    const uint32_t chb = uint32_t(a.x_c) * 4;   // bytes between input channels

    acc_t acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) acc[nb][r] = 0.f;

    // A batch is kDB steps = E entries.  Its channel indices (lane j: entry
    // z + j) are loaded two batches ahead and turned into the byte offset of
    // each entry's input channel -- kBufferOutOfRange for an entry at or past
    // z1 or a channel outside [0, m), which reads zeros.  A step then costs
    // one lane shuffle of that offset and one add per column block besides
    // its loads: the matrix pipe of a SIMD idles while other waves issue, so
    // every instruction per MFMA counts.  The two batches in flight live in
    // register slots with compile-time indices and the loop body is
    // straight-line (scheduling barriers keep each batch's loads in order);
    // otherwise the compiler copies batches and accumulators between
    // registers on every trip and waits for all loads at the loop head.
    constexpr int E = kDB * KS;   // entries per batch
    static_assert(E <= 64, "a batch's indices fit one wave");
    float av[2][kDB], bv[2][kDB][NB];
    int32_t idx[2];
    auto load_idx = [&](int32_t z) { return int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, (z + lane) * 4, 0, 0)); };
    auto issue = [&](int sl, int32_t z) __attribute__((always_inline)) {
        const bool ok = (z + lane < z1) & (uint32_t(idx[sl]) < uint32_t(a.m));
        const uint32_t cw = ok ? uint32_t(idx[sl]) * chb : kBufferOutOfRange;
        idx[sl] = load_idx(z + 2 * E);
        uint32_t co[kDB];
#pragma unroll
        for (int st = 0; st < kDB; ++st)
            co[st] = uint32_t(__builtin_amdgcn_ds_bpermute(4 * (st * KS + kk), int32_t(cw)));
#pragma unroll
        for (int st = 0; st < kDB; ++st) {
            av[sl][st] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                rD, ((z + st * KS) * N + lane) * 4, 0, 0));
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)   // both terms below 2^31: no wrap, out of range stays out
                bv[sl][st][nb] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rX, int32_t(xo[nb] + co[st]), 0, 0));
        }
    };
    auto consume = [&](int sl) __attribute__((always_inline)) {
#pragma unroll
        for (int st = 0; st < kDB; ++st)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[nb] = M::step(av[sl][st], bv[sl][st][nb], acc[nb]);
    };

    // Batches in pairs, each issued one batch ahead of its MFMAs.  An odd
    // count runs one batch of zeros (past the end everything reads zero): a
    // separate tail would merge with the loop body and bring the copies back.
    const int32_t nbat = (z1 - z0 + E - 1) / E;
    if (nbat > 0) {
        idx[0] = load_idx(z0);
        idx[1] = load_idx(z0 + E);
        issue(0, z0);
        const int32_t npair = (nbat + 1) >> 1;
        for (int32_t pi = 0; pi < npair; ++pi) {
            const int32_t z = z0 + 2 * pi * E;
            __builtin_amdgcn_sched_barrier(0);
            issue(1, z + E);
            __builtin_amdgcn_sched_barrier(0);
            consume(0);
            __builtin_amdgcn_sched_barrier(0);
            issue(0, z + 2 * E);
            __builtin_amdgcn_sched_barrier(0);
            consume(1);
        }
    }

    if constexpr (KSPLIT > 1) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < M::ACC; ++r) sR[((wave * NB + nb) * M::ACC + r) * 64 + lane] = acc[nb][r];
        __syncthreads();
        if (kq != 0) return;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < M::ACC; ++r)
#pragma unroll
                for (int k = 1; k < KSPLIT; ++k) acc[nb][r] += sR[(((wave + k) * NB + nb) * M::ACC + r) * 64 + lane];
    }
    if (!live) return;

    float* __restrict__ y = static_cast<float*>(a.y);
    if constexpr (kEp) {
        // Runs of four rows, each fenced off from the next: computed all at
        // once, the epilogue's parameters and results would raise the
        // kernel's register count (and cut its occupancy) far above what its
        // main loop needs.  (The wave wrote sEp itself; its LDS operations
        // complete in order.)
        EpRows<N, true> ep;
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) {
            if (r % 4 == 0) {
                __builtin_amdgcn_sched_barrier(0);
                ep.load_staged_run(sEp + uw * 2 * N, sEp + uw * 2 * N + N, 0, lane, r / 4);
            }
            const int32_t oc = g * N + M::row(lane, r);
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                if (yo[nb] >= 0 && oc < a.n) store_out(&y[yo[nb] + int64_t(oc) * a.y_c], ep.apply(a, r, acc[nb][r]));
        }
    } else {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb) {
            if (yo[nb] < 0) continue;
#pragma unroll
            for (int r = 0; r < M::ACC; ++r) {
                const int32_t oc = g * N + M::row(lane, r);
                if (oc < a.n) store_out(&y[yo[nb] + int64_t(oc) * a.y_c], acc[nb][r]);
            }
        }
    }
}

template <int N, int NB, int KSPLIT>
onexn_status launch_cfg(ConvArgs a, hipStream_t s) {
    constexpr int COLS = PwMfma<N>::COLS, KS = PwMfma<N>::KS;
    const int64_t units = (int64_t(a.npix) + NB * COLS - 1) / (NB * COLS) * a.G;
    const int64_t upw = 4 / KSPLIT;
    const int64_t grid = (units + upw - 1) / upw;
    // A wave's entries run in whole pairs of batches: short shares take
    // small batches.
    const int64_t per_wave = a.G > 0 ? a.t / a.G / KSPLIT : 0;
    int kdb = per_wave < 8 * 8 * KS ? 2 : 8;
    if (tuning(kTuneDirectKdb) >= 0) kdb = tuning(kTuneDirectKdb);
    return with_epilogue(a, [&](auto ep) {
        constexpr bool E = decltype(ep)::value;
        if (kdb == 2) return launch_grid(pw_direct<N, NB, KSPLIT, 2, E>, a, grid, s, kDThreads);
        return launch_grid(pw_direct<N, NB, KSPLIT, 8, E>, a, grid, s, kDThreads);
    });
}

// (column blocks per unit, waves per unit): the largest tile that gives every
// compute unit a few workgroups, splitting the contraction only when the
// col-groups are long.
template <int N>
onexn_status launch_n(ConvArgs a, hipStream_t s) {
    constexpr int COLS = PwMfma<N>::COLS;
    const int64_t want = 4 * int64_t(device_cu_count());
    const int64_t avg_kept = a.G > 0 ? a.t / a.G : 0;
    auto wgs = [&](int nb, int ks) {
        return ((int64_t(a.npix) + nb * COLS - 1) / (nb * COLS) * a.G * ks + 3) / 4;
    };
    int choice = 0;
    if (tuning(kTuneDirectTile) >= 0) choice = tuning(kTuneDirectTile);
    // Widening layers with many col-groups and few pixels (the 14x14 and 7x7
    // expansions of MobileNet-V2, 64->384 to 160->960) run faster with two
    // waves per unit: 34.6 -> 28.2 us and 48 -> 43 us per layer in the
    // whole-step timing at N = 32, batch 128.  (Per-layer sweeps suggested
    // other shapes for more layers, ResNet-50's strided ones among them; in
    // whole steps those measured slower, up to 23 us per layer, and keep the
    // rule below.)
    if (choice == 0 && N == 32 && a.n > a.m && a.G >= 8 && a.npix <= 32768 && a.sh == 1 && a.sw == 1)
        choice = 3;
    if (choice == 0) {
        if (wgs(2, 1) >= want || avg_kept < 64) choice = 1;
        else if (wgs(1, 1) >= want || avg_kept < 128) choice = 2;
        else if (wgs(1, 2) >= want || avg_kept < 256) choice = 3;
        else choice = 4;
    }
    switch (choice) {
        case 1: return launch_cfg<N, 2, 1>(a, s);
        case 2: return launch_cfg<N, 1, 1>(a, s);
        case 3: return launch_cfg<N, 1, 2>(a, s);
        default: return launch_cfg<N, 1, 4>(a, s);
    }
}

}  // namespace

bool pw_direct_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_F32 || ydt != ONEXN_F32 || layout != ONEXN_NCHW) return false;
    if (a.N != 16 && a.N != 32) return false;
    if (a.kh != 1 || a.kw != 1) return false;
    const int64_t batch = a.npix / a.HWo;
    // 32-bit buffer offsets, with room for an out-of-range marker plus a
    // channel offset.
    if (batch * a.x_img * 4 >= (int64_t(1) << 31)) return false;
    if (int64_t(a.t) * a.N * 4 >= (int64_t(1) << 31)) return false;
    return true;
}

onexn_status launch_pw_direct(ConvArgs a, hipStream_t s) {
    return a.N == 16 ? launch_n<16>(a, s) : launch_n<32>(a, s);
}

}  // namespace onexn
