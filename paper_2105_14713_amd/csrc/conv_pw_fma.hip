// Pointwise (1x1, stride 1, no padding, NCHW) 1xN-pruned convolution, fp32,
// N in {1, 2, 4, 8}: per-lane fused multiply-adds.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Each kept block z of col-group g
// multiplies one input value X[I[z]][pixel] by the block's N contiguous
// weights D[z][0..N-1] -- the block-wise vector product the paper executes on
// CPU vector units.  Here a lane owns output pixels, the N weights of a block
// are the same for the whole wave, and every input value feeds N fused
// multiply-adds.  A 16-row matrix-core tile would be at least half padding at
// these N.
//
// Work split.  A workgroup computes a run of pixel tiles (64 lanes x PPT
// pixels each: 64 apart, or 4 consecutive ones) for a set of GSW col-groups: wave w takes col-group w % GSW of the
// set and, when the contraction is split (KSPLIT = 4 / GSW waves per
// col-group, for layers with few pixels and long col-groups), a contiguous
// share of its kept blocks; the partial sums of a split are added through LDS
// at the end.  The waves of a workgroup read the same pixels of X, so the
// channels their col-groups share are mostly served by the L1 cache.
//
// Each wave stages its share of indices and weights in its own LDS window of
// kFWin blocks (buffer loads straight into LDS, range-checked: entries past
// the col-group read zero weights); all lanes then read the same LDS words
// (broadcast).  Input values come straight from global memory: the pixel
// offset is the range-checked vector offset of a buffer load and the channel
// offset its scalar offset, so a load costs no vector arithmetic and pixels
// past the last image read zeros.  Channels outside [0, m) contribute nothing.

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kFThreads = 256;
constexpr int kFWin = 256;   // kept blocks per staged window (per wave)

// V4: a lane owns 4 consecutive pixels (pixels per image a multiple of 4,
// 16-byte aligned x and y), read and written with 16-byte accesses.
template <int N, int PPT, int GSW, bool V4, bool kEp>
__global__ void __launch_bounds__(kFThreads) pw_fma(ConvArgs a) {
    static_assert(!V4 || PPT == 4, "4 consecutive pixels per lane");
    constexpr int KSPLIT = 4 / GSW;
    constexpr int TP = 64 * PPT;           // pixels per tile
    constexpr int RED = KSPLIT > 1 ? 4 * N * PPT * 64 : 1;
    __shared__ __attribute__((aligned(16))) int32_t sI[4][kFWin];
    __shared__ __attribute__((aligned(16))) float sD[4][kFWin * N];
    __shared__ float sR[RED];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int gw = wave % GSW, kq = wave / GSW;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t gsets = (a.G + GSW - 1) / GSW;
    // The workgroup's col-group set and its run of pixel tiles: the grid is
    // gsets x (tile runs), and a run is ceil(tiles / runs) tiles long.
    const int32_t ntiles = (a.npix + TP - 1) / TP;
    const int32_t nruns = a.total / gsets;
    const int32_t tpw = (ntiles + nruns - 1) / nruns;
    const int32_t run = L / gsets;
    const int32_t t0 = run * tpw, t1 = min(ntiles, t0 + tpw);
    const int32_t g = (L - run * gsets) * GSW + gw;
    int32_t zb = 0, ze = 0;
    if (g < a.G) group_range(a, g, zb, ze);
    // This wave's contiguous share of the col-group's kept blocks.
    const int32_t per = (ze - zb + KSPLIT - 1) / KSPLIT;
    const int32_t z0 = min(ze, zb + kq * per), z1 = min(ze, z0 + per);
    const int32_t batch = a.npix / a.HWo;
    const int32_t xbytes = int32_t(int64_t(batch) * a.x_img * 4);

    const __amdgpu_buffer_rsrc_t rX =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.x), 0, xbytes, kRawBufferFlags);
    const v4i32 rI = buffer_rsrc(a.I, z1 * 4);
    const v4i32 rD = buffer_rsrc(a.D, z1 * N * 4);
    const int32_t* const wI = sI[wave];
    const float* const wD = sD[wave];

    uint32_t xo[PPT];   // byte offset of the lane's pixels at channel 0 (past the input: invalid)
    int64_t yo[PPT];    // element offset in y at channel 0, or -1
    float acc[N][PPT];

    // Blocks are taken in batches of kFB: lane j < kFB of the wave reads
    // block j's channel, every lane then issues the batch's input loads at
    // once, and the next batch's loads are issued before this batch's
    // multiply-adds, so a wave keeps up to 2 kFB loads in flight (kFB shrinks
    // as the loads widen, to keep the register count and occupancy).
    constexpr int kFB = V4 ? 8 : (PPT >= 4 ? 4 : 16 / PPT);
    struct Batch {
        float xv[kFB][PPT];
    };
    // Entries past the share (j >= cnt) and channels outside [0, m) take the
    // value 0 (their loads stay inside the input), so a partial batch adds
    // nothing; the window's weights past the share are zeros (range-checked
    // copies of whole 64-entry blocks).
    auto issue = [&](Batch& bt, int32_t e, int32_t cnt) __attribute__((always_inline)) {
        const int32_t chv = wI[e + (lane & (kFB - 1))];
#pragma unroll
        for (int j = 0; j < kFB; ++j) {
            const int32_t ch = __builtin_amdgcn_readlane(chv, j);
            const bool ok = j < cnt && uint32_t(ch) < uint32_t(a.m);
            const int32_t choff = ok ? ch * a.HWo * 4 : 0;
            if constexpr (V4) {
                const f32x4 v = __builtin_bit_cast(f32x4, __builtin_amdgcn_raw_buffer_load_b128(rX, int32_t(xo[0]), choff, 0));
#pragma unroll
                for (int i = 0; i < 4; ++i) bt.xv[j][i] = ok ? v[i] : 0.f;
            } else {
#pragma unroll
                for (int i = 0; i < PPT; ++i) {
                    const float v = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rX, int32_t(xo[i]), choff, 0));
                    bt.xv[j][i] = ok ? v : 0.f;
                }
            }
        }
    };
    auto consume = [&](const Batch& bt, int32_t e) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < kFB; ++j) {
#pragma unroll
            for (int o = 0; o < N; ++o) {
                const float w = wD[(e + j) * N + o];
#pragma unroll
                for (int i = 0; i < PPT; ++i) acc[o][i] = fmaf(w, bt.xv[j][i], acc[o][i]);
            }
        }
    };
    // Stages entries [w0, w0 + nw) of the wave's share into its LDS window.
    auto stage = [&](int32_t w0, int32_t nw) __attribute__((always_inline)) {
        for (int32_t e0 = 0; e0 < nw; e0 += 64)
            copy4_to_lds(rI, (const lds_char*)(wI + e0), (w0 + e0 + lane) * 4, 0);
        for (int32_t e0 = 0; e0 < nw * N; e0 += 64)
            copy4_to_lds(rD, (const lds_char*)(wD + e0), (w0 * N + e0 + lane) * 4, 0);
        vm_wait<0>();   // the window is in this wave's LDS
    };
    auto compute_window = [&](int32_t nw) __attribute__((always_inline)) {
        const int32_t nb = (nw + kFB - 1) / kFB;
        auto cnt = [&](int32_t bi) { return min(kFB, nw - bi * kFB); };
        Batch b0, b1;
        issue(b0, 0, cnt(0));
        for (int32_t bi = 0; bi < nb; bi += 2) {
            if (bi + 1 < nb) issue(b1, (bi + 1) * kFB, cnt(bi + 1));
            consume(b0, bi * kFB);
            if (bi + 1 >= nb) break;
            if (bi + 2 < nb) issue(b0, (bi + 2) * kFB, cnt(bi + 2));
            consume(b1, (bi + 1) * kFB);
        }
    };

    // A share that fits one window is staged once for all the run's tiles.
    const bool one_window = z1 - z0 <= kFWin;
    if (one_window && z1 > z0) stage(z0, z1 - z0);

    float* __restrict__ y = static_cast<float*>(a.y);
    // Fused epilogue: the wave's N channels are the same for every tile of
    // the run, so their scale and bias are read once here (inside the loop
    // the compiler must reload them after each tile's stores, which may
    // alias them, and every store would wait for those loads).
    float eps[kEp ? N : 1], epb[kEp ? N : 1];
    if constexpr (kEp) {
#pragma unroll
        for (int o = 0; o < N; ++o) {
            const int32_t oc = g * N + o;
            const bool in = g < a.G && oc < a.n;
            // (wave-uniform: kept in scalar registers)
            eps[o] = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                         __builtin_bit_cast(int32_t, in && a.ep_scale ? a.ep_scale[oc] : 1.f)));
            epb[o] = __builtin_bit_cast(float, __builtin_amdgcn_readfirstlane(
                         __builtin_bit_cast(int32_t, in && a.ep_bias ? a.ep_bias[oc] : 0.f)));
        }
    }
    auto ep = [&](int o, float v) {
        if constexpr (kEp) return epilogue_act(a, fmaf(v, eps[o], epb[o]));
        else return v;
    };
    for (int32_t tile = t0; tile < t1; ++tile) {
#pragma unroll
        for (int i = 0; i < PPT; ++i) {
            const int32_t p = V4 ? tile * TP + lane * 4 + i : tile * TP + i * 64 + lane;
            xo[i] = uint32_t(xbytes);
            yo[i] = -1;
            if (p < a.npix) {
                const int32_t b = p / a.HWo, hw = p - b * a.HWo;
                xo[i] = uint32_t((int64_t(b) * a.x_img + hw) * 4);
                yo[i] = int64_t(b) * a.y_img + hw;
            }
        }
#pragma unroll
        for (int o = 0; o < N; ++o)
#pragma unroll
            for (int i = 0; i < PPT; ++i) acc[o][i] = 0.f;

        if (one_window) {
            if (z1 > z0) compute_window(z1 - z0);
        } else {
            for (int32_t w0 = z0; w0 < z1; w0 += kFWin) {
                const int32_t nw = min(kFWin, z1 - w0);
                stage(w0, nw);
                compute_window(nw);
                wait_lgkm();    // this wave's reads of the window are done before it is refilled
            }
        }

        if constexpr (KSPLIT > 1) {
#pragma unroll
            for (int o = 0; o < N; ++o)
#pragma unroll
                for (int i = 0; i < PPT; ++i) sR[((wave * N + o) * PPT + i) * 64 + lane] = acc[o][i];
            __syncthreads();
            if (kq == 0) {
#pragma unroll
                for (int o = 0; o < N; ++o)
#pragma unroll
                    for (int i = 0; i < PPT; ++i)
#pragma unroll
                        for (int k = 1; k < KSPLIT; ++k)
                            acc[o][i] += sR[(((wave + k * GSW) * N + o) * PPT + i) * 64 + lane];
            }
            __syncthreads();   // sR is free for the next tile
        }
        if (kq != 0 || g >= a.G) continue;

#pragma unroll
        for (int o = 0; o < N; ++o) {
            const int32_t oc = g * N + o;
            if (oc >= a.n) continue;
            if constexpr (V4) {
                if (yo[0] >= 0) {
                    const f32x4 v = {ep(o, acc[o][0]), ep(o, acc[o][1]), ep(o, acc[o][2]), ep(o, acc[o][3])};
                    store_out(reinterpret_cast<f32x4*>(y + yo[0] + int64_t(oc) * a.y_c), v);
                }
            } else {
#pragma unroll
                for (int i = 0; i < PPT; ++i)
                    if (yo[i] >= 0) store_out(&y[yo[i] + int64_t(oc) * a.y_c], ep(o, acc[o][i]));
            }
        }
    }
}

// Tiles per workgroup: as many as keep at least 8 workgroups per compute
// unit (at most 16), so that layers with many pixels stage their indices and
// weights once per run of tiles.
template <int N, int PPT, int GSW>
onexn_status launch_cfg(ConvArgs a, hipStream_t s) {
    const int64_t ntiles = (int64_t(a.npix) + 64 * PPT - 1) / (64 * PPT);
    const int64_t gsets = (a.G + GSW - 1) / GSW;
    int64_t tpw = std::max<int64_t>(1, std::min<int64_t>(16, ntiles * gsets / (8 * int64_t(device_cu_count()))));
    if (tuning(kTuneFmaTpw) >= 0) tpw = std::max(1, tuning(kTuneFmaTpw));
    const int64_t tiles = (ntiles + tpw - 1) / tpw;   // tile runs
    if constexpr (PPT == 4) {
        const bool v4 = a.HWo % 4 == 0 && (reinterpret_cast<uintptr_t>(a.x) & 15) == 0 &&
                        (reinterpret_cast<uintptr_t>(a.y) & 15) == 0 && tuning(kTuneFmaNoV4) != 1;
        if (v4)
            return with_epilogue(a, [&](auto ep) {
                return launch_grid(pw_fma<N, PPT, GSW, true, decltype(ep)::value>, a, tiles * gsets, s,
                                   kFThreads);
            });
    }
    return with_epilogue(a, [&](auto ep) {
        return launch_grid(pw_fma<N, PPT, GSW, false, decltype(ep)::value>, a, tiles * gsets, s,
                           kFThreads);
    });
}

// Tile shapes (pixels per lane, col-groups per workgroup): four col-groups
// over 256, 128 or 64 pixels, then two or one col-group with the contraction
// split over the other waves.  The first that gives every compute unit a
// few workgroups is taken; a split needs col-groups long enough to share.
template <int N>
onexn_status launch_n(ConvArgs a, hipStream_t s) {
    const int64_t want = 4 * int64_t(device_cu_count());
    const int64_t avg_kept = a.G > 0 ? a.t / a.G : 0;
    const int64_t gs4 = (a.G + 3) / 4, gs2 = (a.G + 1) / 2;
    auto tiles = [&](int tp) { return (int64_t(a.npix) + tp - 1) / tp; };
    int choice = 0;
    if (tuning(kTuneFmaTile) >= 0) choice = tuning(kTuneFmaTile);
    if (choice == 0) {
        // The widest tile also wins with fewer workgroups (down to ~1.5 per
        // compute unit) unless the col-groups are long (measured on the
        // MobileNet-V2 pointwise layers at N = 4 and 8).
        if (tiles(256) * gs4 >= want || (2 * tiles(256) * gs4 >= 3 * int64_t(device_cu_count()) && avg_kept < 400))
            choice = 1;
        else if (tiles(128) * gs4 >= want) choice = 2;
        else if (tiles(64) * gs4 >= want || avg_kept < 64) choice = 3;
        else if (tiles(64) * gs2 >= want || avg_kept < 128) choice = 4;
        else choice = 5;
    }
    switch (choice) {
        case 1: return launch_cfg<N, 4, 4>(a, s);
        case 2: return launch_cfg<N, 2, 4>(a, s);
        case 3: return launch_cfg<N, 1, 4>(a, s);
        case 4: return launch_cfg<N, 1, 2>(a, s);
        default: return launch_cfg<N, 1, 1>(a, s);
    }
}

}  // namespace

bool pw_fma_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_F32 || ydt != ONEXN_F32 || layout != ONEXN_NCHW) return false;
    if (a.N != 1 && a.N != 2 && a.N != 4 && a.N != 8) return false;
    if (a.kh != 1 || a.kw != 1 || a.sh != 1 || a.sw != 1 || a.ph != 0 || a.pw != 0) return false;
    const int64_t batch = a.npix / a.HWo;
    if (batch * a.x_img * 4 >= (int64_t(1) << 31)) return false;   // 32-bit buffer offsets
    if (int64_t(a.t) * a.N * 4 >= (int64_t(1) << 31)) return false;
    return true;
}

onexn_status launch_pw_fma(ConvArgs a, hipStream_t s) {
    switch (a.N) {
        case 1: return launch_n<1>(a, s);
        case 2: return launch_n<2>(a, s);
        case 4: return launch_n<4>(a, s);
        default: return launch_n<8>(a, s);
    }
}

}  // namespace onexn
