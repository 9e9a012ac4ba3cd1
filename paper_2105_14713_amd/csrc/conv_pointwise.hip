// Pointwise (1x1, stride 1, no padding, NCHW) 1xN-pruned convolution, fp32,
// N in {16, 32}, on fp32 matrix cores.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  For a 1x1 kernel col-group g is the
// contraction Y_g[N][pixels] = D_g^T[N][kept_g] * X[I_g][pixels]: its kept
// blocks select rows of the input matrix X[channel][pixel], and the N weights
// of a block are one contiguous row of D.
//
// Work split.  A workgroup has 8 compute waves and one loader wave.  It owns
// 8/WPG consecutive col-groups (each computed by WPG compute waves, one
// 64-pixel slice each) and a contiguous range of pixel tiles of PT = 64*WPG
// pixels, which it walks in order.  Input channels are walked in chunks of
// KC: the X stream of the workgroup is the sequence (tile, chunk), and chunk
// c of a tile (KC rows x PT pixels, 16 KB) is copied once from global memory
// straight into LDS by the loader wave (global_load_lds, 16 bytes per lane
// where rows allow it) into a ring of kPwRing buffers, several chunks ahead
// of use, and shared by all col-groups of the workgroup.  The loader is a
// wave of its own because a wave's vector loads complete in issue order: a
// compute wave that also streamed X would wait for X behind every weight
// load.  A workgroup barrier per chunk hands a landed chunk to the compute
// waves and frees the buffer of the chunk before it.
//
// Each compute wave streams its own col-group's BSR entries: the entries of
// a chunk are a contiguous run (I is ascending; the run bounds are computed
// once per wave), taken in blocks of 8 MFMA steps.  For a block the wave
// reads the I values (one coalesced load, rows handed to lane groups with
// ds_bpermute) and the weights (one coalesced load per step) straight from
// global memory, one block ahead of use, so the inner loop is 8 LDS reads of
// X and 8*NB MFMAs.  Entries whose channel lies outside [0, m) read a row of
// zeros.
//
//   N = 16: v_mfma_f32_16x16x4f32, 4 kept blocks per step (lane group l/16),
//           NB = 4 column blocks per wave: MFMA column n of block e is pixel
//           4n + e of the wave's slice, so a lane reads 4 consecutive pixels.
//   N = 32: v_mfma_f32_32x32x2f32, 2 kept blocks per step, NB = 2.
#include <cstdio>

#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kPwWaves = 8;                        // compute waves
constexpr int kPwThreads = 64 * (kPwWaves + 1);    // + the loader wave
constexpr int kPwWavePx = 64;     // pixels per wave
constexpr int kPwLdsFloats = 4096;   // one X chunk buffer: 16 KB
constexpr int kPwRing = 6;        // X chunk buffers
constexpr int kPwSteps = 8;       // MFMA steps per block
constexpr int kPwMaxChunks = 64;  // channel chunks a layer may have

template <int N, int WPG>
struct PwShape {
    static constexpr int PT = kPwWavePx * WPG;            // pixels per tile
    static constexpr int S = kPwWaves / WPG;              // col-groups per workgroup
    static constexpr int KC = kPwLdsFloats / PT;          // channels per chunk
    static constexpr int NB = kPwWavePx / N;              // MFMA column blocks per wave
    static constexpr int BLK = kPwSteps * PwMfma<N>::KS;  // BSR entries per block
};

template <int N, int WPG, bool kVec4, bool kEp>
__global__ void __launch_bounds__(kPwThreads) pw_mfma_f32(ConvArgs a) {
    typedef PwMfma<N> M;
    typedef PwShape<N, WPG> SH;
    typedef typename M::acc_t acc_t;
    constexpr int PT = SH::PT, S = SH::S, KC = SH::KC, NB = SH::NB, BLK = SH::BLK;
    constexpr int KS = M::KS, STEPS = kPwSteps;
    // Loads into LDS per chunk (loader wave): 16 bytes per lane when pixel
    // quads are aligned and never straddle an image, else 4 bytes per lane.
    constexpr int EB = kVec4 ? 4 : 1;                 // floats per lane per load
    constexpr int ND = kPwLdsFloats / (EB * 64);      // loads per chunk
    constexpr int QPR = PT / EB;                      // lane slots per X row
    constexpr int ROWB = PT * 4;                      // bytes per X row in LDS
    constexpr int ZERO_OFF = kPwRing * kPwLdsFloats * 4;  // byte offset of the zero row
    static_assert(64 / N == KS && BLK <= 64, "lane groups carry a step's kept blocks");
    static_assert(KC * PT == kPwLdsFloats && KC >= 1, "tile shape");
    typedef typename VecF<NB>::T vec_t;

    __shared__ __attribute__((aligned(16))) float sX[kPwRing * kPwLdsFloats + PT];
    __shared__ int32_t sBnd[kPwWaves][kPwMaxChunks + 1];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
    const int32_t GS = (a.G + S - 1) / S;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t gs = L % GS;
    // This workgroup walks pixel tiles [tile0, tile0 + nt) for col-group set
    // gs: range L / GS of a.tile_ranges near-equal ranges.
    const int32_t tiles = (a.npix + PT - 1) / PT;
    const int32_t rg = L / GS;
    const int32_t tile0 = int32_t(int64_t(rg) * tiles / a.tile_ranges);
    const int32_t nt = int32_t(int64_t(rg + 1) * tiles / a.tile_ranges) - tile0;
    const int32_t nch = (a.m + KC - 1) / KC;
    const int32_t nel = nt * nch;   // X stream: element e = chunk e % nch of tile tile0 + e / nch

    if (wave == kPwWaves) {
        // (Issue arbitration favours older waves; the loader, the youngest,
        // gets the highest priority so that its copies are not issued only
        // in the compute waves' gaps.)
        __builtin_amdgcn_s_setprio(3);
        // Loader wave.  Element e goes to ring buffer e % kPwRing.  Load j
        // covers LDS floats [j*64*EB, (j+1)*64*EB) of the buffer
        // (lane-contiguous, as loads into LDS require): lane slot f = j*64 +
        // lane is row f / QPR, pixel EB*(f % QPR) of the tile.  Rows past m
        // and pixels past the last image read a valid element instead (never
        // used: rows past m are never selected, pixels past the end are
        // never stored).
        const float* __restrict__ x = static_cast<const float*>(a.x);
        auto issue_x = [&](int32_t e) {
            const int32_t tile = tile0 + e / nch, c = e % nch;
            float* dst = sX + (e % kPwRing) * kPwLdsFloats;
#pragma unroll 4
            for (int j = 0; j < ND; ++j) {
                const int32_t f = j * 64 + lane;
                int32_t p = tile * PT + EB * (f % QPR);
                p = p < a.npix ? p : 0;
                const int32_t b = p / a.HWo;
                const int32_t ch = min(c * KC + f / QPR, a.m - 1);
                const float* src = x + int64_t(b) * a.x_img + int64_t(ch) * a.x_c + (p - b * a.HWo);
                if constexpr (kVec4)
                    __builtin_amdgcn_global_load_lds(src, dst + j * 64 * EB, 16, 0, 0);
                else
                    __builtin_amdgcn_global_load_lds(src, dst + j * 64 * EB, 4, 0, 0);
            }
        };
        // Waits for element e's loads, `newer` elements having been issued
        // after it.  Loads complete in issue order, so at most newer*ND
        // outstanding loads means e has landed (the count saturates at the
        // counter's range, which only waits longer).
        auto wait_x = [&](int32_t newer) {
            const int32_t k = newer * ND;
            if (k >= 63) wait_vmem<63>();
            else if (k >= 48) wait_vmem<48>();
            else if (k >= 32) wait_vmem<32>();
            else if (k >= 16) wait_vmem<16>();
            else wait_vmem<0>();
        };
        static_assert(ND % 16 == 0, "wait_x counts in steps of 16 loads");
        for (int32_t e = 0; e < min(kPwRing - 1, nel); ++e) issue_x(e);
        for (int i = lane; i < PT; i += 64) sX[kPwRing * kPwLdsFloats + i] = 0.f;
        wait_lgkm();
        __builtin_amdgcn_s_barrier();   // set-up done
        for (int32_t el = 0; el < nel; ++el) {
            wait_x(min(el + kPwRing - 2, nel - 1) - el);
            __builtin_amdgcn_s_barrier();   // element el visible; buffer of el - 1 free
            if (el + kPwRing - 1 < nel) issue_x(el + kPwRing - 1);
        }
        return;
    }

    const int32_t g = gs * S + wave / WPG;      // this wave's col-group
    const int slice = wave % WPG;               // this wave's 64-pixel slice
    const float* __restrict__ D = static_cast<const float*>(a.D);
    int32_t zb = 0, ze = 0;
    if (g < a.G) group_range(a, g, zb, ze);

    // Run bounds: entries [sBnd[w][c], sBnd[w][c+1]) of the col-group have
    // input channels in chunk c.  One pass over the col-group's I entries,
    // 64 at a time, counting the entries below each chunk's end.
    for (int32_t c = lane; c <= nch; c += 64) sBnd[wave][c] = zb;
    for (int32_t z0 = zb; z0 < ze; z0 += 64) {
        const int32_t z = z0 + lane;
        const int32_t iv = z < ze ? a.I[z] : INT32_MAX;
        for (int32_t c = 0; c < nch; ++c) {
            const int32_t below = __popcll(__ballot(iv < (c + 1) * KC));
            if (lane == 0) sBnd[wave][c + 1] += below;
        }
    }

    // One block of the wave's BSR entries: [s, s + len), len <= BLK, all in
    // one chunk.  The loads are only issued here; nothing consumes them until
    // the block is run (one block later), so they stay in flight across the
    // MFMAs of the block before.  Indices past len are clamped to the block's
    // last entry: its weights are loaded again, and the entry reads the zero
    // row of X.
    struct Block {
        int32_t ch;          // lane i: input channel of entry min(i, len - 1)
        float av[STEPS];     // weight of step ks for this lane's (lane group, output)
    };
    const int lg = lane / N, lo = lane % N;
    auto load_block = [&](Block& bk, int32_t s, int32_t len) {
        if (len <= 0) return;   // uniform: nothing left for this wave
        const int32_t* Ib = a.I + s;
        const float* Db = D + int64_t(s) * N;
        bk.ch = Ib[min(lane, len - 1)];
#pragma unroll
        for (int ks = 0; ks < STEPS; ++ks) bk.av[ks] = Db[uint32_t(min(ks * KS + lg, len - 1) * N + lo)];
    };

    acc_t acc[NB];
#pragma unroll
    for (int e = 0; e < NB; ++e)
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) acc[e][r] = 0.f;

    // Multiplies one loaded block against the X rows it names: the block's
    // chunk has base channel c0 and sits in ring buffer buf.  Lanes i >= len
    // and channels outside the chunk or [0, m) read the zero row.
    const char* xs = reinterpret_cast<const char*>(sX + slice * kPwWavePx + NB * lo);
    auto run_block = [&](const Block& bk, int32_t len, int32_t c0, int32_t buf) {
        const int32_t rel = bk.ch - c0;
        const bool ok = lane < len && rel >= 0 && rel < KC && bk.ch < a.m;
        const int32_t off = ok ? (buf * KC + rel) * ROWB : ZERO_OFF;
        vec_t bv[STEPS];
#pragma unroll
        for (int ks = 0; ks < STEPS; ++ks) {
            const int32_t o = __builtin_amdgcn_ds_bpermute(4 * (ks * KS + lg), off);
            bv[ks] = *reinterpret_cast<const vec_t*>(xs + o);
        }
        // Keep all X reads of the block ahead of the (guarded) MFMAs.
#pragma unroll
        for (int ks = 0; ks < STEPS; ++ks) asm volatile("" : "+v"(bv[ks]));
        const int32_t nsteps = (len + KS - 1) / KS;
        if (nsteps == STEPS) {
#pragma unroll
            for (int ks = 0; ks < STEPS; ++ks)
#pragma unroll
                for (int e = 0; e < NB; ++e) acc[e] = M::step(bk.av[ks], bv[ks][e], acc[e]);
        } else {
#pragma unroll
            for (int ks = 0; ks < STEPS; ++ks) {
                if (ks >= nsteps) break;
#pragma unroll
                for (int e = 0; e < NB; ++e) acc[e] = M::step(bk.av[ks], bv[ks][e], acc[e]);
            }
        }
    };

    // Epilogue of one tile: block e, MFMA (row, col n) -> output channel
    // g*N + row, pixel tile*PT + slice*64 + NB*n + e; a lane's NB pixels are
    // consecutive.  The accumulators are cleared for the next tile.
    float* __restrict__ y = static_cast<float*>(a.y);
    auto epilogue = [&](int32_t tile) {
        if (g < a.G) {
            const int32_t p0 = tile * PT + slice * kPwWavePx + NB * lo;
            if (kVec4) {
                // HWo % 4 == 0: an aligned run of NB <= 4 pixels lies in one image.
                if (p0 < a.npix) {
                    const int32_t b = p0 / a.HWo;
                    const int64_t yb = int64_t(b) * a.y_img + (p0 - b * a.HWo);
#pragma unroll
                    for (int r = 0; r < M::ACC; ++r) {
                        const int32_t o = g * N + M::row(lane, r);
                        if (o >= a.n) continue;
                        vec_t v;
#pragma unroll
                        for (int e = 0; e < NB; ++e) v[e] = onexn::epilogue<kEp>(a, o, acc[e][r]);
                        store_out(reinterpret_cast<vec_t*>(y + yb + int64_t(o) * a.y_c), v);
                    }
                }
            } else {
#pragma unroll
                for (int e = 0; e < NB; ++e) {
                    const int32_t p = p0 + e;
                    if (p >= a.npix) continue;
                    const int32_t b = p / a.HWo;
                    const int64_t yb = int64_t(b) * a.y_img + (p - b * a.HWo);
#pragma unroll
                    for (int r = 0; r < M::ACC; ++r) {
                        const int32_t o = g * N + M::row(lane, r);
                        if (o < a.n) store_out(&y[yb + int64_t(o) * a.y_c], onexn::epilogue<kEp>(a, o, acc[e][r]));
                    }
                }
            }
        }
#pragma unroll
        for (int e = 0; e < NB; ++e)
#pragma unroll
            for (int r = 0; r < M::ACC; ++r) acc[e][r] = 0.f;
    };

    // Block schedule: blocks never straddle a chunk; the run of blocks is the
    // same for every tile (it depends on the col-group only) and restarts at
    // each tile.  While a block is multiplied, the next one's loads are in
    // flight, including the first block of the next tile.
    wait_lgkm();   // the run bounds are LDS stores
    __builtin_amdgcn_s_barrier();
    struct Pos {
        int32_t t, c, s, e, len;   // tile, chunk, first entry, end of the chunk's run, entries
    };
    // Positions are wave-uniform; readfirstlane keeps them in scalar registers.
    auto bound = [&](int32_t c) { return __builtin_amdgcn_readfirstlane(sBnd[wave][c]); };
    auto settle = [&](Pos& q) {
        // moves past exhausted chunks; at the end of the col-group len == 0
        while (q.s >= q.e && q.c + 1 < nch) {
            ++q.c;
            q.s = bound(q.c);
            q.e = bound(q.c + 1);
        }
        q.len = max(min(BLK, q.e - q.s), 0);
    };
    auto first = [&](int32_t t) {
        Pos q{t, 0, zb, bound(1), 0};
        settle(q);
        return q;
    };
    auto after = [&](const Pos& q) {
        Pos r{q.t, q.c, q.s + q.len, q.e, 0};
        settle(r);
        if (r.len == 0 && q.t + 1 < nt) r = first(q.t + 1);
        return r;
    };
    auto buf_of = [&](const Pos& q) { return (q.t * nch + q.c) % kPwRing; };
    Pos q0 = first(0);
    Block bk0, bk1;
    // The first block goes through bk1 like every later one, so that bk0's
    // registers are only written by the copy in the loop and the waits for
    // in-flight loads stay exact.
    load_block(bk1, q0.s, q0.len);
    asm volatile("" : "+v"(bk1.ch));
#pragma unroll
    for (int ks = 0; ks < STEPS; ++ks) asm volatile("" : "+v"(bk1.av[ks]));
    bk0 = bk1;

    for (int32_t el = 0; el < nel; ++el) {
        const int32_t tt = el / nch, c = el - tt * nch;
        __builtin_amdgcn_s_barrier();   // element el has landed in LDS
        while (q0.t == tt && q0.c == c && q0.len > 0) {
            const Pos q1 = after(q0);
            load_block(bk1, q1.s, q1.len);
            run_block(bk0, q0.len, q0.c * KC, buf_of(q0));
            // The next block's loads stay in flight across this block's MFMAs.
            asm volatile("" : "+v"(bk1.ch));
#pragma unroll
            for (int ks = 0; ks < STEPS; ++ks) asm volatile("" : "+v"(bk1.av[ks]));
            bk0 = bk1;
            q0 = q1;
        }
        if (c == nch - 1) epilogue(tile0 + tt);
    }
}

// Waves per col-group: 1 when the layer has at least 8 col-groups, more for
// narrower layers so that no wave of a workgroup is idle.  ONEXN_PW_WPG
// overrides it for A/B measurements.
int choose_wpg(const ConvArgs& a) {
    const int32_t v = tuning(kTunePwWpg);
    if (v == 1 || v == 2 || v == 4 || v == 8) return v;
    if (a.G >= 8) return 1;
    if (a.G >= 4) return 2;
    if (a.G >= 2) return 4;
    return 8;
}

// Tile ranges per col-group set: one workgroup per compute unit in total
// (one fits per CU), each walking its range so that its X stream never
// drains; ONEXN_PW_RANGES overrides the count for A/B measurements.
int64_t choose_ranges(int64_t tiles, int64_t gsets) {
    if (tuning(kTunePwRanges) >= 1) return std::min<int64_t>(tuning(kTunePwRanges), tiles);
    const int64_t per_set = std::max<int64_t>(1, int64_t(device_cu_count()) / gsets);
    return std::min<int64_t>(per_set, tiles);
}

template <int N, int WPG>
onexn_status launch_pw(ConvArgs a, hipStream_t s) {
    typedef PwShape<N, WPG> SH;
    const int64_t tiles = (int64_t(a.npix) + SH::PT - 1) / SH::PT;
    const int64_t gsets = (a.G + SH::S - 1) / SH::S;
    const int64_t ranges = choose_ranges(tiles, gsets);
    a.tile_ranges = int32_t(ranges);
    const bool vec4 = a.HWo % 4 == 0 && (reinterpret_cast<uintptr_t>(a.x) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(a.y) & 15) == 0;
    return with_epilogue(a, [&](auto ep) {
        constexpr bool E = decltype(ep)::value;
        if (vec4) return launch_grid(pw_mfma_f32<N, WPG, true, E>, a, ranges * gsets, s, kPwThreads);
        return launch_grid(pw_mfma_f32<N, WPG, false, E>, a, ranges * gsets, s, kPwThreads);
    });
}

template <int N>
onexn_status launch_pw_n(ConvArgs a, hipStream_t s) {
    switch (choose_wpg(a)) {
        case 1: return launch_pw<N, 1>(a, s);
        case 2: return launch_pw<N, 2>(a, s);
        case 4: return launch_pw<N, 4>(a, s);
        default: return launch_pw<N, 8>(a, s);
    }
}

}  // namespace

bool pointwise_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (!(layout == ONEXN_NCHW && xdt == ONEXN_F32 && ydt == ONEXN_F32 && a.kh == 1 &&
          a.kw == 1 && a.sh == 1 && a.sw == 1 && a.ph == 0 && a.pw == 0 &&
          (a.N == 16 || a.N == 32)))
        return false;
    // The per-wave run bounds hold at most kPwMaxChunks channel chunks.
    const int kc = kPwLdsFloats / (kPwWavePx * choose_wpg(a));
    return a.m <= int64_t(kPwMaxChunks) * kc;
}

// The resident-tile kernel where the layer fits it, else the streamed one.
// ONEXN_PW_KERNEL=stream or =tile forces one of them (for tests and A/B
// measurements; =tile on a layer it does not fit is an error).
onexn_status launch_pointwise(ConvArgs a, onexn_dtype, onexn_dtype, hipStream_t s) {
    const int32_t force = tuning(kTunePwKernel);
    if (force == 1 && !pw_tile_applies(a))
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: the resident-tile kernel does not fit this layer");
    if (force != 2 && pw_tile_applies(a)) return launch_pw_tile(a, s);
    return a.N == 16 ? launch_pw_n<16>(a, s) : launch_pw_n<32>(a, s);
}

}  // namespace onexn
