// Pointwise (1x1, stride 1, no padding, NCHW) 1xN-pruned convolution, fp32,
// N in {16, 32}, for layers whose input-channel count lets a whole pixel tile
// of X stay in LDS (m * 16..64 pixels * 4 bytes <= 64 KB).
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  For a 1x1 kernel col-group g is the
// contraction Y_g[N][pixels] = D_g^T[N][kept_g] * X[I_g][pixels]: its kept
// blocks select rows of the input matrix X[channel][pixel], and the N weights
// of a block are one contiguous row of D.
//
// Work split.  A pixel tile is SL slices of SW pixels; a unit of work is one
// (slice, col-group) pair of a tile, and costs kept_g + 1 (the kept blocks,
// plus its stores).  The (tile, unit) sequence, tile-major, is cut into one
// contiguous range of equal cost per workgroup (one workgroup per CU), so
// workgroups finish together however unevenly the col-groups are pruned
// (output-channel rearrangement makes the first col-groups the heaviest).
//
// A workgroup has 15 compute waves and one loader wave, and two LDS buffers
// that each hold all m rows of one tile's X.  The loader copies the tiles of
// the range into the buffers in turn (global_load_lds, 16 bytes per lane
// where pixel quads allow it): a tile is copied while the one before it is
// computed.  It is a wave of its own because a wave's vector loads complete
// in issue order: a compute wave that also copied X would wait for the copy
// behind its next weight load.  Compute waves take the units of the landed
// tile from an LDS counter until none is left and go straight on to the next
// tile, so no wave waits for the others at tile ends.  LDS flags order the
// two sides: `ready` (a buffer's unit counter is reset for its next tile),
// `landed` (that tile's X is in the buffer) and `done` (compute waves
// finished with a buffer's tile, so it may be reused).
//
// A wave computes a unit as a dense contraction over the col-group's kept
// blocks, taken in blocks of 8 MFMA steps: for each block it reads the I
// values (one coalesced load, rows handed to lane groups with ds_bpermute) and
// the weights (one coalesced load per step) from global memory, one block
// ahead of use, then 8 LDS reads of X and 8*NB MFMAs.  Entries whose channel
// lies outside [0, m) read a row of zeros.
//
//   N = 16: v_mfma_f32_16x16x4f32, 4 kept blocks per step (lane group l/16).
//   N = 32: v_mfma_f32_32x32x2f32, 2 kept blocks per step.
//   NB = SW / (MFMA columns) column blocks per unit: MFMA column n of block e
//   is pixel NB*n + e of the slice, so a lane reads NB consecutive pixels.

#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kTileCompute = 15;                        // compute waves
constexpr int kTileThreads = 64 * (kTileCompute + 1);   // + the loader wave
constexpr int kTileBufFloats = 16384;                   // one X tile buffer: 64 KB
constexpr int kTileSteps = 4;                           // MFMA steps per block
constexpr int kTileMaxG = 256;                          // col-groups a layer may have
constexpr int32_t kBufferFlags = 0x00020000;            // buffer resource word 3: 32-bit raw data
constexpr int kTileEarly = 32;                          // copies of the second tile issued before the first is awaited
constexpr int kTileEpMax = 3072;                        // channels whose epilogue parameters LDS holds

__device__ __forceinline__ int32_t lds_load(const int32_t* p) {
    return __hip_atomic_load(p, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}
__device__ __forceinline__ void lds_store(int32_t* p, int32_t v) {
    __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_WORKGROUP);
}

template <int N, int SW, bool kVec4, bool kEp>
__global__ void __launch_bounds__(kTileThreads) pw_tile_f32(ConvArgs a) {
    typedef PwMfma<N> M;
    typedef typename M::acc_t acc_t;
    constexpr int KS = M::KS, STEPS = kTileSteps, BLK = STEPS * KS;
    constexpr int NB = SW / M::COLS;
    constexpr int EB = kVec4 ? 4 : 1;   // floats per lane per X load
    constexpr int ZERO_OFF = 2 * kTileBufFloats * 4;
    static_assert(NB >= 1 && NB * M::COLS == SW, "slice width");
    static_assert(64 / N == KS && BLK <= 64, "lane groups carry a step's kept blocks");
    typedef typename VecF<NB>::T vec_t;

    __shared__ __attribute__((aligned(16))) float sX[2 * kTileBufFloats + SW];
    __shared__ int32_t sP[kTileMaxG + 1];   // P[g] + g: cost of the units before group g
    __shared__ int32_t sNext[2], sReady[2], sLanded[2], sDone[2], sSetup;
    // Fused epilogue: scale then bias of every channel of the col-groups
    // (G * N <= kTileEpMax), staged once so that the stores inside the main
    // loop read them from LDS: a global load there would make the store wait
    // for every weight and index load the pipeline has in flight.
    __shared__ __attribute__((aligned(16))) float sEp[kEp ? 2 * kTileEpMax : 4];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t G = a.G, SL = a.slices, PT = SL * SW;
    const int32_t units = SL * G;
    const int32_t slice_cost = a.t + G;
    const int32_t tile_cost = slice_cost * SL;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t W = a.total;
    // Cost range [c0, c1) of this workgroup; the host split the total cost
    // (below 2^31) into cost_q * W + cost_r.
    const int32_t c0 = a.cost_q * L + a.cost_r * L / W;
    const int32_t c1 = a.cost_q * (L + 1) + a.cost_r * (L + 1) / W;
    if (c0 >= c1) return;   // the whole workgroup: nothing to do

    // X copy of tile T into buffer b (loader wave).  The tile is m rows of
    // spr = PT/EB lane slots (a power of two); lane slot f = j*64 + lane of
    // load j is row f / spr, pixel EB*(f % spr), at LDS float offset f*EB, so
    // each load's 64 slots are contiguous, as loads into LDS require.
    //   spr <= 64: load j covers rows j*(64/spr) + lane/spr, and a lane keeps
    //              one pixel for the whole tile.
    //   spr > 64:  load j covers pixel block pb = j % nb (nb = spr/64) of row
    //              j / nb, so a lane keeps one pixel per block.
    // Each lane computes its pixel's address once per block and steps rows by
    // pointer increments.  Pixels past the last image read a valid element
    // instead (never stored).
    const float* __restrict__ x = static_cast<const float*>(a.x);
    const int32_t spr = PT / EB;
    const int spr_shift = __builtin_ctz(uint32_t(spr));
    auto pixel_src = [&](int32_t T, int32_t slot) {
        int32_t p = T * PT + EB * slot;
        p = p < a.npix ? p : 0;
        const int32_t bi = p / a.HWo;
        return x + int64_t(bi) * a.x_img + (p - bi * a.HWo);
    };
    auto dma = [&](const float* src, float* dst) {
        if constexpr (kVec4)
            __builtin_amdgcn_global_load_lds(src, dst, 16, 0, 0);
        else
            __builtin_amdgcn_global_load_lds(src, dst, 4, 0, 0);
    };
    // `early` (copy of the second tile while the first is in flight): once
    // kTileEarly of its loads are issued, every load of the first tile has
    // completed (loads complete in issue order), so the first tile is
    // published as landed there.  Returns whether that happened.
    auto land_first = [&]() {
        if (lane == 0) lds_store(&sLanded[0], 1);
    };
    auto copy_tile = [&](int32_t T, int b, bool early) {
        float* dst0 = sX + b * kTileBufFloats;
        int32_t issued = 0;
        auto count = [&]() {
            if (early && ++issued == kTileEarly) {
                wait_vmem<kTileEarly>();
                land_first();
            }
        };
        if (spr <= 64) {
            const int32_t rpl = 64 >> spr_shift;           // rows per load
            const int32_t row0 = lane >> spr_shift;
            const float* src = pixel_src(T, lane & (spr - 1)) + int64_t(row0) * a.x_c;
            const int64_t step = int64_t(rpl) * a.x_c;
            for (int32_t j = 0; j * rpl < a.m; ++j, src += step) {
                if (j * rpl + row0 < a.m) dma(src, dst0 + j * 64 * EB);
                count();
            }
        } else {
            const int32_t nb = spr >> 6;
            for (int32_t pb = 0; pb < nb; ++pb) {
                const float* src = pixel_src(T, 64 * pb + lane);
                for (int32_t r = 0; r < a.m; ++r, src += a.x_c) {
                    dma(src, dst0 + (r * nb + pb) * 64 * EB);
                    count();
                }
            }
        }
        return issued >= kTileEarly;
    };

    const bool loader = wave == kTileCompute;
    // The loader is the youngest wave of its SIMD, and issue arbitration
    // favours older waves: without a raised priority its copies are issued
    // only in the compute waves' gaps, and a tile copy takes longer than the
    // tile's compute.
    if (loader) __builtin_amdgcn_s_setprio(3);
    const int32_t Tfirst = c0 / tile_cost;
    if (tid < 2) {
        sReady[tid] = 0;
        sLanded[tid] = 0;
        sDone[tid] = 0;
    }
    if (tid == 0) sSetup = 0;
    wait_lgkm();
    __builtin_amdgcn_s_barrier();   // the flags are set (all waves arrive at once)

    // The loader starts the first tile's copy right away.  The compute waves
    // meanwhile put P into LDS through the scalar cache (each wave loads
    // chunks of 16 entries with uniform addresses clamped to the array) and
    // meet on an LDS counter, not a barrier, so that none of them waits for
    // the loader to finish issuing the copy.
    if (loader) {
        copy_tile(Tfirst, 0, false);
    } else {
        for (int32_t c = wave; c * 16 <= G; c += kTileCompute) {
            int32_t v = 0;
#pragma unroll
            for (int j = 0; j < 16; ++j) {
                const int32_t pj = a.P[min(c * 16 + j, G)];
                v = lane == j ? pj : v;
            }
            const int32_t i = c * 16 + lane;
            if (lane < 16 && i <= G) sP[i] = max(0, min(v, a.t)) + i;
        }
        for (int i = lane; i < SW; i += 64)
            if (wave == 0) sX[2 * kTileBufFloats + i] = 0.f;
        if constexpr (kEp) {
            for (int32_t i = tid; i < G * N; i += kTileCompute * 64) {
                const bool in = i < a.n;
                sEp[i] = in && a.ep_scale ? a.ep_scale[i] : 1.f;
                sEp[kTileEpMax + i] = in && a.ep_bias ? a.ep_bias[i] : 0.f;
            }
        }
        wait_lgkm();
        if (lane == 0) atomicAdd(&sSetup, 1);
    }
    while (__builtin_amdgcn_readfirstlane(lds_load(&sSetup)) < kTileCompute) __builtin_amdgcn_s_sleep(1);

    // First unit at or after cost offset c: the tile's units sorted by
    // start cost s*(t + G) + P[g] + g.
    auto locate = [&](int32_t c, int32_t& tile, int32_t& unit) {
        tile = c / tile_cost;
        const int32_t r = c - tile * tile_cost;
        const int32_t s = r / slice_cost;
        const int32_t rr = r - s * slice_cost;
        int32_t lo = 0, hi = G;   // first g in [0, G] with sP[g] >= rr
        while (lo < hi) {
            const int32_t mid = (lo + hi) >> 1;
            if (sP[mid] >= rr) hi = mid;
            else lo = mid + 1;
        }
        unit = lo == G ? (s + 1) * G : s * G + lo;
        if (unit >= units) {
            ++tile;
            unit = 0;
        }
    };
    int32_t T0, u0, T1, u1;
    locate(c0, T0, u0);
    locate(c1, T1, u1);
    T0 = __builtin_amdgcn_readfirstlane(T0);
    u0 = __builtin_amdgcn_readfirstlane(u0);
    T1 = __builtin_amdgcn_readfirstlane(T1);
    u1 = __builtin_amdgcn_readfirstlane(u1);
    // The workgroup's tiles are T0 .. Tlast; tile k of them (T0 + k) sits in
    // buffer k % 2.  Its units are [ub, ue).
    const int32_t ntiles = (u1 > 0 ? T1 + 1 : T1) - T0;
    auto unit_begin = [&](int32_t k) { return k == 0 ? u0 : 0; };
    auto unit_end = [&](int32_t k) { return T0 + k == T1 ? u1 : units; };

    if (wave == 0 && ntiles > 0) {
        if (lane == 0) lds_store(&sNext[0], unit_begin(0));
        wait_lgkm();
        if (lane == 0) lds_store(&sReady[0], 1);
    }

    if (loader) {
        // Both buffers are free at the start, so the second tile is copied
        // right behind the first instead of after it has landed: a range
        // whose first tile has few units would otherwise leave most waves
        // idle for a whole copy, and even a full first tile ends before a
        // copy issued at its landing (measured: batch 64 of the 256->512
        // 28x28 layer 10 % faster, the 64->256 56x56 one 8 %).
        const bool early = ntiles > 1;
        for (int32_t k = 0; k < ntiles; ++k) {
            const int b = k & 1;
            if (k >= 2) {
                // Buffer b is free once every compute wave is done with tile k - 2.
                while (__builtin_amdgcn_readfirstlane(lds_load(&sDone[b])) < kTileCompute * (k / 2))
                    __builtin_amdgcn_s_sleep(2);
            }
            // The units can be handed out before the tile lands: compute
            // waves load their first blocks' weights and indices meanwhile.
            // (The first tile's counter is set by compute wave 0.)
            if (k > 0 && !(k == 1 && early)) {
                if (lane == 0) lds_store(&sNext[b], unit_begin(k));
                wait_lgkm();
                if (lane == 0) lds_store(&sReady[b], k + 1);
            }
            if ((k > 0 && !(k == 1 && early)) || (k == 0 && Tfirst != T0)) copy_tile(T0 + k, b, false);
            if (k == 0 && early) {
                if (lane == 0) lds_store(&sNext[1], unit_begin(1));
                wait_lgkm();
                if (lane == 0) lds_store(&sReady[1], 2);
                if (copy_tile(T0 + 1, 1, true)) continue;   // the first tile is published
            }
            wait_vmem<0>();   // the tile has landed in LDS
            if (lane == 0) lds_store(&sLanded[b], k + 1);
        }
        wait_vmem<0>();   // no copy into LDS may outlive the workgroup
        return;
    }

    // The wave's work in a tile is a stream of blocks: each unit it takes is
    // cut into blocks of up to BLK entries (STEPS MFMA steps), described by
    // uniform values (entries [s, s + len) of col-group g, X slice at LDS
    // float offset base, whether it ends its unit).  The stream is
    // software-pipelined: while block j is multiplied, the wave reads block
    // j+1's X rows from LDS, hands block j+2's row offsets to its lane groups
    // (ds_bpermute), and loads block j+1's weights and block j+3's channel
    // indices.  These instructions are interleaved with block j's MFMAs
    // because a wave waiting to issue an MFMA holds its SIMD: work issued
    // between MFMAs is nearly free, work issued around a run of MFMAs is
    // not.  Registers of consecutive blocks alternate between two sets (the
    // loop is unrolled by two), so nothing is copied from block to block.
    struct Desc {
        int32_t s, len, ze, base, g, slice;
        bool last, valid;
    };
    // I and D are read through buffer resources with the whole offset (block
    // start plus lane position) in the vector offset, which the hardware
    // range-checks (the scalar offset is not checked): reads past the arrays
    // return 0 and never leave them.  A block always
    // loads BLK entries: entries past len belong to the next col-group (or
    // are zeros past t) and meet the zero row of X.
    const __amdgpu_buffer_rsrc_t rI =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(a.I), 0, a.t * 4, kBufferFlags);
    const __amdgpu_buffer_rsrc_t rD =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.D), 0, a.t * N * 4, kBufferFlags);
    const int lg = lane / N, lo = lane % N;
    const int32_t lane_i = (lane % BLK) * 4, lane_d = lane * 4;
    auto load_ch = [&](int32_t& ch, const Desc& d) {
        ch = __builtin_amdgcn_raw_buffer_load_b32(rI, lane_i + d.s * 4, 0, 0);
    };
    auto load_w = [&](float (&av)[STEPS], const Desc& d) {
#pragma unroll
        for (int ks = 0; ks < STEPS; ++ks)
            av[ks] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rD, lane_d + ks * KS * N * 4 + d.s * N * 4, 0, 0));
    };
    // Row offsets of a block, one per step for this lane's group: lane i of
    // the block names entry i's X row (lanes i >= len and channels outside
    // [0, m) name the zero row); step ks hands entry ks*KS + lg's row to
    // lane group lg.
    auto offsets = [&](int32_t (&o)[STEPS], int32_t ch, const Desc& d) {
        const int32_t row = (d.base + ch * PT) * 4;
        const bool ok = lane < d.len && uint32_t(ch) < uint32_t(a.m);
        const int32_t off = ok ? row : ZERO_OFF;
#pragma unroll
        for (int ks = 0; ks < STEPS; ++ks) o[ks] = __builtin_amdgcn_ds_bpermute(4 * (ks * KS + lg), off);
    };
    const char* xs = reinterpret_cast<const char*>(sX + NB * lo);
    auto read_x = [&](vec_t (&bv)[STEPS], const int32_t (&o)[STEPS]) {
#pragma unroll
        for (int ks = 0; ks < STEPS; ++ks) bv[ks] = *reinterpret_cast<const vec_t*>(xs + o[ks]);
    };

    acc_t acc[NB];
#pragma unroll
    for (int e = 0; e < NB; ++e)
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) acc[e][r] = 0.f;

    // Stores the accumulators of a unit (or zeros, for a unit without kept
    // blocks): MFMA (row, col n) of block e -> output channel g*N + row,
    // pixel T*PT + slice*SW + NB*n + e.  Clears the accumulators.
    float* __restrict__ y = static_cast<float*>(a.y);
    auto store_unit = [&](int32_t tile, int32_t slice, int32_t g, bool zeros) __attribute__((always_inline)) {
        const int32_t p0 = tile * PT + slice * SW + NB * lo;
        EpRows<N, kEp> ep;
        if (kVec4) {
            // HWo % 4 == 0: an aligned run of NB <= 4 pixels lies in one image.
            if (p0 < a.npix) {
                const int32_t b = p0 / a.HWo;
                float* yb = y + int64_t(b) * a.y_img + (p0 - b * a.HWo);
#pragma unroll
                for (int r = 0; r < M::ACC; ++r) {
                    if (r % 4 == 0) ep.load_staged_run(sEp, sEp + kTileEpMax, g, lane, r / 4);
                    const int32_t o = g * N + M::row(lane, r);
                    if (o >= a.n) continue;
                    vec_t v;
#pragma unroll
                    for (int e = 0; e < NB; ++e) vec_set<NB>(v, e, ep.apply(a, r, zeros ? 0.f : acc[e][r]));
                    store_out(reinterpret_cast<vec_t*>(yb + int64_t(o) * a.y_c), v);
                }
            }
        } else {
            ep.load_staged(sEp, sEp + kTileEpMax, g, lane);
#pragma unroll
            for (int e = 0; e < NB; ++e) {
                const int32_t p = p0 + e;
                if (p >= a.npix) continue;
                const int32_t b = p / a.HWo;
                const int64_t yb = int64_t(b) * a.y_img + (p - b * a.HWo);
#pragma unroll
                for (int r = 0; r < M::ACC; ++r) {
                    const int32_t o = g * N + M::row(lane, r);
                    if (o < a.n) store_out(&y[yb + int64_t(o) * a.y_c], ep.apply(a, r, zeros ? 0.f : acc[e][r]));
                }
            }
        }
        if (!zeros) {
#pragma unroll
            for (int e = 0; e < NB; ++e)
#pragma unroll
                for (int r = 0; r < M::ACC; ++r) acc[e][r] = 0.f;
        }
    };

    for (int32_t k = 0; k < ntiles; ++k) {
        const int b = k & 1;
        const int32_t T = T0 + k, ue = unit_end(k);
        while (__builtin_amdgcn_readfirstlane(lds_load(&sReady[b])) < k + 1)
            __builtin_amdgcn_s_sleep(1);

        // Units of this tile, taken from the LDS counter; a unit without
        // kept blocks is stored as zeros right away.
        auto next_unit = [&](Desc& d) {
            while (true) {
                int32_t u = 0;
                if (lane == 0) u = atomicAdd(&sNext[b], 1);
                u = __builtin_amdgcn_readfirstlane(u);
                if (u >= ue) {
                    d.valid = false;
                    return;
                }
                const int32_t slice = SL == 1 ? 0 : __builtin_amdgcn_readfirstlane(u / G);
                const int32_t g = u - slice * G;
                const int32_t zb = __builtin_amdgcn_readfirstlane(sP[g] - g);
                const int32_t ze = max(zb, __builtin_amdgcn_readfirstlane(sP[g + 1] - g - 1));
                if (zb < ze) {
                    d.s = zb;
                    d.ze = ze;
                    d.len = min(BLK, ze - zb);
                    d.last = ze - zb <= BLK;
                    d.base = b * kTileBufFloats + slice * SW;
                    d.g = g;
                    d.slice = slice;
                    d.valid = true;
                    return;
                }
                store_unit(T, slice, g, true);
            }
        };
        auto advance = [&](const Desc& d) {
            Desc r = d;
            if (!d.valid) return r;
            if (!d.last) {
                r.s = d.s + d.len;
                r.len = min(BLK, d.ze - r.s);
                r.last = r.s + r.len >= d.ze;
                return r;
            }
            next_unit(r);
            return r;
        };

        // One pipeline step: multiply block j (d0: weights av0, X bv0) while
        // reading block j+1's X (offsets o1) into bv1, handing out block
        // j+2's row offsets (d2, channels ch2) into o2, and loading block
        // j+1's weights (d1) into av1 and block j+3's channels (d3) into
        // ch3.  Work for a missing block redoes block j, so that every step
        // issues the same instructions (one straight run the scheduler can
        // interleave) and the waits for loads stay exact.
        auto step = [&](const Desc& d0, const Desc& d1, const Desc& d2, const Desc& d3,
                        float (&av0)[STEPS], vec_t (&bv0)[STEPS], float (&av1)[STEPS],
                        vec_t (&bv1)[STEPS], const int32_t (&o1)[STEPS], int32_t (&o2)[STEPS],
                        int32_t ch2, int32_t& ch3) {
            load_ch(ch3, d3.valid ? d3 : d0);
            load_w(av1, d1.valid ? d1 : d0);
            offsets(o2, ch2, d2.valid ? d2 : d0);
            read_x(bv1, o1);
#pragma unroll
            for (int ks = 0; ks < STEPS; ++ks)
#pragma unroll
                for (int e = 0; e < NB; ++e) acc[e] = M::step(av0[ks], vec_el<NB>(bv0[ks], e), acc[e]);
#pragma unroll
            for (int i = 0; i < STEPS * NB; ++i) {
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // one MFMA,
                __builtin_amdgcn_sched_group_barrier(0x020, 1, 0);   // a load,
                __builtin_amdgcn_sched_group_barrier(0x002, 1, 0);   // a vector op
                __builtin_amdgcn_sched_group_barrier(0x080, 1, 0);   // and an LDS op
            }
            if (d0.last) store_unit(T, d0.slice, d0.g, false);
        };

        Desc d0;
        next_unit(d0);
        if (d0.valid) {
            Desc d1 = advance(d0);
            Desc d2 = advance(d1);
            Desc d3 = advance(d2);
            int32_t chA, chB, oA[STEPS], oB[STEPS];
            float avA[STEPS], avB[STEPS];
            vec_t bvA[STEPS], bvB[STEPS];
            // Prologue: blocks 0 and 1's offsets, block 0's weights and X,
            // block 2's channels (block j's registers use set j % 2).
            load_ch(chA, d0);
            load_ch(chB, d1.valid ? d1 : d0);
            load_w(avA, d0);
            offsets(oA, chA, d0);
            offsets(oB, chB, d1.valid ? d1 : d0);
            load_ch(chA, d2.valid ? d2 : d0);
            // Only the X reads need the tile itself.
            while (__builtin_amdgcn_readfirstlane(lds_load(&sLanded[b])) < k + 1)
                __builtin_amdgcn_s_sleep(1);
            read_x(bvA, oA);
            while (true) {
                step(d0, d1, d2, d3, avA, bvA, avB, bvB, oB, oA, chA, chB);
                if (!d1.valid) break;
                d0 = d1;
                d1 = d2;
                d2 = d3;
                d3 = advance(d3);
                step(d0, d1, d2, d3, avB, bvB, avA, bvA, oA, oB, chB, chA);
                if (!d1.valid) break;
                d0 = d1;
                d1 = d2;
                d2 = d3;
                d3 = advance(d3);
            }
        }
        // Every X read of this tile by this wave has completed (its MFMAs
        // consumed them); release the buffer.
        wait_lgkm();
        if (lane == 0) atomicAdd(&sDone[b], 1);
    }
}

// Slice width and slices per tile for a layer, or 0 when the resident-tile
// kernel does not apply: the whole tile (m rows) must fit one 64 KB buffer,
// a tile must hold at least 8 units so that few waves idle, and the total
// cost must stay below 2^31.
struct TileShape {
    int sw, sl;
};
TileShape tile_shape(const ConvArgs& a) {
    if (a.G > kTileMaxG) return {0, 0};
    for (int sw : {64, 32, 16}) {
        if (sw < (a.N == 32 ? 32 : 16)) continue;
        if (int64_t(a.m) * sw > kTileBufFloats) continue;
        // Slices per tile: as many as the buffer holds, but once a tile has 8
        // units not so many that the layer has fewer tiles than compute units
        // (each workgroup would copy a whole tile for a fraction of its units).
        int sl = 1;
        while (int64_t(a.m) * sw * sl * 2 <= kTileBufFloats && int64_t(sl) * sw < a.npix && sl < 64 &&
               (int64_t(sl) * a.G < 8 ||
                (int64_t(a.npix) + int64_t(sw) * sl * 2 - 1) / (int64_t(sw) * sl * 2) >= device_cu_count()))
            sl *= 2;
        if (int64_t(sl) * a.G < 8) continue;
        const int64_t tiles = (int64_t(a.npix) + int64_t(sw) * sl - 1) / (int64_t(sw) * sl);
        if (tiles * sl * (int64_t(a.t) + a.G) >= INT32_MAX) continue;
        return {sw, sl};
    }
    return {0, 0};
}

bool vec4_ok(const ConvArgs& a) {
    return a.HWo % 4 == 0 && (reinterpret_cast<uintptr_t>(a.x) & 15) == 0 &&
           (reinterpret_cast<uintptr_t>(a.y) & 15) == 0;
}

template <int N, int SW>
onexn_status launch_tile_sw(ConvArgs a, hipStream_t s) {
    const int64_t pt = int64_t(SW) * a.slices;
    const int64_t tiles = (int64_t(a.npix) + pt - 1) / pt;
    int64_t wgs = device_cu_count();
    if (tuning(kTunePwWgs) >= 1) wgs = tuning(kTunePwWgs);
    // (at most 2^15 workgroups keeps cost_r * L within int32 in the kernel)
    wgs = std::max<int64_t>(1, std::min<int64_t>({wgs, tiles * a.slices * a.G, int64_t(1) << 15}));
    const int64_t total = tiles * a.slices * (int64_t(a.t) + a.G);
    a.cost_q = int32_t(total / wgs);
    a.cost_r = int32_t(total % wgs);
    return with_epilogue(a, [&](auto ep) {
        constexpr bool E = decltype(ep)::value;
        if (vec4_ok(a)) return launch_grid(pw_tile_f32<N, SW, true, E>, a, wgs, s, kTileThreads);
        return launch_grid(pw_tile_f32<N, SW, false, E>, a, wgs, s, kTileThreads);
    });
}

}  // namespace

bool pw_tile_applies(const ConvArgs& a) {
    if (a.kh != 1 || a.kw != 1 || a.sh != 1 || a.sw != 1 || a.ph != 0 || a.pw != 0) return false;
    if (a.y_c != a.HWo || a.x_c != a.H * a.W) return false;   // NCHW
    if (has_epilogue(a) && int64_t(a.G) * a.N > kTileEpMax) return false;   // parameters do not fit LDS
    return (a.N == 16 || a.N == 32) && tile_shape(a).sw > 0;
}

onexn_status launch_pw_tile(ConvArgs a, hipStream_t s) {
    const TileShape ts = tile_shape(a);
    a.slices = ts.sl;
    if (a.N == 16) {
        if (ts.sw == 64) return launch_tile_sw<16, 64>(a, s);
        if (ts.sw == 32) return launch_tile_sw<16, 32>(a, s);
        return launch_tile_sw<16, 16>(a, s);
    }
    if (ts.sw == 64) return launch_tile_sw<32, 64>(a, s);
    return launch_tile_sw<32, 32>(a, s);
}

}  // namespace onexn
