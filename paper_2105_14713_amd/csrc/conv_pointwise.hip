// Pointwise (1x1, stride 1, no padding, NCHW) 1xN-pruned convolution, fp32,
// N in {16, 32}, on fp32 matrix cores.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  For a 1x1 kernel col-group g is the
// contraction Y_g[N][pixels] = D_g^T[N][kept_g] * X[I_g][pixels]: its kept
// blocks select rows of the input matrix X[channel][pixel], and the N weights
// of a block are one contiguous row of D.
//
// Work split.  A workgroup of 8 waves owns a tile of PT = 64*WPG pixels and
// 8/WPG consecutive col-groups; each col-group is computed by WPG waves, one
// 64-pixel slice each.  Input channels are walked in chunks of KC: a chunk of
// X (KC rows x PT pixels) is read once from global memory (coalesced, one
// chunk ahead) into LDS and shared by all col-groups of the workgroup, so X
// crosses L2 -> CU only G*WPG/8 times.
//
// Each wave streams its own col-group's BSR entries: the entries of a chunk
// are a contiguous run (I is ascending; the run bounds are computed once per
// wave), taken in blocks of 8 MFMA steps.  For a block the wave reads the I
// values (one coalesced load, rows handed to lane groups with ds_bpermute) and
// the weights (one coalesced load per step) straight from global memory, one
// block ahead of use, so the inner loop is 8 LDS reads of X and 8*NB MFMAs.
//
//   N = 16: v_mfma_f32_16x16x4f32, 4 kept blocks per step (lane group l/16),
//           NB = 4 column blocks per wave: MFMA column n of block e is pixel
//           4n + e of the wave's slice, so a lane reads 4 consecutive pixels.
//   N = 32: v_mfma_f32_32x32x2f32, 2 kept blocks per step, NB = 2.
#include <cstdio>
#include <cstdlib>

#include "conv_common.h"

namespace onexn {
namespace {

constexpr int kPwThreads = 512;   // 8 waves
constexpr int kPwWaves = kPwThreads / 64;
constexpr int kPwWavePx = 64;     // pixels per wave
constexpr int kPwLdsFloats = 4096;   // one X chunk buffer: 16 KB
constexpr int kPwSteps = 8;       // MFMA steps per block
constexpr int kPwMaxChunks = 64;  // channel chunks a layer may have

template <int N> struct PwMfma;
template <> struct PwMfma<16> {   // 16x16x4 f32
    typedef f32x4 acc_t;
    static constexpr int KS = 4, ACC = 4;
    __device__ static acc_t step(float a, float b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static int row(int lane, int r) { return 4 * (lane / 16) + r; }
};
template <> struct PwMfma<32> {   // 32x32x2 f32
    typedef f32x16 acc_t;
    static constexpr int KS = 2, ACC = 16;
    __device__ static acc_t step(float a, float b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
    __device__ static int row(int lane, int r) { return 8 * (r / 4) + 4 * (lane / 32) + (r % 4); }
};

template <int NB> struct VecF;
template <> struct VecF<2> { typedef float T __attribute__((ext_vector_type(2))); };
template <> struct VecF<4> { typedef f32x4 T; };

template <int N, int WPG>
struct PwShape {
    static constexpr int PT = kPwWavePx * WPG;            // pixels per workgroup
    static constexpr int S = kPwWaves / WPG;              // col-groups per workgroup
    static constexpr int KC = kPwLdsFloats / PT;          // channels per chunk
    static constexpr int NB = kPwWavePx / N;              // MFMA column blocks per wave
    static constexpr int BLK = kPwSteps * PwMfma<N>::KS;  // BSR entries per block
};

template <int N, int WPG, bool kVec4>
__global__ void __launch_bounds__(kPwThreads) __attribute__((amdgpu_waves_per_eu(4))) pw_mfma_f32(ConvArgs a) {
    typedef PwMfma<N> M;
    typedef PwShape<N, WPG> SH;
    typedef typename M::acc_t acc_t;
    constexpr int PT = SH::PT, S = SH::S, KC = SH::KC, NB = SH::NB, BLK = SH::BLK;
    constexpr int KS = M::KS, STEPS = kPwSteps;
    constexpr int QPR = PT / 4;                 // pixel quads per X row
    constexpr int RG = kPwThreads / QPR;        // X rows loaded in parallel
    constexpr int XJ = KC / RG;                 // quads per thread per chunk
    static_assert(64 / N == KS && BLK <= 64, "lane groups carry a step's kept blocks");
    static_assert(XJ >= 1 && KC % RG == 0, "tile shape");
    typedef typename VecF<NB>::T vec_t;

    __shared__ __attribute__((aligned(16))) float sX[2][KC * PT];
    __shared__ int32_t sBnd[kPwWaves][kPwMaxChunks + 1];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);   // uniform per wave
    const int32_t GS = (a.G + S - 1) / S;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t gs = L % GS;
    // This workgroup walks pixel tiles [tile0, tile0 + nt) for col-group set gs.
    const int32_t tile0 = (L / GS) * a.tpw;
    const int32_t nt = min(a.tpw, (a.npix + PT - 1) / PT - tile0);
    const int32_t g = gs * S + wave / WPG;      // this wave's col-group
    const int slice = wave % WPG;               // this wave's 64-pixel slice
    const float* __restrict__ x = static_cast<const float*>(a.x);
    const float* __restrict__ D = static_cast<const float*>(a.D);
    const int32_t nch = (a.m + KC - 1) / KC;

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

    // X loader role: pixel quad qd of a tile, rows rg, rg + RG, ...  Element e
    // of the X stream is chunk e % nch of tile tile0 + e / nch.
    const int qd = tid % QPR, rg = tid / QPR;
    f32x4 xr[XJ];
    auto fetch_x = [&](int32_t e) {
        const int32_t tile = tile0 + e / nch, c = e % nch;
        int64_t xo[4];
        bool xv[4];
#pragma unroll
        for (int q = 0; q < (kVec4 ? 1 : 4); ++q) {
            const int32_t p = tile * PT + 4 * qd + q;
            xv[q] = p < a.npix;
            const int32_t pp = xv[q] ? p : 0;
            const int32_t b = pp / a.HWo;
            xo[q] = int64_t(b) * a.x_img + (pp - b * a.HWo);
        }
#pragma unroll
        for (int j = 0; j < XJ; ++j) {
            const int32_t ch = c * KC + rg + j * RG;
            const bool chok = ch < a.m;
            const int64_t co = int64_t(ch) * a.x_c;
            if (kVec4) {
                f32x4 v = {0.f, 0.f, 0.f, 0.f};
                if (chok && xv[0]) v = *reinterpret_cast<const f32x4*>(x + xo[0] + co);
                xr[j] = v;
            } else {
#pragma unroll
                for (int q = 0; q < 4; ++q) xr[j][q] = (chok && xv[q]) ? x[xo[q] + co] : 0.f;
            }
        }
    };
    auto stash_x = [&](int buf) {
#pragma unroll
        for (int j = 0; j < XJ; ++j)
            *reinterpret_cast<f32x4*>(&sX[buf][(rg + j * RG) * PT + 4 * qd]) = xr[j];
    };

    // One block of the wave's BSR entries: [s, s + len), len <= BLK, all in
    // one channel chunk with base channel c0.
    struct Block {
        int32_t off;         // lane i < len: LDS byte offset of entry i's X row, else 0
        float av[STEPS];     // weight of step ks for this lane's (lane group, output)
    };
    const int lg = lane / N, lo = lane % N;
    auto load_block = [&](Block& bk, int32_t s, int32_t len, int32_t c0) {
        if (len <= 0) return;   // uniform: nothing left for this wave
        // Clamped indices keep every load inside the block; the selects zero
        // the entries past len (weight 0, X row 0).
        const int32_t* Ib = a.I + s;
        const float* Db = D + int64_t(s) * N;
        const int32_t ch = Ib[min(lane, len - 1)];
        bk.off = lane < len ? min(max(ch - c0, 0), KC - 1) * (PT * 4) : 0;
#pragma unroll
        for (int ks = 0; ks < STEPS; ++ks) {
            const int i = ks * KS + lg;
            const float v = Db[uint32_t(min(i, len - 1) * N + lo)];
            bk.av[ks] = i < len ? v : 0.f;
        }
    };

    acc_t acc[NB];
#pragma unroll
    for (int e = 0; e < NB; ++e)
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) acc[e][r] = 0.f;

    // Multiplies one loaded block against X chunk buffer `buf`.
    auto run_block = [&](const Block& bk, int32_t len, int buf) {
        const char* xs = reinterpret_cast<const char*>(&sX[buf][slice * kPwWavePx + NB * lo]);
        vec_t bv[STEPS];
#pragma unroll
        for (int ks = 0; ks < STEPS; ++ks) {
            const int32_t off = __builtin_amdgcn_ds_bpermute(4 * (ks * KS + lg), bk.off);
            bv[ks] = *reinterpret_cast<const vec_t*>(xs + off);
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
                        for (int e = 0; e < NB; ++e) v[e] = acc[e][r];
                        *reinterpret_cast<vec_t*>(y + yb + int64_t(o) * a.y_c) = v;
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
                        if (o < a.n) y[yb + int64_t(o) * a.y_c] = acc[e][r];
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
    __syncthreads();   // run bounds visible
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
    Pos q0 = first(0);
    Block bk0, bk1;
    load_block(bk0, q0.s, q0.len, q0.c * KC);

    fetch_x(0);
    stash_x(0);
    __syncthreads();
    const int32_t nel = nt * nch;
    for (int32_t el = 0; el < nel; ++el) {
        const int32_t tt = el / nch, c = el % nch;
        if (el + 1 < nel) fetch_x(el + 1);
        const int buf = el & 1;
        while (q0.t == tt && q0.c == c && q0.len > 0) {
            const Pos q1 = after(q0);
            load_block(bk1, q1.s, q1.len, q1.c * KC);
            run_block(bk0, q0.len, buf);
            // The next block's loads stay in flight across this block's MFMAs.
            asm volatile("" : "+v"(bk1.off));
#pragma unroll
            for (int ks = 0; ks < STEPS; ++ks) asm volatile("" : "+v"(bk1.av[ks]));
            bk0 = bk1;
            q0 = q1;
        }
        if (el + 1 < nel) stash_x((el + 1) & 1);
        __syncthreads();
        if (c == nch - 1) epilogue(tile0 + tt);
    }
}

// Waves per col-group: 1 when the layer has at least 8 col-groups, more for
// narrower layers so that no wave of a workgroup is idle.  ONEXN_PW_WPG
// overrides it for A/B measurements.
int choose_wpg(const ConvArgs& a) {
    if (const char* env = std::getenv("ONEXN_PW_WPG")) {
        const int v = std::atoi(env);
        if (v == 1 || v == 2 || v == 4 || v == 8) return v;
    }
    if (a.G >= 8) return 1;
    if (a.G >= 4) return 2;
    if (a.G >= 2) return 4;
    return 8;
}

// Pixel tiles per workgroup: one by default (measured fastest on the 28x28
// layers: a workgroup that walks several tiles serialises their X fetches);
// ONEXN_PW_TPW overrides it for A/B measurements.
int32_t choose_tpw() {
    if (const char* env = std::getenv("ONEXN_PW_TPW")) {
        const int v = std::atoi(env);
        if (v >= 1 && v <= 1024) return v;
    }
    return 1;
}

template <int N, int WPG>
onexn_status launch_pw(ConvArgs a, hipStream_t s) {
    typedef PwShape<N, WPG> SH;
    const int64_t tiles = (int64_t(a.npix) + SH::PT - 1) / SH::PT;
    const int64_t gsets = (a.G + SH::S - 1) / SH::S;
    a.tpw = choose_tpw();
    const int64_t total = ((tiles + a.tpw - 1) / a.tpw) * gsets;
    const bool vec4 = a.HWo % 4 == 0 && (reinterpret_cast<uintptr_t>(a.x) & 15) == 0 &&
                      (reinterpret_cast<uintptr_t>(a.y) & 15) == 0;
    if (vec4) return launch_grid(pw_mfma_f32<N, WPG, true>, a, total, s, kPwThreads);
    return launch_grid(pw_mfma_f32<N, WPG, false>, a, total, s, kPwThreads);
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

onexn_status launch_pointwise(ConvArgs a, onexn_dtype, onexn_dtype, hipStream_t s) {
    return a.N == 16 ? launch_pw_n<16>(a, s) : launch_pw_n<32>(a, s);
}

}  // namespace onexn
