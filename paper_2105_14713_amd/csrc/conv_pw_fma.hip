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
// Work split.  A workgroup computes one pixel tile (64 lanes x PPT pixels,
// 64 apart) for a set of GSW col-groups: wave w takes col-group w % GSW of the
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
#include <cstdlib>

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kFThreads = 256;
constexpr int kFWin = 256;   // kept blocks per staged window (per wave)

template <int N, int PPT, int GSW>
__global__ void __launch_bounds__(kFThreads) pw_fma(ConvArgs a) {
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
    const int32_t tile = L / gsets;
    const int32_t g = (L - tile * gsets) * GSW + gw;
    int32_t zb = 0, ze = 0;
    if (g < a.G) group_range(a, g, zb, ze);
    // This wave's contiguous share of the col-group's kept blocks.
    const int32_t per = (ze - zb + KSPLIT - 1) / KSPLIT;
    const int32_t z0 = min(ze, zb + kq * per), z1 = min(ze, z0 + per);
    const int32_t batch = a.npix / a.HWo;
    const int32_t xbytes = int32_t(int64_t(batch) * a.x_img * 4);

    uint32_t xo[PPT];   // byte offset of the lane's pixels at channel 0 (past the input: invalid)
    int64_t yo[PPT];    // element offset in y at channel 0, or -1
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
        const int32_t p = tile * TP + i * 64 + lane;
        xo[i] = uint32_t(xbytes);
        yo[i] = -1;
        if (p < a.npix) {
            const int32_t b = p / a.HWo, hw = p - b * a.HWo;
            xo[i] = uint32_t((int64_t(b) * a.x_img + hw) * 4);
            yo[i] = int64_t(b) * a.y_img + hw;
        }
    }

    const __amdgpu_buffer_rsrc_t rX =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.x), 0, xbytes, kRawBufferFlags);
    const v4i32 rI = buffer_rsrc(a.I, z1 * 4);
    const v4i32 rD = buffer_rsrc(a.D, z1 * N * 4);
    const int32_t* const wI = sI[wave];
    const float* const wD = sD[wave];

    float acc[N][PPT];
#pragma unroll
    for (int o = 0; o < N; ++o)
#pragma unroll
        for (int i = 0; i < PPT; ++i) acc[o][i] = 0.f;

    // Blocks are taken in batches of kFB: lane j < kFB of the wave reads
    // block j's channel, every lane then issues the batch's input loads at
    // once, and the next batch's loads are issued before this batch's
    // multiply-adds, so a wave keeps up to 2 kFB PPT loads in flight (kFB
    // shrinks as PPT grows, to keep the register count and occupancy).
    constexpr int kFB = PPT >= 4 ? 4 : 16 / PPT;   // loads per batch stay at 16 (or fewer)
    struct Batch {
        float xv[kFB][PPT];
    };
    // Entries past the share (j >= cnt) and channels outside [0, m) take the
    // value 0 (their loads stay inside the input), so a partial batch adds
    // nothing; the window's weights past the share are zeros (range-checked
    // copies of whole 64-entry blocks).
    auto issue = [&](Batch& bt, int32_t e, int32_t cnt) {
        const int32_t chv = wI[e + (lane & (kFB - 1))];
#pragma unroll
        for (int j = 0; j < kFB; ++j) {
            const int32_t ch = __builtin_amdgcn_readlane(chv, j);
            const bool ok = j < cnt && uint32_t(ch) < uint32_t(a.m);
            const int32_t choff = ok ? ch * a.HWo * 4 : 0;
#pragma unroll
            for (int i = 0; i < PPT; ++i) {
                const float v = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rX, int32_t(xo[i]), choff, 0));
                bt.xv[j][i] = ok ? v : 0.f;
            }
        }
    };
    auto consume = [&](const Batch& bt, int32_t e) {
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

    for (int32_t w0 = z0; w0 < z1; w0 += kFWin) {
        const int32_t nw = min(kFWin, z1 - w0);
        for (int32_t e0 = 0; e0 < nw; e0 += 64)
            copy4_to_lds(rI, (const lds_char*)(wI + e0), (w0 + e0 + lane) * 4, 0);
        for (int32_t e0 = 0; e0 < nw * N; e0 += 64)
            copy4_to_lds(rD, (const lds_char*)(wD + e0), (w0 * N + e0 + lane) * 4, 0);
        vm_wait<0>();   // the window is in this wave's LDS
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
        wait_lgkm();    // this wave's reads of the window are done before it is refilled
    }

    if constexpr (KSPLIT > 1) {
#pragma unroll
        for (int o = 0; o < N; ++o)
#pragma unroll
            for (int i = 0; i < PPT; ++i) sR[((wave * N + o) * PPT + i) * 64 + lane] = acc[o][i];
        __syncthreads();
        if (kq != 0) return;
#pragma unroll
        for (int o = 0; o < N; ++o)
#pragma unroll
            for (int i = 0; i < PPT; ++i)
#pragma unroll
                for (int k = 1; k < KSPLIT; ++k) acc[o][i] += sR[(((wave + k * GSW) * N + o) * PPT + i) * 64 + lane];
    }
    if (g >= a.G) return;

    float* __restrict__ y = static_cast<float*>(a.y);
#pragma unroll
    for (int o = 0; o < N; ++o) {
        const int32_t oc = g * N + o;
        if (oc >= a.n) continue;
#pragma unroll
        for (int i = 0; i < PPT; ++i)
            if (yo[i] >= 0) y[yo[i] + int64_t(oc) * a.y_c] = acc[o][i];
    }
}

template <int N, int PPT, int GSW>
onexn_status launch_cfg(ConvArgs a, hipStream_t s) {
    const int64_t tiles = (int64_t(a.npix) + 64 * PPT - 1) / (64 * PPT);
    const int64_t gsets = (a.G + GSW - 1) / GSW;
    return launch_grid(pw_fma<N, PPT, GSW>, a, tiles * gsets, s, kFThreads);
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
    if (const char* env = std::getenv("ONEXN_FMA_TILE")) choice = std::atoi(env);   // testing
    if (choice == 0) {
        if (tiles(256) * gs4 >= want) choice = 1;
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
