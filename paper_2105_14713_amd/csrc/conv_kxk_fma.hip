// 3x3 1xN-pruned convolution (any stride and padding), fp32, NCHW, N in
// {1, 2, 4, 8}: per-lane fused multiply-adds with the taps unrolled.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Kept block z of col-group g holds the
// 3x3 kernels of the group's N output channels for input channel I[z]
// (D[z][N][3][3]); an output pixel's N values of the group are
//     Y[o][pixel] = sum_z sum_{dy,dx} D[z][o][dy][dx] * X[I[z]][ih0+dy][iw0+dx].
// At N <= 8 a matrix-core tile would be mostly padding, so a lane owns one
// output pixel and the N outputs of the wave's col-group, and each input
// value it reads feeds N fused multiply-adds.
//
// Per lane, the byte offsets of the pixel's nine input taps are computed once
// (an offset past the input stands for a tap in the zero padding or a pixel
// past the last image: range-checked buffer loads return zeros there); a kept
// block then costs nine buffer loads, whose channel offset is the scalar
// offset, and 9 N multiply-adds whose weights are wave-uniform (scalar
// registers).  Blocks are taken two at a time, the next pair's loads issued
// before the current pair's multiply-adds.  Channels outside [0, m) and
// blocks past the col-group are skipped (a uniform branch), so they add
// nothing, not even zero times their weights.
//
// Work split.  A unit is (64 consecutive output pixels, col-group).  A
// workgroup of four waves takes four col-groups of one pixel block, or, for
// layers with few pixels (KSPLIT = 4), one unit whose kept blocks the four
// waves share, adding their partial sums through LDS.

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kKFThreads = 256;
constexpr int kKFTaps = 9;
constexpr int kKFPair = 2;   // kept blocks per pipeline stage

template <int N, int KSPLIT, bool kEp>
__global__ void __launch_bounds__(kKFThreads) kxk_fma(ConvArgs a) {
    constexpr int UPW = 4 / KSPLIT;   // units per workgroup
    constexpr int RED = KSPLIT > 1 ? 4 * N * 64 : 1;
    __shared__ float sR[RED];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int uw = wave / KSPLIT, kq = wave % KSPLIT;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    // Units pixel-block-major, so the workgroups that read the same pixels
    // run on one XCD.
    const int32_t gsets = (a.G + UPW - 1) / UPW;
    const int32_t pb = L / gsets;
    const int32_t g = (L - pb * gsets) * UPW + uw;
    int32_t zb = 0, ze = 0;
    if (g < a.G) group_range(a, g, zb, ze);
    const int32_t per = (ze - zb + KSPLIT - 1) / KSPLIT;
    const int32_t z0 = min(ze, zb + kq * per), z1 = min(ze, z0 + per);

    const int32_t p = pb * 64 + lane;
    const bool valid = p < a.npix;
    const int32_t pp = valid ? p : 0;
    const int32_t b = pp / a.HWo, hw = pp - b * a.HWo;
    const int32_t oh = hw / a.Wo, ow = hw - oh * a.Wo;
    const int32_t ih0 = oh * a.sh - a.ph, iw0 = ow * a.sw - a.pw;
    const int32_t batch = a.npix / a.HWo;
    const int32_t xbytes = int32_t(int64_t(batch) * a.x_img * 4);
    // Tap offsets at channel 0 (bytes); past the input where there is no tap.
    uint32_t to[kKFTaps];
#pragma unroll
    for (int t = 0; t < kKFTaps; ++t) {
        const int32_t ih = ih0 + t / 3, iw = iw0 + t % 3;
        const bool in = valid && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
        to[t] = in ? uint32_t((int64_t(b) * a.x_img + int64_t(ih) * a.W + iw) * 4) : kBufferOutOfRange;
    }
    const __amdgpu_buffer_rsrc_t rX = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.x), 0, __builtin_amdgcn_readfirstlane(xbytes), kRawBufferFlags);
    const uint32_t chb = uint32_t(a.x_c) * 4;   // bytes between input channels
    const float* __restrict__ D = static_cast<const float*>(a.D);
    const int32_t* __restrict__ I = a.I;

    float acc[N];
#pragma unroll
    for (int o = 0; o < N; ++o) acc[o] = 0.f;

    // The input values of a pair of kept blocks (a block past z1 or with an
    // invalid channel loads from an offset past the input: zeros).
    float xv[2][kKFPair][kKFTaps];
    bool use[2][kKFPair];   // wave-uniform: the block exists and its channel is in [0, m)
    auto issue = [&](int sl, int32_t z) __attribute__((always_inline)) {
#pragma unroll
        for (int k = 0; k < kKFPair; ++k) {
            const int32_t zk = z + k;
            const int32_t c = zk < z1 ? I[zk] : -1;
            const bool ok = uint32_t(c) < uint32_t(a.m);
            use[sl][k] = ok;
            const uint32_t so = ok ? uint32_t(c) * chb : 0u;
#pragma unroll
            for (int t = 0; t < kKFTaps; ++t)
                xv[sl][k][t] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rX, int32_t(ok ? to[t] : kBufferOutOfRange), int32_t(so), 0));
        }
    };
    auto consume = [&](int sl, int32_t z) __attribute__((always_inline)) {
#pragma unroll
        for (int k = 0; k < kKFPair; ++k) {
            if (!use[sl][k]) continue;   // uniform: nothing to add (not even 0 * weight)
            const float* w = D + int64_t(z + k) * (N * kKFTaps);
#pragma unroll
            for (int o = 0; o < N; ++o)
#pragma unroll
                for (int t = 0; t < kKFTaps; ++t) acc[o] = fmaf(w[o * kKFTaps + t], xv[sl][k][t], acc[o]);
        }
    };

    // Pairs in twos, each issued one pair ahead of its multiply-adds; whole
    // periods keep the register slots compile-time.
    const int32_t npairs = (z1 - z0 + kKFPair - 1) / kKFPair;
    if (npairs > 0) {
        issue(0, z0);
        for (int32_t j = 0; j < npairs; j += 2) {
            const int32_t z = z0 + j * kKFPair;
            __builtin_amdgcn_sched_barrier(0);
            issue(1, z + kKFPair);
            __builtin_amdgcn_sched_barrier(0);
            consume(0, z);
            if (j + 1 >= npairs) break;
            __builtin_amdgcn_sched_barrier(0);
            issue(0, z + 2 * kKFPair);
            __builtin_amdgcn_sched_barrier(0);
            consume(1, z + kKFPair);
        }
    }

    if constexpr (KSPLIT > 1) {
#pragma unroll
        for (int o = 0; o < N; ++o) sR[(wave * N + o) * 64 + lane] = acc[o];
        __syncthreads();
        if (kq != 0) return;
#pragma unroll
        for (int o = 0; o < N; ++o)
#pragma unroll
            for (int k = 1; k < KSPLIT; ++k) acc[o] += sR[((wave + k) * N + o) * 64 + lane];
    }
    if (!valid || g >= a.G) return;
    float* __restrict__ y = static_cast<float*>(a.y);
    const int64_t yb = int64_t(b) * a.y_img + hw;
#pragma unroll
    for (int o = 0; o < N; ++o) {
        const int32_t oc = g * N + o;
        if (oc < a.n) store_out(&y[yb + int64_t(oc) * a.y_c], epilogue<kEp>(a, oc, acc[o]));
    }
}

template <int N>
onexn_status launch_n(ConvArgs a, hipStream_t s) {
    const int64_t pblocks = (int64_t(a.npix) + 63) / 64;
    // Split the contraction over the workgroup's waves when four col-groups
    // per workgroup would give the compute units fewer than 8 workgroups each
    // (3x3 512->512 at 7x7, batch 64, N = 4: 384 us split, 436 us not;
    // 64->64 at 56x56: 243 us not split, 304 us split).
    int ksplit = pblocks * ((a.G + 3) / 4) < 8 * int64_t(device_cu_count()) ? 4 : 1;
    if (tuning(kTuneKxfSplit) >= 1) ksplit = tuning(kTuneKxfSplit) >= 4 ? 4 : 1;
    return with_epilogue(a, [&](auto ep) {
        constexpr bool E = decltype(ep)::value;
        if (ksplit == 4) return launch_grid(kxk_fma<N, 4, E>, a, pblocks * a.G, s, kKFThreads);
        return launch_grid(kxk_fma<N, 1, E>, a, pblocks * ((a.G + 3) / 4), s, kKFThreads);
    });
}

}  // namespace

bool kxk_fma_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_F32 || ydt != ONEXN_F32 || layout != ONEXN_NCHW) return false;
    if (a.N != 1 && a.N != 2 && a.N != 4 && a.N != 8) return false;
    if (a.kh != 3 || a.kw != 3) return false;
    const int64_t batch = a.npix / a.HWo;
    if (batch * a.x_img * 4 >= (int64_t(1) << 31)) return false;   // 32-bit buffer offsets
    return true;
}

onexn_status launch_kxk_fma(ConvArgs a, hipStream_t s) {
    switch (a.N) {
        case 1: return launch_n<1>(a, s);
        case 2: return launch_n<2>(a, s);
        case 4: return launch_n<4>(a, s);
        default: return launch_n<8>(a, s);
    }
}

}  // namespace onexn
