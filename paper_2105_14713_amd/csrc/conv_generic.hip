// Generic kernels of the 1xN-pruned convolution: any kernel size, stride,
// padding, layout and dtype.  One workgroup computes one (pixel tile,
// col-group) output tile, gathering the col-group's kept input channels
// straight from global memory.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the dense contraction
//     Y_g[N][pixels] = A_g[N][K_g] * B_g[K_g][pixels],   K_g = kept_g * kh * kw
// where row kappa = (z, q, r) of B_g is input channel I[z] shifted by tap
// (q, r) under every output pixel (an implicit im2col restricted to the kept
// channels), and A_g[o][kappa] = D[z][o][q][r].
//
//   fma_conv   N <= 8.  One lane per output pixel (or a few); the N weights of
//              a block are wave-uniform (scalar loads); every gathered input
//              value feeds N fused multiply-adds.
//   mfma_conv  N in {16, 32}.  The contraction runs on matrix cores: fp32
//              (v_mfma_f32_16x16x4f32 / 32x32x2f32) or bf16 with fp32
//              accumulation (v_mfma_f32_16x16x32_bf16 / 32x32x16_bf16).  The
//              gathered B_g tile and the A_g tile are staged through LDS in
//              double-buffered chunks of the kappa dimension.
#include "conv_common.h"

namespace onexn {
namespace {

// ---------------------------------------------------------------------------
// fma_conv: N <= 8.
// ---------------------------------------------------------------------------

// KS > 1 splits each col-group's contraction over KS slices of the
// workgroup (whole waves each), for layers with few output pixels and long
// col-groups; the slices' partial sums are added through LDS.
template <int N, int PPT, int KS, bool kUnit, typename TX, typename TY>
__global__ void __launch_bounds__(kThreads) fma_conv(ConvArgs a) {
    constexpr int U = 8;   // kappa per batch: U * PPT gathered loads in flight per lane
    constexpr int TPS = kThreads / KS;   // threads per contraction slice
    static_assert(TPS % 64 == 0, "a slice is whole waves");
    __shared__ float sR[KS > 1 ? (KS - 1) * TPS * PPT * N : 1];
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t g = L % a.G;
    const int32_t tile = L / a.G;
    const int kq = __builtin_amdgcn_readfirstlane(int(threadIdx.x) / TPS);
    const int pt = int(threadIdx.x) % TPS;
    int32_t zb, ze;
    group_range(a, g, zb, ze);
    const int32_t Kg = (ze - zb) * a.KK;
    const int32_t per = (Kg + KS - 1) / KS;
    const int32_t kbeg = min(Kg, kq * per), kend = min(Kg, kbeg + per);

    const TX* __restrict__ x = static_cast<const TX*>(a.x);
    const TX* __restrict__ D = static_cast<const TX*>(a.D);
    PixelPos pp[PPT];
    float acc[PPT][N];
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
        pp[i] = pixel_pos(a, tile * (TPS * PPT) + i * TPS + pt);
#pragma unroll
        for (int o = 0; o < N; ++o) acc[i][o] = 0.f;
    }

    KapWalk w = walk_at<kUnit>(a, kbeg);
    for (int32_t k0 = kbeg; k0 < kend; k0 += U) {
        int32_t cs[U];
        KapWalk ws[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            cs[u] = walk_channel(a, w, zb, ze, k0 + u < kend);
            ws[u] = w;
            walk_step<kUnit>(a, w);
        }
        float xv[U][PPT];
#pragma unroll
        for (int u = 0; u < U; ++u)
#pragma unroll
            for (int i = 0; i < PPT; ++i)
                xv[u][i] = cs[u] >= 0 ? to_f32(gather_x<kUnit>(a, x, pp[i], cs[u], ws[u])) : 0.f;
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (cs[u] < 0) continue;
            const TX* __restrict__ wp =
                D + (int64_t(zb + ws[u].zz) * N) * a.KK + ws[u].q * a.kw + ws[u].r;
            float wv[N];
#pragma unroll
            for (int o = 0; o < N; ++o) wv[o] = to_f32(wp[o * a.KK]);
#pragma unroll
            for (int i = 0; i < PPT; ++i)
#pragma unroll
                for (int o = 0; o < N; ++o) acc[i][o] = fmaf(wv[o], xv[u][i], acc[i][o]);
        }
    }

    if constexpr (KS > 1) {
        if (kq > 0) {
#pragma unroll
            for (int i = 0; i < PPT; ++i)
#pragma unroll
                for (int o = 0; o < N; ++o) sR[(((kq - 1) * PPT + i) * N + o) * TPS + pt] = acc[i][o];
        }
        __syncthreads();
        if (kq > 0) return;
#pragma unroll
        for (int k = 1; k < KS; ++k)
#pragma unroll
            for (int i = 0; i < PPT; ++i)
#pragma unroll
                for (int o = 0; o < N; ++o) acc[i][o] += sR[(((k - 1) * PPT + i) * N + o) * TPS + pt];
    }

    TY* __restrict__ y = static_cast<TY*>(a.y);
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
        if (!pp[i].valid) continue;
#pragma unroll
        for (int o = 0; o < N; ++o) {
            const int32_t oc = g * N + o;
            if (oc < a.n) store_out(&y[pp[i].ybase + int64_t(oc) * a.y_c], from_f32<TY>(epilogue(a, oc, acc[i][o])));
        }
    }
}

// ---------------------------------------------------------------------------
// mfma_conv: N in {16, 32}; fp32 or bf16 inputs, fp32 accumulation.
// ---------------------------------------------------------------------------

template <int N, int WPX, bool kUnit, typename TX, typename TY>
__global__ void __launch_bounds__(kThreads) mfma_conv(ConvArgs a) {
    constexpr bool kBf16 = std::is_same<TX, uint16_t>::value;
    constexpr int KC = kBf16 ? 32 : 16;            // kappa per chunk
    constexpr int ROW = KC + (kBf16 ? 8 : 4);      // LDS row pitch in elements (80 bytes)
    constexpr int PT = 4 * WPX;                    // pixels per workgroup
    constexpr int TPP = kThreads / PT;             // threads sharing one pixel row
    constexpr int KPT = KC / TPP;                  // kappa gathered per thread per chunk
    constexpr int MB = (N == 16) ? 16 : 32;        // MFMA output block edge
    constexpr int NB = WPX / MB;                   // MFMA column blocks per wave
    constexpr int AE = N * KC / kThreads;          // A elements per thread per chunk
    static_assert(KPT % 8 == 0 || (!kBf16 && KPT % 4 == 0), "vector LDS stores");
    static_assert(AE >= 1 && NB >= 1, "tile shape");

    __shared__ __attribute__((aligned(16))) TX sB[2][PT * ROW];
    __shared__ __attribute__((aligned(16))) TX sA[2][N * ROW];

    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t g = L % a.G;
    const int32_t tile = L / a.G;
    int32_t zb, ze;
    group_range(a, g, zb, ze);
    const int32_t Kg = (ze - zb) * a.KK;
    const int32_t nchunks = (Kg + KC - 1) / KC;

    const TX* __restrict__ x = static_cast<const TX*>(a.x);
    const TX* __restrict__ D = static_cast<const TX*>(a.D);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;

    // Gather role: pixel row `prow` of the tile, kappa sub-range `kofs`
    // (the same for all lanes of a wave).
    const int prow = tid % PT;
    const int kofs = __builtin_amdgcn_readfirstlane((tid / PT) * KPT);
    const PixelPos pp = pixel_pos(a, tile * PT + prow);

    TX rb[KPT];     // B prefetch registers
    TX ra[AE];      // A prefetch registers

    auto fetch = [&](int32_t chunk) {
        const int32_t k0 = chunk * KC;
        // B: KPT consecutive kappa of this thread's pixel.
        const int32_t kap0 = k0 + kofs;
        KapWalk w = walk_at<kUnit>(a, kap0);
        int32_t cs[KPT];
        KapWalk ws[KPT];
#pragma unroll
        for (int i = 0; i < KPT; ++i) {
            cs[i] = walk_channel(a, w, zb, ze, kap0 + i < Kg);
            ws[i] = w;
            walk_step<kUnit>(a, w);
        }
#pragma unroll
        for (int i = 0; i < KPT; ++i)
            rb[i] = cs[i] >= 0 ? gather_x<kUnit>(a, x, pp, cs[i], ws[i]) : TX(0);
        // A: element e -> (o = e % N, kk = e / N) of the N x KC chunk.
#pragma unroll
        for (int j = 0; j < AE; ++j) {
            const int e = tid + j * kThreads;
            const int o = e % N, kk = e / N;
            const int32_t k = k0 + kk;
            TX v = TX(0);
            if (k < Kg) {
                if (kUnit) {   // the chunk's blocks are contiguous: [zb + k0, +KC) x N
                    v = D[int64_t(zb + k0) * N + e];
                } else {
                    const int32_t z2 = k / a.KK, tp = k - z2 * a.KK;
                    v = D[(int64_t(zb + z2) * N + o) * a.KK + tp];
                }
            }
            ra[j] = v;
        }
    };
    auto stash = [&](int buf) {
        TX* dstB = &sB[buf][prow * ROW + kofs];
        if constexpr (kBf16) {
#pragma unroll
            for (int i = 0; i < KPT; i += 8) {
                u32x4 v;
                v.x = uint32_t(rb[i + 0]) | (uint32_t(rb[i + 1]) << 16);
                v.y = uint32_t(rb[i + 2]) | (uint32_t(rb[i + 3]) << 16);
                v.z = uint32_t(rb[i + 4]) | (uint32_t(rb[i + 5]) << 16);
                v.w = uint32_t(rb[i + 6]) | (uint32_t(rb[i + 7]) << 16);
                *reinterpret_cast<u32x4*>(dstB + i) = v;
            }
        } else {
#pragma unroll
            for (int i = 0; i < KPT; i += 4) {
                f32x4 v = {rb[i], rb[i + 1], rb[i + 2], rb[i + 3]};
                *reinterpret_cast<f32x4*>(dstB + i) = v;
            }
        }
#pragma unroll
        for (int j = 0; j < AE; ++j) {
            const int e = tid + j * kThreads;
            sA[buf][(e % N) * ROW + e / N] = ra[j];
        }
    };

    typedef typename std::conditional<MB == 16, f32x4, f32x16>::type acc_t;
    acc_t acc[NB];
#pragma unroll
    for (int j = 0; j < NB; ++j)
#pragma unroll
        for (int r = 0; r < int(sizeof(acc_t) / 4); ++r) acc[j][r] = 0.f;

    auto compute = [&](int buf) {
        const TX* A = sA[buf];
        const TX* B = sB[buf] + (wave * WPX) * ROW;
        if constexpr (!kBf16 && MB == 16) {
            // 16x16x4: lane holds row l%16, kappa 4*(l/16) + s at step s.
            const f32x4 av = *reinterpret_cast<const f32x4*>(A + (lane % 16) * ROW + 4 * (lane / 16));
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const f32x4 bv = *reinterpret_cast<const f32x4*>(B + (16 * j + lane % 16) * ROW + 4 * (lane / 16));
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    acc[j] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[s], bv[s], acc[j], 0, 0, 0);
            }
        } else if constexpr (!kBf16) {
            // 32x32x2: lane holds row l%32, kappa 8*(l/32) + s at step s.
            const float* ap = reinterpret_cast<const float*>(A) + (lane % 32) * ROW + 8 * (lane / 32);
            const f32x4 a0 = *reinterpret_cast<const f32x4*>(ap);
            const f32x4 a1 = *reinterpret_cast<const f32x4*>(ap + 4);
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const float* bp = reinterpret_cast<const float*>(B) + (32 * j + lane % 32) * ROW + 8 * (lane / 32);
                const f32x4 b0 = *reinterpret_cast<const f32x4*>(bp);
                const f32x4 b1 = *reinterpret_cast<const f32x4*>(bp + 4);
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a0[s], b0[s], acc[j], 0, 0, 0);
#pragma unroll
                for (int s = 0; s < 4; ++s)
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x2f32(a1[s], b1[s], acc[j], 0, 0, 0);
            }
        } else if constexpr (MB == 16) {
            // 16x16x32 bf16: lane holds row l%16, kappa 8*(l/16) .. +7.
            const bf16x8 av = *reinterpret_cast<const bf16x8*>(A + (lane % 16) * ROW + 8 * (lane / 16));
#pragma unroll
            for (int j = 0; j < NB; ++j) {
                const bf16x8 bv = *reinterpret_cast<const bf16x8*>(B + (16 * j + lane % 16) * ROW + 8 * (lane / 16));
                acc[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(av, bv, acc[j], 0, 0, 0);
            }
        } else {
            // 32x32x16 bf16: lane holds row l%32, kappa 16*u + 8*(l/32) .. +7.
#pragma unroll
            for (int u = 0; u < 2; ++u) {
                const bf16x8 av = *reinterpret_cast<const bf16x8*>(A + (lane % 32) * ROW + 16 * u + 8 * (lane / 32));
#pragma unroll
                for (int j = 0; j < NB; ++j) {
                    const bf16x8 bv = *reinterpret_cast<const bf16x8*>(B + (32 * j + lane % 32) * ROW + 16 * u + 8 * (lane / 32));
                    acc[j] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(av, bv, acc[j], 0, 0, 0);
                }
            }
        }
    };

    if (nchunks > 0) {
        fetch(0);
        stash(0);
        __syncthreads();
        for (int32_t ch = 0; ch < nchunks; ++ch) {
            const bool more = ch + 1 < nchunks;
            if (more) fetch(ch + 1);
            compute(ch & 1);
            if (more) stash((ch + 1) & 1);
            __syncthreads();
        }
    }

    // Epilogue: MFMA output (row, col) -> (output channel g*N + row, pixel col).
    TY* __restrict__ y = static_cast<TY*>(a.y);
#pragma unroll
    for (int j = 0; j < NB; ++j) {
        const int col = (MB == 16) ? (lane % 16) : (lane % 32);
        const PixelPos op = pixel_pos(a, tile * PT + wave * WPX + MB * j + col);
        if (!op.valid) continue;
#pragma unroll
        for (int r = 0; r < int(sizeof(acc_t) / 4); ++r) {
            const int row = (MB == 16) ? (4 * (lane / 16) + r) : (8 * (r / 4) + 4 * (lane / 32) + (r % 4));
            const int32_t oc = g * N + row;
            if (oc < a.n) store_out(&y[op.ybase + int64_t(oc) * a.y_c], from_f32<TY>(epilogue(a, oc, acc[j][r])));
        }
    }
}

// ---------------------------------------------------------------------------
// Host dispatch.
// ---------------------------------------------------------------------------

template <typename TX, typename TY, bool kUnit>
onexn_status launch_typed(ConvArgs a, hipStream_t stream) {
    const int64_t npix = a.npix;
    auto grid_for = [&](int64_t pt) { return ((npix + pt - 1) / pt) * a.G; };
    const int64_t big_grid_min = 2 * 256;   // aim for >= 2 workgroups per CU
    auto go = [&](auto kernel, int64_t pt) { return launch_grid(kernel, a, grid_for(pt), stream); };
    // N <= 8: several pixels per lane when the grid is large, one pixel per
    // lane next, and for small grids 64-pixel tiles with the contraction split
    // over the four waves (if each slice keeps at least a few batches).
    auto go_fma = [&](auto n_const) {
        constexpr int NN = decltype(n_const)::value;
        constexpr int WIDE = NN == 8 ? 2 : 4;
        if (grid_for(256 * WIDE) >= big_grid_min) return go(fma_conv<NN, WIDE, 1, kUnit, TX, TY>, 256 * WIDE);
        const int64_t kg = a.G > 0 ? int64_t(a.t) / a.G * a.KK : 0;
        if (grid_for(256) >= big_grid_min || kg < 4 * 8 * 4) return go(fma_conv<NN, 1, 1, kUnit, TX, TY>, 256);
        return go(fma_conv<NN, 1, 4, kUnit, TX, TY>, 64);
    };
    switch (a.N) {
        case 16:
            if (grid_for(256) >= big_grid_min) return go(mfma_conv<16, 64, kUnit, TX, TY>, 256);
            return go(mfma_conv<16, 32, kUnit, TX, TY>, 128);
        case 32:
            if (grid_for(256) >= big_grid_min) return go(mfma_conv<32, 64, kUnit, TX, TY>, 256);
            return go(mfma_conv<32, 32, kUnit, TX, TY>, 128);
        case 1: return go_fma(std::integral_constant<int, 1>());
        case 2: return go_fma(std::integral_constant<int, 2>());
        case 4: return go_fma(std::integral_constant<int, 4>());
        case 8: return go_fma(std::integral_constant<int, 8>());
    }
    return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: N=%d is not supported", a.N);
}

template <typename TX, typename TY>
onexn_status launch_dtype(const ConvArgs& a, hipStream_t s) {
    const bool unit = a.kh == 1 && a.kw == 1 && a.ph == 0 && a.pw == 0;
    return unit ? launch_typed<TX, TY, true>(a, s) : launch_typed<TX, TY, false>(a, s);
}

}  // namespace

onexn_status launch_generic(ConvArgs a, onexn_dtype xdt, onexn_dtype ydt, hipStream_t s) {
    if (xdt == ONEXN_F32) return launch_dtype<float, float>(a, s);
    if (ydt == ONEXN_BF16) return launch_dtype<uint16_t, uint16_t>(a, s);
    return launch_dtype<uint16_t, float>(a, s);
}

}  // namespace onexn
