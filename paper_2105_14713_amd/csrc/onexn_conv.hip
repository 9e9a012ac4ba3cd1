// Forward convolution of a 1xN-pruned layer on gfx950 (MI355X).
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713).  Sec. 3.4, Eq. 8: every col-group g of N consecutive
// (rearranged) output channels only touches the input channels I[P[g]] ..
// I[P[g+1]-1], each with one dense N x kh x kw block D[z].  So col-group g is a
// dense contraction
//     Y_g[N][pixels] = A_g[N][K_g] * B_g[K_g][pixels],   K_g = kept_g * kh * kw
// where row kappa = (z, q, r) of B_g is input channel I[z] shifted by tap
// (q, r) under every output pixel (an implicit im2col restricted to the kept
// channels), and A_g[o][kappa] = D[z][o][q][r].
//
// Kernels
//   fma_conv   N <= 8.  One lane per output pixel (or a few), the N weights
//              of a block are wave-uniform (scalar loads), every gathered input
//              value feeds N fused multiply-adds.
//   mfma_conv  N in {16, 32}.  The contraction runs on matrix cores: fp32
//              (v_mfma_f32_16x16x4f32 / 32x32x2f32) or bf16 with fp32
//              accumulation (v_mfma_f32_16x16x32_bf16 / 32x32x16_bf16).  The
//              gathered B_g tile and the A_g tile are staged through LDS in
//              double-buffered chunks of the kappa dimension.
//
// One workgroup computes one (pixel tile, col-group) output tile.  Workgroup
// ids are remapped so that the col-groups of a pixel tile run back to back
// on the same XCD, which keeps that tile's input rows in the XCD's L2 while
// the other col-groups read them.
#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "onexn_internal.h"

namespace onexn {
namespace {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x16 __attribute__((ext_vector_type(16)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

constexpr int kThreads = 256;   // 4 waves of 64
constexpr int kXcds = 8;        // MI355X dispatches workgroups round-robin over 8 XCDs

struct ConvArgs {
    const int32_t* P;
    const int32_t* I;
    const void* D;
    const void* x;
    void* y;
    int32_t n, m, kh, kw, KK, N, G;
    int32_t H, W, Ho, Wo, HWo;
    int32_t sh, sw, ph, pw;
    int32_t t;          // entries of I (kept blocks)
    int64_t npix;       // batch * Ho * Wo
    int64_t x_img;      // elements per input image
    int32_t x_c, x_row, x_col;
    int64_t y_img;      // elements per output image
    int32_t y_c, y_pix;
    int32_t total;      // workgroups = pixel tiles * G
};

// ---------------------------------------------------------------------------
// Element helpers.  bf16 is carried as raw uint16_t bits.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// fp32 -> bf16, round to nearest even (NaN stays a quiet NaN).
__device__ __forceinline__ uint16_t f32_to_bf16(float f) {
    uint32_t u = __float_as_uint(f);
    if ((u & 0x7fffffffu) > 0x7f800000u) return uint16_t((u >> 16) | 0x40u);
    u += 0x7fffu + ((u >> 16) & 1u);
    return uint16_t(u >> 16);
}

template <typename T> __device__ __forceinline__ T from_f32(float v);
template <> __device__ __forceinline__ float from_f32<float>(float v) { return v; }
template <> __device__ __forceinline__ uint16_t from_f32<uint16_t>(float v) { return f32_to_bf16(v); }

// Physical workgroup id -> logical id such that each XCD gets a contiguous
// range of logical ids (workgroup i runs on XCD i % 8).
__device__ __forceinline__ int32_t xcd_remap(int32_t i, int32_t total) {
    const int32_t x = i % kXcds, local = i / kXcds;
    const int32_t q = total / kXcds, rmd = total % kXcds;
    return x * q + min(x, rmd) + local;
}

// Kept-block range of col-group g, clamped to [0, t].
__device__ __forceinline__ void group_range(const ConvArgs& a, int32_t g, int32_t& zb, int32_t& ze) {
    zb = a.P[g];
    ze = a.P[g + 1];
    zb = max(0, min(zb, a.t));
    ze = max(zb, min(ze, a.t));
}

struct PixelPos {
    int64_t xbase;   // offset of the pixel's image in x
    int64_t ybase;   // offset of the pixel in y, channel 0
    int32_t ih0, iw0;
    bool valid;
};

__device__ __forceinline__ PixelPos pixel_pos(const ConvArgs& a, int64_t p) {
    PixelPos r;
    r.valid = p < a.npix;
    if (!r.valid) p = 0;
    const int64_t b = p / a.HWo;
    const int32_t hw = int32_t(p - b * a.HWo);
    const int32_t oh = hw / a.Wo, ow = hw - (hw / a.Wo) * a.Wo;
    r.xbase = b * a.x_img;
    r.ybase = b * a.y_img + int64_t(hw) * a.y_pix;
    r.ih0 = oh * a.sh - a.ph;
    r.iw0 = ow * a.sw - a.pw;
    return r;
}

// One gathered input value: channel c at tap (q, r) under the pixel, 0 in the padding.
template <bool kUnit, typename TX>
__device__ __forceinline__ TX gather_x(const ConvArgs& a, const TX* __restrict__ x,
                                       const PixelPos& pp, int32_t c, int32_t q, int32_t r) {
    if (kUnit) {   // 1x1 kernel, no padding: always inside
        if (!pp.valid) return TX(0);
        return x[pp.xbase + int64_t(c) * a.x_c + int64_t(pp.ih0) * a.x_row + int64_t(pp.iw0) * a.x_col];
    }
    const int32_t ih = pp.ih0 + q, iw = pp.iw0 + r;
    const bool in = pp.valid && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
    if (!in) return TX(0);
    return x[pp.xbase + int64_t(c) * a.x_c + int64_t(ih) * a.x_row + int64_t(iw) * a.x_col];
}

// ---------------------------------------------------------------------------
// fma_conv: N <= 8.
// ---------------------------------------------------------------------------

template <int N, int PPT, bool kUnit, typename TX, typename TY>
__global__ void __launch_bounds__(kThreads) fma_conv(ConvArgs a) {
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t g = L % a.G;
    const int64_t tile = L / a.G;
    int32_t zb, ze;
    group_range(a, g, zb, ze);

    const TX* __restrict__ x = static_cast<const TX*>(a.x);
    const TX* __restrict__ D = static_cast<const TX*>(a.D);
    PixelPos pp[PPT];
    float acc[PPT][N];
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
        pp[i] = pixel_pos(a, tile * (kThreads * PPT) + i * kThreads + threadIdx.x);
#pragma unroll
        for (int o = 0; o < N; ++o) acc[i][o] = 0.f;
    }

    for (int32_t z = zb; z < ze; ++z) {
        const int32_t c = a.I[z];
        if (c < 0 || c >= a.m) continue;
        const TX* __restrict__ blk = D + int64_t(z) * N * a.KK;
        for (int32_t q = 0; q < a.kh; ++q) {
            for (int32_t r = 0; r < a.kw; ++r) {
                const int32_t tap = q * a.kw + r;
                float wv[N];
#pragma unroll
                for (int o = 0; o < N; ++o) wv[o] = to_f32(blk[o * a.KK + tap]);
#pragma unroll
                for (int i = 0; i < PPT; ++i) {
                    const float xv = to_f32(gather_x<kUnit>(a, x, pp[i], c, q, r));
#pragma unroll
                    for (int o = 0; o < N; ++o) acc[i][o] = fmaf(wv[o], xv, acc[i][o]);
                }
            }
        }
    }

    TY* __restrict__ y = static_cast<TY*>(a.y);
#pragma unroll
    for (int i = 0; i < PPT; ++i) {
        if (!pp[i].valid) continue;
#pragma unroll
        for (int o = 0; o < N; ++o) {
            const int32_t oc = g * N + o;
            if (oc < a.n) y[pp[i].ybase + int64_t(oc) * a.y_c] = from_f32<TY>(acc[i][o]);
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
    const int64_t tile = L / a.G;
    int32_t zb, ze;
    group_range(a, g, zb, ze);
    const int32_t Kg = (ze - zb) * a.KK;
    const int32_t nchunks = (Kg + KC - 1) / KC;

    const TX* __restrict__ x = static_cast<const TX*>(a.x);
    const TX* __restrict__ D = static_cast<const TX*>(a.D);
    const int tid = threadIdx.x;
    const int lane = tid & 63, wave = tid >> 6;

    // Gather role: pixel row `prow` of the tile, kappa sub-range `kofs`.
    const int prow = tid % PT;
    const int kofs = (tid / PT) * KPT;
    const PixelPos pp = pixel_pos(a, tile * PT + prow);

    TX rb[KPT];     // B prefetch registers
    TX ra[AE];      // A prefetch registers

    auto fetch = [&](int32_t chunk) {
        const int32_t k0 = chunk * KC;
        // B: KPT consecutive kappa of this thread's pixel.
        int32_t kap = k0 + kofs;
        int32_t zz = kap / a.KK, tap = kap - zz * a.KK;
#pragma unroll
        for (int i = 0; i < KPT; ++i) {
            TX v = TX(0);
            if (kap < Kg) {
                const int32_t c = a.I[zb + zz];
                const int32_t q = tap / a.kw, r = tap - q * a.kw;
                if (c >= 0 && c < a.m) v = gather_x<kUnit>(a, x, pp, c, q, r);
            }
            rb[i] = v;
            ++kap;
            if (++tap == a.KK) { tap = 0; ++zz; }
        }
        // A: element e -> (o = e % N, kk = e / N) of the N x KC chunk.
#pragma unroll
        for (int j = 0; j < AE; ++j) {
            const int e = tid + j * kThreads;
            const int o = e % N, kk = e / N;
            const int32_t k = k0 + kk;
            TX v = TX(0);
            if (k < Kg) {
                const int32_t z2 = k / a.KK, tp = k - z2 * a.KK;
                v = D[(int64_t(zb + z2) * N + o) * a.KK + tp];
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
            if (oc < a.n) y[op.ybase + int64_t(oc) * a.y_c] = from_f32<TY>(acc[j][r]);
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
    hipError_t err = hipSuccess;
    auto go = [&](auto kernel, int64_t pt) -> onexn_status {
        const int64_t total = grid_for(pt);
        if (total > INT32_MAX / kThreads)
            return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: grid of %lld workgroups is too large",
                        (long long)total);
        a.total = int32_t(total);
        hipLaunchKernelGGL(kernel, dim3(uint32_t(total)), dim3(kThreads), 0, stream, a);
        err = hipGetLastError();
        if (err != hipSuccess)
            return fail(ONEXN_ERR_HIP, "conv2d_fwd: launch failed: %s", hipGetErrorString(err));
        return ONEXN_OK;
    };
    switch (a.N) {
        case 16:
            if (grid_for(256) >= big_grid_min) return go(mfma_conv<16, 64, kUnit, TX, TY>, 256);
            return go(mfma_conv<16, 32, kUnit, TX, TY>, 128);
        case 32:
            if (grid_for(256) >= big_grid_min) return go(mfma_conv<32, 64, kUnit, TX, TY>, 256);
            return go(mfma_conv<32, 32, kUnit, TX, TY>, 128);
        case 1:
            if (grid_for(1024) >= big_grid_min) return go(fma_conv<1, 4, kUnit, TX, TY>, 1024);
            return go(fma_conv<1, 1, kUnit, TX, TY>, 256);
        case 2:
            if (grid_for(1024) >= big_grid_min) return go(fma_conv<2, 4, kUnit, TX, TY>, 1024);
            return go(fma_conv<2, 1, kUnit, TX, TY>, 256);
        case 4:
            if (grid_for(1024) >= big_grid_min) return go(fma_conv<4, 4, kUnit, TX, TY>, 1024);
            return go(fma_conv<4, 1, kUnit, TX, TY>, 256);
        case 8:
            if (grid_for(512) >= big_grid_min) return go(fma_conv<8, 2, kUnit, TX, TY>, 512);
            return go(fma_conv<8, 1, kUnit, TX, TY>, 256);
    }
    return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: N=%d is not supported", a.N);
}

template <typename TX, typename TY>
onexn_status launch_dtype(const ConvArgs& a, hipStream_t s) {
    const bool unit = a.kh == 1 && a.kw == 1 && a.ph == 0 && a.pw == 0;
    return unit ? launch_typed<TX, TY, true>(a, s) : launch_typed<TX, TY, false>(a, s);
}

}  // namespace
}  // namespace onexn

using namespace onexn;

extern "C" onexn_status onexn_conv2d_fwd(const int32_t* P_dev, const int32_t* I_dev,
                                         const void* D_dev, onexn_dtype wdt, int32_t n, int32_t m,
                                         int32_t kh, int32_t kw, int32_t N, int64_t t,
                                         const void* x_dev, onexn_dtype xdt, onexn_layout layout,
                                         int32_t batch, int32_t H, int32_t W, int32_t stride_h,
                                         int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                         void* y_dev, onexn_dtype ydt, void* stream) {
    clear_error();
    if (!P_dev) return fail(ONEXN_ERR_NULL, "conv2d_fwd: NULL P");
    if (batch != 0 && (!x_dev || !y_dev)) return fail(ONEXN_ERR_NULL, "conv2d_fwd: NULL x or y");
    if (t > 0 && (!I_dev || !D_dev)) return fail(ONEXN_ERR_NULL, "conv2d_fwd: NULL I or D with t > 0");
    if ((wdt != ONEXN_F32 && wdt != ONEXN_BF16) || (xdt != ONEXN_F32 && xdt != ONEXN_BF16) ||
        (ydt != ONEXN_F32 && ydt != ONEXN_BF16))
        return fail(ONEXN_ERR_DTYPE, "conv2d_fwd: unknown dtype");
    if (wdt != xdt) return fail(ONEXN_ERR_DTYPE, "conv2d_fwd: weight and input dtypes differ");
    if (ydt != xdt && ydt != ONEXN_F32)
        return fail(ONEXN_ERR_DTYPE, "conv2d_fwd: output dtype must be the input dtype or F32");
    if (layout != ONEXN_NCHW && layout != ONEXN_NHWC)
        return fail(ONEXN_ERR_ARG, "conv2d_fwd: unknown layout %d", int(layout));
    if (n < 1 || m < 1 || kh < 1 || kw < 1 || N < 1 || batch < 0 || H < 1 || W < 1 ||
        stride_h < 1 || stride_w < 1 || pad_h < 0 || pad_w < 0 || t < 0)
        return fail(ONEXN_ERR_ARG, "conv2d_fwd: sizes, strides and t must be positive, pads >= 0");
    if (N != 1 && N != 2 && N != 4 && N != 8 && N != 16 && N != 32)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: N=%d not in {1,2,4,8,16,32}", N);
    if (kh > 16 || kw > 16 || stride_h > 8 || stride_w > 8 || pad_h >= 16 || pad_w >= 16)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: kernel, stride or pad beyond the supported range");
    const int64_t Ho = (int64_t(H) + 2 * pad_h - kh) / stride_h + 1;
    const int64_t Wo = (int64_t(W) + 2 * pad_w - kw) / stride_w + 1;
    if (int64_t(H) + 2 * pad_h < kh || int64_t(W) + 2 * pad_w < kw || Ho < 1 || Wo < 1)
        return fail(ONEXN_ERR_SHAPE, "conv2d_fwd: empty output (kernel larger than padded input)");
    const int64_t G = (int64_t(n) + N - 1) / N;
    if (int64_t(m) * H * W > INT32_MAX || int64_t(n) * Ho * Wo > INT32_MAX || t > INT32_MAX ||
        t > int64_t(m) * G || G * N * int64_t(kh) * kw > INT32_MAX)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: per-image sizes or t exceed int32 indexing");
    if (batch == 0) return ONEXN_OK;

    ConvArgs a{};
    a.P = P_dev;
    a.I = I_dev;
    a.D = D_dev;
    a.x = x_dev;
    a.y = y_dev;
    a.n = n;
    a.m = m;
    a.kh = kh;
    a.kw = kw;
    a.KK = kh * kw;
    a.N = N;
    a.G = int32_t(G);
    a.H = H;
    a.W = W;
    a.Ho = int32_t(Ho);
    a.Wo = int32_t(Wo);
    a.HWo = int32_t(Ho * Wo);
    a.sh = stride_h;
    a.sw = stride_w;
    a.ph = pad_h;
    a.pw = pad_w;
    a.t = int32_t(t);
    a.npix = int64_t(batch) * Ho * Wo;
    a.x_img = int64_t(m) * H * W;
    a.y_img = int64_t(n) * Ho * Wo;
    if (layout == ONEXN_NCHW) {
        a.x_c = H * W;
        a.x_row = W;
        a.x_col = 1;
        a.y_c = int32_t(Ho * Wo);
        a.y_pix = 1;
    } else {
        a.x_c = 1;
        a.x_row = W * m;
        a.x_col = m;
        a.y_c = 1;
        a.y_pix = n;
    }
    hipStream_t s = static_cast<hipStream_t>(stream);
    if (xdt == ONEXN_F32) return launch_dtype<float, float>(a, s);
    if (ydt == ONEXN_BF16) return launch_dtype<uint16_t, uint16_t>(a, s);
    return launch_dtype<uint16_t, float>(a, s);
}
