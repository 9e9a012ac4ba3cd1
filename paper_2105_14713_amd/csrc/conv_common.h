// Device-side definitions shared by the convolution kernels of libonexn.so.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>
#include <type_traits>

#include "onexn_internal.h"

namespace onexn {

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
    int32_t npix;       // batch * Ho * Wo
    int64_t x_img;      // elements per input image
    int32_t x_c, x_row, x_col;
    int64_t y_img;      // elements per output image
    int32_t y_c, y_pix;
    int32_t total;      // workgroups in the grid
    int32_t slices;        // resident-tile pointwise kernel: slices per pixel tile,
    int32_t cost_q, cost_r;   // and its total work cost divided by the grid (quotient, remainder)
    int32_t kx_rows;       // k x k staged kernel: output rows per tile,
    int32_t kx_wp, kx_vrwp, kx_cp;   // staged row width, input rows x row width, channel pitch (floats)
    int32_t kx_tiles;      // and its tile count (balanced split)
    // Fused epilogue of the store stage: y = act(scale[o] * acc + bias[o]) for
    // output channel o (rearranged order); either array may be absent.
    const float* ep_scale;
    const float* ep_bias;
    int32_t ep_act;        // onexn_act
};

// ---------------------------------------------------------------------------
// Element helpers.  bf16 is carried as raw uint16_t bits.
// ---------------------------------------------------------------------------

__device__ __forceinline__ float to_f32(float v) { return v; }
__device__ __forceinline__ float to_f32(uint16_t v) { return __uint_as_float(uint32_t(v) << 16); }

// Output writes.  A kernel writes each output element once and never reads
// it back, so the stores are non-temporal: the lines do not linger dirty in
// L2, which a launch otherwise writes back before it ends (measured on the
// 1x1 256->512 28x28 layer at batch 32: 54.4 -> 49.9 us).
template <typename T>
__device__ __forceinline__ void store_out(T* p, T v) {
    __builtin_nontemporal_store(v, p);
}

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

// The fused epilogue on one accumulated value of output channel o.  Kernels
// whose stores sit inside their main loop take it as a template flag (kEp):
// the instantiation without it has no epilogue code at all (its parameter
// loads would otherwise make the stores wait for every load in flight).  The
// branches are uniform (kernel arguments).
// The activation of the fused epilogue (after scale and bias).
__device__ __forceinline__ float epilogue_act(const ConvArgs& a, float v) {
    if (a.ep_act == ONEXN_ACT_RELU) v = fmaxf(v, 0.f);
    else if (a.ep_act == ONEXN_ACT_RELU6) v = fminf(fmaxf(v, 0.f), 6.f);
    return v;
}

template <bool kEp = true>
__device__ __forceinline__ float epilogue(const ConvArgs& a, int32_t o, float v) {
    if constexpr (!kEp) return v;
    if (a.ep_scale && a.ep_bias) v = fmaf(v, a.ep_scale[o], a.ep_bias[o]);
    else if (a.ep_scale) v *= a.ep_scale[o];
    else if (a.ep_bias) v += a.ep_bias[o];
    return epilogue_act(a, v);
}

inline bool has_epilogue(const ConvArgs& a) {
    return a.ep_scale || a.ep_bias || a.ep_act != ONEXN_ACT_NONE;
}

// Calls f(std::true_type) when the launch has an epilogue, else
// f(std::false_type): f instantiates the kernel with kEp accordingly.
template <typename F>
onexn_status with_epilogue(const ConvArgs& a, F f) {
    if (has_epilogue(a)) return f(std::true_type{});
    return f(std::false_type{});
}

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

// Per-lane view of one output pixel.  All offsets are element offsets.
struct PixelPos {
    int64_t xoff;    // x offset of (image, ih0, iw0); only dereferenced at in-bounds taps
    int64_t ybase;   // y offset of the pixel at output channel 0
    int32_t ih0, iw0;
    bool valid;
};

__device__ __forceinline__ PixelPos pixel_pos(const ConvArgs& a, int32_t p) {
    PixelPos r;
    r.valid = p < a.npix;
    if (!r.valid) p = 0;
    const int32_t b = p / a.HWo;
    const int32_t hw = p - b * a.HWo;
    const int32_t oh = hw / a.Wo, ow = hw - oh * a.Wo;
    r.ih0 = oh * a.sh - a.ph;
    r.iw0 = ow * a.sw - a.pw;
    r.xoff = int64_t(b) * a.x_img + int64_t(r.ih0) * a.x_row + int64_t(r.iw0) * a.x_col;
    r.ybase = int64_t(b) * a.y_img + int64_t(hw) * a.y_pix;
    return r;
}

// Position along a col-group's contraction: kappa = zz*kh*kw + q*kw + r, i.e.
// block zz (input channel I[zb + zz]) at kernel tap (q, r).  Every field is
// wave-uniform, so the walk, the I[] lookups and the weight lookups stay on the
// scalar unit and the gathered loads of a batch can all be in flight at once.
struct KapWalk {
    int32_t zz, q, r;
};

template <bool kUnit>
__device__ __forceinline__ KapWalk walk_at(const ConvArgs& a, int32_t kap) {
    if (kUnit) return {kap, 0, 0};
    const int32_t zz = kap / a.KK, tap = kap - zz * a.KK;
    const int32_t q = tap / a.kw, r = tap - q * a.kw;
    return {__builtin_amdgcn_readfirstlane(zz), __builtin_amdgcn_readfirstlane(q),
            __builtin_amdgcn_readfirstlane(r)};
}

template <bool kUnit>
__device__ __forceinline__ void walk_step(const ConvArgs& a, KapWalk& w) {
    if (kUnit) {
        ++w.zz;
        return;
    }
    if (++w.r == a.kw) {
        w.r = 0;
        if (++w.q == a.kh) {
            w.q = 0;
            ++w.zz;
        }
    }
}

// Input channel at walk position w, or -1 when kappa is past the end (ok ==
// false) or I holds an out-of-range channel.  The I read is clamped to the
// col-group's last entry, so it never leaves the array.
__device__ __forceinline__ int32_t walk_channel(const ConvArgs& a, const KapWalk& w, int32_t zb,
                                                int32_t ze, bool ok) {
    const int32_t c = a.I[min(zb + w.zz, ze - 1)];
    return (ok && c >= 0 && c < a.m) ? c : -1;
}

// One gathered input value: channel c (>= 0) at tap (w.q, w.r) under the pixel,
// 0 in the zero padding and for invalid pixels.
template <bool kUnit, typename TX>
__device__ __forceinline__ TX gather_x(const ConvArgs& a, const TX* __restrict__ x,
                                       const PixelPos& pp, int32_t c, const KapWalk& w) {
    const int64_t uoff = int64_t(c) * a.x_c + int64_t(w.q) * a.x_row + int64_t(w.r) * a.x_col;
    bool in = pp.valid;
    if (!kUnit) {
        const int32_t ih = pp.ih0 + w.q, iw = pp.iw0 + w.r;
        in = in && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W;
    }
    return in ? x[pp.xoff + uoff] : TX(0);
}


// Compute units of the current device (queried once per device).
int device_cu_count();

// Kernel families (each defined in its own translation unit).
onexn_status launch_generic(ConvArgs a, onexn_dtype xdt, onexn_dtype ydt, hipStream_t stream);
bool pw_tile_applies(const ConvArgs& a);
onexn_status launch_pw_tile(ConvArgs a, hipStream_t stream);
bool pw_bf16r_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout);
onexn_status launch_pw_bf16r(ConvArgs a, onexn_dtype ydt, hipStream_t stream);
bool pw_bf16s_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout);
onexn_status launch_pw_bf16s(ConvArgs a, onexn_dtype ydt, hipStream_t stream);
bool kxk_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout);
bool pw_fma_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout);
bool pw_direct_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout);
onexn_status launch_pw_direct(ConvArgs a, hipStream_t stream);
onexn_status launch_pw_fma(ConvArgs a, hipStream_t stream);
bool kxk_fma_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout);
bool pw_nhwc_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout);
bool bwd_data_pw_applies(const ConvArgs& a, onexn_dtype wdt, onexn_dtype dxdt, int32_t batch);
onexn_status launch_bwd_data_pw(const ConvArgs& a, const void* dy, void* dx, hipStream_t stream);
bool bwd_weight_pw_applies(const ConvArgs& a, onexn_dtype xdt, int32_t batch);
onexn_status launch_bwd_weight_pw(const ConvArgs& a, const void* x, const void* dy, float* dD, hipStream_t stream);
onexn_status launch_pw_nhwc(ConvArgs a, hipStream_t stream);
onexn_status launch_kxk_fma(ConvArgs a, hipStream_t stream);
onexn_status launch_kxk(ConvArgs a, hipStream_t stream);

// Launches `kernel` on a 1-D grid of `total` workgroups.
template <typename K>
onexn_status launch_grid(K kernel, ConvArgs& a, int64_t total, hipStream_t stream,
                         int threads = kThreads) {
    if (total < 1 || total > INT32_MAX / threads)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: grid of %lld workgroups is out of range",
                    (long long)total);
    a.total = int32_t(total);
    hipLaunchKernelGGL(kernel, dim3(uint32_t(total)), dim3(threads), 0, stream, a);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess)
        return fail(ONEXN_ERR_HIP, "conv2d_fwd: launch failed: %s", hipGetErrorString(err));
    return ONEXN_OK;
}

}  // namespace onexn
