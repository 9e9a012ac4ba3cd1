// Entry point of the 1xN-pruned convolution: argument checks and the choice of
// kernel family (pointwise LDS-shared kernels for 1x1 stride-1 NCHW layers
// where they apply, the generic gather kernels otherwise).
#include <atomic>
#include <cstring>

#include "conv_common.h"

namespace onexn {

int device_cu_count() {
    constexpr int kMaxDevices = 64;
    static std::atomic<int> cache[kMaxDevices];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= kMaxDevices) return 256;
    int v = cache[dev].load(std::memory_order_relaxed);
    if (v > 0) return v;
    if (hipDeviceGetAttribute(&v, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess || v <= 0)
        v = 256;
    cache[dev].store(v, std::memory_order_relaxed);
    return v;
}

namespace {

// Stored as value + 1, so that the zero-initialised array reads kTuneAuto.
std::atomic<int32_t> g_tuning[kTuneCount];
const char* const kTuneNames[kTuneCount] = {
    "kernel", "pw_kernel", "pw_wgs", "pwb_gp", "pwb_rp", "direct_kdb", "direct_tile", "fma_tpw",
    "fma_no_v4", "fma_tile", "kxk_split", "kxk_tp", "pwb_kernel", "pwb_wgs", "kxkf_split",
    "nhwc_tile", "bwd_kernel", "bwd_split"};

}  // namespace

int32_t tuning(Tune k) { return g_tuning[k].load(std::memory_order_relaxed) - 1; }

// The generic gather kernels for every layer the specialised ones would take.
bool generic_forced() { return tuning(kTuneKernel) == 1; }

}  // namespace onexn

using namespace onexn;

namespace {

onexn_status conv2d_fwd(const int32_t* P_dev, const int32_t* I_dev, const void* D_dev,
                        onexn_dtype wdt, int32_t n, int32_t m, int32_t kh, int32_t kw, int32_t N,
                        int64_t t, const void* x_dev, onexn_dtype xdt, onexn_layout layout,
                        int32_t batch, int32_t H, int32_t W, int32_t stride_h, int32_t stride_w,
                        int32_t pad_h, int32_t pad_w, void* y_dev, onexn_dtype ydt,
                        const float* scale_dev, const float* bias_dev, onexn_act act,
                        void* stream) {
    clear_error();
    if (!P_dev) return fail(ONEXN_ERR_NULL, "conv2d_fwd: NULL P");
    if (act != ONEXN_ACT_NONE && act != ONEXN_ACT_RELU && act != ONEXN_ACT_RELU6)
        return fail(ONEXN_ERR_ARG, "conv2d_fwd: unknown activation %d", int(act));
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
        int64_t(batch) * Ho * Wo > INT32_MAX - 4096 ||
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
    a.ep_scale = scale_dev;
    a.ep_bias = bias_dev;
    a.ep_act = act;
    a.npix = int32_t(int64_t(batch) * Ho * Wo);
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
    // bf16 1x1 N = 32 layers: the LDS-staged kernel for long contractions
    // (2048 -> 2048 at 14x14, batch 256: 313 us against 360 us register-
    // gathered), the register-gathered one otherwise.  The pwb_kernel tuning
    // forces 1: register-gathered, 2: staged (an error where it does not fit).
    if (!generic_forced()) {
        const int32_t pbk = tuning(kTunePwbKernel);
        const bool staged = pw_bf16s_applies(a, xdt, ydt, layout);
        if (pbk == 2 && !staged)
            return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: the LDS-staged bf16 kernel does not fit this layer");
        if (staged && (pbk == 2 || (pbk != 1 && a.m >= 512))) return launch_pw_bf16s(a, ydt, s);
        if (pw_bf16r_applies(a, xdt, ydt, layout)) return launch_pw_bf16r(a, ydt, s);
    }
    // fp32 1x1 layers: the resident-tile kernel for stride-1 layers that
    // widen the channels over many pixels, the register-operand kernel for
    // the rest (contractions at least as long as the output is wide, few
    // pixels, any stride or padding).  The pw_kernel tuning overrides the
    // choice (1: resident tile, an error where it does not fit; 3: register
    // operands).
    const bool direct = pw_direct_applies(a, xdt, ydt, layout) && !generic_forced();
    if (direct) {
        const int32_t pwk = tuning(kTunePwKernel);
        const bool prefer_direct = pwk == 3 || a.m >= a.n || a.npix <= 8192 ||
                                   (a.N == 32 && a.npix <= 32768 && a.m <= 128);
        const bool tile = pw_tile_applies(a);
        if (pwk == 1 && !tile && a.kh == 1 && a.kw == 1 && a.sh == 1 && a.sw == 1 && a.ph == 0 && a.pw == 0)
            return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: the resident-tile kernel does not fit this layer");
        if (tile && (pwk == 1 || !prefer_direct)) return launch_pw_tile(a, s);
        return launch_pw_direct(a, s);
    }
    if (kxk_applies(a, xdt, ydt, layout) && !generic_forced()) return launch_kxk(a, s);
    if (pw_fma_applies(a, xdt, ydt, layout) && !generic_forced()) return launch_pw_fma(a, s);
    if (kxk_fma_applies(a, xdt, ydt, layout) && !generic_forced()) return launch_kxk_fma(a, s);
    if (pw_nhwc_applies(a, xdt, ydt, layout) && !generic_forced()) return launch_pw_nhwc(a, s);
    return launch_generic(a, xdt, ydt, s);
}

}  // namespace

extern "C" onexn_status onexn_conv2d_fwd(const int32_t* P_dev, const int32_t* I_dev,
                                         const void* D_dev, onexn_dtype wdt, int32_t n, int32_t m,
                                         int32_t kh, int32_t kw, int32_t N, int64_t t,
                                         const void* x_dev, onexn_dtype xdt, onexn_layout layout,
                                         int32_t batch, int32_t H, int32_t W, int32_t stride_h,
                                         int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                         void* y_dev, onexn_dtype ydt, void* stream) {
    return conv2d_fwd(P_dev, I_dev, D_dev, wdt, n, m, kh, kw, N, t, x_dev, xdt, layout, batch, H,
                      W, stride_h, stride_w, pad_h, pad_w, y_dev, ydt, nullptr, nullptr,
                      ONEXN_ACT_NONE, stream);
}

extern "C" onexn_status onexn_conv2d_fwd_fused(
    const int32_t* P_dev, const int32_t* I_dev, const void* D_dev, onexn_dtype wdt, int32_t n,
    int32_t m, int32_t kh, int32_t kw, int32_t N, int64_t t, const void* x_dev, onexn_dtype xdt,
    onexn_layout layout, int32_t batch, int32_t H, int32_t W, int32_t stride_h, int32_t stride_w,
    int32_t pad_h, int32_t pad_w, void* y_dev, onexn_dtype ydt, const float* scale_dev,
    const float* bias_dev, onexn_act act, void* stream) {
    return conv2d_fwd(P_dev, I_dev, D_dev, wdt, n, m, kh, kw, N, t, x_dev, xdt, layout, batch, H,
                      W, stride_h, stride_w, pad_h, pad_w, y_dev, ydt, scale_dev, bias_dev, act,
                      stream);
}

extern "C" onexn_status onexn_set_tuning(const char* name, int32_t value) {
    clear_error();
    if (!name) return fail(ONEXN_ERR_NULL, "set_tuning: NULL name");
    if (value < kTuneAuto || value == INT32_MAX)
        return fail(ONEXN_ERR_ARG, "set_tuning: value %d out of range", value);
    for (int k = 0; k < kTuneCount; ++k)
        if (std::strcmp(name, kTuneNames[k]) == 0) {
            g_tuning[k].store(value + 1, std::memory_order_relaxed);
            return ONEXN_OK;
        }
    return fail(ONEXN_ERR_ARG, "set_tuning: unknown name \"%s\"", name);
}

extern "C" onexn_status onexn_fc_fwd(const int32_t* P_dev, const int32_t* I_dev, const void* D_dev,
                                     onexn_dtype wdt, int32_t n, int32_t m, int32_t N, int64_t t,
                                     const void* x_dev, onexn_dtype xdt, onexn_layout layout,
                                     int32_t batch, void* y_dev, onexn_dtype ydt,
                                     const float* scale_dev, const float* bias_dev, onexn_act act,
                                     void* stream) {
    clear_error();
    if (layout != ONEXN_NCHW && layout != ONEXN_NHWC)
        return fail(ONEXN_ERR_ARG, "fc_fwd: unknown layout %d", int(layout));
    if (batch < 0) return fail(ONEXN_ERR_ARG, "fc_fwd: batch must be >= 0");
    // [batch][m] rows: batch one-pixel images.  [m][batch] columns: one image
    // of batch pixels, so the 1x1 kernels read each feature's row coalesced.
    if (layout == ONEXN_NHWC)
        return conv2d_fwd(P_dev, I_dev, D_dev, wdt, n, m, 1, 1, N, t, x_dev, xdt, ONEXN_NCHW, batch,
                          1, 1, 1, 1, 0, 0, y_dev, ydt, scale_dev, bias_dev, act, stream);
    if (batch == 0) return conv2d_fwd(P_dev, I_dev, D_dev, wdt, n, m, 1, 1, N, t, x_dev, xdt,
                                      ONEXN_NCHW, 0, 1, 1, 1, 1, 0, 0, y_dev, ydt, scale_dev,
                                      bias_dev, act, stream);
    return conv2d_fwd(P_dev, I_dev, D_dev, wdt, n, m, 1, 1, N, t, x_dev, xdt, ONEXN_NCHW, 1, 1,
                      batch, 1, 1, 0, 0, y_dev, ydt, scale_dev, bias_dev, act, stream);
}
