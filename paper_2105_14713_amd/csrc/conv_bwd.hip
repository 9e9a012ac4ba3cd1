// Backward of the 1xN-pruned convolution for fine-tuning with the pattern
// fixed (Sec. 4.1): the input gradient through Omega-bar and the weight
// gradient of the kept blocks, in the BSR layout of D (Sec. 3.4).
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713).  The forward is Eq. 7 with Omega-bar (Eq. 8 over P, I,
// D); its gradients are
//   dX[b][c][ih][iw] = sum over kept blocks z with I[z] = c, rows i, taps
//                      (q, r) with ih = oh*sh - ph + q, iw = ow*sw - pw + r:
//                      D[z][i][q][r] * dY[b][gN + i][oh][ow]
//   dD[z][i][q][r]   = sum over b, oh, ow: dY[b][gN + i][oh][ow] *
//                      X[b][I[z]][oh*sh - ph + q][ow*sw - pw + r]
// (g the col-group of block z; rows gN + i >= n do not exist and get 0).
//
// bwd_data.  A workgroup is (input channel c, tile of 256 input pixels).  Its
// threads first find c's kept blocks: I is ascending within each col-group,
// so one binary search per col-group; the hits are compacted in col-group
// order (a prefix scan), which fixes the summation order.  Each lane then
// gathers its input pixel's contributions: for each kept block, row and tap,
// the output pixel whose window puts that tap on it (when the stride
// divides), weights being wave-uniform loads.
//
// bwd_data_fewc.  Layers with at most four input channels (a network's first
// convolution), fp32: every input channel of a pixel in one lane.  The
// layer's weights (Omega-bar, dense, [tap][output channel][input channel],
// zero where pruned) are scattered into LDS once per workgroup.  A workgroup
// takes a contiguous range of (row, residue, column chunk) tasks, the ranges
// of one XCD consecutive.  A wave takes 64 input pixels of one row whose
// columns share their residue modulo the stride (iw = cb + sw * (64k + lane)), so the taps whose stride divides are
// the same for the whole wave and the others are skipped; for each such tap
// and output channel a lane loads one dY value (consecutive lanes,
// consecutive output columns; out-of-range positions read zeros) and adds it,
// times the broadcast weights, into its MC channel sums.  Fixed summation
// order (tap, then output channel).
//
// bwd_weight.  A workgroup per (kept block z, tap).  Lanes split the output
// pixels and keep N partial sums (one per block row) over their pixels, then
// an LDS tree adds the 256 lanes' sums in a fixed order.  Both
// kernels accumulate in fp32 and their results do not depend on timing.

#include "lds_copy.h"
#include "onexn_internal.h"

namespace onexn {
namespace {

constexpr int kBwdThreads = 256;
constexpr int kBwdMaxG = 2048;   // col-groups bwd_data lists per channel

template <typename T> __device__ __forceinline__ float ld(const T* p, int64_t i) { return to_f32(p[i]); }

template <typename TD, typename TY>
__global__ void __launch_bounds__(kBwdThreads) bwd_data(ConvArgs a, const TD* __restrict__ dy,
                                                         TY* __restrict__ dx) {
    __shared__ int32_t sZ[kBwdMaxG];
    __shared__ int32_t sG[kBwdMaxG];
    __shared__ int32_t sScan[kBwdThreads];
    __shared__ int32_t sBase;
    const int tid = threadIdx.x;
    const int32_t c = blockIdx.y;
    const TD* __restrict__ D = static_cast<const TD*>(a.D);

    // Kept blocks of input channel c, in col-group order.
    if (tid == 0) sBase = 0;
    __syncthreads();
    for (int32_t g0 = 0; g0 < a.G; g0 += kBwdThreads) {
        const int32_t g = g0 + tid;
        int32_t z = -1;
        if (g < a.G) {
            int32_t lo, hi;
            group_range(a, g, lo, hi);
            while (lo < hi) {          // first entry with I >= c
                const int32_t mid = (lo + hi) >> 1;
                if (a.I[mid] < c) lo = mid + 1;
                else hi = mid;
            }
            int32_t zb, ze;
            group_range(a, g, zb, ze);
            if (lo < ze && a.I[lo] == c) z = lo;
        }
        const int32_t hit = z >= 0;
        sScan[tid] = hit;
        __syncthreads();
        for (int d = 1; d < kBwdThreads; d <<= 1) {
            const int32_t v = tid >= d ? sScan[tid - d] : 0;
            __syncthreads();
            sScan[tid] += v;
            __syncthreads();
        }
        const int32_t base = sBase;
        if (hit) {
            sZ[base + sScan[tid] - 1] = z;
            sG[base + sScan[tid] - 1] = g;
        }
        __syncthreads();
        if (tid == kBwdThreads - 1) sBase = base + sScan[tid];
        __syncthreads();
    }
    const int32_t nz = sBase;

    const int64_t HW = int64_t(a.H) * a.W;
    const int64_t pix = int64_t(blockIdx.x) * kBwdThreads + tid;
    const int32_t batch = a.npix / a.HWo;
    if (pix >= int64_t(batch) * HW) return;
    const int32_t b = int32_t(pix / HW);
    const int32_t hw = int32_t(pix - int64_t(b) * HW);
    const int32_t ih = hw / a.W, iw = hw - ih * a.W;
    const int32_t KK = a.kh * a.kw;
    float acc = 0.f;
    for (int32_t e = 0; e < nz; ++e) {
        const int32_t z = sZ[e], g = sG[e];
        const int32_t rows = min(a.N, a.n - g * a.N);
        for (int32_t i = 0; i < rows; ++i) {
            const TD* dz = D + (int64_t(z) * a.N + i) * KK;
            const TD* yrow = dy + (int64_t(b) * a.n + g * a.N + i) * a.HWo;
            for (int32_t q = 0; q < a.kh; ++q) {
                const int32_t th = ih + a.ph - q;
                if (th < 0 || th % a.sh != 0) continue;
                const int32_t oh = th / a.sh;
                if (oh >= a.Ho) continue;
                for (int32_t r = 0; r < a.kw; ++r) {
                    const int32_t tw = iw + a.pw - r;
                    if (tw < 0 || tw % a.sw != 0) continue;
                    const int32_t ow = tw / a.sw;
                    if (ow >= a.Wo) continue;
                    acc += ld(dz, q * a.kw + r) * ld(yrow, int64_t(oh) * a.Wo + ow);
                }
            }
        }
    }
    dx[(int64_t(b) * a.m + c) * HW + hw] = from_f32<TY>(acc);
}

constexpr int kFcWaves = 4;
constexpr int kFcMaxC = 4;                 // input channels bwd_data_fewc takes
constexpr int kFcMaxLds = 64 * 1024;       // bytes of its weight table

template <int MC>
__global__ void __launch_bounds__(64 * kFcWaves) bwd_data_fewc(ConvArgs a, const float* __restrict__ dy,
                                                               float* __restrict__ dx, int32_t cpr,
                                                               int32_t tasks) {
    extern __shared__ float sW[];   // [KK][n][MC]
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t n = a.n, N = a.N, KK = a.KK;
    for (int32_t e = tid; e < KK * n * MC; e += 64 * kFcWaves) sW[e] = 0.f;
    __syncthreads();
    const float* __restrict__ D = static_cast<const float*>(a.D);
    for (int32_t g = 0; g < a.G; ++g) {
        int32_t zb, ze;
        group_range(a, g, zb, ze);
        const int32_t per = N * KK;          // floats of a D row
        for (int32_t e = tid; e < (ze - zb) * per; e += 64 * kFcWaves) {
            const int32_t zz = e / per, rem = e - zz * per;
            const int32_t i = rem / KK, tap = rem - i * KK;
            const int32_t o = g * N + i, c = a.I[zb + zz];
            if (o < n && c >= 0 && c < MC) sW[(tap * n + o) * MC + c] = D[int64_t(zb + zz) * per + rem];
        }
    }
    __syncthreads();

    const int32_t HWo = a.HWo, HWi = a.H * a.W;
    const int32_t batch = a.npix / HWo;
    const __amdgpu_buffer_rsrc_t rY = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<float*>(dy), 0, __builtin_amdgcn_readfirstlane(batch * n * HWo * 4), kRawBufferFlags);
    const uint32_t chb = uint32_t(HWo) * 4;  // bytes between dY channels
    const int32_t per_row = a.sw * cpr;      // wave tasks per input row
    // A workgroup takes a contiguous range of tasks (consecutive input rows,
    // which read overlapping dY rows: a dY row feeds kh consecutive input
    // rows), and consecutive ranges run on one XCD, so those rows are
    // fetched into that XCD's L2 once (round-robin tasks: 19 % L2 hits).
    const int32_t L = xcd_remap(int32_t(blockIdx.x), int32_t(gridDim.x));
    const int32_t t0 = int32_t(int64_t(tasks) * L / gridDim.x);
    const int32_t t1 = int32_t(int64_t(tasks) * (L + 1) / gridDim.x);
    for (int32_t task = t0 + wave; task < t1; task += kFcWaves) {
        const int32_t row = task / per_row, rem = task - row * per_row;
        const int32_t cb = rem / cpr, k = rem - cb * cpr;
        const int32_t b = row / a.H, ih = row - b * a.H;
        const int32_t iw = cb + a.sw * (64 * k + lane);
        const bool in = iw < a.W;
        const int32_t ybase = b * n * HWo;
        float acc[MC];
#pragma unroll
        for (int c = 0; c < MC; ++c) acc[c] = 0.f;
        for (int32_t q = 0; q < a.kh; ++q) {
            const int32_t th = ih + a.ph - q;
            if (th < 0 || th % a.sh != 0 || th / a.sh >= a.Ho) continue;
            const int32_t yrow = ybase + (th / a.sh) * a.Wo;
            for (int32_t r = 0; r < a.kw; ++r) {
                if (((cb + a.pw - r) % a.sw + a.sw) % a.sw != 0) continue;   // the wave's column residue
                const int32_t tw = iw + a.pw - r;
                const bool ok = in && tw >= 0 && tw / a.sw < a.Wo;
                const int32_t voff = ok ? (yrow + tw / a.sw) * 4 : int32_t(kBufferOutOfRange);
                const float* w = sW + (q * a.kw + r) * n * MC;
                int32_t o = 0;
                for (; o + 8 <= n; o += 8) {
                    float v[8];
#pragma unroll
                    for (int u = 0; u < 8; ++u)
                        v[u] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                            rY, voff, int32_t(uint32_t(o + u) * chb), 0));
#pragma unroll
                    for (int u = 0; u < 8; ++u)
#pragma unroll
                        for (int c = 0; c < MC; ++c) acc[c] += w[(o + u) * MC + c] * v[u];
                }
                for (; o < n; ++o) {
                    const float v = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                        rY, voff, int32_t(uint32_t(o) * chb), 0));
#pragma unroll
                    for (int c = 0; c < MC; ++c) acc[c] += w[o * MC + c] * v;
                }
            }
        }
        if (in) {
#pragma unroll
            for (int c = 0; c < MC; ++c) dx[(int64_t(b) * a.m + c) * HWi + int64_t(ih) * a.W + iw] = acc[c];
        }
    }
}

template <int N, typename TX>
__global__ void __launch_bounds__(kBwdThreads) bwd_weight(ConvArgs a, const TX* __restrict__ x,
                                                           const TX* __restrict__ dy,
                                                           float* __restrict__ dD) {
    __shared__ float sR[kBwdThreads * N];
    const int tid = threadIdx.x;
    const int32_t z = blockIdx.x;
    const int32_t q = blockIdx.y / a.kw, r = blockIdx.y - q * a.kw;
    // Col-group of block z: the last g with P[g] <= z (P clamped to [0, t]).
    int32_t lo = 0, hi = a.G - 1;
    while (lo < hi) {
        const int32_t mid = (lo + hi + 1) >> 1;
        if (min(max(a.P[mid], 0), a.t) <= z) lo = mid;
        else hi = mid - 1;
    }
    const int32_t g = lo;
    const int32_t c = a.I[z];
    const int32_t rows = min(N, a.n - g * N);
    const bool chan_ok = c >= 0 && c < a.m;
    const int64_t HW = int64_t(a.H) * a.W;
    const int32_t KK = a.kh * a.kw;

    {
        {
            float acc[N];
#pragma unroll
            for (int i = 0; i < N; ++i) acc[i] = 0.f;
            if (chan_ok) {
                for (int32_t p = tid; p < a.npix; p += kBwdThreads) {
                    const int32_t b = p / a.HWo, hwo = p - b * a.HWo;
                    const int32_t oh = hwo / a.Wo, ow = hwo - oh * a.Wo;
                    const int32_t ih = oh * a.sh - a.ph + q, iw = ow * a.sw - a.pw + r;
                    if (ih < 0 || ih >= a.H || iw < 0 || iw >= a.W) continue;
                    const float xv = to_f32(x[(int64_t(b) * a.m + c) * HW + int64_t(ih) * a.W + iw]);
                    const TX* yp = dy + (int64_t(b) * a.n + g * N) * a.HWo + hwo;
#pragma unroll
                    for (int i = 0; i < N; ++i)
                        if (i < rows) acc[i] += to_f32(yp[int64_t(i) * a.HWo]) * xv;
                }
            }
#pragma unroll
            for (int i = 0; i < N; ++i) sR[i * kBwdThreads + tid] = acc[i];
            __syncthreads();
            for (int s = kBwdThreads / 2; s > 0; s >>= 1) {
                if (tid < s) {
#pragma unroll
                    for (int i = 0; i < N; ++i) sR[i * kBwdThreads + tid] += sR[i * kBwdThreads + tid + s];
                }
                __syncthreads();
            }
            if (tid < N) dD[(int64_t(z) * N + tid) * KK + q * a.kw + r] = sR[tid * kBwdThreads];
        }
    }
}

onexn_status check_common(const int32_t* P, int32_t n, int32_t m, int32_t kh, int32_t kw, int32_t N,
                          int64_t t, int32_t batch, int32_t H, int32_t W, int32_t sh, int32_t sw,
                          int32_t ph, int32_t pw, const char* who, ConvArgs& a) {
    if (!P) return fail(ONEXN_ERR_NULL, "%s: NULL P", who);
    if (n < 1 || m < 1 || kh < 1 || kw < 1 || N < 1 || batch < 0 || H < 1 || W < 1 || sh < 1 ||
        sw < 1 || ph < 0 || pw < 0 || t < 0)
        return fail(ONEXN_ERR_ARG, "%s: sizes, strides and t must be positive, pads >= 0", who);
    if (N != 1 && N != 2 && N != 4 && N != 8 && N != 16 && N != 32)
        return fail(ONEXN_ERR_UNSUPPORTED, "%s: N=%d not in {1,2,4,8,16,32}", who, N);
    if (kh > 16 || kw > 16 || sh > 8 || sw > 8 || ph >= 16 || pw >= 16)
        return fail(ONEXN_ERR_UNSUPPORTED, "%s: kernel, stride or pad beyond the supported range", who);
    const int64_t Ho = (int64_t(H) + 2 * ph - kh) / sh + 1;
    const int64_t Wo = (int64_t(W) + 2 * pw - kw) / sw + 1;
    if (int64_t(H) + 2 * ph < kh || int64_t(W) + 2 * pw < kw || Ho < 1 || Wo < 1)
        return fail(ONEXN_ERR_SHAPE, "%s: empty output (kernel larger than padded input)", who);
    const int64_t G = (int64_t(n) + N - 1) / N;
    if (G > kBwdMaxG) return fail(ONEXN_ERR_UNSUPPORTED, "%s: more than %d col-groups", who, kBwdMaxG);
    if (int64_t(batch) * m * H * W > INT32_MAX || int64_t(batch) * n * Ho * Wo > INT32_MAX ||
        t > int64_t(m) * G || G * N * int64_t(kh) * kw > INT32_MAX)
        return fail(ONEXN_ERR_UNSUPPORTED, "%s: sizes exceed int32 indexing", who);
    a = ConvArgs{};
    a.P = P;
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
    a.sh = sh;
    a.sw = sw;
    a.ph = ph;
    a.pw = pw;
    a.t = int32_t(t);
    a.npix = int32_t(int64_t(batch) * Ho * Wo);
    return ONEXN_OK;
}

onexn_status launched(const char* who) {
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(ONEXN_ERR_HIP, "%s: launch failed: %s", who, hipGetErrorString(err));
    return ONEXN_OK;
}

template <typename TD, typename TY>
onexn_status launch_bwd_data(const ConvArgs& a, int32_t batch, const void* dy, void* dx, hipStream_t s) {
    const int64_t tiles = (int64_t(batch) * a.H * a.W + kBwdThreads - 1) / kBwdThreads;
    if (tiles > INT32_MAX || a.m > 65535)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_bwd_data: grid out of range");
    hipLaunchKernelGGL((bwd_data<TD, TY>), dim3(uint32_t(tiles), uint32_t(a.m)), dim3(kBwdThreads), 0, s, a,
                       static_cast<const TD*>(dy), static_cast<TY*>(dx));
    return launched("conv2d_bwd_data");
}

bool bwd_data_fewc_applies(const ConvArgs& a, onexn_dtype wdt, onexn_dtype dxdt, int32_t batch) {
    return wdt == ONEXN_F32 && dxdt == ONEXN_F32 && a.m <= kFcMaxC &&
           int64_t(a.KK) * a.n * a.m * 4 <= kFcMaxLds &&
           int64_t(batch) * a.n * a.HWo * 4 < (int64_t(1) << 31);   // 32-bit buffer offsets
}

onexn_status launch_bwd_data_fewc(const ConvArgs& a, int32_t batch, const void* dy, void* dx, hipStream_t s) {
    const int32_t cpr = ((a.W + a.sw - 1) / a.sw + 63) / 64;   // 64-column chunks of a residue class
    const int64_t tasks = int64_t(batch) * a.H * a.sw * cpr;
    if (tasks > INT32_MAX) return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_bwd_data: grid out of range");
    const int64_t grid = std::min<int64_t>((tasks + kFcWaves - 1) / kFcWaves, 8 * int64_t(device_cu_count()));
    const size_t lds = size_t(a.KK) * a.n * a.m * 4;
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(uint32_t(grid)), dim3(64 * kFcWaves), lds, s, a,
                           static_cast<const float*>(dy), static_cast<float*>(dx), cpr, int32_t(tasks));
        return launched("conv2d_bwd_data");
    };
    switch (a.m) {
        case 1: return go(bwd_data_fewc<1>);
        case 2: return go(bwd_data_fewc<2>);
        case 3: return go(bwd_data_fewc<3>);
        default: return go(bwd_data_fewc<4>);
    }
}

template <typename TX>
onexn_status launch_bwd_weight(const ConvArgs& a, const void* x, const void* dy, float* dD, hipStream_t s) {
    auto go = [&](auto kern) {
        hipLaunchKernelGGL(kern, dim3(uint32_t(a.t), uint32_t(a.KK)), dim3(kBwdThreads), 0, s, a, static_cast<const TX*>(x),
                           static_cast<const TX*>(dy), dD);
        return launched("conv2d_bwd_weight");
    };
    switch (a.N) {
        case 1: return go(bwd_weight<1, TX>);
        case 2: return go(bwd_weight<2, TX>);
        case 4: return go(bwd_weight<4, TX>);
        case 8: return go(bwd_weight<8, TX>);
        case 16: return go(bwd_weight<16, TX>);
        default: return go(bwd_weight<32, TX>);
    }
}

}  // namespace
}  // namespace onexn

using namespace onexn;

extern "C" onexn_status onexn_conv2d_bwd_data(const int32_t* P_dev, const int32_t* I_dev,
                                              const void* D_dev, onexn_dtype wdt, int32_t n, int32_t m,
                                              int32_t kh, int32_t kw, int32_t N, int64_t t,
                                              const void* dy_dev, onexn_dtype dydt, int32_t batch,
                                              int32_t H, int32_t W, int32_t stride_h, int32_t stride_w,
                                              int32_t pad_h, int32_t pad_w, void* dx_dev,
                                              onexn_dtype dxdt, void* stream) {
    clear_error();
    ConvArgs a;
    if (onexn_status st = check_common(P_dev, n, m, kh, kw, N, t, batch, H, W, stride_h, stride_w, pad_h,
                                       pad_w, "conv2d_bwd_data", a))
        return st;
    if (batch != 0 && (!dy_dev || !dx_dev)) return fail(ONEXN_ERR_NULL, "conv2d_bwd_data: NULL dy or dx");
    if (t > 0 && (!I_dev || !D_dev)) return fail(ONEXN_ERR_NULL, "conv2d_bwd_data: NULL I or D with t > 0");
    if ((wdt != ONEXN_F32 && wdt != ONEXN_BF16) || dydt != wdt || (dxdt != dydt && dxdt != ONEXN_F32))
        return fail(ONEXN_ERR_DTYPE, "conv2d_bwd_data: dy and D share a dtype; dx takes it or F32");
    if (batch == 0) return ONEXN_OK;
    a.I = I_dev;
    a.D = D_dev;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // fp32 layers with at most four input channels: one lane per input pixel
    // and all its channels.  fp32 1x1 and 3x3 layers at N = 16 / 32: the
    // matrix-core kernels.
    if (tuning(kTuneBwdKernel) != 1) {
        if (bwd_data_fewc_applies(a, wdt, dxdt, batch)) return launch_bwd_data_fewc(a, batch, dy_dev, dx_dev, s);
        if (bwd_data_pw_applies(a, wdt, dxdt, batch)) return launch_bwd_data_pw(a, dy_dev, dx_dev, s);
    }
    if (wdt == ONEXN_F32) return launch_bwd_data<float, float>(a, batch, dy_dev, dx_dev, s);
    if (dxdt == ONEXN_BF16) return launch_bwd_data<uint16_t, uint16_t>(a, batch, dy_dev, dx_dev, s);
    return launch_bwd_data<uint16_t, float>(a, batch, dy_dev, dx_dev, s);
}

extern "C" onexn_status onexn_conv2d_bwd_weight(const int32_t* P_dev, const int32_t* I_dev, int32_t n,
                                                int32_t m, int32_t kh, int32_t kw, int32_t N, int64_t t,
                                                const void* x_dev, onexn_dtype xdt, const void* dy_dev,
                                                int32_t batch, int32_t H, int32_t W, int32_t stride_h,
                                                int32_t stride_w, int32_t pad_h, int32_t pad_w,
                                                float* dD_dev, void* stream) {
    clear_error();
    ConvArgs a;
    if (onexn_status st = check_common(P_dev, n, m, kh, kw, N, t, batch, H, W, stride_h, stride_w, pad_h,
                                       pad_w, "conv2d_bwd_weight", a))
        return st;
    if (t > 0 && (!I_dev || !dD_dev || (batch > 0 && (!x_dev || !dy_dev))))
        return fail(ONEXN_ERR_NULL, "conv2d_bwd_weight: NULL I, x, dy or dD with t > 0");
    if (xdt != ONEXN_F32 && xdt != ONEXN_BF16) return fail(ONEXN_ERR_DTYPE, "conv2d_bwd_weight: unknown dtype");
    if (t == 0) return ONEXN_OK;
    a.I = I_dev;
    hipStream_t s = static_cast<hipStream_t>(stream);
    // 1x1 stride-1 fp32 layers at N = 16 / 32: the matrix-core kernel.
    if (bwd_weight_pw_applies(a, xdt, batch) && tuning(kTuneBwdKernel) != 1)
        return launch_bwd_weight_pw(a, x_dev, dy_dev, dD_dev, s);
    if (xdt == ONEXN_F32) return launch_bwd_weight<float>(a, x_dev, dy_dev, dD_dev, s);
    return launch_bwd_weight<uint16_t>(a, x_dev, dy_dev, dD_dev, s);
}
