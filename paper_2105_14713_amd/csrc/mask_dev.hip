// Mask building on the GPU: filter rearrangement, block scoring and the
// per-layer top-(1-p) selection of 1xN pruning, bit-exact with the host's
// onexn_build_mask.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713): Sec. 3.3 (filters in decreasing l1 norm), Sec. 3.2 and
// Eq. 4-5 (the l1 norm of each 1xN block), Eq. 1 and Sec. 4.1 (keep the
// 1 - p fraction of blocks with the largest norms, per layer).
//
// Bit-exactness.  The host sums every l1 norm in fp64 in memory order and
// ranks with a strict total order (filters: norm descending, then index
// ascending; blocks: score descending, then row-major index k*G + g
// ascending).  The kernels here add the same fp64 values in the same order
// (no reassociation, no fused multiply-add: the sums are additions of
// |w| only), and select with the same order, so their perm and mask equal
// the host's bit for bit.
//
//   mask_filter_norms  one wave per filter: lanes load 64 consecutive
//                      elements, and the wave adds them in order through
//                      readlane, so the sum is the sequential one.
//   mask_filter_perm   rank of filter j = filters before it in the order;
//                      perm[rank] = j (the identity without rearrangement).
//   mask_block_scores  one thread per block (k, g), input channel fastest
//                      for coalesced reads; rows of the rearranged layer are
//                      read through perm.
//   mask_select        one workgroup: radix selection over the 64-bit score
//                      bits (non-negative doubles order like their bit
//                      patterns) finds the t-th largest score s*; the blocks
//                      above s* are kept, and of the blocks equal to s* the
//                      ones with the lowest indices, found by a scan in
//                      index order.  Every mask byte is written.
//
// NaN weights, which the host function rejects, give NaN norms and scores;
// here they order above every number, so perm is still a permutation and the
// mask still keeps exactly t blocks.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <cmath>
#include <cstdint>
#include <mutex>

#include "onexn_internal.h"

// Scratch of the no-allocation entry point (onexn_build_mask_dev_noalloc):
// the workspace of one mask build, 8 MiB, so layers with n + m * G up to about
// a million fit (the 2048 -> 2048 layer at N = 32 needs 1.1 MB).  Every GPU the
// library runs on holds its own copy from the program's load until the
// process ends.  In host code this name stands for the array but is not a
// device address: host code uses the address hipGetSymbolAddress returns.
static __device__ __align__(256) unsigned char scratch[size_t(8) << 20];

namespace onexn {
namespace {

constexpr size_t kScratchBytes = size_t(8) << 20;
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mu;
void* g_scratch_addr[kMaxDevices] = {};

// Device address of the current device's scratch array, looked up once per
// device (with that device current) and kept.
onexn_status scratch_address(void** out) {
    int dev = 0;
    const hipError_t e = hipGetDevice(&dev);
    if (e != hipSuccess) return fail(ONEXN_ERR_HIP, "build_mask_dev_noalloc: hipGetDevice: %s", hipGetErrorString(e));
    if (dev < 0 || dev >= kMaxDevices)
        return fail(ONEXN_ERR_UNSUPPORTED, "build_mask_dev_noalloc: device %d beyond %d devices", dev, kMaxDevices);
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    if (!g_scratch_addr[dev]) {
        void* p = nullptr;
        const hipError_t se = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (se != hipSuccess || !p)
            return fail(ONEXN_ERR_HIP, "build_mask_dev_noalloc: hipGetSymbolAddress(scratch): %s",
                        hipGetErrorString(se));
        g_scratch_addr[dev] = p;
    }
    *out = g_scratch_addr[dev];
    return ONEXN_OK;
}

constexpr int kSelThreads = 1024;
constexpr int kSelBins = 256;
constexpr size_t kWsAlign = 256;

__device__ __forceinline__ double abs_elem(const float* w, int64_t e) {
    return fabs(static_cast<double>(w[e]));
}
__device__ __forceinline__ double abs_elem(const uint16_t* w, int64_t e) {
    return fabs(static_cast<double>(__uint_as_float(uint32_t(w[e]) << 16)));
}

// Order key of a non-negative sum: its bit pattern, NaN above +inf.
__device__ __forceinline__ uint64_t order_key(double d) {
    return d != d ? 0x7ff8000000000000ull : static_cast<uint64_t>(__double_as_longlong(d));
}

__device__ __forceinline__ double readlane_f64(double v, int l) {
    const uint64_t u = static_cast<uint64_t>(__double_as_longlong(v));
    const uint32_t lo = __builtin_amdgcn_readlane(uint32_t(u), l);
    const uint32_t hi = __builtin_amdgcn_readlane(uint32_t(u >> 32), l);
    return __longlong_as_double(static_cast<long long>((uint64_t(hi) << 32) | lo));
}

template <typename TW>
__global__ void __launch_bounds__(256) mask_filter_norms(const TW* __restrict__ w, int32_t n,
                                                          int64_t filt, double* __restrict__ norm) {
    const int lane = threadIdx.x & 63;
    const int32_t j = blockIdx.x * 4 + (threadIdx.x >> 6);
    if (j >= n) return;
    const TW* wj = w + int64_t(j) * filt;
    double acc = 0.0;
    for (int64_t e0 = 0; e0 < filt; e0 += 64) {
        const double v = e0 + lane < filt ? abs_elem(wj, e0 + lane) : 0.0;
        if (filt - e0 >= 64) {
#pragma unroll 16
            for (int i = 0; i < 64; ++i) acc += readlane_f64(v, i);
        } else {
            const int cnt = int(filt - e0);
            for (int i = 0; i < cnt; ++i) acc += readlane_f64(v, i);
        }
    }
    if (lane == 0) norm[j] = acc;
}

__global__ void __launch_bounds__(256) mask_filter_perm(const double* __restrict__ norm, int32_t n,
                                                         int32_t rearrange, int32_t* __restrict__ perm) {
    __shared__ uint64_t sk[256];
    const int32_t j = blockIdx.x * 256 + threadIdx.x;
    if (!rearrange) {
        if (j < n) perm[j] = j;
        return;
    }
    const uint64_t kj = j < n ? order_key(norm[j]) : 0;
    int32_t rank = 0;
    for (int32_t i0 = 0; i0 < n; i0 += 256) {
        __syncthreads();
        if (i0 + int32_t(threadIdx.x) < n) sk[threadIdx.x] = order_key(norm[i0 + threadIdx.x]);
        __syncthreads();
        const int32_t cnt = min(256, n - i0);
        for (int32_t i = 0; i < cnt; ++i) {
            const uint64_t ki = sk[i];
            rank += (ki > kj) || (ki == kj && i0 + i < j);
        }
    }
    if (j < n) perm[rank] = j;
}

template <typename TW>
__global__ void __launch_bounds__(256) mask_block_scores(const TW* __restrict__ w, const int32_t* __restrict__ perm,
                                                          int32_t n, int32_t m, int32_t KK, int32_t N,
                                                          int32_t G, double* __restrict__ score) {
    const int64_t id = int64_t(blockIdx.x) * 256 + threadIdx.x;
    if (id >= int64_t(m) * G) return;
    const int32_t g = int32_t(id / m), k = int32_t(id - int64_t(g) * m);
    const int64_t filt = int64_t(m) * KK;
    const int32_t rows = min(N, n - g * N);
    double s = 0.0;
    for (int32_t i = 0; i < rows; ++i) {
        const int64_t base = int64_t(perm[g * N + i]) * filt + int64_t(k) * KK;
        for (int32_t e = 0; e < KK; ++e) s += abs_elem(w, base + e);
    }
    score[int64_t(k) * G + g] = s;
}

__global__ void __launch_bounds__(kSelThreads) mask_select(const double* __restrict__ score, int64_t K,
                                                            int64_t kept, uint8_t* __restrict__ mask) {
    __shared__ uint32_t hist[kSelBins];
    __shared__ uint64_t sPrefix;
    __shared__ int64_t sNeed;
    __shared__ int64_t scan[kSelThreads];
    const int tid = threadIdx.x;

    if (kept <= 0 || kept >= K) {
        const uint8_t v = kept > 0 ? 1 : 0;
        for (int64_t i = tid; i < K; i += kSelThreads) mask[i] = v;
        return;
    }

    // Radix selection, 8 bits at a time from the top: after the pass at
    // `shift`, prefix holds the top bits of the kept-th largest key and need
    // the number of keys with those top bits that still have to be kept.
    if (tid == 0) {
        sPrefix = 0;
        sNeed = kept;
    }
    const int lane = tid & 63;
    uint64_t pmask = 0;
    for (int shift = 56; shift >= 0; shift -= 8) {
        for (int b = tid; b < kSelBins; b += kSelThreads) hist[b] = 0;
        __syncthreads();
        const uint64_t prefix = sPrefix;
        const int64_t need = sNeed;
        // Histogram of the next 8 bits of the candidates.  In the first
        // passes most keys share their top bits: when every candidate lane of
        // a wave hits one bin, a single atomic adds their count (same-address
        // atomics of a whole wave would otherwise serialise).
        for (int64_t i0 = 0; i0 < K; i0 += kSelThreads) {
            const int64_t i = i0 + tid;
            uint64_t key = 0;
            if (i < K) key = order_key(score[i]);
            const bool cand = i < K && (key & pmask) == prefix;
            const uint32_t bin = uint32_t(key >> shift) & 0xff;
            const uint64_t active = __ballot(cand);
            if (active) {
                const int leader = __ffsll(static_cast<unsigned long long>(active)) - 1;
                const uint32_t lb = __shfl(bin, leader);
                if (__ballot(cand && bin == lb) == active) {
                    if (lane == leader) atomicAdd(&hist[lb], uint32_t(__popcll(active)));
                } else if (cand) {
                    atomicAdd(&hist[bin], 1u);
                }
            }
        }
        __syncthreads();
        // Counts from the top bin down (thread c holds bins 255 - c and
        // above): the bin where they reach `need` holds the need-th key.
        if (tid < kSelBins) scan[tid] = hist[kSelBins - 1 - tid];
        __syncthreads();
        for (int d = 1; d < kSelBins; d <<= 1) {
            const int64_t v = (tid < kSelBins && tid >= d) ? scan[tid - d] : 0;
            __syncthreads();
            if (tid < kSelBins) scan[tid] += v;
            __syncthreads();
        }
        if (tid < kSelBins) {
            const int64_t upto = scan[tid], before = tid > 0 ? scan[tid - 1] : 0;
            if (upto >= need && before < need) {
                sNeed = need - before;
                sPrefix = prefix | (uint64_t(kSelBins - 1 - tid) << shift);
            }
        }
        pmask |= uint64_t(0xff) << shift;
        __syncthreads();
    }
    const uint64_t kstar = sPrefix;   // the kept-th largest key
    const int64_t ties = sNeed;       // keys equal to kstar that are kept (the lowest indices)

    // Ties counted in index order: thread tid scans the contiguous slice
    // [tid * per, (tid + 1) * per).
    const int64_t per = (K + kSelThreads - 1) / kSelThreads;
    const int64_t lo = min(K, tid * per), hi = min(K, lo + per);
    int64_t cnt = 0;
    for (int64_t i = lo; i < hi; ++i) cnt += order_key(score[i]) == kstar;
    scan[tid] = cnt;
    __syncthreads();
    for (int d = 1; d < kSelThreads; d <<= 1) {   // inclusive scan
        const int64_t v = tid >= d ? scan[tid - d] : 0;
        __syncthreads();
        scan[tid] += v;
        __syncthreads();
    }
    int64_t before = scan[tid] - cnt;             // ties with a lower index than lo
    for (int64_t i = lo; i < hi; ++i) {
        const uint64_t key = order_key(score[i]);
        uint8_t v = key > kstar ? 1 : 0;
        if (key == kstar) v = before++ < ties ? 1 : 0;
        mask[i] = v;
    }
}

size_t align_up(size_t v) { return (v + kWsAlign - 1) / kWsAlign * kWsAlign; }

// Workspace: norm[n] then score[m*G], fp64.
size_t workspace_bytes(int64_t n, int64_t K) { return align_up(size_t(n) * 8) + align_up(size_t(K) * 8); }

onexn_status check_mask_args(const void* w, onexn_dtype wdt, int32_t n, int32_t m, int32_t kh,
                             int32_t kw, int32_t N, double p, const int32_t* perm,
                             const uint8_t* mask, const int64_t* t) {
    if (!w || !perm || !mask || !t) return fail(ONEXN_ERR_NULL, "build_mask_dev: NULL pointer argument");
    if (wdt != ONEXN_F32 && wdt != ONEXN_BF16)
        return fail(ONEXN_ERR_DTYPE, "build_mask_dev: unknown weight dtype %d", int(wdt));
    if (n < 1 || m < 1 || kh < 1 || kw < 1)
        return fail(ONEXN_ERR_ARG, "build_mask_dev: layer sizes must be >= 1");
    if (N < 1) return fail(ONEXN_ERR_ARG, "build_mask_dev: block length N must be >= 1");
    if (!(p >= 0.0 && p <= 1.0)) return fail(ONEXN_ERR_ARG, "build_mask_dev: p must lie in [0, 1]");
    const int64_t G = (int64_t(n) + N - 1) / N;
    if (int64_t(n) * m * kh * kw > INT32_MAX || int64_t(m) * G > INT32_MAX ||
        G * N * int64_t(kh) * kw > INT32_MAX)
        return fail(ONEXN_ERR_BUFSIZE, "build_mask_dev: layer too large for int32 indexing");
    return ONEXN_OK;
}

template <typename TW>
onexn_status launch_mask(const TW* w, int32_t n, int32_t m, int32_t kh, int32_t kw, int32_t N,
                         int64_t kept, int32_t rearrange, int32_t* perm, uint8_t* mask, void* ws,
                         hipStream_t s) {
    const int32_t G = (n + N - 1) / N;
    const int64_t K = int64_t(m) * G;
    double* norm = static_cast<double*>(ws);
    double* score = reinterpret_cast<double*>(static_cast<char*>(ws) + align_up(size_t(n) * 8));
    const int64_t filt = int64_t(m) * kh * kw;
    if (rearrange) hipLaunchKernelGGL(mask_filter_norms<TW>, dim3((n + 3) / 4), dim3(256), 0, s, w, n, filt, norm);
    hipLaunchKernelGGL(mask_filter_perm, dim3((n + 255) / 256), dim3(256), 0, s, norm, n, rearrange, perm);
    hipLaunchKernelGGL(mask_block_scores<TW>, dim3(uint32_t((K + 255) / 256)), dim3(256), 0, s, w, perm, n, m,
                       kh * kw, N, G, score);
    hipLaunchKernelGGL(mask_select, dim3(1), dim3(kSelThreads), 0, s, score, K, kept, mask);
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess) return fail(ONEXN_ERR_HIP, "build_mask_dev: launch failed: %s", hipGetErrorString(err));
    return ONEXN_OK;
}

int64_t kept_blocks(int64_t K, double p) {
    double pruned = std::floor(p * double(K) + 0.5);
    pruned = std::min(std::max(pruned, 0.0), double(K));
    return K - int64_t(pruned);
}

onexn_status build_mask_dev(const void* w_dev, onexn_dtype wdt, int32_t n, int32_t m, int32_t kh,
                            int32_t kw, int32_t N, double p, int32_t rearrange, int32_t* perm_dev,
                            uint8_t* mask_dev, int64_t* t, void* ws, size_t ws_bytes,
                            void* stream) {
    const int64_t G = (int64_t(n) + N - 1) / N;
    const int64_t K = int64_t(m) * G;
    const int64_t kept = kept_blocks(K, p);
    hipStream_t s = static_cast<hipStream_t>(stream);
    const onexn_status st =
        wdt == ONEXN_F32
            ? launch_mask(static_cast<const float*>(w_dev), n, m, kh, kw, N, kept, rearrange, perm_dev, mask_dev, ws, s)
            : launch_mask(static_cast<const uint16_t*>(w_dev), n, m, kh, kw, N, kept, rearrange, perm_dev, mask_dev, ws, s);
    (void)ws_bytes;
    if (st == ONEXN_OK) *t = kept;
    return st;
}

}  // namespace
}  // namespace onexn

using namespace onexn;

extern "C" size_t onexn_mask_workspace_bytes(int32_t n, int32_t m, int32_t N) {
    if (n < 1 || m < 1 || N < 1) return 0;
    const int64_t G = (int64_t(n) + N - 1) / N;
    return workspace_bytes(n, int64_t(m) * G);
}

extern "C" onexn_status onexn_build_mask_dev(const void* w_dev, onexn_dtype wdt, int32_t n, int32_t m,
                                             int32_t kh, int32_t kw, int32_t N, double p,
                                             int32_t rearrange, int32_t* perm_dev, uint8_t* mask_dev,
                                             int64_t* t, void* workspace_dev, size_t workspace_bytes_,
                                             void* stream) {
    clear_error();
    if (onexn_status st = check_mask_args(w_dev, wdt, n, m, kh, kw, N, p, perm_dev, mask_dev, t)) return st;
    const int64_t G = (int64_t(n) + N - 1) / N;
    const size_t need = workspace_bytes(n, int64_t(m) * G);
    if (!workspace_dev) return fail(ONEXN_ERR_NULL, "build_mask_dev: NULL workspace");
    if (workspace_bytes_ < need)
        return fail(ONEXN_ERR_BUFSIZE, "build_mask_dev: workspace of %zu bytes, %zu needed", workspace_bytes_, need);
    if (reinterpret_cast<uintptr_t>(workspace_dev) % 8 != 0)
        return fail(ONEXN_ERR_ARG, "build_mask_dev: workspace must be 8-byte aligned");
    return build_mask_dev(w_dev, wdt, n, m, kh, kw, N, p, rearrange, perm_dev, mask_dev, t,
                          workspace_dev, workspace_bytes_, stream);
}

extern "C" onexn_status onexn_build_mask_dev_noalloc(const void* w_dev, onexn_dtype wdt, int32_t n,
                                                     int32_t m, int32_t kh, int32_t kw, int32_t N,
                                                     double p, int32_t rearrange, int32_t* perm_dev,
                                                     uint8_t* mask_dev, int64_t* t, void* stream) {
    clear_error();
    if (onexn_status st = check_mask_args(w_dev, wdt, n, m, kh, kw, N, p, perm_dev, mask_dev, t)) return st;
    const int64_t G = (int64_t(n) + N - 1) / N;
    const size_t need = workspace_bytes(n, int64_t(m) * G);
    if (need > kScratchBytes)
        return fail(ONEXN_ERR_BUFSIZE,
                    "build_mask_dev_noalloc: the layer needs %zu bytes of scratch, the entry point holds "
                    "%zu (use onexn_build_mask_dev with a workspace)", need, kScratchBytes);
    void* ws = nullptr;
    if (onexn_status st = scratch_address(&ws)) return st;
    return build_mask_dev(w_dev, wdt, n, m, kh, kw, N, p, rearrange, perm_dev, mask_dev, t, ws,
                          kScratchBytes, stream);
}
