// Host side of libonexn.so: mask building (filter rearrangement, block
// scoring, per-layer top-(1-p) selection) and BSR packing.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.2-3.4.  The results are integer/bit data and are
// defined exactly (fixed fp64 summation order, fixed tie rules, fixed
// rounding of p*K), so they are reproducible bit for bit.
#include <algorithm>
#include <cmath>
#include <cstdio>
#include <cstring>
#include <numeric>
#include <vector>

#include "onexn_internal.h"

namespace onexn {

namespace {

thread_local char g_last_error[512] = "";

inline double bf16_bits_to_double(uint16_t b) {
    uint32_t u = static_cast<uint32_t>(b) << 16;
    float f;
    std::memcpy(&f, &u, sizeof f);
    return static_cast<double>(f);
}

// Absolute value of element e of the weight tensor, exactly, in fp64.
struct AbsReader {
    const void* w;
    onexn_dtype dt;
    double operator()(int64_t e) const {
        if (dt == ONEXN_F32) return std::fabs(static_cast<double>(static_cast<const float*>(w)[e]));
        return std::fabs(bf16_bits_to_double(static_cast<const uint16_t*>(w)[e]));
    }
};

size_t dtype_size(onexn_dtype dt) { return dt == ONEXN_F32 ? 4 : 2; }

bool valid_dtype(int dt) { return dt == ONEXN_F32 || dt == ONEXN_BF16; }

onexn_status check_layer(int32_t n, int32_t m, int32_t kh, int32_t kw, int32_t N) {
    if (n < 1 || m < 1 || kh < 1 || kw < 1)
        return fail(ONEXN_ERR_ARG, "layer sizes must be >= 1 (n=%d m=%d kh=%d kw=%d)", n, m, kh, kw);
    if (N < 1) return fail(ONEXN_ERR_ARG, "block length N must be >= 1 (got %d)", N);
    const int64_t elems = int64_t(n) * m * kh * kw;
    const int64_t G = (int64_t(n) + N - 1) / N;
    if (elems > INT32_MAX || int64_t(m) * G > INT32_MAX || G * N * int64_t(kh) * kw > INT32_MAX)
        return fail(ONEXN_ERR_BUFSIZE, "layer too large for int32 indexing");
    return ONEXN_OK;
}

}  // namespace

onexn_status fail(onexn_status s, const char* fmt, ...) {
    va_list ap;
    va_start(ap, fmt);
    std::vsnprintf(g_last_error, sizeof g_last_error, fmt, ap);
    va_end(ap);
    return s;
}

void clear_error() { g_last_error[0] = '\0'; }

}  // namespace onexn

using namespace onexn;

extern "C" const char* onexn_status_string(onexn_status s) {
    switch (s) {
        case ONEXN_OK: return "ONEXN_OK";
        case ONEXN_ERR_NULL: return "ONEXN_ERR_NULL";
        case ONEXN_ERR_ARG: return "ONEXN_ERR_ARG";
        case ONEXN_ERR_SHAPE: return "ONEXN_ERR_SHAPE";
        case ONEXN_ERR_DTYPE: return "ONEXN_ERR_DTYPE";
        case ONEXN_ERR_UNSUPPORTED: return "ONEXN_ERR_UNSUPPORTED";
        case ONEXN_ERR_BUFSIZE: return "ONEXN_ERR_BUFSIZE";
        case ONEXN_ERR_HIP: return "ONEXN_ERR_HIP";
    }
    return "ONEXN_UNKNOWN";
}

extern "C" const char* onexn_last_error(void) { return g_last_error; }

// Sec. 3.3 (rearrangement) + Eq. 4-5 (block l1 scores) + Eq. 1 / Sec. 4.1
// (per-layer top-(1-p) selection).
extern "C" onexn_status onexn_build_mask(const void* w, onexn_dtype wdt, int32_t n, int32_t m,
                                         int32_t kh, int32_t kw, int32_t N, double p,
                                         int32_t rearrange, int32_t* perm, uint8_t* mask,
                                         int64_t* t) {
    clear_error();
    if (!w || !perm || !mask || !t) return fail(ONEXN_ERR_NULL, "build_mask: NULL pointer argument");
    if (!valid_dtype(wdt)) return fail(ONEXN_ERR_DTYPE, "build_mask: unknown weight dtype %d", int(wdt));
    if (onexn_status s = check_layer(n, m, kh, kw, N)) return s;
    if (!(p >= 0.0 && p <= 1.0)) return fail(ONEXN_ERR_ARG, "build_mask: p must lie in [0, 1]");

    const AbsReader absw{w, wdt};
    const int64_t filt = int64_t(m) * kh * kw;   // elements per filter
    const int32_t KK = kh * kw;
    const int32_t G = (n + N - 1) / N;
    const int64_t K = int64_t(m) * G;

    // Filter order.  A filter is contiguous in memory in (k, q, r) order, so
    // one linear pass sums its l1 norm in that order.
    std::vector<int32_t> order(n);
    std::iota(order.begin(), order.end(), 0);
    if (rearrange) {
        std::vector<double> norm(n);
        for (int32_t j = 0; j < n; ++j) {
            double s = 0.0;
            for (int64_t e = 0; e < filt; ++e) s += absw(j * filt + e);
            if (std::isnan(s)) return fail(ONEXN_ERR_ARG, "build_mask: NaN in filter %d", j);
            norm[j] = s;
        }
        std::stable_sort(order.begin(), order.end(),
                         [&](int32_t a, int32_t b) { return norm[a] > norm[b]; });
    }

    // Block scores of the rearranged matrix, stored by row-major block index
    // k*G + g.  Sum over block rows i, then the kernel's taps.
    std::vector<double> score(K);
    for (int32_t k = 0; k < m; ++k) {
        for (int32_t g = 0; g < G; ++g) {
            double s = 0.0;
            const int32_t rows = std::min(N, n - g * N);
            for (int32_t i = 0; i < rows; ++i) {
                const int64_t base = int64_t(order[g * N + i]) * filt + int64_t(k) * KK;
                for (int32_t e = 0; e < KK; ++e) s += absw(base + e);
            }
            if (std::isnan(s)) return fail(ONEXN_ERR_ARG, "build_mask: NaN in block (%d,%d)", k, g);
            score[int64_t(k) * G + g] = s;
        }
    }

    // Per-layer selection.  The order "higher score first, then lower block
    // index" is a strict total order, so the kept set is the first `kept`
    // elements of it, found with a partial partition.
    double pruned = std::floor(p * double(K) + 0.5);
    pruned = std::min(std::max(pruned, 0.0), double(K));
    const int64_t kept = K - int64_t(pruned);
    std::vector<int64_t> idx(K);
    std::iota(idx.begin(), idx.end(), int64_t(0));
    auto before = [&](int64_t a, int64_t b) {
        return score[a] > score[b] || (score[a] == score[b] && a < b);
    };
    if (kept > 0 && kept < K) std::nth_element(idx.begin(), idx.begin() + kept, idx.end(), before);

    std::memcpy(perm, order.data(), sizeof(int32_t) * size_t(n));
    std::memset(mask, 0, size_t(K));
    for (int64_t i = 0; i < kept; ++i) mask[idx[i]] = 1;
    *t = kept;
    return ONEXN_OK;
}

// Sec. 3.4 / Fig. 3: BSR encoding (D, I, P) of the masked, rearranged weights.
extern "C" onexn_status onexn_pack(const void* w, onexn_dtype wdt, int32_t n, int32_t m,
                                   int32_t kh, int32_t kw, int32_t N, const int32_t* perm,
                                   const uint8_t* mask, int64_t t, int32_t* P, int32_t* I,
                                   void* D) {
    clear_error();
    if (!w || !perm || !mask || !P) return fail(ONEXN_ERR_NULL, "pack: NULL pointer argument");
    if (t > 0 && (!I || !D)) return fail(ONEXN_ERR_NULL, "pack: NULL I or D with t > 0");
    if (!valid_dtype(wdt)) return fail(ONEXN_ERR_DTYPE, "pack: unknown weight dtype %d", int(wdt));
    if (onexn_status s = check_layer(n, m, kh, kw, N)) return s;
    const int32_t G = (n + N - 1) / N;
    const int64_t K = int64_t(m) * G;
    if (t < 0 || t > K) return fail(ONEXN_ERR_ARG, "pack: t=%lld outside [0, m*G]", (long long)t);

    std::vector<uint8_t> seen(n, 0);
    for (int32_t j = 0; j < n; ++j) {
        if (perm[j] < 0 || perm[j] >= n || seen[perm[j]])
            return fail(ONEXN_ERR_ARG, "pack: perm is not a permutation of 0..n-1 (entry %d)", j);
        seen[perm[j]] = 1;
    }
    // Count the kept blocks of every col-group.
    std::vector<int64_t> count(G, 0);
    for (int32_t k = 0; k < m; ++k)
        for (int32_t g = 0; g < G; ++g) {
            const uint8_t v = mask[int64_t(k) * G + g];
            if (v > 1) return fail(ONEXN_ERR_ARG, "pack: mask entry (%d,%d) is not 0/1", k, g);
            count[g] += v;
        }
    int64_t total = 0;
    for (int32_t g = 0; g < G; ++g) total += count[g];
    if (total != t) return fail(ONEXN_ERR_ARG, "pack: t=%lld but mask keeps %lld blocks",
                                (long long)t, (long long)total);

    // Col-group starts (exclusive prefix sum), then scatter the blocks with
    // one cursor per col-group while walking input channels in order, which
    // leaves each col-group's blocks in ascending k.
    std::vector<int64_t> cursor(G);
    int64_t run = 0;
    for (int32_t g = 0; g < G; ++g) {
        P[g] = int32_t(run);
        cursor[g] = run;
        run += count[g];
    }
    P[G] = int32_t(run);

    const size_t es = dtype_size(wdt);
    const int64_t KK = int64_t(kh) * kw;
    const int64_t filt = int64_t(m) * KK;
    const int64_t blk = int64_t(N) * KK;       // elements per stored block
    const auto* src = static_cast<const uint8_t*>(w);
    auto* dst = static_cast<uint8_t*>(D);
    for (int32_t k = 0; k < m; ++k) {
        for (int32_t g = 0; g < G; ++g) {
            if (!mask[int64_t(k) * G + g]) continue;
            const int64_t z = cursor[g]++;
            I[z] = k;
            for (int32_t i = 0; i < N; ++i) {
                uint8_t* out = dst + size_t((z * blk + int64_t(i) * KK) * es);
                const int32_t j = g * N + i;
                if (j < n)
                    std::memcpy(out, src + size_t((int64_t(perm[j]) * filt + int64_t(k) * KK) * es),
                                size_t(KK) * es);
                else
                    std::memset(out, 0, size_t(KK) * es);
            }
        }
    }
    return ONEXN_OK;
}
