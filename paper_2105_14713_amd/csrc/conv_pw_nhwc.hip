// 1x1 1xN-pruned convolution (any stride and padding), fp32, NHWC, N in
// {16, 32}: a pixel tile's input rows staged in LDS once and shared by up to
// eight 16-channel output slices.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the contraction
//     Y[pixel][gN .. gN+N-1] = sum_z X[pixel][I[z]] * D[z][0 .. N-1].
// In NHWC a pixel's input channels are contiguous, so the gather of Eq. 8
// picks single values out of each pixel's row: read from global memory, every
// lane of a step would touch its own cache line.  Here a workgroup copies the
// rows of a tile of T x 16 output pixels' input pixels into LDS (coalesced,
// 16-byte loads where the rows allow, every load of a thread issued before
// the first LDS write), with a row pitch of m + 1 floats, so the 16 lanes that
// read one channel at 16 consecutive pixels hit distinct banks; the extra
// column holds a zero, read by entries whose channel lies outside [0, m).
// Input pixels outside the image (padding) and pixels past the last image
// stage zeros.
//
// Slices.  Every col-group is computed in slices of 16 output channels (one
// for N = 16, two sharing the col-group's kept blocks for N = 32) on
// v_mfma_f32_16x16x4f32: lane l takes entry l / 16 of a step (four kept
// blocks) at pixel l % 16 of a column block.  A: D[z + entry][slice + l % 16];
// B: the staged value at (pixel, I[z + entry]).  A 16-channel slice makes a
// store instruction cover 16 pixels x 64 contiguous bytes (a 32x32 tile's
// would cover 32 pixels x 32 bytes, measured 2-3x slower on write-heavy
// layers).
//
// Work.  A workgroup of eight waves takes one tile and up to eight slices;
// with s < 8 slices, 8 / s waves share each one, taking its column blocks (16
// pixels) in turn, four at a time (four independent accumulators).  The
// workgroups of a tile are consecutive, so they run on one XCD and re-read
// the tile through its L2.
//  - Col-groups of at most 64 kept blocks: the wave loads all of the slice's
//    weights and the LDS offsets of its channels into registers once and
//    reuses them for every column block (the common case for short rows).
//  - Longer col-groups stream: per four column blocks, weights in batches of
//    eight steps loaded a batch ahead; the channel indices in windows of 64
//    entries (one load per lane), handed to the lane groups by ds_bpermute.
// Entries past the col-group's end have zero weights (the weight buffer ends
// at the col-group's last block) and read the zero column.
//
// Store: lane l holds, per column block, 4 consecutive output channels of one
// pixel, written with a 16-byte store where n is a multiple of 4.

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kNWaves = 8;
constexpr int kNThreads = 64 * kNWaves;
constexpr int kNCols = 16;               // pixels per column block
constexpr int kNKS = 4;                  // kept blocks per MFMA step
constexpr int kNBk = 4;                  // column blocks per pass of a wave (at most)
constexpr int kNDB = 8;                  // streamed col-groups: MFMA steps per weight batch
constexpr int kNResEntries = 64;         // longest col-group kept in registers
constexpr int kNStageFloats = 32;        // floats a thread loads per staging batch
constexpr int64_t kNTileLds = 80 * 1024; // LDS of a tile (two workgroups per CU)
constexpr int64_t kNMaxLds = 160 * 1024; // LDS of a CU
constexpr int kNMaxBlocks = 64;          // column blocks per tile

// LDS of a tile of P pixels: P rows of m + 1 floats, then P 8-byte offsets.
int64_t nhwc_tile_bytes(int64_t P, int32_t m) { return (P * (m + 1) + (P & 1)) * 4 + P * 8; }

// Stages the tile's P rows: granules of Q consecutive channels (Q divides m).
// Per batch (kNStageFloats floats, or 16 single floats) a thread first reads
// the row offsets, then issues every load (no branch between them: a granule
// past the tile or of a zero row loads granule 0 and is dropped or zeroed),
// then writes LDS.
template <int Q>
__device__ __forceinline__ void stage_rows(const ConvArgs& a, float* sxn, const int64_t* srco,
                                           int32_t P, int tid) {
    typedef typename VecF<Q>::T V;
    constexpr int SB = Q == 1 ? 16 : kNStageFloats / Q;   // (single floats: registers for 16)
    const int32_t m = a.m, pitch = m + 1, gr = m / Q, total = P * gr;
    const V* __restrict__ x = static_cast<const V*>(a.x);
    for (int32_t e0 = 0; e0 < total; e0 += SB * kNThreads) {
        int64_t src[SB];
        int32_t d[SB];
#pragma unroll
        for (int k = 0; k < SB; ++k) {
            const int32_t e = e0 + k * kNThreads + tid;
            const int32_t ec = e < total ? e : total - 1;
            const int32_t r = ec / gr, c = ec - r * gr;
            const int64_t s = srco[r];
            d[k] = e < total ? r * pitch + c * Q : -1;
            src[k] = s >= 0 ? s / Q + c : -1;
        }
        V v[SB];
#pragma unroll
        for (int k = 0; k < SB; ++k) v[k] = x[src[k] >= 0 ? src[k] : 0];
#pragma unroll
        for (int k = 0; k < SB; ++k)
            if (d[k] >= 0) {
#pragma unroll
                for (int q = 0; q < Q; ++q) sxn[d[k] + q] = src[k] >= 0 ? vec_el<Q>(v[k], q) : 0.f;
            }
    }
}

// H: 16-channel slices per col-group (N = 16 H).
template <int H, int Q, bool kEp>
__global__ void __launch_bounds__(kNThreads) __attribute__((amdgpu_waves_per_eu(4))) pw_nhwc(ConvArgs a) {
    typedef PwMfma<16> M;
    typedef typename M::acc_t acc_t;
    constexpr int N = 16 * H, KS = kNKS, COLS = kNCols;
    constexpr int E = kNDB * KS;                  // streamed: entries per batch
    constexpr int RS = kNResEntries / KS;         // resident: steps
    static_assert(M::KS == KS && M::COLS == COLS, "16x16x4 tiles");
    static_assert(64 % (2 * E) == 0, "pairs of batches tile an index window");
    extern __shared__ __attribute__((aligned(16))) float sxn[];   // [P][m + 1], then P source offsets

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t m = a.m, pitch = m + 1;
    const int32_t T = a.slices, P = T * COLS;     // column blocks and pixels per tile
    const int32_t nsl = a.G * H;                  // slices of the layer
    const int32_t sps = a.cost_q;                 // slices per workgroup
    const int32_t nsets = (nsl + sps - 1) / sps;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t tile = L / nsets;
    const int32_t v0 = (L - tile * nsets) * sps, vn = min(sps, nsl - v0);
    const int32_t p0 = tile * P;
    int64_t* const srco = reinterpret_cast<int64_t*>(sxn + int64_t(P) * pitch + (P & 1));

    // ---- Stage: each pixel's input row offset (-1: padding or past the last
    // image) and zero column, then the rows.
    for (int32_t r = tid; r < P; r += kNThreads) {
        const int32_t p = p0 + r;
        int64_t src = -1;
        if (p < a.npix) {
            const int32_t b = p / a.HWo, hw = p - b * a.HWo;
            const int32_t oh = hw / a.Wo, ow = hw - oh * a.Wo;
            const int32_t ih = oh * a.sh - a.ph, iw = ow * a.sw - a.pw;
            if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
                src = int64_t(b) * a.x_img + (int64_t(ih) * a.W + iw) * m;
        }
        srco[r] = src;
        sxn[r * pitch + m] = 0.f;
    }
    __syncthreads();
    stage_rows<Q>(a, sxn, srco, P, tid);
    __syncthreads();

    // ---- The wave's slice and its share of the tile's column blocks.
    const int32_t wpg = kNWaves / vn;
    if (wave >= vn * wpg) return;
    const int32_t vi = wave / wpg, sub = wave - vi * wpg;
    const int32_t v = v0 + vi, g = v / H, h = v - g * H;
    const int32_t ob = g * N + h * 16;            // the slice's first output channel
    if (ob >= a.n) return;                        // (second slice of a ragged last col-group)
    const int32_t nblk = min(T, (a.npix - p0 + COLS - 1) / COLS);   // blocks holding pixels
    int32_t zb, ze;
    group_range(a, g, zb, ze);
    const __amdgpu_buffer_rsrc_t rD = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.D), 0, __builtin_amdgcn_readfirstlane(ze * N * 4), kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rI = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(a.I), 0, __builtin_amdgcn_readfirstlane(ze * 4), kRawBufferFlags);
    const int col = lane % COLS, kk = lane / COLS;
    const int32_t wl = (kk * N + h * 16 + col) * 4;   // the lane's weight in a step, bytes past D[z]
    const float* const xl = sxn + col * pitch;    // the lane's pixel in column block 0
    const int32_t bstride = COLS * pitch;         // floats between column blocks
    float* __restrict__ y = static_cast<float*>(a.y);
    const bool v4 = (a.n & 3) == 0 && (reinterpret_cast<uintptr_t>(a.y) & 15) == 0;
    const int32_t o = ob + M::row(lane, 0);       // the lane's 4 output channels o .. o+3

    // MFMA (row, col) of column block b -> output channel ob + row, pixel
    // p0 + b*COLS + col.
    auto store = [&](int32_t b, const acc_t& acc) __attribute__((always_inline)) {
        const int32_t p = p0 + b * COLS + col;
        if (p >= a.npix) return;
        float* yp = y + int64_t(p) * a.n + o;
        if (v4 && o + 3 < a.n) {
            f32x4 r;
#pragma unroll
            for (int q = 0; q < 4; ++q) r[q] = epilogue<kEp>(a, o + q, acc[q]);
            store_out(reinterpret_cast<f32x4*>(yp), r);
        } else {
#pragma unroll
            for (int q = 0; q < 4; ++q)
                if (o + q < a.n) store_out(yp + q, epilogue<kEp>(a, o + q, acc[q]));
        }
    };
    // A pass: NB column blocks b0 + j*wpg (NB independent accumulators).
    auto zero = [&](auto& c) __attribute__((always_inline)) {
#pragma unroll
        for (int j = 0; j < int(sizeof(c) / sizeof(c[0])); ++j)
#pragma unroll
            for (int r = 0; r < M::ACC; ++r) c[j][r] = 0.f;
    };
    // The pass loop: four blocks at a time while at least three remain, then
    // two or one (no multiply for a block that is not there).
    auto passes = [&](auto&& pass) __attribute__((always_inline)) {
        for (int32_t b0 = sub; b0 < nblk;) {
            const int32_t left = (nblk - 1 - b0) / wpg + 1;   // blocks of this wave from b0 on
            if (left >= 3) {
                pass(b0, std::integral_constant<int, 4>());
                b0 += 4 * wpg;
            } else if (left == 2) {
                pass(b0, std::integral_constant<int, 2>());
                b0 += 2 * wpg;
            } else {
                pass(b0, std::integral_constant<int, 1>());
                b0 += wpg;
            }
        }
    };
    // Block b0 + j*wpg's row pointer (past the last block: b0's, not stored).
    auto row_of = [&](int32_t b0, int j) __attribute__((always_inline)) {
        const int32_t b = b0 + j * wpg;
        return xl + (b < nblk ? b : b0) * bstride;
    };

    const int32_t ns = (ze - zb + KS - 1) / KS;   // MFMA steps of the col-group
    if (ns <= RS) {
        // ---- Resident: the slice's weights and channel offsets in registers.
        float aw[RS];
        int32_t off[RS];
#pragma unroll
        for (int st = 0; st < RS; ++st) {
            aw[st] = 0.f;
            off[st] = m;
            if (st < ns) {   // uniform
                const int32_t z = zb + st * KS + kk;
                aw[st] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rD, (zb + st * KS) * N * 4 + wl, 0, 0));
                const int32_t ch = int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, z * 4, 0, 0));
                off[st] = (z < ze && uint32_t(ch) < uint32_t(m)) ? ch : m;
            }
        }
        passes([&](int32_t b0, auto nb) __attribute__((always_inline)) {
            constexpr int NB = decltype(nb)::value;
            const float* xs[NB];
            acc_t c[NB];
#pragma unroll
            for (int j = 0; j < NB; ++j) xs[j] = row_of(b0, j);
            zero(c);
#pragma unroll
            for (int st = 0; st < RS; ++st) {
                if (st < ns) {   // uniform
#pragma unroll
                    for (int j = 0; j < NB; ++j) c[j] = M::step(aw[st], xs[j][off[st]], c[j]);
                }
            }
#pragma unroll
            for (int j = 0; j < NB; ++j)
                if (b0 + j * wpg < nblk) store(b0 + j * wpg, c[j]);
        });
        return;
    }

    // ---- Streamed: per pass, batches of kNDB steps with weights loaded a
    // batch ahead into register slot (batch % 2).
    const int32_t nbat = (ze - zb + E - 1) / E;
    passes([&](int32_t b0, auto nb) __attribute__((always_inline)) {
        constexpr int NB = decltype(nb)::value;
        const float* xs[NB];
        acc_t c[NB];
#pragma unroll
        for (int j = 0; j < NB; ++j) xs[j] = row_of(b0, j);
        zero(c);
        float av[2][kNDB];
        auto load_w = [&](int sl, int32_t z) __attribute__((always_inline)) {
#pragma unroll
            for (int st = 0; st < kNDB; ++st)
                av[sl][st] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rD, (z + st * KS) * N * 4 + wl, 0, 0));
        };
        auto mul = [&](int sl, int32_t z, int32_t win) __attribute__((always_inline)) {
            const int32_t base = (z - zb) & 63;   // position of z in its window (windows start at zb + 64 k)
#pragma unroll
            for (int st = 0; st < kNDB; ++st) {
                const int32_t ch = __builtin_amdgcn_ds_bpermute(4 * (base + st * KS + kk), win);
                const bool ok = uint32_t(ch) < uint32_t(m) && z + st * KS + kk < ze;
                const int32_t of = ok ? ch : m;
#pragma unroll
                for (int j = 0; j < NB; ++j) c[j] = M::step(av[sl][st], xs[j][of], c[j]);
            }
        };
        int32_t win = int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, (zb + lane) * 4, 0, 0));
        load_w(0, zb);
        for (int32_t j = 0; j < nbat; j += 2) {
            const int32_t z = zb + j * E;
            load_w(1, z + E);
            mul(0, z, win);
            if (j + 1 >= nbat) break;
            load_w(0, z + 2 * E);
            mul(1, z + E, win);
            if (((j + 2) * E) % 64 == 0)
                win = int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, (z + 2 * E + lane) * 4, 0, 0));
        }
#pragma unroll
        for (int j = 0; j < NB; ++j)
            if (b0 + j * wpg < nblk) store(b0 + j * wpg, c[j]);
    });
}

template <int H, int Q>
onexn_status launch_q(ConvArgs a, int64_t grid, size_t lds, hipStream_t s) {
    return with_epilogue(a, [&](auto ep) {
        constexpr bool E = decltype(ep)::value;
        // (Dynamic LDS above 64 KB must be allowed per kernel.)
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(&pw_nhwc<H, Q, E>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
            return fail(ONEXN_ERR_HIP, "conv2d_fwd: cannot allow %zu bytes of LDS", lds);
        hipLaunchKernelGGL((pw_nhwc<H, Q, E>), dim3(uint32_t(grid)), dim3(kNThreads), lds, s, a);
        const hipError_t err = hipGetLastError();
        if (err != hipSuccess)
            return fail(ONEXN_ERR_HIP, "conv2d_fwd: launch failed: %s", hipGetErrorString(err));
        return ONEXN_OK;
    });
}

template <int H>
onexn_status launch_h(ConvArgs a, hipStream_t s) {
    const int64_t cus = device_cu_count();
    const int64_t blocks = (int64_t(a.npix) + kNCols - 1) / kNCols;
    const int64_t nsl = int64_t(a.G) * H;
    const int64_t sps = nsl < kNWaves ? nsl : kNWaves;
    const int64_t nsets = (nsl + sps - 1) / sps;
    const int64_t wpg = kNWaves / sps;
    // Column blocks per tile: two passes of kNBk blocks per wave, fewer where
    // the tile LDS or two workgroups per CU do not allow it.
    const int64_t fit = kNTileLds / nhwc_tile_bytes(kNCols, a.m);
    int64_t T = std::min<int64_t>({int64_t(kNMaxBlocks), fit, 2 * kNBk * wpg});
    T = std::max<int64_t>(1, std::min<int64_t>(T, blocks * nsets / (2 * cus)));
    if (tuning(kTuneNhwcTile) >= 1)   // (at most what fits the CU's LDS)
        T = std::max<int64_t>(1, std::min<int64_t>(tuning(kTuneNhwcTile),
                                                   kNMaxLds / nhwc_tile_bytes(kNCols, a.m)));
    const int64_t tiles = (blocks + T - 1) / T;
    const int64_t grid = tiles * nsets;
    const size_t lds = size_t(nhwc_tile_bytes(T * kNCols, a.m));
    if (grid < 1 || grid > INT32_MAX / kNThreads || T * kNCols * int64_t(a.m + 1) >= (int64_t(1) << 31) ||
        int64_t(lds) > kNMaxLds)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: NHWC tile of %lld blocks does not fit", (long long)T);
    a.total = int32_t(grid);
    a.slices = int32_t(T);
    a.cost_q = int32_t(sps);
    const bool quads = a.m % 4 == 0 && (reinterpret_cast<uintptr_t>(a.x) & 15) == 0;
    return quads ? launch_q<H, 4>(a, grid, lds, s) : launch_q<H, 1>(a, grid, lds, s);
}

}  // namespace

bool pw_nhwc_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_F32 || ydt != ONEXN_F32 || layout != ONEXN_NHWC) return false;
    if (a.N != 16 && a.N != 32) return false;
    if (a.kh != 1 || a.kw != 1) return false;
    // One column block's tile fits 80 KB (rows of up to 1277 channels).
    if (nhwc_tile_bytes(kNCols, a.m) > kNTileLds) return false;
    if ((int64_t(a.t) + 64) * a.N * 4 >= (int64_t(1) << 31)) return false;
    return true;
}

onexn_status launch_pw_nhwc(ConvArgs a, hipStream_t s) {
    return a.N == 16 ? launch_h<1>(a, s) : launch_h<2>(a, s);
}

}  // namespace onexn
