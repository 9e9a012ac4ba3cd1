// 1x1 1xN-pruned convolution (any stride and padding), fp32, NHWC, N in
// {16, 32}: a pixel tile's input channels staged in LDS once and shared by
// eight col-groups.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the contraction
//     Y[pixel][gN .. gN+N-1] = sum_z X[pixel][I[z]] * D[z][0 .. N-1].
// In NHWC a pixel's input channels are contiguous, so the gather of Eq. 8
// picks single values out of each pixel's row: read from global memory, every
// lane of a step would touch its own cache line.  Here a workgroup copies the
// rows of P consecutive output pixels' input pixels (P x m values, coalesced)
// into LDS, with a row pitch of m + 1 floats, so the 32 (16) lanes that read
// one channel at 32 (16) pixels hit distinct banks; the extra column holds a
// zero, read by entries whose channel lies outside [0, m).
//
// Work.  A workgroup of eight waves takes one pixel tile and eight col-groups
// (one per wave); the workgroups of a tile are consecutive, so they run on one
// XCD and read the tile's input through its L2.  Input pixels outside the
// image (padding) and pixels past the last image stage zeros.
//
// Matrix cores.  N = 32: v_mfma_f32_32x32x2f32, lane l takes entry l / 32 of
// a step (two kept blocks) at tile pixel l % 32; N = 16: v_mfma_f32_16x16x4f32,
// entry l / 16 at pixel l % 16.  A: D[z + entry][l % N], one contiguous run of
// the step's weights, loaded straight into registers a batch of eight steps
// ahead.  B: the staged value at (pixel, I[z + entry]); the channel indices
// come in windows of 64 entries (one load per lane) and reach the lane
// groups through ds_bpermute.  Entries past the col-group's end have zero
// weights (the weight buffer ends at the col-group's last block) and read
// the zero column.
//
// Store: lane l holds, per column block, 4-output runs of one pixel
// (consecutive output channels), written with 16-byte stores where n is a
// multiple of 4.

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kNWaves = 8;
constexpr int kNThreads = 64 * kNWaves;
constexpr int kNDB = 8;   // MFMA steps per weight batch

constexpr int64_t kNMaxLds = 160 * 1024;

template <int N, bool kEp>
__global__ void __launch_bounds__(kNThreads) pw_nhwc(ConvArgs a) {
    typedef PwMfma<N> M;
    typedef typename M::acc_t acc_t;
    constexpr int KS = M::KS, COLS = M::COLS;
    constexpr int E = kNDB * KS;   // entries per batch
    static_assert(64 % (2 * E) == 0, "pairs of batches tile an index window");
    extern __shared__ __attribute__((aligned(16))) float sxn[];   // [P][m + 1], then P source offsets

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t m = a.m, pitch = m + 1;
    const int32_t NBLK = a.slices, P = NBLK * COLS;   // column blocks and pixels per tile
    const int32_t gps = a.cost_q;                      // col-groups per workgroup
    const int32_t nsets = (a.G + gps - 1) / gps;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t tile = L / nsets;
    const int32_t g0 = (L - tile * nsets) * gps, gn = min(gps, a.G - g0);
    const float* __restrict__ x = static_cast<const float*>(a.x);
    int64_t* const srco = reinterpret_cast<int64_t*>(sxn + int64_t(P) * pitch + (P & 1));

    // ---- Stage the tile: each pixel's input row offset (-1: padding or past
    // the last image), then all P x m values with consecutive threads on
    // consecutive channels, then the zero column.
    for (int32_t r = tid; r < P; r += kNThreads) {
        const int32_t p = tile * P + r;
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
    const int32_t total = P * m;
    for (int32_t e = tid; e < total; e += kNThreads) {
        const int32_t r = e / m, c = e - r * m;
        const int64_t src = srco[r];
        sxn[r * pitch + c] = src >= 0 ? x[src + c] : 0.f;
    }
    __syncthreads();

    const int col = lane % COLS, kk = lane / COLS;
    float* __restrict__ y = static_cast<float*>(a.y);
    const bool v4 = (a.n & 3) == 0 && (reinterpret_cast<uintptr_t>(a.y) & 15) == 0;

    // ---- (column block, col-group) pairs of the tile, col-group-major, dealt
    // to the waves in turn.
    const int32_t npairs = NBLK * gn;
    for (int32_t i = wave; i < npairs; i += kNWaves) {
        const int32_t gi = i / NBLK, blk = i - gi * NBLK;
        const int32_t g = g0 + gi;
        int32_t zb, ze;
        group_range(a, g, zb, ze);
        const __amdgpu_buffer_rsrc_t rD = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<void*>(a.D), 0, __builtin_amdgcn_readfirstlane(ze * N * 4), kRawBufferFlags);
        const __amdgpu_buffer_rsrc_t rI = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<int32_t*>(a.I), 0, __builtin_amdgcn_readfirstlane(ze * 4), kRawBufferFlags);
        const float* const xl = sxn + (blk * COLS + col) * pitch;   // the lane's pixel

        acc_t acc;
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) acc[r] = 0.f;

        // Batches of kNDB steps: weights loaded a batch ahead into register
        // slot (batch % 2); channel windows of 64 entries.
        const int32_t nbat = (ze - zb + E - 1) / E;
        float av[2][kNDB];
        auto load_w = [&](int sl, int32_t z) __attribute__((always_inline)) {
#pragma unroll
            for (int st = 0; st < kNDB; ++st)
                av[sl][st] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rD, ((z + st * KS) * N + lane) * 4, 0, 0));
        };
        auto mul = [&](int sl, int32_t z, int32_t win) __attribute__((always_inline)) {
            const int32_t base = (z - zb) & 63;   // position of z in its window (windows start at zb + 64 k)
#pragma unroll
            for (int st = 0; st < kNDB; ++st) {
                const int32_t ch = __builtin_amdgcn_ds_bpermute(4 * (base + st * KS + kk), win);
                const bool ok = uint32_t(ch) < uint32_t(m) && z + st * KS + kk < ze;
                acc = M::step(av[sl][st], xl[ok ? ch : m], acc);
            }
        };
        if (nbat > 0) {
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
        }

        // Store: MFMA (row, col) -> output channel g*N + row, tile pixel
        // blk*COLS + col; a lane's rows r0 .. r0+3 are consecutive channels.
        const int32_t p = tile * P + blk * COLS + col;
        if (p < a.npix) {
            float* yp = y + int64_t(p) * a.n;
#pragma unroll
            for (int r0 = 0; r0 < M::ACC; r0 += 4) {
                const int32_t o = g * N + M::row(lane, r0);
                if (v4 && o + 3 < a.n) {
                    f32x4 v;
#pragma unroll
                    for (int q = 0; q < 4; ++q) v[q] = epilogue<kEp>(a, o + q, acc[r0 + q]);
                    store_out(reinterpret_cast<f32x4*>(yp + o), v);
                } else {
#pragma unroll
                    for (int q = 0; q < 4; ++q)
                        if (o + q < a.n) store_out(yp + o + q, epilogue<kEp>(a, o + q, acc[r0 + q]));
                }
            }
        }
    }
}

// LDS of a tile of P pixels: P rows of m + 1 floats, then P 8-byte offsets.
int64_t nhwc_tile_bytes(int64_t P, int32_t m) { return (P * (m + 1) + (P & 1)) * 4 + P * 8; }

template <int N>
onexn_status launch_n(ConvArgs a, hipStream_t s) {
    constexpr int COLS = PwMfma<N>::COLS;
    const int64_t cus = device_cu_count();
    // Column blocks per tile: as many as fit 64 KB (two workgroups per CU),
    // at most 16, at least one (up to the whole LDS for long rows).
    int64_t nblk = 1;
    while (nblk < 16 && nhwc_tile_bytes((nblk + 1) * COLS, a.m) <= 64 * 1024) ++nblk;
    const int64_t P = nblk * COLS;
    const int64_t tiles = (int64_t(a.npix) + P - 1) / P;
    // Col-groups per workgroup: all of them, unless that leaves fewer than
    // two workgroups per CU; then split them into sets (each set re-stages
    // the tile), keeping at least 8 pairs per workgroup.
    int64_t nsets = 1;
    while (tiles * nsets < 2 * cus && (int64_t(a.G) + nsets) / (nsets + 1) * nblk >= kNWaves && nsets < a.G)
        ++nsets;
    const int64_t gps = (a.G + nsets - 1) / nsets;
    nsets = (a.G + gps - 1) / gps;
    const int64_t grid = tiles * nsets;
    const size_t lds = size_t(nhwc_tile_bytes(P, a.m));
    if (grid < 1 || grid > INT32_MAX / kNThreads || P * int64_t(a.m) >= (int64_t(1) << 31))
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: grid of %lld workgroups is out of range", (long long)grid);
    a.total = int32_t(grid);
    a.slices = int32_t(nblk);
    a.cost_q = int32_t(gps);
    return with_epilogue(a, [&](auto ep) {
        constexpr bool E = decltype(ep)::value;
        // (Dynamic LDS above 64 KB must be allowed per kernel.)
        if (hipFuncSetAttribute(reinterpret_cast<const void*>(&pw_nhwc<N, E>),
                                hipFuncAttributeMaxDynamicSharedMemorySize, int(lds)) != hipSuccess)
            return fail(ONEXN_ERR_HIP, "conv2d_fwd: cannot allow %zu bytes of LDS", lds);
        hipLaunchKernelGGL((pw_nhwc<N, E>), dim3(uint32_t(grid)), dim3(kNThreads), lds, s, a);
        const hipError_t err = hipGetLastError();
        if (err != hipSuccess)
            return fail(ONEXN_ERR_HIP, "conv2d_fwd: launch failed: %s", hipGetErrorString(err));
        return ONEXN_OK;
    });
}

}  // namespace

bool pw_nhwc_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_F32 || ydt != ONEXN_F32 || layout != ONEXN_NHWC) return false;
    if (a.N != 16 && a.N != 32) return false;
    if (a.kh != 1 || a.kw != 1) return false;
    // One column block must fit LDS; weight offsets in 32 bits.
    if (nhwc_tile_bytes(a.N == 32 ? 32 : 16, a.m) > kNMaxLds) return false;
    if ((int64_t(a.t) + 64) * a.N * 4 >= (int64_t(1) << 31)) return false;
    return true;
}

onexn_status launch_pw_nhwc(ConvArgs a, hipStream_t s) {
    return a.N == 16 ? launch_n<16>(a, s) : launch_n<32>(a, s);
}

}  // namespace onexn
