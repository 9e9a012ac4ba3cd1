// Pointwise (1x1, stride 1, no padding, NCHW) 1xN-pruned convolution with
// bf16 inputs and weights, fp32 accumulation, N = 32, bf16 or fp32 output,
// for layers with many input channels: a pixel tile's input rows are staged
// in LDS once and shared by 15 col-groups.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the contraction
//     Y_g[32][pixels] = D_g^T[32][kept_g] * X[I_g][pixels].
// Each col-group keeps its own subset of the input rows, so a kernel in which
// every col-group gathers its rows itself moves each input row through L2 once
// per col-group that keeps it.  Here a workgroup covers one tile of 128
// pixels for 15 col-groups: the tile's rows stream through LDS in chunks of
// 128 channels, each fetched once, and every col-group reads the rows it
// keeps from there.
//
// Work.  A work item is (pixel tile, set of 15 col-groups); the sets of a
// tile are consecutive items, so they run at the same time on one XCD and
// share the tile's rows in its L2.  A tile is 16 granules of 8 consecutive
// pixels of one image (an image's last granule may be half-filled: its extra
// columns are computed and not stored).  Workgroups walk items in a
// persistent loop.
//
// Waves.  Waves 0-14 compute, one col-group each; wave 15 copies X chunks
// into a ring of four LDS buffers (buffer-to-LDS loads, 1 KB per
// instruction) two chunks ahead.  Chunks are handed over at barriers: during
// epoch e of an item, chunks e - 1 and e are resident while chunks e + 1 and
// e + 2 are copied into the other two buffers.  The ring runs on across
// items.  Every wave passes the same number of barriers per item (one per
// chunk), wherever in its loop it waits.
//
// Windows.  v_mfma_f32_32x32x16_bf16 takes 16 contraction entries: window j
// of a col-group is its kept blocks 16 j .. 16 j + 15.  With I ascending, a
// window's channels lie between those of its first and last entries; it is
// multiplied in the epoch of its last entry's chunk when it spans at most
// two chunks, else in several passes over at most two chunks each (A reused,
// entries of other chunks masked).  Entries past the col-group's end and
// channels outside [0, m) read a zero row for both fragments.
//
// Operands.  The compute waves load only through ordinary buffer loads into
// registers, a few windows ahead (their waits are the compiler's): for each
// window, the lane's 16 bytes of its 16 blocks of D (16 x 32 bf16, one
// contiguous kilobyte) and the channels of the lane's two fragment entries.
// The next item's first windows are loaded before this item's results are
// stored: stores and loads share one completion counter, so loads issued
// after the stores would make the next item wait for all of them.
// A: the window's weights are written to the wave's LDS slot and read
// transposed with ds_read_b64_tr_b16.  B: the same instruction reads each
// entry's staged input row, transposed, for each of the tile's four 32-pixel
// column blocks.  Rows are stored in groups of four followed by 64 bytes of
// padding, so the rows one transposed read touches spread over the LDS banks.

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kSCompute = 15;                       // compute waves, one col-group each
constexpr int kSThreads = 64 * (kSCompute + 1);     // + the loader wave
constexpr int kSKc = 128;                           // input channels per chunk
constexpr int kSGran = 16;                          // 8-pixel granules per tile
constexpr int kSBlocks = 4;                         // 32-pixel MFMA column blocks per tile
constexpr int kSRowB = 2 * 8 * kSGran;              // bytes of one channel row of a tile
constexpr int kSQuadB = 4 * kSRowB + 64;            // four rows, then 64 bytes of padding
constexpr int kSRing = 4;                           // chunk buffers
constexpr int kSRingRows = kSRing * kSKc;           // ring rows (a power of two)
constexpr int kSBufB = (kSKc / 4) * kSQuadB;        // one chunk buffer
constexpr int kSZeroOff = kSRing * kSBufB;          // a zero row after the ring
constexpr int kSAOff = kSZeroOff + kSRowB;          // one weight slot per compute wave
constexpr int kSSlotB = 16 * 64;                    // a window's weights: 16 blocks x 32 bf16
constexpr int kSLds = kSAOff + kSCompute * kSSlotB;
constexpr int kSAhead = 3;                          // windows loaded ahead (register slots)
static_assert(kSLds <= 160 * 1024, "LDS of one workgroup");
static_assert(kSRowB * 4 == 1024, "one buffer-to-LDS copy fills four rows");

typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4i16 tr_read(const lds_char* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p);
}

__device__ __forceinline__ bf16x8 join(v4i16 lo, v4i16 hi) {
    return __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// LDS byte offset of ring row R (0 <= R < kSRingRows): R * 256 + (R / 4) * 64.
__device__ __forceinline__ int32_t ring_row_off(int32_t R) { return (R << 8) + ((R >> 2) << 6); }

template <typename TY, bool kEp>
__global__ void __launch_bounds__(kSThreads) pw_bf16s(ConvArgs a) {
    __shared__ __attribute__((aligned(16))) char sX[kSLds];
    // Fused epilogue: one 64-entry slot per compute wave (its current
    // col-group's 32 scales, then 32 biases).
    __shared__ __attribute__((aligned(16))) float sEp[kEp ? kSCompute * 64 : 4];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t batch = a.npix / a.HWo;
    const int32_t gpi = (a.HWo + 7) >> 3;               // granules per image
    const int32_t ngran = batch * gpi;
    const int32_t ntiles = (ngran + kSGran - 1) / kSGran;
    const int32_t nsets = (a.G + kSCompute - 1) / kSCompute;
    const int32_t nitems = ntiles * nsets;
    const int32_t nch = (a.m + kSKc - 1) / kSKc;         // chunks per item
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t nloc = L < nitems ? (nitems - 1 - L) / a.total + 1 : 0;   // items of this workgroup
    const lds_char* const lx = (const lds_char*)sX;

    for (int i = tid; i < kSRowB / 4; i += kSThreads) reinterpret_cast<int32_t*>(sX + kSZeroOff)[i] = 0;

    if (wave == kSCompute) {
        // ---- Loader.  Global epoch s = k * nch + c (item k of this
        // workgroup, chunk c) goes to buffer s % kSRing.  Lane l copies
        // granule l % 16 (16 bytes) of row l / 16 of each four-row copy.
        __builtin_amdgcn_s_setprio(3);
        const int32_t xbytes = int32_t(int64_t(batch) * a.x_img * 2);
        const v4i32 rX = buffer_rsrc(a.x, xbytes);
        const int h = lane >> 4, gran = lane & 15;
        const int32_t rowb = a.HWo * 2;
        auto issue = [&](int32_t s) {
            const int32_t k = s / nch, c = s - k * nch;
            const int32_t tile = (L + k * a.total) / nsets;
            const int32_t id = tile * kSGran + gran;
            uint32_t pbase = uint32_t(xbytes);   // past the last image: reads zeros
            if (id < ngran) {
                const int32_t b = id / gpi, j = id - b * gpi;
                pbase = uint32_t(int64_t(b) * a.x_img * 2) + 16 * j;
            }
            const lds_char* dst = lx + (s % kSRing) * kSBufB;
#pragma unroll 8
            for (int i = 0; i < kSKc / 4; ++i) {
                // rows past m copy a real row (never read)
                const int32_t ch = min(c * kSKc + 4 * i + h, a.m - 1);
                copy16_to_lds(rX, dst + i * kSQuadB, int32_t(pbase + uint32_t(ch) * uint32_t(rowb)), 0);
            }
        };
        // Before epoch s ends, chunk s + 1 has landed (the kSKc / 4 copies
        // of chunk s + 2 may still be in flight).
        const int32_t total_s = nloc * nch;
        if (total_s > 0) issue(0);
        if (total_s > 1) {
            issue(1);
            vm_wait<kSKc / 4>();
        } else {
            vm_wait<0>();
        }
        __syncthreads();
        for (int32_t s = 0; s < total_s; ++s) {
            if (s + 2 < total_s) {
                issue(s + 2);
                vm_wait<kSKc / 4>();
            } else {
                vm_wait<0>();
            }
            __syncthreads();
        }
        return;
    }

    // ---- Compute waves.
    const int w = wave;
    char* const slot = sX + kSAOff + w * kSSlotB;
    const int32_t aoff = kSAOff + w * kSSlotB;
    // Transposed-read roles, the same for both fragments: lane l reads entry
    // k1 (and k1 + 4) at 4 consecutive elements from byte colb of a 64-byte
    // block (A: outputs of the block; B: pixels of a column block).
    const int k1 = 8 * (lane >> 5) + ((lane & 15) >> 2);
    const int colb = 32 * ((lane >> 4) & 1) + 8 * (lane & 3);
    TY* __restrict__ y = static_cast<TY*>(a.y);
    __syncthreads();   // the first chunk has landed

    // A work item as seen by one compute wave.
    struct Item {
        int32_t tile, g, nE, nwin, kbase;
        __amdgpu_buffer_rsrc_t rA, rI;
    };
    auto item_at = [&](int32_t k) {
        Item t;
        const int32_t item = L + k * a.total;
        t.tile = item / nsets;
        t.g = (item - t.tile * nsets) * kSCompute + w;
        int32_t zb = 0, ze = 0;
        if (t.g < a.G) group_range(a, t.g, zb, ze);
        t.nE = ze - zb;
        t.nwin = (t.nE + 15) >> 4;
        // Ring row of channel ch in this item: (ch + kbase) mod kSRingRows.
        t.kbase = ((k * nch) % kSRing) * kSKc;
        // Both resources start at the col-group's first block and end at its
        // last: entries past the end read zero channels and zero weights.
        t.rA = __builtin_amdgcn_make_buffer_rsrc(
            const_cast<char*>(static_cast<const char*>(a.D) + int64_t(zb) * 64), 0, t.nE * 64, kRawBufferFlags);
        t.rI = __builtin_amdgcn_make_buffer_rsrc(const_cast<int32_t*>(a.I + zb), 0, t.nE * 4, kRawBufferFlags);
        return t;
    };

    // Register slots: a window's weights and the lane's two channels.
    i32x4 av[kSAhead];
    int32_t c1[kSAhead], c2[kSAhead];
    auto load = [&](const Item& t, int u, int32_t j) __attribute__((always_inline)) {
        av[u] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(t.rA, j * 1024 + lane * 16, 0, 0));
        c1[u] = int32_t(__builtin_amdgcn_raw_buffer_load_b32(t.rI, (16 * j + k1) * 4, 0, 0));
        c2[u] = int32_t(__builtin_amdgcn_raw_buffer_load_b32(t.rI, (16 * j + k1 + 4) * 4, 0, 0));
    };

    Item it = item_at(0);
    if (nloc > 0) {
#pragma unroll
        for (int u = 0; u < kSAhead; ++u) load(it, u, u);
    }
    for (int32_t k = 0; k < nloc; ++k) {
        f32x16 acc[kSBlocks];
#pragma unroll
        for (int e = 0; e < kSBlocks; ++e)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[e][r] = 0.f;

        int32_t epoch = 0;   // chunks 0 .. epoch of this item have landed
        auto process = [&](int u, int32_t j) __attribute__((always_inline)) {
            const int32_t cnt = min(16, it.nE - 16 * j);
            // First and last entries (entry e sits in lane 4 (e % 4) + 32 (e / 8),
            // in c2 when e % 8 >= 4); channels clamped into [0, m) for gating.
            const int32_t el = cnt - 1;
            const int32_t lanel = 4 * (el & 3) + 32 * (el >> 3);
            const int32_t lastc = (el & 4) ? __builtin_amdgcn_readlane(c2[u], lanel)
                                           : __builtin_amdgcn_readlane(c1[u], lanel);
            const int32_t firstc = __builtin_amdgcn_readlane(c1[u], 0);
            const int32_t qf = min(max(firstc, 0), a.m - 1) / kSKc;
            const int32_t ql = min(max(lastc, 0), a.m - 1) / kSKc;
            *reinterpret_cast<i32x4*>(slot + lane * 16) = av[u];
            const bool ok1 = (k1 < cnt) & (uint32_t(c1[u]) < uint32_t(a.m));
            const bool ok2 = (k1 + 4 < cnt) & (uint32_t(c2[u]) < uint32_t(a.m));
            const int32_t xr1 = ring_row_off((c1[u] + it.kbase) & (kSRingRows - 1));
            const int32_t xr2 = ring_row_off((c2[u] + it.kbase) & (kSRingRows - 1));
            const int32_t q1 = c1[u] >> 7, q2 = c2[u] >> 7;
            // Passes over chunks (lo, hi], at most two each, ending at ql.
            int32_t lo = qf - 1;
            while (true) {
                const int32_t hi = min(lo + 2, ql);
                while (epoch < hi) {
                    __syncthreads();
                    ++epoch;
                }
                const bool in1 = ok1 & (q1 > lo) & (q1 <= hi), in2 = ok2 & (q2 > lo) & (q2 <= hi);
                const int32_t xo1 = in1 ? xr1 : kSZeroOff, xo2 = in2 ? xr2 : kSZeroOff;
                const int32_t ao1 = in1 ? aoff + k1 * 64 : kSZeroOff;
                const int32_t ao2 = in2 ? aoff + (k1 + 4) * 64 : kSZeroOff;
                const bf16x8 af = join(tr_read(lx + ao1 + colb), tr_read(lx + ao2 + colb));
                v4i16 rb[kSBlocks][2];
#pragma unroll
                for (int e = 0; e < kSBlocks; ++e) {
                    rb[e][0] = tr_read(lx + xo1 + colb + 64 * e);
                    rb[e][1] = tr_read(lx + xo2 + colb + 64 * e);
                }
#pragma unroll
                for (int e = 0; e < kSBlocks; ++e)
                    acc[e] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, join(rb[e][0], rb[e][1]), acc[e], 0, 0, 0);
                if (hi >= ql) break;
                lo = hi;
            }
        };

        // Window j is multiplied from slot j % kSAhead, which is then
        // refilled with window j + kSAhead.  Whole periods run with
        // compile-time slot indices, the tail after.
        int32_t j0 = 0;
        for (; j0 + kSAhead <= it.nwin; j0 += kSAhead) {
#pragma unroll
            for (int u = 0; u < kSAhead; ++u) {
                process(u, j0 + u);
                load(it, u, j0 + u + kSAhead);
            }
        }
#pragma unroll
        for (int u = 0; u < kSAhead - 1; ++u)
            if (j0 + u < it.nwin) process(u, j0 + u);

        // Fused epilogue: the item's 32 scales (lanes 0-31) and biases (lanes
        // 32-63) go to the wave's LDS slot here, where this item's loads have
        // all been consumed, so the wait covers these loads alone; at the
        // store (behind the next item's first loads) a global load would wait
        // for those too.
        if constexpr (kEp) {
            if (it.g < a.G) {
                const int32_t o = it.g * 32 + (lane & 31);
                const bool in = o < a.n;
                sEp[w * 64 + lane] = lane < 32 ? (in && a.ep_scale ? a.ep_scale[o] : 1.f)
                                               : (in && a.ep_bias ? a.ep_bias[o] : 0.f);
            }
        }

        // The next item's first windows, then this item's stores.
        const Item nx = item_at(k + 1);
        if (k + 1 < nloc) {
#pragma unroll
            for (int u = 0; u < kSAhead; ++u) load(nx, u, u);
        }

        // Store: MFMA (row, col) of block e -> output channel g*32 + row, tile column 32e + col.
        if (it.g < a.G) {
#pragma unroll
            for (int e = 0; e < kSBlocks; ++e) {
                const int32_t n = 32 * e + (lane & 31);
                const int32_t id = it.tile * kSGran + (n >> 3);
                const int32_t b = id / gpi;
                const int32_t hw = 8 * (id - b * gpi) + (n & 7);
                if (id >= ngran || hw >= a.HWo) continue;
                TY* yb = y + int64_t(b) * a.y_img + hw;
                EpRows<32, kEp> ep;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    if (kEp && r % 4 == 0) ep.load_staged_run(sEp + w * 64, sEp + w * 64 + 32, 0, lane, r / 4);
                    const int32_t o = it.g * 32 + PwMfma<32>::row(lane, r);
                    // Plain stores: with 2-byte elements a half-wave writes
                    // 64 bytes of a row, and non-temporal partial-line writes
                    // measured slower here (366 -> 302 us at 2048 -> 2048,
                    // 14x14, batch 256).
                    if (o < a.n) yb[int64_t(o) * a.y_c] = from_f32<TY>(ep.apply(a, r, acc[e][r]));
                }
            }
        }
        // The item's remaining epochs: one barrier per chunk in all.
        while (epoch < nch) {
            __syncthreads();
            ++epoch;
        }
        it = nx;
    }
}

template <typename TY, bool E>
onexn_status launch_typed(ConvArgs a, hipStream_t s) {
    const int64_t batch = a.npix / a.HWo;
    const int64_t ngran = batch * ((a.HWo + 7) / 8);
    const int64_t ntiles = (ngran + kSGran - 1) / kSGran;
    const int64_t nitems = ntiles * ((a.G + kSCompute - 1) / kSCompute);
    int64_t wgs = std::min<int64_t>(nitems, device_cu_count());
    if (tuning(kTunePwbWgs) >= 1) wgs = std::min<int64_t>(tuning(kTunePwbWgs), nitems);
    return launch_grid(pw_bf16s<TY, E>, a, wgs, s, kSThreads);
}

}  // namespace

bool pw_bf16s_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_BF16 || layout != ONEXN_NCHW || a.N != 32) return false;
    if (a.kh != 1 || a.kw != 1 || a.sh != 1 || a.sw != 1 || a.ph != 0 || a.pw != 0) return false;
    if (a.HWo % 4 != 0 || (reinterpret_cast<uintptr_t>(a.x) & 15) != 0) return false;
    const int64_t batch = a.npix / a.HWo;
    if (batch * a.x_img * 2 >= (int64_t(1) << 31)) return false;   // 32-bit buffer offsets
    // Weight offsets of the windows loaded past a col-group's end.
    if (int64_t(a.t) * 64 + (kSAhead + 1) * 1024 >= (int64_t(1) << 31)) return false;
    (void)ydt;
    return true;
}

onexn_status launch_pw_bf16s(ConvArgs a, onexn_dtype ydt, hipStream_t s) {
    return with_epilogue(a, [&](auto ep) {
        constexpr bool E = decltype(ep)::value;
        if (ydt == ONEXN_BF16) return launch_typed<uint16_t, E>(a, s);
        return launch_typed<float, E>(a, s);
    });
}

}  // namespace onexn
