// 3x3 and 7x7 (any stride and padding) 1xN-pruned convolution, fp32,
// N in {16, 32}, NCHW,
// with the kept channels' input patches and weights staged in LDS.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the contraction
//     Y_g[N][pixels] = A_g[N][kept_g * k * k] * B_g[kept_g * k * k][pixels]
// where B_g's row (z, q, r) is input channel I[z] shifted by kernel tap (q, r)
// under each output pixel (implicit im2col of the kept channels only) and
// A_g[o][(z, q, r)] = D[z][o][q][r].
//
// Work split.  A workgroup computes one (tile, col-group) output block: a tile
// is R whole output rows (consecutive in batch-major row order, so a tile may
// span images), at most 256 pixels.  Its four waves split the tile's pixels
// (NBW MFMA column blocks each) and all of them walk the col-group's kept
// blocks in chunks of CC blocks.
//
// Staging.  For a chunk, the workgroup copies into LDS (buffer loads straight
// into LDS, double-buffered, one chunk ahead):
//   * the input rows the tile reads, for each of the chunk's CC channels: the
//     tile's images' input rows from the first output row's window to the last
//     one's, stacked ("virtual rows"), each Wp = (Wo - 1) * stride + k wide,
//     zero where the window leaves the image (padding) -- the zeros come from
//     out-of-range buffer reads;
//   * the chunk's CC weight blocks D[z][N][k][k], which are contiguous.
// Every output pixel's patch at tap (q, r) of staged channel j then sits at
// LDS float offset j * CP + pofs(pixel) + q * Wp + r.
//
// Matrix cores.  N = 32: v_mfma_f32_32x32x2f32; a step is (channel pair, tap):
// lanes 0-31 take the pair's first channel, lanes 32-63 its second.  N = 16:
// v_mfma_f32_16x16x4f32; a step is (channel quad, tap), lane group l/16 taking
// channel l/16 of the quad.  So a lane's A and B addresses differ from step to
// step by wave-uniform amounts only.  Entries past the col-group's end and
// channels outside [0, m) stage zero weights and zero inputs.

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kKxWaves = 4;
constexpr int kKxThreads = 64 * kKxWaves;
constexpr int kKxMaxRem = 9;   // staged positions per lane per channel: (virtual rows x Wp) <= 9 * 256
constexpr int kKxSplitMaxG = 256;   // col-groups of a layer the balanced split takes

template <int N, int K, int NBW, int CC, bool SPLIT, bool kEp>
__global__ void __launch_bounds__(kKxThreads) kxk_f32(ConvArgs a) {
    typedef PwMfma<N> M;
    typedef typename M::acc_t acc_t;
    constexpr int KS = M::KS, COLS = M::COLS, KK = K * K;
    constexpr int DBUF = CC * N * KK;   // floats of one chunk's weights
    static_assert(CC % KS == 0 && DBUF % 64 == 0, "chunk shape");
    extern __shared__ __attribute__((aligned(16))) float smem[];
    __shared__ int32_t sC[SPLIT ? kKxSplitMaxG + 1 : 1];   // chunks of the col-groups before g
    // Fused epilogue (unsplit kernel: one col-group per workgroup): scale and
    // bias of its N channels, staged at the start, read run by run at the
    // store.
    __shared__ __attribute__((aligned(16))) float sEp[kEp ? 2 * N : 4];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t R = a.kx_rows, Wp = a.kx_wp, VRWp = a.kx_vrwp, CP = a.kx_cp;
    const int32_t XBUF = CC * CP;
    float* const xs = smem;              // [2][CC][CP]
    float* const ds = smem + 2 * XBUF;   // [2][CC][N][KK]
    int32_t* const sI = reinterpret_cast<int32_t*>(ds + 2 * DBUF);   // [3][64]
    const int32_t batch = a.npix / a.HWo;

    // Chunks [ca, cb) of the (tile, col-group g) output block; a part of a
    // block (split) adds its partial sums to y, which holds zeros before.
    auto run = [&](const int32_t tile, const int32_t g, const int32_t ca, const int32_t cb, const bool split)
                   __attribute__((always_inline)) {
    int32_t zb, ze;
    group_range(a, g, zb, ze);
    const int32_t kept = ze - zb;

    // Output rows of the tile, in batch-major order: [rr0, rr1).
    const int32_t rr0 = tile * R;
    const int32_t rr1 = min(rr0 + R, batch * a.Ho);
    const int32_t b0 = rr0 / a.Ho, blast = (rr1 - 1) / a.Ho;
    const int32_t oh_first = rr0 - b0 * a.Ho;
    // Staged input rows of image b (b0 <= b <= blast): its output rows
    // [lo, hi] read input rows lo * sh - ph .. hi * sh - ph + kh - 1.
    auto seg_lo = [&](int32_t b) { return b == b0 ? oh_first : 0; };
    auto seg_rows = [&](int32_t b) {
        const int32_t hi = b == blast ? rr1 - 1 - b * a.Ho : a.Ho - 1;
        return (hi - seg_lo(b)) * a.sh + K;
    };

    // Byte offset in x of each staged position this lane copies (channel 0),
    // or kBufferOutOfRange where the window leaves the image.
    uint32_t spk[kKxMaxRem];
#pragma unroll
    for (int k = 0; k < kKxMaxRem; ++k) {
        const int32_t rem = wave * 64 + lane + k * kKxThreads;
        uint32_t sp = kBufferOutOfRange;
        if (rem < VRWp) {
            int32_t v = rem / Wp;
            const int32_t col = rem - v * Wp;
            int32_t b = b0;
            for (; b <= blast; ++b) {
                const int32_t nv = seg_rows(b);
                if (v < nv) break;
                v -= nv;
            }
            const int32_t ih = seg_lo(b) * a.sh - a.ph + v, iw = col - a.pw;
            if (b <= blast && ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
                sp = uint32_t((int64_t(b) * a.x_img + int64_t(ih) * a.W + iw) * 4);
        }
        spk[k] = sp;
    }

    // This lane's output pixel in each of its column blocks: LDS offset of its
    // patch within a staged channel, and its y offset (-1: not a pixel).
    int32_t pofs[NBW];
    int64_t ybase[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb) {
        const int32_t i = (wave * NBW + nb) * COLS + lane % COLS;
        const int32_t r = i / a.Wo, ow = i - r * a.Wo;
        const int32_t rr = rr0 + r;
        pofs[nb] = 0;
        ybase[nb] = -1;
        if (r < R && rr < rr1) {
            const int32_t b = rr / a.Ho, oh = rr - b * a.Ho;
            int32_t vb = 0;
            for (int32_t bb = b0; bb < b; ++bb) vb += seg_rows(bb);
            pofs[nb] = (vb + (oh - seg_lo(b)) * a.sh) * Wp + ow * a.sw;
            ybase[nb] = int64_t(b) * a.y_img + int64_t(oh) * a.Wo + ow;
        }
    }

    const v4i32 rX = buffer_rsrc(a.x, int32_t(int64_t(batch) * a.x_img * 4));
    const v4i32 rD = buffer_rsrc(a.D, int32_t(int64_t(ze) * N * KK * 4));
    const v4i32 rI = buffer_rsrc(a.I, int32_t(int64_t(ze) * 4));
    const int32_t nchunks = (kept + CC - 1) / CC;

    // The channel indices of chunk c sit in LDS ring slot c % 3 (64 entries,
    // copied by wave 0 two chunks ahead, like the other operands).
    auto copy_channels = [&](int32_t c) {
        if (wave == 0)
            copy4_to_lds(rI, (const lds_char*)(sI + (c % 3) * 64), (zb + c * CC + lane) * 4, 0);
    };
    // Stages chunk c: its weight blocks and its channels' input rows.  The
    // copies are issued straight-line per staged position block k (one
    // uniform test per k, selects rather than branches for the channels), so
    // a chunk's staging costs few instructions besides the copies themselves.
    auto stage = [&](int32_t c, int buf) {
        const lds_char* dd = (const lds_char*)(ds + buf * DBUF);
        const int32_t d0 = (zb + c * CC) * (N * KK * 4);
        // (DBUF is a multiple of 64 floats: every copy lies inside the buffer.)
        for (int32_t e0 = wave * 64; e0 < DBUF; e0 += kKxThreads)
            copy4_to_lds(rD, dd + e0 * 4, d0 + (e0 + lane) * 4, 0);
        // Lane j < CC: block j's channel, or -1 past the col-group's end.
        const int32_t chv = (lane < CC && zb + c * CC + lane < ze) ? sI[(c % 3) * 64 + lane] : -1;
        const lds_char* xd = (const lds_char*)(xs + buf * XBUF);
        // An invalid position or channel carries kBufferOutOfRange: the sum of
        // two offsets below 2^31 stays below 2^32 and an out-of-range one
        // keeps the sum at or above kBufferOutOfRange, past every buffer.
        uint32_t choff[CC];
#pragma unroll
        for (int j = 0; j < CC; ++j) {
            const int32_t ch = __builtin_amdgcn_readlane(chv, j);
            choff[j] = uint32_t(ch) < uint32_t(a.m) ? uint32_t(ch) * uint32_t(a.x_c) * 4u : kBufferOutOfRange;
        }
#pragma unroll
        for (int k = 0; k < kKxMaxRem; ++k) {
            const int32_t rem0 = wave * 64 + k * kKxThreads;
            if (rem0 >= VRWp) break;
#pragma unroll
            for (int j = 0; j < CC; ++j)
                copy4_to_lds(rX, xd + (j * CP + rem0) * 4, int32_t(spk[k] + choff[j]), 0);
        }
    };

    acc_t acc[NBW];
#pragma unroll
    for (int nb = 0; nb < NBW; ++nb)
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) acc[nb][r] = 0.f;

    // Lane roles: row / pixel column o = lane % COLS, staged channel kq of a
    // step.  A chunk is always computed whole: its slots past the col-group's
    // end hold zero weights and zero inputs.
    const int o = lane % COLS, kq = lane / COLS;
    auto compute = [&](int buf) {
        const float* xb = xs + buf * XBUF + kq * CP;
        const float* db = ds + buf * DBUF + (kq * N + o) * KK;
        constexpr int S = (CC / KS) * KK;   // MFMA steps of a chunk: (slot group, tap)
        auto read = [&](int st, float& av, float (&bv)[NBW]) {
            const int jg = st / KK, tap = st % KK;
            const int q = tap / K, r = tap % K;
            av = db[jg * KS * N * KK + tap];
            const float* xj = xb + jg * KS * CP + q * Wp + r;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) bv[nb] = xj[pofs[nb]];
        };
        // Software pipeline: step st + PD's operands are read from LDS while
        // step st's MFMAs run; the scheduling groups put one MFMA between
        // each pair of reads.
        constexpr int PD = 2;
        float av[PD + 1], bv[PD + 1][NBW];
#pragma unroll
        for (int st = 0; st < PD && st < S; ++st) read(st, av[st], bv[st]);
#pragma unroll
        for (int st = 0; st < S; ++st) {
            const int cur = st % (PD + 1);
            if (st + PD < S) read(st + PD, av[(st + PD) % (PD + 1)], bv[(st + PD) % (PD + 1)]);
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) acc[nb] = M::step(av[cur], bv[cur][nb], acc[nb]);
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) {
                __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);   // an LDS read,
                __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);   // an MFMA
            }
            __builtin_amdgcn_sched_group_barrier(0x100, 1, 0);
            __builtin_amdgcn_sched_group_barrier(0x002, 2, 0);       // address arithmetic
        }
    };

    // A chunk whose only kept block is its first slot (the last chunk when
    // kept % CC == 1, e.g. the third input channel of a 3-channel stem) at
    // N = 32: the two lane groups take two taps of that slot, tap 2 st + kq,
    // instead of one tap of two slots, half of them empty; a tap past the
    // kernel reads the second slot's zero row with a zero weight.  Half the
    // MFMA steps for such a chunk.
    auto compute_one = [&](int buf) {
        constexpr int S1 = (KK + 1) / 2;
        const float* xb = xs + buf * XBUF;
        const float* db = ds + buf * DBUF + o * KK;
        auto read = [&](int st, float& av, float (&bv)[NBW]) {
            const int t0 = 2 * st, t1 = 2 * st + 1;
            const int q0 = t0 / K, r0 = t0 % K, q1 = t1 / K, r1 = t1 % K;
            const bool ok1 = t1 < KK;
            const int32_t xo = kq == 0 ? q0 * Wp + r0 : (ok1 ? q1 * Wp + r1 : CP);
            const float w0 = db[t0], w1 = ok1 ? db[ok1 ? t1 : t0] : 0.f;
            av = kq == 0 ? w0 : w1;
            const float* xj = xb + xo;
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) bv[nb] = xj[pofs[nb]];
        };
        constexpr int PD = 2;
        float av[PD + 1], bv[PD + 1][NBW];
#pragma unroll
        for (int st = 0; st < PD && st < S1; ++st) read(st, av[st], bv[st]);
#pragma unroll
        for (int st = 0; st < S1; ++st) {
            const int cur = st % (PD + 1);
            if (st + PD < S1) read(st + PD, av[(st + PD) % (PD + 1)], bv[(st + PD) % (PD + 1)]);
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb) acc[nb] = M::step(av[cur], bv[cur][nb], acc[nb]);
        }
    };
    const bool one_last = N == 32 && CC == 2 && kept % CC == 1;

    // Chunk c + 1 is staged while chunk c is multiplied; one barrier per chunk
    // hands the buffers over.
    if (cb > ca) {
        copy_channels(ca);
        copy_channels(ca + 1);
        vm_wait<0>();
        __syncthreads();
        stage(ca, ca & 1);
        copy_channels(ca + 2);
    }
    vm_wait<0>();
    __syncthreads();
    for (int32_t c = ca; c < cb; ++c) {
        if (c + 1 < cb) {
            stage(c + 1, (c + 1) & 1);
            copy_channels(c + 3);
        }
        if (one_last && c == nchunks - 1) compute_one(c & 1);
        else compute(c & 1);
        vm_wait<0>();
        __syncthreads();
    }

    // Store: MFMA (row, col) of column block nb -> output channel g*N + row.
    float* __restrict__ y = static_cast<float*>(a.y);
    if constexpr (kEp && !SPLIT) {
        // Runs of four rows, each fenced off from the next: computed all at
        // once, the epilogue's parameters and results would raise the
        // register count far above what the main loop needs.
        EpRows<N, true> ep;
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) {
            if (r % 4 == 0) {
                __builtin_amdgcn_sched_barrier(0);
                ep.load_staged_run(sEp, sEp + N, 0, lane, r / 4);
            }
            const int32_t oc = g * N + M::row(lane, r);
#pragma unroll
            for (int nb = 0; nb < NBW; ++nb)
                if (ybase[nb] >= 0 && oc < a.n)
                    store_out(&y[ybase[nb] + int64_t(oc) * a.y_c], ep.apply(a, r, acc[nb][r]));
        }
    } else {
        static_assert(!kEp, "the split kernel adds raw sums: no epilogue");
#pragma unroll
        for (int nb = 0; nb < NBW; ++nb) {
            if (ybase[nb] < 0) continue;
#pragma unroll
            for (int r = 0; r < M::ACC; ++r) {
                const int32_t oc = g * N + M::row(lane, r);
                if (oc >= a.n) continue;
                if (SPLIT && split) unsafeAtomicAdd(&y[ybase[nb] + int64_t(oc) * a.y_c], acc[nb][r]);
                else store_out(&y[ybase[nb] + int64_t(oc) * a.y_c], acc[nb][r]);
            }
        }
    }
    };

    if constexpr (!SPLIT) {
        const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
        const int32_t g = L % a.G, tile = L / a.G;
        int32_t zb, ze;
        group_range(a, g, zb, ze);
        if constexpr (kEp) {
            // (visible at the store: the main loop has barriers)
            const int tid = threadIdx.x;
            if (tid < N) {
                const int32_t o = g * N + tid;
                sEp[tid] = o < a.n && a.ep_scale ? a.ep_scale[o] : 1.f;
                sEp[N + tid] = o < a.n && a.ep_bias ? a.ep_bias[o] : 0.f;
            }
        }
        run(tile, g, 0, (ze - zb + CC - 1) / CC, false);
    } else {
        // Balanced split: the (tile, col-group, chunk) sequence, tile-major,
        // is cut into one contiguous range of equal length per workgroup, so
        // every compute unit gets the same work however the blocks divide
        // among them.  sC[g]: chunks of the col-groups before g.
        if (wave == 0) {
            int32_t carry = 0;
            for (int32_t g0 = 0; g0 < a.G; g0 += 64) {
                const int32_t gg = g0 + lane;
                int32_t v = 0;
                if (gg < a.G) {
                    int32_t zb, ze;
                    group_range(a, gg, zb, ze);
                    v = (ze - zb + CC - 1) / CC;
                }
#pragma unroll
                for (int d = 1; d < 64; d <<= 1) {
                    const int32_t u = __shfl_up(v, d);
                    if (lane >= d) v += u;
                }
                if (gg < a.G) sC[gg + 1] = carry + v;
                carry += __shfl(v, 63);
            }
            if (lane == 0) sC[0] = 0;
        }
        __syncthreads();
        const int32_t G = a.G;
        const int32_t tcost = __builtin_amdgcn_readfirstlane(sC[G]);   // chunks of one tile
        const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
        const int64_t total = int64_t(a.kx_tiles) * tcost;
        // Col-group of position r (< tcost) of a tile: the first g whose
        // chunks extend past r.
        auto group_at = [&](int32_t r) {
            int32_t lo = 1, hi = G;   // first j in [1, G] with sC[j] > r
            while (lo < hi) {
                const int32_t mid = (lo + hi) >> 1;
                if (sC[mid] > r) hi = mid;
                else lo = mid + 1;
            }
            return __builtin_amdgcn_readfirstlane(lo - 1);
        };
        // (A block cut by range ends is computed in parts that add into the
        // zeroed output.  Two parts commute exactly; a block longer than a
        // range can have three or more, which add in arrival order, so the
        // last bits of its outputs may differ from run to run.  Moving every
        // second cut of a block to the block's end bounds the parts at two,
        // but measured 10-40 % slower on the ResNet-50 14x14 and 7x7 layers.)
        int64_t c = total * L / a.total;
        const int64_t c1 = total * (L + 1) / a.total;
        while (c < c1) {
            const int32_t tile = int32_t(c / tcost);
            const int32_t r = int32_t(c - int64_t(tile) * tcost);
            const int32_t g = group_at(r);
            const int32_t base = __builtin_amdgcn_readfirstlane(sC[g]);
            const int32_t nch = __builtin_amdgcn_readfirstlane(sC[g + 1]) - base;
            const int32_t ca = r - base;
            const int32_t cb = int32_t(min<int64_t>(nch, ca + (c1 - c)));
            run(tile, g, ca, cb, ca > 0 || cb < nch);
            c += cb - ca;
        }
    }
}

struct KxShape {
    int32_t rows = 0, wp = 0, vrwp = 0, cp = 0;
    int tp = 0;   // pixel capacity of the tile (4 waves x NBW x MFMA columns)
};

// Largest number of staged input rows any tile of `rows` output rows needs.
// A tile's row structure depends only on where it starts within an image, so
// the first min(tiles, Ho) tiles cover every case.
int32_t max_virtual_rows(const ConvArgs& a, int32_t rows) {
    const int64_t nrows = int64_t(a.npix / a.HWo) * a.Ho;
    const int64_t ntiles = (nrows + rows - 1) / rows;
    int32_t best = 0;
    for (int64_t t = 0; t < std::min<int64_t>(ntiles, a.Ho); ++t) {
        const int64_t r0 = t * rows, r1 = std::min<int64_t>(r0 + rows, nrows);
        int32_t v = 0;
        for (int64_t b = r0 / a.Ho; b <= (r1 - 1) / a.Ho; ++b) {
            const int64_t lo = b == r0 / a.Ho ? r0 - b * a.Ho : 0;
            const int64_t hi = b == (r1 - 1) / a.Ho ? r1 - 1 - b * a.Ho : a.Ho - 1;
            v += int32_t((hi - lo) * a.sh + a.kh);
        }
        best = std::max(best, v);
    }
    return best;
}

template <int N>
constexpr int kx_cols() { return N == 32 ? 32 : 16; }

// Dynamic LDS of a launch: two chunk buffers of inputs and weights, and the
// ring of channel indices.
int64_t kx_lds_bytes(int cc, int cp, int N, int KK) {
    return 2 * 4 * (int64_t(cc) * cp + int64_t(cc) * N * KK) + 3 * 64 * 4;
}

// Tile and LDS shape for a pixel capacity tp, or rows == 0 when it does not fit.
KxShape kx_shape(const ConvArgs& a, int tp, int cc) {
    KxShape s;
    s.tp = tp;
    if (a.Wo > tp) return s;
    s.rows = tp / a.Wo;
    s.wp = (a.Wo - 1) * a.sw + a.kw;
    s.vrwp = max_virtual_rows(a, s.rows) * s.wp;
    const int cols = a.N == 32 ? 32 : 16;
    s.cp = (s.vrwp + 63) / 64 * 64 + cols;   // whole 64-float copies; halves of a step land on other banks
    const int64_t lds = kx_lds_bytes(cc, s.cp, a.N, a.KK);
    if (s.vrwp > kKxMaxRem * kKxThreads || lds > 64 * 1024) s.rows = 0;
    return s;
}

int kx_cc(int N, int k) { return k == 7 ? (N == 32 ? 2 : 4) : 4; }

// Zeros n floats at p (the output of a balanced-split launch, whose parts of
// an output block add into it).
__global__ void __launch_bounds__(256) kx_zero(float* __restrict__ p, int64_t n) {
    const int64_t stride = int64_t(gridDim.x) * 256 * 4;
    for (int64_t i = (int64_t(blockIdx.x) * 256 + threadIdx.x) * 4; i < n; i += stride) {
        if (i + 4 <= n) store_out(reinterpret_cast<f32x4*>(p + i), f32x4{0.f, 0.f, 0.f, 0.f});
        else
            for (int64_t j = i; j < n; ++j) store_out(p + j, 0.f);
    }
}

// The fused epilogue over a finished NCHW output (n floats at p), for a
// split launch: its parts add raw sums into y, so the epilogue can only
// follow them.  Elements are numbered [image][channel][pixel]; n < 2^31.
__global__ void __launch_bounds__(256) kx_epilogue(ConvArgs a, float* __restrict__ p, int32_t n) {
    const int32_t stride = int32_t(gridDim.x) * 256 * 4;
    for (int32_t i = (int32_t(blockIdx.x) * 256 + threadIdx.x) * 4; i < n; i += stride) {
        if (i + 4 <= n) {
            f32x4 v = *reinterpret_cast<const f32x4*>(p + i);
#pragma unroll
            for (int j = 0; j < 4; ++j) v[j] = epilogue(a, (i + j) / a.HWo % a.n, v[j]);
            store_out(reinterpret_cast<f32x4*>(p + i), v);
        } else {
            for (int32_t j = i; j < n; ++j) p[j] = epilogue(a, j / a.HWo % a.n, p[j]);
        }
    }
}

// Largest output (bytes) for which a layer with an epilogue keeps the
// balanced split and runs kx_epilogue after it, rather than taking the
// unsplit kernel with the epilogue in its stores: the extra pass reads and
// writes y once more, which the split's gain outweighs on small outputs only.
constexpr int64_t kKxEpPassMax = int64_t(16) << 20;

// Workgroups per compute unit of the balanced split (0: one workgroup per
// output block).  All blocks of a launch are resident at once, so a launch
// takes as long as its busiest compute unit: with few blocks per unit (800
// blocks on 256 units: 4 on some, 3.125 on average) that loses up to a
// quarter.  Measured on the ResNet-50 3x3 layers at batch 64, the split with
// four workgroups per unit takes 10-21 % off the 128-pixel-tile launches
// (fewer than 8 blocks per unit) and slows the 256-pixel ones (more
// registers: 4 waves per SIMD instead of 7), whose blocks are longer.
int kx_split_choice(const KxShape& s, int64_t units) {
    if (tuning(kTuneKxkSplit) >= 0) return tuning(kTuneKxkSplit);
    return s.tp == 128 && units < 8 * int64_t(device_cu_count()) ? 4 : 0;
}

template <int N, int K, int NBW>
onexn_status launch_nbw(ConvArgs a, const KxShape& s, hipStream_t stream) {
    constexpr int CC = (K == 7) ? (N == 32 ? 2 : 4) : 4;
    a.kx_rows = s.rows;
    a.kx_wp = s.wp;
    a.kx_vrwp = s.vrwp;
    a.kx_cp = s.cp;
    const int64_t nrows = int64_t(a.npix / a.HWo) * a.Ho;
    const int64_t tiles = (nrows + s.rows - 1) / s.rows;
    const int64_t total = tiles * a.G;
    if (total < 1 || total > INT32_MAX / kKxThreads)
        return fail(ONEXN_ERR_UNSUPPORTED, "conv2d_fwd: grid of %lld workgroups is out of range",
                    (long long)total);
    a.total = int32_t(total);
    a.kx_tiles = int32_t(tiles);
    const size_t lds = size_t(kx_lds_bytes(CC, s.cp, N, K * K));
    // (NCHW output, contiguous and 16-byte aligned for the zero fill.)
    // (The parts of a split block add raw sums into y, so with a fused
    // epilogue a small output takes the split and a pass of kx_epilogue, a
    // larger one the unsplit kernel.)
    const int64_t ny = int64_t(a.npix / a.HWo) * a.y_img;
    const bool ep = has_epilogue(a);
    const bool ep_ok = !ep || (ny * 4 <= kKxEpPassMax && a.y_img == int64_t(a.n) * a.HWo);
    const bool can_split = ep_ok && a.G <= kKxSplitMaxG && a.y_c == a.HWo &&
                           reinterpret_cast<uintptr_t>(a.y) % 16 == 0;
    const int split = can_split ? kx_split_choice(s, total) : 0;
    if (split > 0) {
        const int64_t zb = std::min<int64_t>((ny + 1023) / 1024, 4 * int64_t(device_cu_count()));
        hipLaunchKernelGGL(kx_zero, dim3(uint32_t(zb)), dim3(256), 0, stream, static_cast<float*>(a.y), ny);
        const hipError_t zerr = hipGetLastError();
        if (zerr != hipSuccess)
            return fail(ONEXN_ERR_HIP, "conv2d_fwd: launch failed: %s", hipGetErrorString(zerr));
        // (Ranges shorter than an eighth of a block only add partial sums.)
        a.total = int32_t(std::min<int64_t>(8 * total, int64_t(split) * device_cu_count()));
        hipLaunchKernelGGL((kxk_f32<N, K, NBW, CC, true, false>), dim3(uint32_t(a.total)), dim3(kKxThreads), lds, stream, a);
        if (ep) {
            const hipError_t serr = hipGetLastError();
            if (serr != hipSuccess)
                return fail(ONEXN_ERR_HIP, "conv2d_fwd: launch failed: %s", hipGetErrorString(serr));
            hipLaunchKernelGGL(kx_epilogue, dim3(uint32_t(zb)), dim3(256), 0, stream, a, static_cast<float*>(a.y),
                               int32_t(ny));
        }
    } else {
        if (has_epilogue(a))
            hipLaunchKernelGGL((kxk_f32<N, K, NBW, CC, false, true>), dim3(uint32_t(total)), dim3(kKxThreads), lds, stream, a);
        else
            hipLaunchKernelGGL((kxk_f32<N, K, NBW, CC, false, false>), dim3(uint32_t(total)), dim3(kKxThreads), lds, stream, a);
    }
    const hipError_t err = hipGetLastError();
    if (err != hipSuccess)
        return fail(ONEXN_ERR_HIP, "conv2d_fwd: launch failed: %s", hipGetErrorString(err));
    return ONEXN_OK;
}

// Picks the tile size: 256 pixels when that still gives the GPU a few
// workgroups per compute unit, else 128.
template <int N, int K>
onexn_status launch_k(ConvArgs a, hipStream_t stream) {
    constexpr int COLS = kx_cols<N>();
    constexpr int NB_BIG = 256 / (4 * COLS), NB_SMALL = 128 / (4 * COLS);
    const int cc = kx_cc(N, K);
    const KxShape big = kx_shape(a, 256, cc), small = kx_shape(a, 128, cc);
    const int64_t nrows = int64_t(a.npix / a.HWo) * a.Ho;
    const int64_t want = 3 * int64_t(device_cu_count());
    bool big_ok = big.rows > 0 && (nrows + big.rows - 1) / big.rows * a.G >= want;
    const int32_t tp = tuning(kTuneKxkTp);
    if (tp == 256 && big.rows > 0) big_ok = true;
    if (tp == 128 && small.rows > 0) big_ok = false;
    if (big_ok || (big.rows > 0 && small.rows == 0)) return launch_nbw<N, K, NB_BIG>(a, big, stream);
    return launch_nbw<N, K, NB_SMALL>(a, small, stream);
}

}  // namespace

bool kxk_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_F32 || ydt != ONEXN_F32 || layout != ONEXN_NCHW) return false;
    if (a.N != 16 && a.N != 32) return false;
    // 1x1 layers stay on the pointwise and generic kernels, which measured
    // faster for them (a staged 1x1 chunk carries too little work).
    if (a.kh != a.kw || (a.kh != 3 && a.kh != 7)) return false;
    const int64_t batch = a.npix / a.HWo;
    if (batch * a.x_img * 4 >= (int64_t(1) << 31)) return false;        // 32-bit buffer offsets
    if (int64_t(a.t) * a.N * a.KK * 4 >= (int64_t(1) << 31)) return false;
    const int cc = kx_cc(a.N, a.kh);
    return kx_shape(a, 256, cc).rows > 0 || kx_shape(a, 128, cc).rows > 0;
}

onexn_status launch_kxk(ConvArgs a, hipStream_t stream) {
    if (a.N == 32) {
        if (a.kh == 3) return launch_k<32, 3>(a, stream);
        return launch_k<32, 7>(a, stream);
    }
    if (a.kh == 3) return launch_k<16, 3>(a, stream);
    return launch_k<16, 7>(a, stream);
}

}  // namespace onexn
