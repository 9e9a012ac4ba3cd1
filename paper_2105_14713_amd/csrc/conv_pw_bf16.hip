// Pointwise (1x1, stride 1, no padding, NCHW) 1xN-pruned convolution with
// bf16 inputs and weights, fp32 accumulation, N = 32, bf16 or fp32 output.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the contraction
//     Y_g[32][pixels] = D_g^T[32][kept_g] * X[I_g][pixels]:
// its kept blocks select rows of the input matrix X[channel][pixel].
//
// Matrix cores.  v_mfma_f32_32x32x16_bf16 multiplies a 32x16 A fragment (the
// 32 weights of 16 kept blocks) by a 16x32 B fragment (16 gathered input rows
// at 32 pixels); each lane holds 8 consecutive contraction entries of one
// output row (A) or one pixel (B).  For a 1xN layer those 8 entries are 8
// kept channels, i.e. 8 different rows of X, so B cannot be read with plain
// vector loads.  gfx950's ds_read_b64_tr_b16 does exactly this transposition:
// each lane names the row it wants (any row) and receives the 16-bit
// elements of four lanes' rows.  The same instruction transposes the weight
// panel D (stored with the 32 outputs of a block contiguous) into the A
// fragment.
//
// Work split.  A work item is (pixel tile of 128 columns, set of 8
// col-groups); each of the workgroup's 8 compute waves computes one col-group
// over the tile (32 x 128 fp32 accumulators).  A pixel tile is 16 granules of
// 8 pixels; a granule lies in one image (the last granule of an image may be
// partial), so that each granule of a channel is one 16-byte copy.
//
// Input staging.  Three loader waves copy X into LDS in chunks of 32
// channels x 128 columns with buffer loads straight into LDS (16 bytes per
// lane, four 256-byte rows per copy), into a ring of 8 chunk buffers, as far
// ahead as the ring allows.  Each group of 4 rows is followed by 64 bytes of
// padding, so the 8 rows one transposed read touches spread over the LDS
// banks while a row's four 64-byte column blocks stay at fixed offsets
// (immediates of the reads).
// LDS flags, not barriers, order the two sides: each buffer's flag names the
// chunk that has landed in it, each compute wave's `need` is the first chunk
// it may still read; a buffer is refilled once every wave's `need` has passed
// the chunk in it.
//
// Kept blocks.  A compute wave walks its col-group's kept blocks in steps of
// up to 16 (one MFMA k-step): a step takes the next 16 blocks unless their
// channels span more than 4 chunks, in which case it stops short.  The blocks' weights (16 x 64 bytes) and channel indices are copied
// into a per-wave LDS ring in windows of 16 blocks, up to 5 windows ahead.
// Ring sizes are powers of two so that every slot index is a mask.
// Steps are software-pipelined: while step j's four MFMAs run, the wave reads
// step j+1's A and B fragments and step j+2's channel indices.  Entries past
// a step's end, and channels outside [0, m), read a zero row for both A and
// B, so they add exactly nothing.

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kQWaves = 8;                       // compute waves, one col-group each
constexpr int kQLoaders = 3;                     // loader waves
constexpr int kQThreads = 64 * (kQWaves + kQLoaders);
constexpr int kQKcShift = 5;
constexpr int kQKc = 1 << kQKcShift;             // input channels per X chunk
constexpr int kQRing = 8;                        // X chunk buffers (a power of two)
constexpr int kQSpan = 4;                        // chunks one k-step may touch
constexpr int kQInFlight = 2;                    // chunks in flight per loader wave
constexpr int kQGran = 16;                       // 8-pixel granules per tile
constexpr int kQCols = 8 * kQGran;               // pixel columns per tile
constexpr int kQBlocks = kQCols / 32;            // MFMA column blocks
constexpr int kQRowB = kQCols * 2;               // bytes of one X row (one channel of the tile)
constexpr int kQQuadB = 4 * kQRowB + 64;         // LDS bytes per 4 rows: quads of rows shift by 64 bytes of banks
constexpr int kQBufB = (kQKc / 4) * kQQuadB;     // bytes per chunk buffer
constexpr int kQCopies = kQKc / 4;               // 1 KB copies per chunk (4 rows each)
constexpr int kQZeroOff = kQRing * kQBufB;       // a row of zeros after the ring
constexpr int kQWin = 16;                        // kept blocks per window (one k-step)
constexpr int kQWins = 8;                        // windows in a wave's ring (a power of two)
constexpr int kQRingE = kQWin * kQWins;          // ring entries
constexpr int kQARowB = 64;                      // bytes of one block's weights (32 bf16)
constexpr int32_t kQNever = 0x3fffffff;
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;

__device__ __forceinline__ v4i16 tr_read(const lds_char* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p);
}

__device__ __forceinline__ bf16x8 join(v4i16 lo, v4i16 hi) {
    const v8i16 v = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    return __builtin_bit_cast(bf16x8, v);
}

// Waits until at most n (even) copies are outstanding; n is wave-uniform.
__device__ __forceinline__ void vm_wait_upto(int32_t n) {
    if (n <= 0) vm_wait<0>();
    else if (n == 2) vm_wait<2>();
    else if (n == 4) vm_wait<4>();
    else if (n == 6) vm_wait<6>();
    else if (n == 8) vm_wait<8>();
    else if (n == 10) vm_wait<10>();
    else if (n == 12) vm_wait<12>();
    else vm_wait<14>();
}

// One k-step of a col-group: entries [rz, rz + len) (relative to the group's
// first block) whose valid channels lie in chunk sequence numbers [smin, smax]
// (smin < 0: no valid channel).
struct QStep {
    int32_t rz, len, smin, smax;
};

template <typename TY, bool kEp>
__global__ void __launch_bounds__(kQThreads) pw_bf16(ConvArgs a) {
    __shared__ __attribute__((aligned(16))) char sX[kQRing * kQBufB + kQRowB];
    __shared__ __attribute__((aligned(16))) char sA[kQWaves * kQRingE * kQARowB];
    __shared__ __attribute__((aligned(16))) int32_t sI[kQWaves * kQRingE];
    __shared__ int32_t sNeed[kQWaves];
    __shared__ int32_t sFlag[kQRing];   // chunk sequence number that has landed in each buffer

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int32_t batch = a.npix / a.HWo;
    const int32_t gpi = (a.HWo + 7) >> 3;                 // granules per image
    const int32_t ngran = batch * gpi;
    const int32_t ntiles = (ngran + kQGran - 1) / kQGran;
    const int32_t gsets = (a.G + kQWaves - 1) / kQWaves;
    const int32_t nitems = ntiles * gsets;
    const int32_t nchunks = (a.m + kQKc - 1) >> kQKcShift;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t nloc = L < nitems ? (nitems - 1 - L) / a.total + 1 : 0;   // items of this workgroup

    for (int i = tid; i < kQRowB / 4; i += kQThreads) reinterpret_cast<int32_t*>(sX + kQZeroOff)[i] = 0;
    if (tid < kQWaves) sNeed[tid] = 0;
    if (tid < kQRing) sFlag[tid] = -1;
    __syncthreads();

    const lds_char* const lx = (const lds_char*)sX;

    if (wave >= kQWaves) {
        // (Issue arbitration favours older waves; the loaders, the youngest,
        // get the highest priority so that their copies are not issued only
        // in the compute waves' gaps.)
        __builtin_amdgcn_s_setprio(3);
        // ---- Loader waves.  Chunk sequence number s = k * nchunks + c (the
        // workgroup's item k, channel chunk c) goes to buffer s % kQRing;
        // loader wave l copies the chunks with s % kQLoaders == l, up to
        // kQInFlight at a time, and marks each in sFlag once it has landed.
        const int32_t ld = wave - kQWaves;
        const int32_t xbytes = int32_t(int64_t(batch) * a.x_img * 2);
        const v4i32 rX = buffer_rsrc(a.x, xbytes);
        // Lane l copies granule l mod 16 (8 pixels, 16 bytes) of row l / 16
        // of each 4-row copy.
        const int h = lane >> 4, gran = lane & 15;
        const int32_t rowb = a.HWo * 2;                    // bytes between channels
        const int32_t total_seq = nloc * nchunks;
        uint32_t pbase = 0;
        int32_t cur_k = -1;
        auto issue = [&](int32_t s) {
            const int32_t k = s / nchunks, c = s - k * nchunks;
            if (k != cur_k) {
                cur_k = k;
                const int32_t tile = (L + k * a.total) / gsets;
                const int32_t id = tile * kQGran + gran;
                pbase = uint32_t(xbytes);   // past the last image: the copies read zeros
                if (id < ngran) {
                    const int32_t b = id / gpi, j = id - b * gpi;
                    pbase = uint32_t(int64_t(b) * a.x_img * 2) + 16 * j;
                }
            }
            const lds_char* dst = lx + (s & (kQRing - 1)) * kQBufB;
#pragma unroll
            for (int i = 0; i < kQCopies; ++i) {
                const int32_t ch = min(c * kQKc + 4 * i + h, a.m - 1);   // rows past m copy a real row (never read)
                copy16_to_lds(rX, dst + i * kQQuadB, int32_t(pbase + uint32_t(ch * rowb)), 0);
            }
        };
        auto min_need = [&]() {
            const int32_t v = lane < kQWaves ? lds_flag_load(&sNeed[lane]) : kQNever;
            int32_t mn = kQNever;
#pragma unroll
            for (int w = 0; w < kQWaves; ++w) mn = min(mn, __builtin_amdgcn_readlane(v, w));
            return mn;
        };
        int32_t next = ld, oldest = ld, inflight = 0;
        while (next < total_seq || inflight > 0) {
            if (next < total_seq && inflight < kQInFlight && min_need() >= next - (kQRing - 1)) {
                issue(next);
                next += kQLoaders;
                ++inflight;
                continue;
            }
            if (inflight == 0) {
                __builtin_amdgcn_s_sleep(1);
                continue;
            }
            if (inflight == 2) vm_wait<kQCopies>();
            else vm_wait<0>();
            if (lane == 0) lds_flag_store(&sFlag[oldest & (kQRing - 1)], oldest);
            oldest += kQLoaders;
            --inflight;
        }
        return;
    }

    // ---- Compute waves.
    const int w = wave;
    const lds_char* const myA = (const lds_char*)sA + w * (kQRingE * kQARowB);
    const int32_t* const myI = sI + w * kQRingE;
    const lds_char* const zrow = lx + kQZeroOff;
    // Lane roles of a transposed read: lane l names entry k1 (k1 + 4 for the
    // second read) at 4 consecutive columns starting at byte colb of a 64-byte
    // block (the same roles serve the A and the B fragment).
    const int k1 = 8 * (lane >> 5) + ((lane & 15) >> 2);
    const int colb = 32 * ((lane >> 4) & 1) + 8 * (lane & 3);
    TY* __restrict__ y = static_cast<TY*>(a.y);

    f32x16 acc[kQBlocks];
    int32_t need = 0;      // first chunk this wave may still read (published in sNeed)
    int32_t landed = 0;    // chunks in [smin, landed) of the current step are known to have landed
    for (int32_t k = 0; k < nloc; ++k) {
        const int32_t item = L + k * a.total;
        const int32_t tile = item / gsets;
        const int32_t g = (item - tile * gsets) * kQWaves + w;
        const int32_t seq_base = k * nchunks;
#pragma unroll
        for (int e = 0; e < kQBlocks; ++e)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[e][r] = 0.f;

        int32_t zb = 0, ze = 0;
        if (g < a.G) group_range(a, g, zb, ze);
        const int32_t nE = ze - zb;
        if (nE > 0) {
            const int32_t nwin = (nE + kQWin - 1) / kQWin;
            const v4i32 rA = buffer_rsrc(a.D, ze * kQARowB);
            const v4i32 rI = buffer_rsrc(a.I, ze * 4);
            int32_t wi = 0;   // windows issued
            auto issue_windows = [&](int32_t upto) {   // windows [wi, min(upto, nwin))
                upto = min(upto, nwin);
                for (; wi < upto; ++wi) {
                    const int32_t slot = wi & (kQWins - 1);
                    copy16_to_lds(rA, myA + slot * (kQWin * kQARowB), lane * 16 + (zb + wi * kQWin) * kQARowB, 0);
                    if (lane < kQWin)
                        copy4_to_lds(rI, (const lds_char*)myI + slot * (kQWin * 4), lane * 4 + (zb + wi * kQWin) * 4, 0);
                }
            };
            // Waits until the windows holding entries rz .. rz + 15 have landed.
            auto wait_windows = [&](int32_t rz) {
                const int32_t wneed = min((rz + kQWin - 1) / kQWin + 1, nwin) - 1;
                vm_wait_upto(2 * (wi - 1 - wneed));
            };
            // Channel indices for the step at rz: pl (lanes < 16: entry rz +
            // lane), o1 / o2 (entry rz + k1 / rz + k1 + 4).
            auto plan_reads = [&](int32_t rz, int32_t& pl, int32_t& o1, int32_t& o2) {
                pl = myI[(rz + (lane & 15)) & (kQRingE - 1)];
                o1 = myI[(rz + k1) & (kQRingE - 1)];
                o2 = myI[(rz + k1 + 4) & (kQRingE - 1)];
            };
            auto plan = [&](int32_t rz, int32_t pl) {
                QStep st;
                st.rz = rz;
                const bool inE = lane < kQWin && rz + lane < nE;
                const bool okc = inE && pl >= 0 && pl < a.m;
                const int32_t sq = seq_base + (pl >> kQKcShift);
                const int32_t avail = __builtin_popcountll(__ballot(inE));
                const uint64_t mv = __ballot(okc);
                if (mv == 0) {
                    st.len = avail;
                    st.smin = st.smax = -1;
                    return st;
                }
                st.smin = __builtin_amdgcn_readlane(sq, __builtin_ctzll(mv));
                const uint64_t far = __ballot(okc && sq > st.smin + (kQSpan - 1));
                st.len = min(avail, far ? int32_t(__builtin_ctzll(far)) : 64);
                // Channels ascend within a col-group, so the step's last
                // valid entry has its highest chunk.
                const uint64_t in_step = st.len >= 64 ? mv : mv & ((uint64_t(1) << st.len) - 1);
                st.smax = __builtin_amdgcn_readlane(sq, 63 - __builtin_clzll(in_step));
                return st;
            };
            // LDS addresses of one lane's entry (k1 + 4 hh) for a step: its A
            // row and its X row (the four column blocks follow at 64-byte
            // steps), or the zero row.
            struct Addr {
                const lds_char* ap;
                int32_t xoff;
            };
            auto addr = [&](const QStep& st, int32_t ch, int hh) {
                Addr r;
                const int32_t e = k1 + 4 * hh;
                const bool ok = e < st.len && uint32_t(ch) < uint32_t(a.m);
                const int32_t row = ch & (kQKc - 1);
                r.xoff = ok ? ((seq_base + (ch >> kQKcShift)) & (kQRing - 1)) * kQBufB + (row >> 2) * kQQuadB +
                                  (row & 3) * kQRowB + colb
                            : kQZeroOff + colb;
                r.ap = ok ? myA + ((st.rz + e) & (kQRingE - 1)) * kQARowB + colb : zrow + colb;
                return r;
            };
            // Waits until the chunks [smin, smax] of a step have landed.  A
            // buffer's flag only grows (s, s + kQRing, ...), and a buffer
            // holding a chunk this wave has not released is not refilled, so
            // flag >= s means chunk s is in place.  Chunks below smin are
            // never waited for: the wave may have released them unseen.
            auto wait_landed = [&](const QStep& st) {
                for (landed = max(landed, st.smin); landed <= st.smax;) {
                    if (__builtin_amdgcn_readfirstlane(lds_flag_load(&sFlag[landed & (kQRing - 1)])) >= landed) ++landed;
                    else __builtin_amdgcn_s_sleep(1);
                }
                fence_compiler();
            };
            auto release = [&](const QStep& st) {
                if (st.smin > need) {
                    need = st.smin;
                    if (lane == 0) lds_flag_store(&sNeed[w], need);
                }
            };

            // Prologue: step 0 planned and its fragments read; step 1's indices read.
            issue_windows(kQWins - 1);
            wait_windows(0);
            int32_t pl, o1, o2;
            plan_reads(0, pl, o1, o2);
            wait_lgkm();
            QStep cur = plan(0, pl);
            release(cur);
            wait_landed(cur);
            v4i16 ra[2], rb[kQBlocks][2];
            {
                const Addr p1 = addr(cur, o1, 0), p2 = addr(cur, o2, 1);
                ra[0] = tr_read(p1.ap);
                ra[1] = tr_read(p2.ap);
#pragma unroll
                for (int blk = 0; blk < kQBlocks; ++blk) {
                    rb[blk][0] = tr_read(lx + p1.xoff + 64 * blk);
                    rb[blk][1] = tr_read(lx + p2.xoff + 64 * blk);
                }
            }
            int32_t rz_next = cur.len;
            if (rz_next < nE) {
                wait_windows(rz_next);
                plan_reads(rz_next, pl, o1, o2);
            }

            // Step j: multiply the fragments in (ra, rb); plan step j+1 from
            // (pl, o1, o2) and read its fragments into (ra, rb) as each of
            // step j's MFMAs takes its operands; read step j+2's indices.
            while (true) {
                wait_lgkm();
                const bool has_next = rz_next < nE;
                QStep nxt = plan(rz_next, pl);
                if (!has_next) nxt.len = 0;
                if (has_next) {
                    release(nxt);
                    // Windows in use: those of steps j+1 and j+2 (at most 3
                    // from rz_next's); the other slots may be refilled.
                    issue_windows(rz_next / kQWin + kQWins);
                    wait_landed(nxt);
                }
                const int32_t rz2 = rz_next + nxt.len;
                const bool has_next2 = has_next && rz2 < nE;
                const Addr p1 = addr(nxt, o1, 0), p2 = addr(nxt, o2, 1);
                const bf16x8 af = join(ra[0], ra[1]);
                ra[0] = tr_read(p1.ap);
                ra[1] = tr_read(p2.ap);
#pragma unroll
                for (int blk = 0; blk < kQBlocks; ++blk) {
                    acc[blk] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, join(rb[blk][0], rb[blk][1]),
                                                                     acc[blk], 0, 0, 0);
                    rb[blk][0] = tr_read(lx + p1.xoff + 64 * blk);
                    rb[blk][1] = tr_read(lx + p2.xoff + 64 * blk);
                }
                if (has_next2) {
                    wait_windows(rz2);
                    plan_reads(rz2, pl, o1, o2);
                }
                if (!has_next) break;
                rz_next = rz2;
            }
            wait_lgkm();
        }
        // Past this item's chunks.
        if (seq_base + nchunks > need) {
            need = seq_base + nchunks;
            if (lane == 0) lds_flag_store(&sNeed[w], need);
        }

        // Store: MFMA (row, col) of block e -> output channel g*32 + row, tile column 32e + col.
        if (g < a.G) {
#pragma unroll
            for (int e = 0; e < kQBlocks; ++e) {
                const int32_t n = 32 * e + (lane & 31);
                const int32_t id = tile * kQGran + (n >> 3);
                const int32_t b = id / gpi;
                const int32_t hw = 8 * (id - b * gpi) + (n & 7);
                if (id >= ngran || hw >= a.HWo) continue;
                TY* yb = y + int64_t(b) * a.y_img + hw;
#pragma unroll
                for (int r = 0; r < 16; ++r) {
                    const int32_t o = g * 32 + PwMfma<32>::row(lane, r);
                    if (o < a.n) store_out(&yb[int64_t(o) * a.y_c], from_f32<TY>(epilogue<kEp>(a, o, acc[e][r])));
                }
            }
        }
    }
    if (lane == 0) lds_flag_store(&sNeed[w], kQNever);
}

template <typename TY>
onexn_status launch_typed(ConvArgs a, hipStream_t s) {
    const int64_t batch = a.npix / a.HWo;
    const int64_t gpi = (a.HWo + 7) / 8;
    const int64_t ntiles = (batch * gpi + kQGran - 1) / kQGran;
    const int64_t nitems = ntiles * ((a.G + kQWaves - 1) / kQWaves);
    int64_t wgs = nitems;
    if (tuning(kTunePwbWgs) >= 1) wgs = std::min<int64_t>(tuning(kTunePwbWgs), nitems);
    return with_epilogue(a, [&](auto ep) {
        return launch_grid(pw_bf16<TY, decltype(ep)::value>, a, wgs, s, kQThreads);
    });
}

}  // namespace

bool pw_bf16_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_BF16 || layout != ONEXN_NCHW || a.N != 32) return false;
    if (a.kh != 1 || a.kw != 1 || a.sh != 1 || a.sw != 1 || a.ph != 0 || a.pw != 0) return false;
    if (a.HWo % 4 != 0 || (reinterpret_cast<uintptr_t>(a.x) & 15) != 0) return false;
    const int64_t batch = a.npix / a.HWo;
    if (batch * a.x_img * 2 >= (int64_t(1) << 31)) return false;   // 32-bit buffer offsets
    if (int64_t(a.t) * 64 >= (int64_t(1) << 31)) return false;
    (void)ydt;
    return true;
}

onexn_status launch_pw_bf16(ConvArgs a, onexn_dtype ydt, hipStream_t s) {
    if (ydt == ONEXN_BF16) return launch_typed<uint16_t>(a, s);
    return launch_typed<float>(a, s);
}

}  // namespace onexn
