// Pointwise (1x1, stride 1, no padding, NCHW) 1xN-pruned convolution with
// bf16 inputs and weights, fp32 accumulation, N = 32, bf16 or fp32 output:
// the input operand is gathered straight from global memory into registers.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the contraction
//     Y_g[32][pixels] = D_g^T[32][kept_g] * X[I_g][pixels]:
// its kept blocks select rows of the input matrix X[channel][pixel].
//
// Matrix cores.  v_mfma_f32_32x32x16_bf16 multiplies a 32x16 A fragment (the
// 32 weights of 16 kept blocks) by a 16x32 B fragment (16 gathered input rows
// at 32 pixels).  Lane l = 32 h + q holds, for both operands, the contraction
// entries 8 h .. 8 h + 7 of one row (A: output q) or one column (B: pixel q).
//
// B without a transposition buffer.  A wave computes one col-group over a
// tile of 32 granules of GP = 8 (or 4) consecutive pixels of one image, lane
// q owning granule q.  For a step of 16 kept blocks, lane (h, q) loads its
// granule from the 8 input rows of entries 8 h .. 8 h + 7 (16 or 8 bytes
// each), i.e. an 8 x GP block of bf16 values; byte permutes regroup it into
// GP B fragments, one per pixel of the granule, so MFMA column block k is
// pixel k of granule q.  Each load reads 512 (256) contiguous bytes per
// half-wave.  A lane's outputs of a row are consecutive pixels again, stored
// with 8- or 16-byte writes.
//
// A fragments.  A step's 16 blocks of D are one contiguous kilobyte
// (16 x 32 bf16, output-contiguous); a lane loads 16 bytes of it, writes them
// to the wave's LDS slot, and two ds_read_b64_tr_b16 transpose the slot into
// the A fragment (lane (h, q) reads entries 8 h + i of output q).
//
// Pipelining.  The loads of step j + kRP (inputs and weights) are issued
// before the MFMAs of step j, so every load has kRP steps of other waves' and
// its own work to land.  All waits are the compiler's own vmcnt counts over
// these builtin loads; the channel indices come from LDS.
// Entries past the col-group's end, and channels outside [0, m), load zero
// inputs (an out-of-range buffer offset) and zero weights (the weight buffer
// ends at the col-group's last block), so they add exactly nothing.
//
// Work split.  A workgroup is 8 waves, one col-group each, over one pixel
// tile; the workgroups of a tile are consecutive, so they run on one XCD and
// share the tile's input rows in its L2.
#include <type_traits>

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kRWaves = 8;                 // col-groups per workgroup (one per wave)
constexpr int kRThreads = 64 * kRWaves;
constexpr int kRGran = 32;                 // 4-pixel granules per tile
constexpr int kRWin = 2048;                // channel indices staged per wave (input channels at most)
typedef short v4i16 __attribute__((ext_vector_type(4)));
typedef short v8i16 __attribute__((ext_vector_type(8)));
typedef __attribute__((address_space(3))) v4i16 lds_v4i16;
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef int32_t i32x4 __attribute__((ext_vector_type(4)));

__device__ __forceinline__ v4i16 tr_read(const lds_char* p) {
    return __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_v4i16*)p);
}

// A lane's outputs of one row: 4 (or the upper 4 of 8) consecutive pixels.
template <typename TY> struct Out4;
template <> struct Out4<uint16_t> {
    typedef u32x2 T;   // four bf16
    __device__ static T pack(float a, float b, float c, float d) {
        T r;
        r.x = uint32_t(f32_to_bf16(a)) | (uint32_t(f32_to_bf16(b)) << 16);
        r.y = uint32_t(f32_to_bf16(c)) | (uint32_t(f32_to_bf16(d)) << 16);
        return r;
    }
};
template <> struct Out4<float> {
    typedef f32x4 T;
    __device__ static T pack(float a, float b, float c, float d) { return T{a, b, c, d}; }
};
// A lane's 8 consecutive outputs of one row, written with one store where
// the granule has no duplicate pixels.
template <typename TY> struct Out8;
template <> struct Out8<uint16_t> {
    typedef u32x4 T;
    __device__ static T join(u32x2 lo, u32x2 hi) { return T{lo.x, lo.y, hi.x, hi.y}; }
};
template <> struct Out8<float> {
    typedef float T __attribute__((ext_vector_type(8)));
    __device__ static T join(f32x4 lo, f32x4 hi) {
        return __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
    }
};

// kRP: steps of loads in flight ahead of the multiplied step.  GP: pixels
// per granule (4: 8-byte loads, a 128-pixel tile; 8: 16-byte loads, a
// 256-pixel tile, fewer cache lines per gathered byte and half the weight
// reads per MFMA; an image's last granule then starts 8 pixels before its
// end and its first pixels, duplicates of the previous granule's, are not
// stored).
template <typename TY, int kRP, int GP, bool kEp>
__global__ void __launch_bounds__(kRThreads) pw_bf16r(ConvArgs a) {
    static_assert(GP == 4 || GP == 8, "granule of 4 or 8 pixels");
    typedef typename std::conditional<GP == 8, u32x4, u32x2>::type gran_t;
    constexpr int kRSlots = kRP + 1;   // register slots of the pipeline
    __shared__ __attribute__((aligned(16))) char sA[kRWaves * 1024];
    __shared__ __attribute__((aligned(16))) int32_t sI[kRWaves * (kRWin + 16)];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int q = lane & 31, h = lane >> 5;
    const int32_t gsets = (a.G + kRWaves - 1) / kRWaves;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    const int32_t tile = L / gsets;
    const int32_t g = (L - tile * gsets) * kRWaves + wave;
    int32_t zb = 0, ze = 0;
    if (g < a.G) group_range(a, g, zb, ze);
    const int32_t nsteps = (ze - zb + 15) >> 4;

    // The lane's granule: image b, pixels hw0 .. hw0 + GP - 1, of which the
    // first `dup` repeat the previous granule's (an image's last granule).
    const int32_t batch = a.npix / a.HWo;
    const int32_t gpi = (a.HWo + GP - 1) / GP;
    const int32_t gi = tile * kRGran + q;
    const bool gvalid = gi < batch * gpi;
    const int32_t b = gvalid ? gi / gpi : 0, jg = gvalid ? gi - b * gpi : 0;
    const int32_t hw0 = min(GP * jg, a.HWo - GP), dup = GP * jg - hw0;
    const int32_t xbytes = int32_t(int64_t(batch) * a.x_img * 2);
    const uint32_t pixoff = gvalid ? uint32_t((int64_t(b) * a.x_img + hw0) * 2) : kBufferOutOfRange;
    const uint32_t chb = uint32_t(a.HWo) * 2;   // bytes between input channels

    const __amdgpu_buffer_rsrc_t rX =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.x), 0, xbytes, kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rD =
        __builtin_amdgcn_make_buffer_rsrc(const_cast<void*>(a.D), 0, ze * 64, kRawBufferFlags);

    // Transposed-read roles (A fragment): lane l reads entry k1 (k1 + 4) of
    // its slot at 4 consecutive outputs starting at byte colb of a 64-byte row.
    const int k1 = 8 * (lane >> 5) + ((lane & 15) >> 2);
    const int colb = 32 * ((lane >> 4) & 1) + 8 * (lane & 3);
    char* const slot = sA + wave * 1024;
    const lds_char* const lslot = (const lds_char*)slot;

    // Channel indices: all of the col-group's entries (at most m <= kRWin),
    // staged in the wave's LDS once and read back as 8 consecutive entries
    // per lane, so index reads use the LDS counter and never wait behind
    // input loads.  Entries past the col-group read zeros.
    // Each staged index is then turned, once, into the byte offset of its
    // input row (kBufferOutOfRange for a channel outside [0, m) and for the
    // 16 entries past the col-group's end), so a gathered load costs one add.
    int32_t* const win = sI + wave * (kRWin + 16);
    {
        const v4i32 rIw = buffer_rsrc(a.I, ze * 4);
        const int32_t nE = ze - zb;
        for (int32_t e = 0; e < nE; e += 64)
            copy4_to_lds(rIw, (const lds_char*)(win + e), (zb + e + lane) * 4, 0);
        vm_wait<0>();
        for (int32_t e = lane; e < nE + 16; e += 64) {
            const int32_t ch = e < nE ? win[e] : -1;
            win[e] = int32_t(uint32_t(ch) < uint32_t(a.m) ? uint32_t(ch) * chb : kBufferOutOfRange);
        }
    }

    // Pipeline registers, indexed by step % kRSlots.
    gran_t xv[kRSlots][8];   // the lane's granule at the channels of entries 8 h .. 8 h + 7
    i32x4 av[kRSlots];       // the lane's 16 bytes of the step's weights

    // Steps past the last one (only ever prefetched, never multiplied) read
    // clamped window positions: any offset is safe in a range-checked load.
    auto load_step = [&](int s, int32_t step) __attribute__((always_inline)) {
        const int32_t rel = min(step * 16 + 8 * h, kRWin + 8);
        const i32x4 c03 = *reinterpret_cast<const i32x4*>(win + rel);
        const i32x4 c47 = *reinterpret_cast<const i32x4*>(win + rel + 4);
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            // Both terms are below 2^31, and either one out of range keeps
            // the sum out of range (no wrap).
            const uint32_t off = pixoff + uint32_t(j < 4 ? c03[j] : c47[j - 4]);
            if constexpr (GP == 8)
                xv[s][j] = __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(rX, int32_t(off), 0, 0));
            else
                xv[s][j] = __builtin_bit_cast(u32x2, __builtin_amdgcn_raw_buffer_load_b64(rX, int32_t(off), 0, 0));
        }
        av[s] = __builtin_bit_cast(i32x4, __builtin_amdgcn_raw_buffer_load_b128(
                                              rD, (zb + step * 16) * 64 + lane * 16, 0, 0));
    };

    f32x16 acc[GP];
#pragma unroll
    for (int k = 0; k < GP; ++k)
#pragma unroll
        for (int r = 0; r < 16; ++r) acc[k][r] = 0.f;

    auto compute = [&](int s) __attribute__((always_inline)) {
        // A: stage the step's weights in the wave's slot, read them transposed.
        *reinterpret_cast<i32x4*>(slot + lane * 16) = av[s];
        const v4i16 lo = tr_read(lslot + k1 * 64 + colb);
        const v4i16 hi = tr_read(lslot + (k1 + 4) * 64 + colb);
        const bf16x8 af = __builtin_bit_cast(bf16x8, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
        // B: fragment k takes pixel k of the granule from each of the 8 rows.
#pragma unroll
        for (int k = 0; k < GP; ++k) {
            const uint32_t sel = (k & 1) ? 0x07060302u : 0x05040100u;
            u32x4 bw;
#pragma unroll
            for (int d = 0; d < 4; ++d)
                bw[d] = __builtin_amdgcn_perm(xv[s][2 * d + 1][k >> 1], xv[s][2 * d][k >> 1], sel);
            acc[k] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(af, __builtin_bit_cast(bf16x8, bw), acc[k], 0, 0, 0);
        }
    };

    // Prologue: the loads of steps 0 .. kRP-1.
#pragma unroll
    for (int s = 0; s < kRP; ++s) load_step(s, s);
    // Step j: issue step j + kRP's loads, then multiply step j.  Whole
    // periods of kRSlots steps run branch-free (the register slots are
    // compile-time indices); the last partial period after.  Scheduling
    // barriers keep each step's loads in program order.
    auto step = [&](int u, int32_t j) __attribute__((always_inline)) {
        __builtin_amdgcn_sched_barrier(0);
        load_step((u + kRP) % kRSlots, j + kRP);
        __builtin_amdgcn_sched_barrier(0);
        compute(u);
    };
    const int32_t nfull = nsteps / kRSlots * kRSlots;
    for (int32_t j0 = 0; j0 < nfull; j0 += kRSlots) {
#pragma unroll
        for (int u = 0; u < kRSlots; ++u) step(u, j0 + u);
    }
#pragma unroll
    for (int u = 0; u < kRSlots - 1; ++u)
        if (nfull + u < nsteps) step(u, nfull + u);

    // Store: MFMA (row, col) of block k -> output channel g*32 + row, pixel
    // hw0 + k of the lane's granule (col), k >= dup.
    if (g >= a.G || !gvalid) return;
    TY* __restrict__ y = static_cast<TY*>(a.y);
    TY* const yb = y + int64_t(b) * a.y_img + hw0;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        const int32_t o = g * 32 + PwMfma<32>::row(lane, r);
        if (o >= a.n) continue;
        TY* const yr = yb + int64_t(o) * a.y_c;
#pragma unroll
        for (int k = 0; k < GP; ++k) acc[k][r] = epilogue<kEp>(a, o, acc[k][r]);
        if constexpr (GP == 8) {
            const typename Out4<TY>::T lo = Out4<TY>::pack(acc[0][r], acc[1][r], acc[2][r], acc[3][r]);
            const typename Out4<TY>::T hi = Out4<TY>::pack(acc[4][r], acc[5][r], acc[6][r], acc[7][r]);
            if (dup == 0)
                store_out(reinterpret_cast<typename Out8<TY>::T*>(yr), Out8<TY>::join(lo, hi));
            else
                store_out(reinterpret_cast<typename Out4<TY>::T*>(yr + 4), hi);
        } else {
            store_out(reinterpret_cast<typename Out4<TY>::T*>(yr), Out4<TY>::pack(acc[0][r], acc[1][r], acc[2][r], acc[3][r]));
        }
    }
}

template <typename TY, bool E>
onexn_status launch_typed(ConvArgs a, hipStream_t s) {
    const int64_t batch = a.npix / a.HWo;
    const int64_t gsets = (a.G + kRWaves - 1) / kRWaves;
    // 8-pixel granules where an image has at least 8 pixels (2048 -> 2048 at
    // 14x14: 380 us against 445 us with 4-pixel ones, from fewer cache lines
    // per gathered byte), else 4.  Steps in flight: one for 8-pixel granules
    // (their accumulators take twice the registers), two for 4 (deeper
    // pipelines add registers, not bandwidth).
    int gp = a.HWo >= 8 ? 8 : 4, rp = 0;
    if (tuning(kTunePwbGp) >= 0) gp = tuning(kTunePwbGp);
    if (tuning(kTunePwbRp) >= 0) rp = tuning(kTunePwbRp);
    if (gp == 8 && a.HWo >= 8) {
        const int64_t grid = (batch * ((a.HWo + 7) / 8) + kRGran - 1) / kRGran * gsets;
        if (rp == 2) return launch_grid(pw_bf16r<TY, 2, 8, E>, a, grid, s, kRThreads);
        return launch_grid(pw_bf16r<TY, 1, 8, E>, a, grid, s, kRThreads);
    }
    const int64_t grid = (batch * (a.HWo / 4) + kRGran - 1) / kRGran * gsets;
    switch (rp) {
        case 4: return launch_grid(pw_bf16r<TY, 4, 4, E>, a, grid, s, kRThreads);
        case 6: return launch_grid(pw_bf16r<TY, 6, 4, E>, a, grid, s, kRThreads);
        default: return launch_grid(pw_bf16r<TY, 2, 4, E>, a, grid, s, kRThreads);
    }
}

}  // namespace

bool pw_bf16r_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_BF16 || layout != ONEXN_NCHW || a.N != 32) return false;
    if (a.kh != 1 || a.kw != 1 || a.sh != 1 || a.sw != 1 || a.ph != 0 || a.pw != 0) return false;
    if (a.HWo % 4 != 0 || a.m > kRWin) return false;
    // 8-byte input granules; 8-byte (bf16) or 16-byte (fp32) output writes.
    if ((reinterpret_cast<uintptr_t>(a.x) & 7) != 0) return false;
    if ((reinterpret_cast<uintptr_t>(a.y) & (ydt == ONEXN_BF16 ? 7 : 15)) != 0) return false;
    const int64_t batch = a.npix / a.HWo;
    if (batch * a.x_img * 2 >= (int64_t(1) << 31)) return false;   // 32-bit buffer offsets
    if (int64_t(a.t) * 64 + 16384 >= (int64_t(1) << 31)) return false;   // weight offsets of the pipelined steps past the end
    return true;
}

onexn_status launch_pw_bf16r(ConvArgs a, onexn_dtype ydt, hipStream_t s) {
    return with_epilogue(a, [&](auto ep) {
        constexpr bool E = decltype(ep)::value;
        if (ydt == ONEXN_BF16) return launch_typed<uint16_t, E>(a, s);
        return launch_typed<float, E>(a, s);
    });
}

}  // namespace onexn
