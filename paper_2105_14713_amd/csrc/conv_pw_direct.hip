// 1x1 1xN-pruned convolution (any stride and padding), fp32, NCHW,
// N in {16, 32}, with both matrix-core operands loaded straight from global
// memory into registers.
//
// Paper: Lin et al., "1xN Pattern for Pruning Convolutional Neural Networks"
// (arXiv 2105.14713), Sec. 3.4, Eq. 8.  Col-group g is the contraction
//     Y_g[N][pixels] = D_g^T[N][kept_g] * X[I_g][pixels].
//
// Operand layout.  An fp32 MFMA lane holds one contraction entry of one row
// (A) or one column (B):
//   N = 32, v_mfma_f32_32x32x2f32: lane l holds A[row l % 32][entry l / 32],
//     i.e. D[z + l / 32][l % 32] -- the two kept blocks' 64 weights are one
//     contiguous 256-byte run of D -- and B[entry l / 32][pixel l % 32], i.e.
//     input channel I[z + l / 32] at the lane's pixel: 32 consecutive pixels
//     of one gathered input row per half-wave.
//   N = 16, v_mfma_f32_16x16x4f32: the same with four blocks and 16 pixels.
// So neither operand needs a transposition or an LDS staging buffer: each
// step is one weight load and one input load per column block, all
// coalesced, and the input offset of a pixel (stride and padding included)
// is computed once.
//
// Work split.  A unit is (col-group, NB column blocks of pixels).  A
// workgroup of four waves takes 4 / KSPLIT units; KSPLIT waves share a unit's
// kept blocks (contiguous ranges) and add their partial sums through LDS at
// the end, for layers with few pixels and long col-groups.
//
// Pipelining.  Steps are taken in batches of kDB: channel indices come in
// lane-parallel windows of 64 entries loaded a window ahead, a batch's
// weight and input loads are all issued before the previous batch's MFMAs,
// so a wave keeps two batches of loads in flight.  Entries past the wave's
// range and channels outside [0, m) read zeros (out-of-range buffer offsets),
// so they add nothing.
#include <cstdlib>

#include "lds_copy.h"
#include "pw_common.h"

namespace onexn {
namespace {

constexpr int kDThreads = 256;
constexpr int kDB = 8;   // MFMA steps per batch

template <int N, int NB, int KSPLIT>
__global__ void __launch_bounds__(kDThreads) pw_direct(ConvArgs a) {
    typedef PwMfma<N> M;
    typedef typename M::acc_t acc_t;
    constexpr int KS = M::KS, COLS = M::COLS;
    constexpr int UPW = 4 / KSPLIT;                 // units per workgroup
    constexpr int RED = KSPLIT > 1 ? 4 * NB * M::ACC * 64 : 1;
    __shared__ float sR[RED];

    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int uw = wave / KSPLIT, kq = wave % KSPLIT;
    const int32_t L = xcd_remap(int32_t(blockIdx.x), a.total);
    // Units are numbered pixel-block-major, col-group-minor, so the
    // workgroups sharing a pixel range run on one XCD (and its L2).
    const int32_t unit = L * UPW + uw;
    const int32_t pblocks = (a.npix + NB * COLS - 1) / (NB * COLS);
    const int32_t g = unit % a.G, pb = unit / a.G;
    const bool live = pb < pblocks;
    int32_t zb = 0, ze = 0;
    if (live) group_range(a, g, zb, ze);
    const int32_t per = (ze - zb + KSPLIT - 1) / KSPLIT;
    const int32_t z0 = min(ze, zb + kq * per), z1 = min(ze, z0 + per);

    const int32_t batch = a.npix / a.HWo;
    const uint32_t xbytes = uint32_t(int64_t(batch) * a.x_img * 4);
    const int col = lane % COLS, kk = lane / COLS;   // lane's pixel column and entry within a step

    // Byte offset of the lane's input pixel (channel 0) in each column block,
    // or xbytes where there is none (past the last pixel, or in the padding).
    uint32_t xo[NB];
    int64_t yo[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        const int32_t p = (pb * NB + nb) * COLS + col;
        xo[nb] = xbytes;
        yo[nb] = -1;
        if (live && p < a.npix) {
            const int32_t b = p / a.HWo, hw = p - b * a.HWo;
            const int32_t oh = hw / a.Wo, ow = hw - oh * a.Wo;
            const int32_t ih = oh * a.sh - a.ph, iw = ow * a.sw - a.pw;
            if (ih >= 0 && ih < a.H && iw >= 0 && iw < a.W)
                xo[nb] = uint32_t((int64_t(b) * a.x_img + int64_t(ih) * a.W + iw) * 4);
            yo[nb] = int64_t(b) * a.y_img + hw;
        }
    }

    // The sizes are wave-uniform; saying so (readfirstlane) keeps the buffer
    // resources in scalar registers -- a resource the compiler must treat as
    // divergent turns every load into a loop over the distinct values.
    const __amdgpu_buffer_rsrc_t rX = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.x), 0, __builtin_amdgcn_readfirstlane(int32_t(xbytes)), kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rD = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<void*>(a.D), 0, __builtin_amdgcn_readfirstlane(z1 * N * 4), kRawBufferFlags);
    const __amdgpu_buffer_rsrc_t rI = __builtin_amdgcn_make_buffer_rsrc(
        const_cast<int32_t*>(a.I), 0, __builtin_amdgcn_readfirstlane(z1 * 4), kRawBufferFlags);
    const uint32_t chb = uint32_t(a.x_c) * 4;   // bytes between input channels

    acc_t acc[NB];
#pragma unroll
    for (int nb = 0; nb < NB; ++nb)
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) acc[nb][r] = 0.f;

    struct Batch {
        float av[kDB];
        float bv[kDB][NB];
    };
    // Channel indices come in windows of 64 entries (lane j: entry wbase + j),
    // loaded a window ahead of use, so a batch's input addresses never wait
    // for an index load.  Entries at or past z1 and channels outside [0, m)
    // read zeros.
    constexpr int E = kDB * KS;   // entries per batch (divides 64)
    static_assert(64 % E == 0, "batches tile the index windows");
    auto load_idx = [&](int32_t z) { return int32_t(__builtin_amdgcn_raw_buffer_load_b32(rI, (z + lane) * 4, 0, 0)); };
    int32_t wbase = z0;
    int32_t ivw = load_idx(z0), ivn = load_idx(z0 + 64);
    auto issue = [&](Batch& bt, int32_t z) {
        if (z - wbase >= 64) {
            wbase += 64;
            ivw = ivn;
            ivn = load_idx(wbase + 64);
        }
        const int32_t off = z - wbase;
#pragma unroll
        for (int st = 0; st < kDB; ++st) {
            const int32_t ze_ = z + st * KS;
            bt.av[st] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(rD, (ze_ * N + lane) * 4, 0, 0));
            const int32_t ch = __builtin_amdgcn_ds_bpermute(4 * (off + st * KS + kk), ivw);
            const bool ok = ze_ + kk < z1 && uint32_t(ch) < uint32_t(a.m);
            const uint32_t choff = ok ? uint32_t(ch) * chb : xbytes;
#pragma unroll
            for (int nb = 0; nb < NB; ++nb)
                bt.bv[st][nb] = __builtin_bit_cast(float, __builtin_amdgcn_raw_buffer_load_b32(
                    rX, int32_t(min(xo[nb] + choff, xbytes)), 0, 0));
        }
    };
    auto consume = [&](const Batch& bt) {
#pragma unroll
        for (int st = 0; st < kDB; ++st)
#pragma unroll
            for (int nb = 0; nb < NB; ++nb) acc[nb] = M::step(bt.av[st], bt.bv[st][nb], acc[nb]);
    };

    const int32_t nbat = (z1 - z0 + E - 1) / E;
    if (nbat > 0) {
        Batch b0, b1;
        issue(b0, z0);
        for (int32_t bi = 0; bi < nbat; bi += 2) {
            if (bi + 1 < nbat) issue(b1, z0 + (bi + 1) * E);
            consume(b0);
            if (bi + 1 >= nbat) break;
            if (bi + 2 < nbat) issue(b0, z0 + (bi + 2) * E);
            consume(b1);
        }
    }

    if constexpr (KSPLIT > 1) {
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < M::ACC; ++r) sR[((wave * NB + nb) * M::ACC + r) * 64 + lane] = acc[nb][r];
        __syncthreads();
        if (kq != 0) return;
#pragma unroll
        for (int nb = 0; nb < NB; ++nb)
#pragma unroll
            for (int r = 0; r < M::ACC; ++r)
#pragma unroll
                for (int k = 1; k < KSPLIT; ++k) acc[nb][r] += sR[(((wave + k) * NB + nb) * M::ACC + r) * 64 + lane];
    }
    if (!live) return;

    float* __restrict__ y = static_cast<float*>(a.y);
#pragma unroll
    for (int nb = 0; nb < NB; ++nb) {
        if (yo[nb] < 0) continue;
#pragma unroll
        for (int r = 0; r < M::ACC; ++r) {
            const int32_t oc = g * N + M::row(lane, r);
            if (oc < a.n) y[yo[nb] + int64_t(oc) * a.y_c] = acc[nb][r];
        }
    }
}

template <int N, int NB, int KSPLIT>
onexn_status launch_cfg(ConvArgs a, hipStream_t s) {
    constexpr int COLS = PwMfma<N>::COLS;
    const int64_t units = (int64_t(a.npix) + NB * COLS - 1) / (NB * COLS) * a.G;
    const int64_t upw = 4 / KSPLIT;
    return launch_grid(pw_direct<N, NB, KSPLIT>, a, (units + upw - 1) / upw, s, kDThreads);
}

// (column blocks per unit, waves per unit): the largest tile that gives every
// compute unit a few workgroups, splitting the contraction only when the
// col-groups are long.
template <int N>
onexn_status launch_n(ConvArgs a, hipStream_t s) {
    constexpr int COLS = PwMfma<N>::COLS;
    const int64_t want = 4 * int64_t(device_cu_count());
    const int64_t avg_kept = a.G > 0 ? a.t / a.G : 0;
    auto wgs = [&](int nb, int ks) {
        return ((int64_t(a.npix) + nb * COLS - 1) / (nb * COLS) * a.G * ks + 3) / 4;
    };
    int choice = 0;
    if (const char* env = std::getenv("ONEXN_DIRECT_TILE")) choice = std::atoi(env);   // testing
    if (choice == 0) {
        if (wgs(2, 1) >= want || avg_kept < 64) choice = 1;
        else if (wgs(1, 1) >= want || avg_kept < 128) choice = 2;
        else if (wgs(1, 2) >= want || avg_kept < 256) choice = 3;
        else choice = 4;
    }
    switch (choice) {
        case 1: return launch_cfg<N, 2, 1>(a, s);
        case 2: return launch_cfg<N, 1, 1>(a, s);
        case 3: return launch_cfg<N, 1, 2>(a, s);
        default: return launch_cfg<N, 1, 4>(a, s);
    }
}

}  // namespace

bool pw_direct_applies(const ConvArgs& a, onexn_dtype xdt, onexn_dtype ydt, onexn_layout layout) {
    if (xdt != ONEXN_F32 || ydt != ONEXN_F32 || layout != ONEXN_NCHW) return false;
    if (a.N != 16 && a.N != 32) return false;
    if (a.kh != 1 || a.kw != 1) return false;
    const int64_t batch = a.npix / a.HWo;
    // 32-bit buffer offsets, with room for an out-of-range marker plus a
    // channel offset.
    if (batch * a.x_img * 4 >= (int64_t(1) << 31)) return false;
    if (int64_t(a.t) * a.N * 4 >= (int64_t(1) << 31)) return false;
    return true;
}

onexn_status launch_pw_direct(ConvArgs a, hipStream_t s) {
    return a.N == 16 ? launch_n<16>(a, s) : launch_n<32>(a, s);
}

}  // namespace onexn
