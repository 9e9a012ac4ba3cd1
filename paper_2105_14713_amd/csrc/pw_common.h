// Definitions shared by the pointwise (1x1) kernels of libonexn.so.
#pragma once

#include "conv_common.h"

namespace onexn {

template <int N> struct PwMfma;
template <> struct PwMfma<16> {   // 16x16x4 f32
    typedef f32x4 acc_t;
    static constexpr int KS = 4, ACC = 4, COLS = 16;
    __device__ static acc_t step(float a, float b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
    __device__ static int row(int lane, int r) { return 4 * (lane / 16) + r; }
};
template <> struct PwMfma<32> {   // 32x32x2 f32
    typedef f32x16 acc_t;
    static constexpr int KS = 2, ACC = 16, COLS = 32;
    __device__ static acc_t step(float a, float b, acc_t c) {
        return __builtin_amdgcn_mfma_f32_32x32x2f32(a, b, c, 0, 0, 0);
    }
    __device__ static int row(int lane, int r) { return 8 * (r / 4) + 4 * (lane / 32) + (r % 4); }
};

// Fused-epilogue parameters (scale, bias) of the M::ACC output rows a lane of
// an MFMA kernel stores for one col-group g.  Those rows come in runs of four
// consecutive channels (row(lane, 4q + j) = row(lane, 4q) + j), so the
// parameters are read as 4-channel vectors once per store stage: two vector
// loads per four rows instead of two loads per stored value.  An absent
// parameter reads as scale 1 / bias 0 (the result equals the plain product or
// sum).  Without an epilogue (kEp false) the struct holds and does nothing.
template <int N, bool kEp>
struct EpRows {
    typedef PwMfma<N> M;
    static constexpr int ACC = M::ACC, S = kEp ? ACC : 1;
    float s[S], b[S];

    // From global memory: channels at or past n read as scale 1 / bias 0.
    // The loads are issued where this is called: the opaque copy of g keeps
    // the compiler from hoisting them (their addresses are known early) above
    // the caller's main loop, where their registers would stay live and cost
    // occupancy.
    __device__ __forceinline__ void load(const ConvArgs& a, int32_t g, int lane) {
        if constexpr (kEp) {
            asm volatile("" : "+v"(g));
            const bool vec = ((reinterpret_cast<uintptr_t>(a.ep_scale) |
                               reinterpret_cast<uintptr_t>(a.ep_bias)) & 15) == 0;
#pragma unroll
            for (int q = 0; q < ACC / 4; ++q) {
                const int32_t ob = g * N + M::row(lane, 4 * q);
                f32x4 sv = {1.f, 1.f, 1.f, 1.f}, bv = {0.f, 0.f, 0.f, 0.f};
                if (vec && ob + 4 <= a.n) {
                    if (a.ep_scale) sv = *reinterpret_cast<const f32x4*>(a.ep_scale + ob);
                    if (a.ep_bias) bv = *reinterpret_cast<const f32x4*>(a.ep_bias + ob);
                } else {
#pragma unroll
                    for (int j = 0; j < 4; ++j) {
                        if (ob + j >= a.n) continue;
                        if (a.ep_scale) sv[j] = a.ep_scale[ob + j];
                        if (a.ep_bias) bv[j] = a.ep_bias[ob + j];
                    }
                }
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    s[4 * q + j] = sv[j];
                    b[4 * q + j] = bv[j];
                }
            }
        }
    }
    // From full scale and bias arrays (e.g. staged in LDS) that cover every
    // channel of the layer's col-groups, 16-byte aligned.
    // Only the run of rows 4q .. 4q + 3 (a store loop that reads each run
    // just before its rows keeps fewer registers live).
    __device__ __forceinline__ void load_staged_run(const float* sc, const float* bi, int32_t g, int lane,
                                                    int q) {
        if constexpr (kEp) {
            const int32_t ob = g * N + M::row(lane, 4 * q);
            const f32x4 sv = *reinterpret_cast<const f32x4*>(sc + ob);
            const f32x4 bv = *reinterpret_cast<const f32x4*>(bi + ob);
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                s[4 * q + j] = sv[j];
                b[4 * q + j] = bv[j];
            }
        }
    }
    __device__ __forceinline__ void load_staged(const float* sc, const float* bi, int32_t g, int lane) {
#pragma unroll
        for (int q = 0; q < ACC / 4; ++q) load_staged_run(sc, bi, g, lane, q);
    }
    // act(scale * v + bias) for row r.
    __device__ __forceinline__ float apply(const ConvArgs& a, int r, float v) const {
        if constexpr (!kEp) return v;
        else return epilogue_act(a, fmaf(v, s[r], b[r]));
    }
};

// Waits until at most K vector-memory instructions of this wave are
// outstanding (gfx9 s_waitcnt encoding; the other counters are left free).
template <int K>
__device__ __forceinline__ void wait_vmem() {
    static_assert(K >= 0 && K < 64, "vmcnt range");
    __builtin_amdgcn_s_waitcnt((K & 15) | ((K >> 4) << 14) | (7 << 4) | (15 << 8));
}

// Waits until this wave's LDS (and scalar-memory) operations are complete.
__device__ __forceinline__ void wait_lgkm() {
    __builtin_amdgcn_s_waitcnt(15 | (3 << 14) | (7 << 4) | (0 << 8));
}

template <int NB> struct VecF;
template <> struct VecF<1> { typedef float T; };
template <> struct VecF<2> { typedef float T __attribute__((ext_vector_type(2))); };
template <> struct VecF<4> { typedef f32x4 T; };

// Element e of a lane's NB consecutive pixels.
template <int NB>
__device__ __forceinline__ float vec_el(const typename VecF<NB>::T& v, int e) {
    if constexpr (NB == 1) return v;
    else return v[e];
}
template <int NB>
__device__ __forceinline__ void vec_set(typename VecF<NB>::T& v, int e, float f) {
    if constexpr (NB == 1) v = f;
    else v[e] = f;
}

}  // namespace onexn
