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
