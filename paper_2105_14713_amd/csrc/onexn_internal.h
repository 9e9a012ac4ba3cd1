// Internal helpers shared by the translation units of libonexn.so.
#pragma once

#include <cstdarg>
#include <cstdint>

#include "onexn.h"

namespace onexn {

// Records a printf-style message for onexn_last_error() and returns `s`.
onexn_status fail(onexn_status s, const char* fmt, ...) __attribute__((format(printf, 2, 3)));

// Clears the calling thread's last error message.
void clear_error();

// Kernel-choice and launch-shape overrides, set through onexn_set_tuning()
// (for tests that must reach a particular kernel variant and for A/B timing).
// Each is process-wide; kTuneAuto (the initial value) leaves the choice to
// the dispatch rules.
enum Tune : int {
    kTuneKernel,       // 1: the generic gather kernels for every layer
    kTunePwKernel,     // 1x1 fp32 N = 16/32: 1 resident tile, 3 register-operand
    kTunePwWgs,        // resident-tile 1x1: workgroups
    kTunePwbGp,        // register-gathered bf16: pixels per granule (4, 8)
    kTunePwbRp,        // register-gathered bf16: steps in flight
    kTuneDirectKdb,    // register-operand 1x1: MFMA steps per batch (2, 8)
    kTuneDirectTile,   // register-operand 1x1: tile shape 1-4
    kTuneFmaTpw,       // 1x1 FMA: pixel tiles per workgroup
    kTuneFmaNoV4,      // 1x1 FMA: 1 disables 16-byte pixel quads
    kTuneFmaTile,      // 1x1 FMA: tile shape 1-5
    kTuneKxkSplit,     // k x k: workgroups per CU of the balanced split (0: none)
    kTuneKxkTp,        // k x k: tile capacity in pixels (128, 256)
    kTunePwbKernel,    // bf16 1x1 N = 32: 1 register-gathered, 2 LDS-staged
    kTunePwbWgs,       // LDS-staged bf16 1x1: workgroups
    kTuneKxfSplit,     // 3x3 FMA (N <= 8): waves per unit (1, 4)
    kTuneNhwcTile,     // NHWC 1x1: column blocks per tile
    kTuneBwdKernel,    // backward: 1 the general kernels for every layer
    kTuneBwdSplit,     // 1x1 weight gradient: pixel ranges per tile
    kTuneCount
};
constexpr int32_t kTuneAuto = -1;

// Current value of an override (kTuneAuto when not set).
int32_t tuning(Tune k);

}  // namespace onexn
