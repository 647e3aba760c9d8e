// pdssm_io.h -- element formats of the per-step rows D, b, c and of the
// gradient rows dD, db, dc (host and device code).
#pragma once

namespace pdssm {

constexpr int kIoC64 = 0;   // complex64: fp32 (re, im) pairs, 8 bytes
constexpr int kIoBf16 = 1;  // bf16 (re, im) pairs, 4 bytes (App. E, bf16 inputs)
constexpr int kIoReal = 2;  // real fp32, 4 bytes: the real-valued model; imaginary parts are 0

}  // namespace pdssm
