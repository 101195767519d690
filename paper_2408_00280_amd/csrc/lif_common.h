// Constants and the kernel-argument struct shared by the host and device code of the
// fused LIF library.
#pragma once
#include <climits>
#include <cstdint>

#include "snn_lif.h"

namespace snnlif {

constexpr int kBlock = 256;  // 4 wave64 per workgroup
constexpr int kWave = 64;

constexpr int64_t kMaxT = INT32_MAX;
constexpr int64_t kMaxN = int64_t(1) << 31;
constexpr int64_t kMaxTN = int64_t(1) << 44;

// Kernel-side hyper-parameters.
struct LifK {
    float k;      // decay k_tau
    float th;     // V_th
    float rest;   // V_rest
    float alpha;  // surrogate sharpness
    float c_exp;  // -alpha * log2(e): e^{-alpha |u|} = 2^{c_exp |u|}
    float kth;    // k * V_th (soft-reset backward)
};

}  // namespace snnlif
