// Internal declarations shared by the host-side C++ and the device entry points.
#pragma once

#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "../../include/orbitquant.h"

namespace orbit {

constexpr int kMaxDevices = 64;
constexpr int kMaxBits = 6;

// Records a failure for orbit_last_error() and returns its status.
orbit_status fail(orbit_status st, const char* fmt, ...) __attribute__((format(printf, 2, 3)));
void clear_error();

}  // namespace orbit

// Pi_d: permutation (gather), Rademacher signs and block size (Sec. 4.4, Eq. (9)).
struct orbit_plan_s {
    int64_t d = 0;
    int32_t h = 0;
    std::vector<int32_t> perm;  // y_j = x[perm[j]]
    std::vector<int8_t> sign;   // multiplies post-permutation coordinate j
    // Per-device table for the quantizer: meta[j] = (2*perm[j]) | (sign[j] < 0 ? 1u << 31 : 0),
    // i.e. the byte offset of the gathered bf16 element inside a staged row plus the sign bit.
    std::mutex mu;
    uint32_t* dev_meta[orbit::kMaxDevices] = {};
};

// C^(d,b): ascending levels, midpoint thresholds, fp16 image of the levels.
struct orbit_codebook_s {
    int32_t bits = 0;
    int64_t d = 0;
    std::vector<double> levels;
    std::vector<double> thresholds;
    std::vector<uint16_t> lut_f16;
};
