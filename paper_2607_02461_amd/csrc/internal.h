// Internal declarations shared by the host-side C++ and the device entry points.
#pragma once

#include <cstdint>
#include <mutex>
#include <string>
#include <vector>

#include "orbitquant.h"

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
    bool identity = false;      // perm[j] == j for every j (Block-RHT, full-dimension rotations)
    // Per-device tables for the quantizer (gather offsets and sign masks), set up at creation or by
    // rpbh_plan_upload, see plan_upload_dev().
    std::mutex mu;
    uint32_t* dev_meta[orbit::kMaxDevices] = {};
};

// Encoder lookup table over the normalized coordinate u in [-kEncRange, kEncRange].  In cell
// coordinates t = u / w + C, with w below the smallest threshold spacing and C an integer, cell c
// covers t in [c - 0.5, c + 0.5) (the kernel rounds t to the nearest integer), so a cell holds at
// most one threshold.  The code is round-to-nearest-even(0.5*(t - C) + bias[cell]) with
//     bias = base + 0.5 - 0.5*tau/w      in a cell holding threshold tau (code base or base+1),
//     bias = base - 0.5*(c - C)          in a cell without one (the value stays within 0.25 of base),
// where base is the number of thresholds below the cell.
constexpr double kEncRange = 1.001;  // |u| <= 1 up to rounding
struct EncTable {
    float inv_w = 0.f;   // 1 / w
    float center = 0.f;  // C, the cell of u = 0 (an integer)
    int32_t ncell = 0;
    std::vector<float> bias;
};

// C^(d,b): ascending levels, midpoint thresholds, bf16 image of the levels (the GEMM's operands).
struct orbit_codebook_s {
    int32_t bits = 0;
    int64_t d = 0;
    std::vector<double> levels;
    std::vector<double> thresholds;
    std::vector<uint16_t> lut_bf16;
    EncTable enc;
    std::mutex mu;
    float* dev_enc[orbit::kMaxDevices] = {};
};

namespace orbit {
void build_enc_table(orbit_codebook_s* c);
// Set-up of a new handle (exactly one of p, c non-null): copies its device tables to the current
// device when a HIP device is visible; a machine without one keeps host-only handles.
orbit_status upload_on_create(orbit_plan_s* p, orbit_codebook_s* c);
}
