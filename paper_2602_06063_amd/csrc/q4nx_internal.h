// Internal declarations shared by the host packer and the device launchers.
#pragma once

#include <cstddef>
#include <cstdint>
#include <string>

#include "../../include/q4nx.h"

namespace q4nx {

// Q4NX block geometry (Sec. 3.1.1): 32 output rows x 256 input columns,
// groups of 32 consecutive columns of one row.
constexpr int kBlockRows = 32;
constexpr int kBlockCols = 256;
constexpr int kGroup = 32;
constexpr int kGroupsPerRow = kBlockCols / kGroup;             // 8
constexpr int kCodeBytes = kBlockRows * kBlockCols / 2;        // 4096
constexpr int kScaleBytes = kBlockRows * kGroupsPerRow * 2;    // 512
constexpr int kBlockBytes = kCodeBytes + 2 * kScaleBytes;      // 5120

// MXFP4 variant of the block (OCP MX v1.0 element and scale encodings): the
// same 32 x 256 codes as FP4 E2M1 values, one E8M0 scale byte per group,
// no offset.
constexpr int kMxScaleBytes = kBlockRows * kGroupsPerRow;      // 256
constexpr int kMxBlockBytes = kCodeBytes + kMxScaleBytes;      // 4352
constexpr int kMxExpMin = 27, kMxExpMax = 227;                 // accepted scales 2^-100 .. 2^100
constexpr uint8_t kMxPadScale = 127;                           // scale 1 in padded groups

inline int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }

// Records a detail message for q4nx_last_error() and returns `st`.
q4nx_status fail(q4nx_status st, const std::string& msg);
void clear_error();

// Shape check shared by every call: N, K in (0, Q4NX_MAX_DIM], K % 32 == 0.
q4nx_status check_shape(int64_t N, int64_t K, const char* fn);

inline bool aligned(const void* p, size_t a) {
  return (reinterpret_cast<uintptr_t>(p) % a) == 0;
}

}  // namespace q4nx
