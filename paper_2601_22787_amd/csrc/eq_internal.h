// Internal constants shared by the host and device parts of libeq.
#pragma once
#include <cstddef>
#include <cstdint>

namespace eq_detail {

constexpr uint32_t kMaxSlots = 4096;    // 2^P for P <= 12
constexpr uint32_t kStateLow = 1u << 16;
constexpr uint32_t kMinProbBits = 8;   // x >> P must fit a 24-bit multiply
constexpr uint32_t kFmtE4M3 = 1;       // base formats (container header)
constexpr uint32_t kFmtInt8 = 2;
// Device scratch per layer: slot table (kMaxSlots x 2 u32), then the value
// table of the base format's codes as fp32 and as BF16 (256 u32 each).
constexpr size_t kLutBytes = (2 * kMaxSlots + 512) * sizeof(uint32_t);

}  // namespace eq_detail
