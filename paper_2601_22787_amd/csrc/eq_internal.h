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
// Device scratch per layer.  Version 1: slot table (kMaxSlots x 2 u32), then
// the value table of the base format's codes as fp32 and as BF16 (256 u32
// each).  Version 2: kBuckets entries of 16 bytes (state update and the
// phrase's BF16 values), then kBuckets u32 (the phrase's codes).
constexpr size_t kLutBytesV1 = (2 * kMaxSlots + 512) * sizeof(uint32_t);
constexpr uint32_t kBuckets = 4096;  // version 2: slot >> 4 at the finest resolution
constexpr size_t kLutBytesV2 = size_t(kBuckets) * 20;
constexpr size_t kLutBytes = kLutBytesV1 > kLutBytesV2 ? kLutBytesV1 : kLutBytesV2;

}  // namespace eq_detail

