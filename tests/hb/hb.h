// Internal interface of the happens-before checker (test infrastructure).
#pragma once
#include <cstdint>
#include <utility>
#include <vector>

#include "hip/hip_runtime.h"

// [begin, end) byte ranges of one operand
using HbRanges = std::vector<std::pair<uint64_t, uint64_t>>;

void* hb_new_stream(const char* name);
// Records one operation (kernel or copy) on `stream` with the byte ranges it
// reads and writes; reports races against earlier operations.
void hb_op(hipStream_t stream, const char* name, const HbRanges& reads, const HbRanges& writes);
