// probe.hpp -- launcher of the streaming-read probe (probe.hip; internal).
#pragma once

#include <stdint.h>

#include <hip/hip_runtime.h>

namespace dustin {

hipError_t launch_read_probe(const void* data, uint64_t bytes, uint32_t* sums, int blocks, hipStream_t stream);

}  // namespace dustin
