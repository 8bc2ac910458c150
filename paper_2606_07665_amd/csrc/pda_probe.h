// Internal interface of the streaming-read reference kernel (not part of the public ABI).
#pragma once
#include <hip/hip_runtime.h>
#include <cstdint>

namespace pda {

constexpr int kStreamThreads = 256;  // 4 waves per workgroup

// Reads `bytes` of device memory at `buf` once (16-byte non-temporal buffer
// loads, `unroll` of 4, 8 or 16 in flight per wave) with `blocks` workgroups.
hipError_t launch_stream_read(const void* buf, int64_t bytes, uint32_t* sink, int unroll, int blocks,
                              hipStream_t st);

}  // namespace pda
