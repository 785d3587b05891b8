// Internal interface of the tensor-commitment kernels (commit.hip) for the C
// ABI layer (api.cpp).
#pragma once

#include <hip/hip_runtime_api.h>
#include <stdint.h>

namespace repops {

uint64_t commit_leaves(uint64_t nbytes, uint32_t chunk);
// 32 bytes per leaf digest plus 32 per digest of the reduced levels (at most
// half as many).
uint64_t commit_workspace_bytes(uint64_t nbytes, uint32_t chunk);
hipError_t launch_commit(const uint8_t* data, uint64_t nbytes, uint32_t chunk, uint8_t* digest,
                         uint32_t* ws, hipStream_t s);

}  // namespace repops
