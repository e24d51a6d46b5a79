// Shared definitions of the llmig kernels: launch geometry, the 16-byte
// word type, address-space helpers and the library's HIP error record.
// Part of the single translation unit built from llmig.hip.
#pragma once

#include <hip/hip_runtime.h>

#include <cstdint>

#include "llmig.h"

namespace {

constexpr int kThreads = 256;                 // 4 wavefronts of 64 lanes
constexpr uint32_t kRowBytes = kThreads * 16; // one 16-byte word per lane of a workgroup
constexpr int kInlinePairs = 256;             // ids carried in the kernel arguments per launch

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

thread_local int g_last_hip_error = 0;

int hip_error(hipError_t e)
{
    g_last_hip_error = static_cast<int>(e);
    return LLMIG_EHIP;
}

// Address spaces: global for the copied bytes (global_load/global_store
// instead of flat), constant for the small read-only tables so uniform
// reads of them become scalar loads.
#define LLMIG_GLOBAL __attribute__((address_space(1)))
#define LLMIG_CONSTANT __attribute__((address_space(4)))

__device__ __forceinline__ uint32_t uniform(uint32_t x)
{
    return __builtin_amdgcn_readfirstlane(x);
}

__device__ __forceinline__ uint64_t table_entry(const uint64_t *tab, uint32_t k)
{
    return ((const LLMIG_CONSTANT uint64_t *)tab)[k]; // address-space cast
}

__device__ __forceinline__ int32_t id_entry(const int32_t *ids, uint32_t k)
{
    return ((const LLMIG_CONSTANT int32_t *)ids)[k];
}

__device__ __forceinline__ u32x4 load16(const uint8_t *p)
{
    return __builtin_nontemporal_load((const LLMIG_GLOBAL u32x4 *)p);
}

__device__ __forceinline__ void store16(uint8_t *p, u32x4 v)
{
    __builtin_nontemporal_store(v, (LLMIG_GLOBAL u32x4 *)p);
}

} // namespace
