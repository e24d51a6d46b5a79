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
// Grid cap of the grid-stride kernels (copy, conversion, token writes): a
// dispatch counts its work-items in 32 bits, and past a few million
// workgroups more of them would only wait in the queue.
constexpr uint32_t kMaxGridWorkgroups = 1u << 22;

// Where a launch finds its block ids.
enum Ids {
    kIdsDevice = 0, // device arrays src_ids_dev / dst_ids_dev
    kIds32 = 1,     // ids[i] (source) and ids[kInlinePairs + i] (destination)
    kIds16 = 2,     // ids[i] = source | destination << 16 (pool to pool, ids below 65536)
};

typedef unsigned int u32x4 __attribute__((ext_vector_type(4)));

thread_local int g_last_hip_error = 0;

int hip_error(hipError_t e)
{
    g_last_hip_error = static_cast<int>(e);
    return LLMIG_EHIP;
}

// Optional events around a call's kernels: start is recorded on the stream
// right before the first kernel is launched and stop right after the last
// one, so their interval holds the kernels (and one launch's latency) but
// none of the host work that planned them.
struct LaunchEvents {
    hipEvent_t start = nullptr;
    hipEvent_t stop = nullptr;
};

// Launch k of `launches` of one call.
hipError_t launch_kernel(const void *fn, dim3 grid, dim3 block, void **args, hipStream_t stream,
                         const LaunchEvents &ev, int64_t k, int64_t launches)
{
    hipError_t e = hipSuccess;
    if (k == 0 && ev.start)
        e = hipEventRecord(ev.start, stream);
    if (e == hipSuccess)
        e = hipLaunchKernel(fn, grid, block, args, 0, stream);
    if (e == hipSuccess && k == launches - 1 && ev.stop)
        e = hipEventRecord(ev.stop, stream);
    return e;
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

// Raw buffer accesses (the migration copy): a resource over one tile, and
// 16-byte loads and stores with explicit cache-policy bits.  On gfx950 the
// policy bits are sc0 = 1, nt = 2, sc1 = 16 (sc1 alone selects device
// scope).  Loads stream (nt); stores also carry sc1, measured 0.5-1.3%
// faster on the LLaMA-7B stage than nt alone (plain or sc0 stores were
// 2-10% slower).  An access whose offset lies past the resource's
// num_records is out of range: a load returns zeros and a store is dropped.
constexpr int kBufferWord3 = 0x00020000;     // descriptor word 3 for raw 32-bit accesses on gfx9
constexpr int kStreamLoad = 2;               // nt
constexpr int kStreamStore = 16 | 2;         // sc1 nt

__device__ __forceinline__ __amdgpu_buffer_rsrc_t tile_rsrc(const uint8_t *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<uint8_t *>(base), 0, static_cast<int>(bytes), kBufferWord3);
}

__device__ __forceinline__ u32x4 buffer_load16(__amdgpu_buffer_rsrc_t r, uint32_t off)
{
    return __builtin_bit_cast(u32x4, __builtin_amdgcn_raw_buffer_load_b128(r, off, 0, kStreamLoad));
}

__device__ __forceinline__ void buffer_store16(__amdgpu_buffer_rsrc_t r, uint32_t off, u32x4 v)
{
    __builtin_amdgcn_raw_buffer_store_b128(v, r, off, 0, kStreamStore);
}

} // namespace
