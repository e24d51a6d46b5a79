// The tile copy behind llmig_stage, llmig_pack and llmig_unpack, with its
// launch configuration.  Part of the single translation unit built from
// llmig.hip.
//
// What it computes (Llumnix §4.2, §5 "Block fusion"): for every pair i, layer
// l and K/V, the tile_bytes of tile (l, kv) of block src[i] land in tile
// (l, kv) of block dst[i] (pool to pool), or in slot ((l * 2 + kv) * n + i)
// of a contiguous staging buffer (pack), or the reverse (unpack).
//
// Kernel design (CDNA4, wave64):
//  * The work of a call is a list of tiles, one per (pair, layer, K/V); a
//    tile is tile_bytes contiguous bytes on both sides.  A tile is cut into
//    SPAN-KiB spans and each span is one wavefront's work item: the wave
//    issues SPAN 1-KiB loads (64 lanes x 16 bytes) before its first store,
//    so each lane keeps SPAN x 16 bytes in flight and the wave streams one
//    contiguous span in and out.  SPAN is about a quarter of the tile, so
//    the four wavefronts of a workgroup move one whole tile: measured on
//    MI355X, long per-wave spans beat interleaving the wavefronts over
//    shared 4 KiB rows by 5-16% (128 KiB tiles: 32 KiB spans, 6.1-6.3
//    against 5.3-5.4 TB/s).  Launches with few items (a final stage) use
//    2 KiB spans so their tiles spread over more CUs.
//  * Every span runs the same unpredicated sequence of SPAN loads and SPAN
//    stores.  A row of the span that lies past the end of the tile (the
//    last span of a tile that is not a whole number of spans, such as the
//    4 KiB tail of a 52 KiB tile cut into 16 KiB spans) gets an offset past
//    the buffer resource's range, so the hardware's range check returns
//    zeros for its load and drops its store.  Predicating those rows on
//    the lane mask instead makes the compiler wait for every earlier memory
//    operation before each store of the span (it cannot count them across
//    the branches), which serialised the tail's stores.  Measured on 52 KiB
//    tiles in one process, alternating: predicated rows 0.62 of HBM peak; a
//    separate, range-checked code path for short spans only 0.67-0.68; one
//    sequence for every span 0.72-0.75 (128 and 32 KiB tiles gained about
//    1%).
//  * Wave items run pair-major (all spans of all layers of one block pair,
//    then the next pair); one workgroup per four items unless the grid is
//    capped, in which case resident workgroups walk the items.
//  * The block ids of an item are wavefront-uniform; they and the per-layer
//    base addresses are read with scalar loads, so the only vector memory
//    traffic is the copy itself.
//  * A stage's (src, dst) ids travel inside the kernel arguments, so a
//    stage needs no mapping upload and no device allocation: the short
//    final stage costs one launch.  When every id of a pool-to-pool stage
//    fits in 16 bits (pools of up to 65536 blocks) a pair takes one 32-bit
//    word and a launch carries 2 * kInlinePairs pairs (the whole 512-pair
//    LLaMA-7B stage in one launch, measured 0.4-0.7% faster than two);
//    otherwise kInlinePairs pairs of 32-bit ids.
//  * No LDS: both sides have the same byte layout inside a tile, so data
//    goes straight from the load registers to the store.  No MFMA: a copy
//    has no arithmetic.
//  * Loads and stores are raw buffer accesses over one tile with explicit
//    cache policy: non-temporal loads, and stores that are non-temporal
//    with the sc1 scope bit (device scope on gfx950).  Every byte is touched
//    once, and streaming it past the caches leaves them to the decode work
//    beside the migration.
#pragma once

#include <algorithm>
#include <cstring>

#include "common.h"

namespace {

enum Side { kPool = 0, kLinear = 1 };


// Arguments of one copy launch.  Pool sides address tile (l, kv, id) at
// tab[kv * L + l] + id * tile_bytes; linear sides address pair i of plane
// (l, kv) at lin + ((l * 2 + kv) * lin_pairs + lin_first + i) * tile_bytes.
struct CopyArgs {
    const uint64_t *src_tab;
    const uint64_t *dst_tab;
    const uint8_t *src_lin;
    uint8_t *dst_lin;
    const int32_t *src_ids_dev; // device id lists (null when the ids are inline)
    const int32_t *dst_ids_dev;
    uint32_t tile_bytes;
    uint32_t num_layers;
    uint32_t planes;            // 2 * num_layers
    uint32_t pairs;             // pairs in this launch
    uint32_t spans_per_tile;
    uint32_t items;             // wave items: pairs * planes * spans_per_tile
    uint32_t lin_first;         // this launch's first pair within the whole call
    uint32_t lin_pairs;         // pairs in the whole call
    uint32_t ids[2 * kInlinePairs]; // inline ids, laid out as the launch's Ids mode says
};

constexpr uint32_t kWaveRow = 64 * 16;         // one wavefront load: 1 KiB

// Buffer offset of the row starting at byte o of a tile of `bytes` bytes:
// o itself, or kOutOfRange when the row lies past the tile.  Tiles are at
// most 2^31 - 1 bytes, so kOutOfRange plus a lane's offset is always past
// the resource's range: the load returns zeros and the store is dropped.
// A row that is partly inside the tile (a tile that is not a whole number
// of KiB) is cut per lane by the same check.
constexpr uint32_t kOutOfRange = 0x80000000u;

__device__ __forceinline__ uint32_t row_offset(uint32_t o, uint32_t bytes)
{
    return o < bytes ? o : kOutOfRange;
}

template <int IDS>
__device__ __forceinline__ uint32_t src_id(const CopyArgs &a, uint32_t i)
{
    if (IDS == kIds16)
        return a.ids[i] & 0xffffu;
    return IDS == kIds32 ? a.ids[i] : static_cast<uint32_t>(id_entry(a.src_ids_dev, i));
}

template <int IDS>
__device__ __forceinline__ uint32_t dst_id(const CopyArgs &a, uint32_t i)
{
    if (IDS == kIds16)
        return a.ids[i] >> 16;
    return IDS == kIds32 ? a.ids[kInlinePairs + i] : static_cast<uint32_t>(id_entry(a.dst_ids_dev, i));
}

template <int SRC, int DST, int IDS, int SPAN>
__global__ void __launch_bounds__(kThreads) copy_tiles(const CopyArgs a)
{
    const uint32_t lane_off = (threadIdx.x % 64) * 16u;
    const uint32_t waves = gridDim.x * (kThreads / 64);
    for (uint32_t w = blockIdx.x * (kThreads / 64) + threadIdx.x / 64; w < a.items; w += waves) {
        const uint32_t item = uniform(w);
        const uint32_t tile = item / a.spans_per_tile;
        const uint32_t span = item - tile * a.spans_per_tile;
        const uint32_t i = tile / a.planes;
        const uint32_t plane = tile - i * a.planes; // layer * 2 + kv
        const uint32_t layer = plane >> 1, kv = plane & 1u;

        const uint8_t *s;
        uint8_t *d;
        if (SRC == kPool) {
            s = reinterpret_cast<const uint8_t *>(table_entry(a.src_tab, kv * a.num_layers + layer)) +
                static_cast<uint64_t>(uniform(src_id<IDS>(a, i))) * a.tile_bytes;
        } else {
            s = a.src_lin + (static_cast<uint64_t>(plane) * a.lin_pairs + a.lin_first + i) * a.tile_bytes;
        }
        if (DST == kPool) {
            d = reinterpret_cast<uint8_t *>(table_entry(a.dst_tab, kv * a.num_layers + layer)) +
                static_cast<uint64_t>(uniform(dst_id<IDS>(a, i))) * a.tile_bytes;
        } else {
            d = a.dst_lin + (static_cast<uint64_t>(plane) * a.lin_pairs + a.lin_first + i) * a.tile_bytes;
        }

        const __amdgpu_buffer_rsrc_t rs = tile_rsrc(s, a.tile_bytes);
        const __amdgpu_buffer_rsrc_t rd = tile_rsrc(d, a.tile_bytes);
        const uint32_t first = span * SPAN * kWaveRow;
        u32x4 r[SPAN];
#pragma unroll
        for (int u = 0; u < SPAN; ++u)
            r[u] = buffer_load16(rs, row_offset(first + u * kWaveRow, a.tile_bytes) + lane_off);
#pragma unroll
        for (int u = 0; u < SPAN; ++u)
            buffer_store16(rd, row_offset(first + u * kWaveRow, a.tile_bytes) + lane_off, r[u]);
    }
}

uint32_t compute_units()
{
    static const uint32_t cus = [] {
        int dev = 0, n = 256;
        if (hipGetDevice(&dev) != hipSuccess ||
            hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess)
            n = 256;
        return static_cast<uint32_t>(n);
    }();
    return cus;
}

// Span (in 1 KiB rows) for a bulk copy: the power of two nearest above a
// quarter of the tile, between 2 and 32.
int bulk_span(uint32_t tile_bytes)
{
    const uint32_t quarter = (tile_bytes + 4 * kWaveRow - 1) / (4 * kWaveRow);
    int span = 2;
    while (span < 32 && static_cast<uint32_t>(span) < quarter)
        span *= 2;
    return span;
}

template <int SRC, int DST, int IDS>
const void *copy_kernel_span(int span)
{
    switch (span) {
    case 32:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, IDS, 32>);
    case 16:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, IDS, 16>);
    case 8:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, IDS, 8>);
    case 4:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, IDS, 4>);
    default:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, IDS, 2>);
    }
}

template <int SRC, int DST>
const void *copy_kernel(int ids, int span)
{
    if (ids == kIdsDevice)
        return copy_kernel_span<SRC, DST, kIdsDevice>(span);
    if (SRC == kPool && DST == kPool && ids == kIds16)
        return copy_kernel_span<SRC, DST, kIds16>(span);
    return copy_kernel_span<SRC, DST, kIds32>(span);
}

// A launch with fewer wave items than this per CU is small (a final stage).
constexpr uint32_t kBulkWaveItemsPerCU = 16;

// max_workgroups > 0 caps the grid: fewer, resident workgroups walk the
// items, leaving the rest of the chip (and of HBM) to other work.
// ids16: every id of both lists is below 65536 (pool to pool only).
template <int SRC, int DST>
int launch_copy(CopyArgs a, const int32_t *src_ids, const int32_t *dst_ids, int64_t n,
                bool ids_on_device, hipStream_t stream, uint32_t max_workgroups = 0, bool ids16 = false,
                const LaunchEvents &ev = LaunchEvents())
{
    const int ids = ids_on_device ? kIdsDevice : (SRC == kPool && DST == kPool && ids16) ? kIds16 : kIds32;
    const int64_t inline_pairs = ids == kIds16 ? 2 * kInlinePairs : kInlinePairs;
    int span = bulk_span(a.tile_bytes);
    uint32_t spt = (a.tile_bytes + span * kWaveRow - 1) / (span * kWaveRow);
    const uint64_t pairs_first_launch = std::min<int64_t>(n, ids_on_device ? n : inline_pairs);
    if (pairs_first_launch * 2ull * a.num_layers * spt < kBulkWaveItemsPerCU * compute_units()) {
        span = 2;
        spt = (a.tile_bytes + span * kWaveRow - 1) / (span * kWaveRow);
    }
    a.spans_per_tile = spt;
    const uint64_t items_per_pair = 2ull * a.num_layers * spt;
    uint64_t per_launch = std::min<uint64_t>(0x7fffffffull / items_per_pair,
                                             ids_on_device ? UINT64_MAX : static_cast<uint64_t>(inline_pairs));
    if (per_launch == 0)
        return LLMIG_EINVAL;
    a.lin_pairs = static_cast<uint32_t>(n);
    a.planes = 2u * a.num_layers;
    const void *fn = copy_kernel<SRC, DST>(ids, span);
    const int64_t launches = (n + static_cast<int64_t>(per_launch) - 1) / static_cast<int64_t>(per_launch);
    for (int64_t first = 0, k = 0; first < n; first += static_cast<int64_t>(per_launch), ++k) {
        const uint32_t m = static_cast<uint32_t>(std::min<int64_t>(n - first, per_launch));
        a.pairs = m;
        a.lin_first = static_cast<uint32_t>(first);
        a.items = static_cast<uint32_t>(m * items_per_pair);
        if (ids == kIdsDevice) {
            a.src_ids_dev = src_ids ? src_ids + first : nullptr;
            a.dst_ids_dev = dst_ids ? dst_ids + first : nullptr;
        } else if (ids == kIds16) {
            for (uint32_t k = 0; k < m; ++k)
                a.ids[k] = static_cast<uint32_t>(src_ids[first + k]) | (static_cast<uint32_t>(dst_ids[first + k]) << 16);
        } else {
            if (src_ids)
                std::memcpy(a.ids, src_ids + first, m * sizeof(int32_t));
            if (dst_ids)
                std::memcpy(a.ids + kInlinePairs, dst_ids + first, m * sizeof(int32_t));
        }
        void *args[] = {&a};
        uint32_t grid = std::min((a.items + kThreads / 64 - 1) / (kThreads / 64), kMaxGridWorkgroups);
        if (max_workgroups > 0)
            grid = std::min(grid, max_workgroups);
        hipError_t e = launch_kernel(fn, dim3(grid), dim3(kThreads), args, stream, ev, k, launches);
        if (e != hipSuccess)
            return hip_error(e);
    }
    return LLMIG_OK;
}

} // namespace
