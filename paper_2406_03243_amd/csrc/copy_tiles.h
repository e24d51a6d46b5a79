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
//    issues SPAN 1-KiB loads (64 lanes x 16 bytes, global_load_dwordx4)
//    before its first store, so each lane keeps SPAN x 16 bytes in flight
//    and the wave streams one contiguous span in and out.  SPAN is about a
//    quarter of the tile, so the four wavefronts of a workgroup move one
//    whole tile: measured on MI355X, long per-wave spans beat interleaving
//    the wavefronts over shared 4 KiB rows by 5-16% (128 KiB tiles: 32 KiB
//    spans, 6.1-6.3 against 5.3-5.4 TB/s).  Launches with few items (a
//    final stage) use 2 KiB spans so their tiles spread over more CUs.
//  * Wave items run pair-major (all spans of all layers of one block pair,
//    then the next pair); one workgroup per four items unless the grid is
//    capped, in which case resident workgroups walk the items.
//  * The block ids of an item are wavefront-uniform; they and the per-layer
//    base addresses are read with scalar loads, so the only vector memory
//    traffic is the copy itself.
//  * A stage's (src, dst) ids travel inside the kernel arguments (up to
//    kInlinePairs per launch), so a stage needs no mapping upload and no
//    device allocation: the short final stage costs one launch.
//  * No LDS: both sides have the same byte layout inside a tile, so data
//    goes straight from the load registers to the store.  No MFMA: a copy
//    has no arithmetic.
//  * Loads and stores are non-temporal: every byte is touched once, and
//    streaming it past the caches leaves them to the decode work running
//    beside the migration (measured 2-4% faster than cached accesses).
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
    int32_t src_ids[kInlinePairs];
    int32_t dst_ids[kInlinePairs];
};

constexpr uint32_t kWaveRow = 64 * 16;         // one wavefront load: 1 KiB

template <int SRC, int DST, bool INLINE_IDS, int SPAN>
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
            const int32_t id = INLINE_IDS ? a.src_ids[i] : id_entry(a.src_ids_dev, i);
            s = reinterpret_cast<const uint8_t *>(table_entry(a.src_tab, kv * a.num_layers + layer)) +
                static_cast<uint64_t>(uniform(static_cast<uint32_t>(id))) * a.tile_bytes;
        } else {
            s = a.src_lin + (static_cast<uint64_t>(plane) * a.lin_pairs + a.lin_first + i) * a.tile_bytes;
        }
        if (DST == kPool) {
            const int32_t id = INLINE_IDS ? a.dst_ids[i] : id_entry(a.dst_ids_dev, i);
            d = reinterpret_cast<uint8_t *>(table_entry(a.dst_tab, kv * a.num_layers + layer)) +
                static_cast<uint64_t>(uniform(static_cast<uint32_t>(id))) * a.tile_bytes;
        } else {
            d = a.dst_lin + (static_cast<uint64_t>(plane) * a.lin_pairs + a.lin_first + i) * a.tile_bytes;
        }

        const uint32_t first = span * SPAN * kWaveRow + lane_off;
        u32x4 r[SPAN];
        if ((span + 1) * SPAN * kWaveRow <= a.tile_bytes) {
            // Common case: a whole span, no predication at all.
#pragma unroll
            for (int u = 0; u < SPAN; ++u)
                r[u] = load16(s + first + u * kWaveRow);
#pragma unroll
            for (int u = 0; u < SPAN; ++u)
                store16(d + first + u * kWaveRow, r[u]);
        } else {
            // The tile's last span is short: a lane predicate per 1 KiB row.
#pragma unroll
            for (int u = 0; u < SPAN; ++u)
                if (first + u * kWaveRow < a.tile_bytes)
                    r[u] = load16(s + first + u * kWaveRow);
#pragma unroll
            for (int u = 0; u < SPAN; ++u)
                if (first + u * kWaveRow < a.tile_bytes)
                    store16(d + first + u * kWaveRow, r[u]);
        }
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

template <int SRC, int DST, bool INLINE_IDS>
const void *copy_kernel_span(int span)
{
    switch (span) {
    case 32:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, INLINE_IDS, 32>);
    case 16:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, INLINE_IDS, 16>);
    case 8:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, INLINE_IDS, 8>);
    case 4:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, INLINE_IDS, 4>);
    default:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, INLINE_IDS, 2>);
    }
}

template <int SRC, int DST>
const void *copy_kernel(bool ids_on_device, int span)
{
    return ids_on_device ? copy_kernel_span<SRC, DST, false>(span) : copy_kernel_span<SRC, DST, true>(span);
}

// A launch with fewer wave items than this per CU is small (a final stage).
constexpr uint32_t kBulkWaveItemsPerCU = 16;

// max_workgroups > 0 caps the grid: fewer, resident workgroups walk the
// items, leaving the rest of the chip (and of HBM) to other work.
template <int SRC, int DST>
int launch_copy(CopyArgs a, const int32_t *src_ids, const int32_t *dst_ids, int64_t n,
                bool ids_on_device, hipStream_t stream, uint32_t max_workgroups = 0)
{
    int span = bulk_span(a.tile_bytes);
    uint32_t spt = (a.tile_bytes + span * kWaveRow - 1) / (span * kWaveRow);
    const uint64_t pairs_first_launch =
        std::min<int64_t>(n, ids_on_device ? n : static_cast<int64_t>(kInlinePairs));
    if (pairs_first_launch * 2ull * a.num_layers * spt < kBulkWaveItemsPerCU * compute_units()) {
        span = 2;
        spt = (a.tile_bytes + span * kWaveRow - 1) / (span * kWaveRow);
    }
    a.spans_per_tile = spt;
    const uint64_t items_per_pair = 2ull * a.num_layers * spt;
    uint64_t per_launch = std::min<uint64_t>(0x7fffffffull / items_per_pair,
                                             ids_on_device ? UINT64_MAX : kInlinePairs);
    if (per_launch == 0)
        return LLMIG_EINVAL;
    a.lin_pairs = static_cast<uint32_t>(n);
    a.planes = 2u * a.num_layers;
    const void *fn = copy_kernel<SRC, DST>(ids_on_device, span);
    for (int64_t first = 0; first < n; first += static_cast<int64_t>(per_launch)) {
        const uint32_t m = static_cast<uint32_t>(std::min<int64_t>(n - first, per_launch));
        a.pairs = m;
        a.lin_first = static_cast<uint32_t>(first);
        a.items = static_cast<uint32_t>(m * items_per_pair);
        if (ids_on_device) {
            a.src_ids_dev = src_ids ? src_ids + first : nullptr;
            a.dst_ids_dev = dst_ids ? dst_ids + first : nullptr;
        } else {
            if (src_ids)
                std::memcpy(a.src_ids, src_ids + first, m * sizeof(int32_t));
            if (dst_ids)
                std::memcpy(a.dst_ids, dst_ids + first, m * sizeof(int32_t));
        }
        void *args[] = {&a};
        uint32_t grid = (a.items + kThreads / 64 - 1) / (kThreads / 64);
        if (max_workgroups > 0)
            grid = std::min(grid, max_workgroups);
        hipError_t e = hipLaunchKernel(fn, dim3(grid), dim3(kThreads), args, 0, stream);
        if (e != hipSuccess)
            return hip_error(e);
    }
    return LLMIG_OK;
}

} // namespace
