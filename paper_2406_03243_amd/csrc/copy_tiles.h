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
//    rows of 4 KiB (256 lanes x 16 B), and a workgroup item is a chunk of up
//    to ROWS rows of one tile: each lane issues all of its 16-byte loads
//    (global_load_dwordx4) before its first store, so every lane keeps
//    ROWS x 16 B in flight and each wavefront instruction moves 1 KiB of
//    contiguous, fully coalesced memory.  Bulk copies use 8- or 16-row
//    chunks; small copies (a final stage) use 2-row chunks to spread over
//    more CUs.
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
//  * Items run pair-major (all layers of one block pair, then the next
//    pair), one workgroup per item.
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
    uint32_t chunks_per_tile;
    uint32_t rows_per_chunk;    // <= ROWS of the kernel
    uint32_t items;             // pairs * 2 * num_layers * chunks_per_tile
    uint32_t lin_first;         // this launch's first pair within the whole call
    uint32_t lin_pairs;         // pairs in the whole call
    int32_t src_ids[kInlinePairs];
    int32_t dst_ids[kInlinePairs];
};

template <int SRC, int DST, bool INLINE_IDS, int ROWS>
__global__ void __launch_bounds__(kThreads) copy_tiles(const CopyArgs a)
{
    const uint32_t lane_off = threadIdx.x * 16u;
    const uint32_t full_rows = a.tile_bytes / kRowBytes; // complete 4 KiB rows of a tile
    for (uint32_t item = blockIdx.x; item < a.items; item += gridDim.x) {
        // Items run pair-major: consecutive workgroups take the chunks of one
        // block pair across all layers and K/V, so the memory they touch at
        // a time is spread over many layer tensors.
        const uint32_t tile = item / a.chunks_per_tile;
        const uint32_t chunk = item - tile * a.chunks_per_tile;
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

        const uint32_t row0 = chunk * a.rows_per_chunk;
        const uint32_t first = row0 * kRowBytes + lane_off;
        // Rows of this chunk that every lane copies whole (wavefront-uniform).
        const uint32_t whole = full_rows > row0 ? min(a.rows_per_chunk, full_rows - row0) : 0u;
        u32x4 r[ROWS];
        if (whole == ROWS) {
            // Common case: ROWS complete rows, no predication at all.
#pragma unroll
            for (int u = 0; u < ROWS; ++u)
                r[u] = load16(s + first + u * kRowBytes);
#pragma unroll
            for (int u = 0; u < ROWS; ++u)
                store16(d + first + u * kRowBytes, r[u]);
        } else {
            // Fewer rows: uniform branches for the whole rows, a lane
            // predicate only for a final partial row of the tile.
#pragma unroll
            for (int u = 0; u < ROWS; ++u)
                if (u < static_cast<int>(whole))
                    r[u] = load16(s + first + u * kRowBytes);
#pragma unroll
            for (int u = 0; u < ROWS; ++u)
                if (u < static_cast<int>(whole))
                    store16(d + first + u * kRowBytes, r[u]);
            const uint32_t tail = first + whole * kRowBytes;
            if (whole < a.rows_per_chunk && row0 + whole == full_rows && tail < a.tile_bytes)
                store16(d + tail, load16(s + tail));
        }
    }
}

// Row split of one tile: rows of kRowBytes, chunks of at most max_rows
// rows, balanced so every chunk of a tile carries nearly the same number.
void split_tile(uint32_t tile_bytes, uint32_t max_rows, uint32_t *chunks, uint32_t *rows_per_chunk)
{
    const uint32_t rows = (tile_bytes + kRowBytes - 1) / kRowBytes;
    const uint32_t c = (rows + max_rows - 1) / max_rows;
    *chunks = c;
    *rows_per_chunk = (rows + c - 1) / c;
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

// One workgroup per item: measured on MI355X, letting the dispatcher hand
// out items beats a resident grid walking them (the loop in the kernels
// stays, so a capped grid remains correct).
uint32_t grid_for(uint32_t items)
{
    return items;
}

template <int SRC, int DST, bool INLINE_IDS>
const void *copy_kernel_rows(int rows)
{
    switch (rows) {
    case kWideRows:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, INLINE_IDS, kWideRows>);
    case kBulkRows:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, INLINE_IDS, kBulkRows>);
    default:
        return reinterpret_cast<const void *>(&copy_tiles<SRC, DST, INLINE_IDS, kSmallRows>);
    }
}

template <int SRC, int DST>
const void *copy_kernel(bool ids_on_device, int rows)
{
    return ids_on_device ? copy_kernel_rows<SRC, DST, false>(rows) : copy_kernel_rows<SRC, DST, true>(rows);
}

// max_workgroups > 0 caps the grid: fewer, resident workgroups walk the
// items, leaving the rest of the chip (and of HBM) to other work.
template <int SRC, int DST>
int launch_copy(CopyArgs a, const int32_t *src_ids, const int32_t *dst_ids, int64_t n,
                bool ids_on_device, hipStream_t stream, uint32_t max_workgroups = 0)
{
    // Bulk copies take chunks of kBulkRows rows (most bytes in flight per
    // lane); small ones, such as a final stage, take kSmallRows-row chunks so
    // their few tiles spread over more CUs and finish sooner.
    // Tiles of 32 rows or more take 16-row chunks (measured ~1% faster on
    // 128 KiB tiles than 8-row ones).
    uint32_t chunks = 0, rpc = 0;
    const uint32_t tile_rows = (a.tile_bytes + kRowBytes - 1) / kRowBytes;
    int rows = tile_rows >= 2u * kWideRows ? kWideRows : kBulkRows;
    split_tile(a.tile_bytes, rows, &chunks, &rpc);
    const uint64_t pairs_first_launch =
        std::min<int64_t>(n, ids_on_device ? n : static_cast<int64_t>(kInlinePairs));
    const bool bulk = pairs_first_launch * 2ull * a.num_layers * chunks >= kBulkItemsPerCU * compute_units();
    if (!bulk) {
        rows = kSmallRows;
        split_tile(a.tile_bytes, rows, &chunks, &rpc);
    }
    a.chunks_per_tile = chunks;
    a.rows_per_chunk = rpc;
    const uint64_t items_per_pair = 2ull * a.num_layers * a.chunks_per_tile;
    uint64_t per_launch = ids_on_device ? (0x7fffffffull / items_per_pair) : kInlinePairs;
    if (per_launch == 0)
        return LLMIG_EINVAL;
    a.lin_pairs = static_cast<uint32_t>(n);
    a.planes = 2u * a.num_layers;
    const void *fn = copy_kernel<SRC, DST>(ids_on_device, rows);
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
        uint32_t grid = grid_for(a.items);
        if (max_workgroups > 0)
            grid = std::min(grid, max_workgroups);
        hipError_t e = hipLaunchKernel(fn, dim3(grid), dim3(kThreads), args, 0, stream);
        if (e != hipSuccess)
            return hip_error(e);
    }
    return LLMIG_OK;
}

} // namespace
