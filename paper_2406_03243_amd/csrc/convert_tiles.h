// Cross-layout tile conversion: the stage copy between two pools that keep
// the (token, head, dim) elements of a tile in different orders.  Part of
// the single translation unit built from llmig.hip.
//
// What it computes: for every pair i, layer l and K/V, every element
// (t, h, d) of tile (l, kv) of source block src[i] lands in tile (l, kv) of
// destination block dst[i] at the position the destination's layout gives
// it (the layouts are listed with LLMIG_LAYOUT_* in llmig.h).  Whole tiles
// move, as in the same-layout copy (Llumnix §4.2), so a partial last block
// carries its unused slots along.
//
// Kernel design (CDNA4, wave64):
//  * In every layout a head's elements form one slab of block_size *
//    head_dim * 2 bytes: contiguous in HND, HCNX and HDN, and block_size
//    rows of head_dim * 2 bytes, one per token, in NHD.  A wavefront's work
//    item is one (pair, layer, K/V, head) slab; it reads the slab with
//    16-byte loads in the source's own order (whole rows, coalesced) and
//    writes it with 16-byte stores in the destination's own order
//    (contiguous), so neither side of HBM sees a partial row.
//  * Between the two the slab passes through the wavefront's own LDS
//    region, which is where the layouts transpose.  A 16-byte chunk is 8
//    consecutive dims of one token in NHD, HND and HCNX, and 8 consecutive
//    tokens of one dim in HDN.  Between the first three a chunk moves whole
//    (one ds_read_b128 per chunk); to or from HDN every output chunk
//    gathers 8 16-bit elements from 8 source chunks.  The LDS image has one
//    16-byte pad after every 16 chunks, which spreads the strided reads of
//    both cases over distinct banks for the common shapes (block_size 16,
//    head_dim 64 or 128).
//  * A plane whose two layouts agree (say K converts and V does not) moves
//    chunk for chunk, registers straight to the store, without LDS.
//  * Two wavefronts per workgroup (two adjacent heads of one tile).
//    Measured on the LLaMA-7B stage: 8% faster than four when the source is
//    token-major (its slabs are strided rows), equal the other way; one
//    wavefront per workgroup, or several slabs per wavefront, did worse.
//  * XCD-aware workgroup order: MI355X deals workgroups to its eight XCDs
//    round robin, which scattered the sixteen workgroups of one tile over
//    all eight.  Renumbered so that consecutive workgroups share an XCD,
//    the token-major to head-major stage ran 1-9% faster (in-process, three
//    processes), level with the same-layout copy; the copy itself gained
//    nothing from the same change (1-2.5% slower), so it keeps the
//    hardware's order.
//  * Index arithmetic divides chunk numbers (< 2^16) by per-call constants
//    with a multiply-high by ceil(2^32 / divisor), exact in that range.
//  * Block ids, layouts and base addresses are wavefront-uniform and come
//    from the kernel arguments or scalar loads; ids travel inline as in the
//    same-layout copy (512 pairs of packed 16-bit ids a launch when both
//    pools have at most 65536 blocks, else 256 pairs of 32-bit ids).
//  * Global accesses are raw buffer loads and stores over one tile with the
//    same cache policy as the same-layout copy (nt loads, sc1 nt stores).
//  * The source may also be a staging buffer laid out as llmig_pack writes
//    it (the receiving side of block fusion, §5, converting as it scatters).
#pragma once

#include <algorithm>
#include <cstring>

#include "common.h"

namespace {

constexpr int kMaxSlabChunksPerLane = 16;           // slabs of up to 16 KiB
constexpr int kConvertWaves = 2;                    // wavefronts per workgroup
constexpr uint32_t kXcds = 8;                       // accelerator dies the dispatcher deals workgroups to

struct ConvertArgs {
    const uint64_t *src_tab;
    const uint64_t *dst_tab;
    const uint8_t *src_lin;     // staging buffer [L][2][lin_pairs][tile] (null: source is a pool)
    const int32_t *src_ids_dev; // device id lists (null when the ids are inline)
    const int32_t *dst_ids_dev;
    uint64_t magic_row;         // ceil(2^32 / row_chunks)
    uint64_t magic_bs;          // ceil(2^32 / block_size)
    uint64_t magic_t;           // ceil(2^32 / t_chunks)
    uint32_t tile_bytes;
    uint32_t num_layers;
    uint32_t heads;
    uint32_t block_size;
    uint32_t row_chunks;        // head_dim / 8: chunks of one token's head
    uint32_t t_chunks;          // block_size / 8: chunks of one dim's tokens (HDN)
    uint32_t chunks;            // chunks of one head slab
    uint32_t units;             // wave items: pairs * 2 * num_layers * heads
    uint32_t lin_first;         // this launch's first pair within the whole call
    uint32_t lin_pairs;         // pairs in the whole call (plane stride of the staging buffer)
    int32_t layouts[4];         // source K, source V, destination K, destination V
    uint32_t ids[2 * kInlinePairs]; // inline ids, laid out as the launch's Ids mode says
};

__device__ __forceinline__ uint32_t div_magic(uint32_t n, uint64_t magic)
{
    return static_cast<uint32_t>((static_cast<uint64_t>(n) * magic) >> 32);
}

// Byte offset inside a tile of chunk k (in the layout's own order) of head h.
__device__ __forceinline__ uint32_t slab_offset(int32_t layout, uint32_t h, uint32_t k, const ConvertArgs &a)
{
    if (layout == LLMIG_LAYOUT_NHD) {
        const uint32_t t = div_magic(k, a.magic_row);
        const uint32_t c = k - t * a.row_chunks;
        return ((t * a.heads + h) * a.row_chunks + c) * 16u;
    }
    return (h * a.chunks + k) * 16u;
}

// Slab index of the chunk holding dims [8c, 8c + 8) of token t, in a layout
// whose chunks run along the dims (NHD, HND, HCNX).
__device__ __forceinline__ uint32_t dim_chunk_index(int32_t layout, uint32_t t, uint32_t c, const ConvertArgs &a)
{
    return layout == LLMIG_LAYOUT_HCNX ? c * a.block_size + t : t * a.row_chunks + c;
}

__device__ __forceinline__ uint32_t padded(uint32_t k)
{
    return k + (k >> 4);
}

__device__ __forceinline__ void wave_lds_sync()
{
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
}

template <int IDS>
__device__ __forceinline__ uint32_t convert_src_id(const ConvertArgs &a, uint32_t i)
{
    if (IDS == kIds16)
        return a.ids[i] & 0xffffu;
    return IDS == kIds32 ? a.ids[i] : static_cast<uint32_t>(id_entry(a.src_ids_dev, i));
}

template <int IDS>
__device__ __forceinline__ uint32_t convert_dst_id(const ConvertArgs &a, uint32_t i)
{
    if (IDS == kIds16)
        return a.ids[i] >> 16;
    return IDS == kIds32 ? a.ids[kInlinePairs + i] : static_cast<uint32_t>(id_entry(a.dst_ids_dev, i));
}

template <int IDS, int N>
__global__ void __launch_bounds__(kConvertWaves * 64) convert_tiles(const ConvertArgs a)
{
    __shared__ u32x4 lds[kConvertWaves][68 * N];     // 64 N chunks + one pad per 16
    const uint32_t lane = threadIdx.x % 64;
    const uint32_t wave = threadIdx.x / 64;
    u32x4 *mine = lds[wave];
    const uint16_t *mine16 = reinterpret_cast<const uint16_t *>(mine);
    const uint32_t waves = gridDim.x * kConvertWaves;
    const uint32_t per_pair_plane = a.heads;
    const uint32_t planes = 2u * a.num_layers;

    // XCD-aware order: the hardware hands workgroup g to XCD g % 8, so the
    // logical workgroups are renumbered to put consecutive ones (the heads
    // of one tile) on one XCD.
    const uint32_t full = gridDim.x - gridDim.x % kXcds;
    const uint32_t group = blockIdx.x < full ? (blockIdx.x % kXcds) * (full / kXcds) + blockIdx.x / kXcds
                                             : blockIdx.x;
    for (uint32_t w = group * kConvertWaves + wave; w < a.units; w += waves) {
        const uint32_t unit = uniform(w);
        const uint32_t tile = unit / per_pair_plane;
        const uint32_t h = unit - tile * per_pair_plane;
        const uint32_t i = tile / planes;
        const uint32_t plane = tile - i * planes;
        const uint32_t layer = plane >> 1, kv = plane & 1u;
        const int32_t sl = a.layouts[kv], dl = a.layouts[2 + kv];

        const uint8_t *s;
        if (a.src_lin) {
            s = a.src_lin + (static_cast<uint64_t>(plane) * a.lin_pairs + a.lin_first + i) * a.tile_bytes;
        } else {
            s = reinterpret_cast<const uint8_t *>(table_entry(a.src_tab, kv * a.num_layers + layer)) +
                static_cast<uint64_t>(uniform(convert_src_id<IDS>(a, i))) * a.tile_bytes;
        }
        uint8_t *d = reinterpret_cast<uint8_t *>(table_entry(a.dst_tab, kv * a.num_layers + layer)) +
                     static_cast<uint64_t>(uniform(convert_dst_id<IDS>(a, i))) * a.tile_bytes;
        const __amdgpu_buffer_rsrc_t rs = tile_rsrc(s, a.tile_bytes);
        const __amdgpu_buffer_rsrc_t rd = tile_rsrc(d, a.tile_bytes);

        u32x4 r[N];
#pragma unroll
        for (int u = 0; u < N; ++u) {
            const uint32_t k = lane + 64u * u;
            if (k < a.chunks)
                r[u] = buffer_load16(rs, slab_offset(sl, h, k, a));
        }
        if (sl == dl) {
#pragma unroll
            for (int u = 0; u < N; ++u) {
                const uint32_t k = lane + 64u * u;
                if (k < a.chunks)
                    buffer_store16(rd, slab_offset(dl, h, k, a), r[u]);
            }
            continue;
        }
#pragma unroll
        for (int u = 0; u < N; ++u) {
            const uint32_t k = lane + 64u * u;
            if (k < a.chunks)
                mine[padded(k)] = r[u];
        }
        wave_lds_sync();
        // Output chunks: fully unrolled for small slabs; for large ones two at
        // a time, which keeps the gathers' registers within four waves' share.
        constexpr int kGatherUnroll = N > 4 ? 2 : N;
#pragma unroll kGatherUnroll
        for (int u = 0; u < N; ++u) {
            const uint32_t k = lane + 64u * u;
            if (k >= a.chunks)
                continue;
            u32x4 v;
            if (dl == LLMIG_LAYOUT_HDN) {
                // Output chunk: tokens [8 tg, 8 tg + 8) of dim dd.
                const uint32_t dd = div_magic(k, a.magic_t);
                const uint32_t tg = k - dd * a.t_chunks;
                const uint32_t c = dd >> 3, e = dd & 7u;
                uint32_t x[8];
#pragma unroll
                for (int j = 0; j < 8; ++j)
                    x[j] = mine16[padded(dim_chunk_index(sl, 8u * tg + j, c, a)) * 8u + e];
                v = u32x4{x[0] | (x[1] << 16), x[2] | (x[3] << 16), x[4] | (x[5] << 16), x[6] | (x[7] << 16)};
            } else {
                // Output chunk: dims [8 c, 8 c + 8) of token t.
                uint32_t t, c;
                if (dl == LLMIG_LAYOUT_HCNX) {
                    c = div_magic(k, a.magic_bs);
                    t = k - c * a.block_size;
                } else {
                    t = div_magic(k, a.magic_row);
                    c = k - t * a.row_chunks;
                }
                if (sl == LLMIG_LAYOUT_HDN) {
                    const uint32_t tg = t >> 3, e = t & 7u;
                    uint32_t x[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j)
                        x[j] = mine16[padded((8u * c + j) * a.t_chunks + tg) * 8u + e];
                    v = u32x4{x[0] | (x[1] << 16), x[2] | (x[3] << 16), x[4] | (x[5] << 16),
                              x[6] | (x[7] << 16)};
                } else {
                    v = mine[padded(dim_chunk_index(sl, t, c, a))];
                }
            }
            buffer_store16(rd, slab_offset(dl, h, k, a), v);
        }
        wave_lds_sync();
    }
}

template <int IDS>
const void *convert_kernel_n(int n)
{
    switch (n) {
    case 16:
        return reinterpret_cast<const void *>(&convert_tiles<IDS, 16>);
    case 8:
        return reinterpret_cast<const void *>(&convert_tiles<IDS, 8>);
    case 4:
        return reinterpret_cast<const void *>(&convert_tiles<IDS, 4>);
    case 2:
        return reinterpret_cast<const void *>(&convert_tiles<IDS, 2>);
    default:
        return reinterpret_cast<const void *>(&convert_tiles<IDS, 1>);
    }
}

const void *convert_kernel(int ids, int n)
{
    if (ids == kIdsDevice)
        return convert_kernel_n<kIdsDevice>(n);
    return ids == kIds16 ? convert_kernel_n<kIds16>(n) : convert_kernel_n<kIds32>(n);
}

uint64_t magic_for(uint32_t divisor)
{
    return ((1ull << 32) + divisor - 1) / divisor;
}

// Chunks per lane (a power of two) for slabs of `chunks` 16-byte chunks.
int convert_chunks_per_lane(uint32_t chunks)
{
    int n = 1;
    while (static_cast<uint32_t>(n) * 64u < chunks)
        n *= 2;
    return n;
}

// Launches the conversion of n pairs (src_ids null: the source is the staging
// buffer a.src_lin, one tile per pair and plane).  The caller has checked
// that the geometry is supported (16-bit elements, head_dim % 8 == 0,
// block_size % 8 == 0 when a side is HDN, slabs of at most 16 KiB).
// ids16: every id of both lists is below 65536 (pool to pool only).
int launch_convert(ConvertArgs a, const int32_t *src_ids, const int32_t *dst_ids, int64_t n, bool ids_on_device,
                   hipStream_t stream, uint32_t max_workgroups, const LaunchEvents &ev = LaunchEvents(),
                   bool ids16 = false)
{
    const int ids = ids_on_device ? kIdsDevice : (src_ids && ids16) ? kIds16 : kIds32;
    const uint64_t inline_pairs = ids == kIds16 ? 2 * kInlinePairs : kInlinePairs;
    const int per_lane = convert_chunks_per_lane(a.chunks);
    if (per_lane > kMaxSlabChunksPerLane)
        return LLMIG_EINVAL;
    a.magic_row = magic_for(a.row_chunks);
    a.magic_bs = magic_for(a.block_size);
    a.magic_t = magic_for(a.t_chunks > 0 ? a.t_chunks : 1u);
    const uint64_t units_per_pair = 2ull * a.num_layers * a.heads;
    const uint64_t per_launch = std::min<uint64_t>(0x7fffffffull / units_per_pair,
                                                   ids_on_device ? UINT64_MAX : inline_pairs);
    if (per_launch == 0)
        return LLMIG_EINVAL;
    const void *fn = convert_kernel(ids, per_lane);
    a.lin_pairs = static_cast<uint32_t>(n);
    const int64_t launches = (n + static_cast<int64_t>(per_launch) - 1) / static_cast<int64_t>(per_launch);
    for (int64_t first = 0, k = 0; first < n; first += static_cast<int64_t>(per_launch), ++k) {
        const uint32_t m = static_cast<uint32_t>(std::min<int64_t>(n - first, per_launch));
        a.units = static_cast<uint32_t>(m * units_per_pair);
        a.lin_first = static_cast<uint32_t>(first);
        if (ids == kIdsDevice) {
            a.src_ids_dev = src_ids ? src_ids + first : nullptr;
            a.dst_ids_dev = dst_ids + first;
        } else if (ids == kIds16) {
            for (uint32_t k = 0; k < m; ++k)
                a.ids[k] = static_cast<uint32_t>(src_ids[first + k]) | (static_cast<uint32_t>(dst_ids[first + k]) << 16);
        } else {
            if (src_ids)
                std::memcpy(a.ids, src_ids + first, m * sizeof(int32_t));
            std::memcpy(a.ids + kInlinePairs, dst_ids + first, m * sizeof(int32_t));
        }
        void *args[] = {&a};
        uint32_t grid = std::min((a.units + kConvertWaves - 1) / kConvertWaves, kMaxGridWorkgroups);
        if (max_workgroups > 0)
            grid = std::min(grid, max_workgroups);
        hipError_t e = launch_kernel(fn, dim3(grid), dim3(kConvertWaves * 64), args, stream, ev, k, launches);
        if (e != hipSuccess)
            return hip_error(e);
    }
    return LLMIG_OK;
}

} // namespace
