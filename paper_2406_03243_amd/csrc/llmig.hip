// llmig: multi-stage KV-cache live migration on MI355X (gfx950).
//
// Kernels and C-ABI host code behind include/llmig.h.  The method is the
// live migration of Llumnix (arXiv 2406.03243) §4.2 with the block fusion
// of §5; the interface comments in llmig.h state what every call computes.
//
// Sources: common.h (shared kernel definitions, buffer accesses, launch
// helper), copy_tiles.h (the tile copy and its launch configuration),
// convert_tiles.h (the copy between pools of different intra-tile
// layouts), decode_attention.h (paged decode attention, the work measured
// beside a migration), this file (pool registry, planner, coordinator,
// harness kernels, argument checks and the C ABI).

#include <hip/hip_runtime.h>

#include <algorithm>
#include <atomic>
#include <chrono>
#include <cstdint>
#include <cstring>
#include <memory>
#include <mutex>
#include <new>
#include <utility>
#include <vector>

#include "llmig.h"
#include "common.h"
#include "convert_tiles.h"
#include "copy_tiles.h"
#include "decode_attention.h"

struct llmig_pool {
    int32_t num_layers, num_blocks, block_size, num_kv_heads, head_dim, elem_bytes;
    int32_t layouts[2];                               // K, V intra-tile layouts (LLMIG_LAYOUT_*)
    int64_t tile_bytes;
    int device;
    uint64_t *d_tab;                                  // device [2 * L]: K bases, then V bases
    std::vector<std::pair<uint64_t, uint64_t>> spans; // sorted [begin, end) of every layer tensor
};

struct llmig_migration {
    int32_t block_size;
    int32_t state;
    int64_t copied_tok;               // tokens copied by the stages so far
    int64_t stages;
    uint32_t max_workgroups;          // 0: no cap on the copy grid
    LaunchEvents next_events;         // events for the next stage's kernels (then cleared)
    std::vector<int32_t> reserved;    // destination blocks, in logical order
    std::vector<int32_t> plan_src;    // per-stage scratch, reused
    std::vector<int32_t> plan_dst;
};

// Partial results of llmig_decode_attention_noalloc (the entry point for
// callers that cannot allocate): one static array, of which every GPU the
// library runs on holds its own copy until the process ends.  Host code
// never uses the array's name as an address: it reaches each device's copy
// through the address hipGetSymbolAddress gives with that device current
// (scratch_pointer below).
__device__ __align__(256) uint8_t scratch[LLMIG_DECODE_SCRATCH_BYTES];

namespace {

// Decode stand-in: writes whole token slots through a block table.
struct WriteArgs {
    const uint64_t *tab;
    const uint8_t *data;
    uint32_t slot_bytes;
    uint32_t tile_bytes;
    uint32_t block_size;
    uint32_t num_layers;
    uint32_t head_dim;
    uint32_t row_chunks;   // head_dim * elem_bytes / 16 (layouts other than NHD)
    int32_t layouts[2];    // K, V
    uint32_t data_tokens;  // tokens in the whole call (plane stride of data)
    uint32_t first_token;  // this launch's first token within the call
    uint32_t tokens;       // tokens in this launch
    uint32_t first_slot;   // slot of this launch's first token within its block
    int32_t ids[kInlinePairs]; // blocks this launch touches, in logical order
};

__global__ void __launch_bounds__(kThreads) write_token_slots(const WriteArgs a)
{
    const uint32_t items = a.tokens * 2u * a.num_layers;
    for (uint32_t item = blockIdx.x; item < items; item += gridDim.x) {
        const uint32_t plane = item / a.tokens;
        const uint32_t j = item - plane * a.tokens;
        const uint32_t layer = plane >> 1, kv = plane & 1u;
        const uint32_t rel = a.first_slot + j;
        const uint32_t blk = rel / a.block_size;
        const uint32_t slot = rel - blk * a.block_size;
        uint8_t *tile = reinterpret_cast<uint8_t *>(table_entry(a.tab, kv * a.num_layers + layer)) +
                        static_cast<uint64_t>(uniform(static_cast<uint32_t>(a.ids[blk]))) * a.tile_bytes;
        const uint8_t *s = a.data + (static_cast<uint64_t>(plane) * a.data_tokens + a.first_token + j) *
                                        a.slot_bytes;
        const int32_t layout = a.layouts[kv];
        if (layout == LLMIG_LAYOUT_NHD) {
            uint8_t *d = tile + static_cast<uint64_t>(slot) * a.slot_bytes;
            for (uint32_t off = threadIdx.x * 16u; off < a.slot_bytes; off += kRowBytes)
                *(LLMIG_GLOBAL u32x4 *)(d + off) = load16(s + off);
            continue;
        }
        // 16-bit elements: chunk q of the token is dims [8c, 8c + 8) of head h.
        for (uint32_t off = threadIdx.x * 16u; off < a.slot_bytes; off += kRowBytes) {
            const uint32_t q = off / 16u;
            const uint32_t h = q / a.row_chunks, c = q - h * a.row_chunks;
            const u32x4 v = load16(s + off);
            if (layout == LLMIG_LAYOUT_HND) {
                *(LLMIG_GLOBAL u32x4 *)(tile + ((h * a.block_size + slot) * a.row_chunks + c) * 16u) = v;
            } else if (layout == LLMIG_LAYOUT_HCNX) {
                *(LLMIG_GLOBAL u32x4 *)(tile + ((h * a.row_chunks + c) * a.block_size + slot) * 16u) = v;
            } else {
                const uint32_t w[4] = {v.x, v.y, v.z, v.w};
#pragma unroll
                for (uint32_t e = 0; e < 8; ++e) {
                    const uint32_t dim = 8u * c + e;
                    *(LLMIG_GLOBAL uint16_t *)(tile + ((h * a.head_dim + dim) * a.block_size + slot) * 2u) =
                        static_cast<uint16_t>(w[e / 2] >> (16u * (e & 1u)));
                }
            }
        }
    }
}

// Harness: a steady stream of HBM reads standing in for decode's KV reads.
// Each lane sums (as 32-bit integers) the 16-byte words it reads and stores
// its own result to out[global lane]; every lane runs a fixed number of
// passes, so the grid always drains.
__global__ void __launch_bounds__(kThreads) stream_read_words(const uint8_t *region, uint64_t words,
                                                              uint32_t passes, uint64_t *out)
{
    constexpr int kLoads = 8;
    const uint64_t lane = static_cast<uint64_t>(blockIdx.x) * kThreads + threadIdx.x;
    const uint64_t lanes = static_cast<uint64_t>(gridDim.x) * kThreads;
    u32x4 acc = {0u, 0u, 0u, 0u};
    for (uint32_t p = 0; p < passes; ++p) {
        uint64_t w = lane;
        for (; w + (kLoads - 1) * lanes < words; w += kLoads * lanes) {
            u32x4 r[kLoads];
#pragma unroll
            for (int u = 0; u < kLoads; ++u)
                r[u] = load16(region + (w + u * lanes) * 16);
#pragma unroll
            for (int u = 0; u < kLoads; ++u)
                acc += r[u];
        }
        for (; w < words; w += lanes)
            acc += load16(region + w * 16);
    }
    const uint64_t folded = (static_cast<uint64_t>(acc.x + acc.z) << 32) | (acc.y + acc.w);
    ((LLMIG_GLOBAL uint64_t *)out)[lane] = folded;
}

// Completion signal of llmig_migration_finish: one lane stores the call's
// ticket into its slot of pinned host memory, a release store at system
// scope (a vector store), once the stream's earlier work (the final stage's
// copy) has completed.
__global__ void __launch_bounds__(64) signal_host(uint64_t *slot, uint64_t ticket)
{
    if (threadIdx.x == 0)
        __hip_atomic_store(slot, ticket, __ATOMIC_RELEASE, __HIP_MEMORY_SCOPE_SYSTEM);
}

// Runs an entry point's body.  The host code's only exceptions are failed
// allocations (the id bitmaps, plan scratch, pool bookkeeping); they become
// LLMIG_EINVAL here instead of crossing the C ABI.  Bodies allocate before
// they enqueue anything, so such a failure has no effect.
template <typename Body>
int no_throw(Body &&body)
{
    try {
        return body();
    } catch (...) {
        return LLMIG_EINVAL;
    }
}

// Whether the pool lives on the calling thread's current device, where the
// library launches its kernels.
bool on_current_device(const llmig_pool *pool)
{
    int d = -1;
    return hipGetDevice(&d) == hipSuccess && d == pool->device;
}

// Device address of `scratch` on each device, looked up once per device
// with that device current (at its first llmig_pool_create, else at the
// first llmig_decode_attention_noalloc there) and kept for the process.
constexpr int kMaxDevices = 64;
std::mutex g_scratch_mutex;
void *g_scratch_ptr[kMaxDevices] = {};

// The current device's scratch address, looked up on first use.
int scratch_pointer(int device, void **out)
{
    if (device < 0 || device >= kMaxDevices)
        return LLMIG_EINVAL;
    std::lock_guard<std::mutex> lock(g_scratch_mutex);
    if (!g_scratch_ptr[device]) {
        void *p = nullptr;
        const hipError_t e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
        if (e != hipSuccess || !p)
            return hip_error(e != hipSuccess ? e : hipErrorInvalidSymbol);
        g_scratch_ptr[device] = p;
    }
    *out = g_scratch_ptr[device];
    return LLMIG_OK;
}

// Host-visible completion slots of llmig_migration_finish: kFinishSlots
// 64-bit tickets, one cache line apart, in pinned host memory mapped for
// every device, allocated with the first pool (set-up) and kept for the
// process.  Each call takes the next ticket from a counter; its slot is
// ticket % kFinishSlots, and it returns only on reading its own ticket
// there.  A slot can be rewritten by a call kFinishSlots tickets later (on
// another stream, in either order); a waiter whose ticket was overwritten
// before it read it falls back to the runtime wait, so no call returns
// before its own work is done.
constexpr uint64_t kFinishSlots = 1024;
constexpr uint64_t kFinishSlotStride = 64 / sizeof(uint64_t);
// How long llmig_migration_finish reads its slot before it falls back to a
// runtime wait on the stream (a final stage behind other queued work can
// take longer than this).
constexpr double kFinishSpinUs = 2000.0;

struct FinishSlots {
    std::mutex mu;                             // serialises the set-up
    std::atomic<uint64_t *> host{nullptr};
    std::atomic<uint64_t *> dev[kMaxDevices] = {};
    std::atomic<uint64_t> next{1};
};
FinishSlots g_finish;

// Allocates the slots (once) and maps them for `device` (current).
void finish_slots_setup(int device)
{
    if (device < 0 || device >= kMaxDevices)
        return;
    std::lock_guard<std::mutex> lock(g_finish.mu);
    if (!g_finish.host.load()) {
        void *p = nullptr;
        if (hipHostMalloc(&p, kFinishSlots * kFinishSlotStride * sizeof(uint64_t),
                          hipHostMallocMapped | hipHostMallocPortable) != hipSuccess) {
            (void)hipGetLastError();
            return;
        }
        std::memset(p, 0, kFinishSlots * kFinishSlotStride * sizeof(uint64_t));
        g_finish.host.store(static_cast<uint64_t *>(p));
    }
    if (!g_finish.dev[device].load()) {
        void *d = nullptr;
        if (hipHostGetDevicePointer(&d, g_finish.host.load(), 0) == hipSuccess)
            g_finish.dev[device].store(static_cast<uint64_t *>(d));
        else
            (void)hipGetLastError();
    }
}

// Waits until the work enqueued on `stream` so far has completed: through
// a completion slot when the device has them (a signal kernel behind the
// work, the host reading the slot without calling the runtime), else, or
// after kFinishSpinUs, through hipStreamSynchronize.
int wait_stream(int device, hipStream_t stream)
{
    uint64_t *dev_slots = (device >= 0 && device < kMaxDevices) ? g_finish.dev[device].load() : nullptr;
    if (dev_slots) {
        const uint64_t ticket = g_finish.next.fetch_add(1, std::memory_order_relaxed);
        const uint64_t slot = (ticket % kFinishSlots) * kFinishSlotStride;
        uint64_t *dp = dev_slots + slot;
        void *args[] = {&dp, const_cast<uint64_t *>(&ticket)};
        hipError_t e = hipLaunchKernel(reinterpret_cast<const void *>(&signal_host), dim3(1), dim3(64), args, 0,
                                       stream);
        if (e != hipSuccess)
            return hip_error(e);
        const uint64_t *hp = g_finish.host.load() + slot;
        const auto t0 = std::chrono::steady_clock::now();
        for (uint32_t k = 1;; ++k) {
            if (__atomic_load_n(hp, __ATOMIC_ACQUIRE) == ticket)
                return LLMIG_OK;
            if ((k & 1023u) == 0 &&
                std::chrono::duration<double, std::micro>(std::chrono::steady_clock::now() - t0).count() >
                    kFinishSpinUs)
                break;
        }
    }
    const hipError_t e = hipStreamSynchronize(stream);
    return e == hipSuccess ? LLMIG_OK : hip_error(e);
}

bool same_geometry(const llmig_pool *a, const llmig_pool *b)
{
    return a->num_layers == b->num_layers && a->block_size == b->block_size &&
           a->num_kv_heads == b->num_kv_heads && a->head_dim == b->head_dim &&
           a->elem_bytes == b->elem_bytes;
}

// Whether any layer tensor of a overlaps any of b (both span lists sorted).
bool pools_overlap(const llmig_pool *a, const llmig_pool *b)
{
    if (a == b)
        return true;
    size_t i = 0, j = 0;
    while (i < a->spans.size() && j < b->spans.size()) {
        const auto &x = a->spans[i];
        const auto &y = b->spans[j];
        if (x.first < y.second && y.first < x.second)
            return true;
        if (x.second <= y.second)
            ++i;
        else
            ++j;
    }
    return false;
}

int check_ids(const int32_t *ids, int64_t n, int32_t num_blocks)
{
    for (int64_t k = 0; k < n; ++k)
        if (ids[k] < 0 || ids[k] >= num_blocks)
            return LLMIG_ERANGE;
    return LLMIG_OK;
}

// Whether ids[0..n) holds a repeat; ids are known to lie in [0, bound)
// (bound may be 0 when n <= 32).  Pairwise for short lists, else a bitmap.
bool has_repeat(const int32_t *ids, int64_t n, int64_t bound)
{
    if (n <= 32) {
        for (int64_t a = 0; a < n; ++a)
            for (int64_t b = a + 1; b < n; ++b)
                if (ids[a] == ids[b])
                    return true;
        return false;
    }
    std::vector<uint64_t> seen(static_cast<size_t>((bound + 63) / 64), 0);
    for (int64_t k = 0; k < n; ++k) {
        const uint64_t bit = 1ull << (ids[k] & 63);
        uint64_t &word = seen[static_cast<size_t>(ids[k]) >> 6];
        if (word & bit)
            return true;
        word |= bit;
    }
    return false;
}

// Whether ids[0..n) holds a repeat, for non-negative ids of any size: a
// bitmap up to the largest id when that stays small (2 MiB), else a sort.
bool has_repeat_any(const int32_t *ids, int64_t n)
{
    if (n <= 32)
        return has_repeat(ids, n, 0);
    int32_t hi = 0;
    for (int64_t k = 0; k < n; ++k)
        hi = std::max(hi, ids[k]);
    if (hi < (1 << 24))
        return has_repeat(ids, n, static_cast<int64_t>(hi) + 1);
    std::vector<int32_t> v(ids, ids + n);
    std::sort(v.begin(), v.end());
    return std::adjacent_find(v.begin(), v.end()) != v.end();
}

// Device-visible address of a staging buffer: device memory as is, pinned
// host memory through its device mapping.  Pageable memory is refused.
int staging_pointer(const void *p, void **out)
{
    hipPointerAttribute_t attr;
    std::memset(&attr, 0, sizeof(attr));
    hipError_t e = hipPointerGetAttributes(&attr, p);
    if (e != hipSuccess) {
        (void)hipGetLastError();
        return LLMIG_EINVAL;
    }
    if (attr.type == hipMemoryTypeDevice) {
        *out = const_cast<void *>(p);
        return LLMIG_OK;
    }
    if (attr.type == hipMemoryTypeHost && attr.devicePointer != nullptr) {
        *out = attr.devicePointer;
        return LLMIG_OK;
    }
    return LLMIG_EINVAL;
}

int fused_copy_checks(const llmig_pool *pool, const int32_t *blocks, int64_t n, int map_on_device,
                      const void *staging, int64_t staging_bytes, bool reject_repeats)
{
    if (!pool || n < 0 || (map_on_device != 0 && map_on_device != 1) || !on_current_device(pool))
        return LLMIG_EINVAL;
    if (n == 0)
        return LLMIG_OK;
    if (!blocks || !staging || (reinterpret_cast<uintptr_t>(staging) & 15u))
        return LLMIG_EINVAL;
    if (n > (INT64_MAX / 2) / pool->num_layers / pool->tile_bytes)
        return LLMIG_EINVAL;
    if (staging_bytes < n * pool->num_layers * 2 * pool->tile_bytes)
        return LLMIG_EINVAL;
    if (!map_on_device) {
        int rc = check_ids(blocks, n, pool->num_blocks);
        if (rc != LLMIG_OK)
            return rc;
        if (reject_repeats && has_repeat(blocks, n, pool->num_blocks))
            return LLMIG_EINVAL;
    }
    return LLMIG_OK;
}

bool same_layouts(const llmig_pool *src, const llmig_pool *dst)
{
    return src->layouts[0] == dst->layouts[0] && src->layouts[1] == dst->layouts[1];
}

// Whether the conversion kernel supports a pool of this geometry converting
// from (or to) tiles in layouts other[0] (K) and other[1] (V).
bool conversion_supported(const llmig_pool *pool, const int32_t *other)
{
    if (pool->elem_bytes != 2 || pool->head_dim % 8 != 0)
        return false;
    const bool hdn = pool->layouts[0] == LLMIG_LAYOUT_HDN || pool->layouts[1] == LLMIG_LAYOUT_HDN ||
                     other[0] == LLMIG_LAYOUT_HDN || other[1] == LLMIG_LAYOUT_HDN;
    if (hdn && pool->block_size % 8 != 0)
        return false;
    const int64_t chunks = static_cast<int64_t>(pool->block_size) * pool->head_dim / 8;
    return chunks <= 64 * kMaxSlabChunksPerLane;
}

ConvertArgs convert_args(const llmig_pool *pool, const int32_t *src_layouts, const int32_t *dst_layouts)
{
    ConvertArgs c;
    std::memset(&c, 0, sizeof(c));
    c.tile_bytes = static_cast<uint32_t>(pool->tile_bytes);
    c.num_layers = static_cast<uint32_t>(pool->num_layers);
    c.heads = static_cast<uint32_t>(pool->num_kv_heads);
    c.block_size = static_cast<uint32_t>(pool->block_size);
    c.row_chunks = static_cast<uint32_t>(pool->head_dim / 8);
    c.t_chunks = static_cast<uint32_t>(pool->block_size / 8);
    c.chunks = static_cast<uint32_t>(pool->block_size * pool->head_dim / 8);
    c.layouts[0] = src_layouts[0];
    c.layouts[1] = src_layouts[1];
    c.layouts[2] = dst_layouts[0];
    c.layouts[3] = dst_layouts[1];
    return c;
}

bool pools_compatible(const llmig_pool *src, const llmig_pool *dst)
{
    return same_geometry(src, dst) && src->device == dst->device && on_current_device(src) &&
           !pools_overlap(src, dst) && (same_layouts(src, dst) || conversion_supported(src, dst->layouts));
}

int check_pair_ids(const llmig_pool *src, const llmig_pool *dst, const int32_t *ms, const int32_t *md, int64_t n)
{
    int rc = check_ids(ms, n, src->num_blocks);
    return rc == LLMIG_OK ? check_ids(md, n, dst->num_blocks) : rc;
}

int launch_stage(const llmig_pool *src, const llmig_pool *dst, const int32_t *ms, const int32_t *md, int64_t n,
                 bool ids_on_device, hipStream_t stream, uint32_t max_workgroups = 0,
                 const LaunchEvents &ev = LaunchEvents())
{
    if (!same_layouts(src, dst)) {
        ConvertArgs c = convert_args(src, src->layouts, dst->layouts);
        c.src_tab = src->d_tab;
        c.dst_tab = dst->d_tab;
        const bool ids16 = src->num_blocks <= 65536 && dst->num_blocks <= 65536;
        return launch_convert(c, ms, md, n, ids_on_device, stream, max_workgroups, ev, ids16);
    }
    CopyArgs a;
    std::memset(&a, 0, sizeof(a));
    a.src_tab = src->d_tab;
    a.dst_tab = dst->d_tab;
    a.tile_bytes = static_cast<uint32_t>(src->tile_bytes);
    a.num_layers = static_cast<uint32_t>(src->num_layers);
    // ids are range-checked against the pools when they come from the host
    const bool ids16 = src->num_blocks <= 65536 && dst->num_blocks <= 65536;
    return launch_copy<kPool, kPool>(a, ms, md, n, ids_on_device, stream, max_workgroups, ids16, ev);
}

// Token range of the next stage of m for a request now holding len tokens.
int next_range(const llmig_migration *m, int64_t len, int final_stage, int64_t *from, int64_t *to)
{
    if (m->state != LLMIG_MIGRATION_ACTIVE || len < m->copied_tok || (final_stage != 0 && final_stage != 1))
        return LLMIG_EINVAL;
    *from = m->copied_tok;
    *to = final_stage ? len : (len / m->block_size) * m->block_size;
    return LLMIG_OK;
}

// Adds a planned stage to m.  LLMIG_EINVAL, with m unchanged, when the
// reservation cannot grow (no exception leaves the library).
int record_stage(llmig_migration *m, const int32_t *dst_ids, int64_t n, int64_t to, int final_stage)
{
    try {
        m->reserved.insert(m->reserved.end(), dst_ids, dst_ids + n); // n <= free list: memory the caller holds
    } catch (...) {
        return LLMIG_EINVAL;
    }
    m->copied_tok = to;
    m->stages += 1;
    if (final_stage)
        m->state = LLMIG_MIGRATION_FINISHED;
    return LLMIG_OK;
}

} // namespace

extern "C" {

int llmig_pool_create(const llmig_pool_desc *desc, llmig_pool **out)
{
    if (!out)
        return LLMIG_EINVAL;
    *out = nullptr;
    if (!desc || desc->num_layers <= 0 || desc->num_blocks <= 0 || desc->block_size <= 0 ||
        desc->num_kv_heads <= 0 || desc->head_dim <= 0 || desc->elem_bytes <= 0 || !desc->k_ptrs ||
        !desc->v_ptrs)
        return LLMIG_EINVAL;
    const int64_t tile = static_cast<int64_t>(desc->block_size) * desc->num_kv_heads * desc->head_dim *
                         desc->elem_bytes;
    if (tile % 16 != 0 || tile > 0x7fffffffLL)
        return LLMIG_EINVAL;
    for (int32_t layout : {desc->k_layout, desc->v_layout}) {
        if (layout < LLMIG_LAYOUT_NHD || layout > LLMIG_LAYOUT_HDN)
            return LLMIG_EINVAL;
        if (layout == LLMIG_LAYOUT_HCNX &&
            (16 % desc->elem_bytes != 0 || (static_cast<int64_t>(desc->head_dim) * desc->elem_bytes) % 16 != 0))
            return LLMIG_EINVAL;
    }
    return no_throw([&]() -> int {
        const int32_t L = desc->num_layers;
        std::vector<uint64_t> tab(2 * static_cast<size_t>(L));
        for (int32_t l = 0; l < L; ++l) {
            tab[l] = desc->k_ptrs[l];
            tab[L + l] = desc->v_ptrs[l];
        }
        for (uint64_t p : tab)
            if (p == 0 || (p & 15u))
                return LLMIG_EINVAL;

        std::unique_ptr<llmig_pool> pool(new llmig_pool());
        pool->num_layers = L;
        pool->num_blocks = desc->num_blocks;
        pool->block_size = desc->block_size;
        pool->num_kv_heads = desc->num_kv_heads;
        pool->head_dim = desc->head_dim;
        pool->elem_bytes = desc->elem_bytes;
        pool->layouts[0] = desc->k_layout;
        pool->layouts[1] = desc->v_layout;
        pool->tile_bytes = tile;
        pool->d_tab = nullptr;
        const uint64_t tensor_bytes = static_cast<uint64_t>(tile) * static_cast<uint64_t>(desc->num_blocks);
        for (uint64_t p : tab)
            pool->spans.emplace_back(p, p + tensor_bytes);
        std::sort(pool->spans.begin(), pool->spans.end());
        for (size_t k = 1; k < pool->spans.size(); ++k)
            if (pool->spans[k].first < pool->spans[k - 1].second) // layer tensors overlap each other
                return LLMIG_EINVAL;
        hipError_t e = hipGetDevice(&pool->device);
        if (e == hipSuccess)
            e = hipMalloc(reinterpret_cast<void **>(&pool->d_tab), tab.size() * sizeof(uint64_t));
        if (e == hipSuccess)
            e = hipMemcpy(pool->d_tab, tab.data(), tab.size() * sizeof(uint64_t), hipMemcpyHostToDevice);
        if (e != hipSuccess) {
            if (pool->d_tab)
                (void)hipFree(pool->d_tab);
            return hip_error(e);
        }
        // Set-up of the scratch array's address on this device, so that the
        // no-allocation entry point finds it ready; a failure here is
        // reported by that entry point, which looks it up again.
        void *unused = nullptr;
        (void)scratch_pointer(pool->device, &unused);
        finish_slots_setup(pool->device);
        *out = pool.release();
        return LLMIG_OK;
    });
}

void llmig_pool_destroy(llmig_pool *pool)
{
    if (!pool)
        return;
    if (pool->d_tab)
        (void)hipFree(pool->d_tab);
    delete pool;
}

int64_t llmig_pool_tile_bytes(const llmig_pool *pool)
{
    return pool ? pool->tile_bytes : -1;
}

int llmig_plan(const int32_t *src_table, int64_t src_table_len, const int32_t *dst_free_list,
               int64_t dst_free_len, int64_t len, int64_t from_tok, int64_t to_tok, int32_t block_size,
               int32_t *out_src, int32_t *out_dst, int64_t out_cap, int64_t *out_n)
{
    return no_throw([&]() -> int {
        if (!out_n)
            return LLMIG_EINVAL;
        *out_n = 0;
        if (block_size < 1 || len < 0 || from_tok < 0 || from_tok > to_tok || to_tok > len)
            return LLMIG_EINVAL;
        if (from_tok % block_size != 0 || (to_tok % block_size != 0 && to_tok != len))
            return LLMIG_EINVAL;
        if (src_table_len < 0 || dst_free_len < 0 || out_cap < 0)
            return LLMIG_EINVAL;
        const int64_t blocks_of_len = len / block_size + (len % block_size != 0);
        if (src_table_len < blocks_of_len || (blocks_of_len > 0 && !src_table))
            return LLMIG_EINVAL;
        const int64_t first = from_tok / block_size;
        const int64_t n = to_tok / block_size + (to_tok % block_size != 0) - first;
        if (n > dst_free_len)
            return LLMIG_ENOSPC;
        if (n > out_cap || (n > 0 && (!dst_free_list || !out_src || !out_dst)))
            return LLMIG_EINVAL;
        const int32_t *src = src_table + first;
        for (int64_t k = 0; k < n; ++k)
            if (src[k] < 0 || dst_free_list[k] < 0)
                return LLMIG_ERANGE;
        if (has_repeat_any(src, n) || has_repeat_any(dst_free_list, n))
            return LLMIG_EINVAL;
        if (n > 0) { // the output arrays may be NULL for an empty stage
            std::memcpy(out_src, src, static_cast<size_t>(n) * sizeof(int32_t));
            std::memcpy(out_dst, dst_free_list, static_cast<size_t>(n) * sizeof(int32_t));
        }
        *out_n = n;
        return LLMIG_OK;
    });
}

int llmig_stage(const llmig_pool *src, const llmig_pool *dst, const int32_t *map_src,
                const int32_t *map_dst, int64_t n, int map_on_device, void *stream)
{
    return no_throw([&]() -> int {
        if (!src || !dst || n < 0 || (map_on_device != 0 && map_on_device != 1))
            return LLMIG_EINVAL;
        if (!pools_compatible(src, dst))
            return LLMIG_EINVAL;
        if (n == 0)
            return LLMIG_OK;
        if (!map_src || !map_dst)
            return LLMIG_EINVAL;
        if (!map_on_device) {
            int rc = check_pair_ids(src, dst, map_src, map_dst, n);
            if (rc != LLMIG_OK)
                return rc;
            if (has_repeat(map_dst, n, dst->num_blocks))
                return LLMIG_EINVAL;
        }
        return launch_stage(src, dst, map_src, map_dst, n, map_on_device != 0, static_cast<hipStream_t>(stream));
    });
}

int llmig_migration_create(int32_t block_size, llmig_migration **out)
{
    if (!out)
        return LLMIG_EINVAL;
    *out = nullptr;
    if (block_size < 1)
        return LLMIG_EINVAL;
    llmig_migration *m = new (std::nothrow) llmig_migration();
    if (!m)
        return LLMIG_EINVAL;
    m->block_size = block_size;
    m->state = LLMIG_MIGRATION_ACTIVE;
    m->copied_tok = 0;
    m->stages = 0;
    m->max_workgroups = 0;
    m->next_events = LaunchEvents();
    *out = m;
    return LLMIG_OK;
}

void llmig_migration_destroy(llmig_migration *m)
{
    delete m;
}

int llmig_migration_next(llmig_migration *m, const int32_t *src_table, int64_t src_table_len, int64_t len,
                         int final_stage, const int32_t *dst_free_list, int64_t dst_free_len, int32_t *out_src,
                         int32_t *out_dst, int64_t out_cap, int64_t *out_n)
{
    return no_throw([&]() -> int {
        if (!m || !out_n)
            return LLMIG_EINVAL;
        *out_n = 0;
        int64_t from = 0, to = 0;
        int rc = next_range(m, len, final_stage, &from, &to);
        if (rc != LLMIG_OK)
            return rc;
        int64_t n = 0;
        rc = llmig_plan(src_table, src_table_len, dst_free_list, dst_free_len, len, from, to, m->block_size, out_src,
                        out_dst, out_cap, &n);
        if (rc != LLMIG_OK)
            return rc;
        rc = record_stage(m, out_dst, n, to, final_stage);
        if (rc != LLMIG_OK)
            return rc;
        *out_n = n;
        return LLMIG_OK;
    });
}

int llmig_migration_stage(llmig_migration *m, const llmig_pool *src, const llmig_pool *dst,
                          const int32_t *src_table, int64_t src_table_len, int64_t len, int final_stage,
                          const int32_t *dst_free_list, int64_t dst_free_len, void *stream, int64_t *out_n)
{
    return no_throw([&]() -> int {
        if (!m || !out_n)
            return LLMIG_EINVAL;
        *out_n = 0;
        const LaunchEvents ev = m->next_events; // this call's, whatever happens below
        m->next_events = LaunchEvents();
        if (!src || !dst || !pools_compatible(src, dst) || src->block_size != m->block_size)
            return LLMIG_EINVAL;
        int64_t from = 0, to = 0;
        int rc = next_range(m, len, final_stage, &from, &to);
        if (rc != LLMIG_OK)
            return rc;
        // Scratch for the stage's pairs: never more than the free list can give
        // (a longer stage fails in llmig_plan before anything is written).
        const int64_t bs = m->block_size;
        const int64_t need = to / bs + (to % bs != 0) - from / bs;
        if (need < 0 || dst_free_len < 0)
            return LLMIG_EINVAL;
        const size_t cap = static_cast<size_t>(std::max<int64_t>(std::min(need, dst_free_len), 1));
        if (m->plan_src.size() < cap) {
            try {
                m->plan_src.resize(cap);
                m->plan_dst.resize(cap);
            } catch (...) {
                return LLMIG_EINVAL;
            }
        }
        int64_t n = 0;
        rc = llmig_plan(src_table, src_table_len, dst_free_list, dst_free_len, len, from, to, m->block_size,
                        m->plan_src.data(), m->plan_dst.data(), static_cast<int64_t>(cap), &n);
        if (rc != LLMIG_OK)
            return rc;
        rc = check_pair_ids(src, dst, m->plan_src.data(), m->plan_dst.data(), n);
        if (rc != LLMIG_OK)
            return rc;
        rc = record_stage(m, m->plan_dst.data(), n, to, final_stage);
        if (rc != LLMIG_OK)
            return rc;
        *out_n = n;
        if (n == 0)
            return LLMIG_OK;
        return launch_stage(src, dst, m->plan_src.data(), m->plan_dst.data(), n, false,
                            static_cast<hipStream_t>(stream), final_stage ? 0u : m->max_workgroups, ev);
    });
}

int llmig_migration_finish(llmig_migration *m, const llmig_pool *src, const llmig_pool *dst,
                           const int32_t *src_table, int64_t src_table_len, int64_t len,
                           const int32_t *dst_free_list, int64_t dst_free_len, void *stream, int64_t *out_n)
{
    int rc = llmig_migration_stage(m, src, dst, src_table, src_table_len, len, 1, dst_free_list, dst_free_len,
                                   stream, out_n);
    if (rc != LLMIG_OK)
        return rc;
    return no_throw([&]() -> int { return wait_stream(src->device, static_cast<hipStream_t>(stream)); });
}

int llmig_migration_set_stage_events(llmig_migration *m, void *start_event, void *stop_event)
{
    if (!m)
        return LLMIG_EINVAL;
    m->next_events.start = static_cast<hipEvent_t>(start_event);
    m->next_events.stop = static_cast<hipEvent_t>(stop_event);
    return LLMIG_OK;
}

int llmig_migration_set_max_workgroups(llmig_migration *m, int32_t max_workgroups)
{
    if (!m || max_workgroups < 0)
        return LLMIG_EINVAL;
    m->max_workgroups = static_cast<uint32_t>(max_workgroups);
    return LLMIG_OK;
}

int llmig_migration_abort(llmig_migration *m, int32_t *out, int64_t cap, int64_t *out_n)
{
    if (!m || !out_n)
        return LLMIG_EINVAL;
    *out_n = 0;
    if (m->state != LLMIG_MIGRATION_ACTIVE && m->state != LLMIG_MIGRATION_FINISHED)
        return LLMIG_EINVAL;
    const int64_t n = static_cast<int64_t>(m->reserved.size());
    if (cap < n || (n > 0 && !out))
        return LLMIG_EINVAL;
    if (n > 0)
        std::memcpy(out, m->reserved.data(), static_cast<size_t>(n) * sizeof(int32_t));
    m->reserved.clear();
    m->state = LLMIG_MIGRATION_ABORTED;
    *out_n = n;
    return LLMIG_OK;
}

int llmig_migration_commit(llmig_migration *m, int32_t *out, int64_t cap, int64_t *out_n)
{
    if (!m || !out_n)
        return LLMIG_EINVAL;
    *out_n = 0;
    if (m->state != LLMIG_MIGRATION_FINISHED)
        return LLMIG_EINVAL;
    const int64_t n = static_cast<int64_t>(m->reserved.size());
    if (cap < n || (n > 0 && !out))
        return LLMIG_EINVAL;
    if (n > 0)
        std::memcpy(out, m->reserved.data(), static_cast<size_t>(n) * sizeof(int32_t));
    m->state = LLMIG_MIGRATION_COMMITTED;
    *out_n = n;
    return LLMIG_OK;
}

int llmig_migration_info(const llmig_migration *m, int32_t *state, int64_t *copied_tokens,
                         int64_t *reserved_blocks, int64_t *stages)
{
    if (!m)
        return LLMIG_EINVAL;
    if (state)
        *state = m->state;
    if (copied_tokens)
        *copied_tokens = m->copied_tok;
    if (reserved_blocks)
        *reserved_blocks = static_cast<int64_t>(m->reserved.size());
    if (stages)
        *stages = m->stages;
    return LLMIG_OK;
}

int llmig_pack(const llmig_pool *src, const int32_t *blocks, int64_t n, int map_on_device,
               void *staging, int64_t staging_bytes, void *stream)
{
    return no_throw([&]() -> int {
        int rc = fused_copy_checks(src, blocks, n, map_on_device, staging, staging_bytes, false);
        if (rc != LLMIG_OK || n == 0)
            return rc;
        void *lin = nullptr;
        rc = staging_pointer(staging, &lin);
        if (rc != LLMIG_OK)
            return rc;
        CopyArgs a;
        std::memset(&a, 0, sizeof(a));
        a.src_tab = src->d_tab;
        a.dst_lin = static_cast<uint8_t *>(lin);
        a.tile_bytes = static_cast<uint32_t>(src->tile_bytes);
        a.num_layers = static_cast<uint32_t>(src->num_layers);
        return launch_copy<kPool, kLinear>(a, blocks, nullptr, n, map_on_device != 0,
                                           static_cast<hipStream_t>(stream));
    });
}

int llmig_unpack(const llmig_pool *dst, const int32_t *blocks, int64_t n, int map_on_device,
                 const void *staging, int64_t staging_bytes, void *stream)
{
    return no_throw([&]() -> int {
        int rc = fused_copy_checks(dst, blocks, n, map_on_device, staging, staging_bytes, true);
        if (rc != LLMIG_OK || n == 0)
            return rc;
        void *lin = nullptr;
        rc = staging_pointer(staging, &lin);
        if (rc != LLMIG_OK)
            return rc;
        CopyArgs a;
        std::memset(&a, 0, sizeof(a));
        a.dst_tab = dst->d_tab;
        a.src_lin = static_cast<const uint8_t *>(lin);
        a.tile_bytes = static_cast<uint32_t>(dst->tile_bytes);
        a.num_layers = static_cast<uint32_t>(dst->num_layers);
        return launch_copy<kLinear, kPool>(a, nullptr, blocks, n, map_on_device != 0,
                                           static_cast<hipStream_t>(stream));
    });
}

int llmig_unpack_layout(const llmig_pool *dst, const int32_t *blocks, int64_t n, int map_on_device,
                        const void *staging, int64_t staging_bytes, int32_t staging_k_layout,
                        int32_t staging_v_layout, void *stream)
{
    return no_throw([&]() -> int {
        const int32_t from[2] = {staging_k_layout, staging_v_layout};
        for (int32_t layout : from)
            if (layout < LLMIG_LAYOUT_NHD || layout > LLMIG_LAYOUT_HDN)
                return LLMIG_EINVAL;
        if (dst && from[0] == dst->layouts[0] && from[1] == dst->layouts[1])
            return llmig_unpack(dst, blocks, n, map_on_device, staging, staging_bytes, stream);
        int rc = fused_copy_checks(dst, blocks, n, map_on_device, staging, staging_bytes, true);
        if (rc != LLMIG_OK)
            return rc;
        if (!conversion_supported(dst, from))
            return LLMIG_EINVAL;
        if (n == 0)
            return LLMIG_OK;
        void *lin = nullptr;
        rc = staging_pointer(staging, &lin);
        if (rc != LLMIG_OK)
            return rc;
        ConvertArgs c = convert_args(dst, from, dst->layouts);
        c.src_lin = static_cast<const uint8_t *>(lin);
        c.dst_tab = dst->d_tab;
        return launch_convert(c, nullptr, blocks, n, map_on_device != 0, static_cast<hipStream_t>(stream), 0);
    });
}

int llmig_write_tokens(const llmig_pool *pool, const int32_t *table, int64_t table_len, int64_t from_tok,
                       int64_t n_tok, const void *data, void *stream)
{
    if (!pool || from_tok < 0 || n_tok < 0 || table_len < 0 || from_tok > INT64_MAX - n_tok ||
        !on_current_device(pool))
        return LLMIG_EINVAL;
    if (n_tok == 0)
        return LLMIG_OK;
    const int64_t slot_bytes = pool->tile_bytes / pool->block_size;
    if (!table || !data || (reinterpret_cast<uintptr_t>(data) & 15u) || slot_bytes % 16 != 0 ||
        n_tok > 0x7fffffffLL / (2 * pool->num_layers))
        return LLMIG_EINVAL;
    const bool nhd = pool->layouts[0] == LLMIG_LAYOUT_NHD && pool->layouts[1] == LLMIG_LAYOUT_NHD;
    if (!nhd && (pool->elem_bytes != 2 || pool->head_dim % 8 != 0))
        return LLMIG_EINVAL;
    const int64_t bs = pool->block_size;
    const int64_t first_blk = from_tok / bs, last_blk = (from_tok + n_tok - 1) / bs;
    if (last_blk >= table_len)
        return LLMIG_EINVAL;
    int rc = check_ids(table + first_blk, last_blk - first_blk + 1, pool->num_blocks);
    if (rc != LLMIG_OK)
        return rc;
    WriteArgs a;
    std::memset(&a, 0, sizeof(a));
    a.tab = pool->d_tab;
    a.data = static_cast<const uint8_t *>(data);
    a.slot_bytes = static_cast<uint32_t>(slot_bytes);
    a.tile_bytes = static_cast<uint32_t>(pool->tile_bytes);
    a.block_size = static_cast<uint32_t>(bs);
    a.num_layers = static_cast<uint32_t>(pool->num_layers);
    a.head_dim = static_cast<uint32_t>(pool->head_dim);
    a.row_chunks = static_cast<uint32_t>(pool->head_dim / 8);
    a.layouts[0] = pool->layouts[0];
    a.layouts[1] = pool->layouts[1];
    a.data_tokens = static_cast<uint32_t>(n_tok);
    // Each launch covers whole blocks' worth of tokens, at most kInlinePairs blocks.
    int64_t t = from_tok;
    while (t < from_tok + n_tok) {
        const int64_t blk0 = t / bs;
        const int64_t end = std::min(from_tok + n_tok, (blk0 + kInlinePairs) * bs);
        a.first_token = static_cast<uint32_t>(t - from_tok);
        a.tokens = static_cast<uint32_t>(end - t);
        a.first_slot = static_cast<uint32_t>(t - blk0 * bs);
        const int64_t nblk = (end - 1) / bs - blk0 + 1;
        std::memcpy(a.ids, table + blk0, static_cast<size_t>(nblk) * sizeof(int32_t));
        void *args[] = {&a};
        const uint32_t items = a.tokens * 2u * a.num_layers;
        hipError_t e = hipLaunchKernel(reinterpret_cast<const void *>(&write_token_slots),
                                       dim3(std::min(items, kMaxGridWorkgroups)), dim3(kThreads), args, 0,
                                       static_cast<hipStream_t>(stream));
        if (e != hipSuccess)
            return hip_error(e);
        t = end;
    }
    return LLMIG_OK;
}

int llmig_stream_read(const void *region, int64_t bytes, int32_t passes, int32_t workgroups, uint64_t *out,
                      int64_t out_words, void *stream)
{
    if (!region || !out || bytes <= 0 || bytes % 16 != 0 || passes <= 0 || workgroups <= 0 ||
        (reinterpret_cast<uintptr_t>(region) & 15u) || (reinterpret_cast<uintptr_t>(out) & 7u) ||
        out_words < static_cast<int64_t>(workgroups) * kThreads)
        return LLMIG_EINVAL;
    const uint8_t *r = static_cast<const uint8_t *>(region);
    uint64_t words = static_cast<uint64_t>(bytes) / 16u;
    uint32_t np = static_cast<uint32_t>(passes);
    void *args[] = {&r, &words, &np, &out};
    hipError_t e = hipLaunchKernel(reinterpret_cast<const void *>(&stream_read_words), dim3(workgroups),
                                   dim3(kThreads), args, 0, static_cast<hipStream_t>(stream));
    return e == hipSuccess ? LLMIG_OK : hip_error(e);
}

// Work items of a decode-attention call: one per partition of kPartTokens
// tokens of each sequence, in sequence order.  LLMIG_EINVAL for a negative
// length.
static int attn_item_count(const int32_t *ctx_lens, int32_t batch, int64_t *n_items)
{
    int64_t n = 0;
    for (int32_t b = 0; b < batch; ++b) {
        if (ctx_lens[b] < 0)
            return LLMIG_EINVAL;
        n += (static_cast<int64_t>(ctx_lens[b]) + kPartTokens - 1) / kPartTokens;
    }
    *n_items = n;
    return LLMIG_OK;
}

// Workspace of a decode-attention call: per layer, item and query head, the
// partial output (head_dim floats), its running maximum and its sum.
static int attn_workspace_bytes(int64_t num_layers, int64_t n_items, int64_t q_heads, int64_t head_dim,
                                int64_t *bytes)
{
    int64_t v = 0;
    if (__builtin_mul_overflow(num_layers, n_items, &v) || __builtin_mul_overflow(v, q_heads, &v) ||
        __builtin_mul_overflow(v, (head_dim + kAttnHeader) * 4, &v))
        return LLMIG_EINVAL;
    *bytes = v;
    return LLMIG_OK;
}

// Checks the arguments of a decode-attention call (all but the workspace);
// on success gives the kernel, the item count and the workspace size.
static int attn_check(const llmig_pool *pool, int32_t dtype, const void *q, int32_t batch, int32_t q_heads,
                      const int32_t *tables, int32_t table_stride, const int32_t *ctx_lens, const float *out,
                      const void **fn, int64_t *n_items, int64_t *ws_bytes, bool migrating = false)
{
    if (!pool || !on_current_device(pool) || (dtype != 0 && dtype != 1) || pool->elem_bytes != 2 || !q ||
        !tables || !ctx_lens || !out || batch < 1 || batch > kAttnMaxBatch || q_heads < 1 || table_stride < 1 ||
        pool->layouts[0] != LLMIG_LAYOUT_NHD || pool->layouts[1] != LLMIG_LAYOUT_NHD)
        return LLMIG_EINVAL;
    const int32_t hkv = pool->num_kv_heads;
    if (q_heads % hkv != 0)
        return LLMIG_EINVAL;
    *fn = attn_kernel_for(dtype, pool->head_dim, q_heads / hkv, migrating);
    if (!*fn || (reinterpret_cast<uintptr_t>(q) & 15u) || (reinterpret_cast<uintptr_t>(out) & 15u) ||
        (reinterpret_cast<uintptr_t>(tables) & 3u))
        return LLMIG_EINVAL;
    for (int32_t b = 0; b < batch; ++b)
        if (ctx_lens[b] < 0 || (ctx_lens[b] + pool->block_size - 1) / pool->block_size > table_stride)
            return LLMIG_EINVAL;
    if (attn_item_count(ctx_lens, batch, n_items) != LLMIG_OK || *n_items > 0x7fffffffLL)
        return LLMIG_EINVAL;
    return attn_workspace_bytes(pool->num_layers, *n_items, q_heads, pool->head_dim, ws_bytes);
}

// A stage copy carried by a decode-attention launch: logical blocks
// [from, to) of sequence seq into the blocks ids[j - from] of dst.
struct AttnMigration {
    const llmig_pool *dst = nullptr;
    int32_t seq = -1;
    const int32_t *ids = nullptr;
    int32_t from = 0, to = 0;
};

// Enqueues a checked decode-attention call: the partial kernel over the
// items, kAttnItems per launch (their ranges ride in the kernel arguments),
// then the merge.  ws holds the partial results.  Allocates nothing.
static int attn_enqueue(const llmig_pool *pool, const void *fn, const void *q, int32_t batch, int32_t q_heads,
                        const int32_t *tables, int32_t table_stride, const int32_t *ctx_lens, float scale,
                        float *ws, int64_t n_items, float *out, hipStream_t st,
                        const AttnMigration &mig = AttnMigration())
{
    AttnArgs a;
    std::memset(&a, 0, sizeof(a));
    a.mig_seq = -1;
    if (mig.dst) {
        a.dst_tab = mig.dst->d_tab;
        a.mig_ids = mig.ids;
        a.mig_seq = mig.seq;
        a.mig_from = mig.from;
        a.mig_to = mig.to;
        a.dst_layer_bytes = static_cast<uint32_t>(static_cast<uint64_t>(mig.dst->num_blocks) * mig.dst->tile_bytes);
        a.dst_blocks = mig.dst->num_blocks;
    }
    const size_t lds_ids = attn_blk_slots(pool->block_size) * sizeof(int32_t) * (mig.dst ? 2 : 1);
    a.k_tab = pool->d_tab;
    a.q = static_cast<const uint8_t *>(q);
    a.tables = tables;
    a.ws = ws;
    a.scale = scale;
    a.num_layers = static_cast<uint32_t>(pool->num_layers);
    a.batch = static_cast<uint32_t>(batch);
    a.q_heads = static_cast<uint32_t>(q_heads);
    a.kv_heads = static_cast<uint32_t>(pool->num_kv_heads);
    a.block_size = static_cast<uint32_t>(pool->block_size);
    a.table_stride = static_cast<uint32_t>(table_stride);
    a.n_items_total = static_cast<uint32_t>(n_items);
    uint32_t m = 0, first = 0;
    auto flush = [&]() -> hipError_t {
        if (m == 0)
            return hipSuccess;
        a.item_base = first;
        a.items = m;
        void *args[] = {&a};
        hipError_t e = hipLaunchKernel(fn, dim3(m * a.kv_heads, a.num_layers), dim3(kThreads), args, lds_ids, st);
        first += m;
        m = 0;
        return e;
    };
    for (int32_t b = 0; b < batch; ++b)
        for (int32_t t = 0; t < ctx_lens[b]; t += kPartTokens) {
            a.item_seq[m] = b;
            a.item_start[m] = t;
            a.item_end[m] = std::min(ctx_lens[b], t + kPartTokens);
            if (++m == static_cast<uint32_t>(kAttnItems)) {
                hipError_t e = flush();
                if (e != hipSuccess)
                    return hip_error(e);
            }
        }
    hipError_t e = flush();
    if (e != hipSuccess)
        return hip_error(e);
    AttnReduceArgs r;
    std::memset(&r, 0, sizeof(r));
    r.ws = ws;
    r.out = out;
    r.num_layers = a.num_layers;
    r.batch = a.batch;
    r.q_heads = a.q_heads;
    r.head_dim = static_cast<uint32_t>(pool->head_dim);
    r.n_items_total = a.n_items_total;
    for (int32_t b = 0, i = 0; b < batch; ++b) {
        r.seq_first[b] = i;
        r.seq_count[b] = (ctx_lens[b] + kPartTokens - 1) / kPartTokens;
        i += r.seq_count[b];
    }
    // one lane per four dimensions of an output row
    const uint64_t total = static_cast<uint64_t>(pool->num_layers) * batch * q_heads * (pool->head_dim / 4);
    const uint32_t grid = static_cast<uint32_t>(std::min<uint64_t>((total + kThreads - 1) / kThreads, 1u << 20));
    void *rargs[] = {&r};
    e = hipLaunchKernel(reinterpret_cast<const void *>(&attn_reduce), dim3(grid), dim3(kThreads), rargs, 0, st);
    return e == hipSuccess ? LLMIG_OK : hip_error(e);
}

int llmig_decode_attention_workspace(const int32_t *ctx_lens, int32_t batch, int32_t num_layers, int32_t q_heads,
                                     int32_t head_dim, int64_t *bytes)
{
    if (!bytes)
        return LLMIG_EINVAL;
    *bytes = 0;
    if (!ctx_lens || batch < 1 || batch > kAttnMaxBatch || num_layers < 1 || q_heads < 1 || head_dim < 1)
        return LLMIG_EINVAL;
    int64_t n_items = 0;
    if (attn_item_count(ctx_lens, batch, &n_items) != LLMIG_OK)
        return LLMIG_EINVAL;
    return attn_workspace_bytes(num_layers, n_items, q_heads, head_dim, bytes);
}

int llmig_decode_attention(const llmig_pool *pool, int32_t dtype, const void *q, int32_t batch, int32_t q_heads,
                           const int32_t *tables, int32_t table_stride, const int32_t *ctx_lens, float scale,
                           void *workspace, int64_t workspace_bytes, float *out, void *stream)
{
    const void *fn = nullptr;
    int64_t n_items = 0, need = 0;
    int rc = attn_check(pool, dtype, q, batch, q_heads, tables, table_stride, ctx_lens, out, &fn, &n_items, &need);
    if (rc != LLMIG_OK)
        return rc;
    if ((reinterpret_cast<uintptr_t>(workspace) & 15u) || (n_items > 0 && (!workspace || workspace_bytes < need)))
        return LLMIG_EINVAL;
    return attn_enqueue(pool, fn, q, batch, q_heads, tables, table_stride, ctx_lens, scale,
                        static_cast<float *>(workspace), n_items, out, static_cast<hipStream_t>(stream));
}

int llmig_decode_attention_migrate(const llmig_pool *pool, int32_t dtype, const void *q, int32_t batch,
                                   int32_t q_heads, const int32_t *tables, int32_t table_stride,
                                   const int32_t *ctx_lens, float scale, void *workspace, int64_t workspace_bytes,
                                   float *out, const llmig_pool *dst, int32_t seq, const int32_t *dst_ids,
                                   int64_t from_block, int64_t to_block, void *stream)
{
    if (!dst || !pool || !ctx_lens || seq < 0 || seq >= batch || from_block < 0 || from_block > to_block)
        return LLMIG_EINVAL;
    if (from_block == to_block)     // nothing to carry: plain decode attention
        return llmig_decode_attention(pool, dtype, q, batch, q_heads, tables, table_stride, ctx_lens, scale,
                                      workspace, workspace_bytes, out, stream);
    const void *fn = nullptr;
    int64_t n_items = 0, need = 0;
    int rc = attn_check(pool, dtype, q, batch, q_heads, tables, table_stride, ctx_lens, out, &fn, &n_items, &need,
                        true);
    if (rc != LLMIG_OK)
        return rc;
    if ((reinterpret_cast<uintptr_t>(workspace) & 15u) || !workspace || workspace_bytes < need)
        return LLMIG_EINVAL;
    // the destination: a second NHD pool of the same geometry on this device,
    // apart from the source; the stage's blocks lie within the sequence's
    // current length (its last block may be partly filled)
    if (dst == pool || !on_current_device(dst) || !same_geometry(pool, dst) || !same_layouts(pool, dst) ||
        pools_overlap(pool, dst) || !dst_ids || (reinterpret_cast<uintptr_t>(dst_ids) & 3u) ||
        to_block > (static_cast<int64_t>(ctx_lens[seq]) + pool->block_size - 1) / pool->block_size ||
        static_cast<uint64_t>(dst->num_blocks) * dst->tile_bytes > 0x7fffffffull)
        return LLMIG_EINVAL;
    AttnMigration mig;
    mig.dst = dst;
    mig.seq = seq;
    mig.ids = dst_ids;
    mig.from = static_cast<int32_t>(from_block);
    mig.to = static_cast<int32_t>(to_block);
    return attn_enqueue(pool, fn, q, batch, q_heads, tables, table_stride, ctx_lens, scale,
                        static_cast<float *>(workspace), n_items, out, static_cast<hipStream_t>(stream), mig);
}

int llmig_decode_attention_noalloc(const llmig_pool *pool, int32_t dtype, const void *q, int32_t batch,
                                   int32_t q_heads, const int32_t *tables, int32_t table_stride,
                                   const int32_t *ctx_lens, float scale, float *out, void *stream)
{
    return no_throw([&]() -> int { // the mutex is the only thing here that could throw
        const void *fn = nullptr;
        int64_t n_items = 0, need = 0;
        int rc = attn_check(pool, dtype, q, batch, q_heads, tables, table_stride, ctx_lens, out, &fn, &n_items,
                            &need);
        if (rc != LLMIG_OK)
            return rc;
        if (need > static_cast<int64_t>(LLMIG_DECODE_SCRATCH_BYTES))
            return LLMIG_ESCRATCH;
        void *ws = nullptr;
        rc = scratch_pointer(pool->device, &ws);
        if (rc != LLMIG_OK)
            return rc;
        return attn_enqueue(pool, fn, q, batch, q_heads, tables, table_stride, ctx_lens, scale,
                            static_cast<float *>(ws), n_items, out, static_cast<hipStream_t>(stream));
    });
}

const char *llmig_strerror(int code)
{
    switch (code) {
    case LLMIG_OK:
        return "ok";
    case LLMIG_EINVAL:
        return "invalid argument";
    case LLMIG_ENOSPC:
        return "destination free list cannot hold the stage";
    case LLMIG_ERANGE:
        return "block id out of range";
    case LLMIG_EHIP:
        return "HIP runtime error";
    case LLMIG_ESCRATCH:
        return "the call needs more than the library's static scratch array (LLMIG_DECODE_SCRATCH_BYTES) holds";
    default:
        return "unknown error";
    }
}

int llmig_last_hip_error(void)
{
    return g_last_hip_error;
}

} // extern "C"
