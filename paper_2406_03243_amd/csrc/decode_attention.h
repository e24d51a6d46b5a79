// Paged decode attention: the decode work that runs beside a migration and
// whose slowdown Llumnix §6.2 measures.  Part of the single translation unit
// built from llmig.hip.
//
// For layer l, sequence b and query head h (KV head g = h / group):
//     out[l][b][h] = softmax_t(scale * q[l][b][h] . K_l[t][g]) . V_l[t][g]
// over the sequence's ctx tokens, reached through its block table; inputs
// are fp16 or bf16, accumulation and output fp32.
//
// Layout of the work: sequences are cut into partitions of kPartTokens
// tokens (flash-decoding), so a long request does not leave one workgroup
// working alone; a workgroup takes one (layer, partition, KV head) and its
// four wavefronts take alternate 16-token groups of the partition; a second
// kernel merges the partitions of each sequence.  With `group` query heads
// per KV head, every K/V byte feeds `group` multiply-adds, a small dense
// contraction that runs on the matrix cores (see attn_partial_mfma).
#pragma once

#include "common.h"

namespace {

#define LLMIG_LDS __attribute__((address_space(3)))

// s_waitcnt immediates (gfx9 encoding: vmcnt in bits 3:0 and 15:14, expcnt
// in 6:4, lgkmcnt in 11:8; a field at its maximum does not wait): until every
// vector-memory load has returned, and until every LDS access has.
constexpr int kWaitVm0 = 0x0F70;
constexpr int kWaitLgkm0 = 0xC07F;

constexpr int kPartTokens = 2048;    // tokens per partition
constexpr int kAttnItems = 128;      // (sequence, partition) items per launch, in the kernel arguments
constexpr int kAttnMaxBatch = 256;   // sequences per call (per-sequence item ranges ride in the arguments)
// A partial result record: the partition's maximum score m (natural base),
// its weight sum l, two floats of padding, then the D weighted V sums, so
// that records (D + kAttnHeader floats) and their sums start on 16 bytes.
constexpr int kAttnHeader = 4;

struct AttnArgs {
    const uint64_t *k_tab;      // pool tables: K bases then V bases
    const uint8_t *q;           // [L][B][Hq][D]
    const int32_t *tables;      // [B][table_stride]
    float *ws;                  // partial results: [L][n_items][Hq][D + kAttnHeader]
    float scale;
    uint32_t num_layers, batch, q_heads, kv_heads, block_size, table_stride;
    uint32_t item_base;         // global index of this launch's first item
    uint32_t n_items_total;     // items of the whole call
    uint32_t items;             // items in this launch
    int32_t item_seq[kAttnItems];
    int32_t item_start[kAttnItems];
    int32_t item_end[kAttnItems];
    // The stage copy a migrating launch carries (read only when it does):
    // logical blocks [mig_from, mig_to) of sequence mig_seq go to the blocks
    // mig_ids[j - mig_from] of the pool whose K and V bases dst_tab lists.
    const uint64_t *dst_tab;
    const int32_t *mig_ids;
    int32_t mig_seq, mig_from, mig_to;
    uint32_t dst_layer_bytes;   // bytes of one destination layer tensor (< 2^31)
    int32_t dst_blocks;         // blocks of the destination pool
};

struct AttnReduceArgs {
    const float *ws;
    float *out;                 // [L][B][Hq][D]
    uint32_t num_layers, batch, q_heads, head_dim, n_items_total;
    int32_t seq_first[kAttnMaxBatch];   // first item of each sequence
    int32_t seq_count[kAttnMaxBatch];   // its number of items (0 for an empty sequence)
};

// One lane per (layer, sequence, query head, four dimensions): merges the
// partitions of the sequence and normalises.  A lane reads each partition's
// m and l as one 8-byte load and its four sums as one 16-byte load, eight
// partitions at a time so their loads are in flight together; the
// head_dim / 4 lanes of one (layer, sequence, query head) read one record's
// sums whole.
__global__ void __launch_bounds__(kThreads) attn_reduce(const AttnReduceArgs a)
{
    const uint32_t quads = a.head_dim / 4;
    const uint32_t rec = a.head_dim + kAttnHeader;                       // floats per record
    const uint64_t total = static_cast<uint64_t>(a.num_layers) * a.batch * a.q_heads * quads;
    for (uint64_t x = static_cast<uint64_t>(blockIdx.x) * kThreads + threadIdx.x; x < total;
         x += static_cast<uint64_t>(gridDim.x) * kThreads) {
        const uint32_t d4 = x % quads;
        uint64_t r = x / quads;
        const uint32_t h = r % a.q_heads;
        r /= a.q_heads;
        const uint32_t b = r % a.batch;
        const uint32_t layer = static_cast<uint32_t>(r / a.batch);
        float m = -INFINITY, l = 0.f;
        float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
        const int32_t count = a.seq_count[b];
        const uint64_t stride = static_cast<uint64_t>(a.q_heads) * rec;  // one partition
        const float *base = a.ws + ((static_cast<uint64_t>(layer) * a.n_items_total + a.seq_first[b]) * a.q_heads + h) *
                                       rec;
        for (int32_t p0 = 0; p0 < count; p0 += 8) {
            float2 ml[8];
            float4 v[8];
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                ml[u] = make_float2(-INFINITY, 0.f);
                v[u] = make_float4(0.f, 0.f, 0.f, 0.f);
                if (p0 + u < count) {
                    const float *src = base + (p0 + u) * stride;
                    ml[u] = *reinterpret_cast<const float2 *>(src);
                    v[u] = *reinterpret_cast<const float4 *>(src + kAttnHeader + 4 * d4);
                }
            }
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const float mm = fmaxf(m, ml[u].x);
                if (mm == -INFINITY)
                    continue;
                const float c1 = __expf(m - mm), c2 = __expf(ml[u].x - mm);
                l = l * c1 + ml[u].y * c2;
                acc.x = acc.x * c1 + v[u].x * c2;
                acc.y = acc.y * c1 + v[u].y * c2;
                acc.z = acc.z * c1 + v[u].z * c2;
                acc.w = acc.w * c1 + v[u].w * c2;
                m = mm;
            }
        }
        reinterpret_cast<float4 *>(a.out)[x] =
            l > 0.f ? make_float4(acc.x / l, acc.y / l, acc.z / l, acc.w / l) : make_float4(0.f, 0.f, 0.f, 0.f);
    }
}

// ---------------------------------------------------------------------------
// Matrix-core variant.  Per 16-token group of a partition, one wavefront:
//   loads     the group's K and V rows whole, straight from HBM into the
//             wavefront's LDS (global_load_lds_dwordx4: 64 lanes x 16 bytes
//             per instruction, D/8 lanes per row, 256 contiguous bytes a row
//             for D = 128), tokens past the partition's end clamped to its
//             last token (their weights are 0).  The next group's rows are
//             requested as soon as this group's operands have been read out
//             of LDS, so they are in flight while this group computes, and
//             no registers hold rows in transit;
//   S^T = K . Q^T     16 tokens x 16 query rows (the group's heads, zero-padded),
//                     16x16x32 MFMA over head_dim in steps of 32; the K rows
//                     sit in LDS with their 16-byte chunks XOR-swizzled by
//                     token, so the operand reads (token = lane % 16) hit
//                     distinct banks;
//   online softmax per query row (a lane's rows of S^T are the tokens
//                     4*(lane/16) .. +3 of query row lane%16);
//   O^T += V^T . P^T  16x16x16 MFMA per 16 dims; P^T is already in the
//                     B-operand layout, and V^T comes out of the row-major V
//                     rows through gfx950's transposing LDS read
//                     (ds_read_b64_tr_b16).  P is split into a 16-bit high
//                     part and the 16-bit rounding of the remainder, two
//                     MFMAs, so the weights keep ~2^-16 (bf16) / 2^-22 (fp16)
//                     precision.
// The four wavefronts take alternate token groups of the partition and merge
// their states through LDS at the end.  The kernel waits on HBM, not on the
// matrix cores or LDS, so it is built for four wavefronts per SIMD (at most
// 128 registers: the accumulators move from AGPRs to VGPRs; 32 KiB of LDS
// per workgroup for the rows).
// Measured on MI355X, one process, alternating, on a GQA decode step (80
// layers, 8 KV heads of 128, 17 sequences, 65,280 tokens), each step against
// the kernel before it: whole-row K loads rearranged through LDS instead of
// K fragments loaded straight into the operand layout (16 rows x 64 bytes
// per load instruction) +8%; grouping each (layer, partition)'s KV heads on
// one XCD +7%; 2048-token partitions instead of 1024 +4%; rows loaded
// straight into LDS one group ahead instead of through registers, with the
// transposing V^T reads, +2% (bit-identical output).  0.63 -> 0.77 of HBM
// peak for the partial kernel.
typedef _Float16 f16x8_t __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef short i16x4_t __attribute__((ext_vector_type(4)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));

template <int BF16>
__device__ __forceinline__ f32x4_t mfma_qk(u32x4 a, u32x4 b, f32x4_t c)
{
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, a),
                                                        __builtin_bit_cast(bf16x8_t, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(__builtin_bit_cast(f16x8_t, a),
                                                       __builtin_bit_cast(f16x8_t, b), c, 0, 0, 0);
}

template <int BF16>
__device__ __forceinline__ f32x4_t mfma_pv(uint64_t a, uint64_t b, f32x4_t c)
{
    if constexpr (BF16)
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(__builtin_bit_cast(i16x4_t, a),
                                                          __builtin_bit_cast(i16x4_t, b), c, 0, 0, 0);
    else
        return __builtin_amdgcn_mfma_f32_16x16x16f16(__builtin_bit_cast(f16x4_t, a),
                                                      __builtin_bit_cast(f16x4_t, b), c, 0, 0, 0);
}

// Round a float to the 16-bit type (nearest even); returns the bits.
template <int BF16>
__device__ __forceinline__ uint32_t to16(float x)
{
    if constexpr (BF16) {
        const uint32_t u = __builtin_bit_cast(uint32_t, x);
        return (u + 0x7fffu + ((u >> 16) & 1u)) >> 16;
    } else {
        return __builtin_bit_cast(uint16_t, static_cast<_Float16>(x));
    }
}

// Block ids a partition can touch, for the dynamic LDS of attn_partial_mfma:
// a partition starts on a block boundary (kPartTokens is a multiple of every
// block size that divides it) or inside a block, so at most
// ceil(kPartTokens / block_size) + 1 blocks.  A migrating launch keeps the
// destination id of each of them beside it.
__host__ __device__ inline uint32_t attn_blk_slots(uint32_t block_size)
{
    return (kPartTokens + block_size - 1) / block_size + 1;
}

// MIG: the launch also carries a migration stage of one sequence (Llumnix
// §4.2 stage copy, done as a side effect of decode's reads).  Every
// wavefront already brings its token group's K and V rows (one KV head's
// D * 2 bytes of each token) into LDS; for the tokens of the stage's blocks
// it reads them back out of LDS and stores them, unchanged, at the same
// place in the destination blocks.  Across the kv_heads workgroups of every
// (layer, partition) that covers each whole tile, K and V, of those blocks,
// so the destination receives exactly the bytes a pool-to-pool stage copy
// would write, while HBM reads them once, for the attention (of the
// sequence's partly filled last block, which only a final stage includes,
// the rows of its tokens: the slots past them hold no token).
template <int BF16, int D, int MIG>
__global__ void __launch_bounds__(kThreads) __attribute__((amdgpu_waves_per_eu(4, 8)))
attn_partial_mfma(const AttnArgs a)
{
    constexpr int KS = D / 32;            // k-steps of the QK product
    constexpr int MT = D / 16;            // 16-dim tiles of the PV product
    constexpr int LPR = D / 8;            // lanes per row in the K and V loads (16 bytes each)
    constexpr int RPL = 64 / LPR;         // rows per load instruction
    constexpr int RB = D * 2;             // bytes of one K or V row
    constexpr int RPB = 128 / D;          // rows per 256 bytes (one pass over the 64 banks)
    constexpr float kLog2e = 1.4426950408889634f;
    // 4 wavefronts x (16 K rows + 16 V rows) in the loop; reused for the
    // final merge of 4 x D x 16 floats.
    constexpr int kRowBytes = 4 * 2 * 16 * RB, kMergeBytes = 4 * D * 16 * 4;
    static_assert(KS * 64 * 16 == 16 * RB, "KS load instructions of 1 KiB cover the 16 rows of a group");
    __shared__ __align__(16) uint8_t smem[kRowBytes > kMergeBytes ? kRowBytes : kMergeBytes];
    __shared__ float sh_m[4][16], sh_l[4][16];
    // block ids of the partition: dynamic LDS of attn_blk_slots(block_size)
    // entries (a migrating launch: twice that, the destination ids after them)
    extern __shared__ int32_t sh_blk[];

    // The dispatcher deals workgroups to the eight XCDs in turn.  Renumbered
    // here so that the kv_heads workgroups of one (layer, item), which read
    // adjacent 256-byte pieces of the same token rows, run one after another
    // on one XCD: linear workgroup w is the (w / 8)-th on XCD w % 8.  The
    // tail of the grid that does not fill whole rounds of 8 * kv_heads keeps
    // the plain order.
    uint32_t item, g, layer;
    {
        const uint32_t H = a.kv_heads, lin = blockIdx.x + blockIdx.y * gridDim.x;
        const uint32_t total = gridDim.x * gridDim.y, full = total - total % (8u * H);
        uint32_t unit;                    // (layer, item) in row-major order
        if (lin < full) {
            const uint32_t k = lin / 8u;
            g = k % H;
            unit = (k / H) * 8u + lin % 8u;
        } else {
            g = lin % H;
            unit = lin / H;
        }
        layer = unit / a.items;
        item = unit - layer * a.items;
    }
    const uint32_t b = static_cast<uint32_t>(a.item_seq[item]);
    const int32_t start = a.item_start[item], end = a.item_end[item];
    const uint32_t G = a.q_heads / a.kv_heads;
    const uint32_t wave = threadIdx.x / 64, lane = threadIdx.x % 64;
    const uint32_t r16 = lane % 16, g4 = lane / 16;

    const uint8_t *kbase = reinterpret_cast<const uint8_t *>(table_entry(a.k_tab, layer));
    const uint8_t *vbase = reinterpret_cast<const uint8_t *>(table_entry(a.k_tab, a.num_layers + layer));

    // The partition's block ids, once, so no token waits on a table load.
    const int32_t *table = a.tables + static_cast<uint64_t>(b) * a.table_stride;
    const int32_t first_blk = start / static_cast<int32_t>(a.block_size);
    const int32_t n_blk = (end - 1) / static_cast<int32_t>(a.block_size) - first_blk + 1;
    for (int32_t k = threadIdx.x; k < n_blk; k += kThreads)
        sh_blk[k] = table[first_blk + k];
    // A migrating launch: whether this workgroup's rows are the migrating
    // sequence's, and the destination block of each of its logical blocks
    // (-1 outside the stage).
    const bool mig = MIG && static_cast<int32_t>(b) == a.mig_seq;
    int32_t *sh_dst = sh_blk + attn_blk_slots(a.block_size);
    if (mig) {
        for (int32_t k = threadIdx.x; k < n_blk; k += kThreads) {
            const int32_t j = first_blk + k;
            const int32_t id = j >= a.mig_from && j < a.mig_to ? a.mig_ids[j - a.mig_from] : -1;
            sh_dst[k] = id < a.dst_blocks ? id : -1;     // an id past the pool is not written
        }
    }
    __syncthreads();

    // Q^T fragments (B operand): query row r16 of the group, dims 32*ks + 8*g4 .. +8.
    u32x4 qf[KS];
#pragma unroll
    for (int ks = 0; ks < KS; ++ks) {
        qf[ks] = u32x4{0u, 0u, 0u, 0u};
        if (r16 < G) {
            const uint64_t qoff = ((static_cast<uint64_t>(layer) * a.batch + b) * a.q_heads + g * G + r16) * D +
                                  32 * ks + 8 * g4;
            qf[ks] = load16(a.q + qoff * 2);
        }
    }
    const float qk_scale = a.scale * kLog2e;
    float m = -INFINITY, lsum = 0.f;
    f32x4_t acc[MT];
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
        acc[mt] = f32x4_t{0.f, 0.f, 0.f, 0.f};

    // The wavefront's rows of one 16-token group in LDS, D/8 chunks of 16
    // bytes a row.  K chunk c of local token t sits at slot c ^ kswz(t), so
    // that the 16 tokens an operand read touches at once fall on distinct
    // banks; V rows are plain (the transposing reads take them as they are).
    const uint32_t wv = __builtin_amdgcn_readfirstlane(wave);
    uint8_t *kbuf = smem + wv * (2 * 16 * RB);
    uint8_t *vbuf = kbuf + 16 * RB;
    auto kswz = [](uint32_t t) { return (t / RPB) % LPR; };
    // Requests the rows of the group starting at token t0: KS instructions
    // for K and KS for V, instruction j's lane carrying local token
    // j*RPL + lane/LPR into LDS slot lane%LPR of that token's row.  A token
    // past the partition's end loads its last token; its score is masked
    // below, so its weight is 0.
    auto request_group = [&](int32_t t0) {
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            const uint32_t tl = j * RPL + lane / LPR, slot = lane % LPR;
            const int32_t t = min(t0 + static_cast<int32_t>(tl), end - 1);
            const uint64_t row = (static_cast<uint64_t>(sh_blk[t / a.block_size - first_blk]) * a.block_size +
                                  t % a.block_size) * a.kv_heads + g;
            __builtin_amdgcn_global_load_lds((const void LLMIG_GLOBAL *)(kbase + (row * D + 8 * (slot ^ kswz(tl))) * 2),
                                             (void LLMIG_LDS *)(kbuf + j * 1024), 16, 0, kStreamLoad);
            __builtin_amdgcn_global_load_lds((const void LLMIG_GLOBAL *)(vbase + (row * D + 8 * slot) * 2),
                                             (void LLMIG_LDS *)(vbuf + j * 1024), 16, 0, kStreamLoad);
        }
    };
    // A migrating launch: stores the group's rows that belong to the stage's
    // blocks into the destination pool.  Lane `lane` of load instruction j
    // brought token j*RPL + lane/LPR's chunk lane%LPR of the row (K: the
    // swizzled slot of the chunk) into LDS at j * 1024 + lane * 16; it reads
    // that back and stores it where the chunk lives in the destination tile:
    // (slot of the token, head g, the chunk).  Rows of tokens past the
    // partition's end (loaded as copies of its last token) are skipped.
    auto store_group = [&](int32_t tg) {
        // raw buffer stores over the destination layer tensors, with the
        // migration copy's cache policy (streaming, device scope); a whole
        // 10.7 GB stage carried by one GQA decode step added 2.2-2.8 ms to
        // the step with them, 2.8-2.9 ms with plain non-temporal stores.
        // A row that is not the stage's gets an offset past the resource
        // (layer tensors are under 2^31 bytes), so the range check drops
        // its store and every store runs unpredicated.
        constexpr uint32_t kDropped = 0x80000000u;
        const __amdgpu_buffer_rsrc_t rk = tile_rsrc(
            reinterpret_cast<const uint8_t *>(table_entry(a.dst_tab, layer)), a.dst_layer_bytes);
        const __amdgpu_buffer_rsrc_t rv = tile_rsrc(
            reinterpret_cast<const uint8_t *>(table_entry(a.dst_tab, a.num_layers + layer)), a.dst_layer_bytes);
        const uint32_t tile = a.block_size * a.kv_heads * RB;
        const int32_t bs = static_cast<int32_t>(a.block_size);
        const int32_t q = tg / bs, r0 = tg - q * bs;          // the group's first token: block, slot
        uint32_t off[KS];
        u32x4 r[KS];
#pragma unroll
        for (int j = 0; j < KS; ++j) {
            const int32_t tl = j * RPL + static_cast<int32_t>(lane / LPR);
            const int32_t s = r0 + tl, bo = s / bs, slot = s - bo * bs;
            const int32_t d = tg + tl < end ? sh_dst[q + bo - first_blk] : -1;
            off[j] = d < 0 ? kDropped
                           : static_cast<uint32_t>(d) * tile + (static_cast<uint32_t>(slot) * a.kv_heads + g) * RB;
            r[j] = *reinterpret_cast<const u32x4 *>(kbuf + j * 1024 + lane * 16);
        }
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
#pragma unroll
        for (int j = 0; j < KS; ++j)
            buffer_store16(rk, off[j] + 16 * ((lane % LPR) ^ kswz(j * RPL + lane / LPR)), r[j]);
#pragma unroll
        for (int j = 0; j < KS; ++j)
            r[j] = *reinterpret_cast<const u32x4 *>(vbuf + j * 1024 + lane * 16);
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
#pragma unroll
        for (int j = 0; j < KS; ++j)
            buffer_store16(rv, off[j] + 16 * (lane % LPR), r[j]);
    };
    const int32_t tg0 = start + 16 * static_cast<int32_t>(wave);
    if (tg0 < end)
        request_group(tg0);
    for (int32_t tg = tg0; tg < end; tg += 64) {
        // this group's rows have landed (the only loads in flight)
        __builtin_amdgcn_s_waitcnt(kWaitVm0);
        // a migrating launch stores the stage's rows first, while no operand
        // fragments are live yet; a group none of whose tokens lies in the
        // stage's blocks skips it (a wavefront-uniform test)
        if (MIG && mig && (tg + 15) / static_cast<int32_t>(a.block_size) >= a.mig_from &&
            tg / static_cast<int32_t>(a.block_size) < a.mig_to)
            store_group(tg);
        // K fragments (A operand: token r16, dims 32*ks + 8*g4 .. +8)
        u32x4 kf[KS];
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            kf[ks] = *reinterpret_cast<const u32x4 *>(kbuf + r16 * RB + (((4 * ks + g4) ^ kswz(r16)) * 16));
        // V^T fragments (A operand of O^T: dim 16*mt + r16, tokens 4*g4 .. +3)
        // by transposing reads: lane r16 of the 16-lane group g4 receives
        // element r16 % 4 of the 8 bytes that lane 4*q + r16/4 of its group
        // addresses, for q = 0..3; those address token 4*g4 + q, dims
        // 16*mt + 4*(r16 % 4) .. +3.
        uint64_t vf[MT];
#pragma unroll
        for (int mt = 0; mt < MT; ++mt)
            vf[mt] = __builtin_bit_cast(uint64_t, __builtin_amdgcn_ds_read_tr16_b64_v4i16(
                (i16x4_t LLMIG_LDS *)(vbuf + (4 * g4 + r16 / 4) * RB + (16 * mt + 4 * (r16 % 4)) * 2)));
        // the reads have returned before the next group's rows overwrite them
        __builtin_amdgcn_s_waitcnt(kWaitLgkm0);
        if (tg + 64 < end)
            request_group(tg + 64);
        // S^T = K . Q^T
        f32x4_t s = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < KS; ++ks)
            s = mfma_qk<BF16>(kf[ks], qf[ks], s);
        // online softmax for query row r16 over tokens tg + 4*g4 + i
        float sc[4], mx = -INFINITY;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            sc[i] = tg + static_cast<int32_t>(4 * g4) + i < end ? s[i] * qk_scale : -INFINITY;
            mx = fmaxf(mx, sc[i]);
        }
        mx = fmaxf(mx, __shfl_xor(mx, 16));
        mx = fmaxf(mx, __shfl_xor(mx, 32));
        const float m_new = fmaxf(m, mx);          // finite: the group has a valid token
        const float c = exp2f(m - m_new);
        float p[4], ps = 0.f;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            p[i] = exp2f(sc[i] - m_new);
            ps += p[i];
        }
        ps += __shfl_xor(ps, 16);
        ps += __shfl_xor(ps, 32);
        lsum = lsum * c + ps;
        m = m_new;
        uint64_t ph = 0, pl = 0;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const uint32_t hi = to16<BF16>(p[i]);
            const float hv = BF16 ? __builtin_bit_cast(float, hi << 16)
                                  : static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(hi)));
            ph |= static_cast<uint64_t>(hi) << (16 * i);
            pl |= static_cast<uint64_t>(to16<BF16>(p[i] - hv)) << (16 * i);
        }
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            acc[mt] = acc[mt] * c;
            acc[mt] = mfma_pv<BF16>(vf[mt], ph, acc[mt]);
            acc[mt] = mfma_pv<BF16>(vf[mt], pl, acc[mt]);
        }
    }

    // merge the four wavefronts: state of query row r16, O^T rows 16*mt + 4*g4 + i
    __syncthreads();                                // every wave is done with its V^T region
    float *so = reinterpret_cast<float *>(smem);    // [wave][dim][16]
    if (g4 == 0) {
        sh_m[wave][r16] = m;
        sh_l[wave][r16] = lsum;
    }
#pragma unroll
    for (int mt = 0; mt < MT; ++mt)
#pragma unroll
        for (int i = 0; i < 4; ++i)
            so[(wave * D + 16 * mt + 4 * g4 + i) * 16 + r16] = acc[mt][i];
    __syncthreads();
    if (wave == 0 && r16 < G) {
        float mm = -INFINITY;
        for (int w = 0; w < 4; ++w)
            mm = fmaxf(mm, sh_m[w][r16]);
        float cw[4], ll = 0.f;
        for (int w = 0; w < 4; ++w) {
            cw[w] = mm == -INFINITY ? 0.f : exp2f(sh_m[w][r16] - mm);
            ll += sh_l[w][r16] * cw[w];
        }
        const uint64_t slot = (static_cast<uint64_t>(layer) * a.n_items_total + a.item_base + item) * a.q_heads +
                              g * G + r16;
        float *dst = a.ws + slot * (D + kAttnHeader);
#pragma unroll
        for (int mt = 0; mt < MT; ++mt) {
            float o[4];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                const uint32_t dim = 16 * mt + 4 * g4 + i;
                o[i] = 0.f;
                for (int w = 0; w < 4; ++w)
                    o[i] += so[(w * D + dim) * 16 + r16] * cw[w];
            }
            *reinterpret_cast<float4 *>(dst + kAttnHeader + 16 * mt + 4 * g4) = make_float4(o[0], o[1], o[2], o[3]);
        }
        if (g4 == 0) {
            // the reduce kernel merges with natural exponentials: store m in that base
            dst[0] = mm == -INFINITY ? -INFINITY : mm / kLog2e;
            dst[1] = ll;
        }
    }
}

template <int BF16, int D>
const void *attn_kernel(int group, bool migrating)
{
    if (group < 1 || group > 16 || (group & (group - 1)) != 0)
        return nullptr;
    return migrating ? reinterpret_cast<const void *>(&attn_partial_mfma<BF16, D, 1>)
                     : reinterpret_cast<const void *>(&attn_partial_mfma<BF16, D, 0>);
}

const void *attn_kernel_for(int bf16, int head_dim, int group, bool migrating)
{
    if (head_dim == 64)
        return bf16 ? attn_kernel<1, 64>(group, migrating) : attn_kernel<0, 64>(group, migrating);
    if (head_dim == 128)
        return bf16 ? attn_kernel<1, 128>(group, migrating) : attn_kernel<0, 128>(group, migrating);
    return nullptr;
}

} // namespace
