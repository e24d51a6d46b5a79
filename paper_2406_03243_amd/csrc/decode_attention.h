// Paged decode attention: the decode work that runs beside a migration and
// whose slowdown Llumnix §6.2 measures.  Part of the single translation unit
// built from llmig.hip.
//
// For layer l, sequence b and query head h (KV head g = h / group):
//     out[l][b][h] = softmax_t(scale * q[l][b][h] . K_l[t][g]) . V_l[t][g]
// over the sequence's ctx tokens, reached through its block table; inputs
// are fp16 or bf16, arithmetic and output fp32.
//
// Design (decode is HBM-bound: each K/V byte feeds `group` multiply-adds):
//  * split sequences into partitions of kPartTokens tokens (flash-decoding)
//    so a long request does not leave one workgroup working alone; a work
//    item is (layer, partition of a sequence, KV head);
//  * a row of head_dim elements is read by head_dim / 8 lanes with one
//    16-byte load each, so a 256-lane workgroup covers 256 / (head_dim / 8)
//    tokens per step with fully coalesced loads;
//  * the `group` query heads sharing the KV head live in registers; every
//    lane keeps an online softmax (running max, sum and weighted V) per head
//    for the tokens it sees, merged across lanes by shuffles and across the
//    four wavefronts through LDS;
//  * a second kernel merges the partitions of each sequence.
#pragma once

#include "common.h"

namespace {

constexpr int kPartTokens = 512;     // tokens per partition
constexpr int kAttnItems = 128;      // (sequence, partition) items per launch, in the kernel arguments
constexpr int kAttnMaxBatch = 256;   // sequences per call (per-sequence item ranges ride in the arguments)

struct AttnArgs {
    const uint64_t *k_tab;      // pool tables: K bases then V bases
    const uint8_t *q;           // [L][B][Hq][D]
    const int32_t *tables;      // [B][table_stride]
    float *ws;                  // partial results: [L][n_items][Hq][D + 2]
    float scale;
    uint32_t num_layers, batch, q_heads, kv_heads, block_size, table_stride;
    uint32_t item_base;         // global index of this launch's first item
    uint32_t n_items_total;     // items of the whole call
    uint32_t items;             // items in this launch
    int32_t item_seq[kAttnItems];
    int32_t item_start[kAttnItems];
    int32_t item_end[kAttnItems];
};

template <int BF16>
__device__ __forceinline__ float to_float(uint32_t bits16)
{
    if (BF16)
        return __builtin_bit_cast(float, bits16 << 16);
    return static_cast<float>(__builtin_bit_cast(_Float16, static_cast<uint16_t>(bits16)));
}

template <int BF16>
__device__ __forceinline__ void unpack8(u32x4 w, float (&x)[8])
{
    const uint32_t v[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        x[2 * i] = to_float<BF16>(v[i] & 0xffffu);
        x[2 * i + 1] = to_float<BF16>(v[i] >> 16);
    }
}

// Merge online-softmax state (m2, l2, a2) into (m, l, a).
__device__ __forceinline__ void merge_state(float &m, float &l, float (&a)[8], float m2, float l2,
                                            const float (&a2)[8])
{
    const float mm = fmaxf(m, m2);
    if (mm == -INFINITY)
        return;
    const float c1 = __expf(m - mm), c2 = __expf(m2 - mm);
    l = l * c1 + l2 * c2;
#pragma unroll
    for (int i = 0; i < 8; ++i)
        a[i] = a[i] * c1 + a2[i] * c2;
    m = mm;
}

template <int BF16, int D, int G>
__global__ void __launch_bounds__(kThreads) attn_partial(const AttnArgs a)
{
    constexpr int LPT = D / 8;               // lanes per token row
    constexpr int TPI = kThreads / LPT;      // tokens per step
    __shared__ float sh_m[4][G], sh_l[4][G], sh_a[4][G][D];

    const uint32_t item = blockIdx.x / a.kv_heads;
    const uint32_t g = blockIdx.x - item * a.kv_heads;
    const uint32_t layer = blockIdx.y;
    const uint32_t b = static_cast<uint32_t>(a.item_seq[item]);
    const int32_t start = a.item_start[item], end = a.item_end[item];
    const uint32_t lane_tok = threadIdx.x / LPT;
    const uint32_t dslice = (threadIdx.x % LPT) * 8;

    const uint8_t *kbase = reinterpret_cast<const uint8_t *>(table_entry(a.k_tab, layer));
    const uint8_t *vbase = reinterpret_cast<const uint8_t *>(table_entry(a.k_tab, a.num_layers + layer));

    float q[G][8];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        const uint64_t qoff = ((static_cast<uint64_t>(layer) * a.batch + b) * a.q_heads + g * G + j) * D + dslice;
        unpack8<BF16>(load16(a.q + qoff * 2), q[j]);
    }
    float m[G], l[G], acc[G][8];
#pragma unroll
    for (int j = 0; j < G; ++j) {
        m[j] = -INFINITY;
        l[j] = 0.f;
#pragma unroll
        for (int i = 0; i < 8; ++i)
            acc[j][i] = 0.f;
    }

    const int32_t *table = a.tables + static_cast<uint64_t>(b) * a.table_stride;
    for (int32_t t0 = start; t0 < end; t0 += TPI) {
        const int32_t t = t0 + static_cast<int32_t>(lane_tok);
        const bool valid = t < end;
        float k[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        float v[8] = {0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f, 0.f};
        if (valid) {
            const int32_t blk = table[t / a.block_size];
            const uint64_t row = (static_cast<uint64_t>(blk) * a.block_size + t % a.block_size) * a.kv_heads + g;
            unpack8<BF16>(load16(kbase + (row * D + dslice) * 2), k);
            unpack8<BF16>(load16(vbase + (row * D + dslice) * 2), v);
        }
#pragma unroll
        for (int j = 0; j < G; ++j) {
            float s = 0.f;
#pragma unroll
            for (int i = 0; i < 8; ++i)
                s += q[j][i] * k[i];
#pragma unroll
            for (int off = LPT / 2; off > 0; off /= 2)
                s += __shfl_xor(s, off);
            if (valid) {
                s *= a.scale;
                const float mm = fmaxf(m[j], s);
                const float c = __expf(m[j] - mm), e = __expf(s - mm);
                l[j] = l[j] * c + e;
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    acc[j][i] = acc[j][i] * c + e * v[i];
                m[j] = mm;
            }
        }
    }

    // merge the token rows of a wavefront: lanes with the same dslice
#pragma unroll
    for (int j = 0; j < G; ++j) {
#pragma unroll
        for (int off = LPT; off < 64; off *= 2) {
            float a2[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
                a2[i] = __shfl_xor(acc[j][i], off);
            const float m2 = __shfl_xor(m[j], off), l2 = __shfl_xor(l[j], off);
            merge_state(m[j], l[j], acc[j], m2, l2, a2);
        }
    }
    // merge the four wavefronts through LDS
    const uint32_t wave = threadIdx.x / 64, wl = threadIdx.x % 64;
    if (wl < LPT) {
#pragma unroll
        for (int j = 0; j < G; ++j) {
            if (wl == 0) {
                sh_m[wave][j] = m[j];
                sh_l[wave][j] = l[j];
            }
#pragma unroll
            for (int i = 0; i < 8; ++i)
                sh_a[wave][j][dslice + i] = acc[j][i];
        }
    }
    __syncthreads();
    if (threadIdx.x < static_cast<uint32_t>(LPT)) {
        const uint64_t slot = (static_cast<uint64_t>(layer) * a.n_items_total + a.item_base + item) * a.q_heads;
#pragma unroll
        for (int j = 0; j < G; ++j) {
            float mm = sh_m[0][j], ll = sh_l[0][j], aa[8];
#pragma unroll
            for (int i = 0; i < 8; ++i)
                aa[i] = sh_a[0][j][dslice + i];
            for (int w = 1; w < 4; ++w) {
                float a2[8];
#pragma unroll
                for (int i = 0; i < 8; ++i)
                    a2[i] = sh_a[w][j][dslice + i];
                merge_state(mm, ll, aa, sh_m[w][j], sh_l[w][j], a2);
            }
            float *dst = a.ws + (slot + g * G + j) * (D + 2);
#pragma unroll
            for (int i = 0; i < 8; ++i)
                dst[2 + dslice + i] = aa[i];
            if (threadIdx.x == 0) {
                dst[0] = mm;
                dst[1] = ll;
            }
        }
    }
}

struct AttnReduceArgs {
    const float *ws;
    float *out;                 // [L][B][Hq][D]
    uint32_t num_layers, batch, q_heads, head_dim, n_items_total;
    int32_t seq_first[kAttnMaxBatch];   // first item of each sequence
    int32_t seq_count[kAttnMaxBatch];   // its number of items (0 for an empty sequence)
};

// One lane per (layer, sequence, query head, dimension): merges the
// partitions of the sequence and normalises.
__global__ void __launch_bounds__(kThreads) attn_reduce(const AttnReduceArgs a)
{
    const uint64_t total = static_cast<uint64_t>(a.num_layers) * a.batch * a.q_heads * a.head_dim;
    for (uint64_t x = static_cast<uint64_t>(blockIdx.x) * kThreads + threadIdx.x; x < total;
         x += static_cast<uint64_t>(gridDim.x) * kThreads) {
        const uint32_t d = x % a.head_dim;
        uint64_t r = x / a.head_dim;
        const uint32_t h = r % a.q_heads;
        r /= a.q_heads;
        const uint32_t b = r % a.batch;
        const uint32_t layer = static_cast<uint32_t>(r / a.batch);
        float m = -INFINITY, l = 0.f, acc = 0.f;
        for (int32_t p = 0; p < a.seq_count[b]; ++p) {
            const float *src = a.ws + ((static_cast<uint64_t>(layer) * a.n_items_total + a.seq_first[b] + p) *
                                           a.q_heads + h) * (a.head_dim + 2);
            const float m2 = src[0], l2 = src[1], a2 = src[2 + d];
            const float mm = fmaxf(m, m2);
            if (mm == -INFINITY)
                continue;
            const float c1 = __expf(m - mm), c2 = __expf(m2 - mm);
            l = l * c1 + l2 * c2;
            acc = acc * c1 + a2 * c2;
            m = mm;
        }
        a.out[x] = l > 0.f ? acc / l : 0.f;
    }
}

template <int BF16, int D>
const void *attn_kernel(int group)
{
    switch (group) {
    case 1:
        return reinterpret_cast<const void *>(&attn_partial<BF16, D, 1>);
    case 2:
        return reinterpret_cast<const void *>(&attn_partial<BF16, D, 2>);
    case 4:
        return reinterpret_cast<const void *>(&attn_partial<BF16, D, 4>);
    case 8:
        return reinterpret_cast<const void *>(&attn_partial<BF16, D, 8>);
    default:
        return nullptr;
    }
}

const void *attn_kernel_for(int bf16, int head_dim, int group)
{
    if (head_dim == 64)
        return bf16 ? attn_kernel<1, 64>(group) : attn_kernel<0, 64>(group);
    if (head_dim == 128)
        return bf16 ? attn_kernel<1, 128>(group) : attn_kernel<0, 128>(group);
    return nullptr;
}

} // namespace
