/*
 * llmig: multi-stage live migration of a request's paged KV cache between two
 * block pools on one AMD Instinct MI355X (gfx950).
 *
 * What it implements (Llumnix, arXiv 2406.03243, §4.2 "Live Migration of LLM
 * Requests"): the KV cache of a decoding request only ever grows at its end,
 * so the blocks it has already filled can be copied to the destination
 * instance while decoding goes on.  Stage 0 copies every filled block; each
 * later stage copies the blocks filled during the previous one; the final
 * stage, run after the request has been drained from its batch, copies what
 * is left.  Only that last stage is downtime.  Before every stage the
 * destination reserves the blocks the stage needs (the handshake's
 * pre-allocation, §4.2).  §5 "Block fusion" gathers a request's scattered
 * per-layer K/V blocks into one contiguous buffer so they move as one
 * message; llmig_pack / llmig_unpack are that gather and its inverse, and
 * llmig_stage copies pool to pool directly, since both pools sit on one GPU.
 *
 * Pool layout (vLLM paged KV cache, §2 "Batching and memory management"):
 * every layer l has a K tensor and a V tensor of shape
 * [num_blocks, block_size, num_kv_heads, head_dim], each element elem_bytes
 * wide.  One (layer, K or V, block) tile is
 *     tile_bytes = block_size * num_kv_heads * head_dim * elem_bytes
 * contiguous bytes (128 KB for 16 tokens of 16-bit LLaMA-7B, §5).  Between
 * pools of one layout the copy moves whole tiles as raw bytes and never
 * converts them, so any element format (fp16, bf16) and any bit pattern
 * (NaN payloads, -0, subnormals) arrives unchanged; between pools whose
 * intra-tile layouts differ (LLMIG_LAYOUT_*) it moves each 16-bit element,
 * again unchanged, to its place in the destination's layout.
 *
 * Error convention: every entry point returns LLMIG_OK (0) or a negative
 * code.  All argument checks run before anything is enqueued, so a call that
 * fails a check has no effect; only LLMIG_EHIP, a runtime error during a
 * call's launches, may leave part of the call enqueued.  Nothing throws or
 * aborts across this interface.
 *
 * Threads and streams: llmig_plan is pure.  The other calls only enqueue on
 * the stream they are given and may be called from several threads on
 * distinct streams; a pool handle is immutable after creation and may be
 * shared.  Ordering against the writes of decoding is the caller's job
 * (events between the decode stream and the migration stream), and a
 * non-final stage must only contain blocks that decoding will not write
 * again (the full blocks), which llmig_plan enforces.
 */
#ifndef LLMIG_H
#define LLMIG_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define LLMIG_OK 0
#define LLMIG_EINVAL (-1) /* bad argument, range, alignment, shape or duplicate id; also
                             host memory for a call's bookkeeping ran out (no C++
                             exception ever leaves the library) */
#define LLMIG_ENOSPC (-2) /* the destination free list cannot hold the stage (§4.2: the
                             pre-allocation fails and the migration aborts) */
#define LLMIG_ERANGE (-3) /* a block id outside [0, num_blocks) */
#define LLMIG_EHIP (-4)   /* the HIP runtime reported an error: see llmig_last_hip_error */
#define LLMIG_ESCRATCH (-5) /* the call needs more than the library's static scratch array
                               (LLMIG_DECODE_SCRATCH_BYTES) holds; nothing was enqueued */

/* Intra-tile layouts.  A (layer, K or V, block) tile holds block_size
 * tokens x num_kv_heads heads x head_dim dims; x = 16 / elem_bytes dims make
 * one 16-byte group.  Element (t, h, d) sits at element index
 *   LLMIG_LAYOUT_NHD   (t * H + h) * D + d                 [block_size][H][D]
 *                      (token-major: the pool layout above, FlashAttention-
 *                      style engines)
 *   LLMIG_LAYOUT_HND   (h * block_size + t) * D + d        [H][block_size][D]
 *   LLMIG_LAYOUT_HCNX  ((h * D/x + d/x) * block_size + t) * x + d % x
 *                                                          [H][D/x][block_size][x]
 *                      (the key cache of vLLM's paged attention kernel)
 *   LLMIG_LAYOUT_HDN   (h * D + d) * block_size + t        [H][D][block_size]
 *                      (the value cache of vLLM's paged attention kernel)
 * Migration between instances of one engine (§4.2) never converts; a pair
 * of pools whose layouts differ converts inside the stage copy. */
#define LLMIG_LAYOUT_NHD 0
#define LLMIG_LAYOUT_HND 1
#define LLMIG_LAYOUT_HCNX 2
#define LLMIG_LAYOUT_HDN 3

/* Describes a caller-owned pool.  k_ptrs and v_ptrs are HOST arrays of
 * num_layers DEVICE addresses, one per layer tensor of num_blocks tiles;
 * each address must be 16-byte aligned and tile_bytes a multiple of 16.  The
 * arrays are read during llmig_pool_create only.  k_layout and v_layout
 * (LLMIG_LAYOUT_*, 0 = NHD) give the order of the elements inside the K and
 * V tiles; HCNX needs elem_bytes to divide 16 and head_dim * elem_bytes to
 * be a multiple of 16. */
typedef struct llmig_pool_desc {
    int32_t num_layers;
    int32_t num_blocks;
    int32_t block_size;
    int32_t num_kv_heads;
    int32_t head_dim;
    int32_t elem_bytes;
    const uint64_t *k_ptrs;
    const uint64_t *v_ptrs;
    int32_t k_layout;
    int32_t v_layout;
} llmig_pool_desc;

typedef struct llmig_pool llmig_pool;

/* Registers a pool on the current HIP device: validates the description and
 * copies the per-layer address table to device memory once.  The library
 * owns only that table; the pool memory stays the caller's and must outlive
 * the handle.  The first pool registered on a device also looks up that
 * device's copy of the scratch array of llmig_decode_attention_noalloc and
 * maps the completion slots of llmig_migration_finish (a few KB of pinned
 * host memory, allocated once per process and kept until it ends); should
 * either fail, the calls that use them fall back or report it themselves.
 * Errors: LLMIG_EINVAL (a non-positive size, a null array or address,
 * misalignment, a tile over 2^31 bytes), LLMIG_EHIP.
 *
 * Every call that enqueues work on a pool (stage, pack, unpack, write_tokens,
 * decode attention, the coordinator's stage) must be made with the pool's
 * device current, else LLMIG_EINVAL, and on a stream of that device (not
 * checked). */
int llmig_pool_create(const llmig_pool_desc *desc, llmig_pool **out);

/* Frees the handle and its device table (not the pool memory).  The caller
 * must make sure no enqueued work still uses the handle.  NULL is allowed. */
void llmig_pool_destroy(llmig_pool *pool);

/* Bytes of one (layer, K/V, block) tile of the pool, or -1 for NULL. */
int64_t llmig_pool_tile_bytes(const llmig_pool *pool);

/* Plans one migration stage (§4.2: before each stage the destination
 * pre-allocates the blocks the stage migrates).  Pure host function: no GPU
 * call, reentrant; it allocates host scratch only to check a stage of more
 * than 32 blocks for repeated ids.
 *
 * The request has `len` tokens resident in the source pool; logical block j
 * holds tokens [j*block_size, (j+1)*block_size) and lives in source block
 * src_table[j].  The stage covers tokens [from_tok, to_tok): its logical
 * blocks are from_tok/block_size .. ceil(to_tok/block_size)-1, and the k-th
 * of them is paired with dst_free_list[k] (destination blocks are taken from
 * the head of the free list, in ascending logical order).  On success
 * out_src[k], out_dst[k] for k < *out_n hold the pairs; *out_n is also the
 * number of free-list entries consumed, which the caller drops from the
 * head of its free list.
 *
 * A non-final stage copies only whole blocks: from_tok must be a multiple of
 * block_size, and so must to_tok unless to_tok == len (the final stage,
 * which also takes the partially filled last block).
 *
 * Checks, in order (the first failure decides): out_n non-NULL; block_size
 * >= 1 and 0 <= from_tok <= to_tok <= len; the block-boundary rule above;
 * no negative length or capacity; src_table_len >= ceil(len/block_size)
 * (and src_table non-NULL if that is positive) -- all LLMIG_EINVAL; the
 * free list holds the stage -- else LLMIG_ENOSPC; out_cap holds the stage
 * and the arrays are non-NULL when the stage is not empty -- LLMIG_EINVAL;
 * no negative id among the stage's pairs -- LLMIG_ERANGE; no id repeated
 * among the stage's sources nor among its destinations -- LLMIG_EINVAL.
 * On error *out_n = 0 (if out_n is non-NULL) and nothing else is written. */
int llmig_plan(const int32_t *src_table, int64_t src_table_len,
               const int32_t *dst_free_list, int64_t dst_free_len,
               int64_t len, int64_t from_tok, int64_t to_tok, int32_t block_size,
               int32_t *out_src, int32_t *out_dst, int64_t out_cap, int64_t *out_n);

/* Copies one stage pool to pool (§4.2): for every i < n, every layer and
 * both K and V, tile map_dst[i] of dst receives the bytes of tile map_src[i]
 * of src.  Enqueue only: returns once the work is launched on `stream` (a
 * hipStream_t; NULL is the null stream).
 *
 * map_on_device = 0: map_src/map_dst are host arrays, which may be reused as
 * soon as the call returns (the ids travel inside the kernel arguments); ids
 * are range-checked (LLMIG_ERANGE) and repeated destination ids rejected
 * (LLMIG_EINVAL).  map_on_device = 1: device arrays of int32 that must stay
 * valid until the work completes; the caller guarantees the ids are in range
 * and that no destination id repeats.
 *
 * src and dst must be different pools whose layer, block_size, head and
 * element sizes match (num_blocks may differ) and whose memory does not
 * overlap; else LLMIG_EINVAL.  n = 0 does nothing.  A batched migration of
 * several requests concatenates their pairs into one call.
 *
 * When the pools' K or V layouts differ, every element of each tile moves
 * to its place in the destination's layout (see LLMIG_LAYOUT_*).  That
 * needs elem_bytes == 2, head_dim % 8 == 0, block_size % 8 == 0 if either
 * side uses HDN, and block_size * head_dim * 2 <= 16384 (one head's slab of
 * a tile); else LLMIG_EINVAL. */
int llmig_stage(const llmig_pool *src, const llmig_pool *dst,
                const int32_t *map_src, const int32_t *map_dst, int64_t n,
                int map_on_device, void *stream);

/* Block fusion, sending side (§5 "Block fusion"): gathers tiles of the
 * listed source blocks into the contiguous buffer `staging`, laid out
 * [num_layers][K=0, V=1][n][tile_bytes] with i in the order of blocks[].
 * Tiles keep the pool's own intra-tile layout (pack and unpack never
 * convert).
 * staging is device memory or pinned host memory mapped for the device
 * (hipHostMalloc); it is caller-owned, 16-byte aligned, and staging_bytes
 * must be at least n * num_layers * 2 * tile_bytes (else LLMIG_EINVAL).
 * blocks / map_on_device as for llmig_stage (ids checked against the pool
 * when on the host; repeats are allowed). */
int llmig_pack(const llmig_pool *src, const int32_t *blocks, int64_t n, int map_on_device,
               void *staging, int64_t staging_bytes, void *stream);

/* Block fusion, receiving side: scatters a buffer laid out as llmig_pack
 * writes it into the listed destination blocks.  Repeated ids are rejected
 * (LLMIG_EINVAL) when the list is on the host. */
int llmig_unpack(const llmig_pool *dst, const int32_t *blocks, int64_t n, int map_on_device,
                 const void *staging, int64_t staging_bytes, void *stream);

/* Block fusion, receiving side between engines of different layouts: as
 * llmig_unpack, but the staging tiles hold their elements in the layouts
 * staging_k_layout / staging_v_layout (those of the pool that packed them)
 * and every element lands where dst's own layouts put it (see
 * LLMIG_LAYOUT_*).  The receiver converts, so a sender ships its tiles
 * untouched with its two layout codes.  Staging layouts equal to dst's make
 * it llmig_unpack.  Converting needs the conditions of a cross-layout
 * llmig_stage (elem_bytes == 2, head_dim % 8 == 0, block_size % 8 == 0 when
 * a side is HDN, block_size * head_dim * 2 <= 16384); else LLMIG_EINVAL, as
 * for an unknown layout code.  Other arguments and errors as llmig_unpack. */
int llmig_unpack_layout(const llmig_pool *dst, const int32_t *blocks, int64_t n, int map_on_device,
                        const void *staging, int64_t staging_bytes, int32_t staging_k_layout,
                        int32_t staging_v_layout, void *stream);

/* Stand-in for decoding's KV write (§4.2: every iteration appends its
 * token's K and V and leaves earlier ones unchanged): writes tokens
 * [from_tok, from_tok + n_tok) of a request into `pool` through its host
 * block table.  data is device memory laid out
 * [num_layers][K=0, V=1][n_tok][num_kv_heads][head_dim] (elem_bytes each),
 * and each element lands where the pool's layout puts it; a pool with a
 * layout other than NHD needs elem_bytes == 2 and head_dim % 8 == 0.
 * table_len must cover the last token (LLMIG_EINVAL), ids are
 * range-checked (LLMIG_ERANGE).  Used to drive multi-stage migrations
 * without a model. */
int llmig_write_tokens(const llmig_pool *pool, const int32_t *table, int64_t table_len,
                       int64_t from_tok, int64_t n_tok, const void *data, void *stream);

/* ---------------------------------------------------------------------------
 * Migration coordinator: the handshake of §4.2 as a host state machine.
 *
 *   each stage  reserves its destination blocks first (a refusal means
 *               abort), then copies;
 *   between     a request that has meanwhile finished or been preempted
 *   stages      is aborted, which hands every reserved block back;
 *   failures    of either side also end in an abort;
 *   the end     after the final stage, a commit: the destination takes the
 *               request over and the source may free its blocks.
 *
 * A llmig_migration holds the request's progress: tokens copied so far, the
 * destination blocks reserved so far (in logical order), the stage count and
 * its state.  It owns no pool memory and no free list: the caller passes the
 * destination's current free list to each stage and drops the consumed
 * entries from its head.  Stages are planned exactly as llmig_plan plans them
 * (whole blocks only in a non-final stage).  A migration is not thread-safe;
 * use one per request.
 * ------------------------------------------------------------------------- */

#define LLMIG_MIGRATION_ACTIVE 0    /* stages may follow */
#define LLMIG_MIGRATION_FINISHED 1  /* the final stage ran; commit or abort */
#define LLMIG_MIGRATION_COMMITTED 2
#define LLMIG_MIGRATION_ABORTED 3

typedef struct llmig_migration llmig_migration;

/* Starts a migration for pools of the given block size.  Host only; no GPU
 * call.  LLMIG_EINVAL for block_size < 1 or out == NULL. */
int llmig_migration_create(int32_t block_size, llmig_migration **out);

/* Frees the object.  It does not wait for enqueued copies.  NULL allowed. */
void llmig_migration_destroy(llmig_migration *m);

/* Pre-allocates and plans the next stage without copying (host only).  The
 * request now holds `len` tokens whose blocks are src_table[0..]; a
 * non-final stage covers [copied, floor(len/bs)*bs), the final one
 * [copied, len).  Its pairs go to out_src/out_dst (capacity out_cap), *out_n
 * is their count and the number of free-list entries consumed, and the
 * destination ids join the migration's reservation.  Errors leave the
 * migration unchanged: LLMIG_EINVAL (not ACTIVE, len below the tokens already
 * copied, or any llmig_plan argument error), LLMIG_ENOSPC (the destination
 * cannot reserve the stage: the caller should abort), LLMIG_ERANGE. */
int llmig_migration_next(llmig_migration *m, const int32_t *src_table, int64_t src_table_len,
                         int64_t len, int final_stage, const int32_t *dst_free_list, int64_t dst_free_len,
                         int32_t *out_src, int32_t *out_dst, int64_t out_cap, int64_t *out_n);

/* llmig_migration_next followed by llmig_stage of its pairs on `stream`, in
 * one call (the ids travel in the kernel arguments).  *out_n is the number
 * of free-list entries consumed.  src and dst are checked as llmig_stage
 * checks them, and ids against the pools, before anything is reserved.  On
 * LLMIG_EHIP the stage's blocks stay reserved (abort returns them) and part
 * of the copy may have been enqueued. */
int llmig_migration_stage(llmig_migration *m, const llmig_pool *src, const llmig_pool *dst,
                          const int32_t *src_table, int64_t src_table_len, int64_t len, int final_stage,
                          const int32_t *dst_free_list, int64_t dst_free_len, void *stream, int64_t *out_n);

/* The final stage (§4.2: the request has been drained from its batch and
 * what is left is copied; only this stage is downtime): llmig_migration_stage
 * with final_stage = 1, followed by a wait until `stream` has finished all
 * its work, so that on LLMIG_OK the request's whole KV cache is in the
 * destination pool when the call returns (the caller may commit and resume
 * the request there).  One call keeps the downtime path free of any host
 * work between the launch and the wait.  The wait ends as soon as possible:
 * behind the copy a one-lane kernel stores a ticket into pinned host memory
 * that the library allocated with the first pool, and the calling thread
 * reads it without calling the runtime, for up to 2 ms, before it falls
 * back to hipStreamSynchronize (so the thread spins while it waits).
 * Errors as llmig_migration_stage; a failed wait is LLMIG_EHIP (the stage's
 * blocks stay reserved). */
int llmig_migration_finish(llmig_migration *m, const llmig_pool *src, const llmig_pool *dst,
                           const int32_t *src_table, int64_t src_table_len, int64_t len,
                           const int32_t *dst_free_list, int64_t dst_free_len, void *stream, int64_t *out_n);

/* Caps the number of workgroups the migration's non-final stages launch
 * (0, the default, means one per work item); the final stage is the
 * request's downtime and always runs uncapped.  A capped grid keeps fewer workgroups
 * resident, which leaves CUs and HBM bandwidth to the decode work running
 * beside the migration at the cost of a slower copy: the lever for the
 * paper's goal of near-zero overhead on running requests (§6.2), since
 * stream priorities do not preempt running workgroups.  The same-layout
 * copy's workgroups hold four wavefronts, the cross-layout copy's two.
 * LLMIG_EINVAL for a negative value. */
int llmig_migration_set_max_workgroups(llmig_migration *m, int32_t max_workgroups);

/* Times the next llmig_migration_stage call on the GPU: start_event (a
 * hipEvent_t, NULL for none) is recorded on the stage's stream right before
 * its first kernel is launched and stop_event right after its last, so
 * their interval is the stage's kernel time plus one launch latency, without
 * the host work that plans and checks the stage (events recorded on the
 * stream around the call include that).  The events are the caller's,
 * created with timing enabled; they apply to that one call, which records
 * nothing if its stage is empty or fails before launching.  Host only;
 * LLMIG_EINVAL for m == NULL. */
int llmig_migration_set_stage_events(llmig_migration *m, void *start_event, void *stop_event);

/* Aborts (ACTIVE or FINISHED): writes every reserved destination block to
 * out (capacity cap; *out_n = count) so the destination can release them,
 * and moves to ABORTED.  Copies already enqueued may still write into those
 * blocks: synchronise the migration stream before reusing them.
 * LLMIG_EINVAL if already COMMITTED or ABORTED, or cap is too small (then
 * nothing changes). */
int llmig_migration_abort(llmig_migration *m, int32_t *out, int64_t cap, int64_t *out_n);

/* Commits (FINISHED only): writes the request's destination block table
 * (one id per logical block, ceil(len/bs) of them) to out and moves to
 * COMMITTED; the source may now release its blocks.  LLMIG_EINVAL when the
 * final stage has not run, or cap is too small (then nothing changes). */
int llmig_migration_commit(llmig_migration *m, int32_t *out, int64_t cap, int64_t *out_n);

/* Progress: state (LLMIG_MIGRATION_*), tokens copied, blocks reserved,
 * stages run.  Any output pointer may be NULL.  LLMIG_EINVAL for m == NULL. */
int llmig_migration_info(const llmig_migration *m, int32_t *state, int64_t *copied_tokens,
                         int64_t *reserved_blocks, int64_t *stages);

/* Stand-in for the decode work running beside a migration (its reads of
 * the KV cache, §6.2 measures decode speed during migration): reads the
 * `bytes` of device memory at `region` `passes` times with 16-byte loads on
 * `workgroups` workgroups of 256 lanes, and stores what each lane read,
 * summed as 32-bit integers, to out[lane] (so out must hold
 * workgroups * 256 words).  Every
 * lane runs exactly `passes` passes, so the work always completes.  region
 * 16-byte aligned, bytes a positive multiple of 16 (else LLMIG_EINVAL). */
int llmig_stream_read(const void *region, int64_t bytes, int32_t passes, int32_t workgroups,
                      uint64_t *out, int64_t out_words, void *stream);

/* Decode attention over a pool: the per-step KV reads of the requests that
 * keep decoding on an instance while one of them migrates (§6.2 measures
 * their decode speed during migration).  For every layer l, sequence b and
 * query head h (KV head g = h / (q_heads / num_kv_heads)):
 *     out[l][b][h][:] = sum_t p_t V_l[t][g][:],
 *     p = softmax_t(scale * q[l][b][h][:] . K_l[t][g][:]), t < ctx_lens[b],
 * token t of sequence b living in slot t % block_size of block
 * tables[b * table_stride + t / block_size].  q is device memory
 * [num_layers][batch][q_heads][head_dim] of the pool's 16-bit type (dtype 0
 * fp16, 1 bf16), 16-byte aligned; tables device int32, ids the caller
 * guarantees in range; ctx_lens a HOST array; out device float32
 * [num_layers][batch][q_heads][head_dim], 16-byte aligned; a sequence of
 * length 0 gives zeros.  workspace: device memory of at least the size
 * llmig_decode_attention_workspace returns for the same lengths, 16-byte
 * aligned.
 * Supported: NHD pools, head_dim 64 or 128, q_heads / num_kv_heads in
 * {1, 2, 4, 8, 16}, batch <= 256; else LLMIG_EINVAL.  Arithmetic in fp32. */
int llmig_decode_attention_workspace(const int32_t *ctx_lens, int32_t batch, int32_t num_layers,
                                     int32_t q_heads, int32_t head_dim, int64_t *bytes);
int llmig_decode_attention(const llmig_pool *pool, int32_t dtype, const void *q, int32_t batch,
                           int32_t q_heads, const int32_t *tables, int32_t table_stride,
                           const int32_t *ctx_lens, float scale, void *workspace,
                           int64_t workspace_bytes, float *out, void *stream);

/* A migration stage carried by a decode step (§4.2's stage copy of a request
 * that is still decoding, §6.2's cost of it to the batch): exactly
 * llmig_decode_attention on `pool`, which in the same pass also writes the
 * whole blocks [from_block, to_block) of sequence `seq` into `dst`: logical
 * block j (source block tables[seq * table_stride + j]) lands in dst block
 * dst_ids[j - from_block], every layer, K and V, byte for byte as
 * llmig_stage would copy the same pairs.  The attention reads those bytes
 * from HBM anyway; the stage adds only their writes, so it costs the decode
 * batch less than a separate stage copy beside it would (measured: 30-45%
 * less added decode time for a whole stage carried by one step).
 * dst: a second pool on the same device, of the same geometry and (NHD)
 * layouts, not overlapping `pool`, whose layer tensors hold at most
 * 2^31 - 1 bytes each (num_blocks * tile_bytes; the stores address them
 * with 32-bit offsets).  dst_ids: DEVICE int32 array of
 * to_block - from_block ids, 4-byte aligned, valid until the work
 * completes; the caller guarantees they are in [0, dst's num_blocks) and
 * distinct (as for llmig_stage with map_on_device = 1), which the
 * coordinator's llmig_migration_next gives.  The ids are not read on the
 * host, so a bad one is not reported; a block whose id lies outside the
 * pool is not written (no store can leave dst's layer tensors).  The
 * blocks must hold tokens of the sequence:
 * to_block <= ceil(ctx_lens[seq] / block_size).  A stage
 * that ends in the sequence's partly filled last block (the final stage,
 * carried by the request's last decode step on the source, so that no copy
 * is left for after it is drained) writes the rows of its ctx_lens[seq]
 * tokens; the block's slots past them keep the destination's bytes (they
 * hold no token).  from_block == to_block is llmig_decode_attention.  Errors: those of llmig_decode_attention, and
 * LLMIG_EINVAL for a bad seq, block range, dst or dst_ids; nothing is
 * enqueued on an error. */
int llmig_decode_attention_migrate(const llmig_pool *pool, int32_t dtype, const void *q, int32_t batch,
                                   int32_t q_heads, const int32_t *tables, int32_t table_stride,
                                   const int32_t *ctx_lens, float scale, void *workspace,
                                   int64_t workspace_bytes, float *out, const llmig_pool *dst,
                                   int32_t seq, const int32_t *dst_ids, int64_t from_block,
                                   int64_t to_block, void *stream);

/* ---------------------------------------------------------------------------
 * For callers that cannot allocate device memory: code being captured into a
 * HIP graph, serving loops that must not call hipMalloc, harnesses that
 * forbid it.
 *
 * llmig_decode_attention_noalloc is llmig_decode_attention without the
 * workspace: the partial results go to one static device array of
 * LLMIG_DECODE_SCRATCH_BYTES (32 MiB) that every GPU the library runs on
 * holds until the process ends.  The call allocates nothing (no hipMalloc,
 * hipFree or allocating library routine); the array's device address is
 * looked up when the first pool is registered on a GPU (or, failing that,
 * at this call's first use there).  Every call on one GPU shares that GPU's
 * array, which keeps the last call's contents: calls that overlap on one
 * GPU (two streams, two threads) race and give wrong results, so the caller
 * serialises them.  Nothing in the array has to start at zero: a call writes
 * every entry it reads.  A call whose partial results need more than the
 * array (the size llmig_decode_attention_workspace gives for the same
 * lengths) returns LLMIG_ESCRATCH and enqueues nothing.  Other arguments,
 * results and errors as llmig_decode_attention.
 * ------------------------------------------------------------------------- */
#define LLMIG_DECODE_SCRATCH_BYTES (32u << 20)
int llmig_decode_attention_noalloc(const llmig_pool *pool, int32_t dtype, const void *q, int32_t batch,
                                   int32_t q_heads, const int32_t *tables, int32_t table_stride,
                                   const int32_t *ctx_lens, float scale, float *out, void *stream);

/* Static description of a code; never NULL. */
const char *llmig_strerror(int code);

/* The hipError_t behind the calling thread's last LLMIG_EHIP (0 if none). */
int llmig_last_hip_error(void);

#ifdef __cplusplus
}
#endif

#endif /* LLMIG_H */
