/*
 * treekv.h -- C ABI of libtreekv.so: tree-shared paged attention for speculative
 * expand-verify-select search on AMD Instinct MI355X (gfx950).
 *
 * The problem (SpecScale, arXiv 2609.39334): a beam search with a process reward model keeps a
 * tree of candidate reasoning paths (Sec. 2.2).  Speculation multiplies the live candidates and
 * the decode work and fragments verification (Sec. 3.2); computation
 * deduplication runs one forward pass per distinct prefix (Sec. 4.2); early pruning releases
 * losers (Sec. 4.1).  All candidates read one paged KV cache with prefix sharing (Sec. 5.1).
 * This library provides, for one attention layer:
 *   - a prefix-tree KV block manager with refcounted, deduplicated step blocks (host, integer);
 *   - row coalescing of identical candidates (host, integer);
 *   - a planner that turns per-row block tables into shared segments and a device work list;
 *   - decode (q_len 1) and verify (q_len >= 1, causal within the step) attention on the GPU;
 *   - the decode loop's other device steps: K/V append that skips deduplicated blocks, and the
 *     branching sampler of computation deduplication (GPU);
 *   - the controller of early pruning and lazy verification (host).
 *
 * Conventions
 *   - Every function returns TKV_OK (0) or a negative TKV_E* code; nothing throws or aborts across
 *     the ABI.  tkv_last_error() returns a message for the last failure on the calling thread.
 *   - Host arrays are read during the call only (copied where kept).  Device pointers are
 *     caller-owned (e.g. PyTorch tensors); the library never frees caller memory.
 *   - Device work is enqueued on the caller's hipStream_t (passed as void*, NULL = default
 *     stream) and is asynchronous; the caller keeps buffers alive until the stream reaches it.
 *   - bf16 is IEEE bfloat16 bit patterns (uint16); fp32 is IEEE binary32.
 *   - Handles (tkv_bm, tkv_plan, tkv_search) are not thread-safe; use one thread per handle.
 */
#ifndef TREEKV_H
#define TREEKV_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    TKV_OK = 0,
    TKV_EINVAL = -1, /* bad argument, shape, id or state */
    TKV_ENOMEM = -2, /* no free KV block or sequence slot (state unchanged), or host allocation failed */
    TKV_ENOSEQ = -3, /* sequence id not live */
    TKV_ECAP = -4,   /* caller output buffer too small; the n_*_out argument reports the size needed */
    TKV_EHIP = -5    /* a HIP runtime call failed; message names the call */
};

/* Message of the most recent call on this thread ("" if it succeeded).  Valid until the next call. */
const char* tkv_last_error(void);

/* ======================================================================== block manager
 * Prefix tree of reasoning-step blocks over one paged pool (paged attention and prefix sharing,
 * Sec. 5.1; identical prefixes share KV and computation, Sec. 4.2).  Rules (exact, no hashing
 * decides anything):
 *   - Step-aligned blocks: each extension starts a fresh block; n tokens take ceil(n/block_size)
 *     blocks, the last possibly partial.
 *   - Dedup key of a chunk = (preceding block id in the path, or -1 at a root; exact tokens).  A chunk
 *     of a sealed extension reuses the live sealed block with that key (hit); otherwise it takes
 *     the lowest free block id (miss).  Unsealed chunks never hit and are never indexed.
 *   - refcount(b) = number of live sequences whose table holds b; a block is freed and unindexed
 *     when it reaches 0.  New sequence ids are the lowest free id.
 *   - A sequence's open (unsealed) step is private to it: its blocks have refcount 1, are not
 *     indexed, and no sequence can be extended from it.  A decode loop grows it token by token
 *     (tkv_bm_append) and completes it (tkv_bm_seal), when its blocks are deduplicated.
 * Host-only; no device memory is touched.
 */
typedef struct tkv_bm tkv_bm;

/* num_blocks >= 1 pool blocks, block_size >= 1 tokens per block (the attention path needs 16),
 * max_seqs >= 1 live sequences.  *out receives the handle.  EINVAL, ENOMEM. */
int tkv_bm_create(int32_t num_blocks, int32_t block_size, int32_t max_seqs, tkv_bm** out);
void tkv_bm_destroy(tkv_bm* bm);

/* New sequence = parent's path + tokens[0..n).  parent = -1 starts a root (needs n >= 1).
 * seal = 1: a completed step (chunks are deduplicated and indexed); seal = 0: an in-progress step
 * (private chunks; the sequence cannot be extended).  Outputs: *child_out = new sequence id;
 * blk_out[0..*n_blk_out) = the ids of the new step's blocks in order and hit_out[] = 1 where the
 * block was reused (the caller writes K/V only where hit_out is 0).  cap = capacity of blk_out and
 * hit_out.  Errors: EINVAL (n < 0, root without tokens, parent unsealed, seal not 0/1, NULL
 * pointers), ENOSEQ (parent not live), ENOMEM (too few free blocks or no sequence slot), ECAP
 * (cap < ceil(n/block_size); *n_blk_out = that size).  On error nothing changes. */
int tkv_bm_extend(tkv_bm* bm, int32_t parent, const int32_t* tokens, int32_t n, int32_t seal,
                  int32_t* child_out, int32_t* blk_out, uint8_t* hit_out, int32_t cap, int32_t* n_blk_out);

/* Grow a live sequence in place by tokens[0..n) (one decode step appends one token per
 * candidate).  A sealed sequence starts a new open step in a fresh block; an open step fills its
 * last block first, then takes the lowest free block ids one at a time.  dst_out[0..n) = each
 * token's pool slot, block * block_size + slot within the block: where the token's K and V go
 * (tkv_kv_append).  cap = capacity of dst_out.  Errors: EINVAL (n < 0, NULL pointers), ENOSEQ,
 * ENOMEM (too few free blocks), ECAP (cap < n).  On error nothing changes. */
int tkv_bm_append(tkv_bm* bm, int32_t seq, const int32_t* tokens, int32_t n, int32_t* dst_out, int32_t cap);

/* Complete the open step of a live sequence.  Its blocks are taken in path order with the dedup
 * key of the extension rules (the predecessor being the block the path holds after the earlier
 * ones were settled): a hit replaces the sequence's own block with the live sealed block of the same
 * key (refcount +1) and frees its own; a miss indexes the block.  replaced_out[2i], [2i+1] = the
 * i-th (own block, sealed block) pair, i < *n_replaced_out; cap = capacity in pairs, at least the
 * open step's block count (ECAP otherwise, *n_replaced_out = that count, nothing changes).
 * EINVAL if the sequence is already sealed or a pointer is NULL; ENOSEQ. */
int tkv_bm_seal(tkv_bm* bm, int32_t seq, int32_t* replaced_out, int32_t cap, int32_t* n_replaced_out);

/* Branch a live sequence where its candidates' next tokens differ (on-demand branching of
 * computation deduplication, Sec. 4.2: one child per distinct sampled token, e.g. from
 * tkv_cd_sample).  The open step, if any, is sealed first (tkv_bm_seal) -- the point of divergence
 * becomes a step boundary, so the children share every block before it -- then token i starts
 * child_out[i], a new sequence whose open step holds that token (children take the lowest free ids in
 * token order).  The parent stays live; release it with tkv_prune when it is no longer a candidate.
 * A single distinct token needs no branch: append it instead.  Errors: EINVAL (n < 0, NULL),
 * ENOSEQ, ENOMEM (fewer than n free blocks or sequence slots), ECAP (cap < n); nothing changes. */
int tkv_bm_fork(tkv_bm* bm, int32_t seq, const int32_t* tokens, int32_t n, int32_t* child_out, int32_t cap);

/* Pool slots of a new step's tokens for tkv_kv_append, from tkv_bm_extend's outputs: token t of n_tok
 * goes to block blk[t / block_size] at slot t % block_size, or nowhere (-1) where that block was a
 * deduplication hit -- the block already holds the same tokens' K/V, so the write is skipped.
 * n_blk must be ceil(n_tok / block_size).  dst_out[0..n_tok).  EINVAL.  Host-only. */
int tkv_extend_slots(const int32_t* blk, const uint8_t* hit, int32_t n_blk, int32_t n_tok, int32_t block_size,
                     int32_t* dst_out);

/* Release a sequence (early pruning, Sec. 4.1): refcounts of its table drop by one in table order;
 * blocks reaching 0 are freed and written to freed_out[0..*n_freed_out) in that order.  cap =
 * capacity of freed_out; ECAP (nothing changes) if it could be too small, i.e. if cap is below the
 * sequence's table length (*n_freed_out = that length).  ENOSEQ if seq is not live. */
int tkv_prune(tkv_bm* bm, int32_t seq, int32_t* freed_out, int32_t cap, int32_t* n_freed_out);

/* Block table of a live sequence: blk_out[0..*n_out), *kv_len_out = sum of block lengths.
 * ENOSEQ, ECAP (*n_out = table length). */
int tkv_bm_table(const tkv_bm* bm, int32_t seq, int32_t* blk_out, int32_t cap, int32_t* n_out,
                 int32_t* kv_len_out);

/* Reference count of one block (0 = free).  EINVAL if blk is out of range. */
int tkv_bm_refcount(const tkv_bm* bm, int32_t blk, int32_t* rc_out);

/* Token count of every block, len_out[0..num_blocks) (0 = free).  This is the block_len array
 * that tkv_plan_create takes. */
int tkv_bm_block_len(const tkv_bm* bm, int32_t* len_out);

/* Whole state as int32 words, for bit-exact comparison in tests:
 *   num_blocks, block_size, max_seqs, n_live,
 *   refcount[num_blocks], block_len[num_blocks], indexed[num_blocks] (0/1),
 *   then per live sequence in ascending id: seq, sealed, open step's block count, n, table[n].
 * *used = bytes needed; ECAP if cap < *used (buf may be NULL to query the size). */
int tkv_bm_snapshot(const tkv_bm* bm, void* buf, size_t cap, size_t* used);

/* Computation deduplication at the attention boundary (Sec. 4.2: one forward pass per distinct
 * prefix, with a potential size standing for identical candidates): candidates with identical
 * block tables and equal q_len become one row.  Rows are numbered by first appearance.
 * Outputs: row_of_cand_out[n_cand], first_cand_out[*n_rows_out] (first candidate of each row),
 * mult_out[*n_rows_out] (multiplicity); the two row arrays need room for n_cand entries.
 * ENOSEQ for a dead sequence, EINVAL for q_len < 1 or NULL pointers. */
int tkv_bm_coalesce(const tkv_bm* bm, int32_t n_cand, const int32_t* seqs, const int32_t* q_len,
                    int32_t* row_of_cand_out, int32_t* first_cand_out, int32_t* mult_out,
                    int32_t* n_rows_out);

/* ======================================================================== attention
 * One attention layer over the paged cache for a batch of rows (Sec. 2.1 attention; decode of
 * every live candidate and single-pass step verification, Sec. 3.2).  For row r with
 * block table T, q_len L and kv_len N = sum of block_len over T, query token i (0 <= i < L) and
 * query head h (kv head h / (hq/hkv)) attend keys 0 .. N-L+i of the path (bottom-right causal;
 * decode is L = 1 and sees all N keys):
 *   o[i,h] = softmax(q[i,h] . K^T / sqrt(d)) V,   lse[i,h] = natural log of the softmax denominator
 * computed from bf16 inputs with fp32 accumulation; o is rounded to bf16 (nearest even).
 *
 * Device layouts (row-major, contiguous):
 *   q, o   [n_qtok][hq][d] bf16, rows' query tokens concatenated in q_indptr order
 *   k, v   [num_blocks][hkv][block_size][d] bf16 (the paged pool; slots past a block's length are
 *          never read)
 *   lse    [n_qtok][hq] fp32, nullable
 * Supported: block_size 16, d in {64, 128}, hq % hkv == 0, hq / hkv <= 64, hq <= 256.
 * Inputs must be finite: q and the K/V slots a row reads may not hold NaN or infinity (the kernels
 * are built on the assumption that no NaN enters the arithmetic; a NaN input gives an unspecified
 * result, not an error).  Padding slots past a block's length are never read and may hold anything.
 */
typedef struct {
    int32_t hq, hkv, d, block_size, num_blocks;
} tkv_shape;

typedef struct tkv_plan tkv_plan;

/* Build the work plan on the host (host arrays are copied):
 *   n_rows >= 0 rows; q_indptr[n_rows+1] offsets of each row's query tokens (q_indptr[0] = 0);
 *   kv_indptr[n_rows+1] offsets into kv_blocks; kv_blocks = the rows' block tables in path order;
 *   block_len[num_blocks] = tokens per block (tkv_bm_block_len); multiplicity[n_rows] = logical
 *   candidates per row (nullable: all 1; used for accounting only).
 * The planner finds the blocks that several rows share (a trie over the tables).  Rows whose own
 * query tile is small (q_len * G < 64: decode rows and short verify rows) go through the shared
 * segments: the rows that share a segment contract its K/V blocks together, in tiles of up to 128
 * query rows (workgroup kernel) or 16-32 (wave kernel), so that a block is read once per tile rather
 * than once per row (a short segment whose child segments all take 128-row tiles is read as the head
 * of each child's key run instead; option fold_blocks).  A longer verify row fills 128-row tiles of
 * its own tokens, each walking the row's whole
 * path: its shared context is then read once per tile (mostly from L2: tiles of one context are
 * launched together on one XCD), which costs no extra arithmetic, since every query token needs
 * its own dot products with every context key either way.  Long runs are split, and descriptors
 * are laid out for the device.  EINVAL: bad shape, q_len < 1, q_len > kv_len, a block
 * id out of range or with block_len outside [1, block_size], multiplicity < 1. */
int tkv_plan_create(const tkv_shape* shape, int32_t n_rows, const int32_t* q_indptr,
                    const int32_t* kv_indptr, const int32_t* kv_blocks, const int32_t* block_len,
                    const int32_t* multiplicity, tkv_plan** out);

/* Work placement, for tests and tuning: which kernel path and grid the planner uses.  The results
 * do not depend on it (every placement computes the same attention up to fp32 summation order).
 * A negative field keeps the default.
 *   wave_max_rows    widest shared chunk, in query rows, kept on the wave kernel (default 32)
 *   tile_min_items   wider chunks go to 128-row tiles only if they make at least this many items
 *                    (default 0)
 *   waves            size of the wave grid (default 2048, less the 4 waves of each workgroup slot
 *                    that the 128-row tiles take when they are fewer than the 512 slots; 0: default)
 *   tile8_max_items  a plan of at most this many tile items and no wave-grid work runs them as
 *                    8-wave workgroups (default 256)
 *   wide_chunk_blocks  longest key run, in blocks, of a shared chunk on the 128-row tiles
 *                    (default 64)
 *   fold_blocks      a shared segment on the 128-row tiles of at most this many blocks, whose child
 *                    segments all go to the 128-row tiles and hold all of its rows, is read as the
 *                    head of each child's key run instead of on its own (default 16; 0: never) */
typedef struct {
    int32_t wave_max_rows, tile_min_items, waves, tile8_max_items, wide_chunk_blocks, fold_blocks;
} tkv_plan_options;

/* tkv_plan_create with placement options (opts may be NULL: all defaults). */
int tkv_plan_create_ex(const tkv_shape* shape, int32_t n_rows, const int32_t* q_indptr,
                       const int32_t* kv_indptr, const int32_t* kv_blocks, const int32_t* block_len,
                       const int32_t* multiplicity, const tkv_plan_options* opts, tkv_plan** out);

/* Device workspace the plan needs (descriptors + partial results), in bytes (>= 256). */
size_t tkv_plan_workspace_bytes(const tkv_plan* plan);

/* Copy the plan's descriptors into d_workspace (device memory of >= tkv_plan_workspace_bytes,
 * 256-byte aligned, caller-owned) on hip_stream; the plan keeps using that workspace until the
 * next upload.  Into the workspace of the plan's last upload, after in-place tkv_plan_update calls,
 * only the descriptor words those updates changed are sent (index/value pairs through a region of
 * the workspace, written in by a small kernel on hip_stream); so the caller must not write into
 * the descriptor region between uploads.  The library records an event after the copy and waits
 * for it before the plan's host memory changes or is recycled (tkv_plan_update, the next upload,
 * tkv_plan_destroy), so a plan may be updated or destroyed right after an upload; those calls may
 * then wait for the work enqueued on hip_stream before the copy.  EINVAL (size, alignment, NULL),
 * EHIP. */
int tkv_plan_upload(tkv_plan* plan, void* d_workspace, size_t bytes, void* hip_stream);

void tkv_plan_destroy(tkv_plan* plan);

/* Bring a plan to new block tables for the same rows (same count, order, q_len and multiplicity
 * as at creation), as a decode loop needs after every step: kv_indptr[n_rows+1], kv_blocks and
 * block_len[num_blocks] as for tkv_plan_create.
 *   - In place (*in_place = 1: a scan of the tables and of block_len, no planning) when every
 *     row kept its blocks and at most appended new ones (ids in no table before), and the blocks
 *     that changed length
 *     are the last blocks of decode rows (q_len 1) whose path ends in a chunk of their own on the
 *     wave kernel (the blocks a decode step writes).  The new blocks fill that chunk up to 16
 *     blocks; one more chunk per row may open (its partial goes to a slot the plan keeps free for
 *     the row, its work to one of the plan's idle waves).  The plan then does exactly the work of
 *     a plan made from the new tables -- the same items, blocks, tokens, partial slots in path
 *     order and merges, so the same results bit for bit -- but keeps its wave assignment: where
 *     only lengths changed its image equals that plan's byte for byte.
 *   - Otherwise (*in_place = 0) the plan is made again from the new tables, as tkv_plan_create
 *     would (its options kept); its workspace size may change.
 * Either way the plan must be uploaded again before the next attention call (EINVAL until then).
 * in_place may be NULL.  Errors (the plan is then unchanged): EINVAL (NULL arguments, or what
 * tkv_plan_create rejects in the new tables), ENOMEM. */
int tkv_plan_update(tkv_plan* plan, const int32_t* kv_indptr, const int32_t* kv_blocks,
                    const int32_t* block_len, int32_t* in_place);

/* The descriptor words (int32 indices into the image) that in-place updates changed since the
 * plan's last upload (since its creation if never uploaded): *words, *n (repeats possible), and
 * *complete = 0 if they overflowed the plan's patch capacity (the next upload then copies the
 * whole image).  Valid until the next update or upload; for tests and tools. */
int tkv_plan_dirty(const tkv_plan* plan, const int32_t** words, int32_t* n, int32_t* complete);

/* The plan's host descriptor image, what tkv_plan_upload copies (valid until the plan is updated
 * or destroyed; for tests and tools), and where its sections start, in bytes: tile items, their
 * tokens and blocks (the tkv_plan_get_view formats), merge entries, merge slot list, the wave
 * items' 512-byte records (32 16-byte words: words 0-15 the key blocks {id, length, position,
 * header word}, header words KV head, token count, walked block count; words 16-31 the tokens
 * {query token, causal limit, slot, 0}), each wave's further records [off[w], off[w+1])
 * (int32, n_waves + 1), each wave's column tiles (int32, 0: no work); `end` = bytes uploaded.
 * Wave w runs record w, then its further records. */
typedef struct {
    size_t items, toks, blks, merges, merge_slots, wave_records, wave_off, wave_tiles, end;
} tkv_plan_layout;
int tkv_plan_image(const tkv_plan* plan, const void** data, tkv_plan_layout* layout);

/* Counts for accounting and tests. */
typedef struct {
    int32_t n_rows, n_qtok, n_items, n_items_shared, n_items_row, n_slots, n_merge;
    int32_t n_segments, n_shared_segments;
    int32_t n_items_wave;   /* items run by the wave kernel (a subset of the shared items) */
    int32_t n_waves;        /* waves of the wave kernel */
    int32_t n_idle_waves;   /* of those, waves with no work (kept for tkv_plan_update) */
    int64_t logical_qtok;   /* sum of multiplicity * q_len */
    int64_t uniq_kv_tokens; /* tokens in the union of the rows' blocks */
    int64_t path_kv_tokens; /* sum over rows of kv_len (what per-row gathering would read) */
    int64_t flops;          /* 4 * d * hq * sum over query tokens of visible keys */
} tkv_plan_stats;
int tkv_plan_get_stats(const tkv_plan* plan, tkv_plan_stats* out);

/* Read-only view of the plan's host descriptor arrays (valid until the plan is viewed again,
 * updated or destroyed), for tests and tools.  Formats (int32 words):
 *   items[n_items][8]  {kv_head, tok_off, n_tok, blk_off, n_blk, pos0, kind, tiles}: kind 0 shared
 *                      chunk (workgroup kernel), 1 whole-path row tile, 2 shared chunk on the wave
 *                      kernel with `tiles` column tiles of 16 query rows (0 for kinds 0 and 1)
 *   toks[n_toks][4]    {query token, largest visible key position (2^30 for a q_len-1 token,
 *                      which sees its whole path), partial slot or -1, 0}
 *   blks[n_blks][2]    {block id, block length}
 *   merges[n_merge][4] {query token, offset into merge_slots, slot count, 0}
 * An item contracts the G query heads of KV head kv_head of toks[tok_off .. +n_tok) against the
 * keys of blks[blk_off .. +n_blk) (positions pos0, pos0+1, ... along the path).  A token with slot
 * -1 gets its final output from that item; otherwise the merge entry of the token combines its
 * partial slots (n_slots of them in the workspace). */
typedef struct {
    const int32_t *items, *toks, *blks, *merges, *merge_slots;
    int32_t n_items, n_toks, n_blks, n_merge, n_merge_slots, n_slots;
} tkv_plan_view;
int tkv_plan_get_view(const tkv_plan* plan, tkv_plan_view* out);

/* Attention for an uploaded plan.  tkv_decode requires every row's q_len == 1 (EINVAL
 * otherwise); tkv_verify takes any q_len >= 1 (causal), including batches that mix decode and
 * verify rows.  Enqueued on hip_stream; calls that share one plan's workspace must not overlap.
 * EINVAL (not uploaded, NULL pointers), EHIP (launch failure). */
int tkv_decode(const tkv_plan* plan, const void* q, const void* k, const void* v, void* o,
               float* lse, void* hip_stream);
int tkv_verify(const tkv_plan* plan, const void* q, const void* k, const void* v, void* o,
               float* lse, void* hip_stream);

/* For callers that cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid hipMalloc): tkv_verify (decode batches included) with the plan's
 * workspace in a device array of the library's own instead of a caller-uploaded one.  The plan
 * need not be uploaded: each call copies its descriptors into that array (hipMemcpyAsync from the
 * plan's host image on hip_stream) and then runs the same kernels as tkv_verify, with the same
 * results.  The call allocates nothing: no hipMalloc, hipFree or allocating library routine.
 *   - The array is TKV_NOALLOC_MAX_BYTES (64 MiB) on each GPU, held until the process ends; a plan
 *     whose tkv_plan_workspace_bytes exceeds it is refused (EINVAL, nothing enqueued).
 *   - It is the calling thread's current device's array; hip_stream must belong to that device.
 *   - Every call on one GPU shares that array: calls that overlap on one GPU (two streams, or two
 *     threads) race and give undefined results.  Calls ordered on one stream are safe.  Nothing in
 *     the array needs to start at zero, and a call reads nothing that an earlier call left there.
 *   - A plan that has been uploaded once has an event: the copy is recorded with it, and the plan
 *     may be updated or destroyed right after the call, as after tkv_plan_upload.  A plan never
 *     uploaded has none (creating it would allocate): it must then not be updated or destroyed
 *     before hip_stream has passed the call (HIP stages a pageable source before hipMemcpyAsync
 *     returns, which the library's own tests rely on).
 * EINVAL (NULL plan or tensors, plan too large), EHIP (symbol lookup, copy or launch failure). */
#define TKV_NOALLOC_MAX_BYTES ((size_t)64 << 20)
int tkv_verify_noalloc(const tkv_plan* plan, const void* q, const void* k, const void* v, void* o,
                       float* lse, void* hip_stream);

/* Write the K and V of n_tok new tokens into the paged pool: the step before attention in a decode
 * loop.  Token t's rows go to pool slot d_dst[t] = block * block_size + position (tkv_bm_append for
 * tokens decoded one at a time, tkv_extend_slots for a completed step).  A slot of -1 -- a token of a
 * block that was a deduplication hit, which already holds the same tokens' K/V (Sec. 4.2) -- is not
 * written; so is any slot outside [0, num_blocks * block_size).
 *   d_dst          [n_tok] int32, device
 *   k_new, v_new   [n_tok][hkv][d] bf16, device
 *   k, v           the pool, [num_blocks][hkv][block_size][d] bf16, device (written in place)
 * shape: hkv, d, block_size and num_blocks are used (block_size 16, d in {64, 128}).  Enqueued on
 * hip_stream; tokens with the same slot race (the block manager never gives one slot twice).
 * EINVAL (shape, n_tok < 0, NULL pointers when n_tok > 0), EHIP (launch failure). */
int tkv_kv_append(const tkv_shape* shape, const int32_t* d_dst, int32_t n_tok, const void* k_new, const void* v_new,
                  void* k, void* v, void* hip_stream);

/* ======================================================================== CD branching sampler
 * On-demand branching of computation deduplication (Sec. 4.2): a sequence with potential size n
 * stands for n identical candidates; its one row of logits gives n independent draws from the
 * temperature softmax p_j = exp(l_j / T) / sum_i exp(l_i / T) (Sec. 2.1), grouped by token: one child
 * per distinct token (tkv_bm_fork), whose potential is the group's size.  Rows of any potential run
 * in one launch.
 * Draw k of row r is the inverse CDF at uniform u = d_uniform[d_draw_off[r] + k]: the first token j
 * (in token order) whose cumulative weight exceeds u times the total, the weights and their sums in
 * fp32 (exp2 of the scaled logit minus the row maximum); a token with logit -inf is never drawn.
 *   d_logits    [n_rows][vocab] fp32 (finite or -inf, no NaN), device
 *   d_draw_off  [n_rows + 1] int32, device: row r draws potential_r = off[r + 1] - off[r] tokens,
 *               0 <= potential_r <= max_potential <= 1024
 *   d_uniform   [n_draws] fp32 in [0, 1), device (the caller's random numbers; off[n_rows] used)
 *   n_draws     entries of d_uniform, d_token and d_count.  The offsets are device data, so the
 *               kernel checks them: a row whose range [off[r], off[r + 1]) is not inside [0, n_draws)
 *               reads and writes nothing and gets d_n_groups[r] = -1.
 *   d_token, d_count  [n_draws] int32, device: row r's groups at [off[r], off[r] + d_n_groups[r]),
 *               tokens ascending, counts summing to potential_r
 *   d_n_groups  [n_rows] int32, device: distinct tokens of the row (-1: no finite logit, a
 *               potential above 1024, or offsets outside the arrays)
 * Enqueued on hip_stream.  EINVAL (n_rows < 0, vocab < 1, temperature not positive and finite,
 * max_potential outside [0, 1024], n_draws < 0, NULL pointers), EHIP. */
int tkv_cd_sample(int32_t n_rows, int32_t vocab, float temperature, int32_t max_potential, const float* d_logits,
                  const float* d_uniform, const int32_t* d_draw_off, int32_t n_draws, int32_t* d_token,
                  int32_t* d_count, int32_t* d_n_groups, void* hip_stream);

/* ======================================================================== search controller
 * Early pruning (Sec. 4.1) and lazy verification (Sec. 4.3) of a speculative beam search whose
 * rounds keep the top k candidates by verifier score (k = beam size / beam width, Sec. 2.2).
 * Candidates (nodes) are numbered in creation order; the caller maps them to block-manager
 * sequences, verifies flushed batches (tkv_verify) and releases pruned ones (tkv_prune).
 *   - Rounds.  Round d's members are the children of round d-1's selected candidates (the roots for
 *     d = 0).  A candidate expands once it has a score, possibly before its round is decided
 *     (speculation); until then its children are speculative, and their sibling group is all that
 *     is sure to share their round.
 *   - Rule 1 (rank).  A scored candidate is pruned once at least k unpruned, scored candidates that
 *     surely share its round have strictly higher scores.
 *   - Rule 2 (perfect score 1.0).  Once k candidates that surely share a round are perfect, the first
 *     k of them in score arrival order are kept and every other such candidate is pruned; for the
 *     round's members this decides the round with those k selected.
 *   - A round is otherwise decided when every selected parent has expanded and every unpruned member
 *     has a score: the top k by (score descending, arrival ascending) are selected.  Deciding a round
 *     prunes its other candidates.  Pruning a candidate prunes its subtree and drops it from the
 *     queue.
 *   - Lazy verification.  A completed step is queued.  Flush is advised while the queue is not empty
 *     and: the queued tokens exceed token_threshold (policy 1), or the sibling group of a queued
 *     candidate has no candidate still generating (policy 2), or a queued candidate has been deferred
 *     max_deferrals times (policy 3).  A deferral is a tick that passes without a flush advice.
 * Host-only; not thread-safe. */
typedef struct tkv_search tkv_search;

enum {
    TKV_CAND_GENERATING = 0, /* decoding its step */
    TKV_CAND_QUEUED = 1,     /* step complete, waiting in the verification queue */
    TKV_CAND_VERIFYING = 2,  /* flushed in a batch, score not yet reported */
    TKV_CAND_VERIFIED = 3,   /* scored; its round is undecided */
    TKV_CAND_SELECTED = 4,   /* kept by its decided round */
    TKV_CAND_PRUNED = 5      /* pruned (or not selected): its sequence can be released */
};

/* k >= 1 candidates kept per round; max_nodes >= 1 candidates in all; token_threshold >= 0 (the paper
 * profiles 2,048); max_deferrals >= 0 (the paper uses 6).  EINVAL, ENOMEM. */
int tkv_search_create(int32_t k, int32_t max_nodes, int32_t token_threshold, int32_t max_deferrals,
                      tkv_search** out);
void tkv_search_destroy(tkv_search* s);

/* Create n >= 0 children of `parent` with consecutive ids from *first_out; parent = -1 creates the
 * roots (once).  The parent must have a score and not be expanded yet; n = 0 marks a candidate that
 * does not continue (it counts as expanded).  Expanding can decide a round (the caller then drains
 * tkv_search_pruned).  EINVAL (no score yet, already expanded, roots exist, n < 0), ENOSEQ (parent
 * pruned), ENOMEM (more than max_nodes candidates); on error nothing changes. */
int tkv_search_expand(tkv_search* s, int32_t parent, int32_t n, int32_t* first_out);

/* A generating candidate completed its step of n_tokens >= 1 tokens: it is queued for verification.
 * *flush_out = 1 when a lazy-verification policy advises a flush now.  EINVAL (not generating),
 * ENOSEQ (pruned). */
int tkv_search_complete(tkv_search* s, int32_t node, int32_t n_tokens, int32_t* flush_out);

/* One generator iteration: *flush_out = 1 if a policy advises a flush; otherwise every queued
 * candidate's deferral count grows by one.  EINVAL. */
int tkv_search_tick(tkv_search* s, int32_t* flush_out);

/* Take the whole queue as one verification batch: nodes_out[0..*n_out) in enqueue order.  ECAP
 * (cap < queue length, *n_out = that length, nothing changes), EINVAL. */
int tkv_search_flush(tkv_search* s, int32_t* nodes_out, int32_t cap, int32_t* n_out);

/* Verifier scores in [0, 1] of flushed candidates, applied one at a time in the given order (which
 * is their arrival order), each followed by the pruning rules and round decisions.  A candidate
 * pruned while its batch was verified takes no score.  EINVAL (a node not flushed, already scored
 * or repeated; a score outside [0, 1] or NaN); on error nothing changes. */
int tkv_search_score(tkv_search* s, int32_t n, const int32_t* nodes, const float* scores);

/* Candidates pruned since the last call, ascending: nodes_out[0..*n_out).  ECAP (cap < count,
 * *n_out = count, nothing is taken), EINVAL. */
int tkv_search_pruned(tkv_search* s, int32_t* nodes_out, int32_t cap, int32_t* n_out);

/* One candidate: state (TKV_CAND_*), parent (-1 for a root), depth, score (-1 if none).  EINVAL. */
int tkv_search_node(const tkv_search* s, int32_t node, int32_t* state_out, int32_t* parent_out,
                    int32_t* depth_out, float* score_out);

/* Round `depth`: *decided_out = 1 once decided, with its selected candidates ascending in
 * selected_out[0..*n_out) (0 while undecided).  ECAP, EINVAL. */
int tkv_search_round(const tkv_search* s, int32_t depth, int32_t* selected_out, int32_t cap, int32_t* n_out,
                     int32_t* decided_out);

/* Whole state as int32 words, for bit-exact comparison in tests:
 *   k, token_threshold, max_deferrals, n_roots (-1: none yet), queued tokens, n_nodes,
 *   per node: parent, depth, state, n_children (-1: not expanded), tokens, deferrals, arrival (-1:
 *   no score), score bits (0 when none),
 *   queue length, queue[], n_rounds (1 + the deepest decided round), per round: decided,
 *   n_selected, selected[].
 * *used = bytes needed; ECAP if cap < *used (buf may be NULL to query the size). */
int tkv_search_snapshot(const tkv_search* s, void* buf, size_t cap, size_t* used);

/* Instrumentation.  tkv_plan_profile(plan, max_calls) makes the next max_calls attention calls on
 * this plan record HIP events taken from the kernel dispatches' own start and end timestamps: the
 * main attention phase (start of its first kernel to end of its last) and the merge kernel
 * (0 turns recording off and frees the events).
 * tkv_plan_profile_read waits for the recorded events and returns the number of recorded calls
 * and the summed milliseconds of the main kernel and of the merge kernel over those calls, then
 * starts a new recording window.  EINVAL, EHIP. */
int tkv_plan_profile(tkv_plan* plan, int32_t max_calls);
int tkv_plan_profile_read(tkv_plan* plan, int32_t* n_calls, float* ms_main, float* ms_merge);

#ifdef __cplusplus
}
#endif
#endif /* TREEKV_H */
