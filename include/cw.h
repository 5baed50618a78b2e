/*
 * cw.h - C ABI of libcw: prefill of an uncached prompt suffix over a paged,
 * prefix-cached KV store, for AMD Instinct MI355X (gfx950).
 *
 * The computation is the one that cache-aware evidence ordering shortens
 * (CacheWeaver, arXiv 2606.19667): a serving engine stores KV states in
 * fixed-size token blocks, hashes each block together with its prefix history,
 * reuses the longest leading run of stored blocks of a new prompt, and then
 * prefills only the remaining suffix tokens, which attend causally over
 * themselves and fully over the reused prefix (paper Sec. 1; Sec. 2.1 with
 * Fig. 1; Sec. 3.3, the problem statement after Eq. 1).
 *
 * Conventions for every entry point
 *  - Return value: cw_status. CW_OK on success; on failure nothing observable
 *    changed (no partial pool update, no kernel launched) and cw_last_error()
 *    describes the first problem found. No call aborts or throws.
 *  - Host pointers are read or written only during the call. Device pointers
 *    are caller-owned HIP device memory; the library never allocates or frees
 *    device memory and keeps no pointer after returning.
 *  - Device calls are asynchronous on `stream` (a hipStream_t; NULL = the
 *    default stream) and do not synchronise. They are reentrant.
 *  - Pool calls are not thread-safe for one pool; distinct pools are
 *    independent.
 *  - Layouts (all row-major, bf16 = IEEE bfloat16 bit patterns):
 *      q, out        [total_s, Hq, D]        suffix rows of all requests, request-major
 *      k_new, v_new  [total_s, Hkv, D]
 *      k_cache       [num_blocks, Hkv, block_size, D]   block rows are tokens
 *      v_cache       [num_blocks, Hkv, block_size, D]   the same
 *      block_table   int32 [batch, bt_stride]; row r lists the physical blocks of
 *                    request r's logical blocks 0 .. ceil(L_r / block_size) - 1
 *      cu_suffix     int32 [batch + 1]; request r owns rows cu[r] .. cu[r+1]-1,
 *                    S_r = cu[r+1] - cu[r] >= 0, cu[0] = 0
 *      prefix_len    int32 [batch]; P_r cached tokens, a multiple of block_size
 *    Request r's prompt has L_r = P_r + S_r tokens; suffix row i of request r is
 *    token P_r + i.
 *  - Supported shapes: block_size 16, head_dim 64 or 128, num_q_heads a
 *    multiple of num_kv_heads with at most 128 query heads per KV head.
 */
#ifndef CW_H
#define CW_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef int32_t cw_status;
#define CW_OK 0
#define CW_EINVAL (-1)       /* invalid argument */
#define CW_EUNSUPPORTED (-2) /* valid but unsupported shape */
#define CW_ENOSPC (-3)       /* block pool exhausted */
#define CW_EHIP (-4)         /* a HIP runtime call or kernel launch failed */

#define CW_ABI_VERSION 4

/* ABI version of the loaded library (CW_ABI_VERSION at build time). */
int32_t cw_abi_version(void);

/* Message describing the last non-OK status returned on the calling thread
 * (empty string if none). The pointer stays valid until the next cw_ call on
 * this thread. */
const char* cw_last_error(void);

/* ------------------------------------------------------------------------
 * Host: chained block hashes (paper Sec. 2.1: each block is hashed together
 * with its prefix history, so reuse is prefix-sensitive).
 *
 * h_b = XXH64(LE32(tokens[b*bs]) .. LE32(tokens[b*bs + bs - 1]), seed = h_{b-1}),
 * h_{-1} = 0, for the n_tokens / block_size full blocks; a trailing partial
 * block gets no hash. XXH64 is the published xxHash 64-bit function.
 *   tokens      host int32 [n_tokens]
 *   out_hashes  host uint64 [n_tokens / block_size]
 * CW_EINVAL: n_tokens < 0, block_size < 1, or a needed pointer is NULL.
 */
cw_status cw_block_hashes(const int32_t* tokens, int64_t n_tokens, int32_t block_size,
                          uint64_t* out_hashes);

/* ------------------------------------------------------------------------
 * Host: block pool (paper Sec. 2.1 and Sec. 3.4: the engine stores KV in
 * fixed-size blocks, looks up the longest stored prefix, and evicts blocks
 * itself). The pool keeps only host bookkeeping of block IDs; the KV bytes live
 * in the caller's device caches.
 *
 * Per block: a reference count and at most one stored hash. Blocks with count
 * zero wait in a free queue; a free block that still stores a hash remains
 * matchable until it is handed out again (that hand-out evicts the hash).
 */
typedef struct cw_pool cw_pool;

/* New pool of `num_blocks` blocks. free_order (host int32 [num_blocks], a
 * permutation of 0 .. num_blocks-1, or NULL for ascending) is the order in which
 * never-used blocks are handed out, i.e. the physical placement.
 * CW_EINVAL: num_blocks < 1, free_order not a permutation, out NULL. */
cw_status cw_pool_create(int32_t num_blocks, const int32_t* free_order, cw_pool** out);

/* Frees a pool (NULL is ignored). */
void cw_pool_destroy(cw_pool* pool);

/* Deep copy of a pool's state into a new pool. */
cw_status cw_pool_clone(const cw_pool* pool, cw_pool** out);

/* Number of blocks whose reference count is zero (-1 if pool is NULL). */
int32_t cw_pool_num_free(const cw_pool* pool);

/* Longest leading run of `hashes` stored in the pool, at most max_match blocks
 * (paper Sec. 2.1 and Fig. 1: an early mismatch ends all later reuse). Each
 * matched block gains one reference (leaving the free queue if it was free).
 *   hashes         host uint64 [n_hashes]
 *   out_block_ids  host int32 [n_hashes]; the first *out_depth entries are set
 *   out_depth      number of matched blocks
 * Pass max_match = (L - 1) / block_size to keep at least one suffix token.
 * CW_EINVAL: n_hashes < 0 or a needed pointer is NULL. */
cw_status cw_prefix_match(cw_pool* pool, const uint64_t* hashes, int32_t n_hashes,
                          int32_t max_match, int32_t* out_block_ids, int32_t* out_depth);

/* Hands out n blocks from the front of the free queue, each with count 1; a
 * handed-out block forgets its stored hash.
 *   out_block_ids  host int32 [n]
 * CW_ENOSPC: fewer than n free blocks (pool unchanged). CW_EINVAL: n < 0. */
cw_status cw_pool_alloc(cw_pool* pool, int32_t n, int32_t* out_block_ids);

/* Stores hashes[i] -> block_ids[i] so later prompts can match the block. Each
 * block must be held (count > 0) and store no other hash. If a hash is already
 * stored for another block, the pool keeps the first block.
 * CW_EINVAL: a block not held, out of range, or holding another hash. */
cw_status cw_pool_commit(cw_pool* pool, const uint64_t* hashes, const int32_t* block_ids,
                         int32_t n);

/* Drops one reference per listed block. Blocks reaching zero join the back of
 * the free queue in reverse listing order (the tail of a released sequence is
 * reused before its head); they keep their hash until handed out again.
 * CW_EINVAL: a block listed more times than it is held, or out of range. */
cw_status cw_pool_release(cw_pool* pool, const int32_t* block_ids, int32_t n);

/* One call for a batch of prompts, in order: for each request, chained hashes
 * of its full blocks, prefix match capped at (L_r - 1) / block_size blocks,
 * allocation of its remaining ceil(L_r / block_size) - depth blocks, and
 * commit of the hashes of its new full blocks, so later requests of the same
 * batch can reuse them (their K/V is written by cw_kv_append of this batch,
 * which must precede any attention call reading them on the stream).
 *   tokens            host int32, the prompts concatenated
 *   cu_tokens         host int64 [batch + 1], prompt r is tokens[cu[r] .. cu[r+1])
 *   out_block_table   host int32 [batch, bt_stride]; unused entries set to -1
 *   out_prefix_len    host int32 [batch]   (P_r = depth * block_size)
 *   out_cu_suffix     host int32 [batch + 1]
 * On CW_ENOSPC (or any error) every reference taken and hash stored by this
 * call is undone. CW_EINVAL: empty prompt, ceil(L_r / bs) > bt_stride, or
 * total suffix rows > INT32_MAX. */
cw_status cw_schedule_batch(cw_pool* pool, const int32_t* tokens, const int64_t* cu_tokens,
                            int32_t batch, int32_t block_size, int32_t bt_stride,
                            int32_t* out_block_table, int32_t* out_prefix_len,
                            int32_t* out_cu_suffix);

/* Releases every block of every request of a scheduled batch (the first
 * ceil(L_r / block_size) entries of each row). Arguments as produced by
 * cw_schedule_batch. */
cw_status cw_release_batch(cw_pool* pool, const int32_t* block_table, int32_t bt_stride,
                           const int32_t* prefix_len, const int32_t* cu_suffix, int32_t batch,
                           int32_t block_size);

/* ------------------------------------------------------------------------
 * Host: knowledge tree and evidence ordering (paper Sec. 3.2-3.4, Eq. 1,
 * Algorithm 1; baselines of Sec. 4 and Table `baselines`).
 *
 * The tree records the document orders of served requests as root-to-node
 * paths. A node is cached when an order inserted within the last `window`
 * insertions passed through it and it was not marked stale since (recency
 * stands in for residency, Sec. 3.4). l(O, T) is the number of leading
 * documents of O whose nodes are all cached. Documents are int64 IDs; a
 * retrieved set is given in retrieval rank and must hold distinct IDs (at
 * most 4096). The tree is host memory owned by the library; calls on one tree
 * are not thread-safe.
 * ------------------------------------------------------------------------ */
typedef struct cw_tree cw_tree;

#define CW_ORDER_RETRIEVAL 0  /* retrieval rank unchanged */
#define CW_ORDER_SORTED 1     /* lexicographic (ascending) document IDs */
#define CW_ORDER_RECENCY 2    /* documents served within the window first, latest
                                 first (ties in retrieval rank), then the rest in
                                 retrieval rank */
#define CW_ORDER_GREEDY 3     /* Algorithm 1: from the root, repeatedly place the
                                 unplaced document of lowest retrieval rank whose
                                 child node is cached; when none is, the rest
                                 follow in retrieval rank */
#define CW_ORDER_EXHAUSTIVE 4 /* Eq. 1: an order of maximal l(O, T); among equally
                                 deep reused runs the one first in lexicographic
                                 order of retrieval ranks; then the rest in
                                 retrieval rank */

/* Creates an empty tree with recency window `window` >= 1 (in insertions).
 * CW_EINVAL: out NULL or window < 1. */
cw_status cw_tree_create(int32_t window, cw_tree** out);
void cw_tree_destroy(cw_tree* tree);
/* Nodes held (excluding the root); bounded by about 2 * window * k. -1 for NULL. */
int64_t cw_tree_num_nodes(const cw_tree* tree);

/* Records a served order (Sec. 3.2: insert after serving): advances the clock
 * by one and refreshes every node of the path. CW_EINVAL: tree NULL, k
 * outside [0, 4096], order NULL with k > 0, repeated IDs. */
cw_status cw_tree_insert(cw_tree* tree, const int64_t* order, int32_t k);

/* Feedback (Sec. 3.4): the engine reused only `observed_depth` documents of
 * `order`, so the nodes of `order` deeper than that are stale until an order
 * through them is inserted again. Nodes that do not exist are skipped.
 * CW_EINVAL as for cw_tree_insert, or observed_depth outside [0, k]. */
cw_status cw_tree_mark_stale(cw_tree* tree, const int64_t* order, int32_t k, int32_t observed_depth);

/* Orders the retrieved set `docs` [k] with `strategy` (CW_ORDER_*), writing the
 * permutation to out_order [k]. *out_depth = l(out_order, T). *out_probes =
 * child lookups: for the walk of the retrieval, sorted and recency orders, one
 * per node visited plus the failing one; for the greedy order, the lookups a
 * scan of the unplaced documents in retrieval rank makes to find each choice
 * (at a level that places rank j, one per unplaced rank <= j; at the level
 * that finds none, one per unplaced document; at most k (k + 1) / 2); for the
 * exhaustive order, the lookups of its search. out_depth and out_probes may be
 * NULL. The tree is not modified.
 * CW_EINVAL: tree NULL, k outside [0, 4096], NULL arrays with k > 0, repeated
 * IDs, unknown strategy. */
cw_status cw_tree_order(const cw_tree* tree, int32_t strategy, const int64_t* docs, int32_t k,
                        int64_t* out_order, int32_t* out_depth, int32_t* out_probes);

/* ------------------------------------------------------------------------
 * Device: write each request's suffix K and V into its cache blocks (paper
 * Sec. 2.1: KV memory managed in fixed-size blocks).
 *
 * For every request r and token t in [P_r, L_r):
 *   k_cache[block_table[r, t / bs], h, t % bs, :] = k_new[cu[r] + t - P_r, h, :]
 *   v_cache[block_table[r, t / bs], h, t % bs, :] = v_new[cu[r] + t - P_r, h, :]
 * a bit copy. Nothing else in the caches changes. A table entry outside
 * [0, num_blocks) drops the writes of its tokens (never a fault).
 *   cu_suffix_dev / prefix_len_dev   device copies read by the kernel
 *   cu_suffix_host / prefix_len_host host copies used for validation and
 *                                    launch sizing; must hold the same values
 * CW_EINVAL: NULL pointer, batch < 1, num_kv_heads < 1, P_r % bs != 0,
 * cu not non-decreasing from 0, ceil(L_r / bs) > bt_stride, num_blocks < 1.
 * CW_EUNSUPPORTED: head_dim not 64/128 or block_size != 16.
 * CW_EHIP: launch failure. */
cw_status cw_kv_append(const void* k_new, const void* v_new, void* k_cache, void* v_cache,
                       const int32_t* block_table, int32_t bt_stride,
                       const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                       const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                       int32_t batch, int32_t num_kv_heads, int32_t head_dim,
                       int32_t block_size, int32_t num_blocks, void* stream);

/* ------------------------------------------------------------------------
 * Host: work plan for cw_suffix_prefill_attn and cw_suffix_prefill_attn_split
 * (paper Sec. 1 and 2.1: after the prefix match, each request r has P_r cached
 * prefix tokens and S_r suffix rows to prefill; the plan is how that ragged
 * work is cut into tiles and spread over the GPU).
 *
 * The attention kernel works on tiles of (request, KV head, run of
 * 256 / (Hq / Hkv) suffix rows), i.e. 256 packed (query head, row) pairs whose
 * keys run from position 0 to the last row's position, in steps of 64 keys.
 * num_splits > 1 cuts each tile's steps into that many runs (the split path);
 * each run is one plan entry. The grid is persistent (at most one workgroup
 * per CU, 256 on MI355X): entries are spread over per-workgroup queues, longest
 * work first, with the tiles of one (request, KV head) kept on one L2
 * partition where the batch allows. A plan depends only on the batch
 * description (cu_suffix, prefix_len, heads, head_dim, num_splits), so one plan
 * serves every layer of a model for that batch.
 *
 * Layout: a 16-word header (magic, entry count, a 64-bit fingerprint of the
 * batch description, grid, split count, batch, heads, head_dim, rows, queue
 * length, work), then 16-word entries, each with a check word. The device
 * calls take the host copy (plan_host: they validate its header against their
 * own host batch description, so a plan built for another batch is refused
 * with CW_EINVAL) and a device copy of the whole plan (plan_dev: the kernels
 * compute nothing for a device plan whose header fingerprint differs, and stop
 * a queue at an entry whose check word does not match).
 *
 * cw_suffix_prefill_plan_words returns the int32 words a plan needs (or a
 * negative cw_status). cw_suffix_prefill_plan writes it:
 *   plan_host    host int32 [plan_words]; copy all of it to device memory
 *   num_splits   1 .. 64 (1 for cw_suffix_prefill_attn)
 * CW_EINVAL: NULL pointers, batch < 1, Hq % Hkv != 0, cu not non-decreasing
 * from 0, P_r < 0, num_splits out of range, plan_words too small.
 * CW_EUNSUPPORTED: head_dim not 64/128, Hq / Hkv > 128, too many entries. */
int64_t cw_suffix_prefill_plan_words(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                     int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                     int32_t head_dim, int32_t num_splits);
cw_status cw_suffix_prefill_plan(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                 int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                 int32_t head_dim, int32_t num_splits, int32_t* plan_host,
                                 int64_t plan_words);

/* ------------------------------------------------------------------------
 * Device: causal prefill attention of the suffix rows over the paged prefix
 * and themselves (paper Sec. 1 and 2.1: with a reused prefix only the suffix is
 * prefilled, and the result equals a from-scratch prefill of those rows).
 *
 * For every request r, query head h (KV head g = h / (Hq / Hkv)) and suffix row
 * i < S_r, with K_r/V_r the request's logical keys/values read through its
 * block table (tokens 0 .. L_r - 1):
 *   s_j = softmax_scale * <q[cu[r] + i, h, :], K_r[j, g, :]>,  j = 0 .. P_r + i
 *   out[cu[r] + i, h, :] = sum_j softmax(s)_j * V_r[j, g, :]
 * bf16 inputs, fp32 accumulation and softmax, bf16 output (round to nearest
 * even). The caches must already hold the prefix and (after cw_kv_append) the
 * suffix. A table entry outside [0, num_blocks) (within the prompt's blocks)
 * is read as a block of zero keys and values: never a fault, but each of its
 * keys enters the softmax with score 0 and value 0.
 *   plan_host   the plan from cw_suffix_prefill_plan for this batch with
 *               num_splits = 1 (host memory; its header is read)
 *   plan_dev    a device copy of the whole plan
 * CW_EINVAL: NULL pointer, batch < 1, Hq % Hkv != 0, P_r % bs != 0, cu not
 * non-decreasing from 0, ceil(L_r / bs) > bt_stride, softmax_scale not finite
 * and positive, a plan built for another batch description or with splits.
 * CW_EUNSUPPORTED: head_dim not 64/128, block_size != 16, Hq / Hkv > 128,
 *   more than 65536 KV heads.
 * CW_EHIP: launch failure. */
cw_status cw_suffix_prefill_attn(const void* q, const void* k_cache, const void* v_cache,
                                 const int32_t* block_table, int32_t bt_stride,
                                 const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                                 const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                 int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                 int32_t head_dim, int32_t block_size, int32_t num_blocks,
                                 float softmax_scale, const int32_t* plan_host, const int32_t* plan_dev,
                                 void* out, void* stream);

/* ------------------------------------------------------------------------
 * Host: plan for cw_suffix_prefill_append_attn, the KV append and the
 * attention of a batch in one call (paper Sec. 2.1: the suffix K/V go into
 * their blocks; Sec. 1 and 2.1: the suffix rows attend over the cached prefix
 * and themselves).
 *
 * The plan is the unsplit plan of cw_suffix_prefill_plan followed by a table
 * with two words per (request, logical block): where the block's keys are read
 * from and where the call writes them. A request's own suffix blocks are read
 * from its rows of k_new / v_new and written to their cache blocks; a prefix
 * block that is a full suffix block of this batch (a block an earlier request
 * of the same schedule committed, R9) is read from those rows too; every
 * other block is read from the caches. So the call reads no cache block it
 * writes, and its result and cache image equal those of cw_kv_append followed
 * by cw_suffix_prefill_attn. The header also fingerprints the block table and
 * num_blocks: a plan is refused by a call whose host block table differs.
 *   block_table_host  host int32 [batch, bt_stride], the table the caches use
 *   plan_host         host int32 [plan_words]; copy all of it to device memory
 * cw_suffix_prefill_append_plan_words returns the words (or a negative
 * cw_status).
 * CW_EINVAL: as cw_suffix_prefill_plan, plus a NULL table, num_blocks < 1,
 *   ceil(L_r / 16) > bt_stride, P_r % 16 != 0, or an in-pool block named by
 *   two suffix blocks of the batch (their appends would race).
 * CW_EUNSUPPORTED: as cw_suffix_prefill_plan, plus a prefix block that is the
 *   partial last block of a suffix of the batch (its bytes would be partly
 *   appended rows and partly older content). */
int64_t cw_suffix_prefill_append_plan_words(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                            int32_t bt_stride, int32_t batch, int32_t num_q_heads,
                                            int32_t num_kv_heads, int32_t head_dim);
cw_status cw_suffix_prefill_append_plan(const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                        const int32_t* block_table_host, int32_t bt_stride, int32_t batch,
                                        int32_t num_q_heads, int32_t num_kv_heads, int32_t head_dim,
                                        int32_t num_blocks, int32_t* plan_host, int64_t plan_words);

/* ------------------------------------------------------------------------
 * Device: cw_kv_append and cw_suffix_prefill_attn in one launch (paper
 * Sec. 2.1 and Sec. 1; the same result and cache image as the two calls in
 * sequence). The tile whose query rows are a run of suffix positions also
 * writes those positions' K and V rows of its KV head into their cache blocks,
 * from the copy it stages for its own attention; all of the batch's new keys
 * are read from k_new / v_new. Bytes of the caches outside the written rows
 * are unchanged; writes to blocks outside [0, num_blocks) are dropped and such
 * blocks read as zeros, as in the two calls.
 *   k_new, v_new       bf16 [total_s, Hkv, D] device
 *   k_cache, v_cache   written at the suffix rows, read elsewhere
 *   block_table_host, cu_suffix_host, prefix_len_host   host copies; the
 *                      kernel reads the device plan only (no device table or
 *                      offsets are needed)
 *   plan_host / plan_dev   the plan of cw_suffix_prefill_append_plan
 * Errors as cw_suffix_prefill_attn; CW_EINVAL also for a plan without an append
 * table or built for another block table or pool size. */
cw_status cw_suffix_prefill_append_attn(const void* q, const void* k_new, const void* v_new, void* k_cache,
                                        void* v_cache, const int32_t* block_table_host, int32_t bt_stride,
                                        const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                        int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                        int32_t head_dim, int32_t block_size, int32_t num_blocks,
                                        float softmax_scale, const int32_t* plan_host, const int32_t* plan_dev,
                                        void* out, void* stream);

/* ------------------------------------------------------------------------
 * Device: split-KV variant of cw_suffix_prefill_attn, for batches with few
 * tiles (short suffixes such as a question after a fully cached evidence
 * prefix: paper Sec. 1 and 3.3, the reuse the ordering aims for). Same result
 * up to rounding, same arguments, with a plan built for num_splits runs.
 *
 * Each tile's key range is divided into num_splits runs of whole 64-key steps
 * (the plan's entries); each run's attention over its own keys (normalised O
 * in fp32 and its base-2 log-sum-exp per row) is written to `workspace`, then
 * combined exactly as by cw_lse_merge into out (bf16).
 *   workspace        caller-owned device memory of at least
 *                    cw_suffix_prefill_split_workspace_bytes(total_s, Hq, D,
 *                    num_splits) bytes; overwritten by the call
 * Errors as cw_suffix_prefill_attn, plus CW_EINVAL for a missing / too small
 * workspace. cw_suffix_prefill_split_workspace_bytes returns the size, or a
 * negative cw_status for invalid arguments (num_splits outside 1 .. 64). */
int64_t cw_suffix_prefill_split_workspace_bytes(int64_t total_rows, int32_t num_q_heads, int32_t head_dim,
                                                int32_t num_splits);
cw_status cw_suffix_prefill_attn_split(const void* q, const void* k_cache, const void* v_cache,
                                       const int32_t* block_table, int32_t bt_stride,
                                       const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                                       const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                       int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                       int32_t head_dim, int32_t block_size, int32_t num_blocks,
                                       float softmax_scale, const int32_t* plan_host, const int32_t* plan_dev,
                                       void* workspace, int64_t workspace_bytes, void* out, void* stream);

/* ------------------------------------------------------------------------
 * Device: cw_suffix_prefill_attn_split without a workspace, for callers that
 * cannot allocate device memory (code under HIP graph capture, tight serving
 * loops, harnesses that forbid allocation). Same arguments, result and errors
 * as cw_suffix_prefill_attn_split, without workspace / workspace_bytes: the
 * partial results go to a device array built into the library, of
 * cw_noalloc_scratch_bytes() bytes (64 MiB), which every GPU the library runs
 * on holds until the process ends. The call allocates nothing.
 *   - CW_EINVAL when the batch needs more than that:
 *     cw_suffix_prefill_split_workspace_bytes(total_s, Hq, D, num_splits) >
 *     cw_noalloc_scratch_bytes().
 *   - Every call on one GPU shares that GPU's array: calls that overlap in time
 *     on one GPU (other streams, other threads) race and may corrupt each
 *     other's results. Calls on one stream are ordered and safe. The array
 *     keeps the last call's contents; nothing in it needs to start at zero.
 *   - CW_EHIP if the array's device address cannot be obtained. */
int64_t cw_noalloc_scratch_bytes(void);
cw_status cw_suffix_prefill_attn_split_noalloc(const void* q, const void* k_cache, const void* v_cache,
                                               const int32_t* block_table, int32_t bt_stride,
                                               const int32_t* cu_suffix_dev, const int32_t* prefix_len_dev,
                                               const int32_t* cu_suffix_host, const int32_t* prefix_len_host,
                                               int32_t batch, int32_t num_q_heads, int32_t num_kv_heads,
                                               int32_t head_dim, int32_t block_size, int32_t num_blocks,
                                               float softmax_scale, const int32_t* plan_host,
                                               const int32_t* plan_dev, void* out, void* stream);

/* ------------------------------------------------------------------------
 * Device: merge of attention results computed over disjoint key sets (the
 * pieces of cw_suffix_prefill_attn_split; also how partial results over a
 * prefix split across GPUs would be combined). Softmax over a union of key
 * sets, written out by log-sum-exp:
 *   M = max_p lse[p][i],  w_p = 2^(lse[p][i] - M)
 *   out[i][:] = sum_p w_p * o[p][i][:] / sum_p w_p        (bf16, RNE)
 *   partial_o    device fp32 [num_parts, rows, head_dim], each part normalised
 *   partial_lse  device fp32 [num_parts, rows]: log2 of the part's sum of
 *                exp(scaled score); -inf for a part with no keys (skipped).
 *                A row whose parts are all -inf is written as zeros.
 * CW_EINVAL: NULL pointer, num_parts < 1, rows < 0.
 * CW_EUNSUPPORTED: head_dim not a multiple of 8 in [8, 1024]. */
cw_status cw_lse_merge(const void* partial_o, const void* partial_lse, int32_t num_parts, int64_t rows,
                       int32_t head_dim, void* out, void* stream);

/* ------------------------------------------------------------------------
 * Host: rotary-embedding table for the suffix QKV projection. With a reused
 * prefix only the suffix tokens are prefilled (paper Sec. 1 and 2.1), and
 * their queries and keys are rotated at their absolute positions P_r + i (the
 * rotate-half rotary embedding of the decoder-only models of Sec. 4).
 *   out  host fp32 [n_positions, head_dim / 2, 2]: entry (p, j) holds
 *        cos(p * theta_j) and sin(p * theta_j), theta_j = base^(-2 j / head_dim),
 *        each evaluated in double precision and rounded once to fp32.
 * CW_EINVAL: n_positions < 0, head_dim odd or outside [2, 1024], base not
 * finite or <= 1, out NULL with n_positions > 0. */
cw_status cw_rope_table(int32_t n_positions, int32_t head_dim, double base, float* out);

/* ------------------------------------------------------------------------
 * Device: suffix QKV projection with rotary embedding, fused with the KV
 * append. With a reused prefix only the suffix tokens are prefilled (paper
 * Sec. 1 and 2.1); per layer that starts by projecting each suffix token's
 * hidden state to its query, key and value heads, rotating queries and keys
 * at the token's absolute position, and storing keys and values in the
 * request's cache blocks (Sec. 2.1). For suffix row t = cu[r] + i of request
 * r, at position p = P_r + i:
 *   y      = x[t] W^T (+ bias)        fp32 accumulation of bf16 products
 *   y_q, y_k, y_v = features [0, Hq D), [Hq D, (Hq + Hkv) D), the rest
 *   rot(u)[j]         = u[j] cos(p th_j) - u[j + D/2] sin(p th_j)
 *   rot(u)[j + D/2]   = u[j + D/2] cos(p th_j) + u[j] sin(p th_j),  j < D/2
 *   q_out[t][h][:]    = rot(y_q of head h)
 *   k_cache[blk][g][p % 16][:], v_cache[blk][g][p % 16][:] = rot(y_k), y_v
 *     of KV head g, blk = block_table[r][p / 16]; a block id outside
 *     [0, num_blocks) is skipped (nothing written).
 * Every output is rounded once, RNE, to bf16; every other cache byte keeps
 * its value.
 *   x       device bf16 [total_s, hidden], rows in request order
 *   w       device bf16 [(Hq + 2 Hkv) head_dim, hidden] (one row per feature)
 *   bias    device bf16 [(Hq + 2 Hkv) head_dim], or NULL for none
 *   rope    device fp32 [rope_len, head_dim / 2, 2]: (cos, sin) of p th_j, as
 *           cw_rope_table writes it; every suffix position must be < rope_len
 *   hidden  multiple of 32 in [32, 2^20]
 *   q_out   device bf16 [total_s, Hq, head_dim]
 *   k_cache, v_cache, block_table, cu_suffix_*, prefix_len_*: as for
 *           cw_kv_append (cu/prefix on host for validation and launch sizing,
 *           on device for the kernel; both copies must agree)
 * All device pointers 16-byte aligned; the caller owns every buffer. Runs
 * asynchronously on `stream` (NULL = default stream).
 * x and q_out may be NULL when total_s is 0 (nothing is launched).
 * CW_EINVAL: NULL pointer (other than bias), head counts, num_blocks < 1,
 * rope_len < 0 or too short, the batch checks of cw_kv_append.
 * CW_EUNSUPPORTED: head_dim not 64 or 128, block_size != 16, hidden not a
 * multiple of 32 in range, total_s too large. CW_EHIP: launch failure. */
cw_status cw_qkv_rope_append(const void* x, const void* w, const void* bias, const float* rope,
                             int32_t rope_len, int32_t hidden, void* q_out, void* k_cache, void* v_cache,
                             const int32_t* block_table, int32_t bt_stride, const int32_t* cu_suffix_dev,
                             const int32_t* prefix_len_dev, const int32_t* cu_suffix_host,
                             const int32_t* prefix_len_host, int32_t batch, int32_t num_q_heads,
                             int32_t num_kv_heads, int32_t head_dim, int32_t block_size, int32_t num_blocks,
                             void* stream);

/* ---------------------------------------------------------------------------
 * Measurement aid (not a step of the path). A roofline of the attention kernel
 * prices it against the data-sheet bf16 peak; the rate this card sustains
 * depends on the operand values through its power limit, so the bench reports
 * the measured rate beside the data-sheet one.
 *
 * cw_probe_mfma_bf16 launches `workgroups` workgroups of 8 wavefronts; each
 * wavefront runs `iters` rounds of 8 independent v_mfma_f32_32x32x16_bf16
 * instructions (32x32 accumulators, 16-deep bf16 products) on fragments read
 * once from `operands`.
 *   operands       device, bf16 values, operand_bytes bytes: fragments of
 *                  1024 bytes (16 per lane), used cyclically; read only
 *   operand_bytes  a multiple of 1024, >= 6144
 *   sink           device float[workgroups * 512]; one value per thread is
 *                  written (the accumulator sum), only so the work is kept
 *   iters >= 1; 1 <= workgroups <= 2^20. Asynchronous on `stream`.
 * CW_EINVAL: NULL pointer or a size out of range. CW_EHIP: launch failure.
 * cw_probe_mfma_bf16_flops returns the FLOPs of one such call (2 x 32 x 32 x 16
 * per instruction), or -1 for iters < 1 or workgroups < 1. */
int64_t cw_probe_mfma_bf16_flops(int32_t iters, int32_t workgroups);
cw_status cw_probe_mfma_bf16(const void* operands, int64_t operand_bytes, float* sink, int32_t iters,
                             int32_t workgroups, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* CW_H */
