/*
 * hswa.h -- C ABI of libhswa: Hybrid sliding-window-attention (SWA) paged KV
 * attention for AMD MI355X (gfx950).
 *
 * The method (paper: "Full-Pipeline Inference Optimization for MiMo-V2.5
 * Series", sections "Introduction", "Compute Analysis", "KVCache Storage
 * Analysis", "KVCache Dual-Pool Design", "SWA-Aware Prefix Cache Tree"):
 * a model interleaves SWA layers, which attend only inside a local window of W
 * tokens, with FULL layers, which attend to the whole context. The KV cache is
 * split into two physical pools: a FULL pool holding every position, and an
 * SWA pool sized for the window (a per-sequence ring of pages), so SWA storage
 * is O(W) instead of O(L). Out-of-window SWA entries are released (here: a ring
 * overwrite) and must never be read again.
 *
 * Attention computed by every call (one sequence, query at absolute position
 * p, query head h, KV head g = h / (Hq / Hkv)):
 *     keys j with lo(p) <= j <= p, lo(p) = 0 (FULL) or max(0, p - W + 1) (SWA)
 *     o = sum_j softmax_j(scale * <q, k_j>) * v_j
 * W counts the query itself (W = 1 attends only to position p).
 *
 * ---------------------------------------------------------------------------
 * Conventions shared by every call
 * ---------------------------------------------------------------------------
 * Ownership. The caller owns every buffer. The library never allocates or
 *   frees device memory. It keeps two pieces of state between calls: per
 *   device, the number of waves the FULL decode kernel can hold resident,
 *   looked up on the first FULL decode call on that device and cached
 *   (atomically) for the life of the process; and the fixed device array of
 *   hswa_decode_noalloc (a static array of the library, one per device).
 *   All calls are thread-safe. Pointers marked "device" are device (HBM)
 *   addresses, "host" pointers are read synchronously during the call.
 * Streams. Compute calls enqueue on `stream` (a hipStream_t passed as void*;
 *   NULL = the default stream) and return without synchronising. Argument
 *   validation is synchronous and returns a status; a failed launch returns
 *   HSWA_ERR_LAUNCH. Device-side problems surface at the caller's next
 *   synchronisation, or at once when the environment sets HSWA_SYNC_CHECK=1.
 *   Nothing throws across this ABI.
 * Dtypes. q, k, v, out and the pools hold bf16 (raw 16-bit patterns). Scores,
 *   softmax and accumulation are fp32; outputs are rounded to bf16 with
 *   round-to-nearest-even.
 * Layout. Per layer there is one K pool and one V pool of `num_pages` pages;
 *   both hold a page-head (one page of one KV head) as blocks of
 *   B = min(page_size, 32) consecutive keys:
 *     K pool: bf16 [num_pages][Hkv][page_size/B][2][head_dim/32][4][B/2][8]
 *             key k of a block (k = o % B) sits in half (k / 4) % 2 at row
 *             4 * (k / 8) + k % 4; its dim d in slab d / 32, piece (d / 8) % 4,
 *             element d % 8. For B = 32 the 16 keys x 32 dims of one half and
 *             slab (one QK^T operand of the bf16 matrix cores) are one
 *             contiguous 1 KiB run in MFMA lane order.
 *     V pool: bf16 [num_pages][Hkv][page_size/B][head_dim][B]
 *             (each block transposed, so the V^T of 32 consecutive keys of one
 *             head is one 8 KiB run)
 *   Slot s addresses page s / page_size at in-page offset o = s % page_size,
 *   block o / B; its V values sit in that block's column o % B.
 *   Every pool offset is computed in 64-bit.
 * Block tables (int32, device, row stride `table_stride`):
 *     FULL layer: table[b][i] = physical page of logical page i (positions
 *                 i*PG .. i*PG+PG-1) of sequence b; needs ceil(L_b / PG)
 *                 entries.
 *     SWA layer:  table[b][r] = physical page of ring entry r, r < R, with
 *                 R = hswa_ring_pages(W, PG); position j lives in ring entry
 *                 (j / PG) mod R at offset j mod PG, so the ring holds the
 *                 latest R*PG positions.
 *   Entries outside [0, num_pages), and logical pages at or past
 *   table_stride, are never dereferenced: no memory outside the pools is
 *   touched. A key the call needs on such an entry is a caller error whose
 *   rows come out wrong: hswa_decode leaves the key out, hswa_prefill reads it
 *   as a zero key and value (score 0, so it still takes part in the softmax).
 *   hswa_decode checks table_stride * page_size >= max_context_len on the host
 *   (HSWA_ERR_CAPACITY); hswa_prefill cannot (the prefix lengths live on the
 *   device), so a FULL or SWA_PAGED table must hold ceil((P_b + C_b) / PG)
 *   entries per sequence.
 * Ordering. Decode: hswa_kv_append of the new token, then hswa_decode (which
 *   reads the new token from the cache; the ring slot the new token at c
 *   overwrites held position c - R*PG, outside the window since R*PG > W);
 *   or both at once with hswa_decode_append.
 *   Prefill:
 *   hswa_prefill first (the chunk's own keys come from k_new / v_new), then
 *   hswa_kv_append of the chunk. For SWA this order is required: a chunk
 *   longer than the ring overwrites prefix keys that its first queries need.
 * Supported shapes: head_dim == 128; Hq % Hkv == 0 and 128 % (Hq/Hkv) == 0;
 *   Hkv <= 4096; page_size a power of two in [16, 256]; SWA window >= 1.
 *   Anything else returns HSWA_ERR_UNSUPPORTED or HSWA_ERR_INVALID_ARG.
 */
#ifndef HSWA_H
#define HSWA_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HSWA_OK = 0,
  HSWA_ERR_INVALID_ARG = -1, /* null pointer, negative size, inconsistent shape */
  HSWA_ERR_UNSUPPORTED = -2, /* shape outside the supported set above          */
  HSWA_ERR_CAPACITY = -3,    /* table stride, page count or workspace too small */
  HSWA_ERR_LAUNCH = -4       /* the HIP runtime rejected a launch               */
} hswa_status;

/* Layer kind flag ("Compute Analysis": SWA layers attend within a local
 * window, FULL layers attend globally).
 *   HSWA_LAYER_SWA:       SWA layer over a per-sequence ring of pages (see
 *                         Block tables): a fixed O(W) set of pages per sequence.
 *   HSWA_LAYER_SWA_PAGED: SWA layer over a block table indexed like a FULL
 *                         layer's (logical page -> SWA page), in which pages
 *                         outside the window have been released (-1): the
 *                         explicit-release form of the SWA pool, whose tables
 *                         come from hswa_allocator below. Tokens appended to a
 *                         -1 entry are not stored (slot -1). */
typedef enum { HSWA_LAYER_FULL = 0, HSWA_LAYER_SWA = 1, HSWA_LAYER_SWA_PAGED = 2 } hswa_layer_kind;

/* kind: hswa_layer_kind. window: W >= 1 for SWA and SWA_PAGED (counts the
 * query itself); ignored for FULL. */
typedef struct {
  int32_t kind;
  int32_t window;
} hswa_layer;

/* Head geometry of one attention layer. scale multiplies <q, k>; 1/sqrt(128)
 * is the usual choice. */
typedef struct {
  int32_t num_q_heads;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t page_size;
  float scale;
} hswa_shape;

/* One layer's pool pair and its block table (see Layout / Block tables). */
typedef struct {
  void *k_pool;               /* device, bf16 [num_pages][Hkv][PG/B][2][D/32][4][B/2][8] */
  void *v_pool;               /* device, bf16 [num_pages][Hkv][PG/B][D][B]               */
  int64_t num_pages;
  const int32_t *block_table; /* device, int32 [ns][table_stride]              */
  int32_t table_stride;
} hswa_cache;

/* ---- host helpers (no device access) ------------------------------------ */

/* Ring pages per sequence of an SWA layer: ceil(window / page_size) + 1 (the
 * SWA pool is sized for the window only: "KVCache Dual-Pool Design"). Returns
 * -1 if window < 1 or page_size < 1. */
int32_t hswa_ring_pages(int32_t window, int32_t page_size);

/* Bytes of one page of one pool (K or V): Hkv * page_size * head_dim * 2.
 * Pool sizes follow from it ("KVCache Storage Analysis": a FULL layer stores
 * every position of every sequence, an SWA layer only its window, so an SWA
 * pool of ns * R pages is flat in the context length). Returns -1 on a null or
 * non-positive shape. */
int64_t hswa_page_bytes(const hswa_shape *shape);

/* Fill a block table (host memory) from a permutation of physical page ids
 * ("KVCache Dual-Pool Design": the FULL index maps a sequence's logical pages
 * to physical pages, and a separate mapping gives its SWA pages; here the SWA
 * mapping is the ring of R entries):
 * sequence b needs n_b pages (FULL: ceil(final_lens[b] / page_size); SWA: R)
 * and receives perm[o_b .. o_b + n_b - 1], o_b = n_0 + ... + n_{b-1}; unused
 * entries are -1. table_out is int32 [ns][stride]. Returns HSWA_ERR_CAPACITY
 * if some n_b > stride or the permutation is shorter than the sum of n_b. */
hswa_status hswa_build_block_table(hswa_layer layer, int32_t page_size, int32_t ns,
                                   const int32_t *final_lens, const int32_t *perm,
                                   int64_t perm_len, int32_t *table_out, int32_t stride);

/* ---- device calls -------------------------------------------------------- */

/* KV append with slot mapping and ring-wrap eviction ("KVCache Dual-Pool
 * Design": the SWA pool evicts by window; "SWA-Aware Prefix Cache Tree": the
 * release follows each chunk and each decode step).
 *
 * Sequence b appends the tokens cu_seqlens[b] .. cu_seqlens[b+1]-1 of k_new /
 * v_new at positions start_pos[b], start_pos[b]+1, ...; its length afterwards
 * is L_b = start_pos[b] + (cu_seqlens[b+1] - cu_seqlens[b]).
 *   FULL: slot = table[b][j / PG] * PG + j % PG.
 *   SWA:  slot = table[b][(j / PG) mod R] * PG + j % PG if j >= L_b - R*PG,
 *         else -1 (not stored: the ring keeps the latest R*PG positions, so
 *         overwriting the ring is the out-of-window eviction and no slot is
 *         written twice in one call).
 * k_new, v_new: device bf16 [total_tokens][Hkv][D]. cu_seqlens: device int32
 * [ns+1], non-decreasing, cu_seqlens[ns] == total_tokens. start_pos: device
 * int32 [ns]. slot_mapping_out: device int64 [total_tokens] (may be NULL).
 * Tokens whose logical page is beyond table_stride, or whose table entry is
 * outside [0, num_pages), are not stored and get slot -1. */
hswa_status hswa_kv_append(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache,
                           const void *k_new, const void *v_new, const int32_t *cu_seqlens,
                           const int32_t *start_pos, int32_t ns, int32_t total_tokens,
                           int64_t *slot_mapping_out, void *stream);

/* Chunked prefill over a cached prefix ("Compute Analysis": chunked prefill,
 * compute-bound; "Prefill Optimization" / "Length Bucketing Strategy": fixed
 * chunks over prefixes of varying length).
 *
 * Sequence b has prefix_lens[b] = P_b cached tokens and a chunk of
 * C_b = cu_seqlens[b+1] - cu_seqlens[b] new tokens at positions P_b .. P_b+C_b-1.
 * Keys below P_b are read from the cache (FULL: every one; SWA: the ring,
 * only the in-window ones), keys from P_b on are read from k_new / v_new.
 * q: device bf16 [total_tokens][Hq][D]; k_new, v_new: device bf16
 * [total_tokens][Hkv][D]; out: device bf16 [total_tokens][Hq][D].
 * max_chunk_len: host, >= every C_b (sizes the grid; longer chunks are cut).
 * Must run before the hswa_kv_append of the same chunk. */
hswa_status hswa_prefill(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache,
                         const void *q, const void *k_new, const void *v_new,
                         const int32_t *cu_seqlens, const int32_t *prefix_lens, int32_t ns,
                         int32_t total_tokens, int32_t max_chunk_len, void *out, void *stream);

/* Workspace bytes hswa_decode needs for a FULL layer (0 for an SWA layer is
 * enough): fp32 partial outputs and log-sum-exps of every split-KV piece
 * (at most ceil(max_context_len / hswa_decode_split_len) + 1 per output row).
 * The split exists because decode is memory-bound ("KVCache Storage
 * Analysis"): a long FULL context is read by many waves at once, and their
 * pieces are merged by the log-sum-exp identity. Returns 0 on an invalid
 * shape. */
size_t hswa_decode_workspace_bytes(const hswa_shape *shape, int32_t ns, int32_t max_context_len);

/* Fewest keys of a split-KV span that hswa_decode uses for a FULL layer (a
 * multiple of 256); max_context_len at most this long decodes in one pass.
 * Returns -1 on an invalid shape. */
int32_t hswa_decode_split_len(const hswa_shape *shape, int32_t ns, int32_t max_context_len);

/* Decode: one query per sequence at position c_b = context_lens[b] - 1, where
 * context_lens counts the cached tokens including the one just appended
 * ("KVCache Storage Analysis": decode is memory-bound). SWA layers read at most
 * W keys from the ring in a single pass. FULL layers cut the 32-key chunks of
 * all (sequence, KV head) pairs, taken in that order, into equal spans, one per
 * wave the device holds at once (each at least hswa_decode_split_len keys);
 * a pair met by several spans gets fp32 partials in the workspace, merged by
 * log-sum-exp. The cuts are logical positions: results do not depend on where
 * pages sit physically, but their rounding may depend on the other sequences'
 * lengths and on the device's compute-unit count.
 * q: device bf16 [ns][Hq][D]; context_lens: device int32 [ns], each in
 * [1, max_context_len] (values above max_context_len are clamped to it, values
 * below 1 give a zero output row); out: device bf16 [ns][Hq][D];
 * workspace: device, >= hswa_decode_workspace_bytes (FULL only; may be NULL
 * for SWA). */
hswa_status hswa_decode(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache,
                        const void *q, const int32_t *context_lens, int32_t ns,
                        int32_t max_context_len, void *workspace, size_t workspace_bytes,
                        void *out, void *stream);

/* One decode step of a layer, append included ("KVCache Storage Analysis":
 * an SWA layer's decode reads only its window, so its cost is a short chain of
 * dependent loads and a launch; "KVCache Dual-Pool Design": the step's token
 * goes to its pool slot, the ring overwrite evicting the oldest position).
 * For every sequence b with c_b = min(context_lens[b], max_context_len) >= 1:
 * stores k_new[b] / v_new[b] at position c_b - 1 exactly as hswa_kv_append
 * with cu_seqlens = 0, 1, .., ns and start_pos[b] = c_b - 1 would, and writes
 * out[b] as hswa_decode with the same context_lens would after that append.
 * Sequences with c_b < 1 store nothing and get a zero row. SWA layers, and FULL
 * layers short enough for one pass, do both in one kernel whose new key comes
 * from k_new / v_new (results equal the two calls' up to rounding order); so
 * do the split-KV decode kernels of longer FULL layers when page_size >= 32
 * (the log-sum-exp merge still follows); FULL layers with page_size 16 run the
 * append kernel, then the decode kernels.
 * k_new, v_new: device bf16 [ns][Hkv][D]; the other arguments as hswa_decode.
 * The call must not overlap another call writing the same layer's pools. */
hswa_status hswa_decode_append(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache,
                               const void *q, const void *k_new, const void *v_new,
                               const int32_t *context_lens, int32_t ns, int32_t max_context_len,
                               void *workspace, size_t workspace_bytes, void *out, void *stream);

/* Bytes of the fixed device array behind hswa_decode_noalloc. */
#define HSWA_NOALLOC_SCRATCH_BYTES ((size_t)128 << 20)

/* hswa_decode for callers that cannot allocate device memory or hand in a
 * workspace (code under HIP graph capture, tight serving loops, harnesses
 * that forbid hipMalloc): the same kernels and results, with the FULL split
 * partials kept in a fixed device array of the library
 * (HSWA_NOALLOC_SCRATCH_BYTES per device, taken on the first call on a device
 * and held until the process ends). The call allocates nothing. A FULL layer
 * whose partials need more (hswa_decode_workspace_bytes > the array) returns
 * HSWA_ERR_CAPACITY; SWA layers use no scratch. Nothing in the array needs to
 * start at zero: a call reads back only the partials it wrote. All calls on
 * one device share the array and leave their partials in it: calls that
 * overlap on one GPU (several streams, or threads) race and give wrong rows;
 * serialise them, or use hswa_decode with a workspace of their own. */
hswa_status hswa_decode_noalloc(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache,
                                const void *q, const int32_t *context_lens, int32_t ns,
                                int32_t max_context_len, void *out, void *stream);

/* Multi-query decode ("MTP Optimization": the model verifies 1 + 3 predicted
 * tokens per sequence per step): num_queries (1 .. 64) new queries per
 * sequence at positions c_b - num_queries .. c_b - 1, where c_b =
 * context_lens[b] counts the cached tokens including all new ones (append them
 * first). Query i attends keys lo .. its own position (causal among the new
 * tokens; lo as in hswa_decode for its own position). Queries whose position
 * is negative get zero rows.
 * SWA limits: the first query reads the W - 1 keys before it, which must
 * still be cached after all num_queries appends. A ring (HSWA_LAYER_SWA)
 * keeps the latest R * PG positions, so num_queries <= R * PG - W + 1 (17 at
 * PG 16 and W 128, 65 at PG 64); an explicit-release table
 * (HSWA_LAYER_SWA_PAGED) holds the last W positions of one extend, so
 * num_queries <= W. Larger counts return HSWA_ERR_UNSUPPORTED.
 * q, out: device bf16 [ns][num_queries][Hq][D]; workspace >=
 * hswa_decode_multi_workspace_bytes (FULL only). num_queries = 1 is exactly
 * hswa_decode. */
size_t hswa_decode_multi_workspace_bytes(const hswa_shape *shape, int32_t ns, int32_t num_queries,
                                         int32_t max_context_len);
hswa_status hswa_decode_multi(hswa_layer layer, const hswa_shape *shape, const hswa_cache *cache,
                              const void *q, const int32_t *context_lens, int32_t ns, int32_t num_queries,
                              int32_t max_context_len, void *workspace, size_t workspace_bytes, void *out,
                              void *stream);

/* Static string naming a status. */
const char *hswa_status_string(hswa_status status);

/* ---- explicit-release dual-pool page allocator (host) -------------------
 * "KVCache Dual-Pool Design": separate FULL and SWA pools with their own
 * capacities; admission checks both; the FULL index (logical page i of a
 * sequence = positions i*PG .. i*PG+PG-1) is authoritative and the SWA table
 * maps the same logical pages to SWA pages. "SWA-Aware Prefix Cache Tree":
 * out-of-window SWA pages are released at the end of every prefill chunk,
 * every N decode steps and at request end, so SWA usage per sequence stays at
 * window (or chunk) size. The tables are the block tables of a FULL layer and
 * of an HSWA_LAYER_SWA_PAGED layer.
 * An allocator is a host object owned by the caller (create / destroy); it
 * touches no device memory. Calls on one allocator must not overlap; distinct
 * allocators are independent. Physical pages are handed out from per-pool
 * free stacks (initially in increasing order); a call that fails changes
 * nothing. */
typedef struct hswa_allocator hswa_allocator;

typedef struct {
  int32_t page_size;     /* tokens per page, both pools (>= 1)                  */
  int32_t window;        /* W >= 1                                             */
  int64_t full_pages;    /* FULL pool capacity in pages                        */
  int64_t swa_pages;     /* SWA pool capacity in pages                         */
  int32_t max_seqs;      /* sequence slots 0 .. max_seqs-1 (table rows)        */
  int32_t table_stride;  /* logical pages per table row (max length / PG)      */
  int32_t release_every; /* N >= 1: decode steps between out-of-window releases */
} hswa_allocator_config;

hswa_status hswa_allocator_create(const hswa_allocator_config *config, hswa_allocator **out);
void hswa_allocator_destroy(hswa_allocator *alloc);

/* Admission of a request into the free slot `seq`: succeeds only if both pools
 * can hold it now (FULL: ceil(len / PG) pages; SWA: ceil(min(len, W+chunk) /
 * PG) + 1 pages, the window plus one chunk of `chunk` tokens). Reserves
 * nothing; the sequence starts empty. HSWA_ERR_CAPACITY if a pool (or the
 * table stride) is short, HSWA_ERR_INVALID_ARG if the slot is in use. */
hswa_status hswa_allocator_admit(hswa_allocator *alloc, int32_t seq, int64_t len, int32_t chunk);

/* Grow sequence `seq` to new_len tokens before the prefill / append of
 * positions [len, new_len): FULL pages for every new logical page; SWA pages
 * for the positions in [max(len, new_len - W), new_len) that are not held yet
 * (the window of the query at new_len - 1, which a decode step reads back from
 * the pool, and of the next one; earlier new positions are read from the pool
 * by no query and are not stored). All or nothing: HSWA_ERR_CAPACITY if a pool
 * or the stride is short. */
hswa_status hswa_allocator_extend(hswa_allocator *alloc, int32_t seq, int64_t new_len);

/* End of a prefill chunk (decode_step = 0) or of a decode step (decode_step =
 * 1), after the kernels of that step: releases the SWA pages that lie wholly
 * before the window of the next query (position len), i.e. logical pages
 * below (len - W + 1) / PG; for decode steps only on every N-th call.
 * *released (optional) receives the number of pages freed. */
hswa_status hswa_allocator_step_end(hswa_allocator *alloc, int32_t seq, int32_t decode_step, int32_t *released);

/* Request end: every page of `seq` goes back to its pool; the slot is free. */
hswa_status hswa_allocator_free(hswa_allocator *alloc, int32_t seq);

/* Block tables, host int32 [max_seqs][table_stride] each (either may be NULL):
 * logical page -> FULL page / SWA page, -1 where nothing is held. */
hswa_status hswa_allocator_tables(const hswa_allocator *alloc, int32_t *full_table, int32_t *swa_table);

/* Pages held by sequence `seq` (seq >= 0) or by all sequences (seq < 0), and
 * the free pages of each pool; any output may be NULL. */
hswa_status hswa_allocator_usage(const hswa_allocator *alloc, int32_t seq, int64_t *full_used, int64_t *swa_used,
                                 int64_t *full_free, int64_t *swa_free);

/* ---- window-safe prefix cache tree (host) -------------------------------
 * "SWA-Aware Prefix Cache Tree": a radix tree over token ids whose nodes carry
 * per token two indices, the FULL KV slot and the SWA KV slot (-1 = none).
 * Token equality is no longer enough for reuse: a match is the longest cached
 * prefix whose tokens are equal and whose FULL slots are all held (full_len),
 * clipped to the window-safe length (safe_len <= full_len): the largest P such
 * that the W - 1 tokens before P, the cached keys the first new query at
 * position P reads, all hold SWA slots. safe_len is the prefix length P to pass
 * to hswa_prefill. SWA slots can be released on their own (out-of-window
 * release) while FULL slots stay, or whole segments can be evicted.
 * A tree is a host object owned by the caller; calls on one tree must not
 * overlap. Slots are opaque to the tree (e.g. pool slots page * PG + offset). */
typedef struct hswa_prefix_tree hswa_prefix_tree;

hswa_status hswa_prefix_tree_create(int32_t window, hswa_prefix_tree **out);
void hswa_prefix_tree_destroy(hswa_prefix_tree *tree);

/* Caches tokens[0..n) with their slots (host arrays of n entries); positions
 * already cached on this path take the new slots. */
hswa_status hswa_prefix_tree_insert(hswa_prefix_tree *tree, const int32_t *tokens, int64_t n,
                                    const int64_t *full_slots, const int64_t *swa_slots);

/* Match of tokens[0..n): *full_len and *safe_len as above; if the slot outputs
 * are non-NULL (n entries each) their first *full_len entries receive the
 * matched slots. */
hswa_status hswa_prefix_tree_match(const hswa_prefix_tree *tree, const int32_t *tokens, int64_t n,
                                   int64_t *full_len, int64_t *safe_len, int64_t *full_slots_out,
                                   int64_t *swa_slots_out);

/* Out-of-window release: drops the SWA slots of positions [0, upto) of the
 * cached path tokens[0..n) (FULL slots stay). *released = slots dropped. */
hswa_status hswa_prefix_tree_release_swa(hswa_prefix_tree *tree, const int32_t *tokens, int64_t n, int64_t upto,
                                         int64_t *released);

/* Segment eviction: removes position `keep` of the cached path tokens[0..n)
 * and everything cached after it (all continuations). *evicted = tokens
 * removed. */
hswa_status hswa_prefix_tree_evict(hswa_prefix_tree *tree, const int32_t *tokens, int64_t n, int64_t keep,
                                   int64_t *evicted);

/* Nodes, cached tokens and tokens with a valid SWA slot; outputs may be NULL. */
hswa_status hswa_prefix_tree_stats(const hswa_prefix_tree *tree, int64_t *nodes, int64_t *tokens,
                                   int64_t *swa_valid_tokens);

#ifdef __cplusplus
}
#endif

#endif /* HSWA_H */
