/*
 * dms.h -- C ABI of libdms: Dynamic Memory Sparsification (DMS) inference on
 * one AMD Instinct MI355X (gfx950).
 *
 * Method (arxiv 2506.05345, "Inference-Time Hyper-Scaling with KV Cache
 * Compression"):
 *   - every new key/value pair (k_t, v_t) of every KV head carries a binary
 *     eviction decision alpha_t (Sec. 3.1 "Eviction Decisions", Eq. 1;
 *     binarised by rounding at inference, Sec. 3.2);
 *   - a pair flagged at step t stays visible until step t + w and is then
 *     removed (Sec. 3.1 "Delayed Eviction via Sliding Window"): key j is
 *     visible to query t iff j <= t and (j > t - w or alpha_j = 0), the binary
 *     case of the mask M_alpha of Fig. 1b;
 *   - the removed pair's cache slot is overwritten by an incoming pair, and
 *     the cache is paged with pages owned by one attention head (Sec. 3.2,
 *     inference paragraph on performance);
 *   - prefill applies the same mask, passed as a vector of decisions rather
 *     than a T x T matrix (Sec. 3.1 "Performance Considerations", Sec. 3.2).
 *
 * Conventions shared by every call
 * --------------------------------
 *   Hkv = num_kv_heads, g = group_size, Hq = Hkv * g, d = head_dim,
 *   P = page_size, w = window.  Query head q attends with KV head q / g.
 *   Keys and queries are passed after any positional encoding; the library
 *   never applies positions (keys "carry positional information", Sec. 3.2),
 *   so the order of retained slots is irrelevant to attention.
 *
 *   bf16 tensors are IEEE bfloat16 bit patterns (uint16), row-major, densely
 *   packed.  Decode inputs: q [n, Hq, d], k / v [n, Hkv, d], flags [n, Hkv]
 *   (uint8, 0 = keep, nonzero = evict after w steps), seq_ids [n] int32.
 *   Chunk inputs are "varlen": sequence i owns tokens cu_seqlens[i] ..
 *   cu_seqlens[i+1]-1 of q [T, Hq, d], k / v [T, Hkv, d], flags [T, Hkv].
 *   Outputs are float32 [n, Hq, d] (decode) or [T, Hq, d] (prefill).
 *
 *   Pointers named *_dev are device pointers; *_host are host pointers.
 *   `stream` is a hipStream_t (NULL = the null stream).  Every call only
 *   enqueues work on `stream` and returns; device buffers passed in must
 *   stay valid until that work completes.  One context may be used from one
 *   stream at a time (the workspace is shared by all layers).
 *
 * Ownership
 * ---------
 *   The caller allocates and frees every device buffer: the state buffer
 *   (`meta`), one KV pool per layer, and the workspace, sized by
 *   dms_layout().  libdms never allocates or frees device memory; a context
 *   (dms_ctx) is a small host object holding the configuration and the
 *   caller's pointers.
 *
 * Errors
 * ------
 *   Every call returns DMS_OK (0) or a negative code.  Argument errors are
 *   detected on the host before any HIP call and change nothing.  Errors
 *   that only the device can see (page pool exhausted, a head over
 *   max_pages_per_head, out-of-range or duplicate sequence ids) are
 *   recorded in a sticky status word inside `meta`: the offending call
 *   changes no state, and every later state-changing or attention call on
 *   the context does nothing (outputs are left untouched) until
 *   dms_clear_status().  dms_status() reads the word.
 */
#ifndef DMS_H_
#define DMS_H_

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
  DMS_OK = 0,
  DMS_ERR_INVALID = -1,       /* bad configuration or argument (host check) */
  DMS_ERR_UNSUPPORTED = -2,   /* valid but not implemented (e.g. head_dim 96) */
  DMS_ERR_HIP = -3,           /* a HIP runtime call or launch failed */
  DMS_ERR_OUT_OF_PAGES = -4,  /* device: free-page stack exhausted */
  DMS_ERR_CAPACITY = -5,      /* device: a head needs more than max_pages_per_head */
  DMS_ERR_BAD_SEQ = -6,       /* device: sequence id out of range or repeated */
  DMS_ERR_SCRATCH = -7        /* host: call too large for the static scratch of
                                 dms_decode_step_static */
};

typedef struct dms_config {
  int32_t num_layers;         /* >= 1; layers are independent caches */
  int32_t max_seqs;           /* sequence ids are 0 .. max_seqs-1 (<= 65536) */
  int32_t num_kv_heads;       /* Hkv >= 1 */
  int32_t group_size;         /* g = Hq / Hkv, 1 .. 16 (1 .. 128 for DMS_KV_MLA) */
  int32_t head_dim;           /* d: 64 or 128 (576 for DMS_KV_MLA) */
  int32_t window;             /* w >= 1: eviction delay = sliding window */
  int32_t page_size;          /* P tokens per page: 32, 64, 128 or 256 */
  int32_t num_pages;          /* pages in each layer's pool */
  int32_t max_pages_per_head; /* page-table length of one (seq, head) */
  int32_t max_chunk_tokens;   /* largest total token count of one chunk call */
  float softmax_scale;        /* <= 0 selects 1 / sqrt(head_dim) */
  int32_t eviction;           /* DMS_EVICT_DELAYED (0, the method) or
                                 DMS_EVICT_IMMEDIATE (1, the Sec. 5.3 ablation) */
  int32_t decision_source;    /* DMS_DECIDE_CALLER (0) or DMS_DECIDE_QUERY (1) */
  float decision_bias;        /* b added to the borrowed neuron (DMS_DECIDE_QUERY);
                                 -5 is the paper's training offset */
  int32_t kv_format;          /* DMS_KV_BF16 (0), DMS_KV_FP8 (1) or DMS_KV_MLA (2):
                                 how retained rows are stored in the page pools */
  int32_t quest_page_budget;  /* 0: decode attends every retained slot; B > 0:
                                 decode attends the B pages of each head that
                                 Quest's bound ranks highest (see below) */
} dms_config;

/*
 * Eviction timing (dms_config.eviction).
 *   DMS_EVICT_DELAYED: token t's own decision alpha_t evicts it at step t + w
 *     (Sec. 3.1 "Delayed Eviction via Sliding Window").
 *   DMS_EVICT_IMMEDIATE: the decision made at step t + w evicts token t at
 *     that step (Sec. 5.3, the ablation the paper compares against): key j
 *     is visible to query t iff j <= t and (j > t - w or alpha_{j+w} = 0).
 *     In the cache, token t takes token t - w's slot iff alpha_t = 1.
 *
 * Where decisions come from (dms_config.decision_source).
 *   DMS_DECIDE_CALLER: the caller passes flags (uint8, 0 = keep) to
 *     dms_append, dms_decode_step, dms_append_chunk and dms_prefill_chunk.
 *   DMS_DECIDE_QUERY: the decision of a token for KV head h is read from its
 *     query, as in App. C: alpha = round(sigmoid(x)) = (x > 0), with
 *     x = q[first query head of the group, h * g][element 0] + decision_bias,
 *     formed in float32 from the bf16 query (a tie, x = 0, keeps the token);
 *     that element is then treated as 0 by every attention call (App. C
 *     removes the borrowed neuron from attention).  Calls with a query use
 *     dms_decode_step_q / dms_prefill_chunk_q (dms_decode_step and
 *     dms_prefill_chunk return DMS_ERR_INVALID, and vice versa); appends
 *     without a query (dms_append, dms_append_chunk) still take flags.
 */
enum { DMS_EVICT_DELAYED = 0, DMS_EVICT_IMMEDIATE = 1 };

/*
 * KV storage (dms_config.kv_format).  KV quantization is one of the methods
 * the paper names as orthogonal to DMS (App. B); this combines the two.
 *   DMS_KV_BF16: rows are stored as given (bf16), 16 KB per 32-slot tile at
 *     d = 128.
 *   DMS_KV_FP8: each retained K row and V row of a (token, KV head) is
 *     stored as OCP FP8 E4M3 codes with one power-of-two scale 2^e per row,
 *     e the smallest integer with max|x| * 2^-e <= 448; codes are the
 *     round-to-nearest-even E4M3 values of x * 2^-e and the stored value is
 *     code * 2^e.  A 32-slot tile takes 64 d + 256 bytes (8.25 KB at
 *     d = 128), roughly halving the bytes decode reads.  Every key and value
 *     is attended in its stored form, including the token a decode step
 *     appends and the chunk's own tokens in a prefill call.
 *   DMS_KV_MLA: a multi-head latent attention cache, the direction the paper
 *     names for future work (Sec. 6).  Each token caches one bf16 row of
 *     d = 576 shared by all query heads: the compressed latent (dims
 *     0 .. 511) then the decoupled rotary key (dims 512 .. 575).  The cache
 *     is one KV head (num_kv_heads = 1) whose group is every query head
 *     (group_size <= 128: DeepSeek-V2-Lite has 16, DeepSeek-V2 128; decode
 *     attends groups of 16 query heads, each re-reading the rows, which
 *     the groups of one call read close together in time so that the
 *     re-reads mostly hit the L2), and DMS evicts its rows by the same
 *     rule.  Decode
 *     works in the absorbed form: q (per query head, 576 dims) is the query
 *     already mapped into the latent space followed by its rotary part; a
 *     head scores row j by q . row_j over all 576 dims and its output is the
 *     softmax-weighted sum of the rows' latent dims, so `out` holds
 *     [n][group_size][512] float32 (the up-projection of values is the
 *     caller's).  The `v` arguments are ignored (may be NULL).  Requires
 *     decision_source = DMS_DECIDE_CALLER and quest_page_budget = 0;
 *     dms_prefill_chunk attends the chunk's queries ([T][group_size][576])
 *     to the retained rows and the chunk's own rows under the DMS mask,
 *     writes [T][group_size][512] float32 and commits the rows;
 *     dms_prefill_chunk_q returns DMS_ERR_UNSUPPORTED.
 */
enum { DMS_KV_BF16 = 0, DMS_KV_FP8 = 1, DMS_KV_MLA = 2 };

/*
 * Page retrieval within the retained set (dms_config.quest_page_budget).  The
 * paper names Quest (query-aware page selection) as orthogonal to DMS and
 * combinable with it (App. A).  With a budget B > 0 the library keeps, for
 * every cache page, the channel-wise minimum and maximum of the keys in its
 * live slots (exact, recomputed for every page an append writes; bf16; keys
 * as stored, i.e. dequantized for FP8 pages).  Each decode call then scores
 * the pages of a KV head with Quest's bound U = sum_i max(q_i lo_i, q_i hi_i),
 * taking the maximum over the group's query heads (one selection per KV head,
 * shared by its group), keeps the B highest (ties: lower page index; every
 * page when a head has at most B) and attends only their live slots.  Scores
 * are float32 sums in a fixed order.  Prefill attends densely.
 * dms_quest_selection reports the last decode call's selection.  Requires
 * max_pages_per_head <= 4096.
 */
enum { DMS_DECIDE_CALLER = 0, DMS_DECIDE_QUERY = 1 };

typedef struct dms_ctx dms_ctx;

/*
 * Byte offsets of the per-layer state inside `meta` (for dms_export_state
 * readers).  Layer l's region starts at layer0 + l * layer_stride.  Arrays:
 *   pos        int32 [max_seqs]                    tokens appended per sequence
 *   len        int32 [max_seqs][Hkv]               retained slots L per head
 *   ring       int32 [max_seqs][Hkv][w]            slot of position p at p % w,
 *                                                  bit 31 = that token's flag
 *   page_table int32 [max_seqs][Hkv][max_pages_per_head]  page of slots
 *                                                  i*P .. i*P+P-1 (-1 = none)
 *   slot_meta  int32 [max_seqs][Hkv][max_pages_per_head*P] position held by
 *                                                  a live slot, bit 31 = flag
 *   stack      int32 [num_pages]                   free-page stack, entries
 *                                                  0 .. top-1 are free pages
 *   top        int32                               stack height
 * The sticky status word is the int32 at offset `status`.
 * Only entries that the method defines are meaningful: ring entries of
 * positions >= pos - w, page-table entries below ceil(L / P), slot_meta
 * entries below L, stack entries below top.
 */
typedef struct dms_state_offsets {
  size_t status, layer0, layer_stride;
  size_t pos, len, ring, page_table, slot_meta, stack, top;
  size_t page_bounds;   /* quest_page_budget > 0: bf16 [num_pages][2][d], per
                           page (by page id) the channel-wise min then max of
                           the keys in its live slots; 0 otherwise */
} dms_state_offsets;

/*
 * Page layout in a layer's pool (page i at i * page_bytes).  A slot s of a
 * head lives in page page_table[s / P], tile (s % P) / 32, row j = s % 32.
 * With h = (j / 4) % 2 and r = 4 * (j / 8) + j % 4 (row j's place among 16
 * rows), both formats store a tile in the order of the decode kernel's MFMA
 * operand loads (16-byte pieces, one contiguous 1 KB per load instruction):
 * DMS_KV_BF16: page_bytes = 4 * P * d; a page is P/32 tiles of 128 * d bytes:
 *   key (j, e)   bf16 at byte ((((e / 32) * 2 + h) * 4 + (e / 8) % 4) * 16 + r) * 16
 *                         + (e % 8) * 2 of the tile
 *   value (j, e) bf16 at byte 64 * d + (((e / 16) * 4 + j / 8) * 16 + e % 16) * 16
 *                         + (j % 8) * 2 of the tile
 * DMS_KV_FP8: page_bytes = P/32 * (64 * d + 256):
 *   key code (j, e)   at (e / 64) * 2048 + h * 1024 + (16 * ((e / 8) % 4) + r) * 16
 *                        + 8 * ((e / 32) % 2) + e % 8
 *   value code (j, e) at 32 * d + (e / 32) * 1024 + (16 * (j / 8) + e % 16) * 16
 *                        + 8 * ((e / 16) % 2) + j % 8
 *   key scale of row j (float32)   at 64 * d + (j / 8) * 64 + (j % 8) * 4
 *   value scale of row j (float32) at 64 * d + (j / 8) * 64 + 32 + (j % 8) * 4
 * DMS_KV_MLA: page_bytes = 2 * P * d (d = 576); a page is P/32 tiles of
 *   64 * d bytes holding the rows only, element (j, e) at the DMS_KV_BF16
 *   key offset above.
 */

/* Sizes of the caller-owned buffers for `cfg`.  Host only; validates cfg.
 * meta_bytes: state of all layers + status; pool_bytes: ONE layer's pool;
 * workspace_bytes: scratch shared by all calls of a context. */
int dms_layout(const dms_config* cfg, size_t* meta_bytes, size_t* pool_bytes,
               size_t* workspace_bytes, size_t* page_bytes);

/* Offsets of the state arrays in `meta`.  Host only. */
int dms_state_layout(const dms_config* cfg, dms_state_offsets* out);

/* Create a context over caller-owned device buffers.  Host only: no HIP call,
 * the state is NOT initialised (call dms_init_state).  pools_dev_host is a
 * host array of num_layers device pointers (copied). */
int dms_create(const dms_config* cfg, void* meta_dev, void* const* pools_dev_host,
               void* workspace_dev, dms_ctx** out);

/* Free the host context (never touches device memory). */
int dms_destroy(dms_ctx* ctx);

/* Initialise every layer's state: no sequences, all pages free
 * (stack[i] = num_pages-1-i, so pages are popped 0, 1, 2, ...), status 0. */
int dms_init_state(dms_ctx* ctx, void* stream);

/* Release the listed sequences in every layer (layer = -1) or one layer:
 * their pages are pushed back on the free stack (sequences in call order,
 * heads ascending, each head's pages in page-table order), and pos, L and the
 * ring are cleared.  seq_ids_dev: int32 [n]. */
int dms_seq_reset(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev, void* stream);

/* Append one token per listed sequence to one layer (Sec. 3.2 cache
 * management).  For each (sequence, KV head), with t = pos:
 *   if t >= w and the token at t - w was flagged, the new token takes that
 *   token's slot (the flagged token leaves the cache now, w steps after its
 *   decision; with DMS_EVICT_IMMEDIATE: if the new token is flagged);
 *   otherwise it takes the next fresh slot L (L += 1), popping a
 *   page when that slot starts a page.  Pops follow call order, then head.
 * Then the ring remembers (slot, flag) for position t and pos += 1.
 * k_dev, v_dev: bf16 [n, Hkv, d]; flags_dev: uint8 [n, Hkv]. */
int dms_append(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
               const void* k_dev, const void* v_dev, const uint8_t* flags_dev,
               void* stream);

/* Decode attention of one layer over the current cache (with
 * DMS_DECIDE_QUERY the borrowed neuron of q is treated as 0): every query head
 * attends to all live slots of its KV head, which are exactly the keys
 * visible to the latest position (decode reads only retained tokens; the
 * cost is the KV bytes read, Sec. 1 and Appendix I).  Split over the
 * retained tokens of all heads, merged by log-sum-exp.
 * q_dev: bf16 [n, Hq, d]; out_dev: float32 [n, Hq, d] ([n, Hq, 512] for
 * DMS_KV_MLA). */
int dms_decode(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
               const void* q_dev, float* out_dev, void* stream);

/* One decode step of one layer: dms_append of (k, v, flags) followed by
 * dms_decode of q, so the new token attends to itself and to every token
 * still retained (release of t - w, then append of t, then attention). */
int dms_decode_step(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                    const void* q_dev, const void* k_dev, const void* v_dev,
                    const uint8_t* flags_dev, float* out_dev, void* stream);

/* dms_decode_step for callers that cannot allocate device memory (code under
 * HIP graph capture, tight serving loops, harnesses that forbid hipMalloc):
 * the same append, split-K decode and merge, with everything the call needs
 * beyond its inputs, outputs and the context's state and pools (planner
 * output, split-K partials, arrival counters) kept in a static 32 MiB device
 * array inside libdms instead of the context's workspace.  The array exists
 * once per GPU (its address is resolved by dms_init_state, or by this call
 * on a device where that has not happened) and is held until the process
 * ends; the call allocates and frees nothing.
 *   Limit: with W decode waves (4 per compute unit: 1024 on MI355X) and
 *   NH = n * num_kv_heads, the call needs about
 *   (W + NH) * (128 + 4 * group_size * head_dim) + 40 * W + 40 * NH bytes;
 *   a call above 32 MiB returns DMS_ERR_SCRATCH and changes nothing (e.g.
 *   group 16, head_dim 128: up to ~3000 KV heads per call).
 *   Supported: DMS_DECIDE_CALLER, DMS_KV_BF16 or DMS_KV_FP8 pages,
 *   quest_page_budget = 0 (DMS_ERR_UNSUPPORTED otherwise).
 *   Every call on one GPU shares that GPU's array: calls that may overlap in
 *   time on one GPU (different streams, or different contexts on streams not
 *   ordered with each other) race and must not be issued; calls ordered on
 *   one stream are safe.  The array keeps the last call's contents; what must
 *   start at zero is cleared by each call.
 * Arguments, outputs and errors as for dms_decode_step. */
int dms_decode_step_static(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                           const void* q_dev, const void* k_dev, const void* v_dev,
                           const uint8_t* flags_dev, float* out_dev, void* stream);

/* dms_decode_step with decisions read from the queries (DMS_DECIDE_QUERY
 * only): the decision of each (sequence, KV head) comes from q_dev as
 * described above, and is also written to decisions_out_dev (uint8 [n, Hkv],
 * may be NULL). */
int dms_decode_step_q(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                      const void* q_dev, const void* k_dev, const void* v_dev,
                      uint8_t* decisions_out_dev, float* out_dev, void* stream);

/* Append a chunk of tokens per sequence with no attention: the result equals
 * appending them one by one in position order, except that page pops of the
 * whole call go in the order (sequence in call order, head, position).
 * cu_seqlens_dev: int32 [n+1] device array, cu[0] = 0, non-decreasing,
 * cu[n] = total_tokens <= max_chunk_tokens, no sequence longer than
 * max_seqlen (host values used to size the launch; a device array that
 * disagrees with them sets DMS_ERR_INVALID in the sticky status).
 * k_dev, v_dev: bf16 [total_tokens, Hkv, d]; flags_dev: uint8 [total_tokens, Hkv]. */
int dms_append_chunk(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                     const int32_t* cu_seqlens_dev, int total_tokens, int max_seqlen,
                     const void* k_dev, const void* v_dev, const uint8_t* flags_dev,
                     void* stream);

/* Masked chunked prefill of one layer (Sec. 3.2: DMS sparsity also skips
 * prefill work; the mask travels as the decision vector, Sec. 3.1).  Query
 * at position t of a chunk attends to the cached retained tokens and to the
 * chunk's own keys j <= t with j > t - w or flag_j = 0 -- cached tokens
 * flagged within the last w positions expire inside the chunk by the same
 * rule.  Then the chunk is committed as by dms_append_chunk.
 * Arguments as for dms_append_chunk, plus q_dev: bf16 [total_tokens, Hq, d]
 * and out_dev: float32 [total_tokens, Hq, d] (latent rows, DMS_KV_MLA: d = 576
 * for q and the rows, 512 for out; v_dev is ignored and may be NULL). */
int dms_prefill_chunk(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                      const int32_t* cu_seqlens_dev, int total_tokens, int max_seqlen,
                      const void* q_dev, const void* k_dev, const void* v_dev,
                      const uint8_t* flags_dev, float* out_dev, void* stream);

/* dms_prefill_chunk with decisions read from the queries (DMS_DECIDE_QUERY
 * only); the decisions taken are also written to decisions_out_dev (uint8
 * [total_tokens, Hkv], may be NULL). */
int dms_prefill_chunk_q(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                        const int32_t* cu_seqlens_dev, int total_tokens, int max_seqlen,
                        const void* q_dev, const void* k_dev, const void* v_dev,
                        uint8_t* decisions_out_dev, float* out_dev, void* stream);

/* Retained lengths L of the listed sequences of one layer (the paper's
 * per-step "KV-cache token reads", Sec. 5.1): out_dev int32 [n, Hkv]. */
int dms_retained_lengths(dms_ctx* ctx, int layer, int n, const int32_t* seq_ids_dev,
                         int32_t* out_dev, void* stream);

/* Page retrieval (quest_page_budget > 0): the selection of the last decode
 * call on this context, stream-ordered after it.  For its i-th (sequence,
 * KV head) pair in call order (n pairs of Hkv heads): pages_out_dev[i * B ..]
 * (int32, B = quest_page_budget) holds the attended page-table indices in
 * ascending order, and count_out_dev[i] how many (the rest are -1).  Returns
 * DMS_ERR_INVALID for a context without a budget or n outside 1 .. max_seqs
 * (pass the n of that decode call). */
int dms_quest_selection(dms_ctx* ctx, int n, int32_t* pages_out_dev, int32_t* count_out_dev,
                        void* stream);

/* Copy one layer's state region (dms_state_offsets) plus nothing else into
 * host memory: bytes must be >= layer_stride.  Synchronises `stream`. */
int dms_export_state(dms_ctx* ctx, int layer, void* dst_host, size_t bytes, void* stream);

/* Synchronise `stream` and return the sticky device status (DMS_OK or a
 * negative DMS_ERR_* code), or DMS_ERR_HIP if the copy fails. */
int dms_status(dms_ctx* ctx, void* stream);

/* Reset the sticky status to DMS_OK (enqueued on `stream`). */
int dms_clear_status(dms_ctx* ctx, void* stream);

/* Kernel timing instrumentation (not part of the method).  While a session
 * is active the library records a pair of HIP events around each split-K
 * decode kernel and each masked-prefill attention kernel it launches, for at
 * most max_launches launches in total; later launches are not recorded.
 * Events are created here and destroyed by dms_profile_stop (no device
 * memory is allocated). */
int dms_profile_start(dms_ctx* ctx, int max_launches);

enum { DMS_PROFILE_DECODE = 0, DMS_PROFILE_PREFILL = 1 };

/* Wait for the recorded events and end the session.  ms_out[k] = summed
 * duration and launches_out[k] = number of recorded launches of kernel kind
 * k (DMS_PROFILE_DECODE, DMS_PROFILE_PREFILL); both arrays have 2 entries
 * and may be NULL. */
int dms_profile_stop(dms_ctx* ctx, float* ms_out, int* launches_out);

/* Static description of an error code. */
const char* dms_strerror(int code);

/*
 * Training-time DMS attention (retrofitting, Sec. 3.1)
 * -----------------------------------------------------
 * During retrofitting every token j of every KV head carries a continuous
 * decision alpha_j in [0, 1] (Eq. 1: a Gumbel-sigmoid of the decision
 * logit), and attention adds the mask M_alpha of Fig. 1b to the scaled
 * scores: -inf for keys after the query, 0 for the w most recent positions
 * (j > t - w), log(1 - alpha_j) for older keys (alpha_j = 1 hides the key).
 * Every sequence of a call has T tokens.  Layouts (row-major, dense):
 *   q, dout   bf16 [B, T, Hq, d]       k, v      bf16 [B, T, Hkv, d]
 *   alpha     f32  [B, T, Hkv]         out       f32  [B, T, Hq, d]
 *   lse       f32  [B, Hq, T]  natural log of each softmax denominator
 *   dq        f32  [B, T, Hq, d]       dk, dv    f32  [B, T, Hkv, d]
 *   dalpha    f32  [B, T, Hkv]
 * Query head q reads KV head q / g.  Gradients are of sum(out * dout) and
 * overwrite their buffers.  The workspace (dms_train_workspace bytes) holds
 * tiled copies of the inputs; it and every buffer belong to the caller, and
 * one workspace serves one stream at a time.  Errors: DMS_ERR_INVALID /
 * DMS_ERR_UNSUPPORTED (host checks, nothing launched) or DMS_ERR_HIP.
 */
typedef struct dms_train_config {
  int32_t batch;          /* B >= 1 */
  int32_t seq_len;        /* T >= 1 */
  int32_t num_kv_heads;   /* Hkv >= 1 */
  int32_t group_size;     /* g = Hq / Hkv, 1 .. 16 */
  int32_t head_dim;       /* d: 128 */
  int32_t window;         /* w >= 1 */
  float softmax_scale;    /* <= 0 selects 1 / sqrt(head_dim) */
} dms_train_config;

int dms_train_workspace(const dms_train_config* cfg, size_t* workspace_bytes);

/* Forward: out and lse from q, k, v and the decisions. */
int dms_train_attention_fwd(const dms_train_config* cfg, const void* q_dev, const void* k_dev,
                            const void* v_dev, const float* alpha_dev, float* out_dev,
                            float* lse_dev, void* workspace_dev, void* stream);

/* Backward: dq, dk, dv, dalpha from the forward's inputs, out, lse and dout
 * (bf16).  The decision gradient is -sum_t exp(s_tj - lse_t) (dP_tj - D_t)
 * over query positions t >= j + w, finite also where alpha_j = 1. */
int dms_train_attention_bwd(const dms_train_config* cfg, const void* q_dev, const void* k_dev,
                            const void* v_dev, const float* alpha_dev, const float* out_dev,
                            const float* lse_dev, const void* dout_dev, float* dq_dev,
                            float* dk_dev, float* dv_dev, float* dalpha_dev,
                            void* workspace_dev, void* stream);

/* Gumbel-sigmoid of Eq. 1: alpha = sigmoid((logit + log u - log(1 - u)) / tau)
 * for n elements, u in (0, 1) supplied by the caller (u = 0.5 gives the
 * noise-free sigmoid); tau > 0. */
int dms_gumbel_sigmoid_fwd(int n, const float* logits_dev, const float* u_dev, float tau,
                           float* alpha_dev, void* stream);

/* dlogit = dalpha * alpha (1 - alpha) / tau. */
int dms_gumbel_sigmoid_bwd(int n, const float* alpha_dev, const float* dalpha_dev, float tau,
                           float* dlogits_dev, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* DMS_H_ */
