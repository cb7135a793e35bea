/*
 * halo_attn.h -- C ABI of the shared-prefix paged-attention library (gfx950).
 *
 * The operation. A batch of requests (replicated agentic workflows, arXiv
 * 2509.02121 §1) shares prompt prefixes and differs in per-request suffixes
 * (§2, "Context reuse" and intra-batch prefix sharing). Their KV cache is paged
 * (§7, PagedAttention) and the sharing is a prefix forest (§7, RadixAttention):
 * segments of tokens, and for every request an ordered root-to-leaf path of
 * segment ids. Each query attends over the concatenation of its path's
 * segments with ordinary scaled dot-product attention; the result must be
 * exactly that of unshared execution (§3 "Scope", semantic preserving), up to
 * floating-point summation order. Chunked prefill of new tokens over a cached
 * prefix is the prefix-caching case of §4.1.
 *
 *   s_j  = sm_scale * <q, k_j>            for every visible key j
 *   o    = sum_j softmax(s)_j v_j,   lse = ln sum_j exp(s_j)
 *   q head h reads kv head h / (num_q_heads / num_kv_heads).
 *
 * Memory layouts (all row-major, element type = kv_dtype unless stated;
 * E = 16 / sizeof(element): 8 for bf16, 4 for fp32):
 *   k_pool  [num_pool_pages][num_kv_heads][head_dim/E][page_size][E]
 *           token t, dim c of a (page, head) tile at ((c/E)*page_size + t)*E + c%E
 *           (16-byte units, so the 16 tokens of one unit column are contiguous)
 *   v_pool  [num_pool_pages][num_kv_heads][head_dim][page_size]   dim-major;
 *           the page_size slots of a dim row hold tokens 0-3, 8-11, 4-7,
 *           12-15 (token t at slot (t & 3) | (t & 4) << 1 | (t & 8) >> 1),
 *           so the 8 tokens one MFMA lane multiplies are 16 contiguous bytes
 *   q, o    decode:  [num_requests][num_q_heads][head_dim]
 *           prefill: [sum q_len][num_q_heads][head_dim], request r's rows
 *                    follow request r-1's. o has element type out_dtype.
 *   lse     [rows][num_q_heads] float32, natural log; -inf for a row that
 *           sees no key (its o row is 0).
 * A segment of length L occupies ceil(L / page_size) pages; token t sits in
 * page seg_page_ids[seg_page_indptr[s] + t / page_size], slot t % page_size.
 * Slots past L in the last page, and pages no segment lists, may hold any
 * bits (NaN included) and never affect the results.
 *
 * Ownership. Every device buffer belongs to the caller (torch tensors in the
 * Python binding). Run calls allocate nothing and enqueue work on the
 * caller's HIP stream (passed as void*, a hipStream_t); HALO_OK means
 * "validated and enqueued". A plan is host memory owned by the library from
 * halo_plan_create until halo_plan_destroy; only halo_plan_update_lengths
 * changes it, and its uploaded device_meta is only read by runs, so several
 * streams may run one plan concurrently if each has its own workspace.
 *
 * Errors. Every call returns a halo_status_t; halo_last_error_message()
 * gives a thread-local description of the last failure. Structural checks
 * (ids in range, page counts, head ratios, dtypes) happen on the host in
 * halo_plan_create; device memory is never validated by run calls.
 */
#ifndef HALO_ATTN_H
#define HALO_ATTN_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
  HALO_OK = 0,
  HALO_ERR_INVALID_ARGUMENT = 1,   /* malformed forest, null pointer, bad size */
  HALO_ERR_UNSUPPORTED = 2,        /* valid but not built: head_dim, page size, dtype */
  HALO_ERR_WORKSPACE_TOO_SMALL = 3,
  HALO_ERR_HIP = 4,                /* a HIP runtime call or kernel launch failed */
  HALO_ERR_REPLAN = 5              /* halo_plan_update_lengths: the forest changed
                                      beyond what the plan can absorb in place */
} halo_status_t;

typedef enum { HALO_F32 = 0, HALO_BF16 = 1 } halo_dtype_t;

/* Which pool halo_kv_page_gather reads. */
typedef enum { HALO_POOL_K = 0, HALO_POOL_V = 1 } halo_pool_kind_t;

typedef struct {
  int32_t num_q_heads;      /* H_q; a multiple of num_kv_heads */
  int32_t num_kv_heads;     /* H_kv >= 1 */
  int32_t head_dim;         /* 64 or 128 */
  int32_t page_size;        /* tokens per page; 16 */
  int64_t num_pool_pages;   /* capacity of k_pool / v_pool, in pages */
  halo_dtype_t kv_dtype;    /* element type of q, k_pool, v_pool */
  halo_dtype_t out_dtype;   /* HALO_F32, or equal to kv_dtype */
  float sm_scale;           /* score scale > 0, normally 1/sqrt(head_dim) */
} halo_attn_params_t;

/* Prefix forest, HOST arrays in CSR form (§2 intra-batch prefix sharing). */
typedef struct {
  int32_t num_segments;
  const int32_t* seg_len;          /* [S] tokens per segment, >= 0 */
  const int32_t* seg_page_indptr;  /* [S+1], nondecreasing, starts at 0 */
  const int32_t* seg_page_ids;     /* [seg_page_indptr[S]] page ids in [0, num_pool_pages);
                                      segment s lists exactly ceil(seg_len[s]/page_size)
                                      pages; a page may appear in several segments */
  int32_t num_requests;
  const int32_t* req_seg_indptr;   /* [R+1] */
  const int32_t* req_seg_ids;      /* each request's path, root first; no segment twice */
  const int32_t* q_len;            /* NULL: decode, one query per request.
                                      Otherwise prefill: q_len[r] new tokens of request r,
                                      whose K/V are the LAST segment of its path
                                      (seg_len == q_len[r]); that segment may appear in
                                      no other path. Chunk query i sees chunk keys <= i
                                      and every key of the earlier segments. */
} halo_forest_t;

typedef struct halo_plan halo_plan_t;

/* Validate a forest and build the work lists of one batch step.
 * On success *plan is set, *device_meta_bytes is the size of the device
 * buffer halo_plan_upload fills, and *workspace_bytes the scratch the run
 * call needs (0 for prefill). Host arrays are copied; the caller may free
 * them on return. Returns INVALID_ARGUMENT / UNSUPPORTED with a message on
 * any malformed or unsupported input; *plan is then NULL. */
halo_status_t halo_plan_create(const halo_attn_params_t* params,
                               const halo_forest_t* forest,
                               halo_plan_t** plan,
                               size_t* device_meta_bytes,
                               size_t* workspace_bytes);

/* Tuning of the work decomposition (every field 0 or -1 means "chosen by
 * the planner from the batch"). The result never depends on these: any
 * valid setting gives the same attention, up to summation order.
 *   kc_shared        keys per chunk of a shared segment in narrow items
 *                    (multiple of 32, <= 1024; 0: 512)
 *   kc_private       keys per chunk of a request's private keys (multiple of
 *                    32, <= 65536; 0: 2048, 1024, 512 or 256, the longest
 *                    that leaves >= 3 items per CU)
 *   wide             -1: wide items (256-row MFMA workgroups over one key
 *                    stream) when the shared work is large; 0: never; 1:
 *                    always (bf16 only)
 *   wide_rows        rows per wide item (multiple of 32, <= 256; 0: from the
 *                    sharing groups' sizes; prefill: 256)
 *   kc_wide          keys per chunk of a shared segment in wide items
 *                    (multiple of 32; 0: the longest of 4096, 2048, ... that
 *                    gives >= wide_min_items items)
 *   wide_min_items   see kc_wide (0: 128)
 *   shared_unit      narrow items of one shared chunk kept together on one
 *                    workgroup (0: 4)
 *   items_per_block  narrow items per workgroup, at most one per wave
 *                    (0: one per wave, 8 for bf16 and 4 for fp32)
 *   append_reserve   decode plans: tokens every private segment (on one
 *                    path) may gain through halo_plan_update_lengths before
 *                    a new plan is needed; page-table room and span cuts
 *                    are laid out for it (1..256; 0: 256) */
typedef struct {
  int32_t kc_shared;
  int32_t kc_private;
  int32_t wide;
  int32_t wide_rows;
  int32_t kc_wide;
  int32_t wide_min_items;
  int32_t shared_unit;
  int32_t items_per_block;
  int32_t append_reserve;
} halo_plan_options_t;

/* Fill *options with the defaults (every field "chosen by the planner"). */
void halo_plan_options_default(halo_plan_options_t* options);

/* halo_plan_create with explicit tuning options (NULL: the defaults). An
 * out-of-range option is rejected with HALO_ERR_INVALID_ARGUMENT. */
halo_status_t halo_plan_create_with_options(const halo_attn_params_t* params,
                                            const halo_forest_t* forest,
                                            const halo_plan_options_t* options,
                                            halo_plan_t** plan,
                                            size_t* device_meta_bytes,
                                            size_t* workspace_bytes);

/* Decode-append update (§4.1: the plan of a decode batch is rebuilt every
 * step). Brings a decode plan up to date with `forest`, the plan's own
 * forest after tokens were appended to (or removed from) private segments
 * (segments on one path): same requests and paths, every other segment
 * unchanged (length and pages), and each changed segment's page list its
 * old list with pages appended at the end (or dropped from it). A private
 * segment of length n at planning time can take any length in
 * (b, n + append_reserve], b < n being the first key of its last span
 * (for the caller: any length >= its planning-time length up to the
 * reserve); its page table and last span were laid out with that room.
 * Only span ends, the matching inline first-span copies and record page
 * ids, the new page ids, the segment length table and the statistics
 * change; the work decomposition stays the planning-time one. While no
 * segment has changed its page count since planning, the updated host
 * image is byte for byte the image halo_plan_create would build for
 * `forest` (every decision looks at lengths in whole pages).
 * Cost: a comparison of the page tables and work proportional to the spans
 * of the changed segments.
 * Returns HALO_ERR_REPLAN, leaving the plan unchanged, when `forest` is
 * outside these bounds (build a new plan then), and
 * HALO_ERR_INVALID_ARGUMENT, also leaving it unchanged, for a new page id
 * outside [0, num_pool_pages). The caller re-uploads the plan
 * (halo_plan_upload) before the next run, and must not update a plan
 * while an upload of it is still in flight. */
halo_status_t halo_plan_update_lengths(halo_plan_t* plan, const halo_forest_t* forest);

/* Copy the plan's metadata (page ids, work lists) into device_meta, a
 * caller-owned 256-byte aligned device buffer of at least
 * device_meta_bytes, asynchronously on stream. The plan must stay alive
 * until the copy has completed. */
halo_status_t halo_plan_upload(const halo_plan_t* plan, void* device_meta,
                               size_t device_meta_bytes, void* stream);

/* halo_plan_upload of only what halo_plan_update_lengths can change (the
 * segment lengths, page ids, work items, their records and spans: about
 * half of a decode plan's metadata), for a decode loop that updates its
 * plan in place every step. device_meta must already hold an upload of
 * this same plan (halo_plan_upload, or this call, after any number of
 * updates since); after halo_plan_create, use halo_plan_upload. Same
 * arguments, errors and lifetime rules as halo_plan_upload. */
halo_status_t halo_plan_upload_update(const halo_plan_t* plan, void* device_meta,
                                      size_t device_meta_bytes, void* stream);

void halo_plan_destroy(halo_plan_t* plan);

/* Decode attention over the forest (one query per request).
 * q, k_pool, v_pool, o, device_meta, workspace: device pointers, layouts
 * above; lse may be NULL. workspace holds per-chunk partial results (O in
 * the output element type, LSE in fp32) and must be at least the plan's
 * workspace_bytes (its contents on entry do not matter). The plan must be a decode plan whose metadata was uploaded to
 * device_meta. Shared segments are read once per group of stacked query
 * rows (the grouped prefix pass, §2 intra-batch prefix sharing); partial
 * results over disjoint key ranges are combined with the exact log-sum-exp
 * rule, so the result equals unshared attention (§3 "Scope"). Launches:
 * wide items (if any), narrow items, then the merge (if any rows are split). */
halo_status_t halo_prefix_attn_decode(const halo_plan_t* plan, const void* device_meta,
                                      const void* q, const void* k_pool, const void* v_pool,
                                      void* o, float* lse,
                                      void* workspace, size_t workspace_bytes,
                                      void* stream);

/* Chunked prefill over cached prefixes (§4.1 prefix-caching discount):
 * every chunk query attends to its path's earlier segments and causally to
 * its own chunk. Arguments as for decode; the plan must be a prefill plan.
 * workspace may be NULL when the plan's workspace_bytes is 0. */
halo_status_t halo_prefix_attn_prefill(const halo_plan_t* plan, const void* device_meta,
                                       const void* q, const void* k_pool, const void* v_pool,
                                       void* o, float* lse,
                                       void* workspace, size_t workspace_bytes,
                                       void* stream);

/* Largest workspace (bytes) halo_prefix_attn_decode_noalloc can serve. */
#define HALO_NOALLOC_SCRATCH_BYTES ((size_t)64 << 20)

/* halo_prefix_attn_decode for callers that cannot allocate device memory:
 * code under HIP graph capture, tight serving loops, harnesses that forbid
 * hipMalloc. Same arguments and result as halo_prefix_attn_decode, without
 * the workspace: the partial results go to a scratch array of
 * HALO_NOALLOC_SCRATCH_BYTES that the library holds in device memory of its
 * own, one per GPU (a static device variable, so each GPU the library runs
 * on holds it until the process ends). The call allocates nothing and
 * calls no allocating routine; its first call on a device looks up that
 * device's copy of the array (hipGetSymbolAddress) and keeps the address.
 * A plan whose workspace_bytes exceeds HALO_NOALLOC_SCRATCH_BYTES is
 * rejected with HALO_ERR_WORKSPACE_TOO_SMALL and nothing is launched. Every
 * call on one GPU shares that GPU's array and nothing in it has to start at
 * zero (every partial is written before it is read); calls that overlap in
 * time on one GPU (several streams, several host threads) race on it and
 * must be serialised by the caller. */
halo_status_t halo_prefix_attn_decode_noalloc(const halo_plan_t* plan, const void* device_meta,
                                              const void* q, const void* k_pool, const void* v_pool,
                                              void* o, float* lse, void* stream);

/* Page gather (§7 PagedAttention): copy the tokens of num_seqs page lists out
 * of one pool into a dense token-major buffer, bit for bit.
 *   out[out_token_offset[i] + t][h][:] = token t of sequence i, head h
 * for t < seq_len[i], where token t lives in page page_ids[seq_page_indptr[i]
 * + t / page_size]. seq_page_indptr [num_seqs + 1] is nondecreasing and need
 * not start at 0 (a slice of a larger page list works): the slots
 * seq_page_indptr[0] .. seq_page_indptr[num_seqs] - 1 of page_ids are read.
 * pool_kind says whether pool has the k_pool or the v_pool layout. page_ids, seq_page_indptr, seq_len, out_token_offset and
 * out are DEVICE pointers; out is [*][num_kv_heads][head_dim] of kv_dtype;
 * pool and out must be 16-byte aligned.
 * Only params' num_kv_heads, head_dim, page_size, num_pool_pages and
 * kv_dtype are used. Every page of a sequence whose page count is not
 * ceil(seq_len/page_size), and every page whose id is outside
 * [0, num_pool_pages), is skipped (its tokens in out are left untouched);
 * if error_flag (device int32, may be NULL) is given, 1 is then written
 * there. 0 is never written, so the caller clears the flag beforehand. */
halo_status_t halo_kv_page_gather(const void* pool, const halo_attn_params_t* params,
                                  halo_pool_kind_t pool_kind,
                                  const int32_t* page_ids, const int32_t* seq_page_indptr,
                                  const int32_t* seq_len, const int64_t* out_token_offset,
                                  int32_t num_seqs, void* out, int32_t* error_flag,
                                  void* stream);

/* Page scatter, the write path of the paged KV cache (§7 PagedAttention;
 * §2 KV reuse: new tokens are written once, then read by every request
 * that shares them): the inverse of halo_kv_page_gather.
 *   token start + t of sequence i, head h  <-  in[in_token_offset[i] + t][h][:]
 * for 0 <= t < seq_count[i], start = seq_start[i]; the token at position p
 * of sequence i lives in page page_ids[seq_page_indptr[i] + p / page_size],
 * slot p % page_size, stored in the pool_kind layout. A decode step appends
 * one token (count 1, start = the sequence's length so far); a prefill
 * chunk writes its q_len tokens. Slots of tokens outside the written range
 * are left untouched. page_ids, seq_page_indptr, seq_start, seq_count,
 * in_token_offset and in are DEVICE pointers; in is [*][num_kv_heads]
 * [head_dim] of kv_dtype, bits copied unchanged; pool and in must be 16-byte
 * aligned. Only params' num_kv_heads,
 * head_dim, page_size, num_pool_pages and kv_dtype are used. A sequence whose
 * range does not fit its page list (start < 0 or start + count > pages *
 * page_size) is skipped whole, and a touched page whose id is outside
 * [0, num_pool_pages) is skipped (the sequence's other pages are written);
 * either way, if error_flag (device int32, may be NULL) is given, 1 is
 * written there (0 never is). Two sequences must not write the same slot.
 * in_token_offset[i] + seq_count[i] must not exceed the rows of in. */
halo_status_t halo_kv_page_scatter(void* pool, const halo_attn_params_t* params,
                                   halo_pool_kind_t pool_kind,
                                   const int32_t* page_ids, const int32_t* seq_page_indptr,
                                   const int32_t* seq_start, const int32_t* seq_count,
                                   const int64_t* in_token_offset, int32_t num_seqs,
                                   const void* in, int32_t* error_flag, void* stream);

/* halo_kv_page_scatter for the K and the V pool of the same tokens in one
 * launch: k_in goes to k_pool (HALO_POOL_K layout), v_in to v_pool
 * (HALO_POOL_V layout), with one set of page lists, ranges and input offsets.
 * The result equals the two single-pool calls; the error rules are theirs
 * (a flagged sequence or page is skipped in both pools). For a decode step,
 * whose per-pool work is a few KB, one launch instead of two halves the fixed
 * cost of the append. */
halo_status_t halo_kv_page_scatter_kv(void* k_pool, void* v_pool, const halo_attn_params_t* params,
                                      const int32_t* page_ids, const int32_t* seq_page_indptr,
                                      const int32_t* seq_start, const int32_t* seq_count,
                                      const int64_t* in_token_offset, int32_t num_seqs,
                                      const void* k_in, const void* v_in, int32_t* error_flag,
                                      void* stream);

/* Whole-page copy inside one pool, every head, bit for bit: page dst_pages[k]
 * becomes a copy of page src_pages[k], k < num_pages. This is the copy of
 * copy-on-write: before a request writes into a page it shares with others
 * (a shared prefix that ends inside a page), the caller copies that page to
 * a private one, points the request's page list at the copy and writes there.
 * Call once per pool. src_pages and dst_pages are DEVICE int32 arrays; pool
 * must be 16-byte aligned. dst pages must be distinct and none may also be a
 * src page of the same call. Ids outside [0, num_pool_pages) are skipped and
 * flagged as for the scatter. */
halo_status_t halo_kv_page_copy(void* pool, const halo_attn_params_t* params,
                                const int32_t* src_pages, const int32_t* dst_pages,
                                int32_t num_pages, int32_t* error_flag, void* stream);

/* Prefix forest from token ids (host only, no device work). The prompts of
 * a batch that share prefixes (§2 intra-batch prefix sharing: a shared
 * prefix is computed once and its KV cache reused; §1: recurring prompts are
 * detected) become the segments and paths of a halo_forest_t: a trie over
 * page_size-token chunks of the prompts (RadixAttention's radix tree, §7, at
 * page granularity, so that every shared boundary is page-aligned as the
 * paged cache needs), compressed into segments. Chunk k of request r is
 * shared by exactly the requests whose prompts agree with r's on every token
 * up to the end of that chunk and whose chunk k has the same length; a
 * segment is a maximal run of chunks shared by the same requests. So two
 * requests share page_size * floor(lcp / page_size) tokens (lcp = their
 * longest common prefix), or their whole prompts if these are identical.
 * Only a segment that ends a prompt can end inside a page, and such a
 * segment has no children.
 *   prompt_indptr  [num_requests + 1] HOST int32, prompt_indptr[0] = 0,
 *                  nondecreasing; request r's prompt is tokens[prompt_indptr[r]
 *                  .. prompt_indptr[r+1]) (any int32 token ids; empty allowed).
 * On success *tree (owned by the library until halo_prefix_tree_destroy)
 * holds the forest and *info (may be NULL) its sizes. Segment ids follow a
 * depth-first preorder with children in order of first appearance (request
 * order, then position), so the result is deterministic. */
typedef struct halo_prefix_tree halo_prefix_tree_t;

typedef struct {
  int32_t num_segments;
  int32_t num_path_entries;   /* sum over requests of their path lengths */
  int64_t num_pages;          /* sum over segments of ceil(seg_len / page_size) */
  int64_t prompt_tokens;      /* sum of prompt lengths */
  int64_t distinct_tokens;    /* sum of seg_len: tokens whose KV is stored and
                                 prefilled once (prompt_tokens minus the
                                 prefix-caching discount of §4.1) */
} halo_prefix_tree_info_t;

halo_status_t halo_prefix_tree_build(const int32_t* prompt_indptr, const int32_t* tokens,
                                     int32_t num_requests, int32_t page_size,
                                     halo_prefix_tree_t** tree, halo_prefix_tree_info_t* info);

/* Copy the forest into caller-owned HOST arrays (any pointer may be NULL):
 *   seg_len, seg_parent (-1 for a root segment), seg_refcount (requests whose
 *   paths hold the segment), seg_src_request / seg_src_offset (the segment's
 *   tokens are that request's prompt tokens from that offset on)  [num_segments];
 *   req_seg_indptr [num_requests + 1], req_seg_ids [num_path_entries]: each
 *   request's path, root first, in halo_forest_t form. */
halo_status_t halo_prefix_tree_get(const halo_prefix_tree_t* tree, int32_t* seg_len,
                                   int32_t* seg_parent, int32_t* seg_refcount,
                                   int32_t* seg_src_request, int32_t* seg_src_offset,
                                   int32_t* req_seg_indptr, int32_t* req_seg_ids);

void halo_prefix_tree_destroy(halo_prefix_tree_t* tree);

/* Plan statistics for callers and benchmarks (host memory, no device work). */
typedef struct {
  int32_t is_prefill;
  int32_t num_items;          /* narrow work items (one wavefront, <= 16 rows) */
  int32_t num_shared_items;   /* items (narrow or wide) over a segment shared by >= 2 requests */
  int32_t num_merge_rows;     /* output rows combined from several partials */
  int64_t num_partial_rows;   /* partial (o, lse) rows written to the workspace */
  int64_t num_query_rows;     /* rows of q / o */
  int64_t distinct_kv_tokens; /* sum of segment lengths, each segment once */
  int64_t visible_pairs;      /* sum over query rows and q heads of visible keys */
  int32_t num_wide_items;     /* wide work items (one 8-wave workgroup, <= 256 rows) */
  int32_t wide_row_blocks;    /* 1 when the plan has wide items (32 query rows per wave), else 0 */
} halo_plan_stats_t;

halo_status_t halo_plan_get_stats(const halo_plan_t* plan, halo_plan_stats_t* stats);

/* Read-only view of the metadata image halo_plan_upload copies to the device,
 * for inspection and host-side testing of the work lists. Byte offsets of
 * each int32 array inside the image, and the element counts:
 *   items, wide_items: n_items / n_wide x {row_begin, n_rows, span_begin,
 *                       n_spans, kv_head, partial flag (>= 0: the rows write
 *                       partials at their slots; -1: final rows), keys, flags,
 *                       first span's key_begin, key_end, causal, unused x 5}
 *                       narrow item b * narrow_slots + k runs in slot k of
 *                       narrow workgroup b; n_rows = 0 marks an empty slot
 *   item_recs: n_items x {q_row x 16 (-1 past n_rows), per row its chunk
 *                       position (prefill) or partial slot (decode item with
 *                       partials), page ids of the first 32 pages of the
 *                       first span}
 *   spans:  n_spans  x {segment, key_begin, key_end, causal, page-table offset,
 *                       unused x 3}; a span covers at most 1024 keys (512 in
 *                       a narrow item)
 *   rows:   n_rows   x {q_row = token * num_q_heads + head, chunk position,
 *                       merge entry or -1, partial slot or -1}
 *   merge_rows [n_merge], merge_indptr [n_merge + 1], merge_parts: the
 *   workspace slots of the partials combined into each listed output row,
 *   entry m's at merge_parts[merge_indptr[m] .. merge_indptr[m + 1] - 1].
 *   With k0 = min(8, most partials of an entry), entry m's k-th partial
 *   (k < k0) sits at slot k * n_merge + m, so the merge finds it without
 *   reading the list; later partials take consecutive slots after
 *   k0 * n_merge.
 * *image stays valid until halo_plan_destroy. */
typedef struct {
  uint64_t seg_page_off, seg_len, page_ids, items, wide_items, spans, rows;
  uint64_t merge_rows, merge_indptr, merge_parts, total_bytes, item_recs;
  int32_t n_items, n_wide, n_spans, n_rows, n_merge, n_merge_parts, n_pages, n_narrow_blocks;
  int32_t narrow_slots;
} halo_plan_layout_t;

halo_status_t halo_plan_inspect(const halo_plan_t* plan, const void** image,
                                halo_plan_layout_t* layout);

const char* halo_status_string(halo_status_t status);
const char* halo_last_error_message(void);

#ifdef __cplusplus
}
#endif

#endif /* HALO_ATTN_H */
