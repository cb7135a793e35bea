// Internal structures shared by the host planner and the gfx950 kernels.
#pragma once

#include <stdint.h>

#include <memory>
#include <string>
#include <utility>
#include <vector>

#include "halo_attn.h"

namespace halo {

// Rows of one wavefront work item: at most 16 query rows (one MFMA N tile).
constexpr int kRowsPerItem = 16;
// A wide item is one workgroup of kWideWaves waves of 32 query rows each.
constexpr int kWideWaves = 8;
constexpr int kMaxWideRows = kWideWaves * 32;
// Narrow items per workgroup (one per wave): 8 for bf16, 4 for fp32.
inline int narrow_items_per_block(halo_dtype_t dt) { return dt == HALO_BF16 ? 8 : 4; }
// Compute units of an MI355X: a decode plan with no wide items launches one
// narrow workgroup per CU.
constexpr int kNumCUs = 256;
// Fixed cost of one narrow item (metadata, Q load, output write), counted in
// keys when items are dealt to workgroups.
constexpr int kItemOverheadKeys = 64;
// Keys consumed per inner step: two pages of 16 (one K=32 MFMA for P*V).
constexpr int kKeysPerStep = 32;
// Partials per merge entry that sit at fixed workspace slots (k * n_merge + m)
// and that the merge kernel loads together with the entry's metadata.
constexpr int kMergeK0 = 8;

// One work item: up to 16 query rows (narrow, one wavefront) or up to 256
// (wide, one workgroup) against a list of key spans. 64 bytes, read by the
// scalar unit; the first span is repeated inline so that a narrow item can
// start loading keys without first reading the span table.
struct Item {
  int32_t row_begin;   // first entry in the row table
  int32_t n_rows;      // 1..16 narrow, 1..256 wide; 0: an empty slot (narrow)
  int32_t span_begin;  // first entry in the span table
  int32_t n_spans;     // >= 0
  int32_t kv_head;
  int32_t part_base;   // >= 0: the rows write partial results, each to its
                       // row's slot (Row::slot, ItemRec::aux); -1: final rows
                       // written straight to o / lse
  int32_t keys;        // visible keys, each span rounded up to whole pages
                       // (cost, for ordering only)
  int32_t flags;       // kItemStream: keys read by this item only (stream them)
  int32_t s0_key_begin;   // the first span (when n_spans > 0)
  int32_t s0_key_end;
  int32_t s0_causal;
  int32_t pad[5];
};
constexpr int32_t kItemStream = 1;

// What the 64 lanes of a narrow item's wavefront read at its start, one
// 32-bit word each (256 bytes): the q_row of each of its (up to 16) rows, a
// second word per row, and the page ids of the first 32 pages of its first
// span. The second word is the row's chunk position for a prefill item (the
// causal mask needs it; prefill rows are always final) and its partial slot
// for a decode item that writes partials (decode has no mask).
struct ItemRec {
  int32_t q_row[16];   // -1 past n_rows
  int32_t aux[16];
  int32_t page[32];
};
// A narrow item's first span is cut at this many keys, so that its page
// ids fit the record; later spans, like wide items' spans, at kMaxSpanKeys.
constexpr int kNarrowSpanKeys = 512;
// Growth room (tokens) a decode plan leaves every private segment for
// halo_plan_update_lengths: the default, and the largest allowed (the span
// cut that leaves the room assumes it is at most half of kNarrowSpanKeys).
constexpr int kDefaultAppendReserve = 256;
constexpr int kMaxAppendReserve = 256;

// A contiguous range of keys of one segment, [key_begin, key_end).
// key_begin is a multiple of kKeysPerStep and a span covers at most
// kMaxSpanKeys keys, so its page ids fit one 64-lane register.
struct Span {
  int32_t seg;
  int32_t key_begin;
  int32_t key_end;
  int32_t causal;      // 1: key j visible to a row iff j <= row.qpos
  int32_t page_off;    // index in page_ids of the page holding key_begin
  int32_t pad[3];
};
constexpr int kMaxSpanKeys = 1024;

// One query row: its row index into q / o (token * H_q + head), its
// position inside the prefill chunk (for the causal span) and, for a row
// whose keys are split over several items, its merge-list entry and the
// workspace slot of this item's partial result. The partials of merge entry
// m fill slots merge_indptr[m] .. merge_indptr[m + 1] - 1.
struct Row {
  int32_t q_row;
  int32_t qpos;
  int32_t merge_idx;   // entry in the merge list, or -1 when the row is final here
  int32_t slot;        // partial slot, or -1 when the row is final here
};

// Offsets (bytes) of the arrays packed in the device metadata buffer, in
// this order. halo_plan_update_lengths rewrites only arrays from seg_len up
// to (not including) rows, which halo_plan_upload_update relies on.
struct MetaLayout {
  size_t seg_page_off = 0;   // int32 [S]  first page slot of each segment
  size_t seg_len = 0;        // int32 [S]
  size_t page_ids = 0;       // int32 [total pages]
  size_t items = 0;          // Item  [n_narrow_blocks * narrow_slots]  narrow, by workgroup slot
  size_t item_recs = 0;      // ItemRec, one per narrow slot
  size_t wide_items = 0;     // Item  [n_wide]      wide (one kWideWaves-wave workgroup)
  size_t spans = 0;          // Span  [n_spans]
  size_t rows = 0;           // Row   [n_rows]
  size_t merge_rows = 0;     // int32 [n_merge] output row (q_row) per merge entry
  size_t merge_indptr = 0;   // int32 [n_merge + 1]
  size_t merge_parts = 0;    // int32 [n_parts] partial slot ids (merge_indptr[m] + k)
  size_t total = 0;
};

// Allocator whose value-less construct() leaves the bytes as they are, so a
// vector resized to hold the metadata image is not zero-filled first.
template <typename T>
struct DefaultInitAlloc : std::allocator<T> {
  template <typename U>
  struct rebind {
    using other = DefaultInitAlloc<U>;
  };
  DefaultInitAlloc() = default;
  template <typename U>
  DefaultInitAlloc(const DefaultInitAlloc<U>&) noexcept {}
  template <typename U>
  void construct(U* p) noexcept {
    ::new (static_cast<void*>(p)) U;
  }
  template <typename U, typename... A>
  void construct(U* p, A&&... a) {
    ::new (static_cast<void*>(p)) U(std::forward<A>(a)...);
  }
};

// A decode plan's copy of its forest; per segment its page slots in the
// image (page_slot_off, S + 1 entries: a private segment has room for the
// pages its growth reserve needs) and the lengths it may take in place,
// (len_lo, len_hi]; and per segment the spans that end at its last key (CSR
// over segments: tail_span[tail_indptr[s] .. tail_indptr[s+1])), each with
// the image byte offsets of the item whose first span it is and of that
// item's lane record (-1 if none).
struct AppendIndex {
  std::vector<int32_t> seg_len, page_indptr, page_ids, req_indptr, req_ids, refs;
  std::vector<int32_t> page_slot_off, len_lo, len_hi;
  std::vector<int32_t> tail_indptr, tail_span;
  std::vector<int64_t> tail_item, tail_rec;
};

}  // namespace halo

struct halo_plan {
  halo_attn_params_t params;
  bool prefill = false;
  int32_t num_segments = 0;
  int32_t num_requests = 0;
  int64_t num_query_rows = 0;
  int32_t n_items = 0;
  int32_t n_wide = 0;
  int32_t wide_rb = 0;       // 1 when the plan has wide items (32 rows per wave), else 0
  int32_t wide_group = 1;    // wide items that share pages, kept on one XCD
  int32_t n_narrow_blocks = 0;  // workgroups the narrow items are dealt to (a multiple of 8)
  int32_t narrow_slots = 0;     // item slots per narrow workgroup (slot k: wave k)
  int32_t n_shared_items = 0;
  int32_t n_merge = 0;
  int32_t n_spans = 0;
  int32_t n_rows = 0;
  int32_t n_merge_parts = 0;
  int32_t n_pages = 0;
  int64_t n_part_rows = 0;
  int64_t n_part_slots = 0;     // workspace slots (>= n_part_rows)
  int32_t merge_k0 = 0;         // partials per merge entry at slots k * n_merge + m
  int64_t distinct_kv_tokens = 0;
  int64_t visible_pairs = 0;
  size_t workspace_bytes = 0;
  halo::MetaLayout layout;
  std::vector<uint8_t, halo::DefaultInitAlloc<uint8_t>> meta;   // host image of the device metadata
  halo::AppendIndex append;    // decode plans: for halo_plan_update_lengths
};

namespace halo {
// Thread-local error reporting used by every entry point.
halo_status_t fail(halo_status_t st, const std::string& msg);
void clear_error();
const char* last_error();
}  // namespace halo
