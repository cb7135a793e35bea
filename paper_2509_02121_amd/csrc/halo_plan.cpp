// Host planner: validates a prefix forest and turns it into wavefront work
// items for the gfx950 kernels. Pure host C++ (no HIP calls), so it can be
// exercised and sanitized on a machine without a GPU.
//
// Decode (arXiv 2509.02121 §2, intra-batch prefix sharing): a segment on the
// path of two or more requests is "shared". Its query rows -- every (request,
// q head) pair of one kv head -- are stacked into one work item per row
// group, so each of the segment's pages is read once per row group instead of
// once per request (the grouped prefix pass): up to 16 rows in a narrow item
// (one wavefront), or up to 256 in a wide item (one 8-wave workgroup sharing
// the key stream through LDS) when the shared work is large. Segments on one
// path only are "private"; each request's private keys are split into chunks
// (the suffix pass). Every item over a subset of a row's keys writes a
// partial (o, lse); rows with several partials are combined by the
// log-sum-exp merge, rows with exactly one write their final result directly.
//
// Prefill (§4.1, prefix caching): each item holds the (query, head) rows of
// one request and one kv head -- up to 256 in a wide item for bf16, 16 in a
// narrow item otherwise -- and walks all of that request's keys, the cached
// prefix first and its own chunk last, causally; results are final.

#include <stdlib.h>

#include <algorithm>
#include <cmath>
#include <cstring>
#include <limits>
#include <mutex>
#include <new>
#include <queue>
#include <string>
#include <vector>

#include "halo_internal.h"

namespace halo {

namespace {
thread_local std::string g_last_error;

size_t align_up(size_t x, size_t a) { return (x + a - 1) / a * a; }

int64_t ceil_div(int64_t a, int64_t b) { return (a + b - 1) / b; }
}  // namespace

halo_status_t fail(halo_status_t st, const std::string& msg) {
  g_last_error = msg;
  return st;
}

void clear_error() { g_last_error.clear(); }

const char* last_error() { return g_last_error.c_str(); }

}  // namespace halo

using namespace halo;

namespace {

halo_status_t validate(const halo_attn_params_t* p, const halo_forest_t* f) {
  if (!p || !f) return fail(HALO_ERR_INVALID_ARGUMENT, "params and forest must not be NULL");
  if (p->num_kv_heads < 1 || p->num_q_heads < 1)
    return fail(HALO_ERR_INVALID_ARGUMENT, "num_q_heads and num_kv_heads must be >= 1");
  if (p->num_q_heads % p->num_kv_heads != 0)
    return fail(HALO_ERR_INVALID_ARGUMENT, "num_q_heads must be a multiple of num_kv_heads");
  if (p->head_dim != 64 && p->head_dim != 128)
    return fail(HALO_ERR_UNSUPPORTED, "head_dim must be 64 or 128, got " + std::to_string(p->head_dim));
  if (p->page_size != 16)
    return fail(HALO_ERR_UNSUPPORTED, "page_size must be 16, got " + std::to_string(p->page_size));
  if (p->kv_dtype != HALO_F32 && p->kv_dtype != HALO_BF16)
    return fail(HALO_ERR_UNSUPPORTED, "kv_dtype must be HALO_F32 or HALO_BF16");
  if (p->out_dtype != HALO_F32 && p->out_dtype != p->kv_dtype)
    return fail(HALO_ERR_UNSUPPORTED, "out_dtype must be HALO_F32 or equal to kv_dtype");
  if (p->num_pool_pages < 0 || p->num_pool_pages > (int64_t)std::numeric_limits<int32_t>::max())
    return fail(HALO_ERR_INVALID_ARGUMENT, "num_pool_pages must be in [0, 2^31)");
  if (!std::isfinite(p->sm_scale) || !(p->sm_scale > 0.f))
    return fail(HALO_ERR_INVALID_ARGUMENT, "sm_scale must be finite and > 0");
  if (f->num_segments < 0 || f->num_requests < 0)
    return fail(HALO_ERR_INVALID_ARGUMENT, "num_segments and num_requests must be >= 0");
  const int S = f->num_segments, R = f->num_requests;
  if (S > 0 && (!f->seg_len || !f->seg_page_indptr))
    return fail(HALO_ERR_INVALID_ARGUMENT, "seg_len / seg_page_indptr must not be NULL");
  if (!f->req_seg_indptr) return fail(HALO_ERR_INVALID_ARGUMENT, "req_seg_indptr must not be NULL");
  if (S == 0 && f->seg_page_indptr == nullptr) {
    // fine: no segments at all
  } else if (f->seg_page_indptr[0] != 0) {
    return fail(HALO_ERR_INVALID_ARGUMENT, "seg_page_indptr[0] must be 0");
  }
  for (int s = 0; s < S; ++s) {
    const int32_t len = f->seg_len[s];
    if (len < 0) return fail(HALO_ERR_INVALID_ARGUMENT, "seg_len[" + std::to_string(s) + "] < 0");
    const int64_t np = (int64_t)f->seg_page_indptr[s + 1] - f->seg_page_indptr[s];
    if (np != ceil_div(len, p->page_size))
      return fail(HALO_ERR_INVALID_ARGUMENT,
                  "segment " + std::to_string(s) + " lists " + std::to_string(np) +
                      " pages but its length " + std::to_string(len) + " needs " +
                      std::to_string(ceil_div(len, p->page_size)));
  }
  const int64_t total_pages = S ? f->seg_page_indptr[S] : 0;
  if (total_pages > 0 && !f->seg_page_ids)
    return fail(HALO_ERR_INVALID_ARGUMENT, "seg_page_ids must not be NULL");
  for (int64_t i = 0; i < total_pages; ++i) {
    const int32_t pg = f->seg_page_ids[i];
    if (pg < 0 || pg >= p->num_pool_pages)
      return fail(HALO_ERR_INVALID_ARGUMENT, "page id " + std::to_string(pg) + " at slot " +
                                                 std::to_string(i) + " outside [0, num_pool_pages)");
  }
  if (f->req_seg_indptr[0] != 0) return fail(HALO_ERR_INVALID_ARGUMENT, "req_seg_indptr[0] must be 0");
  for (int r = 0; r < R; ++r)
    if (f->req_seg_indptr[r + 1] < f->req_seg_indptr[r])
      return fail(HALO_ERR_INVALID_ARGUMENT, "req_seg_indptr must be nondecreasing");
  const int64_t total_refs = f->req_seg_indptr[R];
  if (total_refs > 0 && !f->req_seg_ids)
    return fail(HALO_ERR_INVALID_ARGUMENT, "req_seg_ids must not be NULL");
  std::vector<int32_t> seen(S, -1);
  for (int r = 0; r < R; ++r) {
    for (int32_t i = f->req_seg_indptr[r]; i < f->req_seg_indptr[r + 1]; ++i) {
      const int32_t s = f->req_seg_ids[i];
      if (s < 0 || s >= S)
        return fail(HALO_ERR_INVALID_ARGUMENT, "request " + std::to_string(r) + " names segment " +
                                                   std::to_string(s) + " outside [0, num_segments)");
      if (seen[s] == r)
        return fail(HALO_ERR_INVALID_ARGUMENT,
                    "request " + std::to_string(r) + " lists segment " + std::to_string(s) + " twice");
      seen[s] = r;
    }
  }
  if (f->q_len) {
    std::vector<int32_t> refs(S, 0);
    for (int64_t i = 0; i < total_refs; ++i) refs[f->req_seg_ids[i]]++;
    for (int r = 0; r < R; ++r) {
      const int32_t n = f->q_len[r];
      if (n < 0) return fail(HALO_ERR_INVALID_ARGUMENT, "q_len must be >= 0");
      const int32_t a = f->req_seg_indptr[r], b = f->req_seg_indptr[r + 1];
      if (a == b) {
        if (n != 0)
          return fail(HALO_ERR_INVALID_ARGUMENT,
                      "prefill request " + std::to_string(r) + " has queries but an empty path");
        continue;
      }
      const int32_t last = f->req_seg_ids[b - 1];
      if (f->seg_len[last] != n)
        return fail(HALO_ERR_INVALID_ARGUMENT, "prefill request " + std::to_string(r) +
                                                   ": last segment length " +
                                                   std::to_string(f->seg_len[last]) +
                                                   " != q_len " + std::to_string(n));
      if (refs[last] != 1)
        return fail(HALO_ERR_INVALID_ARGUMENT, "prefill request " + std::to_string(r) +
                                                   ": its chunk segment appears in another path");
    }
  }
  return HALO_OK;
}

// Split [0, len) into pieces of at most `chunk` keys (chunk % 32 == 0).
void pieces(int32_t seg, int32_t len, int32_t chunk, std::vector<Span>& out) {
  for (int32_t kb = 0; kb < len; kb += chunk)
    out.push_back(Span{seg, kb, std::min(len, kb + chunk), 0, 0, {0, 0, 0}});
}

// The planner's large arrays are thread-local and keep their capacity from
// one call to the next (returned empty): a decode loop plans every step, and
// first touches of fresh multi-megabyte allocations (page faults) cost about
// as much as the planning itself. Tag tells the arrays of one type apart.
template <typename V, int Tag>
V& scratch() {
  static thread_local V v;
  v.clear();
  return v;
}

// The metadata image of the last plan destroyed, kept for the next plan
// (one buffer, the largest seen): same reason.
std::mutex g_spare_mu;
std::vector<uint8_t, DefaultInitAlloc<uint8_t>> g_spare_meta;

}  // namespace

extern "C" void halo_plan_options_default(halo_plan_options_t* o) {
  if (!o) return;
  o->kc_shared = 0;
  o->kc_private = 0;
  o->wide = -1;
  o->wide_rows = 0;
  o->kc_wide = 0;
  o->wide_min_items = 0;
  o->shared_unit = 0;
  o->items_per_block = 0;
  o->append_reserve = 0;
}

namespace {
halo_status_t check_options(const halo_plan_options_t& o) {
  auto bad = [](const char* what) { return fail(HALO_ERR_INVALID_ARGUMENT, std::string("options: ") + what); };
  if (o.kc_shared < 0 || o.kc_shared % 32 || o.kc_shared > kMaxSpanKeys)
    return bad("kc_shared is 0 or a multiple of 32 up to 1024");
  if (o.kc_private < 0 || o.kc_private % 32 || o.kc_private > (1 << 16))
    return bad("kc_private is 0 or a multiple of 32 up to 65536");
  if (o.wide < -1 || o.wide > 1) return bad("wide is -1, 0 or 1");
  if (o.wide_rows < 0 || o.wide_rows % 32 || o.wide_rows > kMaxWideRows)
    return bad("wide_rows is 0 or a multiple of 32 up to 256");
  if (o.kc_wide < 0 || o.kc_wide % 32 || o.kc_wide > (1 << 16)) return bad("kc_wide is 0 or a multiple of 32 up to 65536");
  if (o.wide_min_items < 0) return bad("wide_min_items must be >= 0");
  if (o.shared_unit < 0 || o.shared_unit > 64) return bad("shared_unit is 0..64");
  if (o.items_per_block < 0 || o.items_per_block > 8) return bad("items_per_block is 0..8");
  if (o.append_reserve < 0 || o.append_reserve > kMaxAppendReserve) return bad("append_reserve is 0..256");
  return HALO_OK;
}
}  // namespace

extern "C" halo_status_t halo_plan_create(const halo_attn_params_t* params,
                                          const halo_forest_t* forest, halo_plan_t** plan_out,
                                          size_t* device_meta_bytes, size_t* workspace_bytes) {
  return halo_plan_create_with_options(params, forest, nullptr, plan_out, device_meta_bytes, workspace_bytes);
}

extern "C" halo_status_t halo_plan_create_with_options(const halo_attn_params_t* params,
                                                       const halo_forest_t* forest,
                                                       const halo_plan_options_t* options,
                                                       halo_plan_t** plan_out, size_t* device_meta_bytes,
                                                       size_t* workspace_bytes) {
  clear_error();
  if (!plan_out) return fail(HALO_ERR_INVALID_ARGUMENT, "plan must not be NULL");
  *plan_out = nullptr;
  halo_plan_options_t opt;
  halo_plan_options_default(&opt);
  if (options) opt = *options;
  halo_status_t st = check_options(opt);
  if (st != HALO_OK) return st;
  st = validate(params, forest);
  if (st != HALO_OK) return st;
  const halo_attn_params_t& p = *params;
  const halo_forest_t& f = *forest;
  const int S = f.num_segments, R = f.num_requests;
  const int Hq = p.num_q_heads, Hkv = p.num_kv_heads, G = Hq / Hkv;
  const bool prefill = f.q_len != nullptr;

  int64_t n_q_rows = R;
  std::vector<int64_t> tok0(R + 1, 0);
  if (prefill) {
    for (int r = 0; r < R; ++r) tok0[r + 1] = tok0[r] + f.q_len[r];
    n_q_rows = tok0[R];
  } else {
    for (int r = 0; r <= R; ++r) tok0[r] = r;
  }
  if (n_q_rows * Hq > (int64_t)std::numeric_limits<int32_t>::max())
    return fail(HALO_ERR_INVALID_ARGUMENT, "query rows * num_q_heads must be < 2^31");

  halo_plan* plan = new (std::nothrow) halo_plan();
  if (!plan) return fail(HALO_ERR_INVALID_ARGUMENT, "out of host memory");
  plan->params = p;
  plan->prefill = prefill;
  plan->num_segments = S;
  plan->num_requests = R;
  plan->num_query_rows = n_q_rows;

  auto path_begin = [&](int r) { return f.req_seg_indptr[r]; };
  auto path_end = [&](int r) { return f.req_seg_indptr[r + 1]; };
  // Every decision below (chunk lengths, packing, ordering, dealing) looks
  // at lengths rounded up to whole pages, so tokens appended inside pages a
  // segment already holds change no decision: halo_plan_update_lengths
  // relies on it.
  auto paged = [&](int64_t n) { return ceil_div(n, p.page_size) * p.page_size; };

  std::vector<int32_t> refs(S, 0);
  for (int r = 0; r < R; ++r)
    for (int32_t i = path_begin(r); i < path_end(r); ++i) refs[f.req_seg_ids[i]]++;
  for (int s = 0; s < S; ++s) plan->distinct_kv_tokens += f.seg_len[s];

  // Work items as (rows, spans) before part ids are assigned.
  struct Proto {
    std::vector<Row> rows;
    std::vector<Span> spans;
    int32_t kv_head;
    int64_t keys;
    bool shared;
    bool wide;
    int32_t chunk = -1;   // shared items: id of the (piece, kv head) whose pages they read
  };
  auto& protos = scratch<std::vector<Proto>, 0>();
  int32_t n_chunks = 0;

  if (!prefill) {
    const int kc_shared = opt.kc_shared > 0 ? opt.kc_shared : 512;
    // Private chunks: the longest of 2048, 1024, 512 and 256 keys that
    // still leaves >= 3 items per CU (longer chunks write and merge fewer
    // partials; with fewer items a CU has too few loads in flight), else 256.
    auto private_items = [&](int64_t kc) {
      int64_t n = 0;
      for (int r = 0; r < R; ++r) {
        int64_t priv = 0;
        for (int32_t i = path_begin(r); i < path_end(r); ++i)
          if (refs[f.req_seg_ids[i]] == 1) priv += paged(f.seg_len[f.req_seg_ids[i]]);
        n += ceil_div(priv, kc) * Hkv;
      }
      return n;
    };
    int kc_private_default = 256;
    for (int kc : {2048, 1024, 512})
      if (private_items(kc) >= 3 * kNumCUs) {
        kc_private_default = kc;
        break;
      }
    const int kc_private = opt.kc_private > 0 ? opt.kc_private : kc_private_default;
    for (int r = 0; r < R; ++r) {
      int64_t keys = 0;
      for (int32_t i = path_begin(r); i < path_end(r); ++i) keys += f.seg_len[f.req_seg_ids[i]];
      plan->visible_pairs += keys * Hq;
    }
    // Grouped prefix pass: shared segments, all their rows stacked. With
    // bf16 inputs and enough shared work the rows go to wide items (an 8-wave
    // workgroup reading each page once for up to 256 rows); the rows per item
    // follow the row-weighted size of the shared groups, and the key chunk
    // (at most 4096 keys) shrinks until there are >= 128 wide items. Longer
    // chunks mean fewer partials to write and merge, and a wide item's ring
    // start-up and 256-row epilogue are paid fewer times.
    std::vector<std::vector<int32_t>> seg_reqs(S);
    for (int r = 0; r < R; ++r)
      for (int32_t i = path_begin(r); i < path_end(r); ++i) seg_reqs[f.req_seg_ids[i]].push_back(r);
    // Wide items pay off once the shared work is large: below ~16M
    // (row, key) pairs the grouped pass is a small fraction of the call and
    // narrow items (more of them, no LDS barriers) finish sooner.
    double shared_work = 0, wsum = 0, wrows = 0;
    for (int s = 0; s < S; ++s)
      if (refs[s] >= 2 && f.seg_len[s] > 0) {
        const double w = (double)f.seg_len[s] * refs[s];
        shared_work += w * G * Hkv;
        wsum += w;
        wrows += w * (double)refs[s] * G;
      }
    const bool wide = p.kv_dtype == HALO_BF16 &&
                      (opt.wide == 1 || (opt.wide == -1 && shared_work >= 16.0 * (1 << 20)));
    int rows_per = kRowsPerItem;
    int kc = kc_shared;
    if (wide) {
      const double avg_rows = wsum > 0 ? wrows / wsum : 0;
      plan->wide_rb = 1;
      // rows per wide item: the row-weighted group size rounded up to whole
      // 32-row waves, at most one workgroup
      rows_per = (int)std::min<double>(kMaxWideRows, std::max(32.0, std::ceil(avg_rows / 32.0) * 32.0));
      if (opt.wide_rows > 0) rows_per = opt.wide_rows;
      // row groups of one shared chunk read the same pages: keep up to 8 of
      // them on one XCD
      plan->wide_group = (int)std::min<double>(8, std::max(1.0, std::ceil(avg_rows / rows_per)));
      const int min_items = opt.wide_min_items > 0 ? opt.wide_min_items : 128;
      kc = 4 * kMaxSpanKeys;
      while (kc > 128) {
        int64_t n = 0;
        for (int s = 0; s < S; ++s)
          if (refs[s] >= 2 && f.seg_len[s] > 0)
            n += ceil_div(f.seg_len[s], kc) * ceil_div((int64_t)refs[s] * G, rows_per) * Hkv;
        if (n >= min_items) break;
        kc /= 2;
      }
      if (opt.kc_wide > 0) kc = opt.kc_wide;
    }
    for (int s = 0; s < S; ++s) {
      if (refs[s] < 2 || f.seg_len[s] == 0) continue;
      std::vector<Span> sp;
      pieces(s, f.seg_len[s], kc, sp);
      for (int g = 0; g < Hkv; ++g) {
        std::vector<Row> rows;
        for (int32_t r : seg_reqs[s])
          for (int j = 0; j < G; ++j) rows.push_back(Row{(int32_t)(r * Hq + g * G + j), 0, -1, -1});
        // chunk-major, row group innermost: items reading the same pages
        // are neighbours in the launch order.
        for (const Span& piece : sp) {
          for (size_t rb = 0; rb < rows.size(); rb += rows_per) {
            Proto pr;
            pr.rows.assign(rows.begin() + rb, rows.begin() + std::min(rows.size(), rb + (size_t)rows_per));
            pr.spans = {piece};
            pr.kv_head = g;
            pr.keys = paged(piece.key_end - piece.key_begin);
            pr.shared = true;
            pr.wide = wide;
            pr.chunk = n_chunks;
            protos.push_back(std::move(pr));
          }
          n_chunks++;
        }
      }
    }
    // Suffix pass: each request's private keys, in chunks.
    for (int r = 0; r < R; ++r) {
      std::vector<Span> sp;
      for (int32_t i = path_begin(r); i < path_end(r); ++i) {
        const int32_t s = f.req_seg_ids[i];
        if (refs[s] == 1 && f.seg_len[s] > 0) pieces(s, f.seg_len[s], kc_private, sp);
      }
      // pack consecutive pieces into chunks of at most kc_private keys
      std::vector<std::vector<Span>> chunks;
      int64_t cur = 0;
      for (const Span& piece : sp) {
        const int64_t n = paged(piece.key_end - piece.key_begin);
        if (chunks.empty() || cur + n > kc_private) {
          chunks.emplace_back();
          cur = 0;
        }
        chunks.back().push_back(piece);
        cur += n;
      }
      for (int g = 0; g < Hkv; ++g)
        for (auto& ch : chunks) {
          int64_t keys = 0;
          for (auto& x : ch) keys += paged(x.key_end - x.key_begin);
          for (int j0 = 0; j0 < G; j0 += kRowsPerItem) {
            Proto pr;
            for (int j = j0; j < std::min(G, j0 + kRowsPerItem); ++j)
              pr.rows.push_back(Row{(int32_t)(r * Hq + g * G + j), 0, -1, -1});
            pr.spans = ch;
            pr.kv_head = g;
            pr.keys = keys;
            pr.shared = false;
            pr.wide = false;
            protos.push_back(std::move(pr));
          }
        }
    }
  } else {
    // Prefill: bf16 rows go to wide items of up to kMaxWideRows (query, head) rows.
    const bool wide = p.kv_dtype == HALO_BF16 && opt.wide != 0;
    plan->wide_rb = wide ? 1 : 0;
    plan->wide_group = 1;
    const int rows_per = wide ? (opt.wide_rows > 0 ? opt.wide_rows : kMaxWideRows) : kRowsPerItem;
    for (int r = 0; r < R; ++r) {
      const int32_t n = f.q_len[r];
      if (n == 0) continue;
      const int32_t a = path_begin(r), b = path_end(r);
      const int32_t chunk_seg = f.req_seg_ids[b - 1];
      int64_t prefix_keys = 0;
      std::vector<Span> prefix_spans;
      for (int32_t i = a; i < b - 1; ++i) {
        const int32_t s = f.req_seg_ids[i];
        if (f.seg_len[s] > 0) prefix_spans.push_back(Span{s, 0, f.seg_len[s], 0, 0, {0, 0, 0}});
        prefix_keys += f.seg_len[s];
      }
      plan->visible_pairs += ((int64_t)n * prefix_keys + (int64_t)n * (n + 1) / 2) * Hq;
      for (int g = 0; g < Hkv; ++g) {
        std::vector<Row> rows;
        for (int32_t i = 0; i < n; ++i)
          for (int j = 0; j < G; ++j)
            rows.push_back(Row{(int32_t)((tok0[r] + i) * Hq + g * G + j), i, -1, -1});
        for (size_t rb = 0; rb < rows.size(); rb += rows_per) {
          Proto pr;
          pr.rows.assign(rows.begin() + rb, rows.begin() + std::min(rows.size(), rb + (size_t)rows_per));
          int32_t qmin = n, qmax = 0;
          for (auto& x : pr.rows) {
            qmin = std::min(qmin, x.qpos);
            qmax = std::max(qmax, x.qpos);
          }
          pr.spans = prefix_spans;
          // keys up to the group's first position are visible to every row:
          // that part of the chunk (whole 32-key steps) needs no mask
          const int32_t open = std::min(std::min(n, qmax + 1), (qmin + 1) / 32 * 32);
          if (open > 0) pr.spans.push_back(Span{chunk_seg, 0, open, 0, 0, {0, 0, 0}});
          if (std::min(n, qmax + 1) > open)
            pr.spans.push_back(Span{chunk_seg, open, std::min(n, qmax + 1), 1, 0, {0, 0, 0}});
          pr.kv_head = g;
          pr.keys = prefix_keys + qmax + 1;
          pr.shared = false;
          pr.wide = wide;
          protos.push_back(std::move(pr));
        }
      }
    }
  }

  // Parts per output row; items whose rows all have a single part write
  // their final result directly.
  auto& n_parts = scratch<std::vector<int32_t>, 1>();
  n_parts.assign(n_q_rows * Hq, 0);
  for (auto& pr : protos)
    for (auto& row : pr.rows) n_parts[row.q_row]++;
  // Rows that see no key at all get an item with no spans, which writes
  // O = 0 and LSE = -inf.
  if (!prefill) {
    std::vector<std::vector<Row>> empty(Hkv);
    for (int64_t qr = 0; qr < n_q_rows * Hq; ++qr)
      if (n_parts[qr] == 0) empty[(qr % Hq) / G].push_back(Row{(int32_t)qr, 0, -1, -1});
    for (int g = 0; g < Hkv; ++g)
    for (size_t i = 0; i < empty[g].size(); i += kRowsPerItem) {
      Proto pr;
      pr.rows.assign(empty[g].begin() + i, empty[g].begin() + std::min(empty[g].size(), i + kRowsPerItem));
      pr.kv_head = g;
      pr.keys = 0;
      pr.shared = false;
      pr.wide = false;
      for (auto& row : pr.rows) n_parts[row.q_row] = 1;
      protos.push_back(std::move(pr));
    }
  }
  auto& is_final = scratch<std::vector<char>, 0>();
  is_final.assign(protos.size(), 0);
  for (size_t i = 0; i < protos.size(); ++i) {
    bool all_one = true;
    for (auto& row : protos[i].rows) all_one &= (n_parts[row.q_row] == 1);
    is_final[i] = prefill || all_one;
  }

  // Shared items first, then private ones; longest first within each class
  // (stable: items reading the same pages stay neighbours).
  auto& order = scratch<std::vector<size_t>, 0>();
  order.resize(protos.size());
  for (size_t i = 0; i < order.size(); ++i) order[i] = i;
  std::stable_sort(order.begin(), order.end(), [&](size_t a, size_t b) {
    if (protos[a].shared != protos[b].shared) return protos[a].shared;
    return protos[a].keys > protos[b].keys;
  });

  // Page slots of the image: each segment's pages, and after those of a
  // private segment of a decode plan (on at most one path) room for the
  // pages its growth reserve can open, so that halo_plan_update_lengths
  // never has to move another segment's page ids.
  const int32_t reserve =
      prefill ? 0 : (opt.append_reserve > 0 ? opt.append_reserve : kDefaultAppendReserve);
  auto& slot_off = scratch<std::vector<int32_t>, 20>();
  slot_off.assign(S + 1, 0);
  for (int s = 0; s < S; ++s) {
    const int64_t n = (int64_t)slot_off[s] + (f.seg_page_indptr[s + 1] - f.seg_page_indptr[s]) +
                      (!prefill && refs[s] < 2 ? ceil_div(reserve, p.page_size) : 0);
    if (n > (int64_t)std::numeric_limits<int32_t>::max()) {
      delete plan;
      return fail(HALO_ERR_INVALID_ARGUMENT, "too many pages");
    }
    slot_off[s + 1] = (int32_t)n;
  }
  auto& page_slots = scratch<std::vector<int32_t>, 21>();
  page_slots.assign(slot_off[S], 0);
  for (int s = 0; s < S; ++s)
    std::copy(f.seg_page_ids + f.seg_page_indptr[s], f.seg_page_ids + f.seg_page_indptr[s + 1],
              page_slots.begin() + slot_off[s]);

  auto& items = scratch<std::vector<Item>, 0>();
  auto& witems = scratch<std::vector<Item>, 1>();
  auto& item_chunk = scratch<std::vector<int32_t>, 2>();   // per narrow item: its proto's chunk id
  auto& spans = scratch<std::vector<Span>, 0>();
  auto& rows = scratch<std::vector<Row>, 0>();
  // Partial rows of each output row, in item order (CSR over q rows).
  auto& parts_indptr = scratch<std::vector<int32_t>, 3>();
  auto& parts_of = scratch<std::vector<int32_t>, 4>();
  {
    size_t n_rows_all = 0, n_spans_all = 0, n_wide = 0;
    if (!prefill) parts_indptr.assign(n_q_rows * Hq + 1, 0);
    for (size_t i = 0; i < protos.size(); ++i) {
      const Proto& pr = protos[i];
      n_rows_all += pr.rows.size();
      n_wide += pr.wide ? 1 : 0;
      for (const Span& sp : pr.spans)
        n_spans_all += (size_t)((sp.key_end - sp.key_begin + kNarrowSpanKeys - 1) / kNarrowSpanKeys) + 1;
      if (!prefill && !is_final[i])
        for (const Row& row : pr.rows) parts_indptr[row.q_row + 1]++;
    }
    rows.reserve(n_rows_all);
    spans.reserve(n_spans_all);
    witems.reserve(n_wide);
    items.reserve(protos.size() - n_wide);
    item_chunk.reserve(protos.size() - n_wide);
    if (!prefill) {
      for (size_t q = 0; q + 1 < parts_indptr.size(); ++q) parts_indptr[q + 1] += parts_indptr[q];
      parts_of.resize(parts_indptr.back());
    }
  }
  auto& parts_fill = scratch<std::vector<int32_t>, 5>();
  parts_fill.assign(prefill ? 0 : n_q_rows * Hq, 0);
  int64_t part_rows = 0;
  for (size_t oi : order) {
    Proto& pr = protos[oi];
    Item it{};
    it.row_begin = (int32_t)rows.size();
    it.n_rows = (int32_t)pr.rows.size();
    it.span_begin = (int32_t)spans.size();
    it.kv_head = pr.kv_head;
    it.keys = (int32_t)std::min<int64_t>(pr.keys, std::numeric_limits<int32_t>::max());
    // Private keys of a decode item are read by no other item: stream them
    // past the caches.
    it.flags = (!prefill && !pr.shared && !pr.wide) ? kItemStream : 0;
    if (is_final[oi]) {
      it.part_base = -1;
    } else {
      if (part_rows + it.n_rows > (int64_t)std::numeric_limits<int32_t>::max()) {
        delete plan;
        return fail(HALO_ERR_INVALID_ARGUMENT, "too many partial rows");
      }
      it.part_base = (int32_t)part_rows;
      for (int i = 0; i < it.n_rows; ++i) {
        const int32_t q = pr.rows[i].q_row;
        parts_of[parts_indptr[q] + parts_fill[q]++] = (int32_t)(part_rows + i);
      }
      part_rows += it.n_rows;
    }
    if (pr.shared) plan->n_shared_items++;
    rows.insert(rows.end(), pr.rows.begin(), pr.rows.end());
    // Split spans: a narrow item's first span at kNarrowSpanKeys (its page
    // ids travel in the item's record), every other span at kMaxSpanKeys
    // (its page ids fill one 64-lane register); resolve their page slots.
    // The last span of a private segment of a decode plan keeps `reserve`
    // keys of room below its cap (when it would not, its keys are cut in
    // two, the second part being a later span), so that
    // halo_plan_update_lengths can grow it in place. The cut looks at whole
    // pages only.
    for (const Span& sp : pr.spans) {
      const bool tail = !prefill && refs[sp.seg] == 1 && sp.key_end == f.seg_len[sp.seg];
      const int32_t room = tail ? reserve : 0;
      for (int64_t kb = sp.key_begin; kb < sp.key_end;) {
        const bool first = !pr.wide && (int32_t)spans.size() == it.span_begin;
        const int32_t cap = first ? kNarrowSpanKeys : kMaxSpanKeys;
        const int64_t rest = paged(sp.key_end - kb);
        const int64_t take = rest > cap            ? cap
                             : rest + room <= cap ? rest
                                                  : std::max<int64_t>(kKeysPerStep, rest / 2 / kKeysPerStep * kKeysPerStep);
        Span piece = sp;
        piece.key_begin = (int32_t)kb;
        piece.key_end = (int32_t)std::min<int64_t>(sp.key_end, kb + take);
        piece.page_off = slot_off[sp.seg] + (int32_t)(kb / p.page_size);
        spans.push_back(piece);
        kb += take;
      }
    }
    it.n_spans = (int32_t)spans.size() - it.span_begin;
    if (it.n_spans > 0) {
      const Span& s0 = spans[it.span_begin];
      it.s0_key_begin = s0.key_begin;
      it.s0_key_end = s0.key_end;
      it.s0_causal = s0.causal;
    }
    (pr.wide ? witems : items).push_back(it);
    if (!pr.wide) item_chunk.push_back(pr.chunk);
  }

  // Merge list: every decode row no final item writes, i.e. every row with
  // partial results (several, or one from an item that also holds
  // multi-part rows); the merge kernel combines them after the attention
  // kernels.
  // Workspace slots: the first k0 = min(kMergeK0, most partials of an entry)
  // partials of merge entry m sit at slots k * n_merge + m, so the merge
  // kernel finds them from m alone and loads them in the same round trip as
  // the entry's metadata; partials past k0 take consecutive slots after
  // k0 * n_merge. merge_parts lists every entry's slots in order.
  auto& merge_rows = scratch<std::vector<int32_t>, 6>();
  auto& merge_indptr = scratch<std::vector<int32_t>, 7>();
  auto& merge_parts = scratch<std::vector<int32_t>, 8>();
  merge_indptr.push_back(0);
  int64_t n_slots = 0;
  int32_t merge_k0 = 0;
  if (!prefill) {
    auto& merge_of = scratch<std::vector<int32_t>, 9>();
    merge_of.assign(n_q_rows * Hq, -1);
    auto& slot_of_part = scratch<std::vector<int32_t>, 10>();
    slot_of_part.assign(part_rows, -1);
    size_t most = 0;
    for (int64_t qr = 0; qr < n_q_rows * Hq; ++qr) {
      const size_t np = (size_t)(parts_indptr[qr + 1] - parts_indptr[qr]);
      if (np == 0) continue;   // written by a final item
      merge_of[qr] = (int32_t)merge_rows.size();
      merge_rows.push_back((int32_t)qr);
      most = std::max(most, np);
    }
    merge_parts.reserve(parts_of.size());
    merge_indptr.reserve(merge_rows.size() + 1);
    const int64_t nm = (int64_t)merge_rows.size();
    merge_k0 = (int32_t)std::min<size_t>(kMergeK0, most);
    int64_t next = merge_k0 * nm;
    for (int64_t m = 0; m < nm; ++m) {
      const int32_t qr = merge_rows[m];
      const int32_t b0 = parts_indptr[qr], b1 = parts_indptr[qr + 1];
      for (int32_t k = 0; k < b1 - b0; ++k) {
        const int64_t slot = (int64_t)k < merge_k0 ? (int64_t)k * nm + m : next++;
        slot_of_part[parts_of[b0 + k]] = (int32_t)slot;
        merge_parts.push_back((int32_t)slot);
      }
      merge_indptr.push_back((int32_t)merge_parts.size());
    }
    n_slots = next;
    if (n_slots > (int64_t)std::numeric_limits<int32_t>::max()) {
      delete plan;
      return fail(HALO_ERR_INVALID_ARGUMENT, "too many partial slots");
    }
    for (const std::vector<Item>* list : {&items, &witems})
      for (const Item& it : *list)
        if (it.part_base >= 0)
          for (int32_t k = 0; k < it.n_rows; ++k) {
            Row& row = rows[it.row_begin + k];
            row.merge_idx = merge_of[row.q_row];
            row.slot = slot_of_part[it.part_base + k];
          }
  }

  // Narrow items are dealt to workgroups ahead of time: workgroup b has
  // `slots` item slots (one per wave), and item b * slots + k, if not empty,
  // runs in slot k. Workgroup b runs on XCD b % 8 (dispatch is round-robin),
  // and the row groups of one shared chunk go to workgroups of one XCD, in
  // units of up to shared_unit items on one workgroup, so re-reads of the
  // chunk hit that XCD's L2 or the CU's L1.
  //  * One round (at most one workgroup per CU): a CU ingests only ~30 GB/s
  //    from HBM (~70 GB/s from L2), so the batch is spread over every CU
  //    (256 workgroups) and units go longest first to the least loaded
  //    workgroup of their XCD.
  //  * Several rounds: a workgroup holds its CU until its longest item ends
  //    (a new 8-wave workgroup needs all its wave slots free), so each
  //    workgroup gets units of about the same length: units are taken
  //    longest first and fill the open workgroup of their XCD (shared) or
  //    of the XCD with the fewest items (private). Workgroups then launch
  //    longest first, and the short ones fill the tail.
  auto& recs = scratch<std::vector<ItemRec>, 0>();
  const int64_t n_real_items = (int64_t)items.size();
  if (!items.empty()) {
    const int waves = narrow_items_per_block(p.kv_dtype);
    const int64_t n = (int64_t)items.size();
    const int slots = waves;
    const int cap = opt.items_per_block > 0 ? std::min(opt.items_per_block, slots) : slots;
    if (n > (int64_t)std::numeric_limits<int32_t>::max() / 2) {
      delete plan;
      return fail(HALO_ERR_INVALID_ARGUMENT, "too many narrow work items");
    }
    const bool rounds = (int64_t)witems.size() + (n + cap - 1) / cap > kNumCUs;
    int64_t nb = std::max<int64_t>((n + cap - 1) / cap, std::min<int64_t>(n, kNumCUs));
    nb = (nb + 7) / 8 * 8;
    const int shared_unit = std::min(cap, opt.shared_unit > 0 ? opt.shared_unit : 4);
    // work units: runs of up to shared_unit items of one chunk, or one item
    struct Unit { int32_t first, count, chunk; int64_t cost; };
    std::vector<Unit> units;
    auto cost_of = [&](const Item& it) { return (int64_t)it.keys + kItemOverheadKeys; };
    for (int32_t i = 0; i < (int32_t)n; ++i) {
      const int32_t c = item_chunk[i];
      if (c >= 0 && !units.empty() && units.back().chunk == c && units.back().count < shared_unit &&
          units.back().first + units.back().count == i) {
        units.back().count++;
        units.back().cost += cost_of(items[i]);
      } else {
        units.push_back(Unit{i, 1, c, cost_of(items[i])});
      }
    }
    std::stable_sort(units.begin(), units.end(), [](const Unit& a, const Unit& b) { return a.cost > b.cost; });
    std::vector<std::vector<int32_t>> blk;
    if (rounds) {
      // per XCD, its workgroups in launch order; the last one is open
      std::vector<std::vector<std::vector<int32_t>>> xb(8);
      std::vector<int64_t> xitems(8, 0);
      for (const Unit& u : units) {
        int x = 0;
        if (u.chunk >= 0) {
          x = u.chunk % 8;
        } else {
          for (int y = 1; y < 8; ++y)
            if (xitems[y] < xitems[x]) x = y;
        }
        if (xb[x].empty() || (int)xb[x].back().size() + u.count > cap) xb[x].emplace_back();
        for (int32_t k = 0; k < u.count; ++k) xb[x].back().push_back(u.first + k);
        xitems[x] += u.count;
      }
      size_t per_xcd = 0;
      for (int x = 0; x < 8; ++x) per_xcd = std::max(per_xcd, xb[x].size());
      nb = 8 * (int64_t)per_xcd;
      blk.assign(nb, {});
      for (int x = 0; x < 8; ++x)
        for (size_t j = 0; j < xb[x].size(); ++j) blk[j * 8 + x].swap(xb[x][j]);
    }
    if (nb * slots > (int64_t)std::numeric_limits<int32_t>::max()) {
      delete plan;
      return fail(HALO_ERR_INVALID_ARGUMENT, "too many narrow work items");
    }
    // one round: one min-heap of (load, block) per XCD over the blocks with
    // room left
    using Slot = std::pair<int64_t, int32_t>;
    std::vector<std::priority_queue<Slot, std::vector<Slot>, std::greater<Slot>>> heap(8);
    if (!rounds) {
      blk.assign(nb, {});
      for (int32_t b = 0; b < (int32_t)nb; ++b) heap[b % 8].push(Slot{0, b});
    }
    // place `count` items from `first` on the least loaded block of XCD x
    // with room for them; false if there is none
    auto place_on = [&](int x, int32_t first, int32_t count, int64_t cost) {
      std::vector<Slot> aside;
      bool ok = false;
      while (!heap[x].empty()) {
        Slot s0 = heap[x].top();
        heap[x].pop();
        if ((int)blk[s0.second].size() + count <= cap) {
          for (int32_t k = 0; k < count; ++k) blk[s0.second].push_back(first + k);
          s0.first += cost;
          if ((int)blk[s0.second].size() < cap) heap[x].push(s0);
          ok = true;
          break;
        }
        aside.push_back(s0);
      }
      for (const Slot& s0 : aside) heap[x].push(s0);
      return ok;
    };
    auto least_loaded_xcd = [&]() {
      int x = -1;
      for (int y = 0; y < 8; ++y)
        if (!heap[y].empty() && (x < 0 || heap[y].top() < heap[x].top())) x = y;
      return x;
    };
    for (const Unit& u : units) {
      if (rounds) break;
      if (u.chunk >= 0 && place_on(u.chunk % 8, u.first, u.count, u.cost)) continue;
      const int x = least_loaded_xcd();
      if (x >= 0 && place_on(x, u.first, u.count, u.cost)) continue;
      // no block has room for the whole unit: deal its items one by one
      for (int32_t k = 0; k < u.count; ++k) {
        const int y = least_loaded_xcd();
        if (y < 0 || !place_on(y, u.first + k, 1, cost_of(items[u.first + k]))) {
          delete plan;
          return fail(HALO_ERR_INVALID_ARGUMENT, "internal: narrow items do not fit their workgroups");
        }
      }
    }
    // slot layout, empty slots n_rows = 0; and each slot's lane record
    auto& dealt = scratch<std::vector<Item>, 2>();
    dealt.assign((size_t)(nb * slots), Item{});
    recs.assign((size_t)(nb * slots), ItemRec{});
    for (int64_t b = 0; b < nb; ++b)
      for (size_t k = 0; k < blk[b].size(); ++k) {
        const size_t at = (size_t)(b * slots) + k;
        const Item& it = items[blk[b][k]];
        dealt[at] = it;
        ItemRec& rc = recs[at];
        for (int r = 0; r < 16; ++r) {
          rc.q_row[r] = r < it.n_rows ? rows[it.row_begin + r].q_row : -1;
          rc.aux[r] = r >= it.n_rows ? 0 : it.part_base >= 0 ? rows[it.row_begin + r].slot
                                                             : rows[it.row_begin + r].qpos;
        }
        if (it.n_spans > 0) {
          const Span& s0 = spans[it.span_begin];
          const int32_t np = (s0.key_end - s0.key_begin + p.page_size - 1) / p.page_size;
          for (int32_t j = 0; j < np && j < 32; ++j) rc.page[j] = page_slots[s0.page_off + j];
        }
      }
    items.swap(dealt);
    plan->n_narrow_blocks = (int32_t)nb;
    plan->narrow_slots = slots;
  }
  plan->n_items = (int32_t)n_real_items;
  plan->n_wide = (int32_t)witems.size();
  if (plan->n_wide == 0) plan->wide_rb = 0;
  plan->n_spans = (int32_t)spans.size();
  plan->n_rows = (int32_t)rows.size();
  plan->n_merge_parts = (int32_t)merge_parts.size();
  plan->n_merge = (int32_t)merge_rows.size();
  plan->n_part_rows = part_rows;
  plan->n_part_slots = n_slots;
  plan->merge_k0 = merge_k0;
  const size_t D = (size_t)p.head_dim;
  // partial O rows in the output element type, then one fp32 LSE per row
  const int64_t part_elem = p.out_dtype == HALO_F32 ? 4 : 2;
  plan->workspace_bytes =
      n_slots ? align_up(n_slots * D * part_elem, 256) + align_up(n_slots * sizeof(float), 256) : 0;

  // Pack the device metadata image.
  MetaLayout L;
  size_t off = 0;
  auto place = [&](size_t bytes) {
    size_t o = off;
    off = align_up(off + bytes, 256);
    return o;
  };
  const int64_t total_pages = slot_off[S];
  plan->n_pages = (int32_t)total_pages;
  L.seg_page_off = place(sizeof(int32_t) * std::max(S, 1));
  L.seg_len = place(sizeof(int32_t) * std::max(S, 1));
  L.page_ids = place(sizeof(int32_t) * std::max<int64_t>(total_pages, 1));
  L.items = place(sizeof(Item) * std::max<size_t>(items.size(), 1));
  L.item_recs = place(sizeof(ItemRec) * std::max<size_t>(recs.size(), 1));
  L.wide_items = place(sizeof(Item) * std::max<size_t>(witems.size(), 1));
  L.spans = place(sizeof(Span) * std::max<size_t>(spans.size(), 1));
  L.rows = place(sizeof(Row) * std::max<size_t>(rows.size(), 1));
  L.merge_rows = place(sizeof(int32_t) * std::max<size_t>(merge_rows.size(), 1));
  L.merge_indptr = place(sizeof(int32_t) * merge_indptr.size());
  L.merge_parts = place(sizeof(int32_t) * std::max<size_t>(merge_parts.size(), 1));
  L.total = off;
  plan->layout = L;
  // (the image is not zero-filled first: each array is copied in and the
  // rest of its 256-byte-aligned place is zeroed)
  {
    std::lock_guard<std::mutex> lock(g_spare_mu);
    plan->meta.swap(g_spare_meta);
  }
  plan->meta.clear();
  plan->meta.resize(L.total);
  uint8_t* m = plan->meta.data();
  {
    const struct { size_t at; const void* src; size_t bytes; } parts[] = {
        {L.seg_page_off, slot_off.data(), S ? sizeof(int32_t) * S : 0},
        {L.seg_len, f.seg_len, S ? sizeof(int32_t) * S : 0},
        {L.page_ids, page_slots.data(), sizeof(int32_t) * (size_t)total_pages},
        {L.items, items.data(), sizeof(Item) * items.size()},
        {L.item_recs, recs.data(), sizeof(ItemRec) * recs.size()},
        {L.wide_items, witems.data(), sizeof(Item) * witems.size()},
        {L.spans, spans.data(), sizeof(Span) * spans.size()},
        {L.rows, rows.data(), sizeof(Row) * rows.size()},
        {L.merge_rows, merge_rows.data(), sizeof(int32_t) * merge_rows.size()},
        {L.merge_indptr, merge_indptr.data(), sizeof(int32_t) * merge_indptr.size()},
        {L.merge_parts, merge_parts.data(), sizeof(int32_t) * merge_parts.size()},
    };
    const size_t n = sizeof(parts) / sizeof(parts[0]);
    for (size_t i = 0; i < n; ++i) {
      const size_t end = i + 1 < n ? parts[i + 1].at : L.total;
      if (parts[i].bytes) memcpy(m + parts[i].at, parts[i].src, parts[i].bytes);
      memset(m + parts[i].at + parts[i].bytes, 0, end - parts[i].at - parts[i].bytes);
    }
  }

  // What halo_plan_update_lengths needs: the forest the plan was built for,
  // the page slots, and for every segment the spans that end at its last
  // key (with the image offsets of the item whose first span it is, whose
  // inline copy of the span must follow, and of that item's lane record),
  // and the lengths it may take in place: above the first key of each of
  // those spans, and within their caps and the segment's page slots.
  if (!prefill) {
    AppendIndex& ax = plan->append;
    const int64_t n_refs = f.req_seg_indptr[R];
    ax.seg_len.assign(f.seg_len, f.seg_len + S);
    ax.page_indptr.assign(f.seg_page_indptr, f.seg_page_indptr + S + 1);
    ax.page_ids.assign(f.seg_page_ids, f.seg_page_ids + (S ? f.seg_page_indptr[S] : 0));
    ax.req_indptr.assign(f.req_seg_indptr, f.req_seg_indptr + R + 1);
    ax.req_ids.assign(f.req_seg_ids, f.req_seg_ids + n_refs);
    ax.refs = refs;
    ax.page_slot_off = slot_off;
    std::vector<int64_t> first_of(spans.size(), -1), rec_of(spans.size(), -1);
    for (size_t i = 0; i < items.size(); ++i)
      if (items[i].n_rows > 0 && items[i].n_spans > 0) {
        first_of[items[i].span_begin] = (int64_t)(L.items + i * sizeof(Item));
        rec_of[items[i].span_begin] = (int64_t)(L.item_recs + i * sizeof(ItemRec));
      }
    for (size_t i = 0; i < witems.size(); ++i)
      if (witems[i].n_spans > 0) first_of[witems[i].span_begin] = (int64_t)(L.wide_items + i * sizeof(Item));
    ax.tail_indptr.assign(S + 1, 0);
    for (const Span& sp : spans)
      if (sp.key_end == f.seg_len[sp.seg]) ax.tail_indptr[sp.seg + 1]++;
    for (int s = 0; s < S; ++s) ax.tail_indptr[s + 1] += ax.tail_indptr[s];
    ax.tail_span.resize(ax.tail_indptr[S]);
    ax.tail_item.resize(ax.tail_indptr[S]);
    ax.tail_rec.resize(ax.tail_indptr[S]);
    ax.len_lo.assign(S, -1);
    ax.len_hi.resize(S);
    // (lengths past the int32 range are never reached: clamp)
    auto clamp32 = [](int64_t v) { return (int32_t)std::min<int64_t>(v, std::numeric_limits<int32_t>::max()); };
    for (int s = 0; s < S; ++s)
      ax.len_hi[s] = refs[s] == 0 ? clamp32((int64_t)(slot_off[s + 1] - slot_off[s]) * p.page_size) : f.seg_len[s];
    std::vector<int32_t> fill(ax.tail_indptr.begin(), ax.tail_indptr.end() - 1);
    for (size_t i = 0; i < spans.size(); ++i) {
      const Span& sp = spans[i];
      if (sp.key_end != f.seg_len[sp.seg]) continue;
      const int32_t k = fill[sp.seg]++;
      ax.tail_span[k] = (int32_t)i;
      ax.tail_item[k] = first_of[i];
      ax.tail_rec[k] = rec_of[i];
      if (refs[sp.seg] == 1) {
        const int32_t s = sp.seg;
        const int32_t cap = rec_of[i] >= 0 ? kNarrowSpanKeys : kMaxSpanKeys;
        const int32_t slots_end = clamp32((int64_t)(slot_off[s + 1] - slot_off[s]) * p.page_size);
        const bool first_tail = k == ax.tail_indptr[s];
        ax.len_lo[s] = std::max(ax.len_lo[s], sp.key_begin);
        ax.len_hi[s] = std::min(first_tail ? slots_end : ax.len_hi[s], clamp32((int64_t)sp.key_begin + cap));
      }
    }
  }

  *plan_out = plan;
  if (device_meta_bytes) *device_meta_bytes = L.total;
  if (workspace_bytes) *workspace_bytes = plan->workspace_bytes;
  return HALO_OK;
}

extern "C" void halo_plan_destroy(halo_plan_t* plan) {
  if (plan) {
    std::lock_guard<std::mutex> lock(g_spare_mu);
    if (plan->meta.capacity() > g_spare_meta.capacity()) g_spare_meta.swap(plan->meta);
  }
  delete plan;
}

extern "C" halo_status_t halo_plan_get_stats(const halo_plan_t* plan, halo_plan_stats_t* st) {
  clear_error();
  if (!plan || !st) return fail(HALO_ERR_INVALID_ARGUMENT, "plan and stats must not be NULL");
  st->is_prefill = plan->prefill ? 1 : 0;
  st->num_items = plan->n_items;
  st->num_wide_items = plan->n_wide;
  st->wide_row_blocks = plan->wide_rb;
  st->num_shared_items = plan->n_shared_items;
  st->num_merge_rows = plan->n_merge;
  st->num_partial_rows = plan->n_part_rows;
  st->num_query_rows = plan->num_query_rows;
  st->distinct_kv_tokens = plan->distinct_kv_tokens;
  st->visible_pairs = plan->visible_pairs;
  return HALO_OK;
}

extern "C" halo_status_t halo_plan_inspect(const halo_plan_t* plan, const void** image,
                                           halo_plan_layout_t* out) {
  clear_error();
  if (!plan || !image || !out) return fail(HALO_ERR_INVALID_ARGUMENT, "plan, image and layout must not be NULL");
  const MetaLayout& L = plan->layout;
  *image = plan->meta.data();
  out->seg_page_off = L.seg_page_off;
  out->seg_len = L.seg_len;
  out->page_ids = L.page_ids;
  out->items = L.items;
  out->item_recs = L.item_recs;
  out->wide_items = L.wide_items;
  out->spans = L.spans;
  out->rows = L.rows;
  out->merge_rows = L.merge_rows;
  out->merge_indptr = L.merge_indptr;
  out->merge_parts = L.merge_parts;
  out->total_bytes = L.total;
  out->n_items = plan->n_narrow_blocks * plan->narrow_slots;
  out->n_narrow_blocks = plan->n_narrow_blocks;
  out->narrow_slots = plan->narrow_slots;
  out->n_wide = plan->n_wide;
  out->n_spans = plan->n_spans;
  out->n_rows = plan->n_rows;
  out->n_merge = plan->n_merge;
  out->n_merge_parts = plan->n_merge_parts;
  out->n_pages = plan->n_pages;
  return HALO_OK;
}

extern "C" const char* halo_status_string(halo_status_t s) {
  switch (s) {
    case HALO_OK: return "HALO_OK";
    case HALO_ERR_INVALID_ARGUMENT: return "HALO_ERR_INVALID_ARGUMENT";
    case HALO_ERR_UNSUPPORTED: return "HALO_ERR_UNSUPPORTED";
    case HALO_ERR_WORKSPACE_TOO_SMALL: return "HALO_ERR_WORKSPACE_TOO_SMALL";
    case HALO_ERR_HIP: return "HALO_ERR_HIP";
    case HALO_ERR_REPLAN: return "HALO_ERR_REPLAN";
  }
  return "HALO_ERR_UNKNOWN";
}

extern "C" const char* halo_last_error_message(void) { return halo::last_error(); }

extern "C" halo_status_t halo_plan_update_lengths(halo_plan_t* plan, const halo_forest_t* forest) {
  clear_error();
  if (!plan || !forest) return fail(HALO_ERR_INVALID_ARGUMENT, "plan and forest must not be NULL");
  if (plan->prefill || forest->q_len)
    return fail(HALO_ERR_REPLAN, "only decode plans and decode forests can be updated");
  const AppendIndex& ax = plan->append;
  const int S = plan->num_segments, R = plan->num_requests;
  const halo_forest_t& f = *forest;
  auto same = [](const int32_t* a, const std::vector<int32_t>& b) {
    return b.empty() || (a && memcmp(a, b.data(), sizeof(int32_t) * b.size()) == 0);
  };
  if (f.num_segments != S || f.num_requests != R || !f.seg_len || !f.seg_page_indptr || !f.req_seg_indptr ||
      !same(f.req_seg_indptr, ax.req_indptr) || !same(f.req_seg_ids, ax.req_ids))
    return fail(HALO_ERR_REPLAN, "requests or paths differ from the plan's forest");
  if (f.seg_page_indptr[0] != 0 || (f.seg_page_indptr[S] > 0 && !f.seg_page_ids))
    return fail(HALO_ERR_REPLAN, "malformed page table");
  // Check everything before changing anything.
  const int32_t ps = plan->params.page_size;
  bool pages_moved = false;
  for (int s = 0; s < S; ++s) {
    const int32_t len = f.seg_len[s], old = ax.seg_len[s];
    const int32_t* now = f.seg_page_ids + f.seg_page_indptr[s];
    const int32_t* was = ax.page_ids.data() + ax.page_indptr[s];
    const int64_t np = (int64_t)f.seg_page_indptr[s + 1] - f.seg_page_indptr[s];
    const int64_t np_old = ax.page_indptr[s + 1] - ax.page_indptr[s];
    if (len == old) {
      if (np != np_old || (np && memcmp(now, was, sizeof(int32_t) * np) != 0))
        return fail(HALO_ERR_REPLAN, "the pages of segment " + std::to_string(s) + " changed");
      continue;
    }
    if (ax.refs[s] >= 2) return fail(HALO_ERR_REPLAN, "shared segment " + std::to_string(s) + " changed length");
    if (len <= ax.len_lo[s] || len > ax.len_hi[s])
      return fail(HALO_ERR_REPLAN, "segment " + std::to_string(s) + " left the length range its plan can absorb");
    if (np != ceil_div(len, ps))
      return fail(HALO_ERR_REPLAN, "segment " + std::to_string(s) + " lists the wrong number of pages");
    if (memcmp(now, was, sizeof(int32_t) * std::min(np, np_old)) != 0)
      return fail(HALO_ERR_REPLAN, "the pages segment " + std::to_string(s) + " kept changed");
    for (int64_t j = np_old; j < np; ++j)
      if (now[j] < 0 || now[j] >= plan->params.num_pool_pages)
        return fail(HALO_ERR_INVALID_ARGUMENT, "page id out of range in segment " + std::to_string(s));
    pages_moved |= np != np_old;
  }
  uint8_t* m = plan->meta.data();
  const MetaLayout& L = plan->layout;
  AppendIndex& mx = plan->append;
  int32_t* slots = reinterpret_cast<int32_t*>(m + L.page_ids);
  for (int s = 0; s < S; ++s) {
    const int32_t len = f.seg_len[s], old = mx.seg_len[s];
    if (len == old) continue;
    const int64_t np = ceil_div(len, ps), np_old = ceil_div(old, ps);
    if (np > np_old)
      memcpy(slots + mx.page_slot_off[s] + np_old, f.seg_page_ids + f.seg_page_indptr[s] + np_old,
             sizeof(int32_t) * (np - np_old));
    for (int32_t k = mx.tail_indptr[s]; k < mx.tail_indptr[s + 1]; ++k) {
      Span* sp = reinterpret_cast<Span*>(m + L.spans) + mx.tail_span[k];
      sp->key_end = len;
      if (mx.tail_item[k] >= 0) reinterpret_cast<Item*>(m + mx.tail_item[k])->s0_key_end = len;
      if (mx.tail_rec[k] >= 0 && np != np_old) {
        // the record holds the span's first 32 page ids
        ItemRec* rc = reinterpret_cast<ItemRec*>(m + mx.tail_rec[k]);
        const int64_t n = std::min<int64_t>(32, ceil_div(len - sp->key_begin, ps));
        for (int64_t j = 0; j < n; ++j) rc->page[j] = slots[sp->page_off + j];
      }
    }
    reinterpret_cast<int32_t*>(m + L.seg_len)[s] = len;
    plan->distinct_kv_tokens += len - old;
    plan->visible_pairs += (int64_t)(len - old) * mx.refs[s] * plan->params.num_q_heads;
    mx.seg_len[s] = len;
  }
  if (pages_moved) {
    mx.page_indptr.assign(f.seg_page_indptr, f.seg_page_indptr + S + 1);
    mx.page_ids.assign(f.seg_page_ids, f.seg_page_ids + f.seg_page_indptr[S]);
  }
  return HALO_OK;
}
