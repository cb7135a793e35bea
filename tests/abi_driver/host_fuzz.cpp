// Host-only exercise of the planner and the prefix-tree builder, built by
// the CPU tests together with halo_plan.cpp and halo_forest.cpp under
// AddressSanitizer and UndefinedBehaviorSanitizer (no GPU code, no HIP).
//
// For seeded random prompt sets: prefix tree -> forest -> page table -> plan
// (random valid tuning options, decode and prefill), inspection, statistics,
// in-page length updates checked byte for byte against fresh plans; then
// malformed forests, which must be refused with an error status. Exits 0
// when every check holds; any sanitizer report aborts the run.

#include <stdint.h>
#include <stdio.h>
#include <string.h>

#include <algorithm>
#include <vector>

#include "halo_attn.h"

namespace {

uint64_t g_state = 0x9E3779B97F4A7C15ull;
uint32_t next_u32() {   // xorshift64*
  g_state ^= g_state >> 12;
  g_state ^= g_state << 25;
  g_state ^= g_state >> 27;
  return (uint32_t)((g_state * 0x2545F4914F6CDD1Dull) >> 32);
}
int uniform(int lo, int hi) { return hi <= lo ? lo : lo + (int)(next_u32() % (uint32_t)(hi - lo + 1)); }

int g_fail = 0;
#define CHECK(c)                                                   \
  do {                                                             \
    if (!(c)) {                                                    \
      fprintf(stderr, "check failed at line %d: %s\n", __LINE__, #c); \
      ++g_fail;                                                    \
    }                                                              \
  } while (0)

struct Forest {
  std::vector<int32_t> seg_len, page_indptr, page_ids, req_indptr, req_ids, q_len;
  int32_t pool_pages = 0;
  halo_forest_t view() {
    halo_forest_t f{};
    f.num_segments = (int32_t)seg_len.size();
    f.seg_len = seg_len.data();
    f.seg_page_indptr = page_indptr.data();
    f.seg_page_ids = page_ids.data();
    f.num_requests = (int32_t)req_indptr.size() - 1;
    f.req_seg_indptr = req_indptr.data();
    f.req_seg_ids = req_ids.data();
    f.q_len = q_len.empty() ? nullptr : q_len.data();
    return f;
  }
};

// Prompts with shared prefixes: a few roots, each prompt a root's prefix of
// random length plus its own tokens.
bool tree_forest(int n_req, int max_root, int max_own, bool prefill, Forest& out) {
  std::vector<std::vector<int32_t>> roots(uniform(1, 4));
  for (auto& r : roots) {
    r.resize(uniform(0, max_root));
    for (auto& t : r) t = uniform(0, 50);
  }
  std::vector<int32_t> indptr{0}, tokens;
  for (int i = 0; i < n_req; ++i) {
    const auto& r = roots[uniform(0, (int)roots.size() - 1)];
    const int keep = uniform(0, (int)r.size());
    tokens.insert(tokens.end(), r.begin(), r.begin() + keep);
    const int own = uniform(prefill ? 1 : 0, max_own);
    for (int k = 0; k < own; ++k) tokens.push_back(uniform(0, 50));
    indptr.push_back((int32_t)tokens.size());
  }
  halo_prefix_tree_t* tree = nullptr;
  halo_prefix_tree_info_t info{};
  halo_status_t st = halo_prefix_tree_build(indptr.data(), tokens.data(), n_req, 16, &tree, &info);
  if (st != HALO_OK) {
    // a prompt that is empty (decode with no own tokens and no prefix) is
    // refused; any other refusal is a failure
    CHECK(st == HALO_ERR_INVALID_ARGUMENT);
    return false;
  }
  out.seg_len.assign(info.num_segments, 0);
  std::vector<int32_t> parent(info.num_segments), refc(info.num_segments), src_r(info.num_segments),
      src_o(info.num_segments);
  out.req_indptr.assign(n_req + 1, 0);
  out.req_ids.assign(info.num_path_entries, 0);
  CHECK(halo_prefix_tree_get(tree, out.seg_len.data(), parent.data(), refc.data(), src_r.data(), src_o.data(),
                             out.req_indptr.data(), out.req_ids.data()) == HALO_OK);
  halo_prefix_tree_destroy(tree);
  int64_t pages = 0;
  out.page_indptr.assign(1, 0);
  for (int32_t n : out.seg_len) {
    pages += (n + 15) / 16;
    out.page_indptr.push_back((int32_t)pages);
  }
  CHECK(pages == info.num_pages);
  out.pool_pages = (int32_t)pages + uniform(1, 64);
  std::vector<int32_t> perm(out.pool_pages);
  for (int i = 0; i < out.pool_pages; ++i) perm[i] = i;
  for (int i = out.pool_pages - 1; i > 0; --i) std::swap(perm[i], perm[uniform(0, i)]);
  out.page_ids.assign(perm.begin(), perm.begin() + pages);
  out.q_len.clear();
  if (prefill) {
    // the last segment of every path is the request's chunk
    for (int r = 0; r < n_req; ++r) {
      const int32_t last = out.req_ids[out.req_indptr[r + 1] - 1];
      out.q_len.push_back(out.seg_len[last]);
    }
  }
  return true;
}

std::vector<uint8_t> image_of(const halo_plan_t* plan) {
  const void* img = nullptr;
  halo_plan_layout_t lay{};
  CHECK(halo_plan_inspect(plan, &img, &lay) == HALO_OK);
  const uint8_t* b = static_cast<const uint8_t*>(img);
  return std::vector<uint8_t>(b, b + lay.total_bytes);
}

halo_plan_options_t random_options() {
  halo_plan_options_t o;
  halo_plan_options_default(&o);
  if (uniform(0, 1)) return o;
  const int kcs[] = {0, 32, 96, 256, 512};
  o.kc_shared = kcs[uniform(0, 4)];
  o.kc_private = kcs[uniform(0, 4)] * uniform(1, 4);
  o.wide = uniform(-1, 1);
  o.wide_rows = 32 * uniform(0, 8);
  o.kc_wide = 32 * uniform(0, 64);
  o.wide_min_items = uniform(0, 300);
  o.shared_unit = uniform(0, 8);
  o.items_per_block = uniform(0, 8);
  o.append_reserve = uniform(0, 256);
  return o;
}

void one_case(bool prefill) {
  Forest fo;
  const int n_req = uniform(1, prefill ? 24 : 160);
  if (!tree_forest(n_req, uniform(0, 600), uniform(0, 300), prefill, fo)) return;
  const int hkv = uniform(1, 3), g = 1 << uniform(0, 4);
  halo_attn_params_t p{};
  p.num_q_heads = hkv * g;
  p.num_kv_heads = hkv;
  p.head_dim = uniform(0, 1) ? 128 : 64;
  p.page_size = 16;
  p.num_pool_pages = fo.pool_pages;
  p.kv_dtype = uniform(0, 1) ? HALO_BF16 : HALO_F32;
  p.out_dtype = uniform(0, 1) ? HALO_F32 : p.kv_dtype;
  p.sm_scale = 0.125f;
  const halo_plan_options_t opt = random_options();
  halo_forest_t f = fo.view();
  halo_plan_t* plan = nullptr;
  size_t meta = 0, ws = 0;
  halo_status_t st = halo_plan_create_with_options(&p, &f, &opt, &plan, &meta, &ws);
  CHECK(st == HALO_OK);
  if (st != HALO_OK) {
    fprintf(stderr, "  %s\n", halo_last_error_message());
    return;
  }
  halo_plan_stats_t stats{};
  CHECK(halo_plan_get_stats(plan, &stats) == HALO_OK);
  CHECK(image_of(plan).size() == meta);
  if (!prefill) {
    // tokens appended inside existing pages of private segments
    const std::vector<int32_t> base_len = fo.seg_len;
    std::vector<int32_t> refs(fo.seg_len.size(), 0);
    for (int32_t s : fo.req_ids) refs[s]++;
    for (int round = 0; round < 2; ++round) {
      for (size_t s = 0; s < fo.seg_len.size(); ++s) {
        const int32_t cap = (fo.page_indptr[s + 1] - fo.page_indptr[s]) * 16;
        if (refs[s] == 1 && cap > fo.seg_len[s] && uniform(0, 2)) fo.seg_len[s] = uniform(fo.seg_len[s] + 1, cap);
      }
      f = fo.view();
      CHECK(halo_plan_update_lengths(plan, &f) == HALO_OK);
      halo_plan_t* fresh = nullptr;
      CHECK(halo_plan_create_with_options(&p, &f, &opt, &fresh, &meta, &ws) == HALO_OK);
      if (fresh) {
        CHECK(image_of(plan) == image_of(fresh));
        halo_plan_destroy(fresh);
      }
    }
    // a page opened within the reserve: applied; a private segment grown
    // far past it, or a shared segment that opens a page: refused, plan
    // unchanged
    if (fo.seg_len.empty()) {
      halo_plan_destroy(plan);
      return;
    }
    const int reserve = opt.append_reserve > 0 ? opt.append_reserve : 256;
    auto open_pages = [&](const Forest& from, int s, int32_t len) {
      Forest g = from;
      const int32_t add = (len + 15) / 16 - (g.page_indptr[s + 1] - g.page_indptr[s]);
      g.seg_len[s] = len;
      for (int32_t k = 0; k < add; ++k) {
        g.page_ids.insert(g.page_ids.begin() + g.page_indptr[s + 1], g.pool_pages - 1);
        for (size_t j = s + 1; j < g.page_indptr.size(); ++j) g.page_indptr[j]++;
      }
      return g;
    };
    const int s = uniform(0, (int)fo.seg_len.size() - 1);
    const int32_t len0 = base_len[s];
    if (refs[s] == 1 && len0 > 0 && fo.seg_len[s] >= len0) {
      const int32_t to = std::max(fo.seg_len[s], len0 + uniform(0, reserve));
      Forest g = open_pages(fo, s, to);
      f = g.view();
      CHECK(halo_plan_update_lengths(plan, &f) == HALO_OK);
      fo = g;
    }
    const std::vector<uint8_t> before = image_of(plan);
    Forest grown = open_pages(fo, s, (refs[s] >= 2 ? fo.seg_len[s] : len0) + 1100);
    f = grown.view();
    CHECK(halo_plan_update_lengths(plan, &f) == HALO_ERR_REPLAN);
    CHECK(image_of(plan) == before);
  }
  halo_plan_destroy(plan);
}

// Malformed forests are refused with HALO_ERR_INVALID_ARGUMENT.
void malformed() {
  Forest fo;
  if (!tree_forest(uniform(2, 40), 200, 100, false, fo) || fo.seg_len.empty()) return;
  halo_attn_params_t p{};
  p.num_q_heads = 8;
  p.num_kv_heads = 2;
  p.head_dim = 128;
  p.page_size = 16;
  p.num_pool_pages = fo.pool_pages;
  p.kv_dtype = HALO_BF16;
  p.out_dtype = HALO_BF16;
  p.sm_scale = 0.1f;
  for (int kind = 0; kind < 5; ++kind) {
    Forest bad = fo;
    switch (kind) {
      case 0: bad.seg_len[uniform(0, (int)bad.seg_len.size() - 1)] = -3; break;
      case 1: if (!bad.page_ids.empty()) bad.page_ids[uniform(0, (int)bad.page_ids.size() - 1)] = fo.pool_pages; break;
      case 2: bad.req_ids[uniform(0, (int)bad.req_ids.size() - 1)] = (int32_t)bad.seg_len.size(); break;
      case 3: bad.seg_len[uniform(0, (int)bad.seg_len.size() - 1)] += 17; break;
      default: bad.req_indptr.back() += 1; bad.req_ids.push_back(0); bad.req_indptr[1] = bad.req_indptr[2] + 1; break;
    }
    halo_forest_t f = bad.view();
    halo_plan_t* plan = nullptr;
    size_t meta = 0, ws = 0;
    const halo_status_t st = halo_plan_create(&p, &f, &plan, &meta, &ws);
    if (kind == 1 && fo.page_ids.empty()) continue;
    CHECK(st == HALO_ERR_INVALID_ARGUMENT);
    CHECK(plan == nullptr);
    if (plan) halo_plan_destroy(plan);
  }
}

}  // namespace

int main(int argc, char** argv) {
  const int cases = argc > 1 ? atoi(argv[1]) : 200;
  g_state ^= (uint64_t)(argc > 2 ? atoi(argv[2]) : 1) * 0x100000001B3ull;
  for (int i = 0; i < cases; ++i) {
    one_case(false);
    if (i % 4 == 0) one_case(true);
    if (i % 8 == 0) malformed();
  }
  printf("host_fuzz: %d cases, %d failed checks\n", cases, g_fail);
  return g_fail ? 1 : 0;
}
