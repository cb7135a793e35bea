// Prefix forest construction from token ids (host C++).
//
// A batch of prompts that share prefixes (§2: intra-batch prefix sharing
// computes a shared prefix once and reuses its KV cache; §1 and §3: Halo
// detects recurring prompts) becomes the forest the attention calls take:
// a trie over page-sized chunks of the prompts (the radix tree of
// RadixAttention, §7, at page granularity so that every shared boundary is
// page-aligned, as the paged cache of PagedAttention needs), compressed into
// segments. A chunk node is shared by exactly the requests whose prompts
// agree on every token up to and including it, with the same chunk length;
// a segment is a maximal chain of chunk nodes passed by the same requests.

#include <stdint.h>
#include <string.h>

#include <unordered_map>
#include <vector>

#include "halo_internal.h"

struct halo_prefix_tree {
  int32_t page_size = 0;
  std::vector<int32_t> seg_len, seg_parent, seg_refcount, seg_src_request, seg_src_offset;
  std::vector<int32_t> req_seg_indptr, req_seg_ids;
  int64_t num_pages = 0;
  int64_t prompt_tokens = 0;
  int64_t distinct_tokens = 0;
};

namespace {

using halo::fail;

struct Node {
  int32_t parent;
  int32_t src_req;      // a request whose prompt holds this chunk
  int32_t src_off;      // token offset of the chunk in that prompt
  int32_t len;          // chunk length: page_size, or less for a prompt's last chunk
  int32_t count = 0;    // requests whose prompts pass through this chunk
  int32_t first_child = -1, last_child = -1, next_sibling = -1;   // creation order
  int32_t hash_next = -1;   // next node with the same bucket key
  int32_t seg = -1;
};

// A 64-bit key of (parent node, chunk length, chunk tokens): each 32-bit
// word is folded in with a multiply and an xor-shift (the finaliser of
// splitmix64). Equal keys are confirmed by comparing the tokens.
inline uint64_t fold(uint64_t h, uint32_t v) {
  h = (h ^ v) * 0x9e3779b97f4a7c15ull;
  return h ^ (h >> 29);
}

uint64_t chunk_key(int32_t parent, const int32_t* t, int32_t n) {
  uint64_t h = fold(fold(0x243f6a8885a308d3ull, static_cast<uint32_t>(parent)), static_cast<uint32_t>(n));
  for (int32_t i = 0; i < n; ++i) h = fold(h, static_cast<uint32_t>(t[i]));
  h ^= h >> 31;
  h *= 0xbf58476d1ce4e5b9ull;
  return h ^ (h >> 27);
}

}  // namespace

extern "C" halo_status_t halo_prefix_tree_build(const int32_t* prompt_indptr, const int32_t* tokens,
                                                int32_t num_requests, int32_t page_size,
                                                halo_prefix_tree_t** tree, halo_prefix_tree_info_t* info) {
  halo::clear_error();
  if (!tree) return fail(HALO_ERR_INVALID_ARGUMENT, "tree must not be NULL");
  *tree = nullptr;
  if (num_requests < 0) return fail(HALO_ERR_INVALID_ARGUMENT, "num_requests must be >= 0");
  if (page_size < 1) return fail(HALO_ERR_INVALID_ARGUMENT, "page_size must be >= 1");
  if (num_requests > 0 && !prompt_indptr) return fail(HALO_ERR_INVALID_ARGUMENT, "prompt_indptr must not be NULL");
  if (num_requests > 0) {
    if (prompt_indptr[0] != 0) return fail(HALO_ERR_INVALID_ARGUMENT, "prompt_indptr[0] must be 0");
    for (int32_t r = 0; r < num_requests; ++r)
      if (prompt_indptr[r + 1] < prompt_indptr[r])
        return fail(HALO_ERR_INVALID_ARGUMENT, "prompt_indptr must be nondecreasing");
    if (prompt_indptr[num_requests] > 0 && !tokens)
      return fail(HALO_ERR_INVALID_ARGUMENT, "tokens must not be NULL");
  }

  auto* t = new halo_prefix_tree();
  t->page_size = page_size;
  const int32_t B = page_size;
  std::vector<Node> nodes;
  nodes.push_back(Node{-1, -1, 0, 0});
  nodes[0].count = num_requests;
  const int64_t total = num_requests > 0 ? prompt_indptr[num_requests] : 0;
  nodes.reserve(static_cast<size_t>(total / B + num_requests + 1));
  std::unordered_map<uint64_t, int32_t> bucket;   // key -> first node with that key
  bucket.reserve(static_cast<size_t>(total / B + num_requests + 1));
  std::vector<int32_t> leaf(num_requests, 0);
  for (int32_t r = 0; r < num_requests; ++r) {
    const int32_t* p = tokens + prompt_indptr[r];
    const int32_t len = prompt_indptr[r + 1] - prompt_indptr[r];
    t->prompt_tokens += len;
    int32_t cur = 0;
    for (int32_t off = 0; off < len; off += B) {
      const int32_t n = len - off < B ? len - off : B;
      const uint64_t key = chunk_key(cur, p + off, n);
      auto it = bucket.find(key);
      int32_t hit = -1;
      for (int32_t c = it == bucket.end() ? -1 : it->second; c >= 0; c = nodes[c].hash_next) {
        const Node& nd = nodes[c];
        if (nd.parent == cur && nd.len == n &&
            memcmp(tokens + prompt_indptr[nd.src_req] + nd.src_off, p + off, sizeof(int32_t) * n) == 0) {
          hit = c;
          break;
        }
      }
      if (hit < 0) {
        hit = static_cast<int32_t>(nodes.size());
        Node nd{cur, r, off, n};
        nd.hash_next = it == bucket.end() ? -1 : it->second;
        nodes.push_back(nd);
        bucket[key] = hit;
        if (nodes[cur].last_child < 0) nodes[cur].first_child = hit;
        else nodes[nodes[cur].last_child].next_sibling = hit;
        nodes[cur].last_child = hit;
      }
      nodes[hit].count += 1;
      cur = hit;
    }
    leaf[r] = cur;
  }

  // Segments in depth-first preorder, children in creation order. A node
  // starts a segment unless its parent is passed by the same requests (same
  // count; the parent then has this node as its only child).
  std::vector<int32_t> stack, kids;
  auto push_children = [&](int32_t v) {   // reversed, so they pop in creation order
    kids.clear();
    for (int32_t c = nodes[v].first_child; c >= 0; c = nodes[c].next_sibling) kids.push_back(c);
    for (auto it = kids.rbegin(); it != kids.rend(); ++it) stack.push_back(*it);
  };
  push_children(0);
  while (!stack.empty()) {
    const int32_t v = stack.back();
    stack.pop_back();
    Node& nd = nodes[v];
    const int32_t par = nd.parent;
    if (par == 0 || nodes[par].count != nd.count) {
      nd.seg = static_cast<int32_t>(t->seg_len.size());
      t->seg_len.push_back(nd.len);
      t->seg_parent.push_back(par == 0 ? -1 : nodes[par].seg);
      t->seg_refcount.push_back(nd.count);
      t->seg_src_request.push_back(nd.src_req);
      t->seg_src_offset.push_back(nd.src_off);
    } else {
      nd.seg = nodes[par].seg;
      t->seg_len[nd.seg] += nd.len;
    }
    push_children(v);
  }

  t->req_seg_indptr.assign(num_requests + 1, 0);
  std::vector<int32_t> path;
  for (int32_t r = 0; r < num_requests; ++r) {
    path.clear();
    for (int32_t v = leaf[r]; v > 0; v = nodes[v].parent)
      if (path.empty() || path.back() != nodes[v].seg) path.push_back(nodes[v].seg);
    for (auto it = path.rbegin(); it != path.rend(); ++it) t->req_seg_ids.push_back(*it);
    t->req_seg_indptr[r + 1] = static_cast<int32_t>(t->req_seg_ids.size());
  }
  for (int32_t len : t->seg_len) {
    t->num_pages += (len + B - 1) / B;
    t->distinct_tokens += len;
  }
  *tree = t;
  if (info) {
    info->num_segments = static_cast<int32_t>(t->seg_len.size());
    info->num_path_entries = static_cast<int32_t>(t->req_seg_ids.size());
    info->num_pages = t->num_pages;
    info->prompt_tokens = t->prompt_tokens;
    info->distinct_tokens = t->distinct_tokens;
  }
  return HALO_OK;
}

extern "C" halo_status_t halo_prefix_tree_get(const halo_prefix_tree_t* tree, int32_t* seg_len,
                                              int32_t* seg_parent, int32_t* seg_refcount,
                                              int32_t* seg_src_request, int32_t* seg_src_offset,
                                              int32_t* req_seg_indptr, int32_t* req_seg_ids) {
  halo::clear_error();
  if (!tree) return fail(HALO_ERR_INVALID_ARGUMENT, "tree must not be NULL");
  auto put = [](int32_t* dst, const std::vector<int32_t>& v) {
    if (dst && !v.empty()) memcpy(dst, v.data(), sizeof(int32_t) * v.size());
  };
  put(seg_len, tree->seg_len);
  put(seg_parent, tree->seg_parent);
  put(seg_refcount, tree->seg_refcount);
  put(seg_src_request, tree->seg_src_request);
  put(seg_src_offset, tree->seg_src_offset);
  put(req_seg_indptr, tree->req_seg_indptr);
  put(req_seg_ids, tree->req_seg_ids);
  return HALO_OK;
}

extern "C" void halo_prefix_tree_destroy(halo_prefix_tree_t* tree) { delete tree; }
