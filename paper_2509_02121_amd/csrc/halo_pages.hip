// gfx950 kernels and entry points of the C ABI that move KV tokens between
// the page pools and dense token-major buffers, bit for bit:
// gather_kernel: paged tokens out into a dense buffer (the read-back of the
//   paged KV cache);
// scatter_kernel: new tokens into their pages (a decode append or a prefill
//   chunk), the write path of the cache;
// page_copy_kernel: whole-page copies (the copy of copy-on-write).
// Pool layouts: K pages [H][D/E][16][E] (E elements per 16 bytes), V pages
// [H][D][16] with token slots permuted as below.

#include <hip/hip_runtime.h>

#include <algorithm>
#include <string>

#include "halo_internal.h"

using namespace halo;

namespace {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));

// V pages keep the tokens of a dim row in the slot order 0-3, 8-11, 4-7,
// 12-15 (bits 2 and 3 of the index swapped; the map is its own inverse).
__device__ __forceinline__ int v_token_at_slot(int s) { return (s & 3) | ((s & 4) << 1) | ((s & 8) >> 1); }

// ---------------------------------------------------------------- gather

struct GatherArgs {
  const void* pool;
  const int32_t* page_ids;
  const int32_t* seq_page_indptr;
  const int32_t* seq_len;
  const int64_t* out_token_offset;
  void* out;
  int32_t* error_flag;
  int64_t num_pool_pages;
  int32_t num_seqs;
  int32_t num_kv_heads;
  int32_t head_dim;
  int32_t v_layout;
};

// The last index s < n with indptr[s] <= x, for a nondecreasing indptr with
// indptr[0] <= x (wave-uniform x): the wave compares 64 evenly spaced
// entries at once and keeps the bracket that holds the answer, so up to 4095
// entries take two rounds of loads where a binary search takes twelve.
__device__ __forceinline__ int last_at_or_below(const int32_t* indptr, int n, int64_t x, int lane) {
  int lo = 0, len = n;
  while (len > 64) {
    const int stride = (len + 63) / 64;
    const int off = lane * stride;
    const bool hit = off < len && indptr[lo + off] <= x;
    const uint64_t mask = __ballot(hit);
    const int top = 63 - __clzll(mask);          // lane 0 always hits
    lo += top * stride;
    len = min(stride, len - top * stride);
  }
  const bool hit = lane < len && indptr[lo + lane] <= x;
  const uint64_t mask = __ballot(hit);
  return lo + 63 - __clzll(mask);
}

// The (page slot, head) tiles of all sequences, in order, are cut into equal
// contiguous runs, one per wave, so a few long sequences among many short
// ones spread over the whole grid. A wave finds the sequence of its first
// tile by binary search over seq_page_indptr and walks forward from there.
// Per tile it reads the tile in its stored order with 16-byte loads
// (coalesced), stages it token-major in its own LDS buffer ([16][D + E]
// words, rows 16-byte aligned) and writes the tile's tokens as dense rows,
// 16 bytes per lane. K vectors hold E dims of one token and move whole; V
// vectors hold one dim of E tokens and are split into single words on the
// way into LDS. W is an unsigned word of the element's width, so every bit
// pattern (NaN payloads included) moves unchanged.
template <typename W, int D>
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a) {
  constexpr int E = 16 / (int)sizeof(W);   // elements per 16-byte vector
  constexpr int VPT = D / E;               // vectors per token and head
  constexpr int NV = 16 * VPT / 64;        // vectors per lane for a tile
  constexpr int ROW = D + E;               // staged row, in words (16-byte aligned)
  __shared__ u32x4_t stage[4][16 * ROW / E];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int H = a.num_kv_heads;
  const int64_t row = (int64_t)H * D;      // output elements per token
  const W* pool = static_cast<const W*>(a.pool);
  W* out = static_cast<W*>(a.out);
  W* st = reinterpret_cast<W*>(stage[wave]);

  // page-list slots first .. last-1 are tiled; first need not be 0 (a
  // slice of a larger page list)
  const int first = a.seq_page_indptr[0];
  const int64_t total = ((int64_t)a.seq_page_indptr[a.num_seqs] - first) * H;
  const int64_t waves = (int64_t)gridDim.x * 4;
  const int64_t per = (total + waves - 1) / waves;
  const int64_t w_id = (int64_t)blockIdx.x * 4 + wave;
  const int64_t t_begin = w_id * per;
  const int64_t t_end = min(total, t_begin + per);
  if (t_begin >= t_end) return;
  // indptr[0] <= first + t_begin / H, so the search returns a sequence in
  // [0, num_seqs); the walk below stops at num_seqs - 1 at the latest, since
  // every slot is < indptr[num_seqs]
  int seq = last_at_or_below(a.seq_page_indptr, a.num_seqs, first + t_begin / H, lane);
  int base = a.seq_page_indptr[seq], next = a.seq_page_indptr[seq + 1];
  for (int64_t tl = t_begin; tl < t_end; ++tl) {
    const int slot = first + (int)(tl / H), h = (int)(tl % H);
    while (slot >= next) {             // later sequences (empty ones are passed over)
      ++seq;
      base = next;
      next = a.seq_page_indptr[seq + 1];
    }
    const int len = a.seq_len[seq];
    const int pid = a.page_ids[slot];
    if (len < 0 || next - base != (len + 15) / 16 || pid < 0 || pid >= a.num_pool_pages) {
      if (lane == 0 && a.error_flag) a.error_flag[0] = 1;
      continue;
    }
    const int t0 = (slot - base) * 16;
    const int n = min(16, len - t0);
    const W* src = pool + ((int64_t)pid * H + h) * 16 * D;
    u32x4_t v[NV];
#pragma unroll
    for (int i = 0; i < NV; ++i) v[i] = reinterpret_cast<const u32x4_t*>(src)[lane + 64 * i];
#pragma unroll
    for (int i = 0; i < NV; ++i) {
      const int idx = lane + 64 * i;
      if (!a.v_layout) {             // K: vector idx = (dims j*E.., token t)
        const int j = idx / 16, t = idx % 16;
        *reinterpret_cast<u32x4_t*>(st + t * ROW + j * E) = v[i];
      } else {                       // V: vector idx = (dim c, slots part*E..)
        const int c = idx / (16 / E), part = idx % (16 / E);
        const W* e = reinterpret_cast<const W*>(&v[i]);
#pragma unroll
        for (int q = 0; q < E; ++q) st[v_token_at_slot(part * E + q) * ROW + c] = e[q];
      }
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
    W* dst = out + (a.out_token_offset[seq] + t0) * row + (int64_t)h * D;
    for (int idx = lane; idx < n * VPT; idx += 64) {
      const int tok = idx / VPT, j = idx % VPT;
      *reinterpret_cast<u32x4_t*>(dst + tok * row + j * E) =
          *reinterpret_cast<const u32x4_t*>(st + tok * ROW + j * E);
    }
    __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
    __builtin_amdgcn_wave_barrier();
    __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
  }
}

// ---------------------------------------------------------------- write path

// Up to two (pool, input) pairs written by one launch, pair blockIdx.z: the
// K and V pools of one append share the page lists and the launch.
struct ScatterArgs {
  void* pool[2];
  const void* in[2];
  int32_t v_layout[2];
  const int32_t* page_ids;
  const int32_t* seq_page_indptr;
  const int32_t* seq_start;
  const int32_t* seq_count;
  const int64_t* in_token_offset;
  int32_t* error_flag;
  int64_t num_pool_pages;
  int32_t num_seqs;
  int32_t num_kv_heads;
  int32_t head_dim;
};

// The inverse of the gather: tokens start .. start + count - 1 of each
// sequence are written from the dense input into their (page, head) tiles.
// Blocks (x, y) take sequence x (grid-stride) and its touched tiles; each of
// the block's four waves owns one tile at a time (tiles y*4 + wave, stepping
// by gridDim.y*4), so only the pages the range touches are visited and a
// decode append costs one tile per head whatever the sequence's length.
// A full tile (16 touched tokens) is read with 16-byte loads, transposed in
// the wave's own LDS buffer and written back as the tile's 4 KB (bf16,
// d 128) in stored order, 16 bytes per lane. A partly touched tile (a
// decode append, the ends of a chunk) is written straight from the input:
// 16-byte vectors for K, whose vector (dim group, token) holds one token;
// single elements for V, whose slots interleave tokens. Untouched slots are
// never written. Words of the element's width keep every bit pattern.
template <typename W, int D>
__global__ __launch_bounds__(256) void scatter_kernel(ScatterArgs a) {
  constexpr int E = 16 / (int)sizeof(W);   // elements per 16-byte vector
  constexpr int VPT = D / E;               // vectors per token and head
  constexpr int TV = 16 * VPT;             // vectors per tile
  constexpr int NV = TV / 64;              // vectors per lane for a full tile
  constexpr int KROW = 17;                 // K staging: vector (j, t) at j * KROW + t
  constexpr int KBUF = VPT * KROW;         // 16-byte vectors
  // V staging: the tile in stored order, [D][16] elements, row c held at row
  // c ^ ((c / E) & RMASK): the rows written by one instruction (dims
  // j*E + q of four dim groups j) then fall in different 32-byte bank groups.
  constexpr int RMASK = 128 / (16 * (int)sizeof(W)) - 1;
  constexpr int VBUF = D * 16 / E;
  constexpr int BUF = KBUF > VBUF ? KBUF : VBUF;
  __shared__ u32x4_t stage[4][BUF];
  const int wave = threadIdx.x >> 6, lane = threadIdx.x & 63;
  const int H = a.num_kv_heads;
  const int64_t row = (int64_t)H * D;      // input elements per token
  W* pool = static_cast<W*>(a.pool[blockIdx.z]);
  const W* in = static_cast<const W*>(a.in[blockIdx.z]);
  const bool v_layout = a.v_layout[blockIdx.z] != 0;
  u32x4_t* kst = stage[wave];
  W* vst = reinterpret_cast<W*>(stage[wave]);
  for (int seq = blockIdx.x; seq < a.num_seqs; seq += gridDim.x) {
    const int start = a.seq_start[seq], count = a.seq_count[seq];
    if (count <= 0) continue;
    const int base = a.seq_page_indptr[seq];
    const int npages = a.seq_page_indptr[seq + 1] - base;
    if (start < 0 || (int64_t)start + count > (int64_t)npages * 16) {
      if (blockIdx.y == 0 && blockIdx.z == 0 && threadIdx.x == 0 && a.error_flag) a.error_flag[0] = 1;
      continue;
    }
    const int first = start / 16, last = (start + count - 1) / 16;
    const int ntiles = (last - first + 1) * H;
    for (int k = blockIdx.y * 4 + wave; k < ntiles; k += gridDim.y * 4) {
      const int pslot = first + k / H, h = k % H;
      const int pid = a.page_ids[base + pslot];
      if (pid < 0 || pid >= a.num_pool_pages) {
        if (lane == 0 && a.error_flag) a.error_flag[0] = 1;
        continue;
      }
      const int t0 = pslot * 16;
      const int lo_t = max(start, t0), hi_t = min(start + count, t0 + 16);   // touched tokens
      const int n = hi_t - lo_t;
      const W* src = in + (a.in_token_offset[seq] + (lo_t - start)) * row + (int64_t)h * D;
      W* dst = pool + ((int64_t)pid * H + h) * 16 * D;
      if (n == 16 && !v_layout) {
        u32x4_t v[NV];
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          const int idx = lane + 64 * i, tok = idx / VPT, j = idx % VPT;
          v[i] = *reinterpret_cast<const u32x4_t*>(src + tok * row + j * E);
        }
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          const int idx = lane + 64 * i, tok = idx / VPT, j = idx % VPT;
          kst[j * KROW + tok] = v[i];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int i = 0; i < NV; ++i) {    // K: [D/E][16][E], vector idx = (j, t)
          const int idx = lane + 64 * i;
          *reinterpret_cast<u32x4_t*>(dst + idx * E) = kst[(idx / 16) * KROW + idx % 16];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      } else if (n == 16) {
        // Token fastest across lanes: one instruction's 16 lanes of a dim
        // group fill the 16 slots of one staged row.
        u32x4_t v[NV];
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          const int idx = lane + 64 * i, tok = idx % 16, j = idx / 16;
          v[i] = *reinterpret_cast<const u32x4_t*>(src + tok * row + j * E);
        }
#pragma unroll
        for (int i = 0; i < NV; ++i) {
          const int idx = lane + 64 * i, tok = idx % 16, j = idx / 16;
          const int slot = v_token_at_slot(tok);   // the permutation is its own inverse
          const W* e = reinterpret_cast<const W*>(&v[i]);
#pragma unroll
          for (int q = 0; q < E; ++q) vst[((j * E + q) ^ (j & RMASK)) * 16 + slot] = e[q];
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
#pragma unroll
        for (int i = 0; i < NV; ++i) {    // V: [D][16], vector idx = (dim c, slot group)
          const int idx = lane + 64 * i, c = idx / (16 / E), part = idx % (16 / E);
          *reinterpret_cast<u32x4_t*>(dst + idx * E) =
              *reinterpret_cast<const u32x4_t*>(vst + (c ^ ((c / E) & RMASK)) * 16 + part * E);
        }
        __builtin_amdgcn_fence(__ATOMIC_RELEASE, "wavefront");
        __builtin_amdgcn_wave_barrier();
        __builtin_amdgcn_fence(__ATOMIC_ACQUIRE, "wavefront");
      } else if (!v_layout) {
        for (int idx = lane; idx < n * VPT; idx += 64) {
          const int tok = idx / VPT, j = idx % VPT, t = lo_t - t0 + tok;
          *reinterpret_cast<u32x4_t*>(dst + (j * 16 + t) * E) =
              *reinterpret_cast<const u32x4_t*>(src + tok * row + j * E);
        }
      } else {
        for (int idx = lane; idx < n * D; idx += 64) {
          const int tok = idx / D, c = idx % D, t = lo_t - t0 + tok;
          dst[c * 16 + v_token_at_slot(t)] = src[tok * row + c];
        }
      }
    }
  }
}

struct PageCopyArgs {
  void* pool;
  const int32_t* src_pages;
  const int32_t* dst_pages;
  int32_t* error_flag;
  int64_t num_pool_pages;
  int64_t page_vecs;   // 16-byte units of one page (all heads)
  int32_t num_pages;
};

// Copy whole pages (every head) of one pool, 16 bytes per lane, grid-stride
// over (page, unit). Pages with an id out of range are skipped and flagged.
__global__ __launch_bounds__(256) void page_copy_kernel(PageCopyArgs a) {
  const int64_t total = (int64_t)a.num_pages * a.page_vecs;
  u32x4_t* pool = static_cast<u32x4_t*>(a.pool);
  for (int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; i < total; i += (int64_t)gridDim.x * blockDim.x) {
    const int64_t k = i / a.page_vecs, u = i - k * a.page_vecs;
    const int src = a.src_pages[k], dst = a.dst_pages[k];
    if (src < 0 || src >= a.num_pool_pages || dst < 0 || dst >= a.num_pool_pages) {
      if (u == 0 && a.error_flag) a.error_flag[0] = 1;
      continue;
    }
    pool[dst * a.page_vecs + u] = pool[src * a.page_vecs + u];
  }
}

// ---------------------------------------------------------------- host side

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

halo_status_t hip_check(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(HALO_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return HALO_OK;
}

}  // namespace

extern "C" halo_status_t halo_kv_page_gather(const void* pool, const halo_attn_params_t* params,
                                             halo_pool_kind_t pool_kind, const int32_t* page_ids,
                                             const int32_t* seq_page_indptr, const int32_t* seq_len,
                                             const int64_t* out_token_offset, int32_t num_seqs, void* out,
                                             int32_t* error_flag, void* stream) {
  clear_error();
  if (!params) return fail(HALO_ERR_INVALID_ARGUMENT, "params must not be NULL");
  if (num_seqs < 0) return fail(HALO_ERR_INVALID_ARGUMENT, "num_seqs must be >= 0");
  if (num_seqs == 0) return HALO_OK;
  if (!pool || !page_ids || !seq_page_indptr || !seq_len || !out_token_offset || !out)
    return fail(HALO_ERR_INVALID_ARGUMENT, "pool, page_ids, seq_page_indptr, seq_len, out_token_offset, out "
                                           "must not be NULL");
  if (params->head_dim != 64 && params->head_dim != 128)
    return fail(HALO_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (params->page_size != 16) return fail(HALO_ERR_UNSUPPORTED, "page_size must be 16");
  if (params->num_kv_heads < 1) return fail(HALO_ERR_INVALID_ARGUMENT, "num_kv_heads must be >= 1");
  if (pool_kind != HALO_POOL_K && pool_kind != HALO_POOL_V)
    return fail(HALO_ERR_INVALID_ARGUMENT, "pool_kind must be HALO_POOL_K or HALO_POOL_V");
  GatherArgs g{pool, page_ids, seq_page_indptr, seq_len, out_token_offset, out, error_flag,
               params->num_pool_pages, num_seqs, params->num_kv_heads, params->head_dim,
               pool_kind == HALO_POOL_V ? 1 : 0};
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  if (!aligned16(pool) || !aligned16(out))
    return fail(HALO_ERR_INVALID_ARGUMENT, "pool and out must be 16-byte aligned");
  // 2048 workgroups of four waves; each wave takes an equal run of tiles.
  const dim3 grid(2048);
  const bool d128 = params->head_dim == 128;
  if (params->kv_dtype == HALO_BF16) {
    if (d128) hipLaunchKernelGGL((gather_kernel<uint16_t, 128>), grid, dim3(256), 0, st, g);
    else hipLaunchKernelGGL((gather_kernel<uint16_t, 64>), grid, dim3(256), 0, st, g);
  } else if (params->kv_dtype == HALO_F32) {
    if (d128) hipLaunchKernelGGL((gather_kernel<uint32_t, 128>), grid, dim3(256), 0, st, g);
    else hipLaunchKernelGGL((gather_kernel<uint32_t, 64>), grid, dim3(256), 0, st, g);
  } else {
    return fail(HALO_ERR_UNSUPPORTED, "kv_dtype must be HALO_F32 or HALO_BF16");
  }
  return hip_check("gather launch");
}

namespace {

// Shared checks and launch of the scatter entry points (n_pairs = 1 or 2).
halo_status_t launch_scatter(const halo_attn_params_t* params, ScatterArgs g, int n_pairs, void* stream) {
  if (params->head_dim != 64 && params->head_dim != 128)
    return fail(HALO_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (params->page_size != 16) return fail(HALO_ERR_UNSUPPORTED, "page_size must be 16");
  if (params->num_kv_heads < 1) return fail(HALO_ERR_INVALID_ARGUMENT, "num_kv_heads must be >= 1");
  if (params->kv_dtype != HALO_BF16 && params->kv_dtype != HALO_F32)
    return fail(HALO_ERR_UNSUPPORTED, "kv_dtype must be HALO_F32 or HALO_BF16");
  for (int z = 0; z < n_pairs; ++z)
    if (!aligned16(g.pool[z]) || !aligned16(g.in[z]))
      return fail(HALO_ERR_INVALID_ARGUMENT, "pools and inputs must be 16-byte aligned");
  g.num_pool_pages = params->num_pool_pages;
  g.num_kv_heads = params->num_kv_heads;
  g.head_dim = params->head_dim;
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  // One x-block per sequence (grid-stride past 65536), enough y-blocks per
  // sequence that a call fills the chip with about 2048 workgroups.
  const int bx = std::min(g.num_seqs, 65536);
  const dim3 grid(bx, std::min(std::max(2048 / (bx * n_pairs), 1), 2048), n_pairs);
  const bool d128 = params->head_dim == 128;
  if (params->kv_dtype == HALO_BF16) {
    if (d128) hipLaunchKernelGGL((scatter_kernel<uint16_t, 128>), grid, dim3(256), 0, st, g);
    else hipLaunchKernelGGL((scatter_kernel<uint16_t, 64>), grid, dim3(256), 0, st, g);
  } else {
    if (d128) hipLaunchKernelGGL((scatter_kernel<uint32_t, 128>), grid, dim3(256), 0, st, g);
    else hipLaunchKernelGGL((scatter_kernel<uint32_t, 64>), grid, dim3(256), 0, st, g);
  }
  return hip_check("scatter launch");
}

}  // namespace

extern "C" halo_status_t halo_kv_page_scatter(void* pool, const halo_attn_params_t* params,
                                              halo_pool_kind_t pool_kind, const int32_t* page_ids,
                                              const int32_t* seq_page_indptr, const int32_t* seq_start,
                                              const int32_t* seq_count, const int64_t* in_token_offset,
                                              int32_t num_seqs, const void* in, int32_t* error_flag,
                                              void* stream) {
  clear_error();
  if (!params) return fail(HALO_ERR_INVALID_ARGUMENT, "params must not be NULL");
  if (num_seqs < 0) return fail(HALO_ERR_INVALID_ARGUMENT, "num_seqs must be >= 0");
  if (num_seqs == 0) return HALO_OK;
  if (!pool || !page_ids || !seq_page_indptr || !seq_start || !seq_count || !in_token_offset || !in)
    return fail(HALO_ERR_INVALID_ARGUMENT, "pool, page_ids, seq_page_indptr, seq_start, seq_count, "
                                           "in_token_offset, in must not be NULL");
  if (pool_kind != HALO_POOL_K && pool_kind != HALO_POOL_V)
    return fail(HALO_ERR_INVALID_ARGUMENT, "pool_kind must be HALO_POOL_K or HALO_POOL_V");
  ScatterArgs g{};
  g.pool[0] = pool;
  g.in[0] = in;
  g.v_layout[0] = pool_kind == HALO_POOL_V ? 1 : 0;
  g.page_ids = page_ids;
  g.seq_page_indptr = seq_page_indptr;
  g.seq_start = seq_start;
  g.seq_count = seq_count;
  g.in_token_offset = in_token_offset;
  g.error_flag = error_flag;
  g.num_seqs = num_seqs;
  return launch_scatter(params, g, 1, stream);
}

extern "C" halo_status_t halo_kv_page_scatter_kv(void* k_pool, void* v_pool, const halo_attn_params_t* params,
                                                 const int32_t* page_ids, const int32_t* seq_page_indptr,
                                                 const int32_t* seq_start, const int32_t* seq_count,
                                                 const int64_t* in_token_offset, int32_t num_seqs,
                                                 const void* k_in, const void* v_in, int32_t* error_flag,
                                                 void* stream) {
  clear_error();
  if (!params) return fail(HALO_ERR_INVALID_ARGUMENT, "params must not be NULL");
  if (num_seqs < 0) return fail(HALO_ERR_INVALID_ARGUMENT, "num_seqs must be >= 0");
  if (num_seqs == 0) return HALO_OK;
  if (!k_pool || !v_pool || !page_ids || !seq_page_indptr || !seq_start || !seq_count || !in_token_offset ||
      !k_in || !v_in)
    return fail(HALO_ERR_INVALID_ARGUMENT, "k_pool, v_pool, page_ids, seq_page_indptr, seq_start, seq_count, "
                                           "in_token_offset, k_in, v_in must not be NULL");
  ScatterArgs g{};
  g.pool[0] = k_pool;
  g.pool[1] = v_pool;
  g.in[0] = k_in;
  g.in[1] = v_in;
  g.v_layout[0] = 0;
  g.v_layout[1] = 1;
  g.page_ids = page_ids;
  g.seq_page_indptr = seq_page_indptr;
  g.seq_start = seq_start;
  g.seq_count = seq_count;
  g.in_token_offset = in_token_offset;
  g.error_flag = error_flag;
  g.num_seqs = num_seqs;
  return launch_scatter(params, g, 2, stream);
}

extern "C" halo_status_t halo_kv_page_copy(void* pool, const halo_attn_params_t* params,
                                           const int32_t* src_pages, const int32_t* dst_pages,
                                           int32_t num_pages, int32_t* error_flag, void* stream) {
  clear_error();
  if (!params) return fail(HALO_ERR_INVALID_ARGUMENT, "params must not be NULL");
  if (num_pages < 0) return fail(HALO_ERR_INVALID_ARGUMENT, "num_pages must be >= 0");
  if (num_pages == 0) return HALO_OK;
  if (!pool || !src_pages || !dst_pages)
    return fail(HALO_ERR_INVALID_ARGUMENT, "pool, src_pages, dst_pages must not be NULL");
  if (params->head_dim != 64 && params->head_dim != 128)
    return fail(HALO_ERR_UNSUPPORTED, "head_dim must be 64 or 128");
  if (params->page_size != 16) return fail(HALO_ERR_UNSUPPORTED, "page_size must be 16");
  if (params->num_kv_heads < 1) return fail(HALO_ERR_INVALID_ARGUMENT, "num_kv_heads must be >= 1");
  int elt;
  if (params->kv_dtype == HALO_BF16) elt = 2;
  else if (params->kv_dtype == HALO_F32) elt = 4;
  else return fail(HALO_ERR_UNSUPPORTED, "kv_dtype must be HALO_F32 or HALO_BF16");
  if (!aligned16(pool)) return fail(HALO_ERR_INVALID_ARGUMENT, "pool must be 16-byte aligned");
  const int64_t page_bytes = (int64_t)params->num_kv_heads * 16 * params->head_dim * elt;
  PageCopyArgs g{pool, src_pages, dst_pages, error_flag, params->num_pool_pages, page_bytes / 16, num_pages};
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();
  const int64_t want = ((int64_t)num_pages * g.page_vecs + 255) / 256;
  const int blocks = (int)std::min<int64_t>(std::max<int64_t>(want, 1), 4096);
  hipLaunchKernelGGL(page_copy_kernel, dim3(blocks), dim3(256), 0, st, g);
  return hip_check("page copy launch");
}
