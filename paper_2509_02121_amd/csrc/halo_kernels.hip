// gfx950 kernels and the run-time entry points of the C ABI.
//
// attn_items_kernel: one wavefront per work item (<= 16 query rows against a
//   list of key spans). Per step of 32 keys (two 16-token pages):
//     S^T = K Q^T  on v_mfma_f32_16x16x32_bf16 (one 16-key tile per page,
//                  4 MFMAs per tile at d=128)
//     online softmax in the log2 domain (row max / sum over the 4 lane groups)
//     O^T += V^T P^T on the same MFMA (8 MFMAs at d=128)
//   K pages are stored in 16-byte units ([d/E][16][E]) and V pages dim-major
//   ([d][16]), so every MFMA A operand is a direct load from one page: 1 KB
//   contiguous per wave for K, 512 B for V. The QK output layout is already
//   the PV B operand (no lane exchange).
// merge_kernel: exact log-sum-exp combination of partial results over
//   disjoint key ranges (the merge that makes shared == unshared), in its own
//   launch so the kernel boundary makes every partial visible (an in-kernel
//   last-arriver merge needs agent-scope release/acquire, i.e. L2
//   write-back and invalidate, which measured 4x slower on this path).
// gather_kernel: bit copy of paged tokens into a dense token-major buffer.

#include <hip/hip_runtime.h>

#include <cmath>
#include <string>

#include "halo_internal.h"

using namespace halo;

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef unsigned int u32x2_t __attribute__((ext_vector_type(2)));

constexpr float kNegInf = -__builtin_huge_valf();
constexpr float kLn2 = 0.69314718055994530942f;
constexpr float kLog2e = 1.44269504088896340736f;

// ---------------------------------------------------------------- fragments
// A fragment is the 8 K-slot values one lane feeds to a 16x16x32 MFMA.

template <typename T> struct FragOf;
template <> struct FragOf<__bf16> { using type = bf16x8_t; };
template <> struct FragOf<float> { using type = f32x8_t; };

__device__ __forceinline__ bf16x8_t load8(const __bf16* p) {
  return __builtin_bit_cast(bf16x8_t, *reinterpret_cast<const u32x4_t*>(p));
}
__device__ __forceinline__ f32x8_t load8(const float* p) {
  return *reinterpret_cast<const f32x8_t*>(p);
}

template <typename F> __device__ __forceinline__ F zero_frag() { return F{}; }

// 16-byte global load; NT marks data read once (non-temporal: streamed past
// the caches, measured 7.2 TB/s vs 5.8 TB/s for plain loads on a read stream).
template <bool NT>
__device__ __forceinline__ u32x4_t ld16(const void* p) {
  if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  else return *reinterpret_cast<const u32x4_t*>(p);
}
template <bool NT>
__device__ __forceinline__ u32x2_t ld8(const void* p) {
  if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x2_t*>(p));
  else return *reinterpret_cast<const u32x2_t*>(p);
}

// K fragment: dims d0..d0+7 of key t in a K tile stored as [D/E][16][E]
// (E elements per 16-byte unit).
template <bool NT>
__device__ __forceinline__ bf16x8_t load_k8(const __bf16* tile, int t, int d0) {
  return __builtin_bit_cast(bf16x8_t, ld16<NT>(tile + ((d0 >> 3) * 16 + t) * 8));
}
template <bool NT>
__device__ __forceinline__ f32x8_t load_k8(const float* tile, int t, int d0) {
  const u32x4_t lo = ld16<NT>(tile + ((d0 >> 2) * 16 + t) * 4);
  const u32x4_t hi = ld16<NT>(tile + (((d0 >> 2) + 1) * 16 + t) * 4);
  return __builtin_bit_cast(f32x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// V fragment: keys 4u..4u+3 of dim d from page tiles p0 (slots 0..3) and p1
// (slots 4..7), V tiles stored dim-major as [D][16].
template <bool NT>
__device__ __forceinline__ bf16x8_t load_v8(const __bf16* p0, const __bf16* p1, int off) {
  const u32x2_t a = ld8<NT>(p0 + off);
  const u32x2_t b = ld8<NT>(p1 + off);
  return __builtin_bit_cast(bf16x8_t, u32x4_t{a.x, a.y, b.x, b.y});
}
template <bool NT>
__device__ __forceinline__ f32x8_t load_v8(const float* p0, const float* p1, int off) {
  const u32x4_t lo = ld16<NT>(p0 + off);
  const u32x4_t hi = ld16<NT>(p1 + off);
  return __builtin_bit_cast(f32x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// D(16x16) += A(16x32) B(32x16). bf16: one MFMA. fp32: the same 32-deep
// contraction as eight 16x16x4 MFMAs, slot j of every lane in the j-th one,
// so both element types share one register layout.
__device__ __forceinline__ f32x4_t mma(bf16x8_t a, bf16x8_t b, f32x4_t c) {
  return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
}
__device__ __forceinline__ f32x4_t mma(f32x8_t a, f32x8_t b, f32x4_t c) {
#pragma unroll
  for (int j = 0; j < 8; ++j) c = __builtin_amdgcn_mfma_f32_16x16x4f32(a[j], b[j], c, 0, 0, 0);
  return c;
}

__device__ __forceinline__ bf16x8_t to_frag(const float (&p)[8], bf16x8_t*) {
  bf16x8_t r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = (__bf16)p[j];
  return r;
}
__device__ __forceinline__ f32x8_t to_frag(const float (&p)[8], f32x8_t*) {
  f32x8_t r;
#pragma unroll
  for (int j = 0; j < 8; ++j) r[j] = p[j];
  return r;
}

__device__ __forceinline__ void store4(float* dst, f32x4_t v) {
  *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
}
__device__ __forceinline__ void store4(__bf16* dst, f32x4_t v) {
  typedef __bf16 bf16x4_t __attribute__((ext_vector_type(4)));
  bf16x4_t r;
  r[0] = (__bf16)v[0];
  r[1] = (__bf16)v[1];
  r[2] = (__bf16)v[2];
  r[3] = (__bf16)v[3];
  *reinterpret_cast<uint2*>(dst) = __builtin_bit_cast(uint2, r);
}

// ---------------------------------------------------------------- attention

struct AttnArgs {
  const void* q;
  const void* k_pool;
  const void* v_pool;
  void* o;
  float* lse;
  float* part_o;
  float* part_lse;
  const int32_t* seg_page_off;
  const int32_t* seg_len;
  const int32_t* page_ids;
  const Item* items;        // narrow items (one wavefront each)
  const Item* wide_items;   // wide items (one 4-wave workgroup each)
  const Span* spans;
  const Row* rows;
  int32_t n_items;
  int32_t n_wide;
  int32_t wide_blocks;     // grid blocks of the wide role (n_wide padded, see xcd_remap)
  int32_t narrow_blocks;   // grid blocks of the narrow role (4 items each, padded)
  int32_t wide_group;      // consecutive wide items kept on one XCD
  int32_t narrow_group;    // consecutive narrow blocks kept on one XCD
  int32_t num_kv_heads;
  float scale_log2;   // sm_scale * log2(e)
};

// Workgroups are dealt to the 8 XCDs round-robin by block index, and each
// XCD has its own L2. Blocks that read the same pages (the row groups of one
// shared chunk) are made consecutive on one XCD: physical block p of a
// segment (p % 8 = XCD, p / 8 = its turn there) runs logical block
//   ((p / 8) / S * 8 + p % 8) * S + (p / 8) % S,
// i.e. groups of S logical blocks go round-robin to XCDs, in order. The
// segment length is a multiple of 8 S, so this is a permutation.
__device__ __forceinline__ int xcd_remap(int p, int S) {
  const int x = p & 7, j = p >> 3;
  return ((j / S) * 8 + x) * S + j % S;
}

// A span's keys and its page ids, one page per lane (a span has at most 64
// pages), so a step finds its page ids with two lane reads instead of
// dependent memory loads.
struct SpanState {
  int kb, ke, causal;
  int vpid;      // lane l: page id of the span's l-th page
  bool valid;
};

// Position of one 32-key step.
struct StepPos {
  int t0;          // first key of the step (segment-local, multiple of 32)
  int key_end;     // end of its span
  int causal;
  int pid0, pid1;  // page ids of the step's two pages (pid1 == pid0 if absent)
  bool has1;
  bool valid;
};

// Field-wise choice between two step positions (a conditional on the
// structs themselves would select their addresses and keep them in memory).
__device__ __forceinline__ StepPos pick(bool c, const StepPos& x, const StepPos& y) {
  StepPos r;
  r.t0 = c ? x.t0 : y.t0;
  r.key_end = c ? x.key_end : y.key_end;
  r.causal = c ? x.causal : y.causal;
  r.pid0 = c ? x.pid0 : y.pid0;
  r.pid1 = c ? x.pid1 : y.pid1;
  r.has1 = c ? x.has1 : y.has1;
  r.valid = c ? x.valid : y.valid;
  return r;
}

// Operand registers of one step: K for the two 16-key QK tiles, V^T for
// the NB output blocks.
template <typename F, int NS, int NB>
struct StepRegs {
  F k[2][NS];
  F v[NB];
};

// One work item on one wavefront. Lane l: col = l % 16, grp = l / 16.
//  * QK, one MFMA tile X per page of the 32-key step: A = K rows (A row =
//    key col of page X), B = Q^T (B column = query row col); the result lane
//    (col, grp) holds S[row col][key 16X + 4grp + i] in register i.
//  * PV: B = P^T with slot j = 4X + i, the same key as above; A = V^T rows
//    (A row = dim 16b + col), slot j = V[page X][key 4grp + i][dim]. The
//    result lane (col, grp) holds O^T[d = 16b + 4grp + i][row col].
//  * Loads are software-pipelined: the operands of step i+1 are in flight
//    while step i is computed, and the next span's page ids are loaded when
//    its predecessor starts.
template <typename T, int D, typename TO, bool NT>
__device__ __forceinline__ void run_item(const AttnArgs& a, const Item& it, int lane) {
  using F = typename FragOf<T>::type;
  constexpr int NS = D / 32;   // QK steps over d
  constexpr int NB = D / 16;   // PV output blocks over d
  constexpr int64_t kTile = 16 * D;   // elements of one (page, head) tile
  using Regs = StepRegs<F, NS, NB>;
  const int col = lane & 15;
  const int grp = lane >> 4;

  Row row{-1, 0, -1, 0};
  if (col < it.n_rows) row = a.rows[it.row_begin + col];

  F qf[NS];
  {
    const T* qp = static_cast<const T*>(a.q) + (int64_t)(row.q_row < 0 ? 0 : row.q_row) * D + 8 * grp;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = row.q_row >= 0 ? load8(qp + 32 * s) : zero_frag<F>();
  }

  const int64_t page_stride = (int64_t)a.num_kv_heads * kTile;
  const T* kbase = static_cast<const T*>(a.k_pool) + (int64_t)it.kv_head * kTile;
  const T* vbase = static_cast<const T*>(a.v_pool) + (int64_t)it.kv_head * kTile;
  const int v_off = col * 16 + 4 * grp;   // V^T[dim col][key 4grp] in a tile

  auto load_span = [&](int si) {
    SpanState st;
    st.valid = si < it.n_spans;
    st.kb = st.ke = st.causal = 0;
    st.vpid = 0;
    if (st.valid) {
      const Span sp = a.spans[it.span_begin + si];
      st.kb = sp.key_begin;
      st.ke = sp.key_end;
      st.causal = sp.causal;
      const int np = (sp.key_end - sp.key_begin + 15) >> 4;
      st.vpid = lane < np ? a.page_ids[sp.page_off + lane] : 0;
    }
    return st;
  };
  auto step_at = [&](const SpanState& st, int t0) {
    StepPos p;
    p.valid = st.valid;
    p.t0 = t0;
    p.key_end = st.ke;
    p.causal = st.causal;
    const int j = (t0 - st.kb) >> 4;
    p.has1 = t0 + 16 < st.ke;
    p.pid0 = __builtin_amdgcn_readlane(st.vpid, j);
    p.pid1 = p.has1 ? __builtin_amdgcn_readlane(st.vpid, j + 1) : p.pid0;
    return p;
  };
  auto fetch = [&](const StepPos& p, Regs& r) {
    const T* k0 = kbase + (int64_t)p.pid0 * page_stride;
    const T* k1 = kbase + (int64_t)p.pid1 * page_stride;
#pragma unroll
    for (int s = 0; s < NS; ++s) {
      r.k[0][s] = load_k8<NT>(k0, col, 32 * s + 8 * grp);
      r.k[1][s] = load_k8<NT>(k1, col, 32 * s + 8 * grp);
    }
    const T* v0 = vbase + (int64_t)p.pid0 * page_stride;
    const T* v1 = vbase + (int64_t)p.pid1 * page_stride;
#pragma unroll
    for (int b = 0; b < NB; ++b) r.v[b] = load_v8<NT>(v0, v1, v_off + b * 256);
  };

  // Span cursor: cur is being walked, nxt is loaded one span ahead.
  int si = 0;
  SpanState cur = load_span(0);
  SpanState nxt = load_span(1);
  int t_next = cur.kb;   // first key of the next step to issue
  auto advance = [&]() {
    // position of the next step to issue, moving to the next span if needed
    if (t_next >= cur.ke) {
      cur = nxt;
      ++si;
      nxt = load_span(si + 1);
      t_next = cur.kb;
    }
    StepPos p = step_at(cur, t_next);
    t_next += kKeysPerStep;
    return p;
  };

  float m = kNegInf;
  float lsum = 0.f;
  f32x4_t acc[NB];
#pragma unroll
  for (int b = 0; b < NB; ++b) acc[b] = f32x4_t{0.f, 0.f, 0.f, 0.f};

  auto compute = [&](const StepPos& p, Regs& r) {
    f32x4_t sacc[2];
#pragma unroll
    for (int x = 0; x < 2; ++x) {
      sacc[x] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
      for (int s = 0; s < NS; ++s) sacc[x] = mma(r.k[x][s], qf[s], sacc[x]);
    }
    // slot j = 4X + i holds key t0 + 16X + 4grp + i
    float sv[8];
    if (p.t0 + kKeysPerStep <= p.key_end && !p.causal) {
#pragma unroll
      for (int j = 0; j < 8; ++j) sv[j] = sacc[j >> 2][j & 3] * a.scale_log2;
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int key = p.t0 + 16 * (j >> 2) + 4 * grp + (j & 3);
        const bool vis = key < p.key_end && (!p.causal || key <= row.qpos);
        sv[j] = vis ? sacc[j >> 2][j & 3] * a.scale_log2 : kNegInf;
      }
      // Keys past the span end may be NaN page tails (or a repeated page):
      // zero V there, since P = 0 times NaN would still poison the sum.
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (p.t0 + 16 * (j >> 2) + 4 * grp + (j & 3) >= p.key_end)
#pragma unroll
          for (int b = 0; b < NB; ++b) r.v[b][j] = (T)0.f;
    }
    float mt = sv[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) mt = fmaxf(mt, sv[j]);
    mt = fmaxf(mt, __shfl_xor(mt, 16));
    mt = fmaxf(mt, __shfl_xor(mt, 32));
    const float m_new = fmaxf(m, mt);
    const float m_use = m_new == kNegInf ? 0.f : m_new;
    const float alpha = __builtin_amdgcn_exp2f(m - m_use);
    float pr[8];
    float psum = 0.f;
#pragma unroll
    for (int j = 0; j < 8; ++j) {
      pr[j] = __builtin_amdgcn_exp2f(sv[j] - m_use);
      psum += pr[j];
    }
    lsum = lsum * alpha + psum;
    m = m_new;
    const F pf = to_frag(pr, (F*)nullptr);
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      acc[b] *= alpha;
      acc[b] = mma(r.v[b], pf, acc[b]);
    }
  };

  if (cur.valid) {
    Regs ra, rb;
    StepPos pa = advance();
    fetch(pa, ra);
    while (true) {
      StepPos pb = advance();
      fetch(pick(pb.valid, pb, pa), rb);
      compute(pa, ra);
      if (!pb.valid) break;
      pa = advance();
      fetch(pick(pa.valid, pa, pb), ra);
      compute(pb, rb);
      if (!pa.valid) break;
    }
  }

  lsum += __shfl_xor(lsum, 16);
  lsum += __shfl_xor(lsum, 32);
  const bool has_row = col < it.n_rows;
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  const float lse2 = lsum > 0.f ? m + __log2f(lsum) : kNegInf;
  if (it.part_base >= 0) {
    if (has_row) {
      const int64_t prow = (int64_t)it.part_base + col;
      float* dst = a.part_o + prow * D + 4 * grp;
#pragma unroll
      for (int b = 0; b < NB; ++b) store4(dst + 16 * b, acc[b] * inv);
      if (grp == 0) a.part_lse[prow] = lse2;
    }
  } else if (has_row) {
    TO* dst = static_cast<TO*>(a.o) + (int64_t)row.q_row * D + 4 * grp;
#pragma unroll
    for (int b = 0; b < NB; ++b) store4(dst + 16 * b, acc[b] * inv);
    if (grp == 0 && a.lse) a.lse[row.q_row] = lse2 == kNegInf ? kNegInf : lse2 * kLn2;
  }
}

template <typename T, int D, typename TO>
__device__ __forceinline__ void narrow_block(const AttnArgs& a, int block) {
  const int item_id = __builtin_amdgcn_readfirstlane((int)(block * 4 + (threadIdx.x >> 6)));
  if (item_id >= a.n_items) return;
  const Item it = a.items[item_id];
  if (it.flags & kItemStream) run_item<T, D, TO, true>(a, it, threadIdx.x & 63);
  else run_item<T, D, TO, false>(a, it, threadIdx.x & 63);
}


// ---------------------------------------------------------------- wide items
// A wide item holds up to 4 * RB * 16 query rows of one kv head against a
// span list: a workgroup of 4 waves, RB MFMA row blocks per wave, all rows
// sharing the key stream. Each 32-key step's four tiles (K and V of its two
// pages) are read once per workgroup with coalesced 16-byte loads, two steps
// ahead through registers, into an LDS double buffer; every wave then reads
// its MFMA operands from LDS (1 KB contiguous per K read, 512 B per V read).
// Used for the grouped prefix pass (many rows share one segment, §2
// intra-batch prefix sharing) and for chunked prefill (§4.1).
//
// Softmax rescaling is lazy: a row's reference maximum only moves when a
// step's maximum exceeds it by more than kRescaleLog2 (so weights stay below
// 2^kRescaleLog2); the result is the same softmax, and the accumulator
// rescale runs only on the rare steps where some row moves.
constexpr float kRescaleLog2 = 8.f;

template <int D>
struct WideGeom {
  static constexpr int kTileBytes = 16 * D * 2;           // one bf16 (page, head) tile
  static constexpr int kStepBytes = 4 * kTileBytes;       // K page0, K page1, V page0, V page1
  static constexpr int kChunksPerTile = kTileBytes / 16;  // 16-byte chunks
  static constexpr int kPerThread = 4 * kChunksPerTile / 256;
};

template <int D, int RB, typename TO>
__device__ __forceinline__ void wide_item(const AttnArgs& a, int item_id) {
  using T = __bf16;
  using F = bf16x8_t;
  using G = WideGeom<D>;
  constexpr int NS = D / 32;
  constexpr int NB = D / 16;
  constexpr int64_t kTile = 16 * D;
  __shared__ __attribute__((aligned(16))) uint8_t lds[2 * G::kStepBytes];

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int col = lane & 15;
  const int grp = lane >> 4;
  const Item it = a.wide_items[item_id];

  // This lane's rows: row block rb of this wave, column col.
  Row row[RB];
  F qf[RB][NS];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    const int r = (wave * RB + rb) * 16 + col;
    row[rb] = r < it.n_rows ? a.rows[it.row_begin + r] : Row{-1, 0, -1, 0};
    const T* qp = static_cast<const T*>(a.q) + (int64_t)(row[rb].q_row < 0 ? 0 : row[rb].q_row) * D + 8 * grp;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[rb][s] = row[rb].q_row >= 0 ? load8(qp + 32 * s) : zero_frag<F>();
  }

  const int64_t page_stride = (int64_t)a.num_kv_heads * kTile;
  const T* kbase = static_cast<const T*>(a.k_pool) + (int64_t)it.kv_head * kTile;
  const T* vbase = static_cast<const T*>(a.v_pool) + (int64_t)it.kv_head * kTile;

  // ---- span cursor (identical, wave-uniform, in every wave)
  auto load_span = [&](int si) {
    SpanState st;
    st.valid = si < it.n_spans;
    st.kb = st.ke = st.causal = 0;
    st.vpid = 0;
    if (st.valid) {
      const Span sp = a.spans[it.span_begin + si];
      st.kb = sp.key_begin;
      st.ke = sp.key_end;
      st.causal = sp.causal;
      const int np = (sp.key_end - sp.key_begin + 15) >> 4;
      st.vpid = lane < np ? a.page_ids[sp.page_off + lane] : 0;
    }
    return st;
  };
  int si = 0;
  SpanState cur = load_span(0);
  SpanState nxt = load_span(1);
  int t_next = cur.kb;
  auto advance = [&]() {
    if (t_next >= cur.ke) {
      cur = nxt;
      ++si;
      nxt = load_span(si + 1);
      t_next = cur.kb;
    }
    StepPos p;
    p.valid = cur.valid;
    p.t0 = t_next;
    p.key_end = cur.ke;
    p.causal = cur.causal;
    const int j = (t_next - cur.kb) >> 4;
    p.has1 = t_next + 16 < cur.ke;
    p.pid0 = __builtin_amdgcn_readlane(cur.vpid, j);
    p.pid1 = p.has1 ? __builtin_amdgcn_readlane(cur.vpid, j + 1) : p.pid0;
    t_next += kKeysPerStep;
    return p;
  };

  // ---- staging: thread t moves chunks t + 256k of the step (k < kPerThread)
  struct Stage { u32x4_t v[G::kPerThread]; };
  auto stage_load = [&](const StepPos& p, Stage& st) {
#pragma unroll
    for (int k = 0; k < G::kPerThread; ++k) {
      const int c = threadIdx.x + 256 * k;
      const int tile = c / G::kChunksPerTile;        // 0,1: K pages; 2,3: V pages
      const int off = (c % G::kChunksPerTile) * 8;   // elements
      const int pid = (tile & 1) ? p.pid1 : p.pid0;
      const T* src = ((tile < 2) ? kbase : vbase) + (int64_t)pid * page_stride + off;
      st.v[k] = *reinterpret_cast<const u32x4_t*>(src);
    }
  };
  // LDS image of a step: K tiles of both pages as stored ([D/8][16][8]),
  // then V as 16-byte cells, one per (dim d, lane group g):
  //   {page0 keys 4g..4g+3, page1 keys 4g..4g+3}
  // at cell d * 4 + (g ^ ((d >> 1) & 3)): a wave's V read is then one
  // conflict-free ds_read_b128 per output block (the XOR spreads the eight
  // lanes served together over all banks).
  auto stage_write = [&](const Stage& st, int buf) {
    uint8_t* base = lds + buf * G::kStepBytes;
#pragma unroll
    for (int k = 0; k < G::kPerThread; ++k) {
      const int c = threadIdx.x + 256 * k;
      const int tile = c / G::kChunksPerTile;
      const int chunk = c % G::kChunksPerTile;
      if (tile < 2) {
        *reinterpret_cast<u32x4_t*>(base + tile * G::kTileBytes + chunk * 16) = st.v[k];
      } else {
        const int d = chunk >> 1, h = chunk & 1, pg = tile - 2;
        uint8_t* vb = base + 2 * G::kTileBytes + pg * 8;
        const int sw = (d >> 1) & 3;
        *reinterpret_cast<u32x2_t*>(vb + (d * 4 + ((2 * h) ^ sw)) * 16) = u32x2_t{st.v[k].x, st.v[k].y};
        *reinterpret_cast<u32x2_t*>(vb + (d * 4 + ((2 * h + 1) ^ sw)) * 16) = u32x2_t{st.v[k].z, st.v[k].w};
      }
    }
  };

  float m[RB], lsum[RB];
  f32x4_t acc[RB][NB];
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    m[rb] = kNegInf;
    lsum[rb] = 0.f;
#pragma unroll
    for (int b = 0; b < NB; ++b) acc[rb][b] = f32x4_t{0.f, 0.f, 0.f, 0.f};
  }

  auto compute = [&](const StepPos& p, int buf) {
    const uint8_t* base = lds + buf * G::kStepBytes;
    // All K fragments of the step first, then the QK products.
    F kf[2][NS];
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int s = 0; s < NS; ++s)
        kf[x][s] = __builtin_bit_cast(
            F, *reinterpret_cast<const u32x4_t*>(base + x * G::kTileBytes + ((4 * s + grp) * 16 + col) * 16));
    f32x4_t sacc[RB][2];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) sacc[rb][0] = sacc[rb][1] = f32x4_t{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int x = 0; x < 2; ++x)
#pragma unroll
      for (int s = 0; s < NS; ++s)
#pragma unroll
        for (int rb = 0; rb < RB; ++rb) sacc[rb][x] = mma(kf[x][s], qf[rb][s], sacc[rb][x]);
    // V fragments are read now so the LDS latency overlaps the softmax.
    F vf[NB];
#pragma unroll
    for (int b = 0; b < NB; ++b) {
      const int d = 16 * b + col;
      vf[b] = __builtin_bit_cast(
          F, *reinterpret_cast<const u32x4_t*>(base + 2 * G::kTileBytes + (d * 4 + (grp ^ ((d >> 1) & 3))) * 16));
    }
    const bool full = p.t0 + kKeysPerStep <= p.key_end && !p.causal;
    F pf[RB];
#pragma unroll
    for (int rb = 0; rb < RB; ++rb) {
      // raw scores (masked ones -inf); the scale is applied inside the
      // exponent with one FMA (scale > 0, so it commutes with the max)
      float sv[8];
      if (full) {
#pragma unroll
        for (int j = 0; j < 8; ++j) sv[j] = sacc[rb][j >> 2][j & 3];
      } else {
        const int lim = p.causal ? min(p.key_end, row[rb].qpos + 1) : p.key_end;
#pragma unroll
        for (int j = 0; j < 8; ++j) {
          const int key = p.t0 + 16 * (j >> 2) + 4 * grp + (j & 3);
          sv[j] = key < lim ? sacc[rb][j >> 2][j & 3] : kNegInf;
        }
      }
      float mt = sv[0];
#pragma unroll
      for (int j = 1; j < 8; ++j) mt = fmaxf(mt, sv[j]);
      mt = fmaxf(mt, __shfl_xor(mt, 16));
      mt = fmaxf(mt, __shfl_xor(mt, 32));
      mt *= a.scale_log2;
      const bool move = mt > m[rb] + kRescaleLog2;
      if (__any(move)) {
        const float m_new = move ? mt : m[rb];
        const float alpha = m[rb] == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m[rb] - m_new);
        lsum[rb] *= alpha;
#pragma unroll
        for (int b = 0; b < NB; ++b) acc[rb][b] *= alpha;
        m[rb] = m_new;
      }
      const float m_use = m[rb] == kNegInf ? 0.f : m[rb];
      float pr[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        pr[j] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[j], a.scale_log2, -m_use));
        lsum[rb] += pr[j];
      }
      pf[rb] = to_frag(pr, (F*)nullptr);
    }
    if (!full) {
      // keys past the span end may be NaN page tails: zero V there
#pragma unroll
      for (int j = 0; j < 8; ++j)
        if (p.t0 + 16 * (j >> 2) + 4 * grp + (j & 3) >= p.key_end)
#pragma unroll
          for (int b = 0; b < NB; ++b) vf[b][j] = (T)0.f;
    }
#pragma unroll
    for (int b = 0; b < NB; ++b)
#pragma unroll
      for (int rb = 0; rb < RB; ++rb) acc[rb][b] = mma(vf[b], pf[rb], acc[rb][b]);
  };

  // ---- pipeline: LDS buffers 0/1, register stages r0/r1, two steps ahead
  StepPos p0 = advance();
  StepPos p1 = advance();
  if (p0.valid) {
    Stage r0, r1;
    stage_load(p0, r0);
    stage_load(pick(p1.valid, p1, p0), r1);
    stage_write(r0, 0);
    __syncthreads();
    while (true) {
      StepPos p2 = advance();
      stage_load(pick(p2.valid, p2, p0), r0);
      compute(p0, 0);
      if (!p1.valid) break;
      stage_write(r1, 1);
      __syncthreads();
      StepPos p3 = advance();
      stage_load(pick(p3.valid, p3, p1), r1);
      compute(p1, 1);
      if (!p2.valid) break;
      stage_write(r0, 0);
      __syncthreads();
      p0 = p2;
      p1 = p3;
    }
  }

  // ---- epilogue
#pragma unroll
  for (int rb = 0; rb < RB; ++rb) {
    float l = lsum[rb];
    l += __shfl_xor(l, 16);
    l += __shfl_xor(l, 32);
    const int r = (wave * RB + rb) * 16 + col;
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const float lse2 = l > 0.f ? m[rb] + __log2f(l) : kNegInf;
    if (it.part_base >= 0) {
      if (r < it.n_rows) {
        const int64_t prow = (int64_t)it.part_base + r;
        float* dst = a.part_o + prow * D + 4 * grp;
#pragma unroll
        for (int b = 0; b < NB; ++b) store4(dst + 16 * b, acc[rb][b] * inv);
        if (grp == 0) a.part_lse[prow] = lse2;
      }
    } else if (r < it.n_rows) {
      TO* dst = static_cast<TO*>(a.o) + (int64_t)row[rb].q_row * D + 4 * grp;
#pragma unroll
      for (int b = 0; b < NB; ++b) store4(dst + 16 * b, acc[rb][b] * inv);
      if (grp == 0 && a.lse) a.lse[row[rb].q_row] = lse2 == kNegInf ? kNegInf : lse2 * kLn2;
    }
  }
}

// ---------------------------------------------------------------- launch
// One launch runs both roles: the first wide_blocks blocks are wide items
// (MFMA/LDS-bound grouped prefix or prefill work), the rest hold four narrow
// items each (mostly HBM-bound suffix streaming), so the two kinds of work
// overlap on the GPU. RB = 0: no wide role (fp32 inputs).
// The grid is dealt in rounds of 8 blocks (one per XCD); rounds of the two
// roles are spread evenly over the launch so every CU mixes MFMA-heavy wide
// blocks with HBM-heavy narrow ones, and within a role the block index modulo
// 8 still names the XCD (xcd_remap stays valid).
template <typename T, int D, typename TO, int RB>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(sizeof(T) == 2 ? 2 : 1)))
void attn_kernel(AttnArgs a) {
  const int b = blockIdx.x;
  const int x = b & 7, r = b >> 3;
  if constexpr (RB > 0) {
    const int wr = a.wide_blocks >> 3;
    const int tr = wr + (a.narrow_blocks >> 3);
    const int w_before = (int)((int64_t)r * wr / tr);
    const int w_upto = (int)((int64_t)(r + 1) * wr / tr);
    if (w_upto > w_before) {
      const int item = xcd_remap(w_before * 8 + x, a.wide_group);
      if (item < a.n_wide) wide_item<D, RB, TO>(a, item);
      return;
    }
    narrow_block<T, D, TO>(a, xcd_remap((r - w_upto) * 8 + x, a.narrow_group));
  } else {
    narrow_block<T, D, TO>(a, xcd_remap(b, a.narrow_group));
  }
}

// ---------------------------------------------------------------- merge

struct MergeArgs {
  const float* part_o;
  const float* part_lse;
  const int32_t* merge_rows;
  const int32_t* merge_indptr;
  const int32_t* merge_parts;
  void* o;
  float* lse;
  int32_t n_merge;
};

// Output rows whose keys were split over several items. Partials hold the
// normalized o_i and lse_i (log2) of disjoint key sets:
//   M = max_i lse_i,  w_i = 2^(lse_i - M),  O = sum w_i o_i / sum w_i,
//   LSE = (M + log2 sum w_i) * ln 2
// which is exact in real arithmetic (shared == unshared, §3 "Scope"). One
// group of D/4 threads per row, 4 dims per thread; the partial ids and
// LSEs of up to 8 parts are fetched together so the loads overlap.
template <int D, typename TO>
__global__ __launch_bounds__(256) void merge_kernel(MergeArgs a) {
  constexpr int TPR = D / 4;
  constexpr int RPB = 256 / TPR;
  constexpr int kBatch = 8;
  const int r = blockIdx.x * RPB + threadIdx.x / TPR;
  const int t = threadIdx.x % TPR;
  if (r >= a.n_merge) return;
  const int q_row = a.merge_rows[r];
  const int p0 = a.merge_indptr[r], p1 = a.merge_indptr[r + 1];
  float mx = kNegInf;
  f32x4_t acc = {0.f, 0.f, 0.f, 0.f};
  float wsum = 0.f;
  // online over batches of parts: rescale when the running max moves
  for (int pb = p0; pb < p1; pb += kBatch) {
    int pid[kBatch];
    float l[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) pid[k] = pb + k < p1 ? a.merge_parts[pb + k] : -1;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) l[k] = pid[k] >= 0 ? a.part_lse[pid[k]] : kNegInf;
    f32x4_t v[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const float4 x = pid[k] >= 0 ? *reinterpret_cast<const float4*>(a.part_o + (int64_t)pid[k] * D + 4 * t)
                                   : make_float4(0.f, 0.f, 0.f, 0.f);
      v[k] = f32x4_t{x.x, x.y, x.z, x.w};
    }
    float bm = kNegInf;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) bm = fmaxf(bm, l[k]);
    const float m_new = fmaxf(mx, bm);
    if (m_new == kNegInf) continue;
    const float alpha = mx == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mx - m_new);
    acc *= alpha;
    wsum *= alpha;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const float w = __builtin_amdgcn_exp2f(l[k] - m_new);   // 0 for absent parts
      wsum += w;
      acc += w * v[k];
    }
    mx = m_new;
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
  store4(static_cast<TO*>(a.o) + (int64_t)q_row * D + 4 * t, acc * inv);
  if (t == 0 && a.lse) a.lse[q_row] = wsum > 0.f ? (mx + __log2f(wsum)) * kLn2 : kNegInf;
}

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

// One block per (page slot, head) tile, grid-stride. W is an unsigned word of
// the element's width, so every bit pattern (NaN payloads included) moves
// unchanged.
template <typename W>
__global__ __launch_bounds__(256) void gather_kernel(GatherArgs a) {
  __shared__ W tile[16 * (128 + 1)];
  const int D = a.head_dim;
  const int64_t total_tiles = (int64_t)a.seq_page_indptr[a.num_seqs] * a.num_kv_heads;
  const W* pool = static_cast<const W*>(a.pool);
  W* out = static_cast<W*>(a.out);
  for (int64_t tl = blockIdx.x; tl < total_tiles; tl += gridDim.x) {
    const int64_t slot = tl / a.num_kv_heads;
    const int h = (int)(tl % a.num_kv_heads);
    int lo = 0, hi = a.num_seqs - 1;   // last sequence whose first slot <= slot
    while (lo < hi) {
      const int mid = (lo + hi + 1) >> 1;
      if (a.seq_page_indptr[mid] <= slot) lo = mid; else hi = mid - 1;
    }
    const int len = a.seq_len[lo];
    const int npages = a.seq_page_indptr[lo + 1] - a.seq_page_indptr[lo];
    const int pid = a.page_ids[slot];
    if (len < 0 || npages != (len + 15) / 16 || pid < 0 || pid >= a.num_pool_pages) {
      if (threadIdx.x == 0 && a.error_flag) a.error_flag[0] = 1;
      continue;
    }
    const int t0 = (int)(slot - a.seq_page_indptr[lo]) * 16;
    const int n = min(16, len - t0);
    const int64_t out_tok = a.out_token_offset[lo] + t0;
    const W* src = pool + ((int64_t)pid * a.num_kv_heads + h) * 16 * D;
    // Read the whole (page, head) tile coalesced, in its stored order, and
    // place element (token t, dim c) at tile[t][c] (row stride D + 1).
    constexpr int E = 16 / (int)sizeof(W);
    for (int e = threadIdx.x; e < 16 * D; e += blockDim.x) {
      int t, c;
      if (!a.v_layout) {           // K: [D/E][16][E]
        c = (e / (16 * E)) * E + e % E;
        t = (e / E) % 16;
      } else {                     // V: [D][16]
        c = e >> 4;
        t = e & 15;
      }
      tile[t * (D + 1) + c] = src[e];
    }
    __syncthreads();
    for (int e = threadIdx.x; e < n * D; e += blockDim.x) {
      const int tok = e / D, c = e - tok * D;
      out[((out_tok + tok) * a.num_kv_heads + h) * D + c] = tile[tok * (D + 1) + c];
    }
    __syncthreads();
  }
}

// ---------------------------------------------------------------- host side

size_t align256(size_t x) { return (x + 255) / 256 * 256; }

bool aligned16(const void* p) { return (reinterpret_cast<uintptr_t>(p) & 15) == 0; }

halo_status_t hip_check(const char* what) {
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(HALO_ERR_HIP, std::string(what) + ": " + hipGetErrorString(e));
  return HALO_OK;
}

int pad_to(int n, int m) { return (n + m - 1) / m * m; }

template <typename T, int D, typename TO>
void launch_attention(AttnArgs args, const MergeArgs& margs, int wide_rb, hipStream_t stream) {
  const int rb = sizeof(T) == 2 ? wide_rb : 0;
  args.wide_blocks = (rb > 0 && args.n_wide > 0) ? pad_to(args.n_wide, 8 * args.wide_group) : 0;
  args.narrow_blocks = args.n_items > 0 ? pad_to((args.n_items + 3) / 4, 8 * args.narrow_group) : 0;
  const int grid = args.wide_blocks + args.narrow_blocks;
  if (grid > 0) {
    if constexpr (sizeof(T) == 2) {
      if (rb == 2)
        hipLaunchKernelGGL((attn_kernel<T, D, TO, 2>), dim3(grid), dim3(256), 0, stream, args);
      else if (rb == 1)
        hipLaunchKernelGGL((attn_kernel<T, D, TO, 1>), dim3(grid), dim3(256), 0, stream, args);
      else
        hipLaunchKernelGGL((attn_kernel<T, D, TO, 0>), dim3(grid), dim3(256), 0, stream, args);
    } else {
      hipLaunchKernelGGL((attn_kernel<T, D, TO, 0>), dim3(grid), dim3(256), 0, stream, args);
    }
  }
  if (margs.n_merge > 0) {
    constexpr int rpb = 256 / (D / 4);
    const int blocks = (margs.n_merge + rpb - 1) / rpb;
    hipLaunchKernelGGL((merge_kernel<D, TO>), dim3(blocks), dim3(256), 0, stream, margs);
  }
}

halo_status_t run_attention(const halo_plan_t* plan, bool want_prefill, const void* device_meta,
                            const void* q, const void* k_pool, const void* v_pool, void* o, float* lse,
                            void* workspace, size_t workspace_bytes, void* stream) {
  clear_error();
  if (!plan) return fail(HALO_ERR_INVALID_ARGUMENT, "plan must not be NULL");
  if (plan->prefill != want_prefill)
    return fail(HALO_ERR_INVALID_ARGUMENT,
                want_prefill ? "plan was built for decode (q_len == NULL)" : "plan was built for prefill");
  if (!device_meta || !q || !k_pool || !v_pool || !o)
    return fail(HALO_ERR_INVALID_ARGUMENT, "device_meta, q, k_pool, v_pool and o must not be NULL");
  if (!aligned16(q) || !aligned16(k_pool) || !aligned16(v_pool) || !aligned16(o) ||
      (reinterpret_cast<uintptr_t>(device_meta) & 255) != 0)
    return fail(HALO_ERR_INVALID_ARGUMENT, "q, k_pool, v_pool, o must be 16-byte aligned, device_meta 256-byte");
  if (workspace_bytes < plan->workspace_bytes)
    return fail(HALO_ERR_WORKSPACE_TOO_SMALL, "workspace needs " + std::to_string(plan->workspace_bytes) +
                                                  " bytes, got " + std::to_string(workspace_bytes));
  if (plan->workspace_bytes > 0 && (!workspace || (reinterpret_cast<uintptr_t>(workspace) & 255) != 0))
    return fail(HALO_ERR_INVALID_ARGUMENT, "workspace must be a 256-byte aligned device pointer");

  const halo_attn_params_t& p = plan->params;
  const MetaLayout& L = plan->layout;
  const uint8_t* m = static_cast<const uint8_t*>(device_meta);
  const int D = p.head_dim;
  float* part_o = static_cast<float*>(workspace);
  float* part_lse = plan->n_part_rows
                        ? reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) +
                                                   align256((size_t)plan->n_part_rows * D * sizeof(float)))
                        : nullptr;
  AttnArgs args{q, k_pool, v_pool, o, lse, part_o, part_lse,
                reinterpret_cast<const int32_t*>(m + L.seg_page_off),
                reinterpret_cast<const int32_t*>(m + L.seg_len),
                reinterpret_cast<const int32_t*>(m + L.page_ids),
                reinterpret_cast<const Item*>(m + L.items),
                reinterpret_cast<const Item*>(m + L.wide_items),
                reinterpret_cast<const Span*>(m + L.spans),
                reinterpret_cast<const Row*>(m + L.rows),
                plan->n_items, plan->n_wide, 0, 0, plan->wide_group, plan->narrow_group,
                p.num_kv_heads, p.sm_scale * kLog2e};
  MergeArgs margs{part_o, part_lse,
                  reinterpret_cast<const int32_t*>(m + L.merge_rows),
                  reinterpret_cast<const int32_t*>(m + L.merge_indptr),
                  reinterpret_cast<const int32_t*>(m + L.merge_parts),
                  o, lse, plan->n_merge};
  hipStream_t st = static_cast<hipStream_t>(stream);
  (void)hipGetLastError();   // clear any stale error of the caller
  const bool out_f32 = p.out_dtype == HALO_F32;
  if (p.kv_dtype == HALO_BF16) {
    if (D == 128) {
      if (out_f32) launch_attention<__bf16, 128, float>(args, margs, plan->wide_rb, st);
      else launch_attention<__bf16, 128, __bf16>(args, margs, plan->wide_rb, st);
    } else {
      if (out_f32) launch_attention<__bf16, 64, float>(args, margs, plan->wide_rb, st);
      else launch_attention<__bf16, 64, __bf16>(args, margs, plan->wide_rb, st);
    }
  } else {
    if (D == 128) launch_attention<float, 128, float>(args, margs, plan->wide_rb, st);
    else launch_attention<float, 64, float>(args, margs, plan->wide_rb, st);
  }
  return hip_check("attention launch");
}

}  // namespace

extern "C" halo_status_t halo_plan_upload(const halo_plan_t* plan, void* device_meta,
                                          size_t device_meta_bytes, void* stream) {
  clear_error();
  if (!plan || !device_meta) return fail(HALO_ERR_INVALID_ARGUMENT, "plan and device_meta must not be NULL");
  if (device_meta_bytes < plan->layout.total)
    return fail(HALO_ERR_INVALID_ARGUMENT, "device_meta needs " + std::to_string(plan->layout.total) + " bytes");
  if ((reinterpret_cast<uintptr_t>(device_meta) & 255) != 0)
    return fail(HALO_ERR_INVALID_ARGUMENT, "device_meta must be 256-byte aligned");
  hipError_t e = hipMemcpyAsync(device_meta, plan->meta.data(), plan->layout.total, hipMemcpyHostToDevice,
                                static_cast<hipStream_t>(stream));
  if (e != hipSuccess) return fail(HALO_ERR_HIP, std::string("hipMemcpyAsync: ") + hipGetErrorString(e));
  return HALO_OK;
}

extern "C" halo_status_t halo_prefix_attn_decode(const halo_plan_t* plan, const void* device_meta,
                                                 const void* q, const void* k_pool, const void* v_pool,
                                                 void* o, float* lse, void* workspace,
                                                 size_t workspace_bytes, void* stream) {
  return run_attention(plan, false, device_meta, q, k_pool, v_pool, o, lse, workspace, workspace_bytes,
                       stream);
}

extern "C" halo_status_t halo_prefix_attn_prefill(const halo_plan_t* plan, const void* device_meta,
                                                  const void* q, const void* k_pool, const void* v_pool,
                                                  void* o, float* lse, void* workspace,
                                                  size_t workspace_bytes, void* stream) {
  return run_attention(plan, true, device_meta, q, k_pool, v_pool, o, lse, workspace, workspace_bytes,
                       stream);
}

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
  const int blocks = 2048;
  if (params->kv_dtype == HALO_BF16)
    hipLaunchKernelGGL(gather_kernel<uint16_t>, dim3(blocks), dim3(256), 0, st, g);
  else if (params->kv_dtype == HALO_F32)
    hipLaunchKernelGGL(gather_kernel<uint32_t>, dim3(blocks), dim3(256), 0, st, g);
  else
    return fail(HALO_ERR_UNSUPPORTED, "kv_dtype must be HALO_F32 or HALO_BF16");
  return hip_check("gather launch");
}
