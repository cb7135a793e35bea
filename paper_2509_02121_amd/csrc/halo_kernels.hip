// gfx950 kernels and the run-time entry points of the C ABI.
//
// attn_kernel: one launch for the grouped prefix pass, the suffix pass and
//   chunked prefill, with two kinds of workgroups:
//   * narrow: item slots of one wavefront each (<= 16 query rows against a
//     list of key spans). Per step of 32 keys (two 16-token pages):
//       S^T = K Q^T  on v_mfma_f32_16x16x32_bf16 (one 16-key tile per page,
//                    4 MFMAs per tile at d=128)
//       online softmax in the log2 domain (row max / sum over the 4 lane
//       groups)
//       O^T += V^T P^T on the same MFMA (8 MFMAs at d=128)
//     K pages are stored in 16-byte units ([d/E][16][E]) and V pages
//     dim-major ([d][16], slots permuted so 8 keys of a lane are 16
//     contiguous bytes), so every MFMA operand is a direct 1 KB-per-wave load
//     from one or two pages. The QK output layout is already the PV B
//     operand (no lane exchange).
//   * wide: up to 256 query rows (8 waves x 32) sharing one key stream,
//     staged once per workgroup through an LDS ring by direct global-to-LDS
//     loads, on v_mfma_f32_32x32x16_bf16.
// merge_kernel: exact log-sum-exp combination of partial results over
//   disjoint key ranges (the merge that makes shared == unshared), in its own
//   launch so the kernel boundary makes every partial visible (an in-kernel
//   last-arriver merge needs agent-scope release/acquire, i.e. L2
//   write-back and invalidate, which measured 4x slower on this path).
// The page gather and the write path live in halo_pages.hip.

#include <hip/hip_runtime.h>

#include <atomic>
#include <cmath>
#include <mutex>
#include <string>
#include <type_traits>

#include "halo_internal.h"

using namespace halo;

namespace {

typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x8_t __attribute__((ext_vector_type(8)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));
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

// V fragment: the 8 slot-ordered keys at element offset off of a V tile
// stored dim-major as [D][16] (one dim row holds tokens 0-3, 8-11, 4-7,
// 12-15, so slots 8h..8h+7 are the keys one lane multiplies).
template <bool NT>
__device__ __forceinline__ bf16x8_t load_v8(const __bf16* page, int off) {
  return __builtin_bit_cast(bf16x8_t, ld16<NT>(page + off));
}
template <bool NT>
__device__ __forceinline__ f32x8_t load_v8(const float* page, int off) {
  const u32x4_t lo = ld16<NT>(page + off);
  const u32x4_t hi = ld16<NT>(page + off + 4);
  return __builtin_bit_cast(f32x8_t, __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7));
}

// Key (relative to the first key of a 32-key step) behind slot j of a lane
// in lane group grp. QK tile X (X = j / 4) takes its 16 A rows as keys
// 8X..8X+7 of page 0 (rows 0-7) and of page 1 (rows 8-15); MFMA output
// register i of lane group grp is tile row 4 grp + i, i.e. page grp / 2,
// key 8X + 4 (grp % 2) + i.
__device__ __forceinline__ int slot_key(int grp, int j) {
  return 16 * (grp >> 1) + 8 * (j >> 2) + 4 * (grp & 1) + (j & 3);
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

// D(32x32) += A(32x16) B(16x32), bf16 operands, fp32 accumulate. Lane
// (c = lane % 32, h = lane / 32): A row c and B column c, k = 8h..8h+7;
// result register i holds row 8 (i / 4) + 4h + i % 4, column c.
__device__ __forceinline__ f32x16_t mma32(bf16x8_t a, bf16x8_t b, f32x16_t c) {
  return __builtin_amdgcn_mfma_f32_32x32x16_bf16(a, b, c, 0, 0, 0);
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
// Partial results (read once, by the merge launch): four elements of a row
// per lane, so a row's line is written in 16-byte (fp32) or 8-byte (bf16)
// pieces by several instructions. fp32 pieces go past the caches; bf16
// pieces are half as large, and written past the caches they cost more than
// they save (measured on the 70B-shaped decode: 966 against 934 us of
// attention for fp32 partials), so they go through L2, which assembles the
// lines before they reach HBM.
__device__ __forceinline__ void store4_part(float* dst, f32x4_t v) {
  __builtin_nontemporal_store(v, reinterpret_cast<f32x4_t*>(dst));
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
__device__ __forceinline__ void store4_part(__bf16* dst, f32x4_t v) { store4(dst, v); }

// Reductions over the four 16-lane rows of a wave (lanes l, l^16, l^32,
// l^48) with the gfx950 row-swap instructions, which stay on the VALU
// instead of going through the LDS crossbar like a generic shuffle. Each
// swap leaves, in every lane, the pair {own value, value of lane l^16} (or
// l^32), in some order; max and sum are symmetric in the pair.
__device__ __forceinline__ float rows_max(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = fmaxf(__uint_as_float(a[0]), __uint_as_float(a[1]));
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float rows_sum(float x) {
  auto a = __builtin_amdgcn_permlane16_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  x = __uint_as_float(a[0]) + __uint_as_float(a[1]);
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// Reductions over the two 32-lane halves of a wave (lanes l and l^32).
__device__ __forceinline__ float halves_max(float x) {
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return fmaxf(__uint_as_float(b[0]), __uint_as_float(b[1]));
}
__device__ __forceinline__ float halves_sum(float x) {
  auto b = __builtin_amdgcn_permlane32_swap(__float_as_uint(x), __float_as_uint(x), false, false);
  return __uint_as_float(b[0]) + __uint_as_float(b[1]);
}

// ---------------------------------------------------------------- attention

struct AttnArgs {
  const void* q;
  const void* k_pool;
  const void* v_pool;
  void* o;
  float* lse;
  void* part_o;      // partial O rows, in the output element type
  float* part_lse;
  const int32_t* seg_page_off;
  const int32_t* seg_len;
  const int32_t* page_ids;
  const Item* items;        // narrow item slots: slot k of narrow workgroup b is item b * narrow_slots + k
  const ItemRec* item_recs; // their lane records
  const Item* wide_items;   // wide items (one workgroup each)
  const Span* spans;
  const Row* rows;
  int32_t n_items;
  int32_t n_wide;
  int32_t wide_blocks;     // grid blocks of the wide role (n_wide padded, see xcd_remap)
  int32_t narrow_blocks;   // grid blocks of the narrow role (a multiple of 8)
  int32_t narrow_slots;    // item slots per narrow workgroup (one per wave)
  int32_t wide_group;      // consecutive wide items kept on one XCD
  int32_t wide_span;       // launch rounds (of 8 blocks) the wide rounds are spread over
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
// Within an XCD, workgroups are dispatched in order and in turn to its 4
// shader engines (the XCD's j-th workgroup goes to engine j % 4, in a fixed
// order): a workgroup waits for its engine even when another engine has a
// free CU. The launch therefore mixes wide and narrow workgroups in whole
// cycles of kSeCycle rounds, so every engine gets the same kinds at the same
// time.
constexpr int kSeCycle = 4;

__device__ __forceinline__ int xcd_remap(int p, int S) {
  const int x = p & 7, j = p >> 3;
  return ((j / S) * 8 + x) * S + j % S;
}

// s_waitcnt with only the vector-memory counter limited (gfx9 encoding:
// vmcnt low bits [3:0] and high bits [15:14]; expcnt and lgkmcnt at their
// "no wait" maxima).
template <int N>
__device__ __forceinline__ void wait_vmcnt() {
  static_assert(N >= 0 && N < 64, "vmcnt range");
  __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | 0x70 | 0xF00);
}
__device__ __forceinline__ void wait_lgkmcnt0() { __builtin_amdgcn_s_waitcnt(0xC07F); }

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
  bool full;       // all 32 keys visible to every row: inside the span, no causal mask
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
  r.full = c ? x.full : y.full;
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
// This lane's words of a narrow item's record: its row's q_row and second
// word (lane % 16), and page lane % 32 of the first span.
struct RecLane {
  int32_t q_row, aux, page;
};

template <typename T, int D, typename TO, bool NT, int P>
__device__ __forceinline__ void run_item(const AttnArgs& a, const Item& it, const RecLane& rl, int lane) {
  using F = typename FragOf<T>::type;
  constexpr int NS = D / 32;   // QK steps over d
  constexpr int NB = D / 16;   // PV output blocks over d
  constexpr int64_t kTile = 16 * D;   // elements of one (page, head) tile
  using Regs = StepRegs<F, NS, NB>;
  const int col = lane & 15;
  const int grp = lane >> 4;

  // The item's lane record: this lane's row, and page j of the first span
  // in lane j. (aux: chunk position for a prefill item, partial slot for a
  // decode one)
  Row row{rl.q_row, rl.aux, -1, rl.aux};
  const int32_t vpid0 = rl.page;

  F qf[NS];
  {
    const T* qp = static_cast<const T*>(a.q) + (int64_t)(row.q_row < 0 ? 0 : row.q_row) * D + 8 * grp;
#pragma unroll
    for (int s = 0; s < NS; ++s) qf[s] = row.q_row >= 0 ? load8(qp + 32 * s) : zero_frag<F>();
  }

  const int64_t page_stride = (int64_t)a.num_kv_heads * kTile;
  const T* kbase = static_cast<const T*>(a.k_pool) + (int64_t)it.kv_head * kTile;
  const T* vbase = static_cast<const T*>(a.v_pool) + (int64_t)it.kv_head * kTile;
  const int v_off = col * 16 + 8 * (grp & 1);   // V^T[dim col][slots 8(grp%2)..] in a tile

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
    p.full = t0 + kKeysPerStep <= st.ke && !st.causal;
    p.pid0 = __builtin_amdgcn_readlane(st.vpid, j);
    p.pid1 = p.has1 ? __builtin_amdgcn_readlane(st.vpid, j + 1) : p.pid0;
    return p;
  };
  // bf16: a position past the item's end loads, in every lane, the same one
  // of 16 distinct 16-byte words at the start of the item table (at least
  // 8 workgroups x 8 slots x 64 bytes; cached after its first use) instead
  // of K/V pages: the count of loads in flight stays fixed (the loop's
  // waits are static) without reading pages again and waiting for them
  // when the item ends (measured: 70B-shaped decode 918.6 -> 912 us,
  // two-level tree -1.6%, Llama-8B-shaped -2.5%).
  const uint8_t* idle_words = reinterpret_cast<const uint8_t*>(a.items);
  auto fetch = [&](const StepPos& p, Regs& r) {
    // A rows 0-7 come from page 0, rows 8-15 from page 1; a V lane reads
    // page grp / 2.
    const T* kq = kbase + (int64_t)(col < 8 ? p.pid0 : p.pid1) * page_stride;
    const T* vq = vbase + (int64_t)(grp < 2 ? p.pid0 : p.pid1) * page_stride;
    if constexpr (sizeof(T) == 2) {
      const bool live = p.valid;
      auto word = [&](const T* real, int k) {
        return live ? reinterpret_cast<const uint8_t*>(real) : idle_words + 16 * k;
      };
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        r.k[0][s] = __builtin_bit_cast(F, ld16<NT>(word(kq + ((4 * s + grp) * 16 + (col & 7)) * 8, 2 * s)));
        r.k[1][s] = __builtin_bit_cast(F, ld16<NT>(word(kq + ((4 * s + grp) * 16 + 8 + (col & 7)) * 8, 2 * s + 1)));
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) r.v[b] = __builtin_bit_cast(F, ld16<NT>(word(vq + v_off + b * 256, 2 * NS + b)));
    } else {
#pragma unroll
      for (int s = 0; s < NS; ++s) {
        r.k[0][s] = load_k8<NT>(kq, col & 7, 32 * s + 8 * grp);
        r.k[1][s] = load_k8<NT>(kq, 8 + (col & 7), 32 * s + 8 * grp);
      }
#pragma unroll
      for (int b = 0; b < NB; ++b) r.v[b] = load_v8<NT>(vq, v_off + b * 256);
    }
  };

  // Span cursor. The first span comes with the item and its record; a later
  // span's page ids are loaded when the walk reaches it, and waited for at
  // once: the wait then never has to be repeated on the loop's back edge,
  // where the compiler would otherwise drain every load in flight (the K/V
  // of the next step included) on each iteration.
  int si = 0;
  SpanState cur;
  cur.valid = it.n_spans > 0;
  cur.kb = it.s0_key_begin;
  cur.ke = it.s0_key_end;
  cur.causal = it.s0_causal;
  cur.vpid = vpid0;
  int gs = 0;      // index of the next step among the item's steps
  int sb = 0;      // index of cur's first step
  auto advance = [&]() {
    // position of the next step to issue, moving on to the span holding it
    while (cur.valid && gs >= sb + ((cur.ke - cur.kb + kKeysPerStep - 1) >> 5)) {
      sb += (cur.ke - cur.kb + kKeysPerStep - 1) >> 5;
      ++si;
      cur = load_span(si);
      wait_vmcnt<0>();
    }
    StepPos p = step_at(cur, cur.kb + (gs - sb) * kKeysPerStep);
    ++gs;
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
    // slot j = 4X + i holds key t0 + slot_key(grp, j)
    float sv[8];
    if (p.t0 + kKeysPerStep <= p.key_end && !p.causal) {
#pragma unroll
      for (int j = 0; j < 8; ++j) sv[j] = sacc[j >> 2][j & 3] * a.scale_log2;
    } else {
#pragma unroll
      for (int j = 0; j < 8; ++j) {
        const int key = p.t0 + slot_key(grp, j);
        const bool vis = key < p.key_end && (!p.causal || key <= row.qpos);
        sv[j] = vis ? sacc[j >> 2][j & 3] * a.scale_log2 : kNegInf;
      }
    }
    float mt = sv[0];
#pragma unroll
    for (int j = 1; j < 8; ++j) mt = fmaxf(mt, sv[j]);
    mt = rows_max(mt);
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
    for (int b = 0; b < NB; ++b) acc[b] *= alpha;
    if (p.t0 + kKeysPerStep <= p.key_end) {
#pragma unroll
      for (int b = 0; b < NB; ++b) acc[b] = mma(r.v[b], pf, acc[b]);
    } else {
      // Keys past the span end may be NaN page tails (or a repeated page):
      // zero V there, since P = 0 times NaN would still poison the sum.
      // The operand registers stay untouched (copies are masked), so the
      // register stages keep fixed registers across the loop.
#pragma unroll
      for (int b = 0; b < NB; ++b) {
        F vb = r.v[b];
#pragma unroll
        for (int j = 0; j < 8; ++j)
          if (p.t0 + slot_key(grp, j) >= p.key_end) vb[j] = (T)0.f;
        acc[b] = mma(vb, pf, acc[b]);
      }
    }
  };

  // P register stages rotate: while step s is computed, the next P - 1
  // steps are in flight. A position past the end loads idle words (bf16) or
  // re-fetches the current step's pages (fp32); in bounds, never used.
  Regs r[P];
  StepPos ps[P];
  ps[0] = advance();
  if (ps[0].valid) {
    fetch(ps[0], r[0]);
#pragma unroll
    for (int i = 1; i < P - 1; ++i) {
      ps[i] = advance();
      fetch(sizeof(T) == 2 ? ps[i] : pick(ps[i].valid, ps[i], ps[0]), r[i]);
    }
    bool done = false;
    while (!done) {
#pragma unroll
      for (int s = 0; s < P; ++s) {
        const int w = (s + P - 1) % P;
        ps[w] = advance();
        fetch(sizeof(T) == 2 ? ps[w] : pick(ps[w].valid, ps[w], ps[s]), r[w]);
        compute(ps[s], r[s]);
        if (!ps[(s + 1) % P].valid) {
          done = true;
          break;
        }
      }
    }
  }

  lsum = rows_sum(lsum);
  const bool has_row = col < it.n_rows;
  const float inv = lsum > 0.f ? 1.f / lsum : 0.f;
  const float lse2 = lsum > 0.f ? m + __log2f(lsum) : kNegInf;
  if (it.part_base >= 0) {
    if (has_row) {
      const int64_t prow = row.slot;
      TO* dst = static_cast<TO*>(a.part_o) + prow * D + 4 * grp;
#pragma unroll
      for (int b = 0; b < NB; ++b) store4_part(dst + 16 * b, acc[b] * inv);
      if (grp == 0) a.part_lse[prow] = lse2;
    }
  } else if (has_row) {
    TO* dst = static_cast<TO*>(a.o) + (int64_t)row.q_row * D + 4 * grp;
#pragma unroll
    for (int b = 0; b < NB; ++b) store4(dst + 16 * b, acc[b] * inv);
    if (grp == 0 && a.lse) a.lse[row.q_row] = lse2 == kNegInf ? kNegInf : lse2 * kLn2;
  }
}

// Waves per workgroup: 8 for bf16 (two per SIMD, so one wave's softmax
// overlaps another's MFMAs), 4 for fp32, whose operand registers allow only
// one wave per SIMD.
template <typename T> constexpr int block_waves() { return sizeof(T) == 2 ? 8 : 4; }

// Narrow workgroup `block` runs the items in its narrow_slots slots (dealt
// by the planner; n_rows = 0 marks an empty slot), one per wave; a wave of
// an empty slot runs through without loading a page or writing a row.
template <typename T, int D, typename TO>
__device__ __forceinline__ void narrow_block(const AttnArgs& a, int block) {
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  const int lane = threadIdx.x & 63;
  // one slot per wave (the host checks narrow_slots == block_waves<T>())
  const int64_t item_id = (int64_t)block * block_waves<T>() + wave;
  // The slot's item and lane record go out together (one round trip): no
  // branch waits for the item first. An empty slot (n_rows = 0, no spans)
  // runs through without loading a page or writing a row.
  const Item it = a.items[item_id];
  const ItemRec* rec = a.item_recs + item_id;
  const int col = lane & 15;
  const RecLane rl{rec->q_row[col], rec->aux[col], rec->page[lane & 31]};
  if (it.flags & kItemStream) run_item<T, D, TO, true, 2>(a, it, rl, lane);
  else run_item<T, D, TO, false, 2>(a, it, rl, lane);
}

// ---------------------------------------------------------------- wide items
// A wide item holds up to kWideWaves * 32 query rows of one kv head against
// a span list: a workgroup of kWideWaves waves, 32 rows per wave, all rows
// sharing the key stream. Used for the grouped prefix pass
// (many rows share one segment, §2 intra-batch prefix sharing) and for
// chunked prefill (§4.1).
//
// Loads. Each 32-key step's K and V (two pages) are read once per
// workgroup, by direct global-to-LDS loads into a ring of kWideStages step
// images, so no registers hold data in transit. A step image is
// 2 * D/32 + D/16 blocks of 1 KB (16 KB at d = 128); block k is written by
// one load instruction whose lane L fetches the 16 bytes that lane L of
// every wave later reads with one ds_read_b128 at L * 16, so every LDS read
// is sequential and conflict-free. With c = L % 32, h = L / 32:
//   K block s (dims 16s..16s+15):   page c / 16, key c % 16, unit 2s + h
//   V block (page g, dims 32b..+31): page g, dim 32b + c, slots 8h..8h+7
//
// Products use v_mfma_f32_32x32x16_bf16, the shape that reaches the bf16
// peak on gfx950 (measured 2.48 PFLOP/s, against 1.39 for 16x16x32):
//   S^T (32 keys x 32 rows) = K Q^T, 8 products over d = 128; lane (c, h)
//     holds row c, keys 8 (i / 4) + 4 h + i % 4 in register i;
//   O^T (32 dims x 32 rows) += V^T P^T per page of the step: the B operand of
//     page g is registers 8g..8g+7 of that lane, i.e. keys 8j/4 + 4h + j%4 of
//     page g, which the V slot order keeps in 16 contiguous bytes.
//
// Compute. Iteration t issues the MFMAs of P V for step t-1 and of Q K^T for
// step t+1, and meanwhile runs the softmax of step t on the VALU: the three
// are independent, so the matrix cores and the VALU overlap inside each
// wave (and the two waves of a SIMD fill each other's stalls).
//
// Softmax rescaling is lazy: a row's reference maximum only moves when a
// step's maximum exceeds it by more than kRescaleLog2 (so weights stay below
// 2^kRescaleLog2); the result is the same softmax, and the accumulator
// rescale runs only on the rare steps where some row moves.
constexpr float kRescaleLog2 = 8.f;
constexpr int kWideStages = 6;

// Bytes of the wide items' LDS ring: kWideStages step images of
// 2 * D/32 + D/16 blocks of 1 KB.
template <int D> constexpr int wide_ring_bytes() { return kWideStages * (D / 16 + 2 * (D / 32)) * 1024; }

template <int D, typename TO>
__device__ __forceinline__ void wide_item(const AttnArgs& a, int item_id, uint8_t* smem) {
  using T = __bf16;
  using F = bf16x8_t;
  constexpr int NK = D / 16;                      // 16-dim slices of Q K^T
  constexpr int NO = D / 32;                      // 32-dim output blocks
  constexpr int kBlocks = NK + 2 * NO;            // 1 KB blocks per step image
  constexpr int kStepBytes = kBlocks * 1024;
  static_assert(kBlocks % kWideWaves == 0, "step blocks must split evenly over the waves");
  constexpr int kLoadsPerWave = kBlocks / kWideWaves;
  constexpr int S = kWideStages;
  static_assert(S >= 5 && S % 2 == 0, "the ring needs >= 5 stages, an even count keeps tile parity static");
  constexpr int64_t kTile = 16 * D;
  static_assert(S * kStepBytes == wide_ring_bytes<D>(), "ring size");
  uint8_t (*lds)[kStepBytes] = reinterpret_cast<uint8_t (*)[kStepBytes]>(smem);

  const int wave = threadIdx.x >> 6;
  const int lane = threadIdx.x & 63;
  const int c = lane & 31;
  const int h = lane >> 5;
  const Item it = a.wide_items[item_id];
  // waves without rows still load their share of every step image
  const bool computes = wave * 32 < it.n_rows;

  // This lane's row: row c of this wave's block.
  const int r = wave * 32 + c;
  const Row row = r < it.n_rows ? a.rows[it.row_begin + r] : Row{-1, 0, -1, -1};
  F qf[NK];
  {
    const T* qp = static_cast<const T*>(a.q) + (int64_t)(row.q_row < 0 ? 0 : row.q_row) * D + 8 * h;
#pragma unroll
    for (int s = 0; s < NK; ++s) qf[s] = row.q_row >= 0 ? load8(qp + 16 * s) : zero_frag<F>();
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
    p.full = t_next + kKeysPerStep <= cur.ke && !cur.causal;
    p.pid0 = __builtin_amdgcn_readlane(cur.vpid, j);
    p.pid1 = p.has1 ? __builtin_amdgcn_readlane(cur.vpid, j + 1) : p.pid0;
    t_next += kKeysPerStep;
    return p;
  };

  // ---- loads: this wave writes blocks wave + kWideWaves * k of a step image.
  // Per lane: K or V, which page of the step, and the element offset inside
  // that page's tile. Page bases are computed on the scalar unit.
  int ld_off[kLoadsPerWave];
  bool ld_v[kLoadsPerWave], ld_p1[kLoadsPerWave];
#pragma unroll
  for (int k = 0; k < kLoadsPerWave; ++k) {
    const int blk = wave + kWideWaves * k;
    ld_v[k] = blk >= NK;
    if (!ld_v[k]) {
      ld_p1[k] = c >= 16;
      ld_off[k] = ((2 * blk + h) * 16 + (c & 15)) * 8;
    } else {
      const int g = (blk - NK) / NO, b = (blk - NK) % NO;
      ld_p1[k] = g == 1;
      ld_off[k] = (32 * b + c) * 16 + 8 * h;
    }
  }
  // Byte offsets of the step's two pages, forced onto the scalar unit (the
  // per-lane choice between them is then one select per half).
  auto uniform64 = [](int64_t x) {
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)x);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)((uint64_t)x >> 32));
    return (int64_t)(((uint64_t)hi << 32) | lo);
  };
  auto issue = [&](const StepPos& p, uint8_t* img) {
    const int64_t o0 = uniform64((int64_t)p.pid0 * page_stride);
    const int64_t o1 = uniform64((int64_t)p.pid1 * page_stride);
#pragma unroll
    for (int k = 0; k < kLoadsPerWave; ++k) {
      const T* base = (ld_v[k] ? vbase : kbase) + ld_off[k];
      __builtin_amdgcn_global_load_lds(base + (ld_p1[k] ? o1 : o0), img + (wave + kWideWaves * k) * 1024, 16, 0, 0);
    }
  };

  float m = kNegInf, lsum = 0.f;
  f32x16_t acc[NO];
#pragma unroll
  for (int b = 0; b < NO; ++b) acc[b] = f32x16_t{};

  // Key (within the step) of score register i of this lane.
  auto skey = [&](int i) { return 8 * (i >> 2) + 4 * h + (i & 3); };

  // Q K^T of one step (one accumulation chain over the 16-dim slices).
  auto qk = [&](const uint8_t* img, f32x16_t& sacc) {
    const uint8_t* rd = img + lane * 16;
    F kf[NK];
#pragma unroll
    for (int s = 0; s < NK; ++s) kf[s] = __builtin_bit_cast(F, *reinterpret_cast<const u32x4_t*>(rd + s * 1024));
    f32x16_t sn = f32x16_t{};
#pragma unroll
    for (int s = 0; s < NK; ++s) sn = mma32(kf[s], qf[s], sn);
    sacc = sn;
  };

  // P V of one step. Keys past the span end may be NaN page tails: their V
  // slots are zeroed (P = 0 times NaN would still poison the sum).
  auto read_v = [&](const uint8_t* img, F (&vf)[2][NO]) {
    const uint8_t* rd = img + lane * 16;
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int b = 0; b < NO; ++b)
        vf[g][b] = __builtin_bit_cast(F, *reinterpret_cast<const u32x4_t*>(rd + (NK + g * NO + b) * 1024));
  };
  auto mask_v = [&](const StepPos& p, F (&vf)[2][NO]) {
    if (p.t0 + kKeysPerStep > p.key_end) {
      const int lim = p.key_end - p.t0;
#pragma unroll
      for (int g = 0; g < 2; ++g)
#pragma unroll
        for (int b = 0; b < NO; ++b) {
          u32x4_t w = __builtin_bit_cast(u32x4_t, vf[g][b]);
#pragma unroll
          for (int q = 0; q < 4; ++q) {
            // 32-bit word q holds slots 2q, 2q+1 = registers 8g + 2q, 8g + 2q + 1
            const unsigned keep_lo = skey(8 * g + 2 * q) < lim ? 0xFFFFu : 0u;
            const unsigned keep_hi = skey(8 * g + 2 * q + 1) < lim ? 0xFFFF0000u : 0u;
            w[q] &= keep_lo | keep_hi;
          }
          vf[g][b] = __builtin_bit_cast(F, w);
        }
    }
  };
  auto pv = [&](const F (&vf)[2][NO], const F (&pf)[2]) {
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int b = 0; b < NO; ++b) acc[b] = mma32(vf[g][b], pf[g], acc[b]);
  };

  // Online softmax of one step's scores into P (bf16, RNE), one operand per
  // page of the step (registers 0-7: page 0, 8-15: page 1).
  auto softmax = [&](const StepPos& p, const f32x16_t& sacc, F (&pf)[2]) {
    // raw scores (masked ones -inf); the scale is applied inside the exponent
    // with one FMA (scale > 0, so it commutes with the max)
    float sv[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) sv[i] = sacc[i];
    if (p.t0 + kKeysPerStep > p.key_end || p.causal) {
      const int lim = (p.causal ? min(p.key_end, row.qpos + 1) : p.key_end) - p.t0;
#pragma unroll
      for (int i = 0; i < 16; ++i) sv[i] = skey(i) < lim ? sv[i] : kNegInf;
    }
    float mt = sv[0];
#pragma unroll
    for (int i = 1; i < 16; ++i) mt = fmaxf(mt, sv[i]);
    mt = halves_max(mt) * a.scale_log2;
    const bool move = mt > m + kRescaleLog2;
    if (__any(move)) {
      const float m_new = move ? mt : m;
      const float alpha = m == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m - m_new);
      lsum *= alpha;
#pragma unroll
      for (int b = 0; b < NO; ++b) acc[b] *= alpha;
      m = m_new;
    }
    const float m_use = m == kNegInf ? 0.f : m;
    float pr[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) pr[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sv[i], a.scale_log2, -m_use));
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 16; i += 4) ps += (pr[i] + pr[i + 1]) + (pr[i + 2] + pr[i + 3]);
    lsum += ps;
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      float half[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) half[j] = pr[8 * g + j];
      pf[g] = to_frag(half, (F*)nullptr);
    }
  };

  // One iteration on full, unmasked steps as a single basic block: the 16
  // MFMAs (P V of step t-1, Q K^T of step t+1) are interleaved with the
  // softmax VALU work of step t, so a wave keeps issuing independent VALU
  // instructions while each MFMA runs. V of step t-1 arrives in registers
  // (read during the previous iteration); the K reads of step t+1 go out
  // first and arrive behind the P V products, and the V reads of step t,
  // for the next iteration, go out behind the Q K^T products. The
  // accumulator rescale, which must wait for the P V products, is returned
  // (alpha) and applied afterwards.
  auto fast_iter = [&](F (&vf)[2][NO], const uint8_t* img_qk, const uint8_t* img_v, const F (&pf_prev)[2],
                       const f32x16_t& sacc_cur, f32x16_t& sacc_nxt, F (&pf_cur)[2], float& alpha) {
    const uint8_t* rk = img_qk + lane * 16;
    F kf[NK];
#pragma unroll
    for (int s = 0; s < NK; ++s) kf[s] = __builtin_bit_cast(F, *reinterpret_cast<const u32x4_t*>(rk + s * 1024));
#pragma unroll
    for (int g = 0; g < 2; ++g)
#pragma unroll
      for (int b = 0; b < NO; ++b) acc[b] = mma32(vf[g][b], pf_prev[g], acc[b]);
    f32x16_t sn = f32x16_t{};
#pragma unroll
    for (int s = 0; s < NK; ++s) sn = mma32(kf[s], qf[s], sn);
    read_v(img_v, vf);
    // softmax of step t (no masks: full step); the max as a tree of
    // three-input maxima (v_max3_f32, 8 instructions for 16 scores)
    auto max3 = [](float x, float y, float z) { return fmaxf(fmaxf(x, y), z); };
    const float m0 = max3(sacc_cur[0], sacc_cur[1], sacc_cur[2]);
    const float m1 = max3(sacc_cur[3], sacc_cur[4], sacc_cur[5]);
    const float m2 = max3(sacc_cur[6], sacc_cur[7], sacc_cur[8]);
    const float m3 = max3(sacc_cur[9], sacc_cur[10], sacc_cur[11]);
    const float m4 = max3(sacc_cur[12], sacc_cur[13], sacc_cur[14]);
    float mt = fmaxf(max3(m0, m1, m2), max3(m3, m4, sacc_cur[15]));
    mt = halves_max(mt) * a.scale_log2;
    const bool move = mt > m + kRescaleLog2;
    const float m_new = move ? mt : m;
    alpha = m == kNegInf ? 0.f : __builtin_amdgcn_exp2f(m - m_new);
    m = m_new;
    const float m_use = m == kNegInf ? 0.f : m;
    float pr[16];
#pragma unroll
    for (int i = 0; i < 16; ++i) pr[i] = __builtin_amdgcn_exp2f(__builtin_fmaf(sacc_cur[i], a.scale_log2, -m_use));
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      float half[8];
#pragma unroll
      for (int j = 0; j < 8; ++j) half[j] = pr[8 * g + j];
      pf_cur[g] = to_frag(half, (F*)nullptr);
    }
    float ps = 0.f;
#pragma unroll
    for (int i = 0; i < 16; i += 4) ps += (pr[i] + pr[i + 1]) + (pr[i + 2] + pr[i + 3]);
    lsum = __builtin_fmaf(lsum, alpha, ps);
    sacc_nxt = sn;
    // keep the softmax results in this block (they are consumed only after
    // the next barrier, and would otherwise sink below the rescale branch)
#pragma unroll
    for (int g = 0; g < 2; ++g) {
      const u32x4_t w = __builtin_bit_cast(u32x4_t, pf_cur[g]);
      asm volatile("" ::"v"(w[0]), "v"(w[1]), "v"(w[2]), "v"(w[3]));
    }
    asm volatile("" ::"v"(lsum));
    // schedule: the K reads, the P V MFMAs, then the Q K^T MFMAs with the V
    // reads of step t after the first of them; each MFMA followed by VALU
    // work
    __builtin_amdgcn_sched_group_barrier(0x100, NK, 0);
#pragma unroll
    for (int k = 0; k < 2 * NO + 1; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
    }
    __builtin_amdgcn_sched_group_barrier(0x100, 2 * NO, 0);
#pragma unroll
    for (int k = 0; k < NK - 1; ++k) {
      __builtin_amdgcn_sched_group_barrier(0x008, 1, 0);
      __builtin_amdgcn_sched_group_barrier(0x002, 5, 0);
    }
  };

  // ---- pipeline. Step t lives in stage t % S. Iteration t:
  //   wait for this wave's loads of step t+1 (steps t+2..t+S-2 may still be
  //   in flight) and retire its LDS reads (lgkmcnt 0); barrier: step t+1 is
  //   visible to every wave, and step t-1's stage is free (its K was read in
  //   iteration t-2, its V in iteration t-1); issue step t+S-1 into it;
  //   MFMA: P V of step t-1 (V already in registers), Q K^T of step t+1;
  //   VALU: softmax of step t; LDS: K of step t+1, V of step t.
  // Score and probability tiles alternate by step parity (S is even, so the
  // parity of each unrolled position is fixed). Positions past the end
  // re-load the current step's pages (in bounds, never read) so the count of
  // loads in flight stays fixed.
  StepPos ps[S];
  ps[0] = advance();
  if (ps[0].valid) {
#pragma unroll
    for (int i = 0; i < S - 1; ++i) {
      if (i > 0) ps[i] = advance();
      issue(pick(ps[i].valid, ps[i], ps[0]), lds[i]);
    }
    f32x16_t sacc[2];
    F pf[2][2];
    F vf[2][NO];
    wait_vmcnt<(S - 3) * kLoadsPerWave>();
    __builtin_amdgcn_s_barrier();
    asm volatile("" ::: "memory");
    if (computes) qk(lds[0], sacc[0]);
    bool first = true, done = false;
    while (!done) {
#pragma unroll
      for (int st = 0; st < S; ++st) {
        const int cur_p = st & 1, nxt_p = cur_p ^ 1;
        const int nx = (st + 1) % S, pv_st = (st + S - 1) % S;
        wait_vmcnt<(S - 3) * kLoadsPerWave>();
        wait_lgkmcnt0();
        __builtin_amdgcn_s_barrier();
        asm volatile("" ::: "memory");
        const StepPos prev = ps[pv_st];   // step t-1, whose V is in vf
        ps[pv_st] = advance();
        issue(pick(ps[pv_st].valid, ps[pv_st], ps[st]), lds[pv_st]);
        const bool more = ps[nx].valid;
        const bool fast = !first && more && ps[st].full && prev.full;
        if (computes && fast) {
          float alpha;
          fast_iter(vf, lds[nx], lds[st], pf[nxt_p], sacc[cur_p], sacc[nxt_p], pf[cur_p], alpha);
          if (__any(alpha != 1.f)) {
#pragma unroll
            for (int b = 0; b < NO; ++b) acc[b] *= alpha;
          }
        } else if (computes) {
          if (!first) {
            mask_v(prev, vf);
            pv(vf, pf[nxt_p]);
          }
          if (more) qk(lds[nx], sacc[nxt_p]);
          softmax(ps[st], sacc[cur_p], pf[cur_p]);
          read_v(lds[st], vf);
          if (!more) {
            mask_v(ps[st], vf);
            pv(vf, pf[cur_p]);
          }
        }
        first = false;
        if (!more) {
          done = true;
          break;
        }
      }
    }
  }
  // drain the loads still in flight before the workgroup's LDS is released
  wait_vmcnt<0>();

  // ---- epilogue: lane (c, h) holds dims 32b + 8(i/4) + 4h + i%4 of row c
  const float l = halves_sum(lsum);
  if (computes && r < it.n_rows) {
    const float inv = l > 0.f ? 1.f / l : 0.f;
    const float lse2 = l > 0.f ? m + __log2f(l) : kNegInf;
    if (it.part_base >= 0) {
      const int64_t prow = row.slot;
      TO* dst = static_cast<TO*>(a.part_o) + prow * D + 4 * h;
#pragma unroll
      for (int b = 0; b < NO; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          store4_part(dst + 32 * b + 8 * q, f32x4_t{acc[b][4 * q], acc[b][4 * q + 1], acc[b][4 * q + 2], acc[b][4 * q + 3]} * inv);
      if (h == 0) a.part_lse[prow] = lse2;
    } else {
      TO* dst = static_cast<TO*>(a.o) + (int64_t)row.q_row * D + 4 * h;
#pragma unroll
      for (int b = 0; b < NO; ++b)
#pragma unroll
        for (int q = 0; q < 4; ++q)
          store4(dst + 32 * b + 8 * q, f32x4_t{acc[b][4 * q], acc[b][4 * q + 1], acc[b][4 * q + 2], acc[b][4 * q + 3]} * inv);
      if (h == 0 && a.lse) a.lse[row.q_row] = lse2 == kNegInf ? kNegInf : lse2 * kLn2;
    }
  }
}

// ---------------------------------------------------------------- launch
// One launch runs both roles: wide workgroups (MFMA/LDS-bound grouped
// prefix or prefill work) and narrow ones (lists of one-wave items, mostly
// HBM-bound suffix streaming), so the two kinds of work overlap on the GPU.
// RB = 0: no wide role.
// The grid is dealt in rounds of 8 blocks (one per XCD); the wide rounds
// are spread evenly over the first wide_span rounds, so CUs mix MFMA-heavy
// wide blocks with HBM-heavy narrow ones, and the launch ends on narrow
// blocks (dealt longest first, so its tail is short ones). Within a role
// the block index modulo 8 still names the XCD (xcd_remap, and the
// planner's dealing of narrow items to XCDs, rely on it).
template <typename T, int D, typename TO, int RB>
__global__ __launch_bounds__(64 * block_waves<T>())
__attribute__((amdgpu_waves_per_eu(block_waves<T>() / 4)))
void attn_kernel(AttnArgs a) {
  static_assert(RB == 0 || block_waves<T>() == kWideWaves, "wide items need kWideWaves-wave blocks");
  // the wide role's LDS ring (narrow items use no LDS)
  constexpr int kSmem = RB > 0 ? wide_ring_bytes<D>() : 16;
  __shared__ __attribute__((aligned(1024))) uint8_t smem[kSmem];
  const int b = blockIdx.x;
  const int x = b & 7, r = b >> 3;
  if constexpr (RB > 0) {
    // in cycles of kSeCycle rounds, whole cycles wide or narrow
    const int ws = a.wide_blocks / (8 * kSeCycle);
    const int sp = a.wide_span;
    const int cyc = r / kSeCycle, q = r % kSeCycle;
    const int w_before = cyc < sp ? (int)((int64_t)cyc * ws / sp) : ws;
    const int w_upto = cyc < sp ? (int)((int64_t)(cyc + 1) * ws / sp) : ws;
    if (w_upto > w_before) {
      const int item = xcd_remap((w_before * kSeCycle + q) * 8 + x, a.wide_group);
      if (item < a.n_wide) wide_item<D, TO>(a, item, smem);
      return;
    }
    narrow_block<T, D, TO>(a, ((cyc - w_upto) * kSeCycle + q) * 8 + x);
  } else {
    (void)smem;
    narrow_block<T, D, TO>(a, b);
  }
}

// ---------------------------------------------------------------- merge

// E partial elements (16 bytes) from their raw bits: 4 fp32, or 8 bf16
// (each the upper half of an fp32). Vector elements go through
// __uint_as_float: hipcc's __builtin_bit_cast of a vector element reads
// element 0 whatever the index.
template <typename TO, int E>
__device__ __forceinline__ void unpack16(u32x4_t x, float (&v)[E]) {
  if constexpr (sizeof(TO) == 4) {
#pragma unroll
    for (int j = 0; j < 4; ++j) v[j] = __uint_as_float(x[j]);
  } else {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
      v[2 * j] = __uint_as_float(x[j] << 16);
      v[2 * j + 1] = __uint_as_float(x[j] & 0xffff0000u);
    }
  }
}
template <typename TO, int E>
__device__ __forceinline__ void store16(TO* dst, const float (&v)[E]) {
  if constexpr (sizeof(TO) == 4) {
    *reinterpret_cast<float4*>(dst) = make_float4(v[0], v[1], v[2], v[3]);
  } else {
    typedef __bf16 bf16x8v_t __attribute__((ext_vector_type(8)));
    bf16x8v_t r;
#pragma unroll
    for (int j = 0; j < 8; ++j) r[j] = (__bf16)v[j];
    *reinterpret_cast<u32x4_t*>(dst) = __builtin_bit_cast(u32x4_t, r);
  }
}

struct MergeArgs {
  const void* part_o;     // in the output element type
  const float* part_lse;
  const int32_t* merge_rows;
  const int32_t* merge_indptr;
  const int32_t* merge_parts;
  void* o;
  float* lse;
  int32_t n_merge;
  int32_t k0;   // partials of entry r at slots k * n_merge + r for k < k0
};

// Rows per merge workgroup (256 threads, 16 bytes of a row per thread).
template <int D, typename TO> constexpr int merge_rows_per_block() { return 256 / (D * (int)sizeof(TO) / 16); }

// Output rows whose keys were split over several items. Partials hold the
// normalized o_i and lse_i (log2) of disjoint key sets:
//   M = max_i lse_i,  w_i = 2^(lse_i - M),  O = sum w_i o_i / sum w_i,
//   LSE = (M + log2 sum w_i) * ln 2
// which is exact in real arithmetic (shared == unshared, §3 "Scope").
// Merge entry r has merge_indptr[r + 1] - merge_indptr[r] partials; its
// first k0 sit at slots k * n_merge + r, so they are loaded together with
// the entry's metadata (one round trip); slots past the entry's count are
// read too (in bounds: the workspace holds k0 * n_merge of them) and dropped
// by integer selects, which fast math cannot fold away whatever bits they
// hold. Further partials (entries with more than k0) come from the slot
// list merge_parts. One group of threads per row, 16 bytes of each partial
// (8 bf16 or 4 fp32 dims) per thread.
template <int D, typename TO>
__global__ __launch_bounds__(256) __attribute__((amdgpu_waves_per_eu(6))) void merge_kernel(MergeArgs a) {
  constexpr int E = 16 / (int)sizeof(TO);
  constexpr int TPR = D / E;
  constexpr int RPB = 256 / TPR;
  static_assert(RPB == merge_rows_per_block<D, TO>(), "rows per block");
  constexpr int kBatch = kMergeK0;
  const int r = blockIdx.x * RPB + threadIdx.x / TPR;
  const int t = threadIdx.x % TPR;
  if (r >= a.n_merge) return;
  const TO* part_o = static_cast<const TO*>(a.part_o);
  const int q_row = a.merge_rows[r];
  const int p0 = a.merge_indptr[r], p1 = a.merge_indptr[r + 1];
  uint32_t lb[kBatch];
  u32x4_t vb[kBatch];
#pragma unroll
  for (int k = 0; k < kBatch; ++k) {
    if (k < a.k0) {
      const int64_t slot = (int64_t)k * a.n_merge + r;
      lb[k] = __builtin_bit_cast(uint32_t, a.part_lse[slot]);
      vb[k] = *reinterpret_cast<const u32x4_t*>(part_o + slot * D + E * t);
    } else {
      lb[k] = 0;
      vb[k] = u32x4_t{0u, 0u, 0u, 0u};
    }
  }
  float mx = kNegInf;
  float acc[E];
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] = 0.f;
  float wsum = 0.f;
  // online over batches of parts: rescale when the running max moves
  auto fold = [&](const float (&l)[kBatch], const u32x4_t (&raw)[kBatch]) {
    float bm = kNegInf;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) bm = fmaxf(bm, l[k]);
    const float m_new = fmaxf(mx, bm);
    if (m_new == kNegInf) return;
    const float alpha = mx == kNegInf ? 0.f : __builtin_amdgcn_exp2f(mx - m_new);
#pragma unroll
    for (int e = 0; e < E; ++e) acc[e] *= alpha;
    wsum *= alpha;
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const float w = __builtin_amdgcn_exp2f(l[k] - m_new);   // 0 for absent parts
      float v[E];
      unpack16<TO, E>(raw[k], v);
      wsum += w;
#pragma unroll
      for (int e = 0; e < E; ++e) acc[e] = __builtin_fmaf(w, v[e], acc[e]);
    }
    mx = m_new;
  };
  {
    const int n = p1 - p0;
    const uint32_t neg_inf_bits = 0xff800000u;
    float l[kBatch];
    u32x4_t raw[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) {
      const bool keep = k < n && k < a.k0;
      l[k] = __builtin_bit_cast(float, keep ? lb[k] : neg_inf_bits);
      const uint32_t m = keep ? 0xffffffffu : 0u;
      raw[k] = vb[k] & u32x4_t{m, m, m, m};
    }
    fold(l, raw);
  }
  for (int pb = p0 + a.k0; pb < p1; pb += kBatch) {
    int pid[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) pid[k] = pb + k < p1 ? a.merge_parts[pb + k] : -1;
    float l[kBatch];
    u32x4_t raw[kBatch];
#pragma unroll
    for (int k = 0; k < kBatch; ++k) l[k] = pid[k] >= 0 ? a.part_lse[pid[k]] : kNegInf;
#pragma unroll
    for (int k = 0; k < kBatch; ++k)
      raw[k] = pid[k] >= 0 ? *reinterpret_cast<const u32x4_t*>(part_o + (int64_t)pid[k] * D + E * t)
                           : u32x4_t{0u, 0u, 0u, 0u};
    fold(l, raw);
  }
  const float inv = wsum > 0.f ? 1.f / wsum : 0.f;
#pragma unroll
  for (int e = 0; e < E; ++e) acc[e] *= inv;
  store16<TO, E>(static_cast<TO*>(a.o) + (int64_t)q_row * D + E * t, acc);
  if (t == 0 && a.lse) a.lse[q_row] = wsum > 0.f ? (mx + __log2f(wsum)) * kLn2 : kNegInf;
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

// Share (percent) of the narrow rounds interleaved with the wide ones; the
// rest run after the last wide round.
constexpr int kWideSpanNarrowPct = 80;

int lcm_int(int a, int b) {
  int x = a, y = b;
  while (y) {
    const int t = x % y;
    x = y;
    y = t;
  }
  return a / x * b;
}

template <typename T, int D, typename TO>
void launch_attention(AttnArgs args, const MergeArgs& margs, int wide_rb, hipStream_t stream) {
  const int rb = sizeof(T) == 2 ? wide_rb : 0;
  // whole dispatch cycles of wide rounds, each a multiple of wide_group rounds
  args.wide_blocks =
      (rb > 0 && args.n_wide > 0) ? pad_to(args.n_wide, 8 * lcm_int(args.wide_group, kSeCycle)) : 0;
  {
    const int ws = args.wide_blocks / (8 * kSeCycle), ns = args.narrow_blocks / (8 * kSeCycle);
    args.wide_span = ws + (int)((int64_t)ns * kWideSpanNarrowPct / 100);
  }
  constexpr int W = block_waves<T>();
  const int grid = args.wide_blocks + args.narrow_blocks;
  if (grid > 0) {
    if constexpr (sizeof(T) == 2) {
      if (rb > 0)
        hipLaunchKernelGGL((attn_kernel<T, D, TO, 1>), dim3(grid), dim3(64 * W), 0, stream, args);
      else
        hipLaunchKernelGGL((attn_kernel<T, D, TO, 0>), dim3(grid), dim3(64 * W), 0, stream, args);
    } else {
      hipLaunchKernelGGL((attn_kernel<T, D, TO, 0>), dim3(grid), dim3(64 * W), 0, stream, args);
    }
  }
  if (margs.n_merge > 0) {
    constexpr int rpb = merge_rows_per_block<D, TO>();
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
  // partial O rows in the output element type, then their LSEs
  void* part_o = workspace;
  const size_t part_elem = p.out_dtype == HALO_F32 ? 4 : 2;
  float* part_lse = plan->n_part_slots
                        ? reinterpret_cast<float*>(static_cast<uint8_t*>(workspace) +
                                                   align256((size_t)plan->n_part_slots * D * part_elem))
                        : nullptr;
  AttnArgs args{q, k_pool, v_pool, o, lse, part_o, part_lse,
                reinterpret_cast<const int32_t*>(m + L.seg_page_off),
                reinterpret_cast<const int32_t*>(m + L.seg_len),
                reinterpret_cast<const int32_t*>(m + L.page_ids),
                reinterpret_cast<const Item*>(m + L.items),
                reinterpret_cast<const ItemRec*>(m + L.item_recs),
                reinterpret_cast<const Item*>(m + L.wide_items),
                reinterpret_cast<const Span*>(m + L.spans),
                reinterpret_cast<const Row*>(m + L.rows),
                plan->n_items, plan->n_wide, 0, plan->n_narrow_blocks, plan->narrow_slots,
                plan->wide_group, 0,
                p.num_kv_heads, p.sm_scale * kLog2e};
  MergeArgs margs{part_o, part_lse,
                  reinterpret_cast<const int32_t*>(m + L.merge_rows),
                  reinterpret_cast<const int32_t*>(m + L.merge_indptr),
                  reinterpret_cast<const int32_t*>(m + L.merge_parts),
                  o, lse, plan->n_merge, plan->merge_k0};
  if (plan->n_narrow_blocks > 0 &&
      plan->narrow_slots != (p.kv_dtype == HALO_BF16 ? block_waves<__bf16>() : block_waves<float>()))
    return fail(HALO_ERR_INVALID_ARGUMENT, "internal: narrow slots per workgroup differ from its waves");
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

namespace {
halo_status_t upload_bytes(void* dst, const void* src, size_t n, hipStream_t stream) {
  hipError_t e = hipMemcpyAsync(dst, src, n, hipMemcpyHostToDevice, stream);
  if (e != hipSuccess) return fail(HALO_ERR_HIP, std::string("hipMemcpyAsync: ") + hipGetErrorString(e));
  return HALO_OK;
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
  return upload_bytes(device_meta, plan->meta.data(), plan->layout.total, static_cast<hipStream_t>(stream));
}

extern "C" halo_status_t halo_plan_upload_update(const halo_plan_t* plan, void* device_meta,
                                                 size_t device_meta_bytes, void* stream) {
  clear_error();
  if (!plan || !device_meta) return fail(HALO_ERR_INVALID_ARGUMENT, "plan and device_meta must not be NULL");
  if (device_meta_bytes < plan->layout.total)
    return fail(HALO_ERR_INVALID_ARGUMENT, "device_meta needs " + std::to_string(plan->layout.total) + " bytes");
  if ((reinterpret_cast<uintptr_t>(device_meta) & 255) != 0)
    return fail(HALO_ERR_INVALID_ARGUMENT, "device_meta must be 256-byte aligned");
  // The sections an in-place update rewrites lie between the segment
  // length table and the row table, in that order in the image.
  const size_t at = plan->layout.seg_len, end = plan->layout.rows;
  return upload_bytes(static_cast<uint8_t*>(device_meta) + at, plan->meta.data() + at, end - at,
                      static_cast<hipStream_t>(stream));
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

// ---------------------------------------------------------------- no-alloc decode
// Partial-result scratch of halo_prefix_attn_decode_noalloc: device memory of
// the library's own, one copy per GPU, held until the process ends. In host
// code `scratch` names a host-side stand-in, never a device address: the
// device address of each GPU's copy comes from hipGetSymbolAddress, looked up
// once per device and kept in g_scratch_ptr.
static __device__ __align__(256) uint8_t scratch[HALO_NOALLOC_SCRATCH_BYTES];

namespace {
constexpr int kMaxDevices = 64;
std::atomic<void*> g_scratch_ptr[kMaxDevices];
std::mutex g_scratch_mu;

// The device address of the current device's scratch array (looked up on the
// first call on each device, with that device current).
halo_status_t scratch_of_current_device(void** out) {
  int dev = -1;
  hipError_t e = hipGetDevice(&dev);
  if (e != hipSuccess) return fail(HALO_ERR_HIP, std::string("hipGetDevice: ") + hipGetErrorString(e));
  if (dev < 0 || dev >= kMaxDevices)
    return fail(HALO_ERR_UNSUPPORTED, "device index " + std::to_string(dev) + " beyond the scratch table");
  void* p = g_scratch_ptr[dev].load(std::memory_order_acquire);
  if (!p) {
    std::lock_guard<std::mutex> lock(g_scratch_mu);
    p = g_scratch_ptr[dev].load(std::memory_order_relaxed);
    if (!p) {
      e = hipGetSymbolAddress(&p, HIP_SYMBOL(scratch));
      if (e != hipSuccess || !p)
        return fail(HALO_ERR_HIP, std::string("hipGetSymbolAddress(scratch): ") + hipGetErrorString(e));
      g_scratch_ptr[dev].store(p, std::memory_order_release);
    }
  }
  *out = p;
  return HALO_OK;
}
}  // namespace

extern "C" halo_status_t halo_prefix_attn_decode_noalloc(const halo_plan_t* plan, const void* device_meta,
                                                         const void* q, const void* k_pool,
                                                         const void* v_pool, void* o, float* lse,
                                                         void* stream) {
  clear_error();
  if (!plan) return fail(HALO_ERR_INVALID_ARGUMENT, "plan must not be NULL");
  if (plan->workspace_bytes > HALO_NOALLOC_SCRATCH_BYTES)
    return fail(HALO_ERR_WORKSPACE_TOO_SMALL,
                "the plan needs " + std::to_string(plan->workspace_bytes) + " bytes of workspace; the no-alloc "
                "entry point holds " + std::to_string((size_t)HALO_NOALLOC_SCRATCH_BYTES));
  void* ws = nullptr;
  if (plan->workspace_bytes > 0) {
    halo_status_t st = scratch_of_current_device(&ws);
    if (st != HALO_OK) return st;
  }
  return run_attention(plan, false, device_meta, q, k_pool, v_pool, o, lse, ws,
                       ws ? (size_t)HALO_NOALLOC_SCRATCH_BYTES : 0, stream);
}
