// Context microbenchmarks for the attention kernels' rooflines on gfx950
// (measurement only; no part of the attention path calls them):
//  * stream_read_kernel: a wave reads random 4 KB tiles of a page pool the
//    way the suffix pass reads K/V pages -- 16-byte loads, 1 KB per wave
//    instruction, 16 KB per step, `stages` steps of registers per wave --
//    with plain or non-temporal loads. It gives the HBM read rate reachable
//    for that access pattern at a given number of waves and bytes in flight.
//  * mfma_kernel: back-to-back independent bf16 MFMAs (32x32x16 or
//    16x16x32), the dense matrix-core rate.
//  * exp_kernel: independent v_exp_f32 chains, optionally one MFMA per
//    `valu_per_mfma` of them on the same wave, to measure the transcendental
//    rate and how much VALU work hides behind the matrix cores.
//  * overlap_kernel: MFMA and VALU work on one SIMD, either interleaved in
//    each wave or split between the two waves of the SIMD.

#include <hip/hip_runtime.h>

#include <string>

#include "halo_probe.h"

namespace {

typedef unsigned int u32x4_t __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8_t __attribute__((ext_vector_type(8)));
typedef float f32x4_t __attribute__((ext_vector_type(4)));
typedef float f32x16_t __attribute__((ext_vector_type(16)));

thread_local std::string g_err;

int fail(int st, const std::string& msg) {
  g_err = msg;
  return st;
}

template <bool NT>
__device__ __forceinline__ u32x4_t ld16(const void* p) {
  if constexpr (NT) return __builtin_nontemporal_load(reinterpret_cast<const u32x4_t*>(p));
  else return *reinterpret_cast<const u32x4_t*>(p);
}

// One step = 4 tiles of 4 KB = 16 loads of 16 bytes per lane.
constexpr int kTilesPerStep = 4;
constexpr int kLoadsPerStep = 16;

struct StreamArgs {
  const uint8_t* pool;
  int64_t pool_tiles;     // 4 KB tiles in pool (tile ids are clamped to it)
  const int32_t* tiles;   // tile indices (4 KB units of pool)
  int64_t n_steps;        // steps in the whole stream (n_tiles / 4)
  int32_t steps_per_item; // consecutive steps one wave reads before jumping
  uint32_t* out;          // one word per wave (keeps the loads alive)
};

// Waves take items (runs of steps_per_item steps) round-robin over the grid
// and keep `S` steps of loads in registers: while step s is consumed, steps
// s+1 .. s+S-1 are in flight, across item boundaries too.
template <int S, bool NT, int WAVES>
__global__ __launch_bounds__(64 * WAVES) void stream_read_kernel(StreamArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * WAVES + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * WAVES;
  const int64_t n_items = a.n_steps / a.steps_per_item;
  const int64_t my_items = wave < n_items ? (n_items - 1 - wave) / waves + 1 : 0;
  const int64_t my_steps = my_items * a.steps_per_item;
  // global step of this wave's k-th step
  auto step_of = [&](int64_t k) {
    const int64_t item = wave + (k / a.steps_per_item) * waves;
    return item * a.steps_per_item + k % a.steps_per_item;
  };
  auto issue = [&](int64_t k, u32x4_t (&r)[kLoadsPerStep]) {
    const int64_t st = step_of(k < my_steps ? k : 0);
#pragma unroll
    for (int t = 0; t < kTilesPerStep; ++t) {
      const int64_t tile = min((int64_t)(uint32_t)a.tiles[st * kTilesPerStep + t], a.pool_tiles - 1);
      const uint8_t* base = a.pool + tile * 4096 + lane * 16;
#pragma unroll
      for (int j = 0; j < 4; ++j) r[t * 4 + j] = ld16<NT>(base + j * 1024);
    }
  };
  u32x4_t acc = {0u, 0u, 0u, 0u};
  if (my_steps > 0) {
    u32x4_t r[S][kLoadsPerStep];
#pragma unroll
    for (int i = 0; i < S - 1; ++i) issue(i, r[i]);
    for (int64_t k = 0; k < my_steps; k += S) {
#pragma unroll
      for (int s = 0; s < S; ++s) {
        issue(k + s + S - 1, r[(s + S - 1) % S]);
        if (k + s < my_steps) {
#pragma unroll
          for (int j = 0; j < kLoadsPerStep; ++j) acc ^= r[s][j];
        }
      }
    }
  }
  const uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3];
  if (lane == 0) a.out[wave] = x;
}

// The same reads cut into independent items, as a work-item kernel issues
// them: an item starts with a dependent metadata load (its first tile id),
// fills its own 2-step pipeline, and drains it before the next item starts.
// With COMPUTE, each step also runs 16 v_mfma_f32_16x16x32_bf16 and a
// short softmax-like VALU sequence on the loaded words (the suffix pass's
// per-step work at 8 query rows).
template <bool NT, bool COMPUTE, bool KV>
__global__ __launch_bounds__(512) void stream_items_kernel(StreamArgs a) {
  const int lane = threadIdx.x & 63;
  const int64_t wave = (int64_t)blockIdx.x * 8 + (threadIdx.x >> 6);
  const int64_t waves = (int64_t)gridDim.x * 8;
  const int64_t n_items = a.n_steps / a.steps_per_item;
  u32x4_t acc = {0u, 0u, 0u, 0u};
  f32x4_t macc = {0.f, 0.f, 0.f, 0.f};
  const int col = lane & 15, grp = lane >> 4;
  auto issue = [&](int64_t st, u32x4_t (&r)[kLoadsPerStep]) {
    if constexpr (KV) {
      // the suffix pass's pattern: tiles 0, 1 are the step's two K pages
      // ([16 units][16 tokens][16 B]; lane (col, grp) reads token col % 8 (+8
      // in the second half) of unit 4 s + grp of page col / 8), tiles 2, 3
      // its two V pages (dim-major; lane reads 16 B of dim row 16 b + col,
      // half grp % 2, of page grp / 2)
      int64_t tl[4];
#pragma unroll
      for (int t = 0; t < 4; ++t) tl[t] = min((int64_t)(uint32_t)a.tiles[st * kTilesPerStep + t], a.pool_tiles - 1);
      const uint8_t* kp = a.pool + (col < 8 ? tl[0] : tl[1]) * 4096;
      const uint8_t* vp = a.pool + (grp < 2 ? tl[2] : tl[3]) * 4096;
#pragma unroll
      for (int s4 = 0; s4 < 4; ++s4)
#pragma unroll
        for (int x = 0; x < 2; ++x)
          r[s4 * 2 + x] = ld16<NT>(kp + ((4 * s4 + grp) * 16 + (col & 7) + 8 * x) * 16);
#pragma unroll
      for (int b = 0; b < 8; ++b) r[8 + b] = ld16<NT>(vp + (b * 16 + col) * 32 + 16 * (grp & 1));
    } else {
#pragma unroll
      for (int t = 0; t < kTilesPerStep; ++t) {
        const int64_t tile = min((int64_t)(uint32_t)a.tiles[st * kTilesPerStep + t], a.pool_tiles - 1);
        const uint8_t* base = a.pool + tile * 4096 + lane * 16;
#pragma unroll
        for (int j = 0; j < 4; ++j) r[t * 4 + j] = ld16<NT>(base + j * 1024);
      }
    }
  };
  for (int64_t item = wave; item < n_items; item += waves) {
    // metadata round trip: the item's first step index comes from memory
    const int64_t first = item * a.steps_per_item;
    const int32_t hdr = __builtin_amdgcn_readfirstlane(a.tiles[first * kTilesPerStep] >= 0 ? 0 : 1);
    const int64_t s0 = first + hdr;
    u32x4_t r[2][kLoadsPerStep];
    issue(s0, r[0]);
    for (int k = 0; k < a.steps_per_item; k += 2) {
#pragma unroll
      for (int s = 0; s < 2; ++s) {
        if (k + s + 1 < a.steps_per_item) issue(s0 + k + s + 1, r[(s + 1) & 1]);
        if (k + s < a.steps_per_item) {
          if constexpr (COMPUTE) {
            bf16x8_t x = __builtin_bit_cast(bf16x8_t, r[s][0] ^ r[s][1]);
#pragma unroll
            for (int j = 0; j < 16; ++j)
              macc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8_t, r[s][j]), x, macc, 0, 0, 0);
            float m = fmaxf(fmaxf(macc[0], macc[1]), fmaxf(macc[2], macc[3]));
            m = fmaxf(m, __shfl_xor(m, 16));
            m = fmaxf(m, __shfl_xor(m, 32));
            macc = macc * __builtin_amdgcn_exp2f(-m * 1e-3f);
          } else {
#pragma unroll
            for (int j = 0; j < kLoadsPerStep; ++j) acc ^= r[s][j];
          }
        }
      }
    }
    __builtin_amdgcn_s_waitcnt(0);   // drain: the next item starts from scratch
  }
  const uint32_t x = acc[0] ^ acc[1] ^ acc[2] ^ acc[3] ^ __float_as_uint(macc[0] + macc[3]);
  if (lane == 0) a.out[wave] = x;
}

template <int S, bool NT>
int launch_stream(const StreamArgs& a, int waves_per_simd, int blocks, hipStream_t st) {
  if (waves_per_simd == 2) {
    if constexpr (S <= 3) {
      hipLaunchKernelGGL((stream_read_kernel<S, NT, 8>), dim3(blocks), dim3(512), 0, st, a);
      return 0;
    } else {
      return fail(HALO_PROBE_ERR_ARG, "4 stages need 1 wave per SIMD");
    }
  }
  hipLaunchKernelGGL((stream_read_kernel<S, NT, 4>), dim3(blocks), dim3(256), 0, st, a);
  return 0;
}

// ---------------------------------------------------------------- MFMA

struct MfmaArgs {
  float* out;
  int32_t iters;
};

// 8 independent accumulation chains per wave, so the matrix core never
// waits on a previous result.
template <int SHAPE>
__global__ __launch_bounds__(256) void mfma_kernel(MfmaArgs a) {
  const int lane = threadIdx.x & 63;
  bf16x8_t x, y;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    x[j] = (__bf16)(0.001f * (lane + j));
    y[j] = (__bf16)(0.002f * (lane - j));
  }
  float sum = 0.f;
  if constexpr (SHAPE == 32) {
    f32x16_t c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = f32x16_t{};
    for (int it = 0; it < a.iters; ++it) {
#pragma unroll
      for (int i = 0; i < 8; ++i) c[i] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, c[i], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 16; ++j) sum += c[i][j];
  } else {
    f32x4_t c[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) c[i] = f32x4_t{};
    for (int it = 0; it < a.iters; ++it) {
#pragma unroll
      for (int i = 0; i < 8; ++i) c[i] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(x, y, c[i], 0, 0, 0);
    }
#pragma unroll
    for (int i = 0; i < 8; ++i)
#pragma unroll
      for (int j = 0; j < 4; ++j) sum += c[i][j];
  }
  a.out[blockIdx.x * blockDim.x + threadIdx.x] = sum;
}

// ---------------------------------------------------------------- exp

struct ExpArgs {
  float* out;
  int32_t iters;
};

// 16 independent exp2 chains per lane; with M > 0, one 32x32x16 MFMA per
// M exponentials (chained into 4 accumulators) on the same wave.
template <int M>
__global__ __launch_bounds__(256) void exp_kernel(ExpArgs a) {
  const int lane = threadIdx.x & 63;
  float v[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) v[j] = -0.001f * (lane + j);
  bf16x8_t x, y;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    x[j] = (__bf16)(0.001f * (lane + j));
    y[j] = (__bf16)(0.002f * (lane - j));
  }
  f32x16_t c[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) c[i] = f32x16_t{};
  for (int it = 0; it < a.iters; ++it) {
#pragma unroll
    for (int j = 0; j < 16; ++j) {
      // a bare chain of exponentials (its values run to +inf, which does not
      // change the instruction's rate)
      v[j] = __builtin_amdgcn_exp2f(v[j]);
      if constexpr (M > 0) {
        if (j % M == M - 1) c[(j / M) % 4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, c[(j / M) % 4], 0, 0, 0);
      }
    }
  }
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) sum += v[j];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 16; ++j) sum += c[i][j];
  a.out[blockIdx.x * blockDim.x + threadIdx.x] = sum;
}

// ---------------------------------------------------------------- overlap

// MFMA and VALU work on one SIMD: 8-wave workgroups (two waves per SIMD),
// per iteration and wave pair 16 32x32x16 MFMAs (4 accumulator chains) and
// 16 V VALU instructions (16 independent chains of v_fma_f32, or of
// v_exp_f32 when EXP). SPLIT = false: every wave issues half of both,
// interleaved in its own stream; SPLIT = true: waves 0-3 issue only the
// MFMAs and waves 4-7 only the VALU work (one of each kind per SIMD).
template <bool SPLIT, int V, bool EXP>
__global__ __launch_bounds__(512) void overlap_kernel(ExpArgs a) {
  const int lane = threadIdx.x & 63;
  const int wave = __builtin_amdgcn_readfirstlane((int)(threadIdx.x >> 6));
  float v[16];
#pragma unroll
  for (int j = 0; j < 16; ++j) v[j] = -0.001f * (lane + j);
  bf16x8_t x, y;
#pragma unroll
  for (int j = 0; j < 8; ++j) {
    x[j] = (__bf16)(0.001f * (lane + j));
    y[j] = (__bf16)(0.002f * (lane - j));
  }
  f32x16_t c[4];
#pragma unroll
  for (int i = 0; i < 4; ++i) c[i] = f32x16_t{};
  auto valu = [&](int j) {
    if constexpr (EXP) v[j] = __builtin_amdgcn_exp2f(v[j]);
    else v[j] = __builtin_fmaf(v[j], 0.999f, 0.001f);
  };
  const bool do_mfma = !SPLIT || wave < 4;
  const bool do_valu = !SPLIT || wave >= 4;
  constexpr int NM = SPLIT ? 16 : 8;          // MFMAs per iteration of this wave
  for (int it = 0; it < a.iters; ++it) {
    if (do_mfma && do_valu) {
#pragma unroll
      for (int k = 0; k < NM; ++k) {
        c[k % 4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, c[k % 4], 0, 0, 0);
#pragma unroll
        for (int q = 0; q < V; ++q) valu((k * V + q) % 16);
      }
    } else if (do_mfma) {
#pragma unroll
      for (int k = 0; k < NM; ++k) c[k % 4] = __builtin_amdgcn_mfma_f32_32x32x16_bf16(x, y, c[k % 4], 0, 0, 0);
    } else {
#pragma unroll
      for (int k = 0; k < NM * V; ++k) valu(k % 16);
    }
  }
  float sum = 0.f;
#pragma unroll
  for (int j = 0; j < 16; ++j) sum += v[j];
#pragma unroll
  for (int i = 0; i < 4; ++i)
#pragma unroll
    for (int j = 0; j < 16; ++j) sum += c[i][j];
  a.out[blockIdx.x * blockDim.x + threadIdx.x] = sum;
}

}  // namespace

extern "C" int halo_probe_overlap(int32_t split, int32_t valu_per_mfma, int32_t use_exp, int32_t iters,
                                  int32_t blocks, float* out, void* stream) {
  g_err.clear();
  if (!out || iters < 1 || blocks < 1) return fail(HALO_PROBE_ERR_ARG, "out, iters >= 1, blocks >= 1");
  (void)hipGetLastError();
  ExpArgs a{out, iters};
  hipStream_t st = static_cast<hipStream_t>(stream);
#define HALO_PROBE_OVERLAP(S, V, E) \
  hipLaunchKernelGGL((overlap_kernel<S, V, E>), dim3(blocks), dim3(512), 0, st, a)
  const int key = (split ? 100 : 0) + (use_exp ? 10 : 0) + valu_per_mfma;
  switch (key) {
    case 2: HALO_PROBE_OVERLAP(false, 2, false); break;
    case 4: HALO_PROBE_OVERLAP(false, 4, false); break;
    case 8: HALO_PROBE_OVERLAP(false, 8, false); break;
    case 12: HALO_PROBE_OVERLAP(false, 2, true); break;
    case 14: HALO_PROBE_OVERLAP(false, 4, true); break;
    case 102: HALO_PROBE_OVERLAP(true, 2, false); break;
    case 104: HALO_PROBE_OVERLAP(true, 4, false); break;
    case 108: HALO_PROBE_OVERLAP(true, 8, false); break;
    case 112: HALO_PROBE_OVERLAP(true, 2, true); break;
    case 114: HALO_PROBE_OVERLAP(true, 4, true); break;
    default: return fail(HALO_PROBE_ERR_ARG, "valu_per_mfma is 2, 4 or 8 (2 or 4 with exp)");
  }
#undef HALO_PROBE_OVERLAP
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(HALO_PROBE_ERR_HIP, hipGetErrorString(e));
  return 0;
}

extern "C" int halo_probe_stream_read(const void* pool, int64_t pool_bytes, const int32_t* tiles, int64_t n_tiles,
                                      int32_t steps_per_item, int32_t stages, int32_t waves_per_simd,
                                      int32_t nontemporal, int32_t blocks, uint32_t* out, void* stream) {
  g_err.clear();
  if (!pool || !tiles || !out) return fail(HALO_PROBE_ERR_ARG, "pool, tiles and out must not be NULL");
  if (n_tiles < 0 || n_tiles % (kTilesPerStep * (int64_t)steps_per_item) != 0 || steps_per_item < 1)
    return fail(HALO_PROBE_ERR_ARG, "n_tiles must be a multiple of 4 * steps_per_item");
  if ((stages < 2 || stages > 4) && (stages < 10 || stages > 13))
    return fail(HALO_PROBE_ERR_ARG, "stages must be 2, 3 or 4 (10..13: the item modes)");
  if (waves_per_simd != 1 && waves_per_simd != 2) return fail(HALO_PROBE_ERR_ARG, "waves_per_simd is 1 or 2");
  if (blocks < 1) return fail(HALO_PROBE_ERR_ARG, "blocks must be >= 1");
  if (pool_bytes < 4096) return fail(HALO_PROBE_ERR_ARG, "pool must hold at least one 4 KB tile");
  StreamArgs a{static_cast<const uint8_t*>(pool), pool_bytes / 4096, tiles, n_tiles / kTilesPerStep,
               steps_per_item, out};
  hipStream_t st = static_cast<hipStream_t>(stream);
  int rc = 0;
  (void)hipGetLastError();
  const bool nt = nontemporal != 0;
  if (stages >= 10) {   // item modes: 10 = independent items, 11 = items with per-step compute,
                        // 12, 13: the same with the K/V tile pattern of the suffix pass
    if (waves_per_simd != 2) return fail(HALO_PROBE_ERR_ARG, "item modes use 2 waves per SIMD");
    if (stages == 10) hipLaunchKernelGGL((stream_items_kernel<true, false, false>), dim3(blocks), dim3(512), 0, st, a);
    else if (stages == 11) hipLaunchKernelGGL((stream_items_kernel<true, true, false>), dim3(blocks), dim3(512), 0, st, a);
    else if (stages == 12) hipLaunchKernelGGL((stream_items_kernel<true, false, true>), dim3(blocks), dim3(512), 0, st, a);
    else hipLaunchKernelGGL((stream_items_kernel<true, true, true>), dim3(blocks), dim3(512), 0, st, a);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(HALO_PROBE_ERR_HIP, hipGetErrorString(e));
    return 0;
  }
  switch (stages) {
    case 2: rc = nt ? launch_stream<2, true>(a, waves_per_simd, blocks, st)
                    : launch_stream<2, false>(a, waves_per_simd, blocks, st); break;
    case 3: rc = nt ? launch_stream<3, true>(a, waves_per_simd, blocks, st)
                    : launch_stream<3, false>(a, waves_per_simd, blocks, st); break;
    default: rc = nt ? launch_stream<4, true>(a, waves_per_simd, blocks, st)
                     : launch_stream<4, false>(a, waves_per_simd, blocks, st); break;
  }
  if (rc) return rc;
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(HALO_PROBE_ERR_HIP, hipGetErrorString(e));
  return 0;
}

extern "C" int halo_probe_mfma(int32_t shape, int32_t iters, int32_t blocks, float* out, void* stream) {
  g_err.clear();
  if (!out || iters < 1 || blocks < 1) return fail(HALO_PROBE_ERR_ARG, "out, iters >= 1, blocks >= 1");
  if (shape != 32 && shape != 16) return fail(HALO_PROBE_ERR_ARG, "shape is 32 (32x32x16) or 16 (16x16x32)");
  (void)hipGetLastError();
  MfmaArgs a{out, iters};
  hipStream_t st = static_cast<hipStream_t>(stream);
  if (shape == 32) hipLaunchKernelGGL((mfma_kernel<32>), dim3(blocks), dim3(256), 0, st, a);
  else hipLaunchKernelGGL((mfma_kernel<16>), dim3(blocks), dim3(256), 0, st, a);
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(HALO_PROBE_ERR_HIP, hipGetErrorString(e));
  return 0;
}

extern "C" int halo_probe_exp(int32_t valu_per_mfma, int32_t iters, int32_t blocks, float* out, void* stream) {
  g_err.clear();
  if (!out || iters < 1 || blocks < 1) return fail(HALO_PROBE_ERR_ARG, "out, iters >= 1, blocks >= 1");
  (void)hipGetLastError();
  ExpArgs a{out, iters};
  hipStream_t st = static_cast<hipStream_t>(stream);
  switch (valu_per_mfma) {
    case 0: hipLaunchKernelGGL((exp_kernel<0>), dim3(blocks), dim3(256), 0, st, a); break;
    case 2: hipLaunchKernelGGL((exp_kernel<2>), dim3(blocks), dim3(256), 0, st, a); break;
    case 4: hipLaunchKernelGGL((exp_kernel<4>), dim3(blocks), dim3(256), 0, st, a); break;
    case 8: hipLaunchKernelGGL((exp_kernel<8>), dim3(blocks), dim3(256), 0, st, a); break;
    default: return fail(HALO_PROBE_ERR_ARG, "valu_per_mfma is 0, 2, 4 or 8");
  }
  hipError_t e = hipGetLastError();
  if (e != hipSuccess) return fail(HALO_PROBE_ERR_HIP, hipGetErrorString(e));
  return 0;
}

extern "C" const char* halo_probe_last_error(void) { return g_err.c_str(); }
