/*
 * halo_probe.h -- context microbenchmarks of the gfx950 attention kernels'
 * rooflines (libhalo_probe.so; measurement only, not part of the attention
 * path). They give the rates the kernels are compared with: the HBM read
 * rate for the access pattern of the suffix pass (random 4 KB K/V tiles,
 * 16-byte loads, plain or non-temporal), the dense bf16 matrix-core rate,
 * and the v_exp_f32 rate with and without MFMAs on the same wave.
 *
 * All pointers are device pointers; every call enqueues one kernel on
 * `stream` (a hipStream_t passed as void*) and returns 0, or a nonzero
 * HALO_PROBE_ERR_* code with halo_probe_last_error() describing it. Nothing
 * is allocated.
 */
#ifndef HALO_PROBE_H
#define HALO_PROBE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

#define HALO_PROBE_ERR_ARG 1
#define HALO_PROBE_ERR_HIP 4

/* Read n_tiles 4 KB tiles of pool (pool_bytes long): tile k is bytes
 * tiles[k] * 4096 .. + 4095 (ids are clamped to the pool). A step is 4
 * consecutive list entries (16 KB, 16 loads of 16 bytes per lane); an item
 * is steps_per_item consecutive steps; waves take items round-robin over the
 * grid of `blocks` workgroups and keep `stages` steps (2..4) of loads in
 * registers, across item boundaries. waves_per_simd: 2 (512-thread
 * workgroups, at most 3 stages) or 1 (256-thread workgroups). nontemporal:
 * loads with the non-temporal bit, as the suffix pass reads private keys.
 * stages = 10 or 11 selects the item modes instead (2 waves per SIMD, 2
 * stages): every item starts with a dependent metadata load, fills its own
 * pipeline and drains it before the next item (10), and with 11 each step
 * also runs 16 v_mfma_f32_16x16x32_bf16 and a short max/exp sequence, the
 * per-step work of the suffix pass at 8 query rows. 12 and 13 are 10 and 11
 * with the suffix pass's K/V access pattern: the step's first two tiles are
 * read as K pages (16-byte units, 128-byte runs of 8 tokens per unit) and
 * the other two as dim-major V pages (512-byte runs).
 * out: one uint32 per wave of the grid (an xor of what it read).
 * n_tiles must be a multiple of 4 * steps_per_item. */
int halo_probe_stream_read(const void* pool, int64_t pool_bytes, const int32_t* tiles, int64_t n_tiles,
                           int32_t steps_per_item, int32_t stages, int32_t waves_per_simd,
                           int32_t nontemporal, int32_t blocks, uint32_t* out, void* stream);

/* blocks x 4 waves, each running iters rounds of 8 independent bf16 MFMAs:
 * shape 32 = v_mfma_f32_32x32x16_bf16 (32768 flop each), 16 =
 * v_mfma_f32_16x16x32_bf16 (16384 flop each). out: blocks * 256 floats. */
int halo_probe_mfma(int32_t shape, int32_t iters, int32_t blocks, float* out, void* stream);

/* blocks x 4 waves, each running iters rounds of 16 independent v_exp_f32
 * per lane; with valu_per_mfma in {2, 4, 8}, one 32x32x16 bf16 MFMA is
 * issued after every valu_per_mfma exponentials (0: no MFMA).
 * out: blocks * 256 floats. */
int halo_probe_exp(int32_t valu_per_mfma, int32_t iters, int32_t blocks, float* out, void* stream);

/* blocks x 8 waves (two per SIMD), iters rounds; per round and wave pair
 * 16 v_mfma_f32_32x32x16_bf16 (4 accumulator chains) and 16 * valu_per_mfma
 * VALU instructions on 16 independent chains (v_fma_f32, or v_exp_f32 if
 * use_exp). split = 0: every wave issues half of both, interleaved in its
 * own instruction stream; split = 1: waves 0-3 issue only the MFMAs and
 * waves 4-7 only the VALU work. valu_per_mfma: 2, 4 or 8 (2 or 4 with
 * use_exp). out: blocks * 512 floats. */
int halo_probe_overlap(int32_t split, int32_t valu_per_mfma, int32_t use_exp, int32_t iters, int32_t blocks,
                       float* out, void* stream);

const char* halo_probe_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* HALO_PROBE_H */
