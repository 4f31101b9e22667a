/*
 * alr_debug.h -- kernel-level test hooks of the rollout library.
 *
 * These entry points expose single kernels of the library so that tests can
 * check them in isolation and benchmarks can time them.  They are not needed
 * to run the rollout.
 */
#ifndef ALR_DEBUG_H
#define ALR_DEBUG_H

#include <stdint.h>

#include "alr.h"

#ifdef __cplusplus
extern "C" {
#endif

/* C[M,N] (fp32, row-major) = A[M,K] * W[N,K]^T, on the library's GEMM kernel
 * for `dtype` (ALR_BF16: bf16 MFMA with fp32 accumulation; ALR_F32: fp32 FMA).
 * A, W, C are device pointers, row-major and contiguous; N and K must be
 * multiples of 64 (ALR_E_UNSUPPORTED otherwise).  `tile` picks the bf16
 * kernel: 0 = the library's choice for this shape; W staged through LDS:
 * 1 = 256x128, 2 = 128x128, 3 = 64x128, 4 = 256x256 (8 waves), 5 = 256x256
 * (4 waves); 17 = ping-pong (the two waves of each SIMD alternate LDS and
 * MFMA phases) over register-staged BK = 64 tiles, one tile per workgroup
 * (K a multiple of 64); 18 = split-K over the ping-pong kernel (K slices
 * summed in slice order by a second kernel; 2 or 4 slices by the library's
 * rule, at least 2; K a multiple of 128); 19 = the ping-pong kernel of 17 run
 * persistently (one workgroup per CU looping over the tiles, the next tile's
 * first k-steps loaded during the current tile's last ones); 20 = split-K
 * over the 64x128 kernel of 3 (2 or 4 slices, each a multiple of 64; the
 * unsplit kernel of 3 when K allows no split).  Other values:
 * ALR_E_INVALID_ARG.  Tiles 18 and 20 need a device scratch buffer of at
 * least 2*M*N*4 bytes for the partial sums (up to 4*M*N*4 are used when
 * given); ALR_E_WORKSPACE otherwise.
 * Enqueued on `stream`. */
alr_status alr_debug_gemm(int32_t dtype, const void* A, const void* W, float* C, int32_t M,
                          int32_t N, int32_t K, int32_t tile, void* scratch,
                          size_t scratch_bytes, alr_stream stream);

/* Work plan of the decode attention for a rollout request (host only, no GPU
 * needed; the same planner alr_rollout runs).  n_seq sequences of lengths
 * seq_len[] laid out as alr_prefill lays them out (keys of sequence i from the
 * sum of the earlier lengths; its transposed values from the sum of the
 * earlier lengths each rounded up to 64), n_anchor anchors as for
 * alr_check_rollout, a device of n_cu compute units.  Writes the key-chunk
 * length in 64-key tiles to *ct_out, the simulated makespan (tiles, an item
 * costing its tiles + 3) to *makespan_out and the number of work items,
 * padding included, to *n_items_out; if items_out is not NULL, item b (run on
 * XCD b % 8) as 6 int32 at items_out[6 b]: first anchor in sorted order (by
 * sequence, then position, then the caller's index), anchor count (0 for
 * padding), kv head, first key, end key (exclusive), partial-output index.
 * ALR_E_UNSUPPORTED when the config's attention has no plan (fp32, or a head
 * size other than 64 and 128), ALR_E_WORKSPACE when the items exceed
 * max_items, the statuses of alr_check_config / alr_check_rollout otherwise. */
alr_status alr_debug_decode_plan(const alr_config* cfg, int32_t n_cu, int32_t n_seq,
                                 const int32_t* seq_len, int32_t n_anchor,
                                 const int32_t* anchor_seq, const int32_t* anchor_pos,
                                 int32_t* ct_out, int32_t* makespan_out, int32_t* n_items_out,
                                 int32_t* items_out, int32_t max_items);

/* Kernel launch sites whose device time can be measured with alr_profile_*. */
typedef enum {
  ALR_PROF_PREFILL_QKV = 1,   /* prefill QKV GEMM (+RoPE, shared K/V store)        */
  ALR_PROF_PREFILL_ATTN = 2,  /* prefill causal attention                           */
  ALR_PROF_PREFILL_O = 3,     /* prefill attention-output GEMM (+residual)          */
  ALR_PROF_PREFILL_GU = 4,    /* prefill gate|up GEMM (+SwiGLU)                     */
  ALR_PROF_PREFILL_DOWN = 5,  /* prefill down GEMM (+residual, features)            */
  ALR_PROF_DECODE_QKV = 6,    /* rollout-step QKV GEMM (+RoPE, private K/V append)  */
  ALR_PROF_DECODE_ATTN = 7,   /* rollout-step anchor-branched attention             */
  ALR_PROF_DECODE_O = 8,
  ALR_PROF_DECODE_GU = 9,
  ALR_PROF_DECODE_DOWN = 10,
  ALR_PROF_LM_GEMM = 11,      /* output-head GEMM (logits into the caller's rows)   */
  ALR_PROF_LM_FINALIZE = 12,  /* log-sum-exp, greedy argmax, in-place log-softmax   */
  ALR_PROF_DECODE_COMBINE = 13, /* merge of decode-attention chunk partials (bf16)  */
  ALR_PROF_COUNT = 14
} alr_prof_site;

/* Start timing every launch at `site` with HIP events recorded on the launch
 * stream, for up to `capacity` launches (later launches are not timed).
 * Creates 2*capacity events (host-side HIP objects, no device buffers). */
alr_status alr_profile_start(alr_ctx* ctx, int32_t site, int32_t capacity);

/* Stop timing; waits for the last recorded event and returns the summed
 * device time (ms) and the number of timed launches.  Destroys the events. */
alr_status alr_profile_stop(alr_ctx* ctx, double* total_ms, int32_t* launches);

#ifdef __cplusplus
}
#endif

#endif /* ALR_DEBUG_H */
