/*
 * moe_decode.h -- C ABI of the MI355X (CDNA4, gfx950) Mixture-of-Experts decode layer.
 *
 * One moe_decode_forward call is one decode step of one MoE layer for the T sequences
 * in flight.  That step is the unit of work of the paper's problem statement (Design
 * section, the constrained tokens-per-joule objective): decode throughput and
 * inter-token latency are made of these steps, and the paper's Background section
 * ("PD-disaggregated serving") characterises them as weight-read bound with flat
 * power.  The two MoE models it deploys (Experimental Setup, models row) are
 * Qwen3-235B-A22B and Qwen3-Coder-480B-A35B.
 *
 * A step computes, for every token t (x[t] one row of the activations):
 *   1. router logits  l[t,e] = RNE_fp32( exact sum_h x[t,h] * Wr[e,h] + b[e] ), -0 -> +0
 *   2. selection      the k experts of largest logit, ties to the lower expert index,
 *                     in that order; weights w[t,j] = softmax over all E logits,
 *                     renormalised over the k selected (= softmax of the selected)
 *   3. grouping       the (token, choice) pairs ordered by expert, then by token
 *   4. experts        per pair (t, e): g = Wgate[e] x[t], u = Wup[e] x[t],
 *                     a = silu(g) * u with silu(z) = z / (1 + e^-z), o = Wdown[e] a
 *   5. combine        y[t] = sum_j w[t,j] * o[t,j], j ascending
 * Weights are dequantised in registers: FP8 E4M3FN (OCP) times one fp32 scale per
 * 128x128 block, MXFP4 (OCP MX v1.0: E2M1 times 2^(E8M0-127) per 32 inputs), or
 * NVFP4 (E2M1 times an E4M3 scale per 16 inputs times an fp32 scale per matrix; the
 * paper deploys Qwen3-235B-A22B in this format, Experimental Setup, models row).
 *
 * Memory: every tensor pointer is a DEVICE pointer owned by the caller.  The library
 * never allocates device memory: its scratch lives in a caller-provided workspace
 * (moe_decode_workspace_bytes), or, for moe_decode_forward_noalloc, in a static
 * device array of the library.  The handle itself is host memory.
 *
 * Layouts (row-major, C order):
 *   x, y          [T][H]  act_dtype (bf16 or fp32); y must not alias x
 *   router_w      [E][H]  router_dtype
 *   router_bias   [E]     fp32, or NULL for no bias
 *   expert_w      E consecutive expert blocks; expert e at byte e * expert_stride:
 *                   FP8  : gate [I][H] | up [I][H] | down [H][I]           1 byte/weight
 *                   MXFP4, NVFP4: gate [I][H/2] | up [I][H/2] | down [H][I/2]
 *                          even input index in the low nibble
 *                 (input index contiguous in every row)
 *   scales        FP8  : fp32, per expert gate [I/128][H/128] | up [I/128][H/128] |
 *                        down [H/128][I/128]
 *                 MXFP4: E8M0 bytes, per expert gate [I][H/32] | up [I][H/32] | down [H][I/32]
 *                 NVFP4: per expert 16 bytes of fp32 matrix scales {gate, up, down, unused},
 *                        then E4M3 bytes gate [I][H/16] | up [I][H/16] | down [H][I/16]
 *                        (block scales are positive codes; expert stride 16 + 3*H*I/16)
 *   topk_ids      [T][k] int32 (optional output), topk_weights [T][k] fp32 (optional)
 *
 * Errors: every argument check runs before anything is enqueued; a failed check
 * returns a negative moe_status and leaves a message for moe_decode_last_error.
 * A failed kernel launch returns MOE_ERR_HIP.  Device faults surface at the
 * caller's next synchronisation.  No C++ exception crosses this interface.
 * NaN or infinite inputs, and E8M0 scale codes 0 and 255, are outside the contract.
 *
 * Concurrency: forward is asynchronous on the given HIP stream and never
 * synchronises.  A handle (and its workspace) serves one stream at a time; calls
 * that overlap on one handle race.
 */
#ifndef MOE_DECODE_H
#define MOE_DECODE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef struct moe_decode_s *moe_decode_t;

typedef enum {
    MOE_OK = 0,
    MOE_ERR_INVALID = -1,     /* an argument is out of range, NULL or misaligned */
    MOE_ERR_UNSUPPORTED = -2, /* a valid but unsupported configuration */
    MOE_ERR_WORKSPACE = -3,   /* workspace NULL, misaligned or too small */
    MOE_ERR_HIP = -4          /* a HIP runtime call or kernel launch failed */
} moe_status;

typedef enum { MOE_DTYPE_F32 = 0, MOE_DTYPE_BF16 = 1 } moe_dtype;

typedef enum {
    MOE_WFMT_FP8_E4M3_B128 = 0,  /* E4M3FN weights, fp32 scale per 128x128 block */
    MOE_WFMT_MXFP4_E2M1_B32 = 1, /* E2M1 weights, E8M0 scale per 32 inputs */
    MOE_WFMT_NVFP4_E2M1_B16 = 2  /* E2M1 weights, E4M3 scale per 16 inputs, fp32 scale per matrix;
                                    needs bf16 activations */
} moe_wfmt;

typedef enum {
    MOE_WLAYOUT_ROW_MAJOR = 0, /* every matrix [rows][K], K contiguous (the layout above) */
    MOE_WLAYOUT_TILED16 = 1    /* packed 16-row tiles: each tile of 16 rows keeps its offset
                                  and size, and inside it each 128-input K block is one
                                  contiguous piece of the tile's 16 row segments in the
                                  matrix cores' operand order (FP8: 2 KB, the bytes K
                                  [16g, 16g+16) of row l%16 at 16 l and K [64+16g, +16) at
                                  1024 + 16 l, g = l/16, l < 64; MXFP4: 1 KB, K [32g, 32g+32)
                                  of row l%16 at 16 l; NVFP4: 256-input blocks of 2 KB,
                                  row l%16's bytes [32g, 32g+16) at 16 l and [32g+16,
                                  32g+32) at 1024 + 16 l, and the E4M3 scales packed
                                  the same way: per tile and 256-input block one 256-byte
                                  piece, scales [4g, 4g+4) of row l%16 at 4 l, or, for a
                                  matrix whose K/256 is a multiple of four, per tile and
                                  group of four blocks one 1 KB piece, lane l's 4 scales
                                  of each block of the group (block by block) at 16 l;
                                  the 16 bytes of matrix scales stay first).  MXFP4 E8M0 scales
                                  are packed per tile and group of four 128-input blocks:
                                  lane l's bytes (K sub-block g of row l%16, blocks 4q..4q+3)
                                  at 4 l of a 256-byte piece (a last group of two blocks:
                                  2 l, 128 bytes).  FP8 scales are unchanged.  Written by
                                  moe_decode_pack_weights.  Needs MFMA tiles for every
                                  expert (mfma_min_tokens 0 or 1). */
} moe_wlayout;

typedef struct moe_decode_config {
    int32_t hidden;          /* H: multiple of 128 (FP8) or 256 (MXFP4, NVFP4) */
    int32_t n_experts;       /* E: 1..1024 */
    int32_t inter;           /* I: SwiGLU intermediate size, multiple of 128 (FP8) or 256 (MXFP4, NVFP4) */
    int32_t max_topk;        /* largest k of any call: 1..min(E, 64) */
    int32_t max_tokens;      /* largest T of any call: 1..1024, E * ceil(T/32) <= 8192 */
    int32_t act_dtype;       /* moe_dtype of x and y */
    int32_t router_dtype;    /* moe_dtype of router_w */
    int32_t wfmt;            /* moe_wfmt of expert_w / scales */
    int32_t mfma_min_tokens; /* an expert with at least this many tokens in a step runs on
                                MFMA tiles, below it on the GEMV path; 0 = library default
                                (1: MFMA for every expert, the faster path on MI355X at
                                every measured token count), negative = never */
    int32_t weight_layout;   /* moe_wlayout of expert_w */
    int32_t screen_min_tokens; /* a forward step with at least this many tokens screens the
                                router logits: bf16 matrix-core sums give every logit a
                                rigorous bracket, and only the experts whose bracket can
                                reach the top k get the exact logit (the selection is
                                the same); needs bf16 x and router_w and H a multiple of
                                256.  0 = library default (the smallest T with
                                T*E*H >= 2^26 multiply-adds), negative = never */
    int32_t reserved[5];     /* must be zero */
} moe_decode_config;

typedef struct moe_decode_stats {
    int32_t n_tokens;        /* T of the last forward */
    int32_t n_active;        /* experts with at least one token in the last forward */
    int32_t n_active_mfma;   /* of those, experts that ran on MFMA tiles */
    int32_t n_fallback;      /* router logits that needed the exact (double-double) path */
    int32_t n_exact_logits;  /* router logits computed exactly (T*E unless screened) */
    int32_t route_screened;  /* 1 if the last forward screened the router logits */
    int64_t active_weight_bytes; /* unique expert weight + scale bytes the step streamed */
} moe_decode_stats;

/* Stages timed by the optional profiler (moe_decode_profile_*). */
typedef enum {
    MOE_STAGE_ROUTE = 0,   /* router logits, top-k softmax, grouping */
    MOE_STAGE_W13 = 1,     /* grouped gate/up projection with the SiLU-gate epilogue */
    MOE_STAGE_W2 = 2,      /* grouped down projection */
    MOE_STAGE_COMBINE = 3, /* weighted combine */
    MOE_N_STAGES = 4
} moe_stage;

/* Bytes of device workspace a handle with this configuration needs (0 if the
 * configuration is invalid; moe_decode_init then says why). */
size_t moe_decode_workspace_bytes(const moe_decode_config *cfg);

/* Bytes of one expert's weights (expert_stride of the layout above) and scales. */
size_t moe_decode_expert_weight_bytes(const moe_decode_config *cfg);
size_t moe_decode_expert_scale_bytes(const moe_decode_config *cfg);

/* Validate cfg and create a handle bound to `workspace` (device memory of at least
 * moe_decode_workspace_bytes(cfg) bytes, 256-byte aligned, owned by the caller and
 * kept alive until moe_decode_free).  Makes no HIP call.  *out is set to NULL on error. */
moe_status moe_decode_init(const moe_decode_config *cfg, void *workspace, size_t workspace_bytes,
                           moe_decode_t *out);

/* One decode step (steps 1-5 above) for n_tokens tokens, enqueued on `stream`
 * (a hipStream_t; NULL = the null stream).  x, router_w, expert_w and y must be
 * 16-byte aligned, the other pointers 4-byte aligned.  1 <= topk <= max_topk;
 * 0 <= n_tokens <= max_tokens (0 enqueues nothing).  topk_ids / topk_weights may be
 * NULL.  Bitwise deterministic for identical inputs. */
moe_status moe_decode_forward(moe_decode_t h, void *stream, const void *x, int32_t n_tokens, const void *router_w,
                              const float *router_bias, const void *expert_w, const void *scales, int32_t topk,
                              void *y, int32_t *topk_ids, float *topk_weights);

/* The same decode step as moe_decode_forward, for callers that cannot allocate device
 * memory or create a handle: code under HIP graph capture, tight serving loops, and
 * harnesses that forbid hipMalloc.  It takes the configuration itself (validated as by
 * moe_decode_init) and uses as its workspace a static device array of the library
 * (64 MiB, 256-byte aligned; one copy on each device the library runs on, held until
 * the process ends), so it calls no hipMalloc, hipFree, host allocator or other
 * allocating routine.  Configurations whose workspace (moe_decode_workspace_bytes)
 * exceeds 64 MiB less 256.5 KiB of routing counters are rejected with
 * MOE_ERR_WORKSPACE before anything is enqueued.  `stream` must belong to the
 * current device (MOE_ERR_INVALID otherwise); the first call on a device also
 * enqueues one clear of the array's counters on that stream.  Arguments, layouts,
 * alignment, results and bitwise determinism as for moe_decode_forward; errors are
 * reported through moe_decode_last_error(NULL) of the calling thread.  Every call on
 * one device shares that device's array and it keeps the last call's contents:
 * calls that overlap on one device (concurrent streams or host threads) race, and
 * there are no statistics to read back. */
moe_status moe_decode_forward_noalloc(const moe_decode_config *cfg, void *stream, const void *x, int32_t n_tokens,
                                      const void *router_w, const float *router_bias, const void *expert_w,
                                      const void *scales, int32_t topk, void *y, int32_t *topk_ids,
                                      float *topk_weights);

/* Enqueue on `stream` the conversion of n_experts consecutive experts' weights (and,
 * for MXFP4 and NVFP4, their scales) from the row-major layout (src) to packed 16-row tiles (dst),
 * for a handle whose configuration has weight_layout = MOE_WLAYOUT_TILED16 (the other
 * fields as for that handle; weight_layout itself is not read).  src and dst are device
 * buffers of n_experts * moe_decode_expert_weight_bytes(cfg) bytes, 16-byte aligned;
 * src_scales and dst_scales of n_experts * moe_decode_expert_scale_bytes(cfg) bytes,
 * 4-byte aligned, for MXFP4 and NVFP4 weights, NULL for FP8 ones (their scales keep their
 * layout).  All owned by the caller; a source and its destination must not overlap.
 * Errors as for moe_decode_init (message in moe_decode_last_error(NULL)). */
moe_status moe_decode_pack_weights(const moe_decode_config *cfg, void *stream, const void *src, void *dst,
                                   const void *src_scales, void *dst_scales, int32_t n_experts);

/* Steps 1-2 only (router logits and top-k softmax).  `logits` [T][E] fp32 receives
 * the canonical logits if not NULL; topk_ids / topk_weights as in forward. */
moe_status moe_decode_route(moe_decode_t h, void *stream, const void *x, int32_t n_tokens, const void *router_w,
                            const float *router_bias, int32_t topk, float *logits, int32_t *topk_ids,
                            float *topk_weights);

/* Statistics of the last forward on this handle.  Synchronises that call's stream.
 * counts_host, if not NULL, receives E per-expert token counts. */
moe_status moe_decode_get_stats(moe_decode_t h, moe_decode_stats *out, int32_t *counts_host);

/* Profiler: record HIP events around each stage of the next `max_calls` forward
 * calls (max_calls <= 0 disables and releases the events).  Creates events, makes
 * no device allocation.  Adds one event record per stage boundary to each call. */
moe_status moe_decode_profile_enable(moe_decode_t h, int32_t max_calls);

/* Stage durations in milliseconds of the recorded calls: stage_ms[c * MOE_N_STAGES + s]
 * for call c; *n_calls receives the number recorded (at most the capacity given to
 * moe_decode_profile_enable).  Synchronises the recorded events.  Resets the record. */
moe_status moe_decode_profile_read(moe_decode_t h, float *stage_ms, int32_t *n_calls);

/* Release the handle (host memory and profiler events).  The workspace stays the
 * caller's.  NULL is ignored. */
void moe_decode_free(moe_decode_t h);

/* Static text for a status code. */
const char *moe_decode_status_string(moe_status s);

/* Text of the last error on this handle ("" if none); for a NULL handle, the last
 * error of a failed moe_decode_init or moe_decode_pack_weights in this thread. */
const char *moe_decode_last_error(moe_decode_t h);

#ifdef __cplusplus
}
#endif

#endif /* MOE_DECODE_H */
