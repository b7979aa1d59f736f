/* attn_decode.h -- C ABI of one decode step of grouped-query attention over a paged
 * KV cache on AMD Instinct MI355X (gfx950).
 *
 * A decode step reads the weights and the KV cache (the paper's Background and
 * Motivation section names both as the byte streams that bound decode); this entry
 * point is the KV-cache half.  For sequence b (context length L_b = ctx_lens[b]) and
 * query head h, with G = Hq / Hkv query heads per key/value head and g = h / G:
 *     s_j = scale * q[b][h] . K_b[g][j]              j < L_b
 *     p   = softmax_j(s)
 *     out[b][h] = sum_j p_j V_b[g][j]
 * (scaled dot-product attention with grouped key/value heads).  A sequence with
 * L_b = 0 gets out = 0.
 *
 * Memory: every tensor pointer is a DEVICE pointer owned by the caller; the library
 * never allocates device memory.  Layouts (bf16 = the upper 16 bits of an fp32):
 *   q            [B][Hq][D] bf16
 *   k_cache      [n_pages][Hkv][P][D] bf16   token-major within a page
 *   v_cache      [n_pages][Hkv][D][P] bf16   dimension-major within a page
 *   block_table  [B][max_pages_per_seq] int32: token j of sequence b sits in page
 *                block_table[b][j / P] at slot j % P; entries past the context are
 *                never read
 *   ctx_lens     [B] int32, 0 <= L_b <= max_pages_per_seq * P (device memory)
 *   out          [B][Hq][D] bf16 (must not alias any input)
 * Pointers must be 16-byte aligned.  A page index outside [0, n_pages) is read as a
 * page of zeros; a context length outside its range is clamped to it.
 *
 * Errors: argument checks run before anything is enqueued and return a negative
 * status with a message in attn_decode_last_error() (per thread); launch failures
 * return ATTN_ERR_HIP.  The call is asynchronous on `stream` (a hipStream_t, NULL for
 * the default stream) and bitwise deterministic for identical inputs.  Calls that
 * share a workspace must not overlap.
 */
#ifndef ATTN_DECODE_H
#define ATTN_DECODE_H

#include <stddef.h>
#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

enum {
    ATTN_OK = 0,
    ATTN_ERR_INVALID = -1,     /* argument out of range or inconsistent */
    ATTN_ERR_UNSUPPORTED = -2, /* valid but not implemented (head_dim, page size, group) */
    ATTN_ERR_WORKSPACE = -3,   /* workspace too small */
    ATTN_ERR_HIP = -4          /* a HIP launch failed */
};

typedef struct attn_decode_config {
    int32_t n_q_heads;         /* Hq: multiple of n_kv_heads, Hq / Hkv <= 16 */
    int32_t n_kv_heads;        /* Hkv >= 1 */
    int32_t head_dim;          /* D: 128 */
    int32_t page_size;         /* P: 16 */
    int32_t max_batch;         /* largest B of any call, 1..4096 */
    int32_t max_pages_per_seq; /* block-table row length, 1..65536 */
    int32_t fused_merge_max_splits; /* the context is cut into 256-token pieces.  The grid
                                  has S splits per sequence: the fewest that cover a row
                                  of max_pages_per_seq pages with at most this many, and
                                  fewer when one piece per workgroup would need more than
                                  two rounds of resident workgroups for max_batch
                                  sequences (then the grid is at most three workgroups per
                                  compute unit).  Each sequence walks R = ceil(its own
                                  pieces / S) consecutive pieces per workgroup (online
                                  softmax across them), so a short context uses one piece
                                  per split whatever the capacity.  The split kernel
                                  merges the splits itself (its last workgroup per
                                  sequence and key/value head).  0 = library default 16,
                                  at most 16; negative = one piece per split, merged by a
                                  second kernel.  Where R = 1 both merges give the same
                                  bits; a sequence's result depends only on its own
                                  context, this configuration and the device, never on
                                  the rest of the batch. */
    int32_t reserved[3];       /* must be zero */
} attn_decode_config;

/* Bytes of device workspace forward needs for this configuration (split partials and
 * one merge counter per sequence and key/value head); 0 if the configuration is
 * invalid. */
size_t attn_decode_workspace_bytes(const attn_decode_config *cfg);

/* Enqueue on `stream` the clearing of a workspace's merge counters: once, before the
 * workspace's first forward (each forward leaves them cleared again; after a forward
 * that did not complete, clear them again).  Same workspace rules and status codes as
 * attn_decode_forward. */
int attn_decode_workspace_init(const attn_decode_config *cfg, void *workspace, size_t workspace_bytes, void *stream);

/* One decode step of attention for `batch` sequences (0 <= batch <= max_batch; 0 is a
 * no-op).  `scale` multiplies the scores (1/sqrt(D) for standard attention) and must
 * be finite and positive.  `workspace` holds at least attn_decode_workspace_bytes(cfg)
 * bytes of device memory owned by the caller, initialised once by
 * attn_decode_workspace_init. */
int attn_decode_forward(const attn_decode_config *cfg, void *workspace, size_t workspace_bytes, void *stream,
                        const void *q, const void *k_cache, const void *v_cache, int64_t n_pages,
                        const int32_t *block_table, const int32_t *ctx_lens, int32_t batch, float scale,
                        void *out);

/* Message of the calling thread's last failed call ("" if none). */
const char *attn_decode_last_error(void);

#ifdef __cplusplus
}
#endif

#endif /* ATTN_DECODE_H */
