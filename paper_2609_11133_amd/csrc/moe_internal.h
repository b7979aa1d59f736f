// Internal declarations of the MoE decode library (not part of the C ABI).
#pragma once

#include <hip/hip_runtime.h>
#include <stddef.h>
#include <stdint.h>

namespace moe {

// Workspace carve-up.  Every region starts on a 256-byte boundary.
struct Workspace {
    float *logits;     // [Tmax][E] canonical router logits
    int32_t *ids;      // [Tmax][kmax] selected experts (rank order)
    float *wts;        // [Tmax][kmax] routing weights
    int32_t *meta;     // Meta block, see MetaIdx
    int32_t *slot_of;  // [Tmax*kmax] slot of pair (t, j)
    int32_t *tok_of;   // [Tmax*kmax] token of slot
    float *h;          // [Tmax*kmax][I] SwiGLU activations per slot (GEMV path)
    float *o;          // [Tmax*kmax][H] expert outputs per slot
    int32_t *sync;     // [(Tmax + 2) * kCounterStride] routing counters (zero between launches)
    uint8_t *xs_hi, *xs_lo;  // [Tmax][H] 2-term FP8 split of x (MFMA path)
    uint8_t *xe_hi, *xe_lo;  // [Tmax][H/32] E8M0 exponents of the split
    uint8_t *hs_hi, *hs_lo;  // [Tmax*kmax][I] 2-term FP8 split of h (MFMA path)
    uint8_t *he_hi, *he_lo;  // [Tmax*kmax][I/32]
    __bf16 *hb;              // [Tmax*kmax][I] bf16 SwiGLU activations (NVFP4 MFMA path)
    _Float16 *x16;           // [Tmax][H] x * 2^-k in f16 (NVFP4 MFMA path)
    int32_t *xk;             // [Tmax] the power k of each token
    void *part;              // screened routing: [ks_max][Tmax][E] (sum x*w, sum |x*w|) fp64 pairs
    float *xmax, *wmax;      // [ks_max][Tmax], [ks_max][E] slice maxima of |x| and |w|
    int ks_max;              // K slices the screened routing may use (0: path off)
    size_t bytes;
};

// Layout of the meta block (int32 words).  Records are int4 and start on 16-byte
// boundaries: GEMV records {expert, first slot, tokens, 0}; MFMA chunk records
// {expert, first slot of the chunk, tokens in the chunk (<= 32), 0}, one per 32
// tokens of an MFMA expert.
struct MetaIdx {
    int E;
    int max_chunks;  // E + ceil(Tmax * kmax / 32) bounds the number of MFMA chunks
    __host__ __device__ int n_active() const { return 0; }
    __host__ __device__ int n_gemv() const { return 1; }
    __host__ __device__ int n_mfma() const { return 2; }
    __host__ __device__ int n_fallback() const { return 3; }
    __host__ __device__ int n_mfma_chunks() const { return 4; }
    __host__ __device__ int n_exact() const { return 5; }   // router logits computed exactly
    __host__ __device__ int screened() const { return 6; }  // 1: the step screened its logits
    __host__ __device__ int counts() const { return 8; }        // [E]
    __host__ __device__ int offsets() const { return 8 + E; }   // [E+1]
    __host__ __device__ int gemv_rec() const { return ((8 + 2 * E + 1) + 3) & ~3; }  // int4 [E]
    __host__ __device__ int chunk_rec() const { return gemv_rec() + 4 * E; }         // int4 [max_chunks]
    __host__ __device__ int words() const { return chunk_rec() + 4 * max_chunks; }
};

__host__ __device__ inline int max_mfma_chunks(int E, int Tmax, int kmax) { return E + (Tmax * kmax + 31) / 32; }

constexpr int kMfmaChunk = 32;      // tokens per MFMA pass (two 16-column tiles)
// Screened routing by default from T*E*H >= 2^26 multiply-adds of exact logits: below
// it the fixed costs of the extra pass outweigh the logits it saves.
constexpr long kScreenMinMacs = 1L << 26;
constexpr int kCandCounterOff = 32;  // int32 words from the fallback counter to the candidate counter

// K slices of the screened routing's partial sums: at most 16 and H/256, and the
// partials at most 4 Mi fp64 pairs (64 MB); 0 when H is not a multiple of 256.
constexpr int kScreenMaxKS = 16;
__host__ __device__ inline int screen_ks_max(int H, int E, int Tmax)
{
    if (H % 256) return 0;
    long ks = H / 256;
    ks = ks < kScreenMaxKS ? ks : kScreenMaxKS;
    const long cap = (1L << 22) / ((long)Tmax * E);
    ks = ks < cap ? ks : cap;
    return ks < 1 ? 1 : (int)ks;
}
constexpr int kCounterStride = 64;  // int32 words between routing counters (256 bytes)

// The FP8 split regions are carved for FP8 and MXFP4 weights, hb for NVFP4 weights
// (the other pointers are NULL).
size_t carve_workspace(int H, int E, int I, int kmax, int Tmax, int wfmt, void *base, Workspace *ws);

// Geometry of one layer as the kernels see it.
struct Layer {
    int H, E, I;
    int wfmt;       // 0 FP8-E4M3 (128x128 fp32 scales), 1 MXFP4 (E8M0 per 32),
                    // 2 NVFP4 (E4M3 per 16 + fp32 per matrix)
    int act_bf16;   // activations bf16 (1) or fp32 (0)
    int router_bf16;
    int wlayout;    // expert weights: 0 row-major, 1 packed 16-row tiles
    size_t expert_w_bytes;  // per expert
    size_t expert_s_bytes;  // per expert
};

struct RouteParams {
    const void *x;
    int T, k;
    const void *router_w;
    const float *bias;
    float *logits;
    int32_t *ids, *ids_user;
    float *wts, *wts_user;
    int32_t *meta, *slot_of, *tok_of;
    int32_t *cnt_tok, *cnt_all, *fb_acc;
    uint8_t *xs_hi, *xs_lo, *xe_hi, *xe_lo;  // NULL: no activation split
    _Float16 *x16;                           // NULL: no f16 copy of x (NVFP4 MFMA path)
    int32_t *xk;
    void *part;                               // screened routing buffers (Workspace)
    float *xmax, *wmax;
    int ks_max, Tmax;
    int mstar;
    int do_group;
    int max_chunks;
    int screen;  // 1: screened routing for this step (forward with grouping only)
};

// ---- launchers (all enqueue on `st`, return hipGetLastError())
hipError_t launch_zero(int32_t *p, int n, hipStream_t st);
hipError_t launch_route(const Layer &L, const RouteParams &P, hipStream_t st);
hipError_t launch_pack_weights(const Layer &L, const void *src, void *dst, int n_experts, hipStream_t st);
hipError_t launch_pack_scales(const Layer &L, const void *src, void *dst, int n_experts, hipStream_t st);
hipError_t launch_w13(const Layer &L, const void *expert_w, const void *scales, const void *x, int T, int k,
                      const int32_t *meta, const int32_t *tok_of, float *h, hipStream_t st);
hipError_t launch_w2(const Layer &L, const void *expert_w, const void *scales, int T, int k, const int32_t *meta,
                     const float *h, float *o, hipStream_t st);
hipError_t launch_w13_mfma(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                           const int32_t *meta, const int32_t *tok_of, const Workspace &ws, hipStream_t st);
hipError_t launch_w2_mfma(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                          const int32_t *meta, const Workspace &ws, hipStream_t st);
hipError_t launch_w13_nvfp4(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                            const int32_t *meta, const int32_t *tok_of, const Workspace &ws, hipStream_t st);
hipError_t launch_w2_nvfp4(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                           const int32_t *meta, const Workspace &ws, hipStream_t st);
hipError_t launch_combine(const Layer &L, int T, int k, const int32_t *slot_of, const float *wts, const float *o,
                          void *y, hipStream_t st);

}  // namespace moe
