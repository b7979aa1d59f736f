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
    float *h;          // [Tmax*kmax][I] SwiGLU activations per slot
    float *o;          // [Tmax*kmax][H] expert outputs per slot
    int32_t *fb;       // [Tmax][E] 1 where a router logit took the exact fallback path
    size_t bytes;
};

// Layout of the meta block (int32 words).  Offsets depend on E.
struct MetaIdx {
    int E;
    __host__ __device__ int n_active() const { return 0; }
    __host__ __device__ int n_gemv() const { return 1; }
    __host__ __device__ int n_mfma() const { return 2; }
    __host__ __device__ int n_fallback() const { return 3; }
    __host__ __device__ int counts() const { return 8; }                 // [E]
    __host__ __device__ int offsets() const { return 8 + E; }            // [E+1]
    __host__ __device__ int act_gemv() const { return 8 + 2 * E + 1; }   // [E]
    __host__ __device__ int act_mfma() const { return 8 + 3 * E + 1; }   // [E]
    __host__ __device__ int words() const { return 8 + 4 * E + 1; }
};

size_t carve_workspace(int H, int E, int I, int kmax, int Tmax, void *base, Workspace *ws);

// Geometry of one layer as the kernels see it.
struct Layer {
    int H, E, I;
    int wfmt;       // 0 FP8-E4M3 (128x128 fp32 scales), 1 MXFP4 (E8M0 per 32)
    int act_bf16;   // activations bf16 (1) or fp32 (0)
    int router_bf16;
    size_t expert_w_bytes;  // per expert
    size_t expert_s_bytes;  // per expert
};

// ---- launchers (all enqueue on `st`, return hipGetLastError())
hipError_t launch_router(const Layer &L, const void *x, int T, const void *router_w, const float *bias,
                         float *logits, int32_t *fb_flags, hipStream_t st);
hipError_t launch_topk(const Layer &L, const float *logits, int T, int k, int32_t *ids, float *wts,
                       int32_t *ids_user, float *wts_user, hipStream_t st);
hipError_t launch_group(const Layer &L, const int32_t *ids, int T, int k, int mstar, int32_t *meta,
                        int32_t *slot_of, int32_t *tok_of, const int32_t *fb_flags, hipStream_t st);
hipError_t launch_w13(const Layer &L, const void *expert_w, const void *scales, const void *x, int T, int k,
                      const int32_t *meta, const int32_t *tok_of, float *h, hipStream_t st);
hipError_t launch_w2(const Layer &L, const void *expert_w, const void *scales, int T, int k, const int32_t *meta,
                     const float *h, float *o, hipStream_t st);
hipError_t launch_combine(const Layer &L, int T, int k, const int32_t *slot_of, const float *wts, const float *o,
                          void *y, hipStream_t st);

}  // namespace moe
