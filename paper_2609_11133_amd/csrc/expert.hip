// Grouped expert kernels of the MoE decode step: the gate/up projection with the
// fused SiLU-gate epilogue, the down projection, and the weighted combine.
//
// Decode streams each activated expert's weights once per step and applies them to
// the few tokens routed to it, so these kernels are bound by HBM bandwidth (the
// weight-read-dominated decode of the paper's Background section).  Weights stay in
// their stored format in HBM and are dequantised in registers.
#include <hip/hip_runtime.h>
#include <math.h>

#include "moe_internal.h"

namespace moe {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kMC = 4;  // tokens per pass over a weight tile (GEMV path)

__device__ inline bf16x2 as_bf16x2(uint32_t u) { return __builtin_bit_cast(bf16x2, u); }

__device__ inline uint32_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

// E8M0 code -> fp32 power of two (codes 0 and 255 are outside the contract).
__device__ inline float e8m0_to_f32(uint32_t code) { return __uint_as_float(code << 23); }

// 16 FP8-E4M3 weights . 16 bf16 activations -> fp32.  Conversion to bf16 is exact.
__device__ inline float dot16_fp8_bf16(const uint4 &w, const uint4 &xa, const uint4 &xb, float p)
{
    const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
    const uint32_t xd[8] = {xa.x, xa.y, xa.z, xa.w, xb.x, xb.y, xb.z, xb.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(wd[i], 1.0f, false),
                                            as_bf16x2(xd[2 * i]), p, false);
        p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(wd[i], 1.0f, true),
                                            as_bf16x2(xd[2 * i + 1]), p, false);
    }
    return p;
}

// 32 E2M1 weights (low nibble first) times 2^(scale) . 32 bf16 activations -> fp32.
// The conversion applies the power-of-two scale exactly.
__device__ inline float dot32_fp4_bf16(const uint4 &w, float sc, const uint4 (&x)[4], float p)
{
    const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        const uint4 xv = x[i];
        p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(wd[i], sc, 0), as_bf16x2(xv.x),
                                            p, false);
        p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(wd[i], sc, 1), as_bf16x2(xv.y),
                                            p, false);
        p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(wd[i], sc, 2), as_bf16x2(xv.z),
                                            p, false);
        p = __builtin_amdgcn_fdot2_f32_bf16(__builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(wd[i], sc, 3), as_bf16x2(xv.w),
                                            p, false);
    }
    return p;
}

__device__ inline float fma4(const f32x2 &a, const f32x2 &b, const float4 &x, float p)
{
    p = fmaf(a.x, x.x, p);
    p = fmaf(a.y, x.y, p);
    p = fmaf(b.x, x.z, p);
    return fmaf(b.y, x.w, p);
}

// 16 FP8 weights . 16 fp32 activations.
__device__ inline float dot16_fp8_f32(const uint4 &w, const float4 *x, float p)
{
    const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i)
        p = fma4(__builtin_amdgcn_cvt_scalef32_pk_f32_fp8(wd[i], 1.0f, false),
                 __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(wd[i], 1.0f, true), x[i], p);
    return p;
}

// 32 E2M1 weights times 2^(scale) . 32 fp32 activations.
__device__ inline float dot32_fp4_f32(const uint4 &w, float sc, const float4 *x, float p)
{
    const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        p = fma4(__builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[i], sc, 0),
                 __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[i], sc, 1), x[2 * i], p);
        p = fma4(__builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[i], sc, 2),
                 __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[i], sc, 3), x[2 * i + 1], p);
    }
    return p;
}

// Two weight rows (r0, r1) of length K against up to kMC activation rows staged in
// LDS (`xs`, row stride K elements).  A row is split over the 8 lanes of a row
// group: lane c takes 16 FP8 (or 32 E2M1) weights = one 16-byte load per block of
// 128 (256) inputs.  FP8 block scales are per 128 inputs and uniform over the row
// pair (same 128-row block); E8M0 scales are per lane.
template <int FMT, bool AF32>
__device__ inline void gemv_rows(const uint8_t *__restrict__ r0, const uint8_t *__restrict__ r1, const void *s0p,
                                 const void *s1p, const uint4 *__restrict__ xs, int K, int c, int mc,
                                 float (&a0)[kMC], float (&a1)[kMC])
{
    const int xq = AF32 ? K / 4 : K / 8;  // uint4 per staged activation row
    if constexpr (FMT == 0) {
        const float *s0 = (const float *)s0p, *s1 = (const float *)s1p;
        const int KB = K / 128;
#pragma unroll 4
        for (int kb = 0; kb < KB; ++kb) {
            const int col = kb * 128 + c * 16;
            const uint4 w0 = *reinterpret_cast<const uint4 *>(r0 + col);
            const uint4 w1 = *reinterpret_cast<const uint4 *>(r1 + col);
            const float sc0 = s0[kb], sc1 = s1[kb];
#pragma unroll
            for (int m = 0; m < kMC; ++m) {
                if (m < mc) {
                    float p0, p1;
                    if constexpr (AF32) {
                        const float4 *xv = reinterpret_cast<const float4 *>(xs + m * xq + col / 4);
                        p0 = dot16_fp8_f32(w0, xv, 0.f);
                        p1 = dot16_fp8_f32(w1, xv, 0.f);
                    } else {
                        const uint4 xa = xs[m * xq + col / 8], xb = xs[m * xq + col / 8 + 1];
                        p0 = dot16_fp8_bf16(w0, xa, xb, 0.f);
                        p1 = dot16_fp8_bf16(w1, xa, xb, 0.f);
                    }
                    a0[m] = fmaf(sc0, p0, a0[m]);
                    a1[m] = fmaf(sc1, p1, a1[m]);
                }
            }
        }
    } else {
        const uint8_t *s0 = (const uint8_t *)s0p, *s1 = (const uint8_t *)s1p;
        const int KB = K / 256;
#pragma unroll 4
        for (int kb = 0; kb < KB; ++kb) {
            const int col = kb * 256 + c * 32;
            const uint4 w0 = *reinterpret_cast<const uint4 *>(r0 + col / 2);
            const uint4 w1 = *reinterpret_cast<const uint4 *>(r1 + col / 2);
            const float sc0 = e8m0_to_f32(s0[kb * 8 + c]), sc1 = e8m0_to_f32(s1[kb * 8 + c]);
#pragma unroll
            for (int m = 0; m < kMC; ++m) {
                if (m < mc) {
                    if constexpr (AF32) {
                        const float4 *xv = reinterpret_cast<const float4 *>(xs + m * xq + col / 4);
                        a0[m] = dot32_fp4_f32(w0, sc0, xv, a0[m]);
                        a1[m] = dot32_fp4_f32(w1, sc1, xv, a1[m]);
                    } else {
                        const uint4 xv[4] = {xs[m * xq + col / 8], xs[m * xq + col / 8 + 1],
                                             xs[m * xq + col / 8 + 2], xs[m * xq + col / 8 + 3]};
                        a0[m] = dot32_fp4_bf16(w0, sc0, xv, a0[m]);
                        a1[m] = dot32_fp4_bf16(w1, sc1, xv, a1[m]);
                    }
                }
            }
        }
    }
}

__device__ inline void reduce_row_group(float (&a)[kMC])
{
#pragma unroll
    for (int m = 0; m < kMC; ++m) {
        a[m] += __shfl_xor(a[m], 1);
        a[m] += __shfl_xor(a[m], 2);
        a[m] += __shfl_xor(a[m], 4);
    }
}

// ------------------------------------------------------------------ gate/up + SiLU-gate
//
// Work item = (active expert, tile of 32 consecutive intermediate rows).  A 256-thread
// workgroup = 4 waves x 8 row groups; row group rg of wave w owns intermediate row
// i = 32*tile + 8*w + rg and streams both its gate row and its up row, so the epilogue
// h_i = silu(g_i) * u_i needs no data exchange.  Tokens are staged in LDS kMC at a
// time.  Items are spread over the grid with a grid stride.
template <int FMT, bool AF32>
__global__ __launch_bounds__(256) void w13_gemv_kernel(const uint8_t *__restrict__ ew, const uint8_t *__restrict__ es,
                                                       const void *__restrict__ x, const int32_t *__restrict__ meta,
                                                       const int32_t *__restrict__ tok_of, float *__restrict__ hbuf,
                                                       int H, int I, int E, size_t ewb, size_t esb)
{
    extern __shared__ uint4 lds4[];
    const MetaIdx mi{E};
    const int tiles = I / 32;
    const int n_items = meta[mi.n_gemv()] * tiles;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63, rg = lane >> 3, c = lane & 7;
    const int act_bytes = AF32 ? 4 : 2;
    const int xq = H * act_bytes / 16;  // uint4 per token row
    const size_t rowb = FMT == 0 ? (size_t)H : (size_t)H / 2;

    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int e = meta[mi.act_gemv() + item / tiles];
        const int tile = item % tiles;
        const int s0 = meta[mi.offsets() + e];
        const int M = meta[mi.offsets() + e + 1] - s0;
        const int ibase = tile * 32 + wave * 8;
        const int i = ibase + rg;
        const uint8_t *we = ew + (size_t)e * ewb;
        const uint8_t *se = es + (size_t)e * esb;
        const uint8_t *r0 = we + (size_t)i * rowb;
        const uint8_t *r1 = we + (size_t)(I + i) * rowb;
        const void *sg, *su;
        if constexpr (FMT == 0) {
            const float *sf = (const float *)se + (size_t)(ibase / 128) * (H / 128);
            sg = sf;
            su = sf + (size_t)(I / 128) * (H / 128);
        } else {
            sg = se + (size_t)i * (H / 32);
            su = se + (size_t)(I + i) * (H / 32);
        }
        for (int m0 = 0; m0 < M; m0 += kMC) {
            const int mc = min(kMC, M - m0);
            __syncthreads();
            for (int q = threadIdx.x; q < mc * xq; q += blockDim.x) {
                const int m = q / xq, qq = q % xq;
                const int t = tok_of[s0 + m0 + m];
                lds4[q] = reinterpret_cast<const uint4 *>((const uint8_t *)x + (size_t)t * H * act_bytes)[qq];
            }
            __syncthreads();
            float a0[kMC] = {}, a1[kMC] = {};
            gemv_rows<FMT, AF32>(r0, r1, sg, su, lds4, H, c, mc, a0, a1);
            reduce_row_group(a0);
            reduce_row_group(a1);
            if (c == 0) {
#pragma unroll
                for (int m = 0; m < kMC; ++m)
                    if (m < mc) {
                        const float g = a0[m], u = a1[m];
                        hbuf[(size_t)(s0 + m0 + m) * I + i] = g / (1.0f + expf(-g)) * u;
                    }
            }
        }
    }
}

// ------------------------------------------------------------------ down projection
//
// Work item = (active expert, tile of 64 output rows).  Row group rg of wave w owns
// rows n0 = 64*tile + 16*w + rg and n0 + 8.  The expert's SwiGLU activations are
// staged in LDS (rounded to bf16 for bf16 layers, fp32 otherwise).
template <int FMT, bool AF32>
__global__ __launch_bounds__(256) void w2_gemv_kernel(const uint8_t *__restrict__ ew, const uint8_t *__restrict__ es,
                                                      const int32_t *__restrict__ meta,
                                                      const float *__restrict__ hbuf, float *__restrict__ obuf, int H,
                                                      int I, int E, size_t ewb, size_t esb)
{
    extern __shared__ uint4 lds4[];
    const MetaIdx mi{E};
    const int tiles = H / 64;
    const int n_items = meta[mi.n_gemv()] * tiles;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63, rg = lane >> 3, c = lane & 7;
    const int xq = AF32 ? I / 4 : I / 8;
    const size_t rowb = FMT == 0 ? (size_t)I : (size_t)I / 2;
    const size_t w2off = FMT == 0 ? (size_t)2 * I * H : (size_t)I * H;

    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int e = meta[mi.act_gemv() + item / tiles];
        const int tile = item % tiles;
        const int s0 = meta[mi.offsets() + e];
        const int M = meta[mi.offsets() + e + 1] - s0;
        const int nbase = tile * 64 + wave * 16;
        const int n0 = nbase + rg, n1 = n0 + 8;
        const uint8_t *we = ew + (size_t)e * ewb + w2off;
        const uint8_t *se = es + (size_t)e * esb;
        const uint8_t *r0 = we + (size_t)n0 * rowb;
        const uint8_t *r1 = we + (size_t)n1 * rowb;
        const void *sa, *sb;
        if constexpr (FMT == 0) {
            const float *sf = (const float *)se + (size_t)2 * (I / 128) * (H / 128) + (size_t)(nbase / 128) * (I / 128);
            sa = sf;
            sb = sf;
        } else {
            const uint8_t *sd = se + (size_t)2 * I * (H / 32);
            sa = sd + (size_t)n0 * (I / 32);
            sb = sd + (size_t)n1 * (I / 32);
        }
        for (int m0 = 0; m0 < M; m0 += kMC) {
            const int mc = min(kMC, M - m0);
            __syncthreads();
            for (int q = threadIdx.x; q < mc * xq; q += blockDim.x) {
                const int m = q / xq, qq = q % xq;
                const float *hr = hbuf + (size_t)(s0 + m0 + m) * I;
                if constexpr (AF32) {
                    lds4[q] = reinterpret_cast<const uint4 *>(hr)[qq];
                } else {
                    const float4 a = reinterpret_cast<const float4 *>(hr)[2 * qq];
                    const float4 b = reinterpret_cast<const float4 *>(hr)[2 * qq + 1];
                    lds4[q] = make_uint4(f32_to_bf16_rne(a.x) | (f32_to_bf16_rne(a.y) << 16),
                                         f32_to_bf16_rne(a.z) | (f32_to_bf16_rne(a.w) << 16),
                                         f32_to_bf16_rne(b.x) | (f32_to_bf16_rne(b.y) << 16),
                                         f32_to_bf16_rne(b.z) | (f32_to_bf16_rne(b.w) << 16));
                }
            }
            __syncthreads();
            float a0[kMC] = {}, a1[kMC] = {};
            gemv_rows<FMT, AF32>(r0, r1, sa, sb, lds4, I, c, mc, a0, a1);
            reduce_row_group(a0);
            reduce_row_group(a1);
            if (c == 0) {
#pragma unroll
                for (int m = 0; m < kMC; ++m)
                    if (m < mc) {
                        obuf[(size_t)(s0 + m0 + m) * H + n0] = a0[m];
                        obuf[(size_t)(s0 + m0 + m) * H + n1] = a1[m];
                    }
            }
        }
    }
}

// ------------------------------------------------------------------ combine
//
// y[t] = sum_j w[t,j] * o[slot(t,j)], j ascending; each output element is written by
// exactly one thread, so no atomics and a fixed summation order.
template <bool OUTF32>
__global__ __launch_bounds__(256) void combine_kernel(int k, int H, const int32_t *__restrict__ slot_of,
                                                      const float *__restrict__ wts, const float *__restrict__ obuf,
                                                      void *__restrict__ y)
{
    const int t = blockIdx.y;
    const int n = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
    if (n >= H) return;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j = 0; j < k; ++j) {
        const int s = slot_of[(size_t)t * k + j];
        const float w = wts[(size_t)t * k + j];
        const float4 v = *reinterpret_cast<const float4 *>(obuf + (size_t)s * H + n);
        acc.x = fmaf(w, v.x, acc.x);
        acc.y = fmaf(w, v.y, acc.y);
        acc.z = fmaf(w, v.z, acc.z);
        acc.w = fmaf(w, v.w, acc.w);
    }
    if constexpr (OUTF32) {
        *reinterpret_cast<float4 *>((float *)y + (size_t)t * H + n) = acc;
    } else {
        uint2 pk = make_uint2(f32_to_bf16_rne(acc.x) | (f32_to_bf16_rne(acc.y) << 16),
                              f32_to_bf16_rne(acc.z) | (f32_to_bf16_rne(acc.w) << 16));
        *reinterpret_cast<uint2 *>((uint16_t *)y + (size_t)t * H + n) = pk;
    }
}

int grid_for(int items_upper_bound) { return items_upper_bound < 1 ? 1 : (items_upper_bound > 16384 ? 16384 : items_upper_bound); }

}  // namespace

hipError_t launch_w13(const Layer &L, const void *expert_w, const void *scales, const void *x, int T, int k,
                      const int32_t *meta, const int32_t *tok_of, float *h, hipStream_t st)
{
    const int max_active = T * k < L.E ? T * k : L.E;
    dim3 grid(grid_for(max_active * (L.I / 32))), block(256);
    const size_t lds = (size_t)kMC * L.H * (L.act_bf16 ? 2 : 4);
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
#define W13(F, A) \
    w13_gemv_kernel<F, A><<<grid, block, lds, st>>>(ew, es, x, meta, tok_of, h, L.H, L.I, L.E, L.expert_w_bytes, \
                                                     L.expert_s_bytes)
    if (L.wfmt == 0)
        L.act_bf16 ? W13(0, false) : W13(0, true);
    else
        L.act_bf16 ? W13(1, false) : W13(1, true);
#undef W13
    return hipGetLastError();
}

hipError_t launch_w2(const Layer &L, const void *expert_w, const void *scales, int T, int k, const int32_t *meta,
                     const float *h, float *o, hipStream_t st)
{
    const int max_active = T * k < L.E ? T * k : L.E;
    dim3 grid(grid_for(max_active * (L.H / 64))), block(256);
    const size_t lds = (size_t)kMC * L.I * (L.act_bf16 ? 2 : 4);
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
#define W2(F, A) \
    w2_gemv_kernel<F, A><<<grid, block, lds, st>>>(ew, es, meta, h, o, L.H, L.I, L.E, L.expert_w_bytes, L.expert_s_bytes)
    if (L.wfmt == 0)
        L.act_bf16 ? W2(0, false) : W2(0, true);
    else
        L.act_bf16 ? W2(1, false) : W2(1, true);
#undef W2
    return hipGetLastError();
}

hipError_t launch_combine(const Layer &L, int T, int k, const int32_t *slot_of, const float *wts, const float *o,
                          void *y, hipStream_t st)
{
    dim3 grid((L.H / 4 + 255) / 256, T), block(256);
    if (L.act_bf16)
        combine_kernel<false><<<grid, block, 0, st>>>(k, L.H, slot_of, wts, o, y);
    else
        combine_kernel<true><<<grid, block, 0, st>>>(k, L.H, slot_of, wts, o, y);
    return hipGetLastError();
}

}  // namespace moe
