// Grouped expert kernels of the MoE decode step: the gate/up projection with the
// fused SiLU-gate epilogue, the down projection, and the weighted combine.
//
// Decode streams each activated expert's weights once per step and applies them to
// the few tokens routed to it, so these kernels are bound by HBM bandwidth (the
// weight-read-dominated decode of the paper's Background section).  Weights stay in
// their stored format in HBM and are dequantised in registers.
//
// GEMV path layout.  A work item is a tile of rows of one activated expert.  Each
// wave owns 8 row groups of 8 lanes; a row group streams two weight rows (gate row i
// and up row i for the gate/up projection, rows n and n+8 for the down projection),
// lane c of the group taking one 16-byte load per block of 128 FP8 (256 E2M1)
// inputs.  Weight loads are issued in chunks of kD blocks, double-buffered in
// registers, and the first chunk is in flight while the expert's tokens are staged
// in LDS.  Each weight is converted once and reused for every token of the pass.
#include <hip/hip_runtime.h>
#include <math.h>

#include "moe_internal.h"

namespace moe {
namespace {

typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2 __attribute__((ext_vector_type(2)));

constexpr int kD = 2;     // weight blocks per prefetch chunk
constexpr int kMaxM = 4;  // tokens per pass over a weight tile (larger groups run on MFMA tiles)

typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));

__device__ inline bf16x2 as_bf16x2(uint32_t u) { return __builtin_bit_cast(bf16x2, u); }

// Streaming 16-byte weight load (non-temporal: each weight is read once per step).
__device__ inline uint4 load_stream16(const uint8_t *p)
{
    const u32x4 v = __builtin_nontemporal_load(reinterpret_cast<const u32x4 *>(p));
    return make_uint4(v.x, v.y, v.z, v.w);
}

__device__ inline uint32_t f32_to_bf16_rne(float f)
{
    uint32_t u = __float_as_uint(f);
    u += 0x7FFFu + ((u >> 16) & 1u);
    return u >> 16;
}

// E8M0 code -> fp32 power of two (codes 0 and 255 are outside the contract).
__device__ inline float e8m0_to_f32(uint32_t code) { return __uint_as_float(code << 23); }

// Wait for this wave's LDS traffic, then a workgroup barrier.  Global loads still in
// flight (the prefetched weights) are not waited for.
__device__ inline void block_sync_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// ------------------------------------------------------------------ per-format block math
//
// A "block" is one lane's 16-byte load: 16 FP8 or 32 E2M1 weights.  cvt() turns it
// into bf16 pairs (exact: E4M3 and scaled E2M1 values fit bf16) or fp32 pairs;
// dot() multiplies the converted block with the matching staged activations.

template <int FMT>
struct Blk;

template <>
struct Blk<0> {  // FP8 E4M3, fp32 block scale applied to the partial dot
    static constexpr int kCols = 16;
    static constexpr int kPairs = 8;
    __device__ static inline void cvt_bf16(const uint4 &w, float /*sc*/, uint32_t (&o)[kPairs])
    {
        const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o[2 * i] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(wd[i], 1.0f, false));
            o[2 * i + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp8(wd[i], 1.0f, true));
        }
    }
    __device__ static inline void cvt_f32(const uint4 &w, float /*sc*/, f32x2 (&o)[kPairs])
    {
        const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o[2 * i] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(wd[i], 1.0f, false);
            o[2 * i + 1] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(wd[i], 1.0f, true);
        }
    }
};

template <>
struct Blk<1> {  // MXFP4: E2M1 pairs, E8M0 scale applied exactly in the conversion
    static constexpr int kCols = 32;
    static constexpr int kPairs = 16;
    __device__ static inline void cvt_bf16(const uint4 &w, float sc, uint32_t (&o)[kPairs])
    {
        const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o[4 * i + 0] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(wd[i], sc, 0));
            o[4 * i + 1] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(wd[i], sc, 1));
            o[4 * i + 2] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(wd[i], sc, 2));
            o[4 * i + 3] = __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_scalef32_pk_bf16_fp4(wd[i], sc, 3));
        }
    }
    __device__ static inline void cvt_f32(const uint4 &w, float sc, f32x2 (&o)[kPairs])
    {
        const uint32_t wd[4] = {w.x, w.y, w.z, w.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            o[4 * i + 0] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[i], sc, 0);
            o[4 * i + 1] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[i], sc, 1);
            o[4 * i + 2] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[i], sc, 2);
            o[4 * i + 3] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(wd[i], sc, 3);
        }
    }
};

template <>
struct Blk<2> {  // NVFP4: E2M1 pairs converted exactly; the two E4M3 scales of the
                 // block's 16-input halves multiply the half dots (see apply_chunk)
    static constexpr int kCols = 32;
    static constexpr int kPairs = 16;
    __device__ static inline void cvt_bf16(const uint4 &w, float /*sc*/, uint32_t (&o)[kPairs])
    {
        Blk<1>::cvt_bf16(w, 1.0f, o);
    }
};

// Converted block . staged activations of one token (bf16 pairs in LDS).
template <int NP>
__device__ inline float dot_bf16(const uint32_t (&wc)[NP], const uint4 *xp)
{
    float p = 0.f;
#pragma unroll
    for (int q = 0; q < NP / 4; ++q) {
        const uint4 xv = xp[q];
        p = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(wc[4 * q + 0]), as_bf16x2(xv.x), p, false);
        p = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(wc[4 * q + 1]), as_bf16x2(xv.y), p, false);
        p = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(wc[4 * q + 2]), as_bf16x2(xv.z), p, false);
        p = __builtin_amdgcn_fdot2_f32_bf16(as_bf16x2(wc[4 * q + 3]), as_bf16x2(xv.w), p, false);
    }
    return p;
}

// Converted block . staged activations of one token (fp32 in LDS).
template <int NP>
__device__ inline float dot_f32(const f32x2 (&wc)[NP], const uint4 *xp)
{
    float p = 0.f;
    const float4 *x4 = reinterpret_cast<const float4 *>(xp);
#pragma unroll
    for (int q = 0; q < NP / 2; ++q) {
        const float4 xv = x4[q];
        p = fmaf(wc[2 * q].x, xv.x, p);
        p = fmaf(wc[2 * q].y, xv.y, p);
        p = fmaf(wc[2 * q + 1].x, xv.z, p);
        p = fmaf(wc[2 * q + 1].y, xv.w, p);
    }
    return p;
}

// ------------------------------------------------------------------ two-row streaming GEMV
//
// State of one row group's pass over two weight rows of K inputs.
template <int FMT>
struct TwoRows {
    const uint8_t *r0, *r1;  // row starts (bytes)
    const float *fs0, *fs1;  // FP8: per-128-input scale rows (uniform over the wave)
    const uint8_t *es0, *es1;  // MXFP4: per-32-input E8M0 rows; NVFP4: per-16-input E4M3 rows
    int nblk;                // K / (16*8) FP8 or K / (32*8) MXFP4 / NVFP4 blocks per lane
    int c;                   // lane within the row group
};

template <int FMT>
struct Chunk {
    uint4 w[kD][2];
    uint32_t e[kD][2];  // MXFP4 scale code; NVFP4 the two E4M3 codes of the block's halves
};

template <int FMT>
__device__ inline void load_chunk(const TwoRows<FMT> &R, int b0, Chunk<FMT> &C)
{
    constexpr int kStride = Blk<FMT>::kCols * 8 / (FMT == 0 ? 1 : 2);  // bytes per block row-step
#pragma unroll
    for (int d = 0; d < kD; ++d) {
        const int b = min(b0 + d, R.nblk - 1);  // clamped: tail blocks are loaded, not used
        const size_t off = (size_t)b * kStride + (size_t)R.c * 16;
        C.w[d][0] = load_stream16(R.r0 + off);
        C.w[d][1] = load_stream16(R.r1 + off);
        if constexpr (FMT == 1) {
            C.e[d][0] = R.es0[b * 8 + R.c];
            C.e[d][1] = R.es1[b * 8 + R.c];
        } else if constexpr (FMT == 2) {
            C.e[d][0] = *reinterpret_cast<const uint16_t *>(R.es0 + 2 * (b * 8 + R.c));
            C.e[d][1] = *reinterpret_cast<const uint16_t *>(R.es1 + 2 * (b * 8 + R.c));
        }
    }
}

// E4M3 code (byte `sel` of v) -> fp32, exact.
__device__ inline float e4m3_to_f32(uint32_t v, int sel)
{
    switch (sel) {
    case 0: return __builtin_amdgcn_cvt_f32_fp8((int)v, 0);
    default: return __builtin_amdgcn_cvt_f32_fp8((int)v, 1);
    }
}

// Half-block dots of an NVFP4 block (pairs [0, 8) and [8, 16)) scaled by their E4M3 codes.
__device__ inline float dot_nvfp4(const uint32_t (&wc)[16], uint32_t codes, const uint4 *xp)
{
    uint32_t lo[8], hi[8];
#pragma unroll
    for (int i = 0; i < 8; ++i) {
        lo[i] = wc[i];
        hi[i] = wc[8 + i];
    }
    const float p0 = dot_bf16<8>(lo, xp), p1 = dot_bf16<8>(hi, xp + 2);
    return fmaf(e4m3_to_f32(codes, 1), p1, e4m3_to_f32(codes, 0) * p0);
}

// Apply one chunk (blocks b0 .. b0+kD-1, those below nblk) to M staged tokens.
template <int FMT, bool AF32, int M>
__device__ inline void apply_chunk(const TwoRows<FMT> &R, int b0, const Chunk<FMT> &C, const uint4 *xs, int xq,
                                   float (&a0)[kMaxM], float (&a1)[kMaxM])
{
    constexpr int NP = Blk<FMT>::kPairs;
    constexpr int XQ_PER_BLK = AF32 ? Blk<FMT>::kCols / 4 : Blk<FMT>::kCols / 8;  // uint4 of activations
#pragma unroll
    for (int d = 0; d < kD; ++d) {
        const int b = b0 + d;
        if (b < R.nblk) {
            const int xoff = (b * 8 + R.c) * XQ_PER_BLK;
            float s0 = 1.f, s1 = 1.f;
            if constexpr (FMT == 0) {
                s0 = R.fs0[b];
                s1 = R.fs1[b];
            }
            if constexpr (AF32) {
                f32x2 c0[NP], c1[NP];
                Blk<FMT>::cvt_f32(C.w[d][0], FMT == 1 ? e8m0_to_f32(C.e[d][0]) : 1.f, c0);
                Blk<FMT>::cvt_f32(C.w[d][1], FMT == 1 ? e8m0_to_f32(C.e[d][1]) : 1.f, c1);
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const uint4 *xp = xs + m * xq + xoff;
                    a0[m] = fmaf(s0, dot_f32<NP>(c0, xp), a0[m]);
                    a1[m] = fmaf(s1, dot_f32<NP>(c1, xp), a1[m]);
                }
            } else if constexpr (FMT == 2) {
                uint32_t c0[NP], c1[NP];
                Blk<FMT>::cvt_bf16(C.w[d][0], 1.f, c0);
                Blk<FMT>::cvt_bf16(C.w[d][1], 1.f, c1);
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const uint4 *xp = xs + m * xq + xoff;
                    a0[m] += dot_nvfp4(c0, C.e[d][0], xp);
                    a1[m] += dot_nvfp4(c1, C.e[d][1], xp);
                }
            } else {
                uint32_t c0[NP], c1[NP];
                Blk<FMT>::cvt_bf16(C.w[d][0], FMT == 1 ? e8m0_to_f32(C.e[d][0]) : 1.f, c0);
                Blk<FMT>::cvt_bf16(C.w[d][1], FMT == 1 ? e8m0_to_f32(C.e[d][1]) : 1.f, c1);
#pragma unroll
                for (int m = 0; m < M; ++m) {
                    const uint4 *xp = xs + m * xq + xoff;
                    a0[m] = fmaf(s0, dot_bf16<NP>(c0, xp), a0[m]);
                    a1[m] = fmaf(s1, dot_bf16<NP>(c1, xp), a1[m]);
                }
            }
        }
    }
}

// Stream both rows over all K for M staged tokens.  `A` holds chunk 0 on entry.
template <int FMT, bool AF32, int M>
__device__ inline void stream_rows(const TwoRows<FMT> &R, Chunk<FMT> &A, const uint4 *xs, int xq,
                                   float (&a0)[kMaxM], float (&a1)[kMaxM])
{
    Chunk<FMT> Bc;
    const int nch = (R.nblk + kD - 1) / kD;
    for (int ch = 0; ch < nch; ch += 2) {
        if (ch + 1 < nch) load_chunk<FMT>(R, (ch + 1) * kD, Bc);
        apply_chunk<FMT, AF32, M>(R, ch * kD, A, xs, xq, a0, a1);
        if (ch + 1 >= nch) break;
        if (ch + 2 < nch) load_chunk<FMT>(R, (ch + 2) * kD, A);
        apply_chunk<FMT, AF32, M>(R, (ch + 1) * kD, Bc, xs, xq, a0, a1);
    }
}

template <int FMT, bool AF32>
__device__ inline void stream_rows_m(int m, const TwoRows<FMT> &R, Chunk<FMT> &A, const uint4 *xs, int xq,
                                     float (&a0)[kMaxM], float (&a1)[kMaxM])
{
    switch (m) {
    case 1: stream_rows<FMT, AF32, 1>(R, A, xs, xq, a0, a1); break;
    case 2: stream_rows<FMT, AF32, 2>(R, A, xs, xq, a0, a1); break;
    case 3: stream_rows<FMT, AF32, 3>(R, A, xs, xq, a0, a1); break;
    default: stream_rows<FMT, AF32, 4>(R, A, xs, xq, a0, a1); break;
    }
}

__device__ inline void reduce_row_group(float (&a)[kMaxM], int m)
{
#pragma unroll
    for (int j = 0; j < kMaxM; ++j) {
        if (j < m) {
            a[j] += __shfl_xor(a[j], 1);
            a[j] += __shfl_xor(a[j], 2);
            a[j] += __shfl_xor(a[j], 4);
        }
    }
}

constexpr int kXR = 4;   // activation uint4 held per thread while the weights are in flight

// ------------------------------------------------------------------ gate/up + SiLU-gate
//
// Work item = (active expert, tile of 8*WAVES intermediate rows).  Row group rg of
// wave w owns row i = tile*8*WAVES + 8w + rg and streams its gate and up rows, so the
// epilogue h_i = silu(g_i) * u_i needs no data exchange.
template <int FMT, bool AF32, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void w13_gemv_kernel(const uint8_t *__restrict__ ew,
                                                              const uint8_t *__restrict__ es,
                                                              const void *__restrict__ x,
                                                              const int32_t *__restrict__ meta,
                                                              const int32_t *__restrict__ tok_of,
                                                              float *__restrict__ hbuf, int H, int I, int E,
                                                              size_t ewb, size_t esb, int mmax)
{
    constexpr int NTH = WAVES * 64;
    constexpr int ROWS = 8 * WAVES;
    extern __shared__ uint4 lds4[];
    const MetaIdx mi{E};
    const int tiles = I / ROWS;
    const int n_items = meta[mi.n_gemv()] * tiles;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63, rg = lane >> 3, c = lane & 7;
    const int act_bytes = AF32 ? 4 : 2;
    const int xq = H * act_bytes / 16;  // uint4 per token row
    const size_t rowb = FMT == 0 ? (size_t)H : (size_t)H / 2;

    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int4 rec = reinterpret_cast<const int4 *>(meta + mi.gemv_rec())[item / tiles];
        const int e = rec.x, s0 = rec.y, M = rec.z;
        const int tile = item % tiles;
        const int ibase = tile * ROWS + wave * 8;
        const int i = ibase + rg;
        const uint8_t *we = ew + (size_t)e * ewb;
        const uint8_t *se = es + (size_t)e * esb;
        TwoRows<FMT> R;
        R.r0 = we + (size_t)i * rowb;
        R.r1 = we + (size_t)(I + i) * rowb;
        R.c = c;
        R.nblk = FMT == 0 ? H / 128 : H / 256;
        float tg = 1.f, tu = 1.f;  // NVFP4 matrix scales
        if constexpr (FMT == 0) {
            R.fs0 = (const float *)se + (size_t)(ibase / 128) * (H / 128);
            R.fs1 = R.fs0 + (size_t)(I / 128) * (H / 128);
        } else if constexpr (FMT == 1) {
            R.es0 = se + (size_t)i * (H / 32);
            R.es1 = se + (size_t)(I + i) * (H / 32);
        } else {
            tg = reinterpret_cast<const float *>(se)[0];
            tu = reinterpret_cast<const float *>(se)[1];
            R.es0 = se + 16 + (size_t)i * (H / 16);
            R.es1 = se + 16 + (size_t)(I + i) * (H / 16);
        }
        for (int m0 = 0; m0 < M; m0 += mmax) {
            const int mc = min(mmax, M - m0);
            // token rows of this pass (uniform scalar loads), then their activations
            // into registers, then the first weight chunk, then LDS: the activation
            // wait leaves the weight loads in flight.
            int tk[kMaxM];
#pragma unroll
            for (int m = 0; m < kMaxM; ++m) tk[m] = m < mc ? tok_of[s0 + m0 + m] : 0;
            const int total = mc * xq;
            Chunk<FMT> A;
            for (int r0 = 0; r0 < total; r0 += kXR * NTH) {
                uint4 xv[kXR];
#pragma unroll
                for (int u = 0; u < kXR; ++u) {
                    const int q = r0 + u * NTH + (int)threadIdx.x;
                    if (q < total) {
                        const int m = q / xq;
                        int t = tk[0];
#pragma unroll
                        for (int j = 1; j < kMaxM; ++j) t = m == j ? tk[j] : t;
                        xv[u] = reinterpret_cast<const uint4 *>((const uint8_t *)x + (size_t)t * H * act_bytes)[q - m * xq];
                    }
                }
                if (r0 == 0) load_chunk<FMT>(R, 0, A);
                block_sync_lds();  // the previous pass is done reading LDS
#pragma unroll
                for (int u = 0; u < kXR; ++u) {
                    const int q = r0 + u * NTH + (int)threadIdx.x;
                    if (q < total) lds4[q] = xv[u];
                }
            }
            block_sync_lds();
            float a0[kMaxM] = {}, a1[kMaxM] = {};
            stream_rows_m<FMT, AF32>(mc, R, A, lds4, xq, a0, a1);
            reduce_row_group(a0, mc);
            reduce_row_group(a1, mc);
            if (c == 0) {
#pragma unroll
                for (int m = 0; m < kMaxM; ++m)
                    if (m < mc) {
                        const float g = tg * a0[m], u = tu * a1[m];
                        hbuf[(size_t)(s0 + m0 + m) * I + i] = g / (1.0f + expf(-g)) * u;
                    }
            }
        }
    }
}

// ------------------------------------------------------------------ down projection
//
// Work item = (active expert, tile of 16*WAVES output rows).  Row group rg of wave w
// owns rows n0 = tile*16*WAVES + 16w + rg and n0 + 8.  The expert's SwiGLU
// activations are staged in LDS (rounded to bf16 for bf16 layers, fp32 otherwise).
template <int FMT, bool AF32, int WAVES>
__global__ __launch_bounds__(WAVES * 64) void w2_gemv_kernel(const uint8_t *__restrict__ ew,
                                                             const uint8_t *__restrict__ es,
                                                             const int32_t *__restrict__ meta,
                                                             const float *__restrict__ hbuf,
                                                             float *__restrict__ obuf, int H, int I, int E, size_t ewb,
                                                             size_t esb, int mmax)
{
    constexpr int NTH = WAVES * 64;
    constexpr int ROWS = 16 * WAVES;
    extern __shared__ uint4 lds4[];
    const MetaIdx mi{E};
    const int tiles = H / ROWS;
    const int n_items = meta[mi.n_gemv()] * tiles;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const int lane = threadIdx.x & 63, rg = lane >> 3, c = lane & 7;
    const int xq = AF32 ? I / 4 : I / 8;
    const size_t rowb = FMT == 0 ? (size_t)I : (size_t)I / 2;
    const size_t w2off = FMT == 0 ? (size_t)2 * I * H : (size_t)I * H;

    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int4 rec = reinterpret_cast<const int4 *>(meta + mi.gemv_rec())[item / tiles];
        const int e = rec.x, s0 = rec.y, M = rec.z;
        const int tile = item % tiles;
        const int nbase = tile * ROWS + wave * 16;
        const int n0 = nbase + rg, n1 = n0 + 8;
        const uint8_t *we = ew + (size_t)e * ewb + w2off;
        const uint8_t *se = es + (size_t)e * esb;
        TwoRows<FMT> R;
        R.r0 = we + (size_t)n0 * rowb;
        R.r1 = we + (size_t)n1 * rowb;
        R.c = c;
        R.nblk = FMT == 0 ? I / 128 : I / 256;
        float td = 1.f;  // NVFP4 matrix scale
        if constexpr (FMT == 0) {
            R.fs0 = (const float *)se + (size_t)2 * (I / 128) * (H / 128) + (size_t)(nbase / 128) * (I / 128);
            R.fs1 = R.fs0;
        } else if constexpr (FMT == 1) {
            const uint8_t *sd = se + (size_t)2 * I * (H / 32);
            R.es0 = sd + (size_t)n0 * (I / 32);
            R.es1 = sd + (size_t)n1 * (I / 32);
        } else {
            td = reinterpret_cast<const float *>(se)[2];
            const uint8_t *sd = se + 16 + (size_t)2 * I * (H / 16);
            R.es0 = sd + (size_t)n0 * (I / 16);
            R.es1 = sd + (size_t)n1 * (I / 16);
        }
        for (int m0 = 0; m0 < M; m0 += mmax) {
            const int mc = min(mmax, M - m0);
            const float *hb = hbuf + (size_t)(s0 + m0) * I;  // the pass's slots are consecutive
            const int total = mc * xq;
            Chunk<FMT> A;
            for (int r0 = 0; r0 < total; r0 += (kXR / 2) * NTH) {
                float4 hv[kXR];  // AF32: one float4 per staged uint4; bf16: two
#pragma unroll
                for (int u = 0; u < kXR / 2; ++u) {
                    const int q = r0 + u * NTH + (int)threadIdx.x;
                    if (q < total) {
                        if constexpr (AF32) {
                            hv[u] = reinterpret_cast<const float4 *>(hb)[q];
                        } else {
                            hv[2 * u] = reinterpret_cast<const float4 *>(hb)[2 * q];
                            hv[2 * u + 1] = reinterpret_cast<const float4 *>(hb)[2 * q + 1];
                        }
                    }
                }
                if (r0 == 0) load_chunk<FMT>(R, 0, A);
                block_sync_lds();
#pragma unroll
                for (int u = 0; u < kXR / 2; ++u) {
                    const int q = r0 + u * NTH + (int)threadIdx.x;
                    if (q < total) {
                        if constexpr (AF32) {
                            lds4[q] = __builtin_bit_cast(uint4, hv[u]);
                        } else {
                            const float4 a = hv[2 * u], b = hv[2 * u + 1];
                            lds4[q] = make_uint4(f32_to_bf16_rne(a.x) | (f32_to_bf16_rne(a.y) << 16),
                                                 f32_to_bf16_rne(a.z) | (f32_to_bf16_rne(a.w) << 16),
                                                 f32_to_bf16_rne(b.x) | (f32_to_bf16_rne(b.y) << 16),
                                                 f32_to_bf16_rne(b.z) | (f32_to_bf16_rne(b.w) << 16));
                        }
                    }
                }
            }
            block_sync_lds();
            float a0[kMaxM] = {}, a1[kMaxM] = {};
            stream_rows_m<FMT, AF32>(mc, R, A, lds4, xq, a0, a1);
            reduce_row_group(a0, mc);
            reduce_row_group(a1, mc);
            if (c == 0) {
#pragma unroll
                for (int m = 0; m < kMaxM; ++m)
                    if (m < mc) {
                        obuf[(size_t)(s0 + m0 + m) * H + n0] = td * a0[m];
                        obuf[(size_t)(s0 + m0 + m) * H + n1] = td * a1[m];
                    }
            }
        }
    }
}

// ------------------------------------------------------------------ combine
//
// y[t] = sum_j w[t,j] * o[slot(t,j)], j ascending; each output element is written by
// exactly one thread, so no atomics and a fixed summation order.  Choices are taken
// eight at a time: their slots and weights first, then their rows of o, so a token
// costs two memory round trips per eight choices rather than two per choice.
template <bool OUTF32>
__global__ __launch_bounds__(256) void combine_kernel(int k, int H, const int32_t *__restrict__ slot_of,
                                                      const float *__restrict__ wts, const float *__restrict__ obuf,
                                                      void *__restrict__ y)
{
    constexpr int U = 8;
    const int t = blockIdx.y;
    const int n = (blockIdx.x * blockDim.x + threadIdx.x) * 4;
    if (n >= H) return;
    float4 acc = make_float4(0.f, 0.f, 0.f, 0.f);
    for (int j0 = 0; j0 < k; j0 += U) {
        const int nu = min(U, k - j0);
        int s[U];
        float w[U];
        float4 v[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            s[u] = slot_of[(size_t)t * k + j0 + min(u, nu - 1)];
            w[u] = wts[(size_t)t * k + j0 + min(u, nu - 1)];
        }
#pragma unroll
        for (int u = 0; u < U; ++u) v[u] = *reinterpret_cast<const float4 *>(obuf + (size_t)s[u] * H + n);
#pragma unroll
        for (int u = 0; u < U; ++u) {
            if (u < nu) {
                acc.x = fmaf(w[u], v[u].x, acc.x);
                acc.y = fmaf(w[u], v[u].y, acc.y);
                acc.z = fmaf(w[u], v[u].z, acc.z);
                acc.w = fmaf(w[u], v[u].w, acc.w);
            }
        }
    }
    if constexpr (OUTF32) {
        *reinterpret_cast<float4 *>((float *)y + (size_t)t * H + n) = acc;
    } else {
        uint2 pk = make_uint2(f32_to_bf16_rne(acc.x) | (f32_to_bf16_rne(acc.y) << 16),
                              f32_to_bf16_rne(acc.z) | (f32_to_bf16_rne(acc.w) << 16));
        *reinterpret_cast<uint2 *>((uint16_t *)y + (size_t)t * H + n) = pk;
    }
}

int grid_for(long items) { return items < 1 ? 1 : (items > 65535 ? 65535 : (int)items); }

// Tokens per pass: as many as fit 64 KiB of LDS, at most kMaxM.
int tokens_per_pass(int K, int act_bytes)
{
    int m = 65536 / (K * act_bytes);
    return m < 1 ? 1 : (m > kMaxM ? kMaxM : m);
}

// Two waves per item while few tokens share an expert (more, smaller items balance
// the CUs when only a handful of experts is active), four otherwise.
int waves_for(int T, int k, int E) { return (long)T * k <= 2L * E ? 2 : 4; }

}  // namespace

hipError_t launch_w13(const Layer &L, const void *expert_w, const void *scales, const void *x, int T, int k,
                      const int32_t *meta, const int32_t *tok_of, float *h, hipStream_t st)
{
    const int max_active = T * k < L.E ? T * k : L.E;
    const int ab = L.act_bf16 ? 2 : 4;
    const int mmax = tokens_per_pass(L.H, ab);
    const size_t lds = (size_t)mmax * L.H * ab;
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
    const int waves = waves_for(T, k, L.E);
#define W13(F, A, WV)                                                                                        \
    w13_gemv_kernel<F, A, WV><<<grid_for((long)max_active * (L.I / (8 * WV))), WV * 64, lds, st>>>(          \
        ew, es, x, meta, tok_of, h, L.H, L.I, L.E, L.expert_w_bytes, L.expert_s_bytes, mmax)
#define W13W(F, A) (waves == 2 ? (W13(F, A, 2)) : (W13(F, A, 4)))
    if (L.wfmt == 0)
        L.act_bf16 ? W13W(0, false) : W13W(0, true);
    else if (L.wfmt == 1)
        L.act_bf16 ? W13W(1, false) : W13W(1, true);
    else
        W13W(2, false);  // NVFP4 layers have bf16 activations
#undef W13W
#undef W13
    return hipGetLastError();
}

hipError_t launch_w2(const Layer &L, const void *expert_w, const void *scales, int T, int k, const int32_t *meta,
                     const float *h, float *o, hipStream_t st)
{
    const int max_active = T * k < L.E ? T * k : L.E;
    const int ab = L.act_bf16 ? 2 : 4;
    const int mmax = tokens_per_pass(L.I, ab);
    const size_t lds = (size_t)mmax * L.I * ab;
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
    const int waves = waves_for(T, k, L.E);
#define W2(F, A, WV)                                                                                          \
    w2_gemv_kernel<F, A, WV><<<grid_for((long)max_active * (L.H / (16 * WV))), WV * 64, lds, st>>>(           \
        ew, es, meta, h, o, L.H, L.I, L.E, L.expert_w_bytes, L.expert_s_bytes, mmax)
#define W2W(F, A) (waves == 2 ? (W2(F, A, 2)) : (W2(F, A, 4)))
    if (L.wfmt == 0)
        L.act_bf16 ? W2W(0, false) : W2W(0, true);
    else if (L.wfmt == 1)
        L.act_bf16 ? W2W(1, false) : W2W(1, true);
    else
        W2W(2, false);
#undef W2W
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
