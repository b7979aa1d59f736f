// MFMA path of the grouped expert FFN: experts that received enough tokens in a
// step run as real dense contractions on the CDNA4 scaled matrix cores
// (v_mfma_scale_f32_16x16x128_f8f6f4), consuming the stored FP8-E4M3 or E2M1
// weights directly.  Activations enter as a 2-term FP8 split (hi + lo, E8M0 scale
// per 32 inputs, see fp8split.h): two MFMAs per tile, with the same error as bf16.
//
// Operand layout of the 16x16x128 instruction on gfx950 (pinned by an on-device
// probe): lane l holds row/column l%16; with g = l/16 an FP8 operand holds K
// [16g, 16g+16) and [64+16g, 64+16g+16) (two 16-byte pieces), an E2M1 operand K
// [32g, 32g+32) (16 bytes, low nibble first); the operand scale of lane l covers
// (row/column l%16, K block [32g, 32g+32)); the 16x16 fp32 result gives lane l rows
// 4g..4g+3 of column l%16.
//
// Work item = (32 weight rows, chunk of up to 32 tokens of one expert) for one wave;
// consecutive items walk the row tiles of a chunk, so the four waves of a workgroup
// share the chunk's activation fragments through the L1 cache.
#include <hip/hip_runtime.h>
#include <math.h>

#include "fp8split.h"
#include "moe_internal.h"

namespace moe {
namespace {

typedef int i32x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));

__device__ inline uint4 ld16(const uint8_t *p) { return *reinterpret_cast<const uint4 *>(p); }

// FP8 operand fragment of K block kb (p = row start + kb*128).  Weight fragments use
// ordinary loads: on this path they measured faster than non-temporal ones.
__device__ inline i32x8 frag_fp8(const uint8_t *p, int g)
{
    const uint4 a = ld16(p + 16 * g);
    const uint4 b = ld16(p + 64 + 16 * g);
    return (i32x8){(int)a.x, (int)a.y, (int)a.z, (int)a.w, (int)b.x, (int)b.y, (int)b.z, (int)b.w};
}

// E2M1 operand fragment of K block kb (p = row start + kb*64).
__device__ inline i32x8 frag_fp4(const uint8_t *p, int g)
{
    const uint4 a = ld16(p + 16 * g);
    return (i32x8){(int)a.x, (int)a.y, (int)a.z, (int)a.w, 0, 0, 0, 0};
}

// acc += s * (A . (Bhi*2^eh + Blo*2^el)) for FP8 weights (fp32 block scale s);
// acc += A*2^ea . (...) for E2M1 weights (E8M0 scale ea in the instruction).
template <int FMT>
__device__ inline void mma2(f32x4 &acc, const i32x8 &a, int ea, float s, const i32x8 &bh, int eh, const i32x8 &bl,
                            int el)
{
    if constexpr (FMT == 0) {
        f32x4 t = {0.f, 0.f, 0.f, 0.f};
        t = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bh, t, 0, 0, 0, 127, 0, eh);
        t = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bl, t, 0, 0, 0, 127, 0, el);
        acc += s * t;
    } else {
        acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bh, acc, 4, 0, 0, ea, 0, eh);
        acc = __builtin_amdgcn_mfma_scale_f32_16x16x128_f8f6f4(a, bl, acc, 4, 0, 0, ea, 0, el);
    }
}

// Fragments of one K block: NA weight tiles and NT token tiles.
template <int NA, int NT>
struct Frags {
    i32x8 a[NA];
    int ea[NA];
    i32x8 bh[NT], bl[NT];
    int eh[NT], el[NT];
};

// K loop over KB blocks with an S-stage register ring: the loads of block kb+S-1 are
// issued before block kb is multiplied, so S-1 blocks of weights stay in flight.
template <int S, typename FR, typename LoadF, typename CompF>
__device__ inline void k_pipeline(int KB, FR (&F)[S], LoadF load, CompF compute)
{
#pragma unroll
    for (int s = 0; s < S - 1; ++s)
        if (s < KB) load(F[s], s);
    for (int kb = 0; kb < KB; kb += S) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
            const int cur = kb + s;
            if (cur >= KB) break;
            if (cur + S - 1 < KB) load(F[(s + S - 1) % S], cur + S - 1);
            compute(F[s], cur);
        }
    }
}

// ------------------------------------------------------------------ gate/up + SiLU-gate

template <int FMT, int NT, int S>
__device__ inline void w13_item(const uint8_t *__restrict__ we, const uint8_t *__restrict__ se, int H, int I, int i0,
                                int slot0, int mc, const int32_t *__restrict__ tok_of,
                                const uint8_t *__restrict__ xs_hi, const uint8_t *__restrict__ xs_lo,
                                const uint8_t *__restrict__ xe_hi, const uint8_t *__restrict__ xe_lo,
                                uint8_t *__restrict__ hs_hi, uint8_t *__restrict__ hs_lo, uint8_t *__restrict__ he_hi,
                                uint8_t *__restrict__ he_lo, int lane)
{
    const int r = lane & 15, g = lane >> 4;
    const int KB = H / 128;
    const size_t rowb = FMT == 0 ? (size_t)H : (size_t)H / 2;
    // weight rows of the four tiles: gate [i0, i0+16), gate [i0+16, i0+32), up likewise
    const uint8_t *arow[4];
    const uint8_t *erow[4];
#pragma unroll
    for (int at = 0; at < 4; ++at) {
        const int row = (at < 2 ? 0 : I) + i0 + 16 * (at & 1) + r;
        arow[at] = we + (size_t)row * rowb;
        erow[at] = se + (size_t)row * (H / 32);  // MXFP4 scale rows (gate then up, same stride)
    }
    const float *sg = (const float *)se + (size_t)(i0 / 128) * (H / 128);  // FP8 block scales
    const float *su = sg + (size_t)(I / 128) * (H / 128);
    // this lane's token in each 16-column tile
    int tok[NT];
    bool valid[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int m = 16 * j + r;
        valid[j] = m < mc;
        tok[j] = valid[j] ? tok_of[slot0 + m] : 0;
    }
    auto load = [&](Frags<4, NT> &F, int kb) {
#pragma unroll
        for (int at = 0; at < 4; ++at) {
            if constexpr (FMT == 0) {
                F.a[at] = frag_fp8(arow[at] + (size_t)kb * 128, g);
                F.ea[at] = 127;
            } else {
                F.a[at] = frag_fp4(arow[at] + (size_t)kb * 64, g);
                F.ea[at] = erow[at][kb * 4 + g];
            }
        }
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const size_t xo = (size_t)tok[j] * H + (size_t)kb * 128;
            const size_t eo = (size_t)tok[j] * (H / 32) + kb * 4 + g;
            F.bh[j] = frag_fp8(xs_hi + xo, g);
            F.bl[j] = frag_fp8(xs_lo + xo, g);
            F.eh[j] = xe_hi[eo];
            F.el[j] = xe_lo[eo];
            if (!valid[j]) {
                F.bh[j] = (i32x8){0, 0, 0, 0, 0, 0, 0, 0};
                F.bl[j] = F.bh[j];
            }
        }
    };
    f32x4 acc[4][NT];
#pragma unroll
    for (int at = 0; at < 4; ++at)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[at][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const Frags<4, NT> &F, int kb) {
        const float s_g = FMT == 0 ? sg[kb] : 1.f, s_u = FMT == 0 ? su[kb] : 1.f;
#pragma unroll
        for (int at = 0; at < 4; ++at)
#pragma unroll
            for (int j = 0; j < NT; ++j)
                mma2<FMT>(acc[at][j], F.a[at], F.ea[at], at < 2 ? s_g : s_u, F.bh[j], F.eh[j], F.bl[j], F.el[j]);
    };
    Frags<4, NT> F[S];
    k_pipeline<S>(KB, F, load, compute);
    // epilogue: h = silu(g) * u for rows i0 + {4g+i, 16+4g+i}, then the 2-term split of
    // the 32-row group [i0, i0+32) of each token (the group spans the four lanes of a
    // column: l, l^16, l^32, l^48).
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        float h[8], res[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float g0 = acc[0][j][i], g1 = acc[1][j][i];
            h[i] = g0 / (1.0f + expf(-g0)) * acc[2][j][i];
            h[4 + i] = g1 / (1.0f + expf(-g1)) * acc[3][j][i];
        }
        float am = amax_of(h);
        am = fmaxf(am, __shfl_xor(am, 16));
        am = fmaxf(am, __shfl_xor(am, 32));
        const int ch = exp_for_group(am);
        uint32_t qh[2], ql[2];
        split_hi(h, ch, qh, res);
        float rm = amax_of(res);
        rm = fmaxf(rm, __shfl_xor(rm, 16));
        rm = fmaxf(rm, __shfl_xor(rm, 32));
        const int cl = exp_for_group(rm);
        split_lo(res, cl, ql);
        if (valid[j]) {
            const size_t slot = (size_t)slot0 + 16 * j + r;
            uint8_t *ph = hs_hi + slot * I + i0 + 4 * g;
            uint8_t *pl = hs_lo + slot * I + i0 + 4 * g;
            *reinterpret_cast<uint32_t *>(ph) = qh[0];
            *reinterpret_cast<uint32_t *>(ph + 16) = qh[1];
            *reinterpret_cast<uint32_t *>(pl) = ql[0];
            *reinterpret_cast<uint32_t *>(pl + 16) = ql[1];
            if (g == 0) {
                he_hi[slot * (I / 32) + i0 / 32] = (uint8_t)ch;
                he_lo[slot * (I / 32) + i0 / 32] = (uint8_t)cl;
            }
        }
    }
}

template <int FMT>
__global__ __launch_bounds__(256) void w13_mfma_kernel(const uint8_t *__restrict__ ew, const uint8_t *__restrict__ es,
                                                       const int32_t *__restrict__ meta,
                                                       const int32_t *__restrict__ tok_of,
                                                       const uint8_t *__restrict__ xs_hi,
                                                       const uint8_t *__restrict__ xs_lo,
                                                       const uint8_t *__restrict__ xe_hi,
                                                       const uint8_t *__restrict__ xe_lo, uint8_t *__restrict__ hs_hi,
                                                       uint8_t *__restrict__ hs_lo, uint8_t *__restrict__ he_hi,
                                                       uint8_t *__restrict__ he_lo, int H, int I, int E, size_t ewb,
                                                       size_t esb)
{
    const MetaIdx mi{E};
    const int tiles = I / 32;
    const int n_items = meta[mi.n_mfma_chunks()] * tiles;
    const int4 *recs = reinterpret_cast<const int4 *>(meta + mi.chunk_rec());
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    for (int item = blockIdx.x * 4 + wave; item < n_items; item += gridDim.x * 4) {
        const int4 rec = recs[item / tiles];  // {expert, first slot, tokens, -}
        const int i0 = (item % tiles) * 32;
        const uint8_t *we = ew + (size_t)rec.x * ewb;
        const uint8_t *se = es + (size_t)rec.x * esb;
        if (rec.z > 16)
            w13_item<FMT, 2, 2>(we, se, H, I, i0, rec.y, rec.z, tok_of, xs_hi, xs_lo, xe_hi, xe_lo, hs_hi, hs_lo,
                                he_hi, he_lo, lane);
        else
            w13_item<FMT, 1, 3>(we, se, H, I, i0, rec.y, rec.z, tok_of, xs_hi, xs_lo, xe_hi, xe_lo, hs_hi, hs_lo,
                                he_hi, he_lo, lane);
    }
}

// ------------------------------------------------------------------ down projection

template <int FMT, int NT, int S>
__device__ inline void w2_item(const uint8_t *__restrict__ we2, const uint8_t *__restrict__ se, int H, int I, int n0,
                               int slot0, int mc, const uint8_t *__restrict__ hs_hi,
                               const uint8_t *__restrict__ hs_lo, const uint8_t *__restrict__ he_hi,
                               const uint8_t *__restrict__ he_lo, float *__restrict__ obuf, int lane)
{
    const int r = lane & 15, g = lane >> 4;
    const int KB = I / 128;
    const size_t rowb = FMT == 0 ? (size_t)I : (size_t)I / 2;
    const uint8_t *arow[2];
    const uint8_t *erow[2];
    const uint8_t *sd8 = se + (size_t)2 * I * (H / 32);  // MXFP4 down scales
#pragma unroll
    for (int at = 0; at < 2; ++at) {
        const int row = n0 + 16 * at + r;
        arow[at] = we2 + (size_t)row * rowb;
        erow[at] = sd8 + (size_t)row * (I / 32);
    }
    const float *sd = (const float *)se + (size_t)2 * (I / 128) * (H / 128) + (size_t)(n0 / 128) * (I / 128);
    size_t slot[NT];
    bool valid[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int m = 16 * j + r;
        valid[j] = m < mc;
        slot[j] = (size_t)slot0 + (valid[j] ? m : 0);
    }
    auto load = [&](Frags<2, NT> &F, int kb) {
#pragma unroll
        for (int at = 0; at < 2; ++at) {
            if constexpr (FMT == 0) {
                F.a[at] = frag_fp8(arow[at] + (size_t)kb * 128, g);
                F.ea[at] = 127;
            } else {
                F.a[at] = frag_fp4(arow[at] + (size_t)kb * 64, g);
                F.ea[at] = erow[at][kb * 4 + g];
            }
        }
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const size_t ho = slot[j] * I + (size_t)kb * 128;
            const size_t eo = slot[j] * (I / 32) + kb * 4 + g;
            F.bh[j] = frag_fp8(hs_hi + ho, g);
            F.bl[j] = frag_fp8(hs_lo + ho, g);
            F.eh[j] = he_hi[eo];
            F.el[j] = he_lo[eo];
            if (!valid[j]) {
                F.bh[j] = (i32x8){0, 0, 0, 0, 0, 0, 0, 0};
                F.bl[j] = F.bh[j];
            }
        }
    };
    f32x4 acc[2][NT];
#pragma unroll
    for (int at = 0; at < 2; ++at)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[at][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const Frags<2, NT> &F, int kb) {
        const float s = FMT == 0 ? sd[kb] : 1.f;
#pragma unroll
        for (int at = 0; at < 2; ++at)
#pragma unroll
            for (int j = 0; j < NT; ++j) mma2<FMT>(acc[at][j], F.a[at], F.ea[at], s, F.bh[j], F.eh[j], F.bl[j], F.el[j]);
    };
    Frags<2, NT> F[S];
    k_pipeline<S>(KB, F, load, compute);
#pragma unroll
    for (int j = 0; j < NT; ++j)
        if (valid[j])
#pragma unroll
            for (int at = 0; at < 2; ++at)
                *reinterpret_cast<f32x4 *>(obuf + slot[j] * H + n0 + 16 * at + 4 * g) = acc[at][j];
}

template <int FMT>
__global__ __launch_bounds__(256) void w2_mfma_kernel(const uint8_t *__restrict__ ew, const uint8_t *__restrict__ es,
                                                      const int32_t *__restrict__ meta,
                                                      const uint8_t *__restrict__ hs_hi,
                                                      const uint8_t *__restrict__ hs_lo,
                                                      const uint8_t *__restrict__ he_hi,
                                                      const uint8_t *__restrict__ he_lo, float *__restrict__ obuf,
                                                      int H, int I, int E, size_t ewb, size_t esb)
{
    const MetaIdx mi{E};
    const int tiles = H / 32;
    const int n_items = meta[mi.n_mfma_chunks()] * tiles;
    const int4 *recs = reinterpret_cast<const int4 *>(meta + mi.chunk_rec());
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const size_t w2off = FMT == 0 ? (size_t)2 * I * H : (size_t)I * H;
    for (int item = blockIdx.x * 4 + wave; item < n_items; item += gridDim.x * 4) {
        const int4 rec = recs[item / tiles];
        const int n0 = (item % tiles) * 32;
        const uint8_t *we2 = ew + (size_t)rec.x * ewb + w2off;
        const uint8_t *se = es + (size_t)rec.x * esb;
        if (rec.z > 16)
            w2_item<FMT, 2, 2>(we2, se, H, I, n0, rec.y, rec.z, hs_hi, hs_lo, he_hi, he_lo, obuf, lane);
        else
            w2_item<FMT, 1, 3>(we2, se, H, I, n0, rec.y, rec.z, hs_hi, hs_lo, he_hi, he_lo, obuf, lane);
    }
}

int mfma_grid(const Layer &L, int T, int k, int tiles)
{
    const long pairs = (long)T * k;
    const long recs = pairs < L.E ? pairs : L.E;
    const long chunks = recs + (pairs + kMfmaChunk - 1) / kMfmaChunk;  // >= number of chunk records
    const long blocks = (chunks * tiles + 3) / 4;
    return blocks < 1 ? 1 : (blocks > 65535 ? 65535 : (int)blocks);
}

}  // namespace

hipError_t launch_w13_mfma(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                           const int32_t *meta, const int32_t *tok_of, const Workspace &ws, hipStream_t st)
{
    dim3 grid(mfma_grid(L, T, k, L.I / 32)), block(256);
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
    if (L.wfmt == 0)
        w13_mfma_kernel<0><<<grid, block, 0, st>>>(ew, es, meta, tok_of, ws.xs_hi, ws.xs_lo, ws.xe_hi, ws.xe_lo,
                                                   ws.hs_hi, ws.hs_lo, ws.he_hi, ws.he_lo, L.H, L.I, L.E,
                                                   L.expert_w_bytes, L.expert_s_bytes);
    else
        w13_mfma_kernel<1><<<grid, block, 0, st>>>(ew, es, meta, tok_of, ws.xs_hi, ws.xs_lo, ws.xe_hi, ws.xe_lo,
                                                   ws.hs_hi, ws.hs_lo, ws.he_hi, ws.he_lo, L.H, L.I, L.E,
                                                   L.expert_w_bytes, L.expert_s_bytes);
    return hipGetLastError();
}

hipError_t launch_w2_mfma(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                          const int32_t *meta, const Workspace &ws, hipStream_t st)
{
    dim3 grid(mfma_grid(L, T, k, L.H / 32)), block(256);
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
    if (L.wfmt == 0)
        w2_mfma_kernel<0><<<grid, block, 0, st>>>(ew, es, meta, ws.hs_hi, ws.hs_lo, ws.he_hi, ws.he_lo, ws.o, L.H,
                                                  L.I, L.E, L.expert_w_bytes, L.expert_s_bytes);
    else
        w2_mfma_kernel<1><<<grid, block, 0, st>>>(ew, es, meta, ws.hs_hi, ws.hs_lo, ws.he_hi, ws.he_lo, ws.o, L.H,
                                                  L.I, L.E, L.expert_w_bytes, L.expert_s_bytes);
    return hipGetLastError();
}

}  // namespace moe
