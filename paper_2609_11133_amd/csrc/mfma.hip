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
// Every wave streams two 16-row weight tiles per work item (see stream_tiles).
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
// issued before block kb is multiplied, so S-1 blocks stay in flight.  Neither the
// prologue nor the steady state has conditional loads: the compiler's wait counts
// are exact only when every path issues the same loads, and a guarded load before
// the loop makes every iteration wait for all outstanding loads.  So the prologue
// always fills S-1 slots, with block KB-1 standing in for blocks past the end, and
// issues them slot by slot: the wait at the top of the loop is one count for the
// path from the prologue and the path from the previous iteration, and a slot's
// loads scheduled after a later slot's (the scheduler likes to sink the byte loads)
// would make it wait for nearly all.
template <int S, typename FR, typename LoadF, typename CompF>
__device__ inline void k_pipeline(int KB, FR (&F)[S], LoadF load, CompF compute)
{
#pragma unroll
    for (int s = 0; s < S - 1; ++s) {
        load(F[s], s < KB ? s : KB - 1);
        __builtin_amdgcn_sched_barrier(0);
    }
    int kb = 0;
    for (; kb + 2 * S - 1 <= KB; kb += S) {
#pragma unroll
        for (int s = 0; s < S; ++s) {
            load(F[(s + S - 1) % S], kb + s + S - 1);
            compute(F[s], kb + s);
        }
    }
    // fewer than 2S-1 blocks remain; block kb+s sits in F[s % S]
#pragma unroll
    for (int s = 0; s < 2 * S - 2; ++s) {
        if (kb + s < KB) {
            if (kb + s + S - 1 < KB) load(F[(s + S - 1) % S], kb + s + S - 1);
            compute(F[s % S], kb + s);
        }
    }
}

// ------------------------------------------------------------------ activation operand
//
// Activation fragments are read through raw buffer resources sized to the step's
// data.  Lanes whose token column lies past the chunk use an offset beyond the
// resource, which the hardware answers with zeros and no memory request: the
// activation traffic through the L1 then scales with the chunk's real tokens, and
// no branch guards the loads (a branch around loads makes every K block wait for
// all outstanding loads).  An output column depends only on its own activation
// column, and columns past the chunk are never stored.

typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kRawBufferWord3 = 0x00020000;  // untyped 32-bit data format, no swizzle

__device__ inline __amdgpu_buffer_rsrc_t raw_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRawBufferWord3);
}

// FP8 fragment of a K block: bytes [16g, 16g+16) and [64+16g, 64+16g+16) at voff+soff.
__device__ inline i32x8 frag_buf(__amdgpu_buffer_rsrc_t r, uint32_t voff, uint32_t soff)
{
    const u32x4v a = __builtin_amdgcn_raw_buffer_load_b128(r, voff, soff, 0);
    const u32x4v b = __builtin_amdgcn_raw_buffer_load_b128(r, voff + 64, soff, 0);
    return (i32x8){(int)a.x, (int)a.y, (int)a.z, (int)a.w, (int)b.x, (int)b.y, (int)b.z, (int)b.w};
}

// The four resources of a split activation buffer [rows][K] (hi, lo codes) and
// [rows][K/32] (hi, lo exponents) holding `rows` rows.
struct ActRsrc {
    __amdgpu_buffer_rsrc_t hi, lo, ehi, elo;
};

__device__ inline ActRsrc act_rsrc(const uint8_t *hi, const uint8_t *lo, const uint8_t *ehi, const uint8_t *elo,
                                   uint32_t rows, uint32_t K)
{
    return ActRsrc{raw_rsrc(hi, rows * K), raw_rsrc(lo, rows * K), raw_rsrc(ehi, rows * (K / 32)),
                   raw_rsrc(elo, rows * (K / 32))};
}

// Weight layouts.  Row-major (PK = false): a matrix [rows][K] with K contiguous.
// Packed 16-row tiles (PK = true): each tile of 16 rows keeps its place and size, and
// inside it each 128-input K block is one contiguous piece holding the operand
// fragments in lane order: FP8 2 KB, lane l's bytes K [16g, 16g+16) of row l%16 at
// 16l and K [64+16g, 64+16g+16) at 1024 + 16l (g = l/16); E2M1 1 KB, lane l's 16
// bytes (K [32g, 32g+32) of row l%16) at 16l.  A load instruction of a wave then reads
// 1 KB of contiguous bytes; on this GPU such a stream runs at 6.8-6.9 TB/s with
// non-temporal loads, against 6.0-6.2 TB/s for the row-major walk with either kind.
// The tile is the same for the whole wave, so packed fragments are read through a
// buffer resource on it (scalar registers), the lane's offset 16l and the block's
// offset as a scalar.  With packed E2M1 weights the E8M0 scales are packed too: inside
// each 16-row tile, per group of four K blocks, lane l's four scale bytes (K sub-block
// g of row l%16 in blocks 4q..4q+3) sit together at 4l of a 256-byte piece (a final
// group of two blocks: 2 bytes per lane, 128 bytes).  Read row by row, one byte per
// lane and block, the scales bound the E2M1 kernels.
constexpr int kNonTemporal = 2;  // cache policy of a non-temporal buffer load

// This lane's weight pointer for the 16-row tile starting at row `row0` (a multiple of
// 16) of a matrix with `rowb` bytes per row: its row (row-major) or the tile (packed).
template <bool PK>
__device__ inline const uint8_t *wlane(const uint8_t *mat, int row0, size_t rowb, int lane)
{
    return PK ? mat + (size_t)row0 * rowb : mat + (size_t)(row0 + (lane & 15)) * rowb;
}

__device__ inline __amdgpu_buffer_rsrc_t tile_rsrc(const uint8_t *tile)
{
    const uint64_t a = (uint64_t)tile;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), (short)0, -1, kRawBufferWord3);
}

// E8M0 scale byte of K block kb (of KB) from a packed tile's scales `et` (byte reads:
// the two-tile kernels; the staged ones read a word per four blocks).
__device__ inline int e8m0_packed(const uint8_t *et, int kb, int KB, int lane)
{
    const int q = kb >> 2, rem = min(4, KB - 4 * q);
    return et[256 * q + lane * rem + (kb & 3)];
}

// Weight operand fragment of K block kb from a pointer of wlane.
template <int FMT, bool PK>
__device__ inline i32x8 wfrag(const uint8_t *a, int kb, int g)
{
    if constexpr (PK) {
        const __amdgpu_buffer_rsrc_t r = tile_rsrc(a);
        const uint32_t v = 16u * (uint32_t)__lane_id();
        if constexpr (FMT == 0) {
            const u32x4v x = __builtin_amdgcn_raw_buffer_load_b128(r, v, kb * 2048, kNonTemporal);
            const u32x4v y = __builtin_amdgcn_raw_buffer_load_b128(r, v + 1024, kb * 2048, kNonTemporal);
            return (i32x8){(int)x.x, (int)x.y, (int)x.z, (int)x.w, (int)y.x, (int)y.y, (int)y.z, (int)y.w};
        } else {
            // ordinary loads for E2M1 tiles: an expert with several token chunks re-reads
            // its tiles, and the non-temporal policy made those re-reads miss the caches
            // (4-bit MXFP4 layer at 256 tokens per step: 1.31x its algorithmic bytes
            // fetched, 997k against 1,036k tokens/s with ordinary loads)
            const u32x4v x = __builtin_amdgcn_raw_buffer_load_b128(r, v, kb * 1024, 0);
            return (i32x8){(int)x.x, (int)x.y, (int)x.z, (int)x.w, 0, 0, 0, 0};
        }
    } else {
        if constexpr (FMT == 0)
            return frag_fp8(a + (size_t)kb * 128, g);
        else
            return frag_fp4(a + (size_t)kb * 64, g);
    }
}

// ------------------------------------------------------------------ two weight tiles
//
// A wave streams two 16-row weight tiles (this lane's rows arow[0], arow[1]) over KB
// K blocks against NT 16-token tiles, accumulating acc[t][j] (lane l: rows 4g..4g+3
// of token column l%16).  Two tiles per wave balance the two costs measured on this
// GPU: each extra concurrently streamed tile lowers the HBM rate (one: 6.3 TB/s,
// four: 5.2 TB/s), each activation fragment load is paid per tile pair.
//   arow[t]  weight row of this lane in tile t (FP8: KB*128 bytes, E2M1: KB*64 bytes)
//   erow[t]  E8M0 scales of that row (E2M1 only), one per 32 inputs
//   sblk[t]  fp32 block scale of tile t per K block (FP8 only)
//   voff[j], eoff[j]  this lane's byte offset of its token row in the code and
//                     exponent buffers (kOutOfRange past the chunk)
template <int FMT, int NT, int S, bool PK>
__device__ inline void stream_tiles(f32x4 (&acc)[2][NT], const uint8_t *const (&arow)[2],
                                    const uint8_t *const (&erow)[2], const float *const (&sblk)[2], int KB,
                                    const ActRsrc &B, const uint32_t (&voff)[NT], const uint32_t (&eoff)[NT], int g)
{
    auto load = [&](Frags<2, NT> &F, int kb) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            F.a[t] = wfrag<FMT, PK>(arow[t], kb, g);
            F.ea[t] = FMT == 0 ? 127 : (PK ? e8m0_packed(erow[t], kb, KB, __lane_id()) : erow[t][kb * 4 + g]);
        }
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            F.bh[j] = frag_buf(B.hi, voff[j], kb * 128);
            F.bl[j] = frag_buf(B.lo, voff[j], kb * 128);
            F.eh[j] = __builtin_amdgcn_raw_buffer_load_b8(B.ehi, eoff[j], kb * 4, 0);
            F.el[j] = __builtin_amdgcn_raw_buffer_load_b8(B.elo, eoff[j], kb * 4, 0);
        }
    };
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[t][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const Frags<2, NT> &F, int kb) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const float s = FMT == 0 ? sblk[t][kb] : 1.f;
#pragma unroll
            for (int j = 0; j < NT; ++j)
                mma2<FMT>(acc[t][j], F.a[t], F.ea[t], s, F.bh[j], F.eh[j], F.bl[j], F.el[j]);
        }
    };
    Frags<2, NT> F[S];
    k_pipeline<S>(KB, F, load, compute);
}

// stream_tiles for a block count KBC fixed at compile time and fully unrolled.  The
// activations' E8M0 exponents of the lane's token rows are read up front, 16 bytes
// (four K blocks) per load, instead of one byte load per block and token tile: on
// the 235B-shaped down projection (12 K blocks) the byte loads were a fifth of the
// K loop's memory instructions.
//   erow_off[j]  byte offset of the lane's token row in the exponent buffers
//                (kOutOfRange past the chunk)
template <int FMT, int NT, int S, int KBC, bool PK>
__device__ inline void stream_tiles_fixed(f32x4 (&acc)[2][NT], const uint8_t *const (&arow)[2],
                                          const uint8_t *const (&erow)[2], const float *const (&sblk)[2],
                                          const ActRsrc &B, const uint32_t (&voff)[NT],
                                          const uint32_t (&erow_off)[NT], int g)
{
    static_assert(KBC % 4 == 0 && S >= 2, "whole 16-byte exponent loads");
    constexpr int Q = KBC / 4;
    u32x4v exh[NT][Q], exl[NT][Q];
#pragma unroll
    for (int j = 0; j < NT; ++j)
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            exh[j][q] = __builtin_amdgcn_raw_buffer_load_b128(B.ehi, erow_off[j], q * 16, 0);
            exl[j][q] = __builtin_amdgcn_raw_buffer_load_b128(B.elo, erow_off[j], q * 16, 0);
        }
    auto load = [&](Frags<2, NT> &F, int kb) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            F.a[t] = wfrag<FMT, PK>(arow[t], kb, g);
            F.ea[t] = FMT == 0 ? 127 : (PK ? e8m0_packed(erow[t], kb, KBC, __lane_id()) : erow[t][kb * 4 + g]);
        }
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            F.bh[j] = frag_buf(B.hi, voff[j], kb * 128);
            F.bl[j] = frag_buf(B.lo, voff[j], kb * 128);
        }
    };
#pragma unroll
    for (int t = 0; t < 2; ++t)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[t][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    auto compute = [&](const Frags<2, NT> &F, int kb) {
#pragma unroll
        for (int t = 0; t < 2; ++t) {
            const float sc = FMT == 0 ? sblk[t][kb] : 1.f;
#pragma unroll
            for (int j = 0; j < NT; ++j) {
                const int eh = (int)__builtin_amdgcn_ubfe(exh[j][kb / 4][kb % 4], 8 * g, 8);
                const int el = (int)__builtin_amdgcn_ubfe(exl[j][kb / 4][kb % 4], 8 * g, 8);
                mma2<FMT>(acc[t][j], F.a[t], F.ea[t], sc, F.bh[j], eh, F.bl[j], el);
            }
        }
    };
    Frags<2, NT> F[S];
#pragma unroll
    for (int kb = 0; kb < S - 1; ++kb) load(F[kb], kb);
#pragma unroll
    for (int kb = 0; kb < KBC; ++kb) {
        if (kb + S - 1 < KBC) load(F[(kb + S - 1) % S], kb + S - 1);
        compute(F[kb % S], kb);
    }
}

// This lane's token-row offsets for the NT token tiles of a chunk.
template <int NT>
__device__ inline void token_offsets(uint32_t (&voff)[NT], uint32_t (&eoff)[NT], const int32_t *__restrict__ row_of,
                                     int slot0, int mc, int K, int r, int g)
{
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int m = 16 * j + r;
        const uint32_t row = m < mc ? (uint32_t)(row_of ? row_of[slot0 + m] : slot0 + m) : 0u;
        voff[j] = m < mc ? row * (uint32_t)K + 16u * g : kOutOfRange;
        eoff[j] = m < mc ? row * (uint32_t)(K / 32) + (uint32_t)g : kOutOfRange;
    }
}

// ------------------------------------------------------------------ gate/up + SiLU-gate
//
// Work item = (chunk of up to 32 tokens of one expert, rows [i0, i0+64) of the
// intermediate dimension) for a workgroup of four waves.  Wave w takes rows
// r0 = i0 + 16w .. r0+16 of both the gate and the up matrix, so h = silu(g)*u forms
// in its registers.  The 2-term split of h groups 32 rows (one E8M0 exponent per
// token and group): waves 2q and 2q+1 share group q and exchange their column
// maxima through LDS.

template <int FMT, int NT, int S, bool PK>
__device__ inline void w13_rows(int w, const uint8_t *__restrict__ we, const uint8_t *__restrict__ se, int H, int I,
                                int i0, int slot0, int mc, const int32_t *__restrict__ tok_of, const ActRsrc &X,
                                uint8_t *__restrict__ hs_hi, uint8_t *__restrict__ hs_lo,
                                uint8_t *__restrict__ he_hi, uint8_t *__restrict__ he_lo, float (&s_am)[4][2][16],
                                float (&s_rm)[4][2][16], int lane)
{
    const int r = lane & 15, g = lane >> 4;
    const int r0 = i0 + 16 * w;  // first row of this wave in the gate and in the up matrix
    const size_t rowb = FMT == 0 ? (size_t)H : (size_t)H / 2;
    const uint8_t *arow[2] = {wlane<PK>(we, r0, rowb, lane), wlane<PK>(we, I + r0, rowb, lane)};
    const int er = PK ? 0 : r;  // packed scales: the tile's
    const uint8_t *erow[2] = {se + (size_t)(r0 + er) * (H / 32), se + (size_t)(I + r0 + er) * (H / 32)};
    const float *sblk[2] = {(const float *)se + (size_t)(r0 / 128) * (H / 128),
                            (const float *)se + (size_t)((I + r0) / 128) * (H / 128)};
    uint32_t voff[NT], eoff[NT];
    token_offsets<NT>(voff, eoff, tok_of, slot0, mc, H, r, g);
    f32x4 acc[2][NT];
    stream_tiles<FMT, NT, S, PK>(acc, arow, erow, sblk, H / 128, X, voff, eoff, g);

    // epilogue: h = silu(g)*u for rows r0 + 4g + i of token column r of each tile
    float h[NT][4], res[NT][4];
    float am[NT];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const float gi = acc[0][j][i];
            h[j][i] = gi / (1.0f + expf(-gi)) * acc[1][j][i];
        }
        float m = amax_of(h[j]);
        m = fmaxf(m, __shfl_xor(m, 16));
        am[j] = fmaxf(m, __shfl_xor(m, 32));
        if (g == 0) s_am[w][j][r] = am[j];
    }
    __syncthreads();
    int ch[NT];
    uint32_t qh[NT][1], ql[NT][1];
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        ch[j] = exp_for_group(fmaxf(am[j], s_am[w ^ 1][j][r]));
        split_hi(h[j], ch[j], qh[j], res[j]);
        float m = amax_of(res[j]);
        m = fmaxf(m, __shfl_xor(m, 16));
        am[j] = fmaxf(m, __shfl_xor(m, 32));
        if (g == 0) s_rm[w][j][r] = am[j];
    }
    __syncthreads();
#pragma unroll
    for (int j = 0; j < NT; ++j) {
        const int cl = exp_for_group(fmaxf(am[j], s_rm[w ^ 1][j][r]));
        split_lo(res[j], cl, ql[j]);
        if (16 * j + r < mc) {
            const size_t slot = (size_t)slot0 + 16 * j + r;
            *reinterpret_cast<uint32_t *>(hs_hi + slot * I + r0 + 4 * g) = qh[j][0];
            *reinterpret_cast<uint32_t *>(hs_lo + slot * I + r0 + 4 * g) = ql[j][0];
            if ((w & 1) == 0 && g == 0) {
                he_hi[slot * (I / 32) + r0 / 32] = (uint8_t)ch[j];
                he_lo[slot * (I / 32) + r0 / 32] = (uint8_t)cl;
            }
        }
    }
}

template <int FMT, bool PK>
__global__ __launch_bounds__(256) void w13_mfma_kernel(const uint8_t *__restrict__ ew, const uint8_t *__restrict__ es,
                                                       const int32_t *__restrict__ meta,
                                                       const int32_t *__restrict__ tok_of,
                                                       const uint8_t *__restrict__ xs_hi,
                                                       const uint8_t *__restrict__ xs_lo,
                                                       const uint8_t *__restrict__ xe_hi,
                                                       const uint8_t *__restrict__ xe_lo, uint8_t *__restrict__ hs_hi,
                                                       uint8_t *__restrict__ hs_lo, uint8_t *__restrict__ he_hi,
                                                       uint8_t *__restrict__ he_lo, int T, int H, int I, int E,
                                                       size_t ewb, size_t esb)
{
    __shared__ float s_am[4][2][16], s_rm[4][2][16];
    const MetaIdx mi{E};
    const int tiles = I / 64;
    const int n_items = meta[mi.n_mfma_chunks()] * tiles;
    const int4 *recs = reinterpret_cast<const int4 *>(meta + mi.chunk_rec());
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const ActRsrc X = act_rsrc(xs_hi, xs_lo, xe_hi, xe_lo, (uint32_t)T, (uint32_t)H);
    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int4 rec = recs[item / tiles];  // {expert, first slot, tokens, -}
        const int i0 = (item % tiles) * 64;
        const uint8_t *we = ew + (size_t)rec.x * ewb;
        const uint8_t *se = es + (size_t)rec.x * esb;
        if (rec.z > 16)
            w13_rows<FMT, 2, 2, PK>(wave, we, se, H, I, i0, rec.y, rec.z, tok_of, X, hs_hi, hs_lo, he_hi, he_lo, s_am,
                                s_rm, lane);
        else
            w13_rows<FMT, 1, 3, PK>(wave, we, se, H, I, i0, rec.y, rec.z, tok_of, X, hs_hi, hs_lo, he_hi, he_lo, s_am,
                                s_rm, lane);
    }
}

// ------------------------------------------------------------------ down projection
//
// Work item = (chunk of up to 32 tokens of one expert, 32 output rows [n0, n0+32)) for
// one wave; the four waves of a workgroup take consecutive row pairs of a chunk and
// so share its activation fragments through the L1 cache.  A chunk of at most 16
// tokens keeps three K blocks in flight on packed weights (the 480B TP4 shard's down
// projection: 81.7 -> 78.2 us at T=48), two on row-major ones.

template <int FMT, int NT, int S, bool PK>
__device__ inline void w2_rows(const uint8_t *__restrict__ we2, const uint8_t *__restrict__ se, int H, int I, int n0,
                               int slot0, int mc, const ActRsrc &Hs, float *__restrict__ obuf, int lane)
{
    const int r = lane & 15, g = lane >> 4;
    const size_t rowb = FMT == 0 ? (size_t)I : (size_t)I / 2;
    const uint8_t *sd8 = se + (size_t)2 * I * (H / 32);  // MXFP4 down scales
    const uint8_t *arow[2] = {wlane<PK>(we2, n0, rowb, lane), wlane<PK>(we2, n0 + 16, rowb, lane)};
    const int er = PK ? 0 : r;  // packed scales: the tile's
    const uint8_t *erow[2] = {sd8 + (size_t)(n0 + er) * (I / 32), sd8 + (size_t)(n0 + 16 + er) * (I / 32)};
    const float *sd = (const float *)se + (size_t)2 * (I / 128) * (H / 128);
    const float *sblk[2] = {sd + (size_t)(n0 / 128) * (I / 128), sd + (size_t)((n0 + 16) / 128) * (I / 128)};
    uint32_t voff[NT], eoff[NT];
    token_offsets<NT>(voff, eoff, nullptr, slot0, mc, I, r, g);
    f32x4 acc[2][NT];
    if (I == 12 * 128) {  // the 235B-shaped layer
        uint32_t erow_off[NT];
#pragma unroll
        for (int j = 0; j < NT; ++j) erow_off[j] = eoff[j] - (uint32_t)g;
        stream_tiles_fixed<FMT, NT, S, 12, PK>(acc, arow, erow, sblk, Hs, voff, erow_off, g);
    } else {
        stream_tiles<FMT, NT, S, PK>(acc, arow, erow, sblk, I / 128, Hs, voff, eoff, g);
    }
#pragma unroll
    for (int j = 0; j < NT; ++j)
        if (16 * j + r < mc) {
            const size_t slot = (size_t)slot0 + 16 * j + r;
#pragma unroll
            for (int t = 0; t < 2; ++t)
                *reinterpret_cast<f32x4 *>(obuf + slot * H + n0 + 16 * t + 4 * g) = acc[t][j];
        }
}

template <int FMT, bool PK>
__global__ __launch_bounds__(256) void w2_mfma_kernel(const uint8_t *__restrict__ ew, const uint8_t *__restrict__ es,
                                                      const int32_t *__restrict__ meta,
                                                      const uint8_t *__restrict__ hs_hi,
                                                      const uint8_t *__restrict__ hs_lo,
                                                      const uint8_t *__restrict__ he_hi,
                                                      const uint8_t *__restrict__ he_lo, float *__restrict__ obuf,
                                                      int P, int H, int I, int E, size_t ewb, size_t esb)
{
    const MetaIdx mi{E};
    const int tiles = H / 32;
    const int n_items = meta[mi.n_mfma_chunks()] * tiles;
    const int4 *recs = reinterpret_cast<const int4 *>(meta + mi.chunk_rec());
    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);
    const size_t w2off = FMT == 0 ? (size_t)2 * I * H : (size_t)I * H;
    const ActRsrc Hs = act_rsrc(hs_hi, hs_lo, he_hi, he_lo, (uint32_t)P, (uint32_t)I);
    for (int item = blockIdx.x * 4 + wave; item < n_items; item += gridDim.x * 4) {
        const int4 rec = recs[item / tiles];
        const int n0 = (item % tiles) * 32;
        const uint8_t *we2 = ew + (size_t)rec.x * ewb + w2off;
        const uint8_t *se = es + (size_t)rec.x * esb;
        if (rec.z > 16)
            w2_rows<FMT, 2, 2, PK>(we2, se, H, I, n0, rec.y, rec.z, Hs, obuf, lane);
        else
            w2_rows<FMT, 1, PK ? 4 : 3, PK>(we2, se, H, I, n0, rec.y, rec.z, Hs, obuf, lane);
    }
}

// ------------------------------------------------------------------ LDS-staged activations
//
// When K spans a multiple of four 128-input blocks (every production shape), a work
// item is one workgroup of four waves over one chunk, and each wave streams exactly
// one 16-row weight tile with a four-deep register ring.  The chunk's split
// activations are staged once per workgroup in LDS, in double-buffered segments of
// four K blocks, and every wave reads its fragments from there.  Measured on this GPU,
// a wave streaming one tile reaches 6.3 TB/s and one streaming two 5.6 TB/s, but one
// tile per wave pays a full activation fragment per weight fragment when each wave
// fetches its own; staging removes that cost.

constexpr int kSegK = 4;                // K blocks per staged segment
constexpr int kSegBytes = kSegK * 128;  // activation bytes per token row and segment
constexpr int kStageTok = 32;           // token rows of a chunk

struct alignas(16) ActSeg {
    uint8_t code[2][kStageTok][kSegBytes];  // [hi, lo][token][16-byte pieces, swizzled]
    uint8_t ex[2][kStageTok][kSegK * 4];    // [hi, lo][token][E8M0 per 32 inputs]
    uint8_t sink[kSegK * 4];                // target of the threads that stage no exponents
};

// Piece c (16 bytes) of token t's 512-byte segment row is stored at piece swz(c, t):
// the low four bits of the piece index are XORed with the token, so the 16 tokens of a
// fragment read (one 16-lane group) fall on 16 distinct 16-byte bank groups of the
// 64-bank LDS.  A three-bit XOR left pairs of tokens on one bank group: the counters
// showed bank-conflict stalls in about 40 % of the LDS's active cycles.
__device__ inline int swz(int c, int t) { return (c & ~15) | ((c ^ t) & 15); }

__device__ inline void sync_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

// One thread's share of staging a segment for a workgroup of W waves: piece tid%32
// of token rows 2W*q + tid/32 (q < 8*NT/W) in both the hi and lo codes; threads
// tid < 32 also stage token tid's exponent bytes of each.  Every thread issues the
// same loads (tokens past the chunk read out of range), so the loads need no branch.
template <int NT, int W>
struct Stager {
    static_assert(W == 4 || W == 8, "four or eight waves per workgroup");
    static constexpr int Q = 8 * NT / W;
    uint32_t voff[Q];  // byte offset of this thread's piece in its token rows, segment 0
    uint32_t eoff;     // exponent offset of token tid, segment 0 (out of range if none)
    int tok[Q];
    int piece;
    u32x4v code[2][Q];
    u32x4v ex[2];

    __device__ void init(const int32_t *__restrict__ row_of, int slot0, int mc, int K, int tid)
    {
        piece = tid & 31;
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int t = 2 * W * q + (tid >> 5);
            tok[q] = t;
            const uint32_t row = t < mc ? (uint32_t)(row_of ? row_of[slot0 + t] : slot0 + t) : 0u;
            voff[q] = t < mc ? row * (uint32_t)K + 16u * piece : kOutOfRange;
        }
        const uint32_t erow = tid < mc ? (uint32_t)(row_of ? row_of[slot0 + tid] : slot0 + tid) : 0u;
        eoff = (tid < 32 && tid < mc) ? erow * (uint32_t)(K / 32) : kOutOfRange;
    }
    // segment sg (callers clamp it to the last segment)
    __device__ void load(const ActRsrc &B, int sg)
    {
        const uint32_t d = (uint32_t)sg * kSegBytes, de = (uint32_t)sg * (kSegK * 4);
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            code[0][q] = __builtin_amdgcn_raw_buffer_load_b128(B.hi, voff[q] + d, 0, 0);
            code[1][q] = __builtin_amdgcn_raw_buffer_load_b128(B.lo, voff[q] + d, 0, 0);
        }
        ex[0] = __builtin_amdgcn_raw_buffer_load_b128(B.ehi, eoff + de, 0, 0);
        ex[1] = __builtin_amdgcn_raw_buffer_load_b128(B.elo, eoff + de, 0, 0);
    }
    __device__ void store(ActSeg &S, int tid) const
    {
#pragma unroll
        for (int h = 0; h < 2; ++h)
#pragma unroll
            for (int q = 0; q < Q; ++q)
                *reinterpret_cast<u32x4v *>(&S.code[h][tok[q]][swz(piece, tok[q]) * 16]) = code[h][q];
        uint8_t *e0 = tid < 32 ? &S.ex[0][tid][0] : S.sink;
        uint8_t *e1 = tid < 32 ? &S.ex[1][tid][0] : S.sink;
        *reinterpret_cast<u32x4v *>(e0) = ex[0];
        *reinterpret_cast<u32x4v *>(e1) = ex[1];
    }
};

// Streams this wave's NA weight tiles (this lane's rows arow[a]) over KB K blocks (KB a
// multiple of 4) against NT staged token tiles; acc[a][j] as in stream_tiles.  Each
// activation fragment read from LDS feeds the NA tiles' MFMAs.  All W waves of the
// workgroup call it together: it synchronises them once per staged segment (four K
// blocks).  On return no wave reads `seg` any more.
template <int FMT, int NT, int W, int NA, bool PK>
__device__ inline void stream_tile_lds(f32x4 (&acc)[NA][NT], const uint8_t *const (&arow)[NA],
                                       const uint8_t *const (&erow)[NA], const float *const (&sblk)[NA], int KB,
                                       const ActRsrc &B, Stager<NT, W> &st, ActSeg (&seg)[2], int lane, int tid)
{
    const int r = lane & 15, g = lane >> 4;
    const int nseg = KB / kSegK;
    i32x8 A[4][NA];
    int EA[4][NA];
    // packed E8M0 scales: one word per lane, tile and segment of four blocks, a segment ahead
    __amdgpu_buffer_rsrc_t er[NA];
    if constexpr (PK && FMT == 1) {
#pragma unroll
        for (int a = 0; a < NA; ++a) er[a] = tile_rsrc(erow[a]);
    }
    auto eword = [&](uint32_t (&w)[NA], int sg) {
#pragma unroll
        for (int a = 0; a < NA; ++a) {
            if constexpr (PK && FMT == 1)
                w[a] = __builtin_amdgcn_raw_buffer_load_b32(er[a], 4u * lane, sg * 256, 0);
            else
                w[a] = 0u;
        }
    };
    // Packed E8M0 scales are taken from the segment's words when the block is multiplied,
    // not when its weights are loaded: the next segment's words arrive during this one,
    // and reading them at the load of the next segment's first block made every wave
    // wait there for all but its five newest loads (MXFP4 Zipf layer at T=256: gate/up
    // 120.0 -> 118.8 us in four-wave workgroups, 116.0 -> 115.5 us in eight-wave ones).
    uint32_t wc[NA], wn[NA];  // words of the segment being multiplied and of the next one
    auto loadA = [&](int slot, int kb) {
#pragma unroll
        for (int a = 0; a < NA; ++a) {
            A[slot][a] = wfrag<FMT, PK>(arow[a], kb, g);
            if constexpr (FMT == 0)
                EA[slot][a] = 127;
            else if constexpr (!PK)
                EA[slot][a] = erow[a][kb * 4 + g];
        }
    };
    auto compute = [&](int slot, const ActSeg &S, int kk, int kb) {
        float sc[NA];
#pragma unroll
        for (int a = 0; a < NA; ++a) sc[a] = FMT == 0 ? sblk[a][kb] : 1.f;
        if constexpr (FMT == 1 && PK) {
#pragma unroll
            for (int a = 0; a < NA; ++a) EA[slot][a] = (int)__builtin_amdgcn_ubfe(wc[a], 8 * kk, 8);
        }
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            const int t = 16 * j + r;
            const u32x4v h0 = *reinterpret_cast<const u32x4v *>(&S.code[0][t][swz(kk * 8 + g, t) * 16]);
            const u32x4v h1 = *reinterpret_cast<const u32x4v *>(&S.code[0][t][swz(kk * 8 + 4 + g, t) * 16]);
            const u32x4v l0 = *reinterpret_cast<const u32x4v *>(&S.code[1][t][swz(kk * 8 + g, t) * 16]);
            const u32x4v l1 = *reinterpret_cast<const u32x4v *>(&S.code[1][t][swz(kk * 8 + 4 + g, t) * 16]);
            const i32x8 bh = {(int)h0.x, (int)h0.y, (int)h0.z, (int)h0.w, (int)h1.x, (int)h1.y, (int)h1.z, (int)h1.w};
            const i32x8 bl = {(int)l0.x, (int)l0.y, (int)l0.z, (int)l0.w, (int)l1.x, (int)l1.y, (int)l1.z, (int)l1.w};
            const int eh = S.ex[0][t][kk * 4 + g], el = S.ex[1][t][kk * 4 + g];
#pragma unroll
            for (int a = 0; a < NA; ++a) mma2<FMT>(acc[a][j], A[slot][a], EA[slot][a], sc[a], bh, eh, bl, el);
        }
    };
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int j = 0; j < NT; ++j) acc[a][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    eword(wc, 0);
    loadA(0, 0);
    loadA(1, 1);
    loadA(2, 2);
    st.load(B, 0);
    st.store(seg[0], tid);
    st.load(B, nseg > 1 ? 1 : 0);
    sync_lds();
    for (int kb = 0; kb < KB; kb += kSegK) {  // one staged segment per iteration
        const int sg = kb / kSegK;
        const ActSeg &cur = seg[sg & 1];
        eword(wn, min(sg + 1, nseg - 1));  // the last segment's past the end
#pragma unroll
        for (int u = 0; u < kSegK; ++u) {
            // block kb+3 is this segment's, kb+4.. the next one's; past the end: reload the last block.
            // The scheduling barrier keeps each block's loads here: left to itself the
            // scheduler sinks the next segment's loads to the end of the segment, and every
            // segment then starts with a full memory latency.
            loadA((u + 3) & 3, min(kb + u + 3, KB - 1));
            __builtin_amdgcn_sched_barrier(0);
            compute(u, cur, u, kb + u);
        }
#pragma unroll
        for (int a = 0; a < NA; ++a) wc[a] = wn[a];
        st.store(seg[(sg + 1) & 1], tid);
        st.load(B, min(sg + 2, nseg - 1));
        sync_lds();
    }
}

// gate/up: item = (chunk, NA*8W rows of the intermediate dimension) for W waves; wave w
// streams NA gate (w < W/2) or up (w >= W/2) tiles, rows i0 + 16*q for tiles
// q = NA*(w % (W/2)) + a.  The accumulators meet in LDS (over the staging buffer the
// last segment no longer needs) and wave w forms h and its 2-term split for the pairs
// e = w, w + W, ... < NT*NA*W/4 of token tile e % NT and 32-row group e / NT (32 rows are
// one E8M0 group per token).
template <int FMT, int NT, int W, int NA, bool PK>
__device__ inline void w13_item_lds(const uint8_t *__restrict__ we, const uint8_t *__restrict__ se, int H, int I,
                                    int i0, int slot0, int mc, const int32_t *__restrict__ tok_of, const ActRsrc &X,
                                    uint8_t *__restrict__ hs_hi, uint8_t *__restrict__ hs_lo,
                                    uint8_t *__restrict__ he_hi, uint8_t *__restrict__ he_lo, ActSeg (&seg)[2],
                                    int wave, int lane, int tid)
{
    constexpr int HW = W / 2;       // waves per projection
    constexpr int NQ = HW * NA;     // tiles per projection
    constexpr int NG = NQ / 2;      // 32-row groups per item
    const int r = lane & 15, g = lane >> 4;
    const size_t rowb = FMT == 0 ? (size_t)H : (size_t)H / 2;
    const uint8_t *arow[NA];
    const uint8_t *erow[NA];
    const float *sblk[NA];
#pragma unroll
    for (int a = 0; a < NA; ++a) {
        const int row0 = (wave >= HW ? I : 0) + i0 + 16 * (NA * (wave % HW) + a);
        arow[a] = wlane<PK>(we, row0, rowb, lane);
        erow[a] = se + (size_t)(row0 + (PK ? 0 : r)) * (H / 32);
        sblk[a] = (const float *)se + (size_t)(row0 / 128) * (H / 128);
    }
    Stager<NT, W> st;
    st.init(tok_of, slot0, mc, H, tid);
    f32x4 acc[NA][NT];
    stream_tile_lds<FMT, NT, W, NA, PK>(acc, arow, erow, sblk, H / 128, X, st, seg, lane, tid);
    // red[(proj*NQ + q)*NT + j][lane]: 2*NQ*NT*64 f32x4.  Where they fit in seg[1].code,
    // which the next item first writes after its first barrier, no wave still reads red
    // by then; otherwise red starts at seg[0] and a barrier follows its last read.
    constexpr bool kRedAll = sizeof(f32x4) * 2 * NQ * NT * 64 > sizeof(seg[1].code);
    static_assert(sizeof(f32x4) * 2 * NQ * NT * 64 <= sizeof(seg), "reduction buffer");
    f32x4 *red = kRedAll ? reinterpret_cast<f32x4 *>(&seg[0]) : reinterpret_cast<f32x4 *>(&seg[1].code[0][0][0]);
    auto ridx = [&](int proj, int q, int j) { return ((proj * NQ + q) * NT + j) * 64 + lane; };
#pragma unroll
    for (int a = 0; a < NA; ++a)
#pragma unroll
        for (int j = 0; j < NT; ++j) red[ridx(wave / HW, NA * (wave % HW) + a, j)] = acc[a][j];
    sync_lds();
    for (int e = wave; e < NG * NT; e += W) {  // one (group, token tile) per wave and pass
        const int j = e % NT, grp = e / NT;
        const f32x4 g0 = red[ridx(0, 2 * grp, j)], g1 = red[ridx(0, 2 * grp + 1, j)];
        const f32x4 u0 = red[ridx(1, 2 * grp, j)], u1 = red[ridx(1, 2 * grp + 1, j)];
        float h[8], res[8];
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            h[i] = g0[i] / (1.0f + expf(-g0[i])) * u0[i];
            h[4 + i] = g1[i] / (1.0f + expf(-g1[i])) * u1[i];
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
        if (16 * j + r < mc) {
            const size_t slot = (size_t)slot0 + 16 * j + r;
            const int c0 = i0 + 32 * grp;
            uint8_t *ph = hs_hi + slot * I + c0 + 4 * g;
            uint8_t *pl = hs_lo + slot * I + c0 + 4 * g;
            *reinterpret_cast<uint32_t *>(ph) = qh[0];
            *reinterpret_cast<uint32_t *>(ph + 16) = qh[1];
            *reinterpret_cast<uint32_t *>(pl) = ql[0];
            *reinterpret_cast<uint32_t *>(pl + 16) = ql[1];
            if (g == 0) {
                he_hi[slot * (I / 32) + c0 / 32] = (uint8_t)ch;
                he_lo[slot * (I / 32) + c0 / 32] = (uint8_t)cl;
            }
        }
    }
    if constexpr (kRedAll) sync_lds();
}

template <int FMT, int W, int NA, bool PK>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(W == 8 ? (FMT == 1 ? 2 : 4) : 1))) void w13_mfma_lds_kernel(
    const uint8_t *__restrict__ ew, const uint8_t *__restrict__ es, const int32_t *__restrict__ meta,
    const int32_t *__restrict__ tok_of, const uint8_t *__restrict__ xs_hi, const uint8_t *__restrict__ xs_lo,
    const uint8_t *__restrict__ xe_hi, const uint8_t *__restrict__ xe_lo, uint8_t *__restrict__ hs_hi,
    uint8_t *__restrict__ hs_lo, uint8_t *__restrict__ he_hi, uint8_t *__restrict__ he_lo, int T, int H, int I,
    int E, size_t ewb, size_t esb)
{
    __shared__ ActSeg seg[2];
    const MetaIdx mi{E};
    const int tiles = I / (8 * W * NA);
    const int n_items = meta[mi.n_mfma_chunks()] * tiles;
    const int4 *recs = reinterpret_cast<const int4 *>(meta + mi.chunk_rec());
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const ActRsrc X = act_rsrc(xs_hi, xs_lo, xe_hi, xe_lo, (uint32_t)T, (uint32_t)H);
    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int4 rec = recs[item / tiles];  // {expert, first slot, tokens, -}
        const int i0 = (item % tiles) * 8 * W * NA;
        const uint8_t *we = ew + (size_t)rec.x * ewb;
        const uint8_t *se = es + (size_t)rec.x * esb;
        if (rec.z > 16)
            w13_item_lds<FMT, 2, W, NA, PK>(we, se, H, I, i0, rec.y, rec.z, tok_of, X, hs_hi, hs_lo, he_hi, he_lo,
                                            seg, wave, lane, tid);
        else
            w13_item_lds<FMT, 1, W, NA, PK>(we, se, H, I, i0, rec.y, rec.z, tok_of, X, hs_hi, hs_lo, he_hi, he_lo,
                                            seg, wave, lane, tid);
    }
}

// down: item = (chunk, rows [n0, n0+16*NA*W)) for W waves; wave w streams rows
// n0 + 16*(NA*w + a), a < NA.
template <int FMT, int NT, int W, int NA, bool PK>
__device__ inline void w2_item_lds(const uint8_t *__restrict__ we2, const uint8_t *__restrict__ se, int H, int I,
                                   int n0, int slot0, int mc, const ActRsrc &Hs, float *__restrict__ obuf,
                                   ActSeg (&seg)[2], int wave, int lane, int tid)
{
    const int r = lane & 15, g = lane >> 4;
    const size_t rowb = FMT == 0 ? (size_t)I : (size_t)I / 2;
    const uint8_t *arow[NA];
    const uint8_t *erow[NA];
    const float *sblk[NA];
#pragma unroll
    for (int a = 0; a < NA; ++a) {
        const int row0 = n0 + 16 * (NA * wave + a);
        arow[a] = wlane<PK>(we2, row0, rowb, lane);
        erow[a] = se + (size_t)2 * I * (H / 32) + (size_t)(row0 + (PK ? 0 : r)) * (I / 32);
        sblk[a] = (const float *)se + (size_t)2 * (I / 128) * (H / 128) + (size_t)(row0 / 128) * (I / 128);
    }
    Stager<NT, W> st;
    st.init(nullptr, slot0, mc, I, tid);
    f32x4 acc[NA][NT];
    stream_tile_lds<FMT, NT, W, NA, PK>(acc, arow, erow, sblk, I / 128, Hs, st, seg, lane, tid);
#pragma unroll
    for (int j = 0; j < NT; ++j)
        if (16 * j + r < mc) {
            const size_t slot = (size_t)slot0 + 16 * j + r;
#pragma unroll
            for (int a = 0; a < NA; ++a)
                *reinterpret_cast<f32x4 *>(obuf + slot * H + n0 + 16 * (NA * wave + a) + 4 * g) = acc[a][j];
        }
}

template <int FMT, int W, int NA, bool PK>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(W == 8 ? 4 : 1))) void w2_mfma_lds_kernel(
    const uint8_t *__restrict__ ew, const uint8_t *__restrict__ es, const int32_t *__restrict__ meta,
    const uint8_t *__restrict__ hs_hi, const uint8_t *__restrict__ hs_lo, const uint8_t *__restrict__ he_hi,
    const uint8_t *__restrict__ he_lo, float *__restrict__ obuf, int P, int H, int I, int E, size_t ewb, size_t esb)
{
    __shared__ ActSeg seg[2];
    const MetaIdx mi{E};
    const int tiles = H / (16 * W * NA);
    const int n_items = meta[mi.n_mfma_chunks()] * tiles;
    const int4 *recs = reinterpret_cast<const int4 *>(meta + mi.chunk_rec());
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const size_t w2off = FMT == 0 ? (size_t)2 * I * H : (size_t)I * H;
    const ActRsrc Hs = act_rsrc(hs_hi, hs_lo, he_hi, he_lo, (uint32_t)P, (uint32_t)I);
    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int4 rec = recs[item / tiles];
        const int n0 = (item % tiles) * 16 * W * NA;
        const uint8_t *we2 = ew + (size_t)rec.x * ewb + w2off;
        const uint8_t *se = es + (size_t)rec.x * esb;
        if (rec.z > 16)
            w2_item_lds<FMT, 2, W, NA, PK>(we2, se, H, I, n0, rec.y, rec.z, Hs, obuf, seg, wave, lane, tid);
        else
            w2_item_lds<FMT, 1, W, NA, PK>(we2, se, H, I, n0, rec.y, rec.z, Hs, obuf, seg, wave, lane, tid);
    }
}

// Waves per workgroup of the staged kernels.  FP8 weights stream at 4 waves and two
// workgroups per CU: eight waves per CU hold the HBM stream at its best, and more
// waves per CU slowed it (the 235B- and 480B-shaped layers lost 9-18%).  E2M1
// weights carry half the bytes per activation fragment, so the activation staging, not
// HBM, bounds them: 4 waves with several tiles each (kStagedTiles), and 8 waves for the
// three-tile gate/up (kThreeTileWaves), which stage each segment once for more rows.
// Eight-wave workgroups held to 128 VGPRs to run two per CU lost (the MXFP4 layer at
// T=256, one tile per wave: 570k against 604k tokens/s).
template <int FMT>
constexpr int kStagedWaves = 4;
// Weight tiles per wave of the staged kernels (NA).  E2M1 tiles: four on packed weights
// (each staged activation fragment then feeds four tiles; MXFP4 Zipf layer at T=256
// 1,035k -> 1,094k tokens/s), two on row-major ones (four need more than the 256
// registers two waves per SIMD allow there).
template <int FMT, bool PK>
constexpr int kStagedTiles = FMT == 0 ? 1 : (PK ? 4 : 2);
// Packed E2M1 gate/up takes three tiles per wave in eight-wave workgroups (one per CU,
// up to 256 VGPRs) where I is a multiple of 1536: an item then covers 192 rows, a chunk
// a multiple of 8 items, and since consecutive workgroups go round-robin over the 8
// XCDs, tile q of every chunk of one expert runs on one XCD, at about the same time, and
// its later chunks find the weights in that XCD's L2.  At four tiles (12 items per
// chunk at I = 1536) consecutive chunks land 4 XCDs apart.  MXFP4 Zipf layer at T=256:
// three tiles in four-wave workgroups (96 rows, 16 items per chunk) took gate/up fetch
// 760 -> 629 MB and 126.0 -> 120.0 us; eight waves, which stage each activation
// segment once for twice the rows, 120.0 -> 116.0 us (1,124k -> 1,140k tokens/s).
// Padding 12 items to a stride of 16 instead put twice the work on half the XCDs (126 ->
// 138 us).  The down projection stays at four waves (eight: 69.5 -> 72.4 us).
constexpr int kThreeTileWaves = 8;  // waves per workgroup of the three-tile gate/up
template <int FMT, bool PK>
constexpr bool w13_three_tiles(const Layer &L)
{
    return FMT == 1 && PK && L.I % (8 * kThreeTileWaves * 3 * 8) == 0;
}

// Workgroups for `items_per_chunk` items per chunk record, `per_block` items per workgroup.
int mfma_grid(const Layer &L, int T, int k, int items_per_chunk, int per_block)
{
    const long pairs = (long)T * k;
    const long recs = pairs < L.E ? pairs : L.E;
    const long chunks = recs + (pairs + kMfmaChunk - 1) / kMfmaChunk;  // >= number of chunk records
    const long blocks = (chunks * items_per_chunk + per_block - 1) / per_block;
    return blocks < 1 ? 1 : (blocks > 65535 ? 65535 : (int)blocks);
}

template <int FMT, bool PK, int NA, int W = kStagedWaves<FMT>>
hipError_t launch_w13_lds(const Layer &L, const uint8_t *ew, const uint8_t *es, int T, int k, const int32_t *meta,
                          const int32_t *tok_of, const Workspace &ws, hipStream_t st)
{
    dim3 grid(mfma_grid(L, T, k, L.I / (8 * W * NA), 1)), block(64 * W);
    w13_mfma_lds_kernel<FMT, W, NA, PK><<<grid, block, 0, st>>>(ew, es, meta, tok_of, ws.xs_hi, ws.xs_lo, ws.xe_hi, ws.xe_lo,
                                                        ws.hs_hi, ws.hs_lo, ws.he_hi, ws.he_lo, T, L.H, L.I, L.E,
                                                        L.expert_w_bytes, L.expert_s_bytes);
    return hipGetLastError();
}

template <int FMT, bool PK>
hipError_t launch_w2_lds(const Layer &L, const uint8_t *ew, const uint8_t *es, int T, int k, const int32_t *meta,
                         const Workspace &ws, hipStream_t st)
{
    constexpr int W = kStagedWaves<FMT>, NA = kStagedTiles<FMT, PK>;
    dim3 grid(mfma_grid(L, T, k, L.H / (16 * W * NA), 1)), block(64 * W);
    w2_mfma_lds_kernel<FMT, W, NA, PK><<<grid, block, 0, st>>>(ew, es, meta, ws.hs_hi, ws.hs_lo, ws.he_hi, ws.he_lo, ws.o,
                                                       T * k, L.H, L.I, L.E, L.expert_w_bytes, L.expert_s_bytes);
    return hipGetLastError();
}

template <int FMT, bool PK>
hipError_t w13_launch(const Layer &L, const uint8_t *ew, const uint8_t *es, int T, int k, const int32_t *meta,
                      const int32_t *tok_of, const Workspace &ws, hipStream_t st)
{
    if ((L.H / 128) % 4 == 0) {
        if constexpr (FMT == 1 && PK)
            if (w13_three_tiles<FMT, PK>(L))
                return launch_w13_lds<FMT, PK, 3, kThreeTileWaves>(L, ew, es, T, k, meta, tok_of, ws, st);
        return launch_w13_lds<FMT, PK, kStagedTiles<FMT, PK>>(L, ew, es, T, k, meta, tok_of, ws, st);
    }
    dim3 grid(mfma_grid(L, T, k, L.I / 64, 1)), block(256);
    w13_mfma_kernel<FMT, PK><<<grid, block, 0, st>>>(ew, es, meta, tok_of, ws.xs_hi, ws.xs_lo, ws.xe_hi, ws.xe_lo,
                                                     ws.hs_hi, ws.hs_lo, ws.he_hi, ws.he_lo, T, L.H, L.I, L.E,
                                                     L.expert_w_bytes, L.expert_s_bytes);
    return hipGetLastError();
}

template <int FMT, bool PK>
hipError_t w2_launch(const Layer &L, const uint8_t *ew, const uint8_t *es, int T, int k, const int32_t *meta,
                     const Workspace &ws, hipStream_t st)
{
    // Staging pays a per-item prologue; with fewer than 16 K blocks per row (I < 2048)
    // the two-tile kernel measured faster for FP8 weights (235B-shaped layer: 155
    // against 160 us at T=64).  E2M1 weights carry half the bytes per activation
    // fragment, so they always take the staged kernel.
    if ((L.I / 128) % 4 == 0 && (L.I / 128 >= 16 || FMT == 1)) return launch_w2_lds<FMT, PK>(L, ew, es, T, k, meta, ws, st);
    dim3 grid(mfma_grid(L, T, k, L.H / 32, 4)), block(256);
    w2_mfma_kernel<FMT, PK><<<grid, block, 0, st>>>(ew, es, meta, ws.hs_hi, ws.hs_lo, ws.he_hi, ws.he_lo, ws.o, T * k,
                                                    L.H, L.I, L.E, L.expert_w_bytes, L.expert_s_bytes);
    return hipGetLastError();
}

// Row-major expert weights -> packed 16-row tiles (the layout above), one thread per
// 16-byte piece of the destination.  Per expert: the [2I][K = H] gate/up rows, then
// the [H][K = I] down rows; FP8 one byte per input, E2M1 half a byte.  fmt 0 FP8
// (128-input blocks), 1 MXFP4 (128-input blocks), 2 NVFP4 (256-input blocks of the
// bf16 kernels: lane l's bytes [32g, 32g+16) at 16l, [32g+16, 32g+32) at 1024 + 16l).
__global__ void pack_kernel(const uint8_t *__restrict__ src, uint8_t *__restrict__ dst, int64_t n_pieces, int H,
                            int I, int fmt, int64_t expert_bytes)
{
    const bool fp4 = fmt != 0;
    const int blk = fmt == 1 ? 1024 : 2048;     // bytes of a (16-row tile, K block) piece
    const int kbb = fmt == 1 ? 64 : 128;        // bytes of a row per K block
    const int64_t w13 = (int64_t)2 * I * H / (fp4 ? 2 : 1);  // gate/up bytes of an expert
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n_pieces; p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t off = p * 16;                     // destination byte
        const int64_t e = off / expert_bytes, eo = off % expert_bytes;
        const bool down = eo >= w13;
        const int64_t mo = down ? eo - w13 : eo;        // byte within the matrix
        const int64_t rowb = (down ? I : H) / (fp4 ? 2 : 1);
        const int64_t tile = mo / (16 * rowb), to = mo % (16 * rowb);
        const int64_t kb = to / blk;
        const int q = (int)(to % blk) / 16;             // piece within the block
        const int half = fmt == 1 ? 0 : q / 64, l = q % 64;  // 2 KB pieces: two halves of 1 KB
        const int r = l & 15, g = l >> 4;
        const int lb = fmt == 2 ? 32 * g + 16 * half : 16 * g + 64 * half;  // byte within the row's block
        const int64_t so = e * expert_bytes + (down ? w13 : 0) + (tile * 16 + r) * rowb + kb * kbb + lb;
        *reinterpret_cast<uint4 *>(dst + off) = *reinterpret_cast<const uint4 *>(src + so);
    }
}

// MXFP4 E8M0 scales, row-major -> packed 16-row tiles (the layout above): per expert the
// [2I][H/32] gate/up scales, then the [H][I/32] down scales.  One thread per byte of the
// destination.
__global__ void pack_e8m0_kernel(const uint8_t *__restrict__ src, uint8_t *__restrict__ dst, int64_t n_bytes, int H,
                                 int I, int64_t expert_bytes)
{
    const int64_t w13 = (int64_t)2 * I * (H / 32);
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n_bytes; p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t e = p / expert_bytes, eo = p % expert_bytes;
        const bool down = eo >= w13;
        const int64_t mo = down ? eo - w13 : eo;
        const int K = down ? I : H, KB = K / 128;
        const int64_t rowb = K / 32;
        const int64_t tile = mo / (16 * rowb);
        const int o = (int)(mo % (16 * rowb));
        const int nfull = KB / 4;
        int q, rem, oo;
        if (o < 256 * nfull) {
            q = o / 256, rem = 4, oo = o % 256;
        } else {
            q = nfull, rem = KB % 4, oo = o - 256 * nfull;
        }
        const int l = oo / rem, kb = 4 * q + oo % rem, r = l & 15, g = l >> 4;
        dst[p] = src[e * expert_bytes + (down ? w13 : 0) + (tile * 16 + r) * rowb + kb * 4 + g];
    }
}

// NVFP4 E4M3 scales, row-major -> packed 16-row tiles: per matrix [rows][K/16] bytes
// after each expert's 16 bytes of matrix scales.  Per (16-row tile, 256-input block) one
// 256-byte piece, lane l's 4 bytes (scales [4g, 4g+4) of row l%16) at 4l; where the
// matrix's block count K/256 is a multiple of four, per (16-row tile, group of four
// blocks) one 1 KB piece instead, lane l's 16 bytes (its 4 bytes of each block of the
// group, block by block) at 16l.  One thread per 4-byte word of the destination.
__global__ void pack_scales_kernel(const uint8_t *__restrict__ src, uint8_t *__restrict__ dst, int64_t n_words, int H,
                                   int I, int64_t expert_bytes)
{
    const int64_t w13 = (int64_t)2 * I * (H / 16);  // gate/up scale bytes of an expert
    const int64_t body = w13 + (int64_t)H * (I / 16);
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n_words; p += (int64_t)gridDim.x * blockDim.x) {
        const int64_t off = p * 4;                       // byte within the experts' scale bodies
        const int64_t e = off / body, eo = off % body;
        const bool down = eo >= w13;
        const int64_t mo = down ? eo - w13 : eo;
        const int K = down ? I : H;
        const int64_t rowb = K / 16;                     // scale bytes per row
        const int64_t tile = mo / (16 * rowb);
        const int w = (int)(mo % (16 * rowb)) / 4;       // word within the tile's scales
        int l, kb;
        if ((K / 256) % 4 == 0) {
            l = (w % 256) / 4, kb = 4 * (w / 256) + w % 4;
        } else {
            l = w % 64, kb = w / 64;
        }
        const int r = l & 15, g = l >> 4;
        const int64_t base = e * expert_bytes + 16 + (down ? w13 : 0);
        *reinterpret_cast<uint32_t *>(dst + base + mo) =
            *reinterpret_cast<const uint32_t *>(src + base + (tile * 16 + r) * rowb + kb * 16 + 4 * g);
    }
    // the 16 bytes of matrix scales of each expert, unchanged
    const int64_t n_e = n_words * 4 / body;
    for (int64_t p = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; p < n_e * 4; p += (int64_t)gridDim.x * blockDim.x)
        *reinterpret_cast<uint32_t *>(dst + (p / 4) * expert_bytes + (p % 4) * 4) =
            *reinterpret_cast<const uint32_t *>(src + (p / 4) * expert_bytes + (p % 4) * 4);
}

}  // namespace

hipError_t launch_w13_mfma(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                           const int32_t *meta, const int32_t *tok_of, const Workspace &ws, hipStream_t st)
{
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
    if (L.wfmt == 0)
        return L.wlayout ? w13_launch<0, true>(L, ew, es, T, k, meta, tok_of, ws, st)
                         : w13_launch<0, false>(L, ew, es, T, k, meta, tok_of, ws, st);
    return L.wlayout ? w13_launch<1, true>(L, ew, es, T, k, meta, tok_of, ws, st)
                     : w13_launch<1, false>(L, ew, es, T, k, meta, tok_of, ws, st);
}

hipError_t launch_w2_mfma(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                          const int32_t *meta, const Workspace &ws, hipStream_t st)
{
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
    if (L.wfmt == 0)
        return L.wlayout ? w2_launch<0, true>(L, ew, es, T, k, meta, ws, st)
                         : w2_launch<0, false>(L, ew, es, T, k, meta, ws, st);
    return L.wlayout ? w2_launch<1, true>(L, ew, es, T, k, meta, ws, st)
                     : w2_launch<1, false>(L, ew, es, T, k, meta, ws, st);
}

hipError_t launch_pack_scales(const Layer &L, const void *src, void *dst, int n_experts, hipStream_t st)
{
    if (L.wfmt == 1) {
        const int64_t bytes = (int64_t)n_experts * (int64_t)L.expert_s_bytes;
        const int64_t blocks = (bytes + 255) / 256;
        pack_e8m0_kernel<<<(unsigned)(blocks < 16384 ? blocks : 16384), 256, 0, st>>>(
            (const uint8_t *)src, (uint8_t *)dst, bytes, L.H, L.I, (int64_t)L.expert_s_bytes);
        return hipGetLastError();
    }
    const int64_t body = (int64_t)2 * L.I * (L.H / 16) + (int64_t)L.H * (L.I / 16);
    const int64_t words = (int64_t)n_experts * body / 4;
    const int64_t blocks = (words + 255) / 256;
    pack_scales_kernel<<<(unsigned)(blocks < 16384 ? blocks : 16384), 256, 0, st>>>(
        (const uint8_t *)src, (uint8_t *)dst, words, L.H, L.I, (int64_t)L.expert_s_bytes);
    return hipGetLastError();
}

hipError_t launch_pack_weights(const Layer &L, const void *src, void *dst, int n_experts, hipStream_t st)
{
    const int64_t pieces = (int64_t)n_experts * (int64_t)L.expert_w_bytes / 16;
    const int64_t blocks = (pieces + 255) / 256;
    pack_kernel<<<(unsigned)(blocks < 16384 ? blocks : 16384), 256, 0, st>>>(
        (const uint8_t *)src, (uint8_t *)dst, pieces, L.H, L.I, L.wfmt, (int64_t)L.expert_w_bytes);
    return hipGetLastError();
}

}  // namespace moe
