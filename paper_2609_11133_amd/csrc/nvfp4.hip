// NVFP4 path of the grouped expert FFN on the bf16 matrix cores.
//
// NVFP4 weights are E2M1 codes with one E4M3 scale per 16 inputs and one fp32 scale
// per matrix.  The scaled f8f6f4 MFMA takes E8M0 (power-of-two) scales per 32 inputs
// only, and the gfx950 conversions with an fp32 scale apply only its exponent (checked
// on the device), so a 16-input E4M3 scale cannot ride along with the stored codes.
// Each weight is therefore converted in registers: E2M1 -> fp32 (exact), times its
// block scale (exact in fp32), packed to bf16 (exact: an E2M1 value times an E4M3
// scale has at most 6 significant bits).  The activations are the layer's bf16 x
// itself and, for the down projection, h rounded once to bf16; the 16x16x32 bf16 MFMA
// accumulates in fp32 and the matrix scales multiply the accumulators.
//
// The gate/up projection runs on f16 operands instead, which halves the conversion
// work that bounds it: an E2M1 pair converts to f16 with the block scale's power of
// two applied by the conversion, and one packed f16 multiply applies the scale's
// mantissa 1 + j/8 (every product has at most 5 significant bits and lies in
// [2^-13, 2688]: exact).  x enters as the routing kernel's f16 copy x * 2^-k (k per
// token, so that every value at least 2^-31 of the token's maximum converts exactly),
// and the accumulators are multiplied by 2^k.
//
// Operand layout of v_mfma_f32_16x16x32_bf16 (checked on the device): lane l holds
// row/column l%16 and K [8g, 8g+8) with g = l/16; the result gives lane l rows
// 4g..4g+3 of column l%16.  The K order inside one instruction is free as long as
// both operands agree.  A K block is 256 inputs (128 weight bytes per row, the access
// shape of the FP8 kernels); instruction q (0..7) of a block takes, in lane group g,
// the inputs [64g + 8q, 64g + 8q + 8), so a lane's 32 contiguous weight bytes (inputs
// [64g, 64g+64)) feed all eight and one 32-bit load brings their four block scales.
//
// Weights are row-major or packed in 16-row tiles (PK): each 256-input block of a tile
// is one contiguous 2 KB piece, lane l's weight bytes [32g, 32g+16) of row l%16 at 16l and
// [32g+16, 32g+32) at 1024 + 16l, read with non-temporal buffer loads off the tile (a
// wave-uniform resource), so each load instruction of a wave reads 1 KB of contiguous
// bytes.  The E4M3 scales are packed the same way: a block's 16 rows x 16 scales are one
// 256-byte piece, lane l's four (scales [4g, 4g+4) of row l%16) at 4l; where a matrix's
// block count is a multiple of four, per group of four blocks one 1 KB piece instead,
// lane l's 16 bytes (its four scales of each block of the group, block by block) at 16l,
// so one 16-byte load per lane brings four blocks' scales (GS below).  Read row by row,
// the scales were the packed kernels' bound (16 segments of 16 bytes per load), and one
// 32-bit load per lane and block still cost about a tenth of the gate/up kernel's time.
//
// Work items follow the FP8 staged kernels (mfma.hip): one workgroup of W waves per
// (chunk of <= 32 tokens of one expert, rows), one 16-row weight tile per wave through
// a four-deep register ring, the chunk's activations staged once per workgroup in LDS
// (double-buffered segments of 512 inputs, 16-byte pieces XOR-swizzled by token).
#include <hip/hip_runtime.h>
#include <math.h>

#include "moe_internal.h"

namespace moe {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));

constexpr uint32_t kOutOfRange = 0x80000000u;
constexpr int kRawBufferWord3 = 0x00020000;  // untyped 32-bit data format, no swizzle
constexpr int kNonTemporal = 2;              // cache policy of a non-temporal buffer load

constexpr int kBlk = 256;                 // inputs per K block
constexpr int kSegBlk = 2;                // K blocks per staged segment
constexpr int kRowBytes = kSegBlk * kBlk * 2;  // bf16 bytes of one token row per segment
constexpr int kTok = 32;                  // token rows of a chunk

// A staged segment of ROWS token rows.
template <int ROWS>
struct alignas(16) SegT {
    uint8_t row[ROWS][kRowBytes];
};
using Seg = SegT<kTok>;

// Piece p (16 bytes) of token t's segment row is stored at piece swz(p, t): the low
// four bits of the piece index are XORed with the token's low three bits.  A fragment
// read gives lane (token r, group g) piece 8g + q of a block.  Measured in an LDS probe
// at eight waves per CU, cycles per 1 KB ds_read_b128: 5.2 for these reads (one or two
// token tiles) and for contiguous ones; 8.1, two-way bank conflicts, when all four
// token bits were XORed in.  The stager's row writes run at the same rate either way.
__device__ inline int swz(int p, int t) { return (p & ~15) | ((p ^ (t & 7)) & 15); }

__device__ inline void sync_lds() { asm volatile("s_waitcnt lgkmcnt(0)\n\ts_barrier" ::: "memory"); }

__device__ inline __amdgpu_buffer_rsrc_t raw_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRawBufferWord3);
}

// One thread's share of staging a segment of a chunk's bf16 activation rows (K
// inputs each) for a workgroup of W waves: piece tid%64 of token rows W*q + tid/64
// (q < Q).  Tokens past the chunk read out of range (zeros, no memory request), so
// every thread issues the same loads and no branch guards them.  A segment that runs
// past K (an odd block count) stages bytes no block reads.
template <int NT, int W>
struct Stager {
    static_assert(W == 4 || W == 8, "four or eight waves per workgroup");
    static constexpr int kPieces = kRowBytes / 16;  // per token row and segment
    static constexpr int Q = 16 * NT * kPieces / (64 * W);
    uint32_t voff[Q];
    int tok[Q];
    int piece;
    u32x4v code[Q];

    __device__ void init(const int32_t *__restrict__ row_of, int slot0, int mc, int K, int tid)
    {
        piece = tid & (kPieces - 1);
#pragma unroll
        for (int q = 0; q < Q; ++q) {
            const int t = (64 * W / kPieces) * q + tid / kPieces;
            tok[q] = t;
            const uint32_t row = t < mc ? (uint32_t)(row_of ? row_of[slot0 + t] : slot0 + t) : 0u;
            voff[q] = t < mc ? row * (uint32_t)K * 2u + 16u * piece : kOutOfRange;
        }
    }
    // segment sg (callers clamp it to the last segment)
    __device__ void load(__amdgpu_buffer_rsrc_t rs, int sg)
    {
#pragma unroll
        for (int q = 0; q < Q; ++q)
            code[q] = __builtin_amdgcn_raw_buffer_load_b128(rs, voff[q] + (uint32_t)sg * kRowBytes, 0, 0);
    }
    template <class S_>
    __device__ void store(S_ &S) const
    {
#pragma unroll
        for (int q = 0; q < Q; ++q)
            *reinterpret_cast<u32x4v *>(&S.row[tok[q]][swz(piece, tok[q]) * 16]) = code[q];
    }
};

// Four bf16x8 operands (instructions q = 4h..4h+3 of a block) from 16 of a lane's
// weight bytes (w: inputs [64g + 32h, 64g + 32h + 32)) and their two E4M3 block
// scales (s0: the first 16 inputs, s1: the next 16).
__device__ inline void dequant(const u32x4v &w, float s0, float s1, bf16x8 (&a)[4])
{
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const float s = q < 2 ? s0 : s1;
        f32x2 v[4];
        v[0] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[q], 1.0f, 0);
        v[1] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[q], 1.0f, 1);
        v[2] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[q], 1.0f, 2);
        v[3] = __builtin_amdgcn_cvt_scalef32_pk_f32_fp4(w[q], 1.0f, 3);
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            const bf16x2 p = __builtin_convertvector(v[b] * s, bf16x2);
            a[q][2 * b] = p.x;
            a[q][2 * b + 1] = p.y;
        }
    }
}

// A raw buffer over memory the whole wave addresses from one base (scalar registers).
__device__ inline __amdgpu_buffer_rsrc_t uniform_rsrc(const void *p)
{
    const uint64_t a = (uint64_t)p;
    const uint32_t lo = __builtin_amdgcn_readfirstlane((uint32_t)a);
    const uint32_t hi = __builtin_amdgcn_readfirstlane((uint32_t)(a >> 32));
    return __builtin_amdgcn_make_buffer_rsrc((void *)(((uint64_t)hi << 32) | lo), (short)0, -1, kRawBufferWord3);
}

// The f16 form of dequant: E2M1 pairs to f16 (exact), times the block scale, which the
// E4M3 conversion gave as f16 (s.x: the first 16 inputs, s.y: the next 16), by packed
// multiplies whose operand selection broadcasts one half of s.  A product of an E2M1
// value and an E4M3 scale has at most 6 significant bits and lies in [2^-10, 2688] or is
// zero: exact in f16.
__device__ inline void dequant16(const u32x4v &w, f16x2 s, f16x8 (&a)[4])
{
    const f16x2 m0 = {s.x, s.x}, m1 = {s.y, s.y};
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const f16x2 m = q < 2 ? m0 : m1;
        f16x2 v[4];
        v[0] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w[q], 1.0f, 0) * m;
        v[1] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w[q], 1.0f, 1) * m;
        v[2] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w[q], 1.0f, 2) * m;
        v[3] = __builtin_amdgcn_cvt_scalef32_pk_f16_fp4(w[q], 1.0f, 3) * m;
#pragma unroll
        for (int b = 0; b < 4; ++b) {
            a[q][2 * b] = v[b].x;
            a[q][2 * b + 1] = v[b].y;
        }
    }
}

// Streams this wave's 16-row weight tile (this lane's row `arow`, its E4M3 scale row
// `srow`) over KB 256-input blocks against NT staged token tiles.  All W waves of the
// workgroup call it together; it synchronises them once per staged segment.  On
// return every wave has passed a barrier after its last read of either buffer.
//   arow  row-major: this lane's weight row; packed: the wave's 16-row tile
//   srow  row-major: this lane's scale row; packed: the tile's scales
//   F16   f16 operands (the staged activations are f16), else bf16
//   GS    packed scales in groups of four blocks (PK, KB a multiple of 4): one 16-byte
//         load per lane and group, issued a group ahead, at a fixed place in the loop
//         (a conditional load in the steady state would make every wait conservative)
template <int NT, int W, bool PK, bool F16, bool GS, class S_>
__device__ inline void stream_tile(f32x4 (&acc)[NT], const uint8_t *__restrict__ arow,
                                   const uint8_t *__restrict__ srow, int KB, __amdgpu_buffer_rsrc_t rs,
                                   Stager<NT, W> &st, S_ (&seg)[2], int lane)
{
    static_assert(!GS || PK, "grouped scales are a packed layout");
    const int r = lane & 15, g = lane >> 4;
    const int nseg = (KB + kSegBlk - 1) / kSegBlk;
    u32x4v A[4][2];
    uint32_t S[4];
    __amdgpu_buffer_rsrc_t tr, sr;
    if constexpr (PK) {
        tr = uniform_rsrc(arow);
        sr = uniform_rsrc(srow);
    }
    auto loadA = [&](int slot, int kb) {
        if constexpr (PK) {
            A[slot][0] = __builtin_amdgcn_raw_buffer_load_b128(tr, 16u * lane, kb * 2048, kNonTemporal);
            A[slot][1] = __builtin_amdgcn_raw_buffer_load_b128(tr, 16u * lane + 1024u, kb * 2048, kNonTemporal);
            if constexpr (!GS) S[slot] = __builtin_amdgcn_raw_buffer_load_b32(sr, 4u * lane, kb * 256, 0);
        } else {
            const uint8_t *p = arow + (size_t)kb * (kBlk / 2) + 32 * g;
            A[slot][0] = *reinterpret_cast<const u32x4v *>(p);
            A[slot][1] = *reinterpret_cast<const u32x4v *>(p + 16);
            S[slot] = *reinterpret_cast<const uint32_t *>(srow + (size_t)kb * (kBlk / 16) + 4 * g);
        }
    };
    // Each half block's activation fragments are read from LDS before its weights are
    // dequantised, so the LDS latency hides behind that VALU work; instructions q
    // accumulate into acc2[q % 2], so consecutive MFMAs do not wait on each other.
    f32x4 acc2[2][NT];
    // the four scales of group q of a grouped layout
    auto load_group = [&](int q) { return __builtin_amdgcn_raw_buffer_load_b128(sr, 16u * lane, q * 1024, 0); };
    auto compute = [&](int slot, const S_ &sg, int kk, uint32_t sw) {
        // the four E4M3 scales of this lane's 64 inputs, as fp32 for the bf16 path and
        // as f16 pairs for the f16 one (the unused pair is dead code)
        const f32x2 s01 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(sw, 1.0f, false);
        const f32x2 s23 = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(sw, 1.0f, true);
        const f16x2 h01 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sw, 1.0f, false);
        const f16x2 h23 = __builtin_amdgcn_cvt_scalef32_pk_f16_fp8(sw, 1.0f, true);
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            u32x4v b[4][NT];
#pragma unroll
            for (int q = 0; q < 4; ++q)
#pragma unroll
                for (int j = 0; j < NT; ++j) {
                    const int t = 16 * j + r;
                    b[q][j] = *reinterpret_cast<const u32x4v *>(&sg.row[t][swz(kk * 32 + 8 * g + 4 * h + q, t) * 16]);
                }
            __builtin_amdgcn_sched_barrier(0);
            if constexpr (F16) {
                f16x8 a[4];
                dequant16(A[slot][h], h ? h23 : h01, a);
#pragma unroll
                for (int q = 0; q < 4; ++q)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc2[q & 1][j] = __builtin_amdgcn_mfma_f32_16x16x32_f16(a[q], __builtin_bit_cast(f16x8, b[q][j]),
                                                                                acc2[q & 1][j], 0, 0, 0);
            } else {
                bf16x8 a[4];
                dequant(A[slot][h], h ? s23.x : s01.x, h ? s23.y : s01.y, a);
#pragma unroll
                for (int q = 0; q < 4; ++q)
#pragma unroll
                    for (int j = 0; j < NT; ++j)
                        acc2[q & 1][j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(a[q], __builtin_bit_cast(bf16x8, b[q][j]),
                                                                                 acc2[q & 1][j], 0, 0, 0);
            }
        }
    };
#pragma unroll
    for (int j = 0; j < NT; ++j) acc2[0][j] = acc2[1][j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    loadA(0, 0);
    loadA(1, min(1, KB - 1));
    loadA(2, min(2, KB - 1));
    u32x4v SG0 = {0u, 0u, 0u, 0u}, SG1 = {0u, 0u, 0u, 0u};
    if constexpr (GS) SG0 = load_group(0);
    st.load(rs, 0);
    st.store(seg[0]);
    st.load(rs, min(1, nseg - 1));
    sync_lds();
    int sg = 0, kb = 0;
    // Four blocks (two segments) per step: blocks kb..kb+3 are multiplied while kb+3..kb+6
    // load; with grouped scales the next group's load leads the step and `cur` holds
    // this group's.
    auto step = [&](const u32x4v &cur, u32x4v &nxt) {
        if constexpr (GS) nxt = load_group(min((kb >> 2) + 1, KB / 4 - 1));
        loadA(3, min(kb + 3, KB - 1));  // past the end: reload the last block
        compute(0, seg[0], 0, GS ? cur[0] : S[0]);
        loadA(0, min(kb + 4, KB - 1));
        compute(1, seg[0], 1, GS ? cur[1] : S[1]);
        st.store(seg[1]);
        st.load(rs, min(sg + 2, nseg - 1));
        sync_lds();
        loadA(1, min(kb + 5, KB - 1));
        compute(2, seg[1], 0, GS ? cur[2] : S[2]);
        loadA(2, min(kb + 6, KB - 1));
        compute(3, seg[1], 1, GS ? cur[3] : S[3]);
        st.store(seg[0]);
        st.load(rs, min(sg + 3, nseg - 1));
        sync_lds();
        sg += 2;
        kb += 4;
    };
    if constexpr (GS) {
        // One step per iteration, the next group's words copied into the current ones at
        // its end.  Two steps per iteration that traded the registers by name made the
        // compiler wait for all but the step's first three loads at the top of every
        // iteration (NVFP4 Zipf layer at T=256: gate/up 180.8 -> 179.1 us).
        while (kb + 4 <= KB) {
            step(SG0, SG1);
            SG0 = SG1;
        }
    } else {
        while (kb + 4 <= KB) step(SG0, SG1);
        // Fewer than four blocks remain, in ring slots 0..2: segment sg sits in seg[0] and
        // segment sg + 1 in the stager's registers.
        if (kb < KB) compute(0, seg[0], 0, S[0]);
        if (kb + 1 < KB) compute(1, seg[0], 1, S[1]);
        if (kb + 2 < KB) {
            st.store(seg[1]);
            sync_lds();
            compute(2, seg[1], 0, S[2]);
        }
    }
    if (kb < KB) sync_lds();
#pragma unroll
    for (int j = 0; j < NT; ++j) acc[j] = acc2[0][j] + acc2[1][j];
}

// gate/up: item = (chunk, rows [i0, i0 + 8W)); wave w < W/2 streams gate rows
// i0 + 16w, wave w >= W/2 the up rows of the same 16.  The up accumulators reach the
// gate waves through LDS (seg[1], free once stream_tile returns; the next item first
// writes it after its first barrier), and the gate waves form h = silu(g) * u, round
// it to bf16 and store it.
template <int NT, int W, bool PK, bool GS, class S_>
__device__ inline void w13_item(const uint8_t *__restrict__ we, const uint8_t *__restrict__ se, int H, int I, int i0,
                                int slot0, int mc, const int32_t *__restrict__ tok_of, __amdgpu_buffer_rsrc_t xr,
                                const int32_t *__restrict__ xk, __bf16 *__restrict__ hb, S_ (&seg)[2], int wave,
                                int lane, int tid)
{
    constexpr int HW = W / 2;
    const int r = lane & 15, g = lane >> 4;
    const bool up = wave >= HW;
    const int rr = i0 + 16 * (wave % HW) + r;  // this lane's intermediate row
    const uint8_t *arow = we + (size_t)((up ? I : 0) + rr - (PK ? r : 0)) * (H / 2);
    const uint8_t *srow = se + 16 + (size_t)((up ? I : 0) + rr - (PK ? r : 0)) * (H / 16);
    Stager<NT, W> st;
    st.init(tok_of, slot0, mc, H, tid);
    f32x4 acc[NT];
    stream_tile<NT, W, PK, true, GS>(acc, arow, srow, H / kBlk, xr, st, seg, lane);
    f32x4 *red = reinterpret_cast<f32x4 *>(&seg[1].row[0][0]);
    static_assert(sizeof(f32x4) * (W / 2) * 2 * 64 <= sizeof(S_), "reduction buffer");
    if (up) {
#pragma unroll
        for (int j = 0; j < NT; ++j) red[((wave - HW) * 2 + j) * 64 + lane] = acc[j];
    }
    sync_lds();
    if (!up) {
#pragma unroll
        for (int j = 0; j < NT; ++j) {
            // token column 16j + r: undo its 2^-k (2^k is exact: -112 <= k <= 113)
            const int kt = 16 * j + r < mc ? xk[tok_of[slot0 + 16 * j + r]] : 0;
            const float p2k = __uint_as_float((uint32_t)(127 + kt) << 23);
            const float tg = reinterpret_cast<const float *>(se)[0] * p2k, tu = reinterpret_cast<const float *>(se)[1] * p2k;
            const f32x4 u = red[(wave * 2 + j) * 64 + lane];
            bf16x2 hv[2];
#pragma unroll
            for (int i = 0; i < 2; ++i) {
                const float g0 = tg * acc[j][2 * i], g1 = tg * acc[j][2 * i + 1];
                const f32x2 h = {g0 / (1.0f + expf(-g0)) * (tu * u[2 * i]), g1 / (1.0f + expf(-g1)) * (tu * u[2 * i + 1])};
                hv[i] = __builtin_convertvector(h, bf16x2);
            }
            if (16 * j + r < mc) {
                const size_t slot = (size_t)slot0 + 16 * j + r;
                *reinterpret_cast<uint2 *>(hb + slot * I + i0 + 16 * wave + 4 * g) =
                    make_uint2(__builtin_bit_cast(uint32_t, hv[0]), __builtin_bit_cast(uint32_t, hv[1]));
            }
        }
    }
}

// T16: every chunk in passes of at most 16 tokens (one token tile), staged in
// 16-row segments: half the LDS and none of the two-tile registers, for three waves
// per SIMD.  A chunk of more than 16 tokens streams its weights once per pass.
template <int W, bool PK, bool GS, bool T16>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(T16 ? 3 : 2))) void w13_nvfp4_kernel(const uint8_t *__restrict__ ew,
                                                           const uint8_t *__restrict__ es,
                                                           const int32_t *__restrict__ meta,
                                                           const int32_t *__restrict__ tok_of,
                                                           const _Float16 *__restrict__ x16,
                                                           const int32_t *__restrict__ xk, __bf16 *__restrict__ hb,
                                                           int T, int H, int I, int E, size_t ewb, size_t esb)
{
    __shared__ SegT<T16 ? 16 : kTok> seg[2];
    const MetaIdx mi{E};
    const int tiles = I / (8 * W);
    const int n_items = meta[mi.n_mfma_chunks()] * tiles;
    const int4 *recs = reinterpret_cast<const int4 *>(meta + mi.chunk_rec());
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const __amdgpu_buffer_rsrc_t xr = raw_rsrc(x16, (uint32_t)T * (uint32_t)H * 2u);
    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int4 rec = recs[item / tiles];  // {expert, first slot, tokens, -}
        const int i0 = (item % tiles) * 8 * W;
        const uint8_t *we = ew + (size_t)rec.x * ewb;
        const uint8_t *se = es + (size_t)rec.x * esb;
        if constexpr (T16) {
            for (int s0 = 0; s0 < rec.z; s0 += 16)
                w13_item<1, W, PK, GS>(we, se, H, I, i0, rec.y + s0, min(16, rec.z - s0), tok_of, xr, xk, hb, seg, wave,
                                       lane, tid);
        } else if (rec.z > 16) {
            w13_item<2, W, PK, GS>(we, se, H, I, i0, rec.y, rec.z, tok_of, xr, xk, hb, seg, wave, lane, tid);
        } else {
            w13_item<1, W, PK, GS>(we, se, H, I, i0, rec.y, rec.z, tok_of, xr, xk, hb, seg, wave, lane, tid);
        }
    }
}

// down: item = (chunk, rows [n0, n0 + 16W)); wave w streams rows n0 + 16w.
template <int NT, int W, bool PK, bool GS, class S_>
__device__ inline void w2_item(const uint8_t *__restrict__ we, const uint8_t *__restrict__ se, int H, int I, int n0,
                               int slot0, int mc, __amdgpu_buffer_rsrc_t hr, float *__restrict__ obuf, S_ (&seg)[2],
                               int wave, int lane, int tid)
{
    const int r = lane & 15, g = lane >> 4;
    const int row0 = n0 + 16 * wave;
    const uint8_t *arow = we + (size_t)I * H + (size_t)(row0 + (PK ? 0 : r)) * (I / 2);
    const uint8_t *srow = se + 16 + (size_t)2 * I * (H / 16) + (size_t)(row0 + (PK ? 0 : r)) * (I / 16);
    Stager<NT, W> st;
    st.init(nullptr, slot0, mc, I, tid);
    f32x4 acc[NT];
    stream_tile<NT, W, PK, false, GS>(acc, arow, srow, I / kBlk, hr, st, seg, lane);
    const float td = reinterpret_cast<const float *>(se)[2];
#pragma unroll
    for (int j = 0; j < NT; ++j)
        if (16 * j + r < mc)
            *reinterpret_cast<f32x4 *>(obuf + ((size_t)slot0 + 16 * j + r) * H + row0 + 4 * g) = td * acc[j];
}

// T16 as for the gate/up kernel.
template <int W, bool PK, bool GS, bool T16>
__global__ __launch_bounds__(64 * W) __attribute__((amdgpu_waves_per_eu(T16 ? 3 : 2))) void w2_nvfp4_kernel(const uint8_t *__restrict__ ew,
                                                          const uint8_t *__restrict__ es,
                                                          const int32_t *__restrict__ meta,
                                                          const __bf16 *__restrict__ hb, float *__restrict__ obuf,
                                                          int P, int H, int I, int E, size_t ewb, size_t esb)
{
    __shared__ SegT<T16 ? 16 : kTok> seg[2];
    const MetaIdx mi{E};
    const int tiles = H / (16 * W);
    const int n_items = meta[mi.n_mfma_chunks()] * tiles;
    const int4 *recs = reinterpret_cast<const int4 *>(meta + mi.chunk_rec());
    const int tid = threadIdx.x, lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const __amdgpu_buffer_rsrc_t hr = raw_rsrc(hb, (uint32_t)P * (uint32_t)I * 2u);
    for (int item = blockIdx.x; item < n_items; item += gridDim.x) {
        const int4 rec = recs[item / tiles];
        const int n0 = (item % tiles) * 16 * W;
        const uint8_t *we = ew + (size_t)rec.x * ewb;
        const uint8_t *se = es + (size_t)rec.x * esb;
        if constexpr (T16) {
            for (int s0 = 0; s0 < rec.z; s0 += 16)
                w2_item<1, W, PK, GS>(we, se, H, I, n0, rec.y + s0, min(16, rec.z - s0), hr, obuf, seg, wave, lane, tid);
        } else if (rec.z > 16) {
            w2_item<2, W, PK, GS>(we, se, H, I, n0, rec.y, rec.z, hr, obuf, seg, wave, lane, tid);
        } else {
            w2_item<1, W, PK, GS>(we, se, H, I, n0, rec.y, rec.z, hr, obuf, seg, wave, lane, tid);
        }
    }
}

constexpr int kWaves = 4;

// Workgroups for `items_per_chunk` items per chunk record (see mfma_grid in mfma.hip).
int nvfp4_grid(const Layer &L, int T, int k, int items_per_chunk)
{
    const long pairs = (long)T * k;
    const long recs = pairs < L.E ? pairs : L.E;
    const long chunks = recs + (pairs + kMfmaChunk - 1) / kMfmaChunk;
    const long blocks = chunks * items_per_chunk;
    return blocks < 1 ? 1 : (blocks > 65535 ? 65535 : (int)blocks);
}

}  // namespace

// Grouped packed scales (four blocks per 16-byte load) where the matrix's 256-input block
// count is a multiple of four; moe_decode_pack_weights writes that layout for such
// matrices.
bool grouped_scales(const Layer &L, int K) { return L.wlayout && (K / kBlk) % 4 == 0; }

// Gate/up workgroups of eight waves from 1024 (token, expert) pairs per step: with full
// chunks each staged activation segment then serves twice the rows.  235B-shaped NVFP4
// layer (four waves -> eight): Zipf T=256 gate/up 180.4 -> 169.6 us; T=64 152.0 -> 151.2
// (equal within the spread); T=8 67.4 -> 70.0 and T=32 134.5 -> 137.3 us, so smaller
// batches keep four.  Both give the same bits: a wave's rows and its K order do not
// change.  The down projection keeps four (eight: 108.5 -> 121.0 us at Zipf T=256).
constexpr int kWideBatchPairs = 1024;

// One-tile passes (T16) on packed weights up to this many (token, expert) pairs per
// expert on average (T=128 at top-8 of 128 experts; the gate/up kernel takes its
// eight-wave form from 1024 pairs first).  Three waves per SIMD against two,
// 235B-shaped NVFP4 layer, gate/up and down us: T=8 66.7/43.4 -> 63.3/39.0, T=32
// 132.0/87.8 -> 125.9/78.3, T=64 149.8/101.4 -> 142.2/93.0; T=96 155.6/104.3 ->
// 147.3/96.4 and T=127 159.4/105.6 -> 152.0/99.2, where hot experts take several
// passes.  Row-major weights keep the two-tile kernels (their T16 form spills at
// three waves).
constexpr long kTileOnlyPairsPerExpert = 8;

static bool tile_only(const Layer &L, int T, int k) { return L.wlayout && (long)T * k <= kTileOnlyPairsPerExpert * (long)L.E; }

template <int W, bool T16>
hipError_t w13_nvfp4_launch(const Layer &L, const uint8_t *ew, const uint8_t *es, int T, int k, const int32_t *meta,
                            const int32_t *tok_of, const Workspace &ws, hipStream_t st)
{
    dim3 grid(nvfp4_grid(L, T, k, L.I / (8 * W))), block(64 * W);
    __bf16 *hb = (__bf16 *)ws.hb;
    if (grouped_scales(L, L.H))
        w13_nvfp4_kernel<W, true, true, T16><<<grid, block, 0, st>>>(ew, es, meta, tok_of, ws.x16, ws.xk, hb, T, L.H,
                                                                     L.I, L.E, L.expert_w_bytes, L.expert_s_bytes);
    else if (L.wlayout)
        w13_nvfp4_kernel<W, true, false, T16><<<grid, block, 0, st>>>(ew, es, meta, tok_of, ws.x16, ws.xk, hb, T, L.H,
                                                                      L.I, L.E, L.expert_w_bytes, L.expert_s_bytes);
    else
        w13_nvfp4_kernel<W, false, false, false><<<grid, block, 0, st>>>(ew, es, meta, tok_of, ws.x16, ws.xk, hb, T,
                                                                         L.H, L.I, L.E, L.expert_w_bytes,
                                                                         L.expert_s_bytes);
    return hipGetLastError();
}

// Packed weights only: row-major ones take the four-wave two-tile kernel
// (launch_w2_nvfp4).
template <int W, bool T16>
hipError_t w2_nvfp4_launch(const Layer &L, const uint8_t *ew, const uint8_t *es, int T, int k, const int32_t *meta,
                           const Workspace &ws, hipStream_t st)
{
    dim3 grid(nvfp4_grid(L, T, k, L.H / (16 * W))), block(64 * W);
    const __bf16 *hb = (const __bf16 *)ws.hb;
    if (grouped_scales(L, L.I))
        w2_nvfp4_kernel<W, true, true, T16><<<grid, block, 0, st>>>(ew, es, meta, hb, ws.o, T * k, L.H, L.I, L.E,
                                                                    L.expert_w_bytes, L.expert_s_bytes);
    else
        w2_nvfp4_kernel<W, true, false, T16><<<grid, block, 0, st>>>(ew, es, meta, hb, ws.o, T * k, L.H, L.I, L.E,
                                                                     L.expert_w_bytes, L.expert_s_bytes);
    return hipGetLastError();
}

hipError_t launch_w13_nvfp4(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                            const int32_t *meta, const int32_t *tok_of, const Workspace &ws, hipStream_t st)
{
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
    if ((long)T * k >= kWideBatchPairs && L.I % (8 * 8) == 0)
        return w13_nvfp4_launch<8, false>(L, ew, es, T, k, meta, tok_of, ws, st);
    if (tile_only(L, T, k)) {
        // Eight-wave one-tile workgroups (126 VGPRs, four waves per SIMD) where chunks
        // are fuller, from four pairs per expert on average, or where the four-wave grid
        // would leave most CUs with one workgroup (fewer than 512 items on 256 CUs).
        // 235B-shaped layer, gate/up us (four -> eight waves): T=1 17.35 -> 16.4, T=127
        // 152.6 -> 149.2; T=8 63.4 -> 64.3, T=32 125.7 -> 128.6, T=64 142.0 -> 142.9.
        const long pairs = (long)T * k;
        if ((pairs > 4L * L.E || pairs * (L.I / (8 * kWaves)) < 512) && L.I % (8 * 8) == 0)
            return w13_nvfp4_launch<8, true>(L, ew, es, T, k, meta, tok_of, ws, st);
        return w13_nvfp4_launch<kWaves, true>(L, ew, es, T, k, meta, tok_of, ws, st);
    }
    return w13_nvfp4_launch<kWaves, false>(L, ew, es, T, k, meta, tok_of, ws, st);
}
hipError_t launch_w2_nvfp4(const Layer &L, const void *expert_w, const void *scales, int T, int k,
                           const int32_t *meta, const Workspace &ws, hipStream_t st)
{
    const uint8_t *ew = (const uint8_t *)expert_w, *es = (const uint8_t *)scales;
    if (!L.wlayout) {
        dim3 grid(nvfp4_grid(L, T, k, L.H / (16 * kWaves))), block(64 * kWaves);
        w2_nvfp4_kernel<kWaves, false, false, false><<<grid, block, 0, st>>>(
            ew, es, meta, (const __bf16 *)ws.hb, ws.o, T * k, L.H, L.I, L.E, L.expert_w_bytes, L.expert_s_bytes);
        return hipGetLastError();
    }
    // One-tile passes in eight-wave workgroups (124-133 VGPRs, three or four waves per
    // SIMD), 128 rows per item (H is a multiple of 256 for NVFP4 weights, checked at
    // init).  235B-shaped layer, down us (four -> eight waves): T=32 78.7 -> 77.9, T=64
    // 92.8 -> 91.5, T=127 99.0 -> 97.4; T=1 and T=8 equal.
    if (tile_only(L, T, k)) return w2_nvfp4_launch<8, true>(L, ew, es, T, k, meta, ws, st);
    return w2_nvfp4_launch<kWaves, false>(L, ew, es, T, k, meta, ws, st);
}

}  // namespace moe
