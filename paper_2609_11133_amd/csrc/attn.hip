// Decode attention over a paged KV cache: one decode step of grouped-query attention
// (scaled dot-product attention with Hq / Hkv query heads per key/value head), the
// KV-cache half of the decode step's byte streams, on the gfx950 bf16 matrix cores.
//
// Split over the context.  Workgroup (c, g, b) of four waves takes tokens
// [256c, 256c + 256) of sequence b for key/value head g and its (up to 16) query heads;
// each wave takes 64 of those tokens as four 16-token tiles (one cache page each).
//   S^T = K_tile . Q^T   v_mfma_f32_16x16x32_bf16, A = keys (rows = tokens, K = dims),
//                        B = queries (columns = heads): lane l ends with the scores of
//                        head l%16 for tokens 4(l/16)..4(l/16)+3 of the tile.
//   O  += P . V          A = probabilities (rows = heads), B = values (columns = dims):
//                        the lane's eight K slots are its four tokens of two tiles,
//                        which is exactly what the S^T accumulators hold, so P needs no
//                        transpose; the values are read dimension-major (a page stores
//                        V as [D][16]), four contiguous tokens per tile.
// The workgroup shares one score maximum per head (through LDS), so its four waves' P.V
// partials add directly; it writes (max, sum, O) of its split, and the splits of each
// (sequence, query head) are merged in split order: by the last of the sequence's
// workgroups for that key/value head (a device-scope counter, the partials written and
// read with device-coherent accesses) when a sequence has at most kFusedSplits splits,
// else by a second kernel.  A sequence with one split writes its output directly.
//
// Operand layout of v_mfma_f32_16x16x32_bf16 (checked on the device): lane l holds
// row/column l%16 and K [8g, 8g+8) with g = l/16; the result gives lane l rows
// 4g..4g+3 of column l%16.
#include <hip/hip_runtime.h>

#include <atomic>
#include <math.h>
#include <stdarg.h>
#include <stdio.h>
#include <string.h>

#include "../../include/attn_decode.h"

namespace attn {
namespace {

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x2 __attribute__((ext_vector_type(2)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef float f32x2 __attribute__((ext_vector_type(2)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2v __attribute__((ext_vector_type(2)));

constexpr int kD = 128;                    // head dimension
constexpr int kP = 16;                     // tokens per page
constexpr int kWaves = 4;                  // waves per workgroup
constexpr int kWaveTok = 64;               // tokens per wave
constexpr int kTiles = kWaveTok / kP;      // 16-token tiles (pages) per wave
constexpr int kChunk = kWaves * kWaveTok;  // tokens per split
constexpr int kDT = kD / 16;               // 16-column tiles of the output
constexpr float kLog2e = 1.44269504088896340736f;
constexpr int kRawBufferWord3 = 0x00020000;  // untyped 32-bit data format, no swizzle
constexpr int kFusedSplits = 16;             // splits merged inside the split kernel, at most

// Device-coherent accesses for the hand-off between workgroups (relaxed atomics at agent
// scope bypass the per-XCD L2), and a wait for this thread's stores.
template <typename T>
__device__ inline void st_dev(T *p, T v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
template <typename T>
__device__ inline T ld_dev(const T *p) { return __hip_atomic_load(const_cast<T *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
// The memory clobber keeps the compiler from moving memory accesses across the wait,
// so every store issued before it has completed when the counter is bumped.
__device__ inline void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

__device__ inline uint16_t to_bf16(float y)
{
    const bf16x2 yb = __builtin_convertvector((f32x2){y, 0.f}, bf16x2);
    return __builtin_bit_cast(uint16_t, yb.x);
}

// A raw buffer over `bytes` bytes at `base`: loads past the end return zeros and make
// no memory request, so a page the kernel must not read gets bytes = 0.
__device__ inline __amdgpu_buffer_rsrc_t rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, kRawBufferWord3);
}

__device__ inline bf16x8 as_bf16x8(const u32x4v &u) { return __builtin_bit_cast(bf16x8, u); }

// Split kernel: partial (max, sum, O) of one 256-token split for one (sequence, key/value
// head) and its query heads.  Grid (splits, Hkv, B), 256 threads.  Scores are kept in
// log2 units (scale * log2 e folded in), so p = exp2(s - m).  A split is R consecutive
// chunks (online softmax across them); with FUSED each sequence sets its own R.  FUSED: the merge of the splits happens here
// (S <= kFusedSplits; `cnt` holds one zeroed counter per (b, g), left at zero again), and
// `out` is written here.
template <bool FUSED>
__global__ __launch_bounds__(256) void attn_split_kernel(const uint16_t *__restrict__ q,
                                                         const uint16_t *__restrict__ kc,
                                                         const uint16_t *__restrict__ vc, int64_t n_pages,
                                                         const int32_t *__restrict__ block_table, int max_pages,
                                                         const int32_t *__restrict__ ctx, int Hkv, int G,
                                                         float scale_log2, float *__restrict__ po,
                                                         float *__restrict__ pml, int S, int R,
                                                         int32_t *__restrict__ cnt, uint16_t *__restrict__ out)
{
    __shared__ float s_max[2][kWaves][16], s_sum[kWaves][16];
    __shared__ f32x4 red[kWaves][kDT][64];
    __shared__ float s_w[FUSED ? kFusedSplits : 1][16], s_den[16];
    __shared__ int s_last;
    const int c = blockIdx.x, g = blockIdx.y, b = blockIdx.z;
    const int L = min(max(ctx[b], 0), max_pages * kP);
    // FUSED: each sequence spreads its own chunks over the S splits of the grid, at least
    // one chunk per split (R = ceil(chunks / S), at most the configuration's R): a short
    // context in a configuration sized for long ones still gets one workgroup per chunk,
    // and a sequence's result depends on its own length only, never on its batch.
    if (FUSED) R = max(1, ((L + kChunk - 1) / kChunk + S - 1) / S);
    const int t0 = c * R * kChunk;  // first token of this split
    const int tid = threadIdx.x, lane = tid & 63;
    uint16_t *orow = out + ((size_t)b * Hkv + g) * G * kD;  // the group's [G][D] outputs
    if (t0 >= L) {  // uniform over the workgroup
        if (FUSED && c == 0)  // empty context: zeros
            for (int e = tid; e < G * kD; e += 256) orow[e] = 0;
        return;
    }
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int r = lane & 15, lg = lane >> 4;

    // Q^T operand: head r of the group (zeros past it), dims [32i + 8lg, 32i + 8lg + 8)
    bf16x8 qop[4];
    {
        const bool live = r < G;
        const uint16_t *qrow = q + ((size_t)b * Hkv * G + (size_t)g * G + (live ? r : 0)) * kD;
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            const u32x4v w = live ? *reinterpret_cast<const u32x4v *>(qrow + 32 * i + 8 * lg) : (u32x4v){0, 0, 0, 0};
            qop[i] = as_bf16x8(w);
        }
    }

    // R consecutive 256-token chunks of the context per workgroup (online softmax across
    // them: a running maximum per head rescales the sums and the P.V accumulators)
    float m_run = -INFINITY, l_run = 0.f, m = -INFINITY;
    f32x4 o[kDT];
#pragma unroll
    for (int j = 0; j < kDT; ++j) o[j] = (f32x4){0.f, 0.f, 0.f, 0.f};
    for (int rr = 0; rr < R; ++rr) {
        const int t0 = (c * R + rr) * kChunk;
        if (t0 >= L) break;  // uniform over the workgroup
        // This wave's four pages: keys (token r, dims [32i + 8lg, +8)) and values (dims
        // 16j + r, tokens [4lg, 4lg + 4)).  Pages past the context or outside the cache
        // read as zeros.
        const int tw = t0 + kWaveTok * wave;
        u32x4v ka[kTiles][4];
        u32x2v vb[kTiles][kDT];
    #pragma unroll
        for (int tt = 0; tt < kTiles; ++tt) {
            const int ts = tw + kP * tt;  // first token of the tile (page aligned)
            int pg = ts < L ? block_table[(size_t)b * max_pages + ts / kP] : -1;
            pg = __builtin_amdgcn_readfirstlane(pg);
            const bool ok = pg >= 0 && (int64_t)pg < n_pages;
            const int64_t p = ok ? pg : 0;
            const __amdgpu_buffer_rsrc_t kr = rsrc(kc + (p * Hkv + g) * (int64_t)(kP * kD), ok ? kP * kD * 2 : 0);
            const __amdgpu_buffer_rsrc_t vr = rsrc(vc + (p * Hkv + g) * (int64_t)(kP * kD), ok ? kP * kD * 2 : 0);
    #pragma unroll
            for (int i = 0; i < 4; ++i)
                ka[tt][i] = __builtin_amdgcn_raw_buffer_load_b128(kr, (uint32_t)((r * kD + 32 * i + 8 * lg) * 2), 0, 0);
    #pragma unroll
            for (int j = 0; j < kDT; ++j)
                vb[tt][j] = __builtin_amdgcn_raw_buffer_load_b64(vr, (uint32_t)(((16 * j + r) * kP + 4 * lg) * 2), 0, 0);
        }

        // scores of this lane's 16 (token, head r) pairs, masked past the context
        float s[kTiles][4];
        m = -INFINITY;
    #pragma unroll
        for (int tt = 0; tt < kTiles; ++tt) {
            f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    #pragma unroll
            for (int i = 0; i < 4; ++i) acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(as_bf16x8(ka[tt][i]), qop[i], acc, 0, 0, 0);
    #pragma unroll
            for (int e = 0; e < 4; ++e) {
                const bool live = tw + kP * tt + 4 * lg + e < L;
                s[tt][e] = live ? acc[e] * scale_log2 : -INFINITY;
                m = fmaxf(m, s[tt][e]);
            }
        }
        m = fmaxf(m, __shfl_xor(m, 16));
        m = fmaxf(m, __shfl_xor(m, 32));
        if (lg == 0) s_max[rr & 1][wave][r] = m;
        __syncthreads();
        m = fmaxf(fmaxf(s_max[rr & 1][0][r], s_max[rr & 1][1][r]), fmaxf(s_max[rr & 1][2][r], s_max[rr & 1][3][r]));
        // running maximum (finite: token t0 < L); alpha rescales what earlier chunks added
        // (0 on the first chunk, whose sums start at zero)
        const float m_new = fmaxf(m_run, m);
        const float alpha = exp2f(m_run - m_new);
        m_run = m_new;
        m = m_new;

        // probabilities (bf16 for the P.V product; the sum uses the same rounded values)
        float l = 0.f;
        bf16x8 pa[kTiles / 2];
    #pragma unroll
        for (int st = 0; st < kTiles / 2; ++st)
    #pragma unroll
            for (int h = 0; h < 2; ++h)
    #pragma unroll
                for (int e = 0; e < 4; e += 2) {
                    const f32x2 pv = {exp2f(s[2 * st + h][e] - m), exp2f(s[2 * st + h][e + 1] - m)};
                    const bf16x2 pb = __builtin_convertvector(pv, bf16x2);
                    pa[st][4 * h + e] = pb.x;
                    pa[st][4 * h + e + 1] = pb.y;
                    l += (float)pb.x + (float)pb.y;
                }
        l += __shfl_xor(l, 16);
        l += __shfl_xor(l, 32);
        l_run = l_run * alpha + l;

        // values past the context are zeroed: a cache slot past it may hold any bits, and
        // 0 * NaN would not vanish
    #pragma unroll
        for (int tt = 0; tt < kTiles; ++tt) {
            const int nv = min(max(L - (tw + kP * tt + 4 * lg), 0), 4);
            const uint32_t m0 = nv >= 2 ? 0xFFFFFFFFu : (nv == 1 ? 0x0000FFFFu : 0u);
            const uint32_t m1 = nv >= 4 ? 0xFFFFFFFFu : (nv == 3 ? 0x0000FFFFu : 0u);
    #pragma unroll
            for (int j = 0; j < kDT; ++j) {
                vb[tt][j].x &= m0;
                vb[tt][j].y &= m1;
            }
        }
        // o holds heads 4lg..4lg+3 of the P.V result: their rescale factors come from the
        // lanes that hold those heads in the score layout
        {
            float a4[4];
    #pragma unroll
            for (int i = 0; i < 4; ++i) a4[i] = __shfl(alpha, 4 * lg + i);
    #pragma unroll
            for (int j = 0; j < kDT; ++j)
    #pragma unroll
                for (int i = 0; i < 4; ++i) o[j][i] *= a4[i];
        }
    #pragma unroll
        for (int st = 0; st < kTiles / 2; ++st)
    #pragma unroll
            for (int j = 0; j < kDT; ++j) {
                const u32x4v vv = {vb[2 * st][j].x, vb[2 * st][j].y, vb[2 * st + 1][j].x, vb[2 * st + 1][j].y};
                o[j] = __builtin_amdgcn_mfma_f32_16x16x32_bf16(pa[st], as_bf16x8(vv), o[j], 0, 0, 0);
            }
    }
    m = m_run;
    if (lg == 0) s_sum[wave][r] = l_run;

    // the workgroup's O: the four waves' partials in wave order
#pragma unroll
    for (int j = 0; j < kDT; ++j) red[wave][j][lane] = o[j];
    __syncthreads();
    const int ns = (L + R * kChunk - 1) / (R * kChunk);  // splits of this sequence
    if (FUSED && ns == 1) {
        // the only split: out = O / l (what the merge of one split gives)
#pragma unroll
        for (int k = 0; k < 16 * kD / 256; ++k) {
            const int e = tid + 256 * k;  // (head n, dim d); n is uniform over a wave
            const int n = e / kD, d = e % kD;
            if (n < G) {
                const int j = d / 16, ln = 16 * (n / 4) + d % 16, comp = n % 4;
                const float v = ((red[0][j][ln][comp] + red[1][j][ln][comp]) + red[2][j][ln][comp]) + red[3][j][ln][comp];
                const float l = ((s_sum[0][n] + s_sum[1][n]) + s_sum[2][n]) + s_sum[3][n];
                orow[e] = to_bf16(fmaf(1.f, v, 0.f) / fmaf(1.f, l, 0.f));
            }
        }
        return;
    }
    const size_t part0 = ((size_t)b * Hkv + g) * S, part = part0 + c;
#pragma unroll
    for (int k = 0; k < 16 * kD / 256; ++k) {
        const int e = tid + 256 * k;  // (head n, dim d)
        const int n = e / kD, d = e % kD;
        const int j = d / 16, ln = 16 * (n / 4) + d % 16, comp = n % 4;
        const float v = ((red[0][j][ln][comp] + red[1][j][ln][comp]) + red[2][j][ln][comp]) + red[3][j][ln][comp];
        if (FUSED)
            st_dev(&po[part * 16 * kD + e], v);
        else
            po[part * 16 * kD + e] = v;
    }
    if (tid < 16) {
        const float l = ((s_sum[0][tid] + s_sum[1][tid]) + s_sum[2][tid]) + s_sum[3][tid];
        if (FUSED) {
            st_dev(&pml[(part * 16 + tid) * 2], m);
            st_dev(&pml[(part * 16 + tid) * 2 + 1], l);
        } else {
            reinterpret_cast<f32x2 *>(pml)[part * 16 + tid] = (f32x2){m, l};
        }
    }
    if constexpr (FUSED) {
        // the last of the sequence's workgroups for head g merges its ns splits
        wait_stores();
        __syncthreads();
        int32_t *ctr = cnt + (size_t)b * Hkv + g;
        if (tid == 0) s_last = atomicAdd(ctr, 1) == ns - 1;
        __syncthreads();
        if (!s_last) return;
        if (tid == 0) st_dev(ctr, 0);
        // thread: element pairs (2 e2, 2 e2 + 1), e2 = tid + 256 k2, of head e2 / 64 (uniform
        // over a wave); eight splits' 64-bit loads in flight per round, the first round
        // issued before the weights are formed
        constexpr int kRound = 8;
        const uint64_t *po2 = reinterpret_cast<const uint64_t *>(po);
        uint64_t v[kRound][4];
        auto load_round = [&](int c0) {
#pragma unroll
            for (int u = 0; u < kRound; ++u)
#pragma unroll
                for (int k2 = 0; k2 < 4; ++k2) {
                    const int e2 = tid + 256 * k2;
                    v[u][k2] = c0 + u < ns && e2 / 64 < G ? ld_dev(&po2[(part0 + c0 + u) * (16 * kD / 2) + e2]) : 0;
                }
        };
        load_round(0);
        // weights 2^(m_c - M) and the denominator per head, splits in ascending order
        if (tid < 16) {
            float mc[kFusedSplits], lc[kFusedSplits];
#pragma unroll
            for (int cc = 0; cc < kFusedSplits; ++cc) {
                const size_t pc = (part0 + min(cc, ns - 1)) * 16 + tid;
                mc[cc] = ld_dev(&pml[pc * 2]);
                lc[cc] = ld_dev(&pml[pc * 2 + 1]);
            }
            float M = -INFINITY;
#pragma unroll
            for (int cc = 0; cc < kFusedSplits; ++cc) M = fmaxf(M, mc[cc]);  // repeats of the last split
            float den = 0.f;
#pragma unroll
            for (int cc = 0; cc < kFusedSplits; ++cc)
                if (cc < ns) {
                    const float w = exp2f(mc[cc] - M);
                    den = fmaf(w, lc[cc], den);
                    s_w[cc][tid] = w;
                }
            s_den[tid] = den;
        }
        __syncthreads();
        float num[4][2];
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2) num[k2][0] = num[k2][1] = 0.f;
        for (int c0 = 0; c0 < ns; c0 += kRound) {
            if (c0) load_round(c0);
#pragma unroll
            for (int u = 0; u < kRound; ++u)
                if (c0 + u < ns)
#pragma unroll
                    for (int k2 = 0; k2 < 4; ++k2) {
                        const float w = s_w[c0 + u][(tid + 256 * k2) / 64];
                        num[k2][0] = fmaf(w, __uint_as_float((uint32_t)v[u][k2]), num[k2][0]);
                        num[k2][1] = fmaf(w, __uint_as_float((uint32_t)(v[u][k2] >> 32)), num[k2][1]);
                    }
        }
#pragma unroll
        for (int k2 = 0; k2 < 4; ++k2) {
            const int e2 = tid + 256 * k2, n = e2 / 64;
            if (n < G) {
                const uint32_t lo = to_bf16(num[k2][0] / s_den[n]), hi = to_bf16(num[k2][1] / s_den[n]);
                reinterpret_cast<uint32_t *>(orow)[e2] = lo | (hi << 16);
            }
        }
    }
}

// Counters of the fused merge: zero.
__global__ void attn_zero_kernel(int32_t *p, int n)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

// Combine kernel: out[b][g*G + n][d] = sum_c 2^(m_c - M) O_c[n][d] / sum_c 2^(m_c - M) l_c
// over the splits c of (b, g) in ascending order, M = max_c m_c; zeros for an empty
// context.  Grid (G, Hkv, B), 128 threads: thread d of workgroup (n, g, b) owns one
// output and keeps sixteen splits' loads in flight; every thread forms the same
// denominator in the same order.
__global__ __launch_bounds__(128) void attn_combine_kernel(const float *__restrict__ po, const float *__restrict__ pml,
                                                           const int32_t *__restrict__ ctx, int max_pages, int Hkv,
                                                           int G, int S, uint16_t *__restrict__ out)
{
    constexpr int U = 16;
    __shared__ float s_m[2];
    const int n = blockIdx.x, g = blockIdx.y, b = blockIdx.z, d = threadIdx.x;
    const int L = min(max(ctx[b], 0), max_pages * kP);
    const int ns = (L + kChunk - 1) / kChunk;
    const size_t part0 = ((size_t)b * Hkv + g) * S;
    const f32x2 *ml = reinterpret_cast<const f32x2 *>(pml);
    float M = -INFINITY;
    for (int c = d; c < ns; c += 128) M = fmaxf(M, ml[(part0 + c) * 16 + n].x);
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) M = fmaxf(M, __shfl_xor(M, o));
    if ((d & 63) == 0) s_m[d >> 6] = M;
    __syncthreads();
    M = fmaxf(s_m[0], s_m[1]);
    float num = 0.f, den = 0.f;
    for (int c0 = 0; c0 < ns; c0 += U) {
        f32x2 mlv[U];
        float ov[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const size_t c = part0 + min(c0 + u, ns - 1);
            mlv[u] = ml[c * 16 + n];
            ov[u] = po[(c * 16 + n) * kD + d];
        }
#pragma unroll
        for (int u = 0; u < U; ++u)
            if (c0 + u < ns) {
                const float w = exp2f(mlv[u].x - M);
                den = fmaf(w, mlv[u].y, den);
                num = fmaf(w, ov[u], num);
            }
    }
    const float y = ns ? num / den : 0.f;
    out[(((size_t)b * Hkv + g) * G + n) * kD + d] = to_bf16(y);
}

thread_local char g_err[256];

int fail(int code, const char *fmt, ...)
{
    va_list ap;
    va_start(ap, fmt);
    vsnprintf(g_err, sizeof g_err, fmt, ap);
    va_end(ap);
    return code;
}

int check_config(const attn_decode_config *c)
{
    if (!c) return fail(ATTN_ERR_INVALID, "config is NULL");
    for (int i = 0; i < 3; ++i)
        if (c->reserved[i] != 0) return fail(ATTN_ERR_INVALID, "config.reserved[%d] must be zero", i);
    if (c->fused_merge_max_splits > kFusedSplits)
        return fail(ATTN_ERR_INVALID, "fused_merge_max_splits=%d exceeds %d", c->fused_merge_max_splits, kFusedSplits);
    if (c->n_kv_heads < 1) return fail(ATTN_ERR_INVALID, "n_kv_heads=%d must be positive", c->n_kv_heads);
    if (c->n_q_heads < 1 || c->n_q_heads % c->n_kv_heads)
        return fail(ATTN_ERR_INVALID, "n_q_heads=%d must be a positive multiple of n_kv_heads=%d", c->n_q_heads,
                    c->n_kv_heads);
    if (c->n_q_heads / c->n_kv_heads > 16)
        return fail(ATTN_ERR_UNSUPPORTED, "at most 16 query heads per key/value head (got %d)",
                    c->n_q_heads / c->n_kv_heads);
    if (c->n_kv_heads > 65535) return fail(ATTN_ERR_INVALID, "n_kv_heads=%d exceeds 65535", c->n_kv_heads);
    if (c->head_dim != kD) return fail(ATTN_ERR_UNSUPPORTED, "head_dim=%d (only %d)", c->head_dim, kD);
    if (c->page_size != kP) return fail(ATTN_ERR_UNSUPPORTED, "page_size=%d (only %d)", c->page_size, kP);
    if (c->max_batch < 1 || c->max_batch > 4096) return fail(ATTN_ERR_INVALID, "max_batch=%d outside 1..4096", c->max_batch);
    if (c->max_pages_per_seq < 1 || c->max_pages_per_seq > 65536)
        return fail(ATTN_ERR_INVALID, "max_pages_per_seq=%d outside 1..65536", c->max_pages_per_seq);
    return ATTN_OK;
}

int max_splits(const attn_decode_config *c) { return (c->max_pages_per_seq * kP + kChunk - 1) / kChunk; }

// Partials per (sequence, key/value head) the workspace holds: every 256-token chunk's
// when the second kernel merges; with the merge in the split kernel at most the split
// limit (the grid's S never exceeds it, whatever the device), so the workspace does not
// grow with the context capacity.
int partial_slots(const attn_decode_config *c)
{
    const int sf = max_splits(c);
    if (c->fused_merge_max_splits < 0) return sf;
    const int lim = c->fused_merge_max_splits == 0 ? kFusedSplits : c->fused_merge_max_splits;
    return sf < lim ? sf : lim;
}

size_t partial_o_bytes(const attn_decode_config *c)
{
    return ((size_t)c->max_batch * c->n_kv_heads * partial_slots(c) * 16 * kD * 4 + 255) & ~(size_t)255;
}

size_t partial_ml_bytes(const attn_decode_config *c)
{
    return ((size_t)c->max_batch * c->n_kv_heads * partial_slots(c) * 16 * 8 + 255) & ~(size_t)255;
}

size_t counter_words(const attn_decode_config *c) { return (size_t)c->max_batch * c->n_kv_heads; }

// The split kernel merges the splits itself when every sequence has at most this many.
// Compute units of the current device (cached per device, safe across host threads; 0 if
// the query fails).
int compute_units()
{
    static std::atomic<int> cus[64];
    int dev = 0;
    if (hipGetDevice(&dev) != hipSuccess || dev < 0 || dev >= 64) return 0;
    int n = cus[dev].load(std::memory_order_relaxed);
    if (n == 0) {
        if (hipDeviceGetAttribute(&n, hipDeviceAttributeMultiprocessorCount, dev) != hipSuccess) return 0;
        cus[dev].store(n, std::memory_order_relaxed);
    }
    return n;
}

// 256-token chunks per workgroup for a full row of the block table, which sets the
// grid's split count S = ceil(row chunks / R); 0 when the configuration asks for the
// second kernel's merge (every chunk its own split).  At least enough that `lim` splits
// cover a row.  When one chunk per split would need more than two rounds of resident
// workgroups (two per compute unit), the splits grow until the grid is at most three
// workgroups per compute unit: the walk inside a workgroup keeps as many loads in flight
// as more workgroups would, with fewer partials to merge.  Only the configuration enters;
// the kernel spreads each sequence's own chunks over the S splits.
int chunks_per_split(const attn_decode_config *c)
{
    if (c->fused_merge_max_splits < 0) return 0;
    const int lim = c->fused_merge_max_splits == 0 ? kFusedSplits : c->fused_merge_max_splits;
    const int sf = max_splits(c);
    int R = (sf + lim - 1) / lim;
    const long rows = (long)c->n_kv_heads * c->max_batch;  // workgroups per split index
    const long slots = 2L * compute_units();
    if (slots > 0 && (long)sf * rows > 2 * slots)
        while (R < sf && (long)((sf + R - 1) / R) * rows > slots * 3 / 2) ++R;
    return R;
}

bool aligned(const void *p, size_t a) { return ((uintptr_t)p & (a - 1)) == 0; }

}  // namespace
}  // namespace attn

extern "C" size_t attn_decode_workspace_bytes(const attn_decode_config *cfg)
{
    using namespace attn;
    if (check_config(cfg) != ATTN_OK) return 0;
    return partial_o_bytes(cfg) + partial_ml_bytes(cfg) + counter_words(cfg) * 4;
}

extern "C" int attn_decode_workspace_init(const attn_decode_config *cfg, void *workspace, size_t workspace_bytes,
                                          void *stream)
{
    using namespace attn;
    g_err[0] = 0;
    const int rc = check_config(cfg);
    if (rc != ATTN_OK) return rc;
    if (!workspace || !aligned(workspace, 256)) return fail(ATTN_ERR_WORKSPACE, "workspace is NULL or not 256-byte aligned");
    if (workspace_bytes < attn_decode_workspace_bytes(cfg))
        return fail(ATTN_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes,
                    attn_decode_workspace_bytes(cfg));
    int32_t *cnt = (int32_t *)((char *)workspace + partial_o_bytes(cfg) + partial_ml_bytes(cfg));
    const int n = (int)counter_words(cfg);
    attn_zero_kernel<<<(n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024, 256, 0, (hipStream_t)stream>>>(cnt, n);
    const hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(ATTN_ERR_HIP, "zero kernel launch: %s", hipGetErrorString(e));
    return ATTN_OK;
}

extern "C" int attn_decode_forward(const attn_decode_config *cfg, void *workspace, size_t workspace_bytes, void *stream,
                                   const void *q, const void *k_cache, const void *v_cache, int64_t n_pages,
                                   const int32_t *block_table, const int32_t *ctx_lens, int32_t batch, float scale,
                                   void *out)
{
    using namespace attn;
    g_err[0] = 0;
    const int rc = check_config(cfg);
    if (rc != ATTN_OK) return rc;
    if (batch < 0 || batch > cfg->max_batch) return fail(ATTN_ERR_INVALID, "batch=%d outside 0..%d", batch, cfg->max_batch);
    if (!(scale > 0.f) || !isfinite(scale)) return fail(ATTN_ERR_INVALID, "scale must be finite and positive");
    if (n_pages < 1) return fail(ATTN_ERR_INVALID, "n_pages=%lld must be positive", (long long)n_pages);
    const void *ptrs[] = {q, k_cache, v_cache, out};
    const char *names[] = {"q", "k_cache", "v_cache", "out"};
    for (int i = 0; i < 4; ++i) {
        if (!ptrs[i]) return fail(ATTN_ERR_INVALID, "%s is NULL", names[i]);
        if (!aligned(ptrs[i], 16)) return fail(ATTN_ERR_INVALID, "%s must be 16-byte aligned", names[i]);
    }
    if (!block_table || !aligned(block_table, 4)) return fail(ATTN_ERR_INVALID, "block_table is NULL or misaligned");
    if (!ctx_lens || !aligned(ctx_lens, 4)) return fail(ATTN_ERR_INVALID, "ctx_lens is NULL or misaligned");
    if (out == q || out == k_cache || out == v_cache) return fail(ATTN_ERR_INVALID, "out must not alias an input");
    if (!workspace || !aligned(workspace, 256)) return fail(ATTN_ERR_WORKSPACE, "workspace is NULL or not 256-byte aligned");
    if (workspace_bytes < attn_decode_workspace_bytes(cfg))
        return fail(ATTN_ERR_WORKSPACE, "workspace of %zu bytes, %zu needed", workspace_bytes,
                    attn_decode_workspace_bytes(cfg));
    if (batch == 0) return ATTN_OK;
    const int Hkv = cfg->n_kv_heads, G = cfg->n_q_heads / Hkv, R = chunks_per_split(cfg);
    float *po = (float *)workspace;
    float *pml = (float *)((char *)workspace + partial_o_bytes(cfg));
    int32_t *cnt = (int32_t *)((char *)workspace + partial_o_bytes(cfg) + partial_ml_bytes(cfg));
    hipStream_t st = (hipStream_t)stream;
    if (R > 0) {
        const int S = (max_splits(cfg) + R - 1) / R;  // at most the limit, and at most partial_slots
        if (S > partial_slots(cfg)) return fail(ATTN_ERR_INVALID, "internal: %d splits exceed the workspace", S);
        attn_split_kernel<true><<<dim3(S, Hkv, batch), 256, 0, st>>>(
            (const uint16_t *)q, (const uint16_t *)k_cache, (const uint16_t *)v_cache, n_pages, block_table,
            cfg->max_pages_per_seq, ctx_lens, Hkv, G, scale * kLog2e, po, pml, S, R, cnt, (uint16_t *)out);
        const hipError_t e = hipGetLastError();
        if (e != hipSuccess) return fail(ATTN_ERR_HIP, "split kernel launch: %s", hipGetErrorString(e));
        return ATTN_OK;
    }
    const int S = max_splits(cfg);
    attn_split_kernel<false><<<dim3(S, Hkv, batch), 256, 0, st>>>(
        (const uint16_t *)q, (const uint16_t *)k_cache, (const uint16_t *)v_cache, n_pages, block_table,
        cfg->max_pages_per_seq, ctx_lens, Hkv, G, scale * kLog2e, po, pml, S, 1, cnt, (uint16_t *)out);
    hipError_t e = hipGetLastError();
    if (e != hipSuccess) return fail(ATTN_ERR_HIP, "split kernel launch: %s", hipGetErrorString(e));
    attn_combine_kernel<<<dim3(G, Hkv, batch), 128, 0, st>>>(po, pml, ctx_lens, cfg->max_pages_per_seq, Hkv, G, S,
                                                             (uint16_t *)out);
    e = hipGetLastError();
    if (e != hipSuccess) return fail(ATTN_ERR_HIP, "combine kernel launch: %s", hipGetErrorString(e));
    return ATTN_OK;
}

extern "C" const char *attn_decode_last_error(void) { return attn::g_err; }
