// Routing kernels of the MoE decode step: router logits, top-k softmax and the
// token-to-expert grouping.  One decode step of a MoE layer starts here (the decode
// lane of the paper's Background section; the MoE models of its Experimental Setup).
#include <hip/hip_runtime.h>
#include <math.h>

#include "fp8split.h"
#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kWave = 64;

// Values exchanged between workgroups of this kernel (logits, selected experts) are
// written and read with device-scope atomic stores and loads, which bypass the
// per-XCD L2 caches; a producer waits for its stores to complete before it bumps a
// counter.  This avoids whole-cache write-back / invalidate fences, which serialise
// per XCD.
template <typename T>
__device__ inline void st_dev(T *p, T v) { __hip_atomic_store(p, v, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
template <typename T>
__device__ inline T ld_dev(const T *p) { return __hip_atomic_load(const_cast<T *>(p), __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_AGENT); }
// The memory clobber keeps the compiler from moving memory accesses across the wait,
// so every store issued before it has completed when the counter is bumped.
__device__ inline void wait_stores() { asm volatile("s_waitcnt vmcnt(0)" ::: "memory"); }

// ------------------------------------------------------------------ router logits
//
// Canonical logit: one round-to-nearest-even to fp32 of the exact value of
// sum_h x[h] * w[h] + b.  Products of bf16 or fp32 operands are exact in fp64.
// Fast path: each lane sums its products in fp64 (one FMA each) together with
// sum |x*w|; the wave combines lanes by a butterfly.  Every product then passes
// through at most D roundings (D = products per lane + 6 butterfly levels + 1 for
// the bias), so |sum - exact| <= gamma_D * (sum|x*w| + |b|), gamma_D = D u/(1-D u),
// u = 2^-53.  If the interval sum +- bound (plus one fp64 ulp of slack) lies
// strictly between the two fp32 rounding midpoints around RNE(sum), every value in
// it rounds to the same fp32 number, which is then the canonical logit.  Otherwise
// the wave recomputes the sum in double-double (error-free TwoSum accumulation,
// about 106 significant bits) and rounds hi + lo with the tie resolved by lo.

__device__ inline double bf16_to_f64(uint32_t bits16) { return (double)__uint_as_float(bits16 << 16); }

__device__ inline void two_sum(double a, double b, double &s, double &e)
{
    s = a + b;
    double bb = s - a;
    e = (a - (s - bb)) + (b - bb);
}

// (h, l) += (h2, l2); symmetric in its operands, so butterfly partners agree.
__device__ inline void dd_add(double &h, double &l, double h2, double l2)
{
    double s, e;
    two_sum(h, h2, s, e);
    e += l + l2;
    h = s + e;
    l = e - (h - s);
}

// Round hi + lo (|lo| <= ulp(hi)/2) to fp32, nearest, ties to even.
__device__ inline float round_dd_to_f32(double hi, double lo)
{
    float r = (float)hi;
    double rd = (double)r;
    if (rd == hi) return r;
    float other = hi > rd ? nextafterf(r, INFINITY) : nextafterf(r, -INFINITY);
    double mid = 0.5 * (rd + (double)other);
    if (hi != mid || lo == 0.0) return r;  // not a tie, or an exact tie already resolved to even
    return ((lo > 0.0) == ((double)other > rd)) ? other : r;
}

// True if every real number within `bound` of v rounds to the same fp32 value r.
__device__ inline bool certain_f32(double v, double bound, float &r)
{
    r = (float)v;
    double rd = (double)r;
    double lo_mid = 0.5 * (rd + (double)nextafterf(r, -INFINITY));
    double hi_mid = 0.5 * (rd + (double)nextafterf(r, INFINITY));
    double margin = bound + fabs(v) * 0x1p-51;
    return (v - lo_mid > margin) && (hi_mid - v > margin);
}

template <typename T>
__device__ inline void load8(const T *p, double (&v)[8]);

template <>
__device__ inline void load8<uint16_t>(const uint16_t *p, double (&v)[8])
{
    uint4 q = *reinterpret_cast<const uint4 *>(p);
    uint32_t w[4] = {q.x, q.y, q.z, q.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = bf16_to_f64(w[i] & 0xFFFFu);
        v[2 * i + 1] = bf16_to_f64(w[i] >> 16);
    }
}

template <>
__device__ inline void load8<float>(const float *p, double (&v)[8])
{
    float4 a = *reinterpret_cast<const float4 *>(p);
    float4 b = *reinterpret_cast<const float4 *>(p + 4);
    v[0] = a.x; v[1] = a.y; v[2] = a.z; v[3] = a.w;
    v[4] = b.x; v[5] = b.y; v[6] = b.z; v[7] = b.w;
}

// Exact (double-double) logit of one (token, expert) pair, computed by one wave: the
// slow path taken when the fp64 sum cannot certify its fp32 rounding.
template <typename XT, typename WT>
__device__ __attribute__((always_inline)) inline float wave_logit_exact(const XT *__restrict__ xr, const WT *__restrict__ wrow, double b, int H,
                                         int lane)
{
    double hi = 0.0, lo = 0.0;
    for (int h = lane * 8; h < H; h += 512) {
        double xv[8], wv[8];
        load8<XT>(xr + h, xv);
        load8<WT>(wrow + h, wv);
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            double p = xv[i] * wv[i], ss, ee;  // exact product
            two_sum(hi, p, ss, ee);
            hi = ss;
            lo += ee;
        }
    }
    double nh = hi + lo;  // normalise the lane's pair before combining
    lo = lo - (nh - hi);
    hi = nh;
#pragma unroll
    for (int o = kWave / 2; o >= 1; o >>= 1) {
        double h2 = __shfl_xor(hi, o), l2 = __shfl_xor(lo, o);
        dd_add(hi, lo, h2, l2);
    }
    dd_add(hi, lo, b, 0.0);
    return round_dd_to_f32(hi, lo);
}

// Eight consecutive inputs of one lane, as raw bits (bf16: 4 words, fp32: 8 words).
template <typename T>
struct Chunk8 {
    uint32_t d[sizeof(T) == 2 ? 4 : 8];
};

template <typename T>
__device__ inline void ld_chunk(const T *p, Chunk8<T> &c)
{
#pragma unroll
    for (int q = 0; q < (int)(sizeof(c.d) / 16); ++q) {
        const uint4 u = reinterpret_cast<const uint4 *>(p)[q];
        c.d[4 * q] = u.x;
        c.d[4 * q + 1] = u.y;
        c.d[4 * q + 2] = u.z;
        c.d[4 * q + 3] = u.w;
    }
}

template <typename T>
__device__ inline double elem(const Chunk8<T> &c, int i)
{
    if constexpr (sizeof(T) == 2)
        return (double)__uint_as_float((i & 1) ? (c.d[i >> 1] & 0xFFFF0000u) : (c.d[i >> 1] << 16));
    else
        return (double)__uint_as_float(c.d[i]);
}

constexpr int kEPW = 4;  // experts per wave, at most

// One fp64 value moved by a DPP lane permutation (ctrl: an immediate DPP control).
template <int CTRL>
__device__ inline double dpp_f64(double v)
{
    const uint64_t u = __double_as_longlong(v);
    const uint32_t lo = __builtin_amdgcn_update_dpp(0u, (uint32_t)u, CTRL, 0xF, 0xF, false);
    const uint32_t hi = __builtin_amdgcn_update_dpp(0u, (uint32_t)(u >> 32), CTRL, 0xF, 0xF, false);
    return __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
}

// Sum of v over the wave, the same in every lane: DPP quad permutes and the half-row
// and row mirrors give each 16-lane row its sum, and the four row sums are added from
// scalar registers.  Six additions deep, like a butterfly, so the recursive-summation
// bound of the caller holds.
__device__ inline double wave_sum_f64(double v)
{
    v += dpp_f64<0xB1>(v);   // quad_perm [1,0,3,2]
    v += dpp_f64<0x4E>(v);   // quad_perm [2,3,0,1]
    v += dpp_f64<0x141>(v);  // row_half_mirror
    v += dpp_f64<0x140>(v);  // row_mirror
    double r[4];
#pragma unroll
    for (int row = 0; row < 4; ++row) {
        const uint64_t u = __double_as_longlong(v);
        const uint32_t lo = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)u, 16 * row);
        const uint32_t hi = (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)(u >> 32), 16 * row);
        r[row] = __longlong_as_double((long long)(((uint64_t)hi << 32) | lo));
    }
    return (r[0] + r[1]) + (r[2] + r[3]);
}

__device__ inline float bf16_lo(uint32_t w) { return __uint_as_float(w << 16); }
__device__ inline float bf16_hi(uint32_t w) { return __uint_as_float(w & 0xFFFF0000u); }

// Canonical logits of one token row xr against router rows e0 .. e0+ne-1 (ne <= EPW),
// or the rows elist[0 .. ne-1],
// computed by one wave and written to lrow[e].  The lane's inputs are loaded once per
// segment and reused for every expert; the next expert's router row is in flight
// while the current one accumulates.  Returns the number of fallbacks taken.
//
// Each lane sums exact products in fp64 (two accumulators per expert) next to a bound
// on the sum of their magnitudes; the wave-reduced sum is certified against the fp32
// rounding midpoints with the recursive-summation error bound, else recomputed exactly.
// With bf16 inputs a product of two bf16 values is exact in fp32 (16-bit significand),
// so it is formed in fp32 and added in fp64, and the magnitude bound is summed in fp32
// and inflated by its own worst-case rounding; products below the fp32 subnormal grain
// add at most H*2^-149 in absolute error, which the margin covers.  fp32 inputs use
// fp64 fused multiply-adds throughout.
//
// EPW is the wave's expert capacity (ne <= EPW) and SEG the 8-input chunks per lane
// held at once: one expert per wave loads a 4096-input row in one round trip.
template <typename XT, typename WT, int EPW, int SEG>
__device__ __attribute__((always_inline)) inline int wave_logits(const XT *__restrict__ xr, const WT *__restrict__ wr, const float *bias, int H,
                                  int e0, int ne, int lane, float *lrow, const int *elist = nullptr)
{
    // expert i of the call: elist[i] if a list is given, else e0 + i
    int ex[EPW];
#pragma unroll
    for (int i = 0; i < EPW; ++i) ex[i] = elist ? elist[i < ne ? i : 0] : e0 + (i < ne ? i : 0);
    constexpr bool kBf16 = sizeof(XT) == 2 && sizeof(WT) == 2;
    const int nck = (H + 511) / 512;  // chunks of the lane with the most
    // Two accumulators per expert (even and odd chunks): each sums at most
    // ceil(nck/2)*8 products, then they are added and reduced over the wave.
    const int per_acc = ((nck + 1) / 2) * 8;
    const double gamma = (double)(per_acc + 1 + 6 + 1 + 2) * 0x1p-52;  // >= 2 gamma_D
    const double infl = 1.0 + (double)(per_acc + 2) * 0x1p-23;         // fp32 magnitude sums
    double s[EPW][2], a[EPW][2];
    float a32[EPW][2];
#pragma unroll
    for (int i = 0; i < EPW; ++i) {
        s[i][0] = s[i][1] = a[i][0] = a[i][1] = 0.0;
        a32[i][0] = a32[i][1] = 0.f;
    }
    for (int seg = 0; seg < nck; seg += SEG) {
        Chunk8<XT> xc[SEG];
        bool valid[SEG];
        int off[SEG];
#pragma unroll
        for (int j = 0; j < SEG; ++j) {
            const int h = lane * 8 + 512 * (seg + j);
            valid[j] = h < H;
            off[j] = valid[j] ? h : H - 8;  // clamped: an invalid chunk is loaded but its x is 0
            ld_chunk<XT>(xr + off[j], xc[j]);
            if (!valid[j])
#pragma unroll
                for (int q = 0; q < (int)(sizeof(xc[j].d) / 4); ++q) xc[j].d[q] = 0u;
        }
        float xf[SEG][8];
        if constexpr (kBf16)
#pragma unroll
            for (int j = 0; j < SEG; ++j)
#pragma unroll
                for (int q = 0; q < 4; ++q) {
                    xf[j][2 * q] = bf16_lo(xc[j].d[q]);
                    xf[j][2 * q + 1] = bf16_hi(xc[j].d[q]);
                }
        // every expert's slice of this segment in flight at once (one memory latency)
        Chunk8<WT> wc[EPW][SEG];
#pragma unroll
        for (int i = 0; i < EPW; ++i)
#pragma unroll
            for (int j = 0; j < SEG; ++j)
                ld_chunk<WT>(wr + (size_t)ex[i] * H + off[j], wc[i][j]);
#pragma unroll
        for (int i = 0; i < EPW; ++i) {
            if (i < ne) {
#pragma unroll
                for (int j = 0; j < SEG; ++j)
#pragma unroll
                    for (int q = 0; q < 8; ++q) {
                        if constexpr (kBf16) {
                            const uint32_t wd = wc[i][j].d[q >> 1];
                            const float wv = (q & 1) ? bf16_hi(wd) : bf16_lo(wd);
                            const float pv = xf[j][q] * wv;  // exact
                            s[i][j & 1] += (double)pv;
                            a32[i][j & 1] = fmaf(fabsf(xf[j][q]), fabsf(wv), a32[i][j & 1]);
                        } else {
                            const double xv = elem<XT>(xc[j], q), wv = elem<WT>(wc[i][j], q);
                            s[i][j & 1] = fma(xv, wv, s[i][j & 1]);
                            a[i][j & 1] = fma(fabs(xv), fabs(wv), a[i][j & 1]);
                        }
                    }
            }
        }
    }
    int nfb = 0;
#pragma unroll
    for (int i = 0; i < EPW; ++i) {
        if (i < ne) {
            const double si = wave_sum_f64(s[i][0] + s[i][1]);
            const double ai = wave_sum_f64(kBf16 ? ((double)a32[i][0] + (double)a32[i][1]) * infl : a[i][0] + a[i][1]);
            const int e = ex[i];
            const double b = bias ? (double)bias[e] : 0.0;
            const double slack = kBf16 ? (double)H * 0x1p-148 : 0.0;
            float r;
            if (!certain_f32(si + b, gamma * (ai + fabs(b)) + slack, r)) {
                r = wave_logit_exact<XT, WT>(xr, wr + (size_t)e * H, b, H, lane);
                ++nfb;
            }
            if (lane == 0) st_dev(&lrow[e], r + 0.0f);  // -0 -> +0
        }
    }
    return nfb;
}

// ------------------------------------------------------------------ top-k keys
//
// A key is (order-preserving integer image of the fp32 logit) << 32 | (~expert): the
// largest key is the largest logit, ties going to the lower expert index.

__device__ inline uint32_t ordered_bits(float f)
{
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float from_ordered(uint32_t o) { return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o); }

template <typename XT>
__device__ inline void load32_f32(const XT *p, float (&v)[32]);

template <>
__device__ inline void load32_f32<uint16_t>(const uint16_t *p, float (&v)[32])
{
#pragma unroll
    for (int q = 0; q < 4; ++q) {
        const uint4 u = reinterpret_cast<const uint4 *>(p)[q];
        const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
        for (int i = 0; i < 4; ++i) {
            v[8 * q + 2 * i] = __uint_as_float(w[i] << 16);
            v[8 * q + 2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
        }
    }
}

template <>
__device__ inline void load32_f32<float>(const float *p, float (&v)[32])
{
#pragma unroll
    for (int q = 0; q < 8; ++q) {
        const float4 u = reinterpret_cast<const float4 *>(p)[q];
        v[4 * q] = u.x;
        v[4 * q + 1] = u.y;
        v[4 * q + 2] = u.z;
        v[4 * q + 3] = u.w;
    }
}

// ------------------------------------------------------------------ block scan

// Inclusive prefix sum over a wave with DPP row shifts (each 16-lane row), then the
// row totals read from lanes 15, 31, 47 and 63.  Returns the wave total.
__device__ inline int wave_inclusive_scan(int &v, int lane)
{
    v += __builtin_amdgcn_update_dpp(0, v, 0x111, 0xF, 0xF, false);  // row_shr:1
    v += __builtin_amdgcn_update_dpp(0, v, 0x112, 0xF, 0xF, false);  // row_shr:2
    v += __builtin_amdgcn_update_dpp(0, v, 0x114, 0xF, 0xF, false);  // row_shr:4
    v += __builtin_amdgcn_update_dpp(0, v, 0x118, 0xF, 0xF, false);  // row_shr:8
    const int t0 = __builtin_amdgcn_readlane(v, 15), t1 = __builtin_amdgcn_readlane(v, 31),
              t2 = __builtin_amdgcn_readlane(v, 47), t3 = __builtin_amdgcn_readlane(v, 63);
    const int row = lane >> 4;
    v += (row >= 1 ? t0 : 0) + (row >= 2 ? t1 : 0) + (row >= 3 ? t2 : 0);
    return t0 + t1 + t2 + t3;
}

// Exclusive prefix sums of four counters over the 256 threads of a workgroup.
__device__ inline void block_exscan4(int (&v)[4], int (&tot)[4], int *sh /* [4 waves][4] */)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    int inc[4] = {v[0], v[1], v[2], v[3]};
    int wt[4];
#pragma unroll
    for (int c = 0; c < 4; ++c) wt[c] = wave_inclusive_scan(inc[c], lane);
    if (lane == 0)
        for (int c = 0; c < 4; ++c) sh[wave * 4 + c] = wt[c];
    __syncthreads();
    for (int c = 0; c < 4; ++c) {
        int before = 0, all = 0;
        for (int w = 0; w < 4; ++w) {
            const int s = sh[w * 4 + c];
            if (w < wave) before += s;
            all += s;
        }
        tot[c] = all;
        v[c] = before + inc[c] - v[c];
    }
    __syncthreads();
}

// Wave-wide maximum of 64-bit keys with DPP lane permutations: two quad permutes
// and the half-row and row mirrors leave every lane of a 16-lane row with the row's
// maximum; the four row maxima are combined in scalar registers.
__device__ inline uint64_t dpp_max64(uint64_t v, int ctrl_sel)
{
    uint32_t lo = (uint32_t)v, hi = (uint32_t)(v >> 32), olo, ohi;
    switch (ctrl_sel) {  // the DPP control is an immediate
    case 0:
        olo = __builtin_amdgcn_update_dpp(0u, lo, 0xB1, 0xF, 0xF, false);  // quad_perm [1,0,3,2]
        ohi = __builtin_amdgcn_update_dpp(0u, hi, 0xB1, 0xF, 0xF, false);
        break;
    case 1:
        olo = __builtin_amdgcn_update_dpp(0u, lo, 0x4E, 0xF, 0xF, false);  // quad_perm [2,3,0,1]
        ohi = __builtin_amdgcn_update_dpp(0u, hi, 0x4E, 0xF, 0xF, false);
        break;
    case 2:
        olo = __builtin_amdgcn_update_dpp(0u, lo, 0x141, 0xF, 0xF, false);  // row_half_mirror
        ohi = __builtin_amdgcn_update_dpp(0u, hi, 0x141, 0xF, 0xF, false);
        break;
    default:
        olo = __builtin_amdgcn_update_dpp(0u, lo, 0x140, 0xF, 0xF, false);  // row_mirror
        ohi = __builtin_amdgcn_update_dpp(0u, hi, 0x140, 0xF, 0xF, false);
        break;
    }
    const uint64_t o = ((uint64_t)ohi << 32) | olo;
    return o > v ? o : v;
}

__device__ inline uint64_t wave_max64(uint64_t v)
{
    v = dpp_max64(v, 0);
    v = dpp_max64(v, 1);
    v = dpp_max64(v, 2);
    v = dpp_max64(v, 3);
    uint64_t m = 0;
#pragma unroll
    for (int row = 0; row < 4; ++row) {
        // readlane returns a signed int: widen through uint32_t
        const uint64_t r = ((uint64_t)(uint32_t)__builtin_amdgcn_readlane((int)(v >> 32), 16 * row) << 32) |
                           (uint32_t)__builtin_amdgcn_readlane((int)(uint32_t)v, 16 * row);
        m = r > m ? r : m;
    }
    return m;
}

// Top-k softmax of one token by one wave.  Keys are (ordered logit bits, complemented
// expert index): a larger logit wins, and among equal logits the lower index.  Lane
// owns keys of experts lane, lane+64, ... (V per lane, E <= 64V).  k rounds of a
// wave-wide argmax (DPP lane permutations, see wave_max64) each take the largest
// remaining key; lane j keeps choice j.  Weights are the softmax of the selected logits in
// fp32 relative to the largest, normalised by their butterfly sum, which every lane
// forms from the same pairs.
template <int V, bool MASK>
__device__ __attribute__((always_inline)) inline void wave_topk(const float *__restrict__ l, int E, int k, int32_t *ids, float *wts,
                                 int32_t *ids_user, float *wts_user, int lane, const uint32_t *cand)
{
    uint64_t key[V];
#pragma unroll
    for (int v = 0; v < V; ++v) {
        const int e = 64 * v + lane;
        bool in = e < E;
        if constexpr (MASK) in = in && ((cand[e >> 5] >> (e & 31)) & 1u);
        key[v] = in ? ((uint64_t)ordered_bits(ld_dev(&l[e])) << 32) | (uint32_t)(~(uint32_t)e) : 0;
    }
    uint64_t mine = 0;  // lane j < k: key of choice j
    for (int j = 0; j < k; ++j) {
        uint64_t best = key[0];
#pragma unroll
        for (int v = 1; v < V; ++v) best = key[v] > best ? key[v] : best;
        best = wave_max64(best);
        if (lane == j) mine = best;
#pragma unroll
        for (int v = 0; v < V; ++v) key[v] = key[v] == best ? 0 : key[v];  // keys are unique
    }
    const float top = from_ordered((uint32_t)__shfl((uint32_t)(mine >> 32), 0));
    const float p = lane < k ? expf(from_ordered((uint32_t)(mine >> 32)) - top) : 0.f;
    float den = p;
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) den += __shfl_xor(den, o);
    if (lane < k) {
        const int e = (int)(~(uint32_t)mine);
        const float w = p / den;
        st_dev(&ids[lane], e);
        wts[lane] = w;
        if (ids_user) ids_user[lane] = e;
        if (wts_user) wts_user[lane] = w;
    }
}

// MASK: only the experts of the bitmask `cand` may be selected (the others' logits need
// not be valid).
template <bool MASK = false>
__device__ __attribute__((always_inline)) inline void token_topk(const float *__restrict__ l, int E, int k, int32_t *ids, float *wts,
                                  int32_t *ids_user, float *wts_user, int lane, const uint32_t *cand = nullptr)
{
    if (E <= 64)
        wave_topk<1, MASK>(l, E, k, ids, wts, ids_user, wts_user, lane, cand);
    else if (E <= 128)
        wave_topk<2, MASK>(l, E, k, ids, wts, ids_user, wts_user, lane, cand);
    else if (E <= 256)
        wave_topk<4, MASK>(l, E, k, ids, wts, ids_user, wts_user, lane, cand);
    else if (E <= 512)
        wave_topk<8, MASK>(l, E, k, ids, wts, ids_user, wts_user, lane, cand);
    else
        wave_topk<16, MASK>(l, E, k, ids, wts, ids_user, wts_user, lane, cand);
}

// ------------------------------------------------------------------ fused routing kernel
//
// Grid = T x bpt workgroups of 4 waves.  Workgroup (t, q) computes the logits of token
// t for experts [4*q*epw, 4*(q+1)*epw).  The last workgroup of token t to finish (a
// device-scope counter) runs that token's top-k softmax in one wave while its other
// three waves write the token's 2-term FP8 activation split (when the MFMA path is
// on).  The last token to finish then groups all (token, choice) pairs by expert.  The
// counters are reset by the workgroup that consumes them, so they read zero at the
// start of every launch.


struct RouteArgs {
    const void *x;
    const void *wr;
    const float *bias;
    float *logits;
    int32_t *ids, *ids_user;
    float *wts, *wts_user;
    int32_t *meta, *slot_of, *tok_of;
    int32_t *cnt_tok;  // [Tmax][kCounterStride], one counter per 256-byte line
    int32_t *cnt_all;  // [1]
    int32_t *fb_acc;   // [1]
    uint8_t *xs_hi, *xs_lo, *xe_hi, *xe_lo;  // activation split (NULL: MFMA path off)
    _Float16 *x16;                           // f16 copy of x * 2^-k (NULL: none)
    int32_t *xk;                             // [T] the token's k
    int T, E, H, k, epw, bpt, mstar, do_group, max_chunks;
    int id_cache;  // the grouping keeps the choices in LDS (sized by the launch)
    // screened routing (large T): per K slice ks, partial sums part[ks][t][e] =
    // (sum x*w, sum |x*w|) and the slice's max |x[t,.]|, max |w[e,.]|
    double2 *part;
    float *xmax, *wmax;
    int KS, Tmax;
};

// The 2-term FP8 split of token t's activations (groups of 32 inputs, see fp8split.h),
// groups first, first + stride, ... written by the calling thread.
template <typename XT>
__device__ __attribute__((always_inline)) inline void write_split(const RouteArgs &A, const XT *xr, int t, int first, int stride)
{
    const int H = A.H, G = H / 32;
    for (int g = first; g < G; g += stride) {
        float v[32], res[32];
        uint32_t qh[8], ql[8];
        load32_f32<XT>(xr + g * 32, v);
        const int ch = exp_for_group(amax_of(v));
        split_hi(v, ch, qh, res);
        const int cl = exp_for_group(amax_of(res));
        split_lo(res, cl, ql);
        const size_t o = (size_t)t * H + g * 32;
        reinterpret_cast<uint4 *>(A.xs_hi + o)[0] = make_uint4(qh[0], qh[1], qh[2], qh[3]);
        reinterpret_cast<uint4 *>(A.xs_hi + o)[1] = make_uint4(qh[4], qh[5], qh[6], qh[7]);
        reinterpret_cast<uint4 *>(A.xs_lo + o)[0] = make_uint4(ql[0], ql[1], ql[2], ql[3]);
        reinterpret_cast<uint4 *>(A.xs_lo + o)[1] = make_uint4(ql[4], ql[5], ql[6], ql[7]);
        A.xe_hi[(size_t)t * (H / 32) + g] = (uint8_t)ch;
        A.xe_lo[(size_t)t * (H / 32) + g] = (uint8_t)cl;
    }
}

// The token's bf16 x as f16 scaled by 2^-k, with k such that max|x| * 2^-k lies in
// [2^14, 2^15) (k = 0 for a zero row; k >= -112): every value at least 2^-31 of the
// row's maximum converts exactly.  Called by `nw` waves (wave index w), each of which
// takes the row maximum on its own (no barrier among them) and converts every nw-th
// group of eight inputs.
__device__ inline void bf16x8_f32(const uint16_t *p, float (&v)[8])
{
    const uint4 u = *reinterpret_cast<const uint4 *>(p);
    const uint32_t w[4] = {u.x, u.y, u.z, u.w};
#pragma unroll
    for (int i = 0; i < 4; ++i) {
        v[2 * i] = __uint_as_float(w[i] << 16);
        v[2 * i + 1] = __uint_as_float(w[i] & 0xFFFF0000u);
    }
}

__device__ __attribute__((always_inline)) inline void write_x16(const RouteArgs &A, const uint16_t *xr, int t, int w,
                                                                int nw, int lane)
{
    const int H = A.H;
    float m = 0.f;
    for (int h = lane * 8; h < H; h += 512) {
        float v[8];
        bf16x8_f32(xr + h, v);
#pragma unroll
        for (int i = 0; i < 8; ++i) m = fmaxf(m, fabsf(v[i]));
    }
#pragma unroll
    for (int o = 32; o >= 1; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    const int ex = m > 0.f ? (int)((__float_as_uint(m) >> 23) & 0xFF) - 127 : 14;  // floor(log2 m) for normal m
    const int kk = max(ex - 14, -112);
    const float sc = __uint_as_float((uint32_t)(127 - kk) << 23);  // 2^-k
    for (int h = (w * 64 + lane) * 8; h < H; h += nw * 512) {
        float v[8];
        bf16x8_f32(xr + h, v);
        _Float16 q[8];
#pragma unroll
        for (int i = 0; i < 8; ++i) q[i] = (_Float16)(v[i] * sc);
        *reinterpret_cast<uint4 *>(A.x16 + (size_t)t * H + h) = __builtin_bit_cast(uint4, q);
    }
    if (w == 0 && lane == 0) A.xk[t] = kk;
}

// Last token of a step: group the T*k (token, choice) pairs by expert.  LDS holds one
// bit per (expert, token): expert e's tokens in token order.  counts = popcounts,
// offsets = exclusive prefix sum, slot of pair (t, j) choosing e = offsets[e] +
// (number of earlier tokens that chose e).  Experts with at least `mstar` tokens go
// to the MFMA list, the others to the GEMV list, each in expert order.  All threads
// of the workgroup call it.
__device__ __attribute__((always_inline)) inline void group_pairs(const RouteArgs &A, uint32_t *lds, int *s_scan)
{
    const int E = A.E;
    const int T = A.T, k = A.k, P = T * k;
    const int W = (T + 31) / 32;
    uint32_t *mask = lds;                        // [E][W]
    int32_t *offs = (int32_t *)(lds + E * W);    // [E]
    int32_t *idc = offs + E;                     // [P] when the launch sized LDS for it: the choices, read once
    const bool cached = A.id_cache != 0;
    const MetaIdx mi{E, A.max_chunks};
    int nfb_total = 0, n_exact = A.T * E;
    if (threadIdx.x == 0) {  // in flight during the grouping; each counter is reset by its reader
        nfb_total = atomicExch(A.fb_acc, 0);
        if (A.KS) n_exact = atomicExch(A.fb_acc + kCandCounterOff, 0);
    }
    for (int i = threadIdx.x; i < E * W; i += blockDim.x) mask[i] = 0u;
    __syncthreads();
    // this thread's choices, eight loads in flight at a time
    for (int p0 = threadIdx.x; p0 < P; p0 += 8 * blockDim.x) {
        int e8[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int p = p0 + u * blockDim.x;
            e8[u] = p < P ? ld_dev(&A.ids[p]) : 0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            const int p = p0 + u * blockDim.x;
            if (p < P) {
                const int tt = p / k;
                atomicOr(&mask[e8[u] * W + tt / 32], 1u << (tt % 32));
                if (cached) idc[p] = e8[u];
            }
        }
    }
    __syncthreads();
    // each thread owns up to 4 consecutive experts
    const int per = (E + 255) / 256;
    const int eb = threadIdx.x * per;
    int cnt[4] = {0, 0, 0, 0};
    int v[4] = {0, 0, 0, 0};  // tokens, gemv experts, mfma experts, mfma token chunks
    for (int j = 0; j < per; ++j) {
        const int e = eb + j;
        if (e < E) {
            int c = 0;
            for (int w = 0; w < W; ++w) c += __popc(mask[e * W + w]);
            cnt[j] = c;
            v[0] += c;
            if (c > 0) {
                if (A.mstar > 0 && c >= A.mstar) {
                    v[2]++;
                    v[3] += (c + kMfmaChunk - 1) / kMfmaChunk;
                } else {
                    v[1]++;
                }
            }
        }
    }
    int tot[4];
    block_exscan4(v, tot, s_scan);
    for (int j = 0; j < per; ++j) {
        const int e = eb + j;
        if (e < E) {
            const int c = cnt[j];
            offs[e] = v[0];
            A.meta[mi.counts() + e] = c;
            A.meta[mi.offsets() + e] = v[0];
            if (c > 0) {
                if (A.mstar > 0 && c >= A.mstar) {
                    int4 *cr = reinterpret_cast<int4 *>(A.meta + mi.chunk_rec());
                    for (int m0 = 0; m0 < c; m0 += kMfmaChunk)
                        cr[v[3]++] = make_int4(e, v[0] + m0, min(kMfmaChunk, c - m0), 0);
                    v[2]++;
                } else {
                    reinterpret_cast<int4 *>(A.meta + mi.gemv_rec())[v[1]++] = make_int4(e, v[0], c, 0);
                }
            }
            v[0] += c;
        }
    }
    if (threadIdx.x == 0) {
        A.meta[mi.offsets() + E] = tot[0];
        A.meta[mi.n_active()] = tot[1] + tot[2];
        A.meta[mi.n_gemv()] = tot[1];
        A.meta[mi.n_mfma()] = tot[2];
        A.meta[mi.n_fallback()] = nfb_total;
        A.meta[mi.n_mfma_chunks()] = tot[3];
        A.meta[mi.n_exact()] = n_exact;
        A.meta[mi.screened()] = A.KS ? 1 : 0;
        st_dev(A.cnt_all, 0);
    }
    __syncthreads();
    for (int p = threadIdx.x; p < P; p += blockDim.x) {
        const int tt = p / k, e = cached ? idc[p] : ld_dev(&A.ids[p]);
        int rank = __popc(mask[e * W + tt / 32] & ((1u << (tt % 32)) - 1u));
        for (int w = 0; w < tt / 32; ++w) rank += __popc(mask[e * W + w]);
        const int slot = offs[e] + rank;
        A.slot_of[p] = slot;
        A.tok_of[slot] = tt;
    }
}

template <typename XT, typename WT>
__global__ __launch_bounds__(256) void route_kernel(RouteArgs A)
{
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    __shared__ int s_flag;
    __shared__ int s_scan[16];
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
    const int t = blockIdx.x / A.bpt;
    const int q = blockIdx.x % A.bpt;
    const int E = A.E, H = A.H;
    const XT *xr = (const XT *)A.x + (size_t)t * H;

    // 1. logits of this workgroup's experts
    {
        const int e0 = (q * 4 + wave) * A.epw;
        const int ne = min(E, e0 + A.epw) - e0;
        if (ne > 0) {
            const WT *wr = (const WT *)A.wr;
            float *lrow = A.logits + (size_t)t * E;
            // one expert per wave: no loads for empty expert slots, and a row of up to
            // 4096 bf16 inputs in one round trip
            int nfb;
            if (A.epw > 1)
                nfb = wave_logits<XT, WT, kEPW, 4>(xr, wr, A.bias, H, e0, ne, lane, lrow);
            else if (sizeof(XT) == 2 && H <= 8 * 512)
                nfb = wave_logits<XT, WT, 1, 8>(xr, wr, A.bias, H, e0, ne, lane, lrow);
            else
                nfb = wave_logits<XT, WT, 1, 4>(xr, wr, A.bias, H, e0, ne, lane, lrow);
            if (lane == 0 && nfb) atomicAdd(A.fb_acc, nfb);
        }
    }
    // Publish this workgroup's logits, then count it; the last workgroup of the token
    // goes on.
    wait_stores();
    __syncthreads();
    if (threadIdx.x == 0) s_flag = atomicAdd(&A.cnt_tok[t * kCounterStride], 1) == A.bpt - 1;
    __syncthreads();
    if (!s_flag) return;

    // 2. last workgroup of token t: top-k softmax in wave 0 while waves 1-3 write the
    // token's 2-term activation split when the MFMA path is on (groups of 32 inputs), or
    // its scaled f16 copy for NVFP4 weights
    if (wave == 0) {
        token_topk(A.logits + (size_t)t * E, E, A.k, A.ids + (size_t)t * A.k, A.wts + (size_t)t * A.k,
                   A.ids_user ? A.ids_user + (size_t)t * A.k : nullptr,
                   A.wts_user ? A.wts_user + (size_t)t * A.k : nullptr, lane);
    } else if (A.xs_hi) {
        write_split<XT>(A, xr, t, threadIdx.x - kWave, blockDim.x - kWave);
    } else if constexpr (sizeof(XT) == 2) {
        if (A.x16) write_x16(A, xr, t, wave - 1, 3, lane);
    }
    if (threadIdx.x == 0) st_dev(&A.cnt_tok[t * kCounterStride], 0);
    if (!A.do_group) return;
    wait_stores();
    __syncthreads();
    // One token: its last workgroup is the step's last, without the second counter's
    // round trip (group_pairs leaves that counter at zero, where it already is).
    if (A.T > 1) {
        if (threadIdx.x == 0) s_flag = atomicAdd(A.cnt_all, 1) == A.T - 1;
        __syncthreads();
        if (!s_flag) return;
    }

    group_pairs(A, lds, s_scan);
}

// ------------------------------------------------------------------ screened routing
//
// At large T the exact logits of every (token, expert) pair are the step's largest
// vector-ALU cost.  Only the top-k of each token need them, so the screened path
// first brackets every logit and then computes exactly only the experts whose
// bracket can reach the top k:
//   screen_kernel    bf16 MFMA sums of x.w and |x|.|w| over 256-input chunks (fp32
//                    inside a chunk, fp64 across chunks), per K slice;
//   route_cand_kernel per token: the bracket [lo_e, hi_e] of every canonical logit
//                    l_e, LB = the k-th largest lo; e can be selected only if
//                    hi_e >= LB (k experts f have l_f >= lo_f >= LB > hi_e >= l_e
//                    otherwise); exact logits of those candidates (wave_logits), top-k
//                    among them by (l desc, e asc), softmax; the last token groups.
// Bracket.  A chunk of 256 exact products summed in fp32 in any order with any
// rounding is within g = 256u/(1-256u), u = 2^-23, of its exact sum times the sum of
// |products|; flushed denormal inputs, products or partial sums add at most
// 2^-126 (max|x| + max|w| + 2) per product; the fp64 sums across chunks and slices
// add at most 2^-40 of sum|products|; the bias add one fp64 rounding; the canonical
// rounding to fp32 at most 2^-23 relative plus 2^-149.

constexpr int kScreenChunk = 256;  // inputs per fp32 MFMA chunk
constexpr int kMaxE = 1024;
constexpr int kMaxKS = kScreenMaxKS;  // K slices of the screen at most
constexpr size_t kCandStaticLds = 12800;  // bytes, at least route_cand_kernel's static LDS

typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4v __attribute__((ext_vector_type(4)));
typedef uint16_t u16x2 __attribute__((ext_vector_type(2)));
constexpr uint32_t kScreenOOR = 0x80000000u;  // buffer offset past every resource: zeros, no request

__device__ inline __amdgpu_buffer_rsrc_t screen_rsrc(const void *base, uint32_t bytes)
{
    return __builtin_amdgcn_make_buffer_rsrc(const_cast<void *>(base), (short)0, (int)bytes, 0x00020000);
}

// Grid (ceil(T/16), ceil(E/64), KS), 256 threads.  Wave w: experts e0 = 64y + 16w .. +16
// (MFMA rows: A = router rows), tokens 16x .. +16 (columns: B = x rows), chunks of
// slice z.  Writes part[z][t][e] = (sum x*w, sum |x*w|) and the slice's max |x|, max |w|.
__global__ __launch_bounds__(256) void screen_kernel(RouteArgs A)
{
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int r = lane & 15, lg = lane >> 4;
    const int T = A.T, E = A.E, H = A.H;
    const int t0 = blockIdx.x * 16, e0 = blockIdx.y * 64 + wave * 16, ks = blockIdx.z;
    const int nch = H / kScreenChunk, cps = (nch + A.KS - 1) / A.KS;
    const int c0 = min(nch, ks * cps), c1 = min(nch, c0 + cps);
    const __amdgpu_buffer_rsrc_t xr = screen_rsrc(A.x, (uint32_t)T * H * 2u);
    const __amdgpu_buffer_rsrc_t wr = screen_rsrc(A.wr, (uint32_t)E * H * 2u);
    const uint32_t xo = t0 + r < T ? (uint32_t)(t0 + r) * H * 2u : kScreenOOR;
    const uint32_t wo = e0 + r < E ? (uint32_t)(e0 + r) * H * 2u : kScreenOOR;
    double S[4] = {0.0, 0.0, 0.0, 0.0}, Aa[4] = {0.0, 0.0, 0.0, 0.0};
    u16x2 mx = {0, 0}, mw = {0, 0};
    u32x4v xa[2][8], wa[2][8];
    auto load = [&](int b, int c) {
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const uint32_t k2 = (uint32_t)(c * kScreenChunk + 32 * i + 8 * lg) * 2u;
            xa[b][i] = __builtin_amdgcn_raw_buffer_load_b128(xr, xo + k2, 0, 0);
            wa[b][i] = __builtin_amdgcn_raw_buffer_load_b128(wr, wo + k2, 0, 0);
        }
    };
    auto compute = [&](int b) {
        f32x4 acc = {0.f, 0.f, 0.f, 0.f}, acca = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int i = 0; i < 8; ++i) {
            const u32x4v m = {0x7FFF7FFFu, 0x7FFF7FFFu, 0x7FFF7FFFu, 0x7FFF7FFFu};
            const u32x4v xabs = xa[b][i] & m, wabs = wa[b][i] & m;
            acc = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wa[b][i]),
                                                          __builtin_bit_cast(bf16x8, xa[b][i]), acc, 0, 0, 0);
            acca = __builtin_amdgcn_mfma_f32_16x16x32_bf16(__builtin_bit_cast(bf16x8, wabs),
                                                           __builtin_bit_cast(bf16x8, xabs), acca, 0, 0, 0);
#pragma unroll
            for (int q = 0; q < 4; ++q) {  // |bf16| bit patterns order like their values
                mx = __builtin_elementwise_max(mx, __builtin_bit_cast(u16x2, xabs[q]));
                mw = __builtin_elementwise_max(mw, __builtin_bit_cast(u16x2, wabs[q]));
            }
        }
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            S[j] += (double)acc[j];
            Aa[j] += (double)acca[j];
        }
    };
    if (c0 < c1) {
        // chunk c sits in buffer (c - c0) % 2; loads of the next chunk are in flight
        // while one is multiplied (the last chunk is reloaded past the end)
        load(0, c0);
        int c = c0;
        for (; c + 2 <= c1; c += 2) {
            load(1, c + 1);
            compute(0);
            load(0, min(c + 2, c1 - 1));
            compute(1);
        }
        if (c < c1) compute(0);
    }
    // lane: experts e0 + 4lg + j (rows), token t0 + r (column)
    const int t = t0 + r;
    if (t < T) {
#pragma unroll
        for (int j = 0; j < 4; ++j) {
            const int e = e0 + 4 * lg + j;
            if (e < E) A.part[((size_t)ks * A.Tmax + t) * E + e] = make_double2(S[j], Aa[j]);
        }
    }
    // slice maxima: lane (r, lg) saw row r of x and of the router block; combine the
    // four lane groups
    uint32_t m1 = max((uint32_t)mx.x, (uint32_t)mx.y), m2 = max((uint32_t)mw.x, (uint32_t)mw.y);
    m1 = max(m1, (uint32_t)__shfl_xor((int)m1, 16));
    m1 = max(m1, (uint32_t)__shfl_xor((int)m1, 32));
    m2 = max(m2, (uint32_t)__shfl_xor((int)m2, 16));
    m2 = max(m2, (uint32_t)__shfl_xor((int)m2, 32));
    if (lg == 0) {
        if (t < T) A.xmax[(size_t)ks * A.Tmax + t] = __uint_as_float(m1 << 16);
        if (e0 + r < E) A.wmax[(size_t)ks * E + e0 + r] = __uint_as_float(m2 << 16);
    }
}

// fp32 rounded down / up from fp64.
__device__ inline float f32_down(double v)
{
    float f = (float)v;
    return (double)f > v ? nextafterf(f, -INFINITY) : f;
}
__device__ inline float f32_up(double v)
{
    float f = (float)v;
    return (double)f < v ? nextafterf(f, INFINITY) : f;
}

// k-th largest of v[0 .. E-1] (E <= 64 V) in the key order of the top-k (value desc,
// index asc), by one wave: k rounds of the wave argmax.
template <int V>
__device__ __attribute__((always_inline)) inline float kth_largest(const float *v, int E, int k, int lane)
{
    uint64_t key[V];
#pragma unroll
    for (int i = 0; i < V; ++i) {
        const int e = 64 * i + lane;
        key[i] = e < E ? ((uint64_t)ordered_bits(v[e]) << 32) | (uint32_t)(~(uint32_t)e) : 0;
    }
    uint64_t best = 0;
    for (int j = 0; j < k; ++j) {
        best = key[0];
#pragma unroll
        for (int i = 1; i < V; ++i) best = key[i] > best ? key[i] : best;
        best = wave_max64(best);
#pragma unroll
        for (int i = 0; i < V; ++i) key[i] = key[i] == best ? 0 : key[i];
    }
    return from_ordered((uint32_t)(best >> 32));
}

// One workgroup per token (grid T), 256 threads; dynamic LDS as route_kernel's grouping.
__global__ __launch_bounds__(256) void route_cand_kernel(RouteArgs A)
{
    extern __shared__ __attribute__((aligned(16))) uint32_t lds[];
    __shared__ float s_lo[kMaxE], s_hi[kMaxE];
    __shared__ uint32_t s_cand[kMaxE / 32];
    __shared__ int s_list[kMaxE];
    __shared__ int s_n, s_flag;
    __shared__ int s_scan[16];
    static_assert(sizeof(float) * 2 * kMaxE + sizeof(uint32_t) * (kMaxE / 32) + sizeof(int) * (kMaxE + 2 + 16) <=
                  kCandStaticLds);
    const int lane = threadIdx.x & (kWave - 1), wave = threadIdx.x >> 6;
    const int t = blockIdx.x, E = A.E, H = A.H, k = A.k;
    const uint16_t *xr = (const uint16_t *)A.x + (size_t)t * H;
    const uint16_t *wr = (const uint16_t *)A.wr;

    // 1. brackets of every expert's canonical logit
    // (the slices' loads are issued together: KS <= kMaxKS, unrolled and predicated)
    float xm[kMaxKS];
#pragma unroll
    for (int s2 = 0; s2 < kMaxKS; ++s2) xm[s2] = s2 < A.KS ? A.xmax[(size_t)s2 * A.Tmax + t] : 0.f;
    float mxt = 0.f;
#pragma unroll
    for (int s2 = 0; s2 < kMaxKS; ++s2) mxt = fmaxf(mxt, xm[s2]);
    const double u = 0x1p-23, g = kScreenChunk * u / (1.0 - kScreenChunk * u);
    for (int e = threadIdx.x; e < E; e += blockDim.x) {
        double2 d[kMaxKS];
        float wm[kMaxKS];
#pragma unroll
        for (int s2 = 0; s2 < kMaxKS; ++s2) {
            d[s2] = s2 < A.KS ? A.part[((size_t)s2 * A.Tmax + t) * E + e] : make_double2(0.0, 0.0);
            wm[s2] = s2 < A.KS ? A.wmax[(size_t)s2 * E + e] : 0.f;
        }
        double S = 0.0, Aa = 0.0;
        float mwe = 0.f;
#pragma unroll
        for (int s2 = 0; s2 < kMaxKS; ++s2) {
            S += d[s2].x;
            Aa += d[s2].y;
            mwe = fmaxf(mwe, wm[s2]);
        }
        const double flush = (double)H * 0x1p-126 * ((double)mxt + (double)mwe + 2.0);
        const double Ab = (Aa * (1.0 + 0x1p-40) + flush) / (1.0 - g);
        const double Sb = S + (A.bias ? (double)A.bias[e] : 0.0);
        const double dsum = (g + 0x1p-40) * Ab + flush;
        const double D = dsum + fabs(Sb) * 0x1p-52 + (fabs(Sb) + dsum) * 0x1p-23 + 0x1p-149;
        s_lo[e] = f32_down(Sb - D);
        s_hi[e] = f32_up(Sb + D);
    }
    for (int i = threadIdx.x; i < kMaxE / 32; i += blockDim.x) s_cand[i] = 0u;
    __syncthreads();

    // 2. wave 0: LB = k-th largest lower bound, the candidates hi >= LB in expert
    // order; waves 1-3: the token's activation split (MFMA path)
    if (wave == 0) {
        const int V = (E + 63) / 64;
        const float LB = V <= 1   ? kth_largest<1>(s_lo, E, k, lane)
                         : V <= 2 ? kth_largest<2>(s_lo, E, k, lane)
                         : V <= 4 ? kth_largest<4>(s_lo, E, k, lane)
                         : V <= 8 ? kth_largest<8>(s_lo, E, k, lane)
                                  : kth_largest<16>(s_lo, E, k, lane);
        int n = 0;
        for (int v = 0; v < V; ++v) {
            const int e = 64 * v + lane;
            const bool c = e < E && !(s_hi[e] < LB);  // a NaN bracket or LB keeps e: n >= k always
            const uint64_t bal = __ballot(c);
            if (c) {
                s_list[n + __popcll(bal & ((1ull << lane) - 1ull))] = e;
                atomicOr(&s_cand[e >> 5], 1u << (e & 31));
            }
            n += __popcll(bal);
        }
        if (lane == 0) {
            s_n = n;
            atomicAdd(A.fb_acc + kCandCounterOff, n);
        }
    } else if (A.xs_hi) {
        write_split<uint16_t>(A, xr, t, threadIdx.x - kWave, blockDim.x - kWave);
    } else if (A.x16) {
        write_x16(A, xr, t, wave - 1, 3, lane);
    }
    __syncthreads();

    // 3. exact canonical logits of the candidates: an even share per wave, up to kEPW
    // router rows in flight per call; they go to LDS over the lower bounds, which are
    // no longer needed
    float *lrow = s_lo;
    int nfb = 0;
    const int n = s_n, per = (n + 3) / 4, i0 = wave * per, i1 = min(n, i0 + per);
    for (int i = i0; i < i1; i += kEPW)
        nfb += wave_logits<uint16_t, uint16_t, kEPW, 4>(xr, wr, A.bias, H, 0, min(kEPW, i1 - i), lane, lrow, s_list + i);
    if (lane == 0 && nfb) atomicAdd(A.fb_acc, nfb);
    __syncthreads();

    // 4. top-k among the candidates, softmax of the selected logits
    if (wave == 0)
        token_topk<true>(lrow, E, k, A.ids + (size_t)t * k, A.wts + (size_t)t * k,
                   A.ids_user ? A.ids_user + (size_t)t * k : nullptr, A.wts_user ? A.wts_user + (size_t)t * k : nullptr,
                   lane, s_cand);
    wait_stores();
    __syncthreads();
    if (threadIdx.x == 0) s_flag = atomicAdd(A.cnt_all, 1) == A.T - 1;
    __syncthreads();
    if (!s_flag) return;
    group_pairs(A, lds, s_scan);
}

__global__ void zero_kernel(int32_t *p, int n)
{
    for (int i = blockIdx.x * blockDim.x + threadIdx.x; i < n; i += gridDim.x * blockDim.x) p[i] = 0;
}

}  // namespace

hipError_t launch_zero(int32_t *p, int n, hipStream_t st)
{
    zero_kernel<<<(n + 255) / 256 < 1024 ? (n + 255) / 256 : 1024, 256, 0, st>>>(p, n);
    return hipGetLastError();
}

hipError_t launch_route(const Layer &L, const RouteParams &P, hipStream_t st)
{
    // Experts per wave: one up to 6400 (token, expert) pairs, four above.  Timed on the
    // 235B- and 480B-shaped routers with one to four experts per wave at 2048-12288
    // pairs: one is best or within 1.3 us up to 6400 pairs (480B-shaped, 32 tokens:
    // 16.5 us against 17.3 / 17.9 / 18.9 with two / three / four), four from 7168 pairs on
    // or within 0.8 us (235B-shaped, 64 tokens: 15.6 against 18.5 with one).
    const int epw = P.T * L.E <= 6400 ? 1 : kEPW;
    const int bpt = (L.E + 4 * epw - 1) / (4 * epw);
    RouteArgs A;
    A.x = P.x;
    A.wr = P.router_w;
    A.bias = P.bias;
    A.logits = P.logits;
    A.ids = P.ids;
    A.ids_user = P.ids_user;
    A.wts = P.wts;
    A.wts_user = P.wts_user;
    A.meta = P.meta;
    A.slot_of = P.slot_of;
    A.tok_of = P.tok_of;
    A.cnt_tok = P.cnt_tok;
    A.cnt_all = P.cnt_all;
    A.fb_acc = P.fb_acc;
    A.xs_hi = P.xs_hi;
    A.xs_lo = P.xs_lo;
    A.xe_hi = P.xe_hi;
    A.xe_lo = P.xe_lo;
    A.x16 = P.x16;
    A.xk = P.xk;
    A.T = P.T;
    A.E = L.E;
    A.H = L.H;
    A.k = P.k;
    A.epw = epw;
    A.bpt = bpt;
    A.mstar = P.mstar;
    A.do_group = P.do_group;
    A.max_chunks = P.max_chunks;
    A.part = (double2 *)P.part;
    A.xmax = P.xmax;
    A.wmax = P.wmax;
    A.Tmax = P.Tmax;
    A.KS = 0;
    const int W = (P.T + 31) / 32;
    // grouping LDS: bitmasks [E][W] and offsets [E], plus the choices [T*k] while the
    // whole stays within 64 KiB
    const size_t base_words = (size_t)L.E * W + L.E, pairs = (size_t)P.T * P.k;
    A.id_cache = P.do_group && (base_words + pairs) * sizeof(uint32_t) <= 65536 ? 1 : 0;
    const size_t lds = P.do_group ? sizeof(uint32_t) * (base_words + (A.id_cache ? pairs : 0)) : 0;
    // screened routing: bf16 activations and router, H a multiple of 256, enough work
    if (P.do_group && P.screen && L.act_bf16 && L.router_bf16 && P.ks_max > 0 && L.E <= kMaxE) {
        const int tiles = (P.T + 15) / 16, groups = (L.E + 63) / 64;
        const int waves = tiles * groups * 4;
        int ks = (2048 + waves - 1) / waves;  // about two waves per SIMD
        ks = ks < 1 ? 1 : (ks > P.ks_max ? P.ks_max : ks);
        A.KS = ks;
        // route_cand_kernel's static arrays take about 12.3 KiB: keep the total within 64 KiB
        A.id_cache = (base_words + pairs) * sizeof(uint32_t) + kCandStaticLds <= 65536 ? 1 : 0;
        const size_t lds_c = sizeof(uint32_t) * (base_words + (A.id_cache ? pairs : 0));
        screen_kernel<<<dim3(tiles, groups, ks), 256, 0, st>>>(A);
        route_cand_kernel<<<dim3(P.T), 256, lds_c, st>>>(A);
        return hipGetLastError();
    }
    dim3 grid(P.T * bpt), block(256);
    if (L.act_bf16 && L.router_bf16)
        route_kernel<uint16_t, uint16_t><<<grid, block, lds, st>>>(A);
    else if (L.act_bf16)
        route_kernel<uint16_t, float><<<grid, block, lds, st>>>(A);
    else if (L.router_bf16)
        route_kernel<float, uint16_t><<<grid, block, lds, st>>>(A);
    else
        route_kernel<float, float><<<grid, block, lds, st>>>(A);
    return hipGetLastError();
}

}  // namespace moe
