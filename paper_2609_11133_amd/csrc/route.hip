// Routing kernels of the MoE decode step: router logits, top-k softmax and the
// token-to-expert grouping.  One decode step of a MoE layer starts here (the decode
// lane of the paper's Background section; the MoE models of its Experimental Setup).
#include <hip/hip_runtime.h>
#include <math.h>

#include "moe_internal.h"

namespace moe {
namespace {

constexpr int kWave = 64;

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

// One wave per (token, group of `epw` experts).
template <typename XT, typename WT>
__global__ __launch_bounds__(256) void router_logits_kernel(const XT *__restrict__ x, const WT *__restrict__ wr,
                                                            const float *__restrict__ bias, float *__restrict__ logits,
                                                            int32_t *__restrict__ fb_flags, int T, int E, int H,
                                                            int epw)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int wave = blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    const int groups = (E + epw - 1) / epw;
    const int t = wave / groups;
    if (t >= T) return;
    const int e0 = (wave % groups) * epw;
    const int e1 = min(E, e0 + epw);
    const XT *xr = x + (size_t)t * H;
    const int per_lane = ((H + 511) / 512) * 8;
    const double gamma = (double)(per_lane + 6 + 1 + 2) * 0x1p-52;  // >= 2 gamma_D

    for (int e = e0; e < e1; ++e) {
        const WT *wrow = wr + (size_t)e * H;
        double s = 0.0, a = 0.0;
        for (int h = lane * 8; h < H; h += 512) {
            double xv[8], wv[8];
            load8<XT>(xr + h, xv);
            load8<WT>(wrow + h, wv);
#pragma unroll
            for (int i = 0; i < 8; ++i) {
                s = fma(xv[i], wv[i], s);
                a = fma(fabs(xv[i]), fabs(wv[i]), a);
            }
        }
#pragma unroll
        for (int o = kWave / 2; o >= 1; o >>= 1) {
            s += __shfl_xor(s, o);
            a += __shfl_xor(a, o);
        }
        const double b = bias ? (double)bias[e] : 0.0;
        const double v = s + b;
        float r;
        int fallback = 0;
        if (!certain_f32(v, gamma * (a + fabs(b)), r)) {
            // Exact path: error-free accumulation of the same (exact) products.
            double hi = 0.0, lo = 0.0;
            for (int h = lane * 8; h < H; h += 512) {
                double xv[8], wv[8];
                load8<XT>(xr + h, xv);
                load8<WT>(wrow + h, wv);
#pragma unroll
                for (int i = 0; i < 8; ++i) {
                    double p = xv[i] * wv[i], ss, ee;
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
            r = round_dd_to_f32(hi, lo);
            fallback = 1;
        }
        if (lane == 0) {
            logits[(size_t)t * E + e] = r + 0.0f;  // -0 -> +0
            if (fb_flags) fb_flags[(size_t)t * E + e] = fallback;
        }
    }
}

// ------------------------------------------------------------------ top-k softmax
//
// One wave per token.  Each lane holds the keys of experts lane, lane+64, ...; a key
// is (order-preserving integer image of the fp32 logit) << 32 | (~expert), so the
// largest key is the largest logit, ties going to the lower expert index.  k rounds
// of a wave-wide arg-max (xor butterfly) pick the experts in rank order.  Weights are
// the softmax of the selected logits (equal to the full softmax renormalised over
// the selection), computed in fp32 relative to the largest one.

__device__ inline uint32_t ordered_bits(float f)
{
    uint32_t u = __float_as_uint(f);
    return (u & 0x80000000u) ? ~u : (u | 0x80000000u);
}

__device__ inline float from_ordered(uint32_t o) { return __uint_as_float((o & 0x80000000u) ? (o & 0x7FFFFFFFu) : ~o); }

constexpr int kMaxKeysPerLane = 16;  // E <= 1024

__global__ __launch_bounds__(256) void topk_softmax_kernel(const float *__restrict__ logits, int T, int E, int k,
                                                           int32_t *__restrict__ ids, float *__restrict__ wts,
                                                           int32_t *__restrict__ ids_user, float *__restrict__ wts_user)
{
    const int lane = threadIdx.x & (kWave - 1);
    const int t = blockIdx.x * (blockDim.x / kWave) + (threadIdx.x / kWave);
    if (t >= T) return;
    const float *l = logits + (size_t)t * E;
    uint64_t key[kMaxKeysPerLane];
    const int nk = (E + kWave - 1) / kWave;
#pragma unroll
    for (int c = 0; c < kMaxKeysPerLane; ++c) {
        int e = lane + c * kWave;
        key[c] = (c < nk && e < E) ? (((uint64_t)ordered_bits(l[e]) << 32) | (uint32_t)(~(uint32_t)e)) : 0ull;
    }
    float top_l = 0.f, denom = 0.f;
    float my_l = 0.f;
    int my_e = 0;
    for (int j = 0; j < k; ++j) {
        uint64_t best = 0;
#pragma unroll
        for (int c = 0; c < kMaxKeysPerLane; ++c) best = key[c] > best ? key[c] : best;
#pragma unroll
        for (int o = kWave / 2; o >= 1; o >>= 1) {
            uint64_t other = __shfl_xor(best, o);
            best = other > best ? other : best;
        }
        const int e = (int)(~(uint32_t)best);
        const float lv = from_ordered((uint32_t)(best >> 32));
        if ((e & (kWave - 1)) == lane) {
#pragma unroll
            for (int c = 0; c < kMaxKeysPerLane; ++c)
                if (c == e / kWave) key[c] = 0ull;
        }
        if (j == 0) top_l = lv;
        const float p = expf(lv - top_l);
        denom += p;  // same order (j ascending) in every lane
        if (lane == j) {
            my_e = e;
            my_l = p;
        }
    }
    if (lane < k) {
        const float w = my_l / denom;
        ids[(size_t)t * k + lane] = my_e;
        wts[(size_t)t * k + lane] = w;
        if (ids_user) ids_user[(size_t)t * k + lane] = my_e;
        if (wts_user) wts_user[(size_t)t * k + lane] = w;
    }
}

// ------------------------------------------------------------------ grouping
//
// One workgroup.  LDS holds one bit per (expert, token): expert e's tokens in token
// order.  counts[e] = popcount of its row, offsets = exclusive prefix sum, and the
// slot of pair (t, j) choosing e is offsets[e] + (number of earlier tokens that chose
// e).  Every result is independent of thread timing.  Experts with at least `mstar`
// tokens go to the MFMA list, the others to the GEMV list, each in expert order.

__global__ __launch_bounds__(1024) void group_kernel(const int32_t *__restrict__ ids, int T, int k, int E, int mstar,
                                                     int32_t *__restrict__ meta, int32_t *__restrict__ slot_of,
                                                     int32_t *__restrict__ tok_of,
                                                     const int32_t *__restrict__ fb_flags)
{
    extern __shared__ uint32_t lds[];
    const int W = (T + 31) / 32;
    uint32_t *mask = lds;                  // [E][W]
    int32_t *offs = (int32_t *)(lds + E * W);  // [E+1]
    __shared__ int32_t fb_total;
    const MetaIdx mi{E};
    const int tid = threadIdx.x, nth = blockDim.x;

    for (int i = tid; i < E * W; i += nth) mask[i] = 0u;
    if (tid == 0) fb_total = 0;
    __syncthreads();
    for (int p = tid; p < T * k; p += nth) {
        const int t = p / k;
        atomicOr(&mask[ids[p] * W + t / 32], 1u << (t % 32));
    }
    int fb = 0;
    if (fb_flags)
        for (int i = tid; i < T * E; i += nth) fb += fb_flags[i];
    __syncthreads();
    for (int e = tid; e < E; e += nth) {
        int c = 0;
        for (int w = 0; w < W; ++w) c += __popc(mask[e * W + w]);
        meta[mi.counts() + e] = c;
        offs[e] = c;  // counts for the scan below
    }
    if (fb) atomicAdd(&fb_total, fb);
    __syncthreads();
    if (tid == 0) {
        int run = 0, na = 0, ng = 0, nm = 0;
        for (int e = 0; e < E; ++e) {
            const int c = offs[e];
            offs[e] = run;
            meta[mi.offsets() + e] = run;
            run += c;
            if (c > 0) {
                ++na;
                if (mstar > 0 && c >= mstar)
                    meta[mi.act_mfma() + nm++] = e;
                else
                    meta[mi.act_gemv() + ng++] = e;
            }
        }
        offs[E] = run;
        meta[mi.offsets() + E] = run;
        meta[mi.n_active()] = na;
        meta[mi.n_gemv()] = ng;
        meta[mi.n_mfma()] = nm;
        meta[mi.n_fallback()] = fb_total;
    }
    __syncthreads();
    for (int p = tid; p < T * k; p += nth) {
        const int t = p / k, e = ids[p];
        int rank = __popc(mask[e * W + t / 32] & ((1u << (t % 32)) - 1u));
        for (int w = 0; w < t / 32; ++w) rank += __popc(mask[e * W + w]);
        const int slot = offs[e] + rank;
        slot_of[p] = slot;
        tok_of[slot] = t;
    }
}

}  // namespace

hipError_t launch_router(const Layer &L, const void *x, int T, const void *router_w, const float *bias,
                         float *logits, int32_t *fb_flags, hipStream_t st)
{
    // Experts per wave: enough waves to cover the GPU, few experts per wave at small T.
    const int target_waves = 4096;
    int epw = (T * L.E + target_waves - 1) / target_waves;
    epw = epw < 1 ? 1 : (epw > 16 ? 16 : epw);
    const int groups = (L.E + epw - 1) / epw;
    const int waves = T * groups;
    dim3 grid((waves + 3) / 4), block(256);
    if (L.act_bf16 && L.router_bf16)
        router_logits_kernel<uint16_t, uint16_t><<<grid, block, 0, st>>>(
            (const uint16_t *)x, (const uint16_t *)router_w, bias, logits, fb_flags, T, L.E, L.H, epw);
    else if (L.act_bf16)
        router_logits_kernel<uint16_t, float><<<grid, block, 0, st>>>(
            (const uint16_t *)x, (const float *)router_w, bias, logits, fb_flags, T, L.E, L.H, epw);
    else if (L.router_bf16)
        router_logits_kernel<float, uint16_t><<<grid, block, 0, st>>>(
            (const float *)x, (const uint16_t *)router_w, bias, logits, fb_flags, T, L.E, L.H, epw);
    else
        router_logits_kernel<float, float><<<grid, block, 0, st>>>((const float *)x, (const float *)router_w, bias,
                                                                   logits, fb_flags, T, L.E, L.H, epw);
    return hipGetLastError();
}

hipError_t launch_topk(const Layer &L, const float *logits, int T, int k, int32_t *ids, float *wts,
                       int32_t *ids_user, float *wts_user, hipStream_t st)
{
    dim3 grid((T + 3) / 4), block(256);
    topk_softmax_kernel<<<grid, block, 0, st>>>(logits, T, L.E, k, ids, wts, ids_user, wts_user);
    return hipGetLastError();
}

hipError_t launch_group(const Layer &L, const int32_t *ids, int T, int k, int mstar, int32_t *meta,
                        int32_t *slot_of, int32_t *tok_of, const int32_t *fb_flags, hipStream_t st)
{
    const int W = (T + 31) / 32;
    const size_t lds = sizeof(uint32_t) * ((size_t)L.E * W + L.E + 1);
    group_kernel<<<1, 1024, lds, st>>>(ids, T, k, L.E, mstar, meta, slot_of, tok_of, fb_flags);
    return hipGetLastError();
}

}  // namespace moe
