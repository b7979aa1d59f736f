/*
 * Seeded synthetic inputs for the MoE decode layer.
 *
 * This module produces the tensors a decode step consumes (activations, router
 * weights, router bias, quantised expert weights and their scales).  It holds none
 * of the layer's own arithmetic: no routing, no dequantisation, no expert FFN.
 * Both the fp64 reference and the HIP library are fed from here.
 *
 * Random numbers
 *   A counter-based generator: every value is a pure function of
 *   (seed, tag, layer, sub, index), so any slice of any tensor can be produced
 *   independently and in parallel.  The mixing function is SplitMix64
 *   (Steele, Lea and Flood, "Fast splittable pseudorandom number generators",
 *   OOPSLA 2014; constants as in Vigna's public-domain splitmix64.c).
 *   Gaussian draws use the Irwin-Hall construction: the sum of twelve uniform
 *   16-bit integers, centred and scaled, which has mean 0 and variance 1 and is
 *   computed exactly in integer arithmetic plus one exact power-of-two scaling,
 *   so the bits are identical on every IEEE-754 platform.
 *
 * Quantisers (weight preparation, not part of the layer)
 *   FP8 E4M3FN (OCP 8-bit floating point spec): one fp32 scale per 128x128
 *     (output x input) block, s = amax/448 (1 if the block is all zero), codes
 *     are round-to-nearest-even of w/s, saturated to +-448.
 *   MXFP4 (OCP Microscaling Formats v1.0): E2M1 elements, one E8M0 scale per 32
 *     consecutive inputs of a row, shared exponent floor(log2(amax)) - 2, codes are
 *     round-to-nearest-even of w/X, saturated to +-6.  Two codes per byte, the even
 *     input index in the low nibble.
 *   NVFP4 (NVIDIA's two-level 4-bit format): E2M1 elements, one E4M3 scale per 16
 *     consecutive inputs of a row and one fp32 scale per matrix.  The matrix scale is
 *     ts = amax(matrix) / (6 * 448) rounded to fp32 (1 if the matrix is zero), so the
 *     block scales s = RNE_E4M3(amax(block) / (6 * ts)) use the whole E4M3 range;
 *     codes are round-to-nearest-even of w / (s * ts), saturated to +-6, and 0 where
 *     s rounds to 0.  Packing as MXFP4.
 *
 * Expert weight packing (per expert e, one contiguous block):
 *   FP8  : gate [I][H] bytes | up [I][H] | down [H][I]            (3*H*I bytes)
 *          scales fp32: gate [I/128][H/128] | up [I/128][H/128] | down [H/128][I/128]
 *   MXFP4: gate [I][H/2] | up [I][H/2] | down [H][I/2]             (3*H*I/2 bytes)
 *          scales E8M0: gate [I][H/32] | up [I][H/32] | down [H][I/32]
 *   NVFP4: weights as MXFP4
 *          scales: fp32 matrix scales {gate, up, down, 0} (16 bytes), then E4M3 block
 *          scales gate [I][H/16] | up [I][H/16] | down [H][I/16]
 */
#include <math.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

#define GOLDEN 0x9E3779B97F4A7C15ULL

enum { TAG_X = 1, TAG_ROUTER = 2, TAG_BIAS = 3, TAG_GATE = 4, TAG_UP = 5, TAG_DOWN = 6, TAG_PERM = 7 };

static inline uint64_t sm64_mix(uint64_t z)
{
    z = (z ^ (z >> 30)) * 0xBF58476D1CE4E5B9ULL;
    z = (z ^ (z >> 27)) * 0x94D049BB133111EBULL;
    return z ^ (z >> 31);
}

uint64_t synth_stream_key(uint64_t seed, uint32_t tag, uint32_t layer, uint32_t sub)
{
    uint64_t k = sm64_mix(seed + GOLDEN);
    return sm64_mix(k ^ (((uint64_t)tag << 56) | ((uint64_t)(layer & 0xFFFFFF) << 32) | sub));
}

static inline uint64_t draw(uint64_t key, uint64_t i) { return sm64_mix(key + (i + 1) * GOLDEN); }

/* Irwin-Hall(12): the sum of twelve uniforms (u + 1/2) / 2^16, u a 16-bit integer,
 * minus 6.  Three 64-bit draws supply the twelve 16-bit integers.  Exact in fp64. */
static inline double normal_at(uint64_t key, uint64_t i)
{
    uint64_t s = 0;
    for (int j = 0; j < 3; j++) {
        uint64_t d = draw(key, 3 * i + (uint64_t)j);
        s += (d & 0xFFFF) + ((d >> 16) & 0xFFFF) + ((d >> 32) & 0xFFFF) + (d >> 48);
    }
    /* (2*s + 12 - 12*2^16) / 2^17 */
    int64_t num = (int64_t)(2 * s + 12) - (int64_t)(12 << 16);
    return (double)num * 0x1p-17;
}

void synth_normal_f64(uint64_t key, uint64_t start, uint64_t n, double sigma, double *out)
{
    for (uint64_t i = 0; i < n; i++) out[i] = sigma * normal_at(key, start + i);
}

/* Exponent of a finite double a > 0 (a in [2^e, 2^(e+1))); a must be normal. */
static inline int exp_of(double a)
{
    uint64_t u;
    memcpy(&u, &a, 8);
    return (int)((u >> 52) & 0x7FF) - 1023;
}

static inline double pow2(int k) /* 2^k for -1022 <= k <= 1023 */
{
    uint64_t u = (uint64_t)(k + 1023) << 52;
    double d;
    memcpy(&d, &u, 8);
    return d;
}

/* Round a >= 0 to the nearest value with p significant bits whose smallest normal
 * exponent is emin (below it the grid is fixed at 2^(emin-p+1)); ties to even.
 * a is a normal double or zero. */
static double round_fmt(double a, int p, int emin)
{
    if (a == 0.0) return 0.0;
    int e = exp_of(a);
    if (e < emin) e = emin;
    int k = e - p + 1;
    return __builtin_rint(a * pow2(-k)) * pow2(k); /* scaling is exact; rint rounds half to even */
}

uint16_t synth_bf16_from_f64(double v)
{
    double a = round_fmt(fabs(v), 8, -126);
    float f = (float)a; /* exact: a has at most 8 significant bits */
    uint32_t u;
    memcpy(&u, &f, 4);
    uint16_t b = (uint16_t)(u >> 16);
    return signbit(v) ? (uint16_t)(b | 0x8000) : b;
}

uint8_t synth_e4m3_from_f64(double v)
{
    double a = round_fmt(fabs(v), 4, -6);
    if (a > 448.0) a = 448.0;
    uint8_t code;
    if (a == 0.0) {
        code = 0;
    } else {
        int e = exp_of(a);
        if (e < -6) {
            code = (uint8_t)(a * 512.0); /* subnormal: a = m * 2^-9 */
        } else {
            int m = (int)(a * pow2(-e) * 8.0) - 8;
            code = (uint8_t)(((e + 7) << 3) | m);
        }
    }
    return signbit(v) ? (uint8_t)(code | 0x80) : code;
}

uint8_t synth_e2m1_from_f64(double v)
{
    double a = round_fmt(fabs(v), 2, 0);
    if (a > 6.0) a = 6.0;
    static const double grid[8] = {0.0, 0.5, 1.0, 1.5, 2.0, 3.0, 4.0, 6.0};
    uint8_t code = 0;
    for (int c = 0; c < 8; c++)
        if (grid[c] == a) code = (uint8_t)c;
    return signbit(v) ? (uint8_t)(code | 0x8) : code;
}

/* ---------------------------------------------------------------- activations */

/* n values sigma * N(0,1) of one stream (draws start..start+n-1), rounded to bf16. */
void synth_normal_bf16(uint64_t key, uint64_t start, int64_t n, double sigma, uint16_t *out)
{
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < n; i++) out[i] = synth_bf16_from_f64(sigma * normal_at(key, start + (uint64_t)i));
}

void synth_x_bf16(uint64_t seed, uint32_t batch, int64_t T, int64_t H, uint16_t *out)
{
    uint64_t key = synth_stream_key(seed, TAG_X, batch, 0);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < T * H; i++) out[i] = synth_bf16_from_f64(normal_at(key, (uint64_t)i));
}

void synth_x_f32(uint64_t seed, uint32_t batch, int64_t T, int64_t H, float *out)
{
    uint64_t key = synth_stream_key(seed, TAG_X, batch, 0);
    for (int64_t i = 0; i < T * H; i++) out[i] = (float)normal_at(key, (uint64_t)i);
}

/* ---------------------------------------------------------------- router */

void synth_router_bf16(uint64_t seed, uint32_t layer, int64_t E, int64_t H, uint16_t *out)
{
    uint64_t key = synth_stream_key(seed, TAG_ROUTER, layer, 0);
    double sigma = 1.0 / sqrt((double)H);
#pragma omp parallel for schedule(static)
    for (int64_t i = 0; i < E * H; i++) out[i] = synth_bf16_from_f64(sigma * normal_at(key, (uint64_t)i));
}

void synth_router_f32(uint64_t seed, uint32_t layer, int64_t E, int64_t H, float *out)
{
    uint64_t key = synth_stream_key(seed, TAG_ROUTER, layer, 0);
    double sigma = 1.0 / sqrt((double)H);
    for (int64_t i = 0; i < E * H; i++) out[i] = (float)(sigma * normal_at(key, (uint64_t)i));
}

/* b_e ~ N(0, sd) rounded to fp32. */
void synth_bias_normal(uint64_t seed, uint32_t layer, int64_t E, double sd, float *out)
{
    uint64_t key = synth_stream_key(seed, TAG_BIAS, layer, 0);
    for (int64_t e = 0; e < E; e++) out[e] = (float)(sd * normal_at(key, (uint64_t)e));
}

/* Zipf(s) popularity through the router: b_e = -s * ln(rank_e), rank_e in 1..E a
 * seeded permutation (Fisher-Yates on the counter stream).  Under Gumbel noise this
 * gives exactly Zipf(s) top-1 marginals; under Gaussian logits it is a skew of the
 * same shape. */
void synth_bias_zipf(uint64_t seed, uint32_t layer, int64_t E, double s, float *out)
{
    uint64_t key = synth_stream_key(seed, TAG_PERM, layer, 0);
    int64_t *perm = (int64_t *)malloc(sizeof(int64_t) * (size_t)E);
    for (int64_t i = 0; i < E; i++) perm[i] = i;
    for (int64_t i = E - 1; i > 0; i--) {
        int64_t j = (int64_t)(draw(key, (uint64_t)i) % (uint64_t)(i + 1));
        int64_t t = perm[i];
        perm[i] = perm[j];
        perm[j] = t;
    }
    for (int64_t r = 0; r < E; r++) out[perm[r]] = (float)(-s * log((double)(r + 1))) + 0.0f; /* -0 -> +0 */
    free(perm);
}

/* ---------------------------------------------------------------- expert weights */

static void quant_fp8_matrix(uint64_t key, double sigma, int64_t N, int64_t K, uint8_t *q, float *sc,
                             double *scratch)
{
    int64_t nb = N / 128, kb = K / 128;
    for (int64_t rb = 0; rb < nb; rb++)
        for (int64_t cb = 0; cb < kb; cb++) {
            double amax = 0.0;
            for (int64_t r = 0; r < 128; r++)
                for (int64_t c = 0; c < 128; c++) {
                    int64_t n = rb * 128 + r, k = cb * 128 + c;
                    double v = sigma * normal_at(key, (uint64_t)(n * K + k));
                    scratch[r * 128 + c] = v;
                    if (fabs(v) > amax) amax = fabs(v);
                }
            float s = amax > 0.0 ? (float)(amax / 448.0) : 1.0f;
            sc[rb * kb + cb] = s;
            for (int64_t r = 0; r < 128; r++)
                for (int64_t c = 0; c < 128; c++) {
                    int64_t n = rb * 128 + r, k = cb * 128 + c;
                    q[n * K + k] = synth_e4m3_from_f64(scratch[r * 128 + c] / (double)s);
                }
        }
}

static void quant_mxfp4_matrix(uint64_t key, double sigma, int64_t N, int64_t K, uint8_t *q, uint8_t *sc)
{
    double v[32];
    for (int64_t n = 0; n < N; n++)
        for (int64_t g = 0; g < K / 32; g++) {
            double amax = 0.0;
            for (int c = 0; c < 32; c++) {
                v[c] = sigma * normal_at(key, (uint64_t)(n * K + g * 32 + c));
                if (fabs(v[c]) > amax) amax = fabs(v[c]);
            }
            int code = 127;
            if (amax > 0.0) {
                code = exp_of(amax) - 2 + 127; /* floor(log2 amax) - emax(E2M1) */
                if (code < 0) code = 0;
                if (code > 254) code = 254;
            }
            sc[n * (K / 32) + g] = (uint8_t)code;
            double X = pow2(code - 127);
            for (int c = 0; c < 32; c += 2) {
                uint8_t lo = synth_e2m1_from_f64(v[c] / X);
                uint8_t hi = synth_e2m1_from_f64(v[c + 1] / X);
                q[(n * K + g * 32 + c) / 2] = (uint8_t)(lo | (hi << 4));
            }
        }
}

/* NVFP4 matrix [N][K]: codes q (packed as MXFP4), E4M3 block scales sc [N][K/16], and
 * the fp32 matrix scale *ts.  Two passes over the counter stream: the matrix maximum
 * first, then the blocks. */
static void quant_nvfp4_matrix(uint64_t key, double sigma, int64_t N, int64_t K, uint8_t *q, uint8_t *sc, float *ts)
{
    double amax_m = 0.0;
    for (int64_t i = 0; i < N * K; i++) {
        double a = fabs(sigma * normal_at(key, (uint64_t)i));
        if (a > amax_m) amax_m = a;
    }
    float t = amax_m > 0.0 ? (float)(amax_m / (6.0 * 448.0)) : 1.0f;
    *ts = t;
    double v[16];
    for (int64_t n = 0; n < N; n++)
        for (int64_t b = 0; b < K / 16; b++) {
            double amax = 0.0;
            for (int c = 0; c < 16; c++) {
                v[c] = sigma * normal_at(key, (uint64_t)(n * K + b * 16 + c));
                if (fabs(v[c]) > amax) amax = fabs(v[c]);
            }
            uint8_t s = synth_e4m3_from_f64(amax / (6.0 * (double)t));
            sc[n * (K / 16) + b] = s;
            /* decode the (positive) scale code: (1 + m/8) 2^(e-7), subnormal m 2^-9 */
            int e = (s >> 3) & 15, m = s & 7;
            double sv = e == 0 ? ldexp((double)m, -9) : ldexp((double)(8 + m), e - 10);
            double X = sv * (double)t;
            for (int c = 0; c < 16; c += 2) {
                uint8_t lo = X > 0.0 ? synth_e2m1_from_f64(v[c] / X) : 0;
                uint8_t hi = X > 0.0 ? synth_e2m1_from_f64(v[c + 1] / X) : 0;
                q[(n * K + b * 16 + c) / 2] = (uint8_t)(lo | (hi << 4));
            }
        }
}

int64_t synth_expert_bytes(int wfmt, int64_t H, int64_t I) { return wfmt == 0 ? 3 * H * I : 3 * H * I / 2; }

int64_t synth_expert_scale_bytes(int wfmt, int64_t H, int64_t I)
{
    if (wfmt == 0) return 4 * 3 * (H / 128) * (I / 128);
    if (wfmt == 1) return 3 * H * I / 32;
    return 16 + 3 * H * I / 16;
}

/* One expert of one layer, FP8-E4M3 with 128x128 fp32 block scales. */
void synth_expert_fp8(uint64_t seed, uint32_t layer, int64_t e, int64_t H, int64_t I, uint8_t *w, float *s)
{
    double *scratch = (double *)malloc(sizeof(double) * 128 * 128);
    double sg = 1.0 / sqrt((double)H), sd = 1.0 / sqrt((double)I);
    int64_t nsg = (I / 128) * (H / 128);
    quant_fp8_matrix(synth_stream_key(seed, TAG_GATE, layer, (uint32_t)e), sg, I, H, w, s, scratch);
    quant_fp8_matrix(synth_stream_key(seed, TAG_UP, layer, (uint32_t)e), sg, I, H, w + I * H, s + nsg, scratch);
    quant_fp8_matrix(synth_stream_key(seed, TAG_DOWN, layer, (uint32_t)e), sd, H, I, w + 2 * I * H, s + 2 * nsg,
                     scratch);
    free(scratch);
}

/* One expert of one layer, MXFP4 (E2M1 + E8M0 per 32). */
void synth_expert_mxfp4(uint64_t seed, uint32_t layer, int64_t e, int64_t H, int64_t I, uint8_t *w, uint8_t *s)
{
    double sg = 1.0 / sqrt((double)H), sd = 1.0 / sqrt((double)I);
    quant_mxfp4_matrix(synth_stream_key(seed, TAG_GATE, layer, (uint32_t)e), sg, I, H, w, s);
    quant_mxfp4_matrix(synth_stream_key(seed, TAG_UP, layer, (uint32_t)e), sg, I, H, w + I * H / 2, s + I * H / 32);
    quant_mxfp4_matrix(synth_stream_key(seed, TAG_DOWN, layer, (uint32_t)e), sd, H, I, w + I * H, s + 2 * I * H / 32);
}

/* One expert of one layer, NVFP4 (E2M1 + E4M3 per 16 + fp32 per matrix). */
void synth_expert_nvfp4(uint64_t seed, uint32_t layer, int64_t e, int64_t H, int64_t I, uint8_t *w, uint8_t *s)
{
    double sg = 1.0 / sqrt((double)H), sd = 1.0 / sqrt((double)I);
    float ts[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    uint8_t *blk = s + 16;
    quant_nvfp4_matrix(synth_stream_key(seed, TAG_GATE, layer, (uint32_t)e), sg, I, H, w, blk, &ts[0]);
    quant_nvfp4_matrix(synth_stream_key(seed, TAG_UP, layer, (uint32_t)e), sg, I, H, w + I * H / 2, blk + I * H / 16,
                       &ts[1]);
    quant_nvfp4_matrix(synth_stream_key(seed, TAG_DOWN, layer, (uint32_t)e), sd, H, I, w + I * H,
                       blk + 2 * I * H / 16, &ts[2]);
    memcpy(s, ts, sizeof ts);
}

/* Experts [e0, e1) of a layer; the tensors for expert e are written at offset
 * (e - e0) * per-expert size.  Parallel over experts. */
void synth_experts(uint64_t seed, uint32_t layer, int wfmt, int64_t e0, int64_t e1, int64_t H, int64_t I,
                   uint8_t *w, void *s)
{
    int64_t wb = synth_expert_bytes(wfmt, H, I), sb = synth_expert_scale_bytes(wfmt, H, I);
#pragma omp parallel for schedule(dynamic, 1)
    for (int64_t e = e0; e < e1; e++) {
        uint8_t *we = w + (e - e0) * wb;
        uint8_t *se = (uint8_t *)s + (e - e0) * sb;
        if (wfmt == 0)
            synth_expert_fp8(seed, layer, e, H, I, we, (float *)se);
        else if (wfmt == 1)
            synth_expert_mxfp4(seed, layer, e, H, I, we, se);
        else
            synth_expert_nvfp4(seed, layer, e, H, I, we, se);
    }
}
