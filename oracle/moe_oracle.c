/*
 * TEST INFRASTRUCTURE -- the fp64 CPU oracle of the MoE decode layer.
 *
 * A plain, slow, obviously correct reference.  Only the test suite, the smoke check
 * and the benchmark's CPU-baseline leg may load it; the product library never does,
 * and the two share no code.
 *
 * What it computes, per decode step of one MoE layer (the decode-lane step that the
 * paper's Background section describes as dominated by weight reads, and that its
 * appendix on why MoE benefits most ties to the fraction of parameters a token
 * activates):
 *
 *   O1 router logit   l[t,e] = RNE_fp32( exact( sum_h x[t,h] * Wr[e,h] + b[e] ) ), -0 -> +0
 *   O2 selection      rank(e) = #{f : l_f > l_e  or  (l_f == l_e and f < e)};
 *                     expert e is the rank(e)-th choice iff rank(e) < k
 *   O3 softmax        p[t,e] = exp(l_e - m) / sum_e' exp(l_e' - m), m = max_e l_e   (fp64)
 *   O4 renormalise    w[t,j] = p[t,id_j] / sum_{i<k} p[t,id_i]
 *   O5 dequantise     FP8 : W[n][c] = e4m3(q[n][c]) * s[n/128][c/128]
 *                     MXFP4: W[n][c] = e2m1(q[n][c]) * 2^(e8m0[n][c/32] - 127)
 *                     NVFP4: W[n][c] = e2m1(q[n][c]) * e4m3(sb[n][c/16]) * ts
 *   O6 expert FFN     g = Wgate x, u = Wup x, a_i = g_i / (1 + exp(-g_i)) * u_i, o = Wdown a
 *   O7 combine        y[t] = sum_{j=0..k-1} w[t,j] * o[t,j]   (j ascending)
 *
 * All arithmetic after O1 is fp64.  Products of bf16 or fp32 inputs are exact in
 * fp64, and O1 sums them exactly in a fixed-point long accumulator (Kulisch-style)
 * before one round-to-nearest-even to fp32, so the logit does not depend on any
 * summation order.
 *
 * Formats: OCP FP8 E4M3FN (bias 7, max 448, S.1111.111 = NaN, no infinities);
 * OCP MX v1.0 E2M1 (bias 1, values 0, 0.5, 1, 1.5, 2, 3, 4, 6) and E8M0
 * (2^(e-127), 0xFF = NaN); bf16 = the upper 16 bits of an fp32.  NVFP4, NVIDIA's
 * two-level 4-bit format: E2M1 elements, an E4M3 scale per 16 consecutive inputs
 * and an fp32 scale ts per matrix.
 *
 * Expert weight packing (per expert, contiguous): gate [I][H], up [I][H] (input
 * index contiguous), down [H][I]; FP8 one byte per weight, MXFP4 two per byte with
 * the even input index in the low nibble (NVFP4 packed as MXFP4).  Scales: FP8 fp32
 * gate [I/128][H/128] | up | down [H/128][I/128]; MXFP4 E8M0 bytes gate [I][H/32] | up |
 * down [H][I/32]; NVFP4 four fp32 {ts gate, ts up, ts down, unused}, then E4M3 bytes
 * gate [I][H/16] | up | down [H][I/16].
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

enum { DT_F32 = 0, DT_BF16 = 1 };
enum { WF_FP8 = 0, WF_MXFP4 = 1, WF_NVFP4 = 2 };

/* ------------------------------------------------------------------ formats */

double oracle_dec_e4m3(uint8_t c)
{
    int s = c >> 7, e = (c >> 3) & 15, m = c & 7;
    if (e == 15 && m == 7) return NAN;
    double v = (e == 0) ? ldexp((double)m, -9) : ldexp((double)(8 + m), e - 10); /* (1+m/8) 2^(e-7) */
    return s ? -v : v;
}

double oracle_dec_e2m1(uint8_t nib)
{
    int s = (nib >> 3) & 1, e = (nib >> 1) & 3, m = nib & 1;
    double v = (e == 0) ? 0.5 * m : ldexp((double)(2 + m), e - 2); /* (1+m/2) 2^(e-1) */
    return s ? -v : v;
}

double oracle_dec_e8m0(uint8_t c) { return c == 255 ? NAN : ldexp(1.0, (int)c - 127); }

double oracle_dec_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

static double load_act(const void *p, int64_t i, int dtype)
{
    return dtype == DT_BF16 ? oracle_dec_bf16(((const uint16_t *)p)[i]) : (double)((const float *)p)[i];
}

/* ------------------------------------------------------------------ O1: exact logit */

/* The value sum_i d[i] * 2^(ACC_LSB + 32 i), with 32-bit digits held in int64 so
 * that up to 2^31 additions cannot overflow before carries are propagated.  It
 * covers every product of two fp32 (hence bf16) numbers and their sums. */
#define ACC_LSB (-384)
#define ACC_DIGITS 24
typedef struct {
    int64_t d[ACC_DIGITS];
} longacc;

static void acc_add(longacc *a, double v)
{
    if (v == 0.0) return;
    int e;
    double m = frexp(v, &e);                /* v = m 2^e, 0.5 <= |m| < 1 */
    int64_t q = (int64_t)ldexp(m, 53);      /* exact: v = q 2^(e-53) */
    int off = (e - 53) - ACC_LSB;
    if (off < 0 || off / 32 + 3 > ACC_DIGITS) abort(); /* outside fp32-product range */
    uint64_t mag = q < 0 ? (uint64_t)(-q) : (uint64_t)q;
    unsigned __int128 sh = (unsigned __int128)mag << (off % 32);
    for (int i = 0; i < 3; i++) {
        int64_t dig = (int64_t)(uint32_t)(sh >> (32 * i));
        a->d[off / 32 + i] += q < 0 ? -dig : dig;
    }
}

/* Propagate carries so that every digit lies in [0, 2^32), except the top one,
 * which then carries the sign of the whole value. */
static void acc_normalise(longacc *a)
{
    for (int i = 0; i + 1 < ACC_DIGITS; i++) {
        int64_t c = a->d[i] >> 32; /* floor division by 2^32 */
        a->d[i] -= c * ((int64_t)1 << 32);
        a->d[i + 1] += c;
    }
}

static int acc_bit(const longacc *a, int pos) /* pos = absolute bit exponent */
{
    int off = pos - ACC_LSB;
    if (off < 0) return 0;
    return (int)((a->d[off / 32] >> (off % 32)) & 1);
}

static int acc_any_below(const longacc *a, int pos)
{
    for (int p = ACC_LSB; p < pos; p++)
        if (acc_bit(a, p)) return 1;
    return 0;
}

/* Round the exact value held in *a to fp32, to nearest, ties to even. */
static float acc_round_f32(longacc *a)
{
    acc_normalise(a);
    int neg = a->d[ACC_DIGITS - 1] < 0;
    if (neg) {
        for (int i = 0; i < ACC_DIGITS; i++) a->d[i] = -a->d[i];
        acc_normalise(a);
    }
    int top = ACC_LSB - 1; /* exponent of the leading set bit */
    for (int p = ACC_LSB + 32 * ACC_DIGITS - 1; p >= ACC_LSB; p--)
        if (acc_bit(a, p)) {
            top = p;
            break;
        }
    if (top < ACC_LSB) return 0.0f; /* the exact sum is zero */
    int lsb = top - 23;             /* 24 significant bits */
    if (lsb < -149) lsb = -149;     /* fixed subnormal grid below 2^-126 */
    uint64_t mant = 0;
    for (int p = top; p >= lsb; p--) mant = (mant << 1) | (uint64_t)acc_bit(a, p);
    int rnd = acc_bit(a, lsb - 1);
    int sticky = acc_any_below(a, lsb - 1);
    if (rnd && (sticky || (mant & 1))) mant++;
    float r = ldexpf((float)mant, lsb); /* mant <= 2^24: exact unless it overflows */
    return neg ? -r : r;
}

/* One canonical router logit.  x_row and w_row hold H values of the given dtype. */
float oracle_logit(const void *x_row, int x_dtype, const void *w_row, int w_dtype, int64_t H, const float *bias)
{
    longacc acc;
    memset(&acc, 0, sizeof acc);
    for (int64_t h = 0; h < H; h++) acc_add(&acc, load_act(x_row, h, x_dtype) * load_act(w_row, h, w_dtype));
    if (bias) acc_add(&acc, (double)*bias);
    float r = acc_round_f32(&acc);
    return r + 0.0f; /* -0 -> +0 */
}

/* ------------------------------------------------------------------ O2-O4: routing */

/* Routing of one token: logits l[E] (O1), ids[k] in rank order (O2), weights w[k]
 * (O3-O4) and, if p is not NULL, the full softmax p[E]. */
void oracle_route_token(const void *x_row, int x_dtype, const void *router_w, int w_dtype, const float *bias,
                        int64_t H, int E, int k, float *l, int32_t *ids, double *w, double *p)
{
    for (int e = 0; e < E; e++) {
        const void *wr = w_dtype == DT_BF16 ? (const void *)((const uint16_t *)router_w + (int64_t)e * H)
                                            : (const void *)((const float *)router_w + (int64_t)e * H);
        l[e] = oracle_logit(x_row, x_dtype, wr, w_dtype, H, bias ? bias + e : NULL);
    }
    for (int e = 0; e < E; e++) {
        int rank = 0;
        for (int f = 0; f < E; f++)
            if (l[f] > l[e] || (l[f] == l[e] && f < e)) rank++;
        if (rank < k) ids[rank] = e;
    }
    double m = l[0];
    for (int e = 1; e < E; e++)
        if (l[e] > m) m = l[e];
    double *pe = (double *)malloc(sizeof(double) * (size_t)E);
    double z = 0.0;
    for (int e = 0; e < E; e++) {
        pe[e] = exp((double)l[e] - m);
        z += pe[e];
    }
    for (int e = 0; e < E; e++) pe[e] /= z;
    double zk = 0.0;
    for (int j = 0; j < k; j++) zk += pe[ids[j]];
    for (int j = 0; j < k; j++) w[j] = pe[ids[j]] / zk;
    if (p) memcpy(p, pe, sizeof(double) * (size_t)E);
    free(pe);
}

/* ------------------------------------------------------------------ O5-O6: experts */

typedef struct {
    int64_t H, I;
    int E, wfmt;
    const uint8_t *expert_w; /* E blocks, packed as in the header comment */
    const void *scales;
} experts_t;

static int64_t expert_w_bytes(const experts_t *X) { return X->wfmt == WF_FP8 ? 3 * X->H * X->I : 3 * X->H * X->I / 2; }
static int64_t expert_s_bytes(const experts_t *X)
{
    if (X->wfmt == WF_FP8) return 4 * 3 * (X->H / 128) * (X->I / 128);
    if (X->wfmt == WF_MXFP4) return 3 * X->H * X->I / 32;
    return 16 + 3 * X->H * X->I / 16;
}

/* E2M1 code of input c of row n of a packed [N][K] 4-bit matrix q (the even input
 * index in the low nibble). */
static uint8_t nibble(const uint8_t *q, int64_t n, int64_t K, int64_t c)
{
    uint8_t byte = q[(n * K + c) / 2];
    return (c % 2 == 0) ? (byte & 15) : (byte >> 4);
}

/* Dequantised weight of matrix `mat` (0 gate, 1 up, 2 down) of expert e, row n, input c. */
static double weight(const experts_t *X, int e, int mat, int64_t n, int64_t c)
{
    int64_t H = X->H, I = X->I;
    int64_t K = mat == 2 ? I : H;          /* inputs per row */
    int64_t N = mat == 2 ? H : I;          /* rows */
    const uint8_t *w = X->expert_w + (int64_t)e * expert_w_bytes(X);
    const uint8_t *s = (const uint8_t *)X->scales + (int64_t)e * expert_s_bytes(X);
    if (X->wfmt == WF_FP8) {
        const uint8_t *q = w + (int64_t)mat * I * H;
        const float *sc = (const float *)s + (int64_t)mat * (I / 128) * (H / 128);
        return oracle_dec_e4m3(q[n * K + c]) * (double)sc[(n / 128) * (K / 128) + c / 128];
    } else if (X->wfmt == WF_MXFP4) {
        const uint8_t *q = w + (int64_t)mat * I * H / 2;
        const uint8_t *sc = s + (int64_t)mat * I * H / 32;
        (void)N;
        return oracle_dec_e2m1(nibble(q, n, K, c)) * oracle_dec_e8m0(sc[n * (K / 32) + c / 32]);
    } else {
        const uint8_t *q = w + (int64_t)mat * I * H / 2;
        float ts;
        memcpy(&ts, s + 4 * mat, 4);
        const uint8_t *sb = s + 16 + (int64_t)mat * I * H / 16;
        return oracle_dec_e2m1(nibble(q, n, K, c)) * oracle_dec_e4m3(sb[n * (K / 16) + c / 16]) * (double)ts;
    }
}

/* O6 for one token vector xv[H] through expert e -> o[H].  a is scratch [I]. */
static void expert_ffn(const experts_t *X, int e, const double *xv, double *o, double *a)
{
    for (int64_t i = 0; i < X->I; i++) {
        double g = 0.0, u = 0.0;
        for (int64_t h = 0; h < X->H; h++) g += weight(X, e, 0, i, h) * xv[h];
        for (int64_t h = 0; h < X->H; h++) u += weight(X, e, 1, i, h) * xv[h];
        a[i] = g / (1.0 + exp(-g)) * u;
    }
    for (int64_t n = 0; n < X->H; n++) {
        double acc = 0.0;
        for (int64_t i = 0; i < X->I; i++) acc += weight(X, e, 2, n, i) * a[i];
        o[n] = acc;
    }
}

/* ------------------------------------------------------------------ the layer */

typedef struct {
    const experts_t *X;
    const double *xv;   /* [n_pairs][H] token vectors */
    const int32_t *eid; /* [n_pairs] expert of each pair */
    double *o;          /* [n_pairs][H] */
    int64_t n_pairs;
    int64_t next;       /* shared work counter */
    pthread_mutex_t mu;
} work_t;

static void *worker(void *arg)
{
    work_t *W = (work_t *)arg;
    double *a = (double *)malloc(sizeof(double) * (size_t)W->X->I);
    for (;;) {
        pthread_mutex_lock(&W->mu);
        int64_t i = W->next++;
        pthread_mutex_unlock(&W->mu);
        if (i >= W->n_pairs) break;
        expert_ffn(W->X, W->eid[i], W->xv + i * W->X->H, W->o + i * W->X->H, a);
    }
    free(a);
    return NULL;
}

/*
 * The whole layer for the tokens listed in `tokens` (n_sel of them; NULL = all T in
 * order).  Outputs are per selected token, in the order given: logits [n_sel][E],
 * ids [n_sel][k], w [n_sel][k], y [n_sel][H].  `threads` workers share the (token,
 * choice) pairs; each pair is computed exactly as the single-threaded definition.
 * Returns 0, or -1 on an invalid argument.
 */
int oracle_forward(int64_t H, int E, int64_t I, int act_dtype, int router_dtype, int wfmt, const void *x,
                   int64_t T, const void *router_w, const float *bias, const void *expert_w, const void *scales,
                   int k, const int64_t *tokens, int64_t n_sel, int threads, float *logits, int32_t *ids, double *w,
                   double *y)
{
    if (k < 1 || k > E || H <= 0 || I <= 0 || T <= 0) return -1;
    if (wfmt == WF_FP8 && (H % 128 || I % 128)) return -1;
    if (wfmt == WF_MXFP4 && (H % 32 || I % 32)) return -1;
    if (wfmt == WF_NVFP4 && (H % 16 || I % 16)) return -1;
    if (wfmt < WF_FP8 || wfmt > WF_NVFP4) return -1;
    if (!tokens) n_sel = T;
    experts_t X = {H, I, E, wfmt, (const uint8_t *)expert_w, scales};
    int64_t esz = act_dtype == DT_BF16 ? 2 : 4;
    for (int64_t s = 0; s < n_sel; s++) {
        int64_t t = tokens ? tokens[s] : s;
        if (t < 0 || t >= T) return -1;
        oracle_route_token((const uint8_t *)x + t * H * esz, act_dtype, router_w, router_dtype, bias, H, E, k,
                           logits + s * E, ids + s * k, w + s * k, NULL);
    }
    int64_t n_pairs = n_sel * k;
    double *xv = (double *)malloc(sizeof(double) * (size_t)(n_pairs * H));
    double *o = (double *)malloc(sizeof(double) * (size_t)(n_pairs * H));
    int32_t *eid = (int32_t *)malloc(sizeof(int32_t) * (size_t)n_pairs);
    for (int64_t s = 0; s < n_sel; s++) {
        int64_t t = tokens ? tokens[s] : s;
        for (int j = 0; j < k; j++) {
            eid[s * k + j] = ids[s * k + j];
            for (int64_t h = 0; h < H; h++) xv[(s * k + j) * H + h] = load_act(x, t * H + h, act_dtype);
        }
    }
    work_t W;
    W.X = &X;
    W.xv = xv;
    W.eid = eid;
    W.o = o;
    W.n_pairs = n_pairs;
    W.next = 0;
    pthread_mutex_init(&W.mu, NULL);
    if (threads < 1) threads = 1;
    if (threads == 1) {
        worker(&W);
    } else {
        pthread_t *th = (pthread_t *)malloc(sizeof(pthread_t) * (size_t)threads);
        for (int i = 0; i < threads; i++) pthread_create(&th[i], NULL, worker, &W);
        for (int i = 0; i < threads; i++) pthread_join(th[i], NULL);
        free(th);
    }
    pthread_mutex_destroy(&W.mu);
    for (int64_t s = 0; s < n_sel; s++)
        for (int64_t n = 0; n < H; n++) {
            double acc = 0.0;
            for (int j = 0; j < k; j++) acc += w[s * k + j] * o[(s * k + j) * H + n];
            y[s * H + n] = acc;
        }
    free(xv);
    free(o);
    free(eid);
    return 0;
}

/* O6 alone, for pins that bypass routing: one token vector through one expert. */
int oracle_expert_ffn(int64_t H, int E, int64_t I, int wfmt, const void *expert_w, const void *scales, int e,
                      const double *xv, double *o)
{
    if (e < 0 || e >= E) return -1;
    experts_t X = {H, I, E, wfmt, (const uint8_t *)expert_w, scales};
    double *a = (double *)malloc(sizeof(double) * (size_t)I);
    expert_ffn(&X, e, xv, o, a);
    free(a);
    return 0;
}
