/* TEST INFRASTRUCTURE -- fp64 CPU oracle of one decode step of grouped-query attention
 * over a paged KV cache.  Only tests/, __graft_entry__.smoke() and bench.py's
 * CPU-baseline leg load it; it shares no code with the HIP library.
 *
 * What it computes.  The paper names the KV-cache reads as the second byte stream that
 * bounds a decode step (Background and Motivation, PD-disaggregated serving) and gives
 * no formula for attention; the definition is the standard scaled dot-product attention
 * (Vaswani et al., 2017) with grouped key/value heads (Ainslie et al., 2023, GQA): for
 * sequence b and query head h, with G = Hq / Hkv query heads per key/value head and
 * g = h / G (integer division),
 *     s_j = scale * sum_d q[b][h][d] * K_b[g][j][d]          for j < L_b = ctx[b]
 *     p_j = exp(s_j - max_i s_i) / sum_i exp(s_i - max_i s_i)
 *     o[b][h][d] = sum_j p_j * V_b[g][j][d]
 * in fp64 with bf16 inputs decoded exactly.  A sequence with L_b = 0 has o = 0.
 *
 * Paged cache.  Token j of sequence b lives in physical page block_table[b][j / P] at
 * slot j % P (P tokens per page).  Per page and key/value head:
 *     K cache [n_pages][Hkv][P][D]   (token-major: a token's D values contiguous)
 *     V cache [n_pages][Hkv][D][P]   (dimension-major: a dimension's P values contiguous)
 * bf16 = the upper 16 bits of an fp32.
 */
#include <math.h>
#include <stdint.h>
#include <string.h>

static double attn_dec_bf16(uint16_t b)
{
    uint32_t u = (uint32_t)b << 16;
    float f;
    memcpy(&f, &u, 4);
    return (double)f;
}

/* o[B][Hq][D] (fp64).  Returns 0, or -1 for inconsistent sizes or a page index outside
 * [0, n_pages). */
int oracle_attn_decode(int B, int Hq, int Hkv, int D, int P, const uint16_t *q, const uint16_t *kc,
                       const uint16_t *vc, int64_t n_pages, const int32_t *block_table, int max_pages,
                       const int32_t *ctx, double scale, double *o)
{
    if (B < 0 || Hq <= 0 || Hkv <= 0 || Hq % Hkv || D <= 0 || P <= 0 || max_pages < 0) return -1;
    const int G = Hq / Hkv;
    for (int b = 0; b < B; b++) {
        const int L = ctx[b];
        if (L < 0 || L > max_pages * P) return -1;
        for (int j = 0; j < L; j++) {
            const int32_t pg = block_table[(int64_t)b * max_pages + j / P];
            if (pg < 0 || pg >= n_pages) return -1;
        }
        for (int h = 0; h < Hq; h++) {
            const int g = h / G;
            const uint16_t *qv = q + ((int64_t)b * Hq + h) * D;
            double *ov = o + ((int64_t)b * Hq + h) * D;
            for (int d = 0; d < D; d++) ov[d] = 0.0;
            if (L == 0) continue;
            /* scores */
            double m = -INFINITY;
            for (int j = 0; j < L; j++) {
                const int64_t pg = block_table[(int64_t)b * max_pages + j / P];
                const uint16_t *kv = kc + ((pg * Hkv + g) * P + j % P) * (int64_t)D;
                double s = 0.0;
                for (int d = 0; d < D; d++) s += attn_dec_bf16(qv[d]) * attn_dec_bf16(kv[d]);
                s *= scale;
                if (s > m) m = s;
            }
            /* softmax weights and the weighted sum of values */
            double den = 0.0;
            for (int j = 0; j < L; j++) {
                const int64_t pg = block_table[(int64_t)b * max_pages + j / P];
                const uint16_t *kv = kc + ((pg * Hkv + g) * P + j % P) * (int64_t)D;
                double s = 0.0;
                for (int d = 0; d < D; d++) s += attn_dec_bf16(qv[d]) * attn_dec_bf16(kv[d]);
                const double e = exp(s * scale - m);
                den += e;
                const uint16_t *vp = vc + (pg * Hkv + g) * (int64_t)D * P;
                for (int d = 0; d < D; d++) ov[d] += e * attn_dec_bf16(vp[(int64_t)d * P + j % P]);
            }
            for (int d = 0; d < D; d++) ov[d] /= den;
        }
    }
    return 0;
}
