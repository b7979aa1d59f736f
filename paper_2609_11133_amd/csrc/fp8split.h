// Two-term FP8 (E4M3) split of activation groups for the scaled MFMA path.
//
// A group of 32 consecutive inputs is held as x ~= hi * 2^(ehi-127) + lo * 2^(elo-127):
// hi and lo are FP8-E4M3 codes, ehi and elo E8M0 exponents (the operand scales of
// the CDNA4 scaled MFMA).  The group's largest magnitude maps into [128, 256), below
// the E4M3 maximum; the residual x - hi*2^ehi is exact in fp32 and is encoded the
// same way.  The split error is at most half an E4M3 step of the residual, about
// 2^-9 of the group's largest magnitude.  Multi-term splitting of a wide operand
// into narrow ones follows the error-free splitting idea of Ozaki et al. (2012) and
// the bf16x3 scheme of Henry, Tang and Heinecke (2019).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace moe {

typedef short i16x2 __attribute__((ext_vector_type(2)));
typedef float f32x2v __attribute__((ext_vector_type(2)));

// E8M0 exponent code for a group whose largest magnitude is amax (127 for a zero group).
__device__ inline int exp_for_group(float amax)
{
    if (!(amax > 0.f)) return 127;
    const int e = (int)((__float_as_uint(amax) >> 23) & 0xFF) - 127;  // floor(log2 amax) for normals
    const int code = e - 7 + 127;
    return code < 1 ? 1 : (code > 254 ? 254 : code);
}

__device__ inline float pow2_of_code(int code) { return __uint_as_float((uint32_t)code << 23); }  // 2^(code-127)

// Encode 4 fp32 values (already divided by the group scale, |v| < 256) as 4 FP8 bytes.
__device__ inline uint32_t enc4_e4m3(float a, float b, float c, float d)
{
    i16x2 lo = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32((i16x2){0, 0}, a, b, 1.0f, false);
    i16x2 hi = __builtin_amdgcn_cvt_scalef32_pk_fp8_f32(lo, c, d, 1.0f, true);
    return __builtin_bit_cast(uint32_t, hi);
}

__device__ inline void dec4_e4m3(uint32_t q, float &a, float &b, float &c, float &d)
{
    const f32x2v x = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(q, 1.0f, false);
    const f32x2v y = __builtin_amdgcn_cvt_scalef32_pk_f32_fp8(q, 1.0f, true);
    a = x.x;
    b = x.y;
    c = y.x;
    d = y.y;
}

// Split N values of one group, given the group's largest magnitude and the largest
// magnitude of the residual (computed by the caller, possibly across lanes, with
// residual_amax()).  Two-phase use: split_hi() then split_lo().
template <int N>
__device__ inline void split_hi(const float (&v)[N], int ch, uint32_t (&qh)[N / 4], float (&res)[N])
{
    const float inv = pow2_of_code(254 - ch), sc = pow2_of_code(ch);
#pragma unroll
    for (int i = 0; i < N / 4; ++i) {
        qh[i] = enc4_e4m3(v[4 * i] * inv, v[4 * i + 1] * inv, v[4 * i + 2] * inv, v[4 * i + 3] * inv);
        float a, b, c, d;
        dec4_e4m3(qh[i], a, b, c, d);
        res[4 * i] = v[4 * i] - a * sc;  // exact residuals
        res[4 * i + 1] = v[4 * i + 1] - b * sc;
        res[4 * i + 2] = v[4 * i + 2] - c * sc;
        res[4 * i + 3] = v[4 * i + 3] - d * sc;
    }
}

template <int N>
__device__ inline void split_lo(const float (&res)[N], int cl, uint32_t (&ql)[N / 4])
{
    const float inv = pow2_of_code(254 - cl);
#pragma unroll
    for (int i = 0; i < N / 4; ++i)
        ql[i] = enc4_e4m3(res[4 * i] * inv, res[4 * i + 1] * inv, res[4 * i + 2] * inv, res[4 * i + 3] * inv);
}

template <int N>
__device__ inline float amax_of(const float (&v)[N])
{
    float m = 0.f;
#pragma unroll
    for (int i = 0; i < N; ++i) m = fmaxf(m, fabsf(v[i]));
    return m;
}

}  // namespace moe
