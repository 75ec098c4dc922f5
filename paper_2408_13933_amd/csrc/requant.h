// Device-side requantization shared by every qlinear kernel: the per-column
// fixed-point parameters and the per-element epilogue
//   c = sat_int32(acc + off[n]),  off[n] = bias_q[n] - a_zp * colsum[n]
//   r = floor((c * M0[n] + 2^(sh[n]-1)) / 2^sh[n])
//   y = clamp(r + out_zp, qmin, qmax)
// (the integer-only rescale between layers; the paper requires fixed-point
// integer arithmetic throughout, Section 1 and Section 3.1).
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mq {

struct ColParams {
    int32_t off;  // bias_q - a_zp * colsum, saturated to int32
    int32_t m0;   // Q31 multiplier in [2^30, 2^31), or 0
    int32_t sh;   // right shift; >= 63 means r = 0, <= 0 means saturate
    int32_t bq;   // bias_q alone, |bias_q| <= 2^30
};

// Fixed-point form of M = (a_scale * w_scale) / out_scale and the bias in
// accumulator units.  fp64 throughout: the product of two fp32 values is
// exact in fp64, the division is one correctly rounded operation, and
// frexp/ldexp/rint are exact, so the integers do not depend on the device.
__device__ inline ColParams derive_col_params_v(float a_scale, float w_scale, float out_scale,
                                                bool has_bias, float bias_n, int32_t colsum,
                                                int32_t a_zp)
{
#pragma clang fp contract(off)
    ColParams p;
    const double prod = (double)a_scale * (double)w_scale;
    const double M = prod / (double)out_scale;
    if (!(M > 0.0)) {
        p.m0 = 0;
        p.sh = 31;
    } else if (__builtin_isinf(M)) {
        p.m0 = 1 << 30;
        p.sh = 0;
    } else {
        int e = 0;
        const double f = frexp(M, &e);
        long long m0 = (long long)rint(ldexp(f, 31));
        if (m0 == (1LL << 31)) {
            m0 = 1LL << 30;
            e += 1;
        }
        p.m0 = (int32_t)m0;
        p.sh = 31 - e;
    }
    long long bq = 0;
    if (has_bias) {
        double t = (double)bias_n / prod;
        t = fmin(fmax(t, -1073741824.0), 1073741824.0);
        bq = (long long)rint(t);
    }
    long long off = bq - (long long)a_zp * (long long)colsum;
    off = off < INT32_MIN ? INT32_MIN : (off > INT32_MAX ? INT32_MAX : off);
    p.off = (int32_t)off;
    p.bq = (int32_t)bq;
    return p;
}

__device__ inline ColParams derive_col_params(float a_scale, float w_scale, float out_scale,
                                              const float* bias_n, int32_t colsum,
                                              int32_t a_zp)
{
    return derive_col_params_v(a_scale, w_scale, out_scale, bias_n != nullptr,
                               bias_n != nullptr ? *bias_n : 0.0f, colsum, a_zp);
}

// r for one corrected accumulator c (int32).
__device__ inline int32_t requant_round(int32_t c, int32_t m0, int32_t sh)
{
    if (sh >= 63) return 0;
    if (sh >= 1) {
        const long long prod = (long long)c * (long long)m0 + (1LL << (sh - 1));
        const long long r = prod >> sh;  // arithmetic shift = floor division
        // |r| <= 2^31 here; anything beyond int16 saturates later anyway
        return (int32_t)(r < -(1LL << 30) ? -(1LL << 30) : (r > (1LL << 30) ? (1LL << 30) : r));
    }
    return c > 0 ? (1 << 30) : (c < 0 ? -(1 << 30) : 0);
}

// y from the corrected accumulator c.
__device__ inline int32_t requant_c(int32_t c, const ColParams& p, int32_t out_zp, int32_t qmin,
                                    int32_t qmax)
{
    const int32_t r = requant_round(c, p.m0, p.sh);
    int32_t y = r + out_zp;  // |r| <= 2^30, |out_zp| <= 2^15: no overflow
    y = y < qmin ? qmin : (y > qmax ? qmax : y);
    return y;
}

__device__ inline int32_t requant_out(int32_t acc, const ColParams& p, int32_t out_zp,
                                      int32_t qmin, int32_t qmax)
{
    return requant_c(__builtin_elementwise_add_sat(acc, p.off), p, out_zp, qmin, qmax);
}

// The dequantized value of an output code (the inverse of Eq.(4), the
// arithmetic of mq_dequant: one exact integer subtraction, one fp32
// multiply), for the layers that write it in the same pass.
__device__ inline float dequant_code(int32_t q, float alpha, int32_t zp)
{
#pragma clang fp contract(off)
    return alpha * (float)(q - zp);
}

// 16-bit activations (W8A16): the kernels split each code a into an int8
// high part h = a >> 8 and an offset low part l = (a & 255) - 128, so that
// a = 256 h + l + 128 and
//   sum_k (a - a_zp) w = 256 sum h w + sum l w + (128 - a_zp) colsum,
// two exact int8 products.  |(128 - a_zp) colsum| < 2^39: int64.
__device__ inline int64_t a16_offset(const ColParams& cp, int32_t a_zp, int32_t colsum)
{
    return (int64_t)cp.bq + (int64_t)(128 - a_zp) * (int64_t)colsum;
}

// 16 int16 codes in k order (32 bytes: x0 = codes 0-7, x1 = codes 8-15; a
// dword holds two codes, the even one in its low half) -> the int8 MFMA
// operands h (high bytes) and l (low bytes - 128), 16 lanes each in k order.
// v_perm_b32 selector bytes 0-3 pick from the second source, 4-7 from the
// first.
typedef int a16_v4i __attribute__((ext_vector_type(4)));
__device__ inline void split_a16(const a16_v4i& x0, const a16_v4i& x1, a16_v4i& h, a16_v4i& l)
{
    h[0] = (int)__builtin_amdgcn_perm((uint32_t)x0[1], (uint32_t)x0[0], 0x07050301u);
    h[1] = (int)__builtin_amdgcn_perm((uint32_t)x0[3], (uint32_t)x0[2], 0x07050301u);
    h[2] = (int)__builtin_amdgcn_perm((uint32_t)x1[1], (uint32_t)x1[0], 0x07050301u);
    h[3] = (int)__builtin_amdgcn_perm((uint32_t)x1[3], (uint32_t)x1[2], 0x07050301u);
    l[0] = (int)(__builtin_amdgcn_perm((uint32_t)x0[1], (uint32_t)x0[0], 0x06040200u) ^ 0x80808080u);
    l[1] = (int)(__builtin_amdgcn_perm((uint32_t)x0[3], (uint32_t)x0[2], 0x06040200u) ^ 0x80808080u);
    l[2] = (int)(__builtin_amdgcn_perm((uint32_t)x1[1], (uint32_t)x1[0], 0x06040200u) ^ 0x80808080u);
    l[3] = (int)(__builtin_amdgcn_perm((uint32_t)x1[3], (uint32_t)x1[2], 0x06040200u) ^ 0x80808080u);
}

__device__ inline int32_t sat32(int64_t c)
{
    return (int32_t)(c < INT32_MIN ? INT32_MIN : (c > INT32_MAX ? INT32_MAX : c));
}

// Asymmetric per-channel weights (codes W - w_zp[n]): the zero-point adds
// the term -w_zp[n] * sum_k (A[m][k] - a_zp) = -w_zp[n] * rs[m], where
// rs[m] = rowsum[m] - K * a_zp (|rs| <= 255 K).  Exact in int64, then
//   c = sat_int32(acc + off + nzw * rs),  nzw = -w_zp[n].
__device__ inline int32_t corrected_acc_asym(int32_t acc, int32_t off, int32_t nzw, int32_t rs)
{
    const long long c = (long long)acc + (long long)off + (long long)nzw * (long long)rs;
    return (int32_t)(c < INT32_MIN ? INT32_MIN : (c > INT32_MAX ? INT32_MAX : c));
}

// ---------------------------------------------------------------------------
// Branch-free integer form for the tiled kernels; it computes exactly the
// value of requant_out.
//
// integer form: r = floor((c*M0 + 2^(sh-1)) / 2^sh) is rewritten with an
// effective shift s >= 33, where it equals (mulhi(c, M0) + 2^(s-33)) >> (s-32)
// (the low 32 bits of the product cannot carry into the rounding).  For
// 3 <= sh <= 32 the accumulator is first limited to +-2^(sh-3), which cannot
// change the saturated result, and shifted left by 33 - sh without overflow;
// for sh <= 2 every non-zero c saturates and c is limited to +-1 and shifted
// by 30.
struct EpiInt {
    int32_t m0, rnd, shr, pre, bnd;
};

__device__ inline EpiInt epi_int_params(const ColParams& cp)
{
    EpiInt e;
    e.m0 = cp.m0;
    if (cp.m0 == 0) {  // r = 0 for every c
        e.rnd = 1; e.shr = 1; e.pre = 0; e.bnd = 0x7FFFFFFF;
    } else if (cp.sh >= 33) {
        const int s = cp.sh < 63 ? cp.sh : 63;
        e.rnd = 1 << (s - 33); e.shr = s - 32; e.pre = 0; e.bnd = 0x7FFFFFFF;
    } else if (cp.sh >= 3) {
        e.rnd = 1; e.shr = 1; e.pre = 33 - cp.sh; e.bnd = 1 << (cp.sh - 3);
    } else {
        e.rnd = 1; e.shr = 1; e.pre = 30; e.bnd = 1;
    }
    return e;
}

__device__ inline int32_t requant_int(int32_t acc, int32_t off, const EpiInt& e, int32_t zp,
                                      int32_t qmin, int32_t qmax)
{
    int32_t c = __builtin_elementwise_add_sat(acc, off);
    c = max(min(c, e.bnd), -e.bnd);  // v_med3_i32
    c = (int32_t)((uint32_t)c << e.pre);
    const int32_t h = __mulhi(c, e.m0);
    const int32_t r = (h + e.rnd) >> e.shr;
    return max(min(r + zp, qmax), qmin);  // v_med3_i32
}

}  // namespace mq
