// Bandwidth-bound kernels around the integer linear layer: the static
// activation quantizer (Section 4.2, Eq.(4)), its inverse, the fold of the
// smoothing vector (Section 3.2, Eq.(1)) and the per-channel weight packer.
//
// All of them stream HBM: 16-byte vector loads on consecutive lanes,
// grid-stride loops sized to the 256 CUs, and scalar code only for ragged
// tails and unaligned buffers.
// Floating point is IEEE: correctly rounded fp32 division, rint = round
// half to even, no contraction.
#include "mq_internal.h"

namespace mq {
namespace {

constexpr int kThreads = 256;

inline int grid_for(int64_t items, int per_block)
{
    int64_t b = (items + per_block - 1) / per_block;
    if (b < 1) b = 1;
    // enough blocks for every CU many times over; the loops stride.  Large
    // streams run best with about one iteration per thread: dequantizing
    // 512 x 256000 int16 codes (786 MB moved) takes 158 us on 4096 blocks
    // and 135 us (5.8 TB/s) on 65536 (measured on MI355X)
    if (b > 256 * 256) b = 256 * 256;
    return (int)b;
}

inline bool aligned(const void* p, uintptr_t a) { return ((uintptr_t)p % a) == 0; }

template <int BITS>
__device__ inline int32_t quant1(float x, float alpha, int32_t zp)
{
#pragma clang fp contract(off)
    constexpr int32_t qmin = -(1 << (BITS - 1));
    constexpr int32_t qmax = (1 << (BITS - 1)) - 1;
    float t = x / alpha;
    t = fminf(fmaxf(t, -1048576.0f), 1048576.0f);
    int32_t v = (int32_t)rintf(t) + zp;
    return v < qmin ? qmin : (v > qmax ? qmax : v);
}

// x / alpha as far as rint() can tell.  The product with the rounded
// reciprocal is within 2.5 ulp of the quotient (reciprocal error 0.5 ulp,
// product rounding 0.5 ulp, quotient rounding 0.5 ulp, relative to |t|), so
// where it lies more than 4 ulp (|t| * 2^-21) from every half-integer,
// rounding it to an integer gives the same result as rounding the correctly
// rounded quotient.  Other lanes (and NaN, infinities, |t| >= 2^20) take
// the correctly rounded division, behind a wave-uniform branch so the
// division is not evaluated speculatively on every lane.
__device__ inline bool product_decides_rint(float t)
{
#pragma clang fp contract(off)
    const float d = fabsf(t - rintf(t));  // exact for |t| < 2^23
    return fabsf(0.5f - d) > fabsf(t) * 0x1p-21f;
}

template <int BITS>
__device__ inline int32_t code_from_quotient(float t, int32_t zp)
{
    constexpr int32_t qmin = -(1 << (BITS - 1));
    constexpr int32_t qmax = (1 << (BITS - 1)) - 1;
    t = fminf(fmaxf(t, -1048576.0f), 1048576.0f);
    int32_t v = (int32_t)rintf(t) + zp;
    return v < qmin ? qmin : (v > qmax ? qmax : v);
}

// One float4 -> 4 codes per thread and step, lanes on consecutive float4s
// (every load and store instruction covers a contiguous span); two steps
// per loop trip keep two loads in flight.  Returns the sum of the 4 codes.
template <int BITS>
__device__ inline int32_t quant_store4(const float4 a, float alpha, float inv, int32_t zp, void* q,
                                       int64_t i)
{
#pragma clang fp contract(off)
    const float xs[4] = {a.x, a.y, a.z, a.w};
    float t[4];
    bool ok = true;
#pragma unroll
    for (int k = 0; k < 4; ++k) {
        t[k] = xs[k] * inv;
        ok = ok && product_decides_rint(t[k]);
    }
    if (__builtin_expect(__ballot(!ok) != 0, 0)) {
#pragma unroll
        for (int k = 0; k < 4; ++k)
            if (!product_decides_rint(xs[k] * inv)) t[k] = xs[k] / alpha;
    }
    const int32_t v0 = code_from_quotient<BITS>(t[0], zp);
    const int32_t v1 = code_from_quotient<BITS>(t[1], zp);
    const int32_t v2 = code_from_quotient<BITS>(t[2], zp);
    const int32_t v3 = code_from_quotient<BITS>(t[3], zp);
    if constexpr (BITS == 8) {
        reinterpret_cast<uint32_t*>(q)[i] = ((uint32_t)v0 & 0xFFu) | (((uint32_t)v1 & 0xFFu) << 8) |
                                            (((uint32_t)v2 & 0xFFu) << 16) | ((uint32_t)v3 << 24);
    } else {
        reinterpret_cast<uint2*>(q)[i] =
            make_uint2(((uint32_t)v0 & 0xFFFFu) | ((uint32_t)v1 << 16),
                       ((uint32_t)v2 & 0xFFFFu) | ((uint32_t)v3 << 16));
    }
    return v0 + v1 + v2 + v3;
}

template <int BITS>
__global__ __launch_bounds__(kThreads) void quantize_act_vec(const float4* __restrict__ x,
                                                             int64_t n4, float alpha,
                                                             float inv_alpha, int32_t zp,
                                                             void* __restrict__ q)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + stride < n4; i += 2 * stride) {
        const float4 a = x[i];
        const float4 b = x[i + stride];
        quant_store4<BITS>(a, alpha, inv_alpha, zp, q, i);
        quant_store4<BITS>(b, alpha, inv_alpha, zp, q, i + stride);
    }
    if (i < n4) quant_store4<BITS>(x[i], alpha, inv_alpha, zp, q, i);
}

template <int BITS>
__global__ __launch_bounds__(kThreads) void quantize_act_scalar(const float* __restrict__ x,
                                                                int64_t begin, int64_t n,
                                                                float alpha, int32_t zp,
                                                                void* __restrict__ q)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = begin + (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        const int32_t v = quant1<BITS>(x[i], alpha, zp);
        if constexpr (BITS == 8)
            static_cast<int8_t*>(q)[i] = (int8_t)v;
        else
            static_cast<int16_t*>(q)[i] = (int16_t)v;
    }
}

// Sum over the block of one int32 per thread (every thread gets it).
__device__ inline int32_t block_sum(int32_t v)
{
    __shared__ int32_t red[kThreads / 64];
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    int32_t t = 0;
#pragma unroll
    for (int i = 0; i < kThreads / 64; ++i) t += red[i];
    return t;
}

// Eq.(4) quantizer on int8 rows fused with their code sums (the term that
// asymmetric weights multiply): one block per row, the codes are those of
// quantize_act_vec / quantize_act_scalar, bit for bit.
__global__ __launch_bounds__(kThreads) void quantize_rowsum_vec(const float4* __restrict__ x,
                                                                int64_t K4, float alpha,
                                                                float inv_alpha, int32_t zp,
                                                                int8_t* __restrict__ q,
                                                                int32_t* __restrict__ rowsum)
{
    const int64_t m = blockIdx.x;
    const float4* xr = x + m * K4;
    int8_t* qr = q + m * K4 * 4;
    int32_t sum = 0;
    int64_t i = threadIdx.x;
    for (; i + kThreads < K4; i += 2 * kThreads) {
        const float4 a = xr[i];
        const float4 b = xr[i + kThreads];
        sum += quant_store4<8>(a, alpha, inv_alpha, zp, qr, i);
        sum += quant_store4<8>(b, alpha, inv_alpha, zp, qr, i + kThreads);
    }
    if (i < K4) sum += quant_store4<8>(xr[i], alpha, inv_alpha, zp, qr, i);
    sum = block_sum(sum);
    if (threadIdx.x == 0) rowsum[m] = sum;
}

__global__ __launch_bounds__(kThreads) void quantize_rowsum_scalar(const float* __restrict__ x,
                                                                   int64_t K, float alpha,
                                                                   int32_t zp,
                                                                   int8_t* __restrict__ q,
                                                                   int32_t* __restrict__ rowsum)
{
    const int64_t m = blockIdx.x;
    int32_t sum = 0;
    for (int64_t k = threadIdx.x; k < K; k += kThreads) {
        const int32_t v = quant1<8>(x[m * K + k], alpha, zp);
        q[m * K + k] = (int8_t)v;
        sum += v;
    }
    sum = block_sum(sum);
    if (threadIdx.x == 0) rowsum[m] = sum;
}

template <int BITS>
__device__ inline float deq1(int32_t q, float alpha, int32_t zp)
{
#pragma clang fp contract(off)
    return alpha * (float)(q - zp);
}

template <int BITS>
__device__ inline void deq_store4(const void* __restrict__ q, float alpha, int32_t zp,
                                  float4* __restrict__ y, int64_t i)
{
    int32_t v[4];
    if constexpr (BITS == 8) {
        const uint32_t p = reinterpret_cast<const uint32_t*>(q)[i];
#pragma unroll
        for (int k = 0; k < 4; ++k) v[k] = (int32_t)(int8_t)(p >> (8 * k));
    } else {
        const uint2 p = reinterpret_cast<const uint2*>(q)[i];
        v[0] = (int32_t)(int16_t)(p.x & 0xFFFFu);
        v[1] = (int32_t)(int16_t)(p.x >> 16);
        v[2] = (int32_t)(int16_t)(p.y & 0xFFFFu);
        v[3] = (int32_t)(int16_t)(p.y >> 16);
    }
    y[i] = make_float4(deq1<BITS>(v[0], alpha, zp), deq1<BITS>(v[1], alpha, zp),
                       deq1<BITS>(v[2], alpha, zp), deq1<BITS>(v[3], alpha, zp));
}

// 4 codes -> one float4 per thread and step, lanes on consecutive groups
template <int BITS>
__global__ __launch_bounds__(kThreads) void dequant_vec(const void* __restrict__ q, int64_t n4,
                                                        float alpha, int32_t zp,
                                                        float4* __restrict__ y)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    for (; i + stride < n4; i += 2 * stride) {
        deq_store4<BITS>(q, alpha, zp, y, i);
        deq_store4<BITS>(q, alpha, zp, y, i + stride);
    }
    if (i < n4) deq_store4<BITS>(q, alpha, zp, y, i);
}

template <int BITS>
__global__ __launch_bounds__(kThreads) void dequant_scalar(const void* __restrict__ q,
                                                           int64_t begin, int64_t n, float alpha,
                                                           int32_t zp, float* __restrict__ y)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = begin + (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        const int32_t v = BITS == 8 ? (int32_t) static_cast<const int8_t*>(q)[i]
                                    : (int32_t) static_cast<const int16_t*>(q)[i];
        y[i] = deq1<BITS>(v, alpha, zp);
    }
}

// w_hat[n][k] = w[n][k] * s[k]  (DIVIDE = false)
// x_hat[m][k] = x[m][k] / s[k]  (DIVIDE = true)
template <bool DIVIDE>
__global__ __launch_bounds__(kThreads) void fold_kernel(const float* __restrict__ in,
                                                        const float* __restrict__ sv,
                                                        int64_t rows, int64_t K,
                                                        float* __restrict__ out)
{
#pragma clang fp contract(off)
    const int64_t total = rows * K;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < total; i += stride) {
        const float s = sv[i % K];
        out[i] = DIVIDE ? in[i] / s : in[i] * s;
    }
}

// One block per weight row: absmax, scale, then codes and their sum.
template <int BITS>
__global__ __launch_bounds__(kThreads) void pack_weights_kernel(const float* __restrict__ w,
                                                                int64_t K, void* __restrict__ wq,
                                                                float* __restrict__ scale_out,
                                                                int32_t* __restrict__ colsum)
{
#pragma clang fp contract(off)
    constexpr float Q = BITS == 8 ? 127.0f : 7.0f;
    __shared__ float red_f[kThreads / 64];
    __shared__ int32_t red_i[kThreads / 64];
    const int64_t n = blockIdx.x;
    const float* row = w + n * K;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    float m = 0.0f;
    for (int64_t k = threadIdx.x; k < K; k += kThreads) m = fmaxf(m, fabsf(row[k]));
    for (int o = 32; o > 0; o >>= 1) m = fmaxf(m, __shfl_xor(m, o));
    if (lane == 0) red_f[wave] = m;
    __syncthreads();
    m = red_f[0];
#pragma unroll
    for (int i = 1; i < kThreads / 64; ++i) m = fmaxf(m, red_f[i]);
    float s = m / Q;
    if (!(s > 0.0f)) s = 1.0f;

    int32_t sum = 0;
    if constexpr (BITS == 8) {
        int8_t* dst = static_cast<int8_t*>(wq) + n * K;
        for (int64_t k = threadIdx.x; k < K; k += kThreads) {
            const float t = fminf(fmaxf(row[k] / s, -Q), Q);
            const int32_t v = (int32_t)rintf(t);
            dst[k] = (int8_t)v;
            sum += v;
        }
    } else {
        uint8_t* dst = static_cast<uint8_t*>(wq) + n * (K / 2);
        for (int64_t j = threadIdx.x; j < K / 2; j += kThreads) {
            const float t0 = fminf(fmaxf(row[2 * j] / s, -Q), Q);
            const float t1 = fminf(fmaxf(row[2 * j + 1] / s, -Q), Q);
            const int32_t v0 = (int32_t)rintf(t0);
            const int32_t v1 = (int32_t)rintf(t1);
            dst[j] = (uint8_t)(((uint32_t)v0 & 0xFu) | (((uint32_t)v1 & 0xFu) << 4));
            sum += v0 + v1;
        }
    }
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) red_i[wave] = sum;
    __syncthreads();
    if (threadIdx.x == 0) {
        int32_t t = 0;
#pragma unroll
        for (int i = 0; i < kThreads / 64; ++i) t += red_i[i];
        colsum[n] = t;
        scale_out[n] = s;
    }
}

// Asymmetric weights (Section 5.1): the Eq.(2)-(4) quantizer over a range
// [lo, hi] that contains 0 -- the finite values of one row (per channel)
// or of the whole matrix (per tensor).  alpha = (hi - lo)/(2^bits - 1) in
// fp64, rounded to fp32; the unsigned zero-point rint(-lo/alpha) clamped to
// the grid; codes clamp(rint(w/alpha) + zp) with one correctly rounded fp32
// division.  A zero-width range takes alpha = 1 and zero-point -2^(bits-1).
template <int BITS>
__device__ inline void asym_format(float lo, float hi, float* alpha_out, int32_t* zp_out)
{
#pragma clang fp contract(off)
    constexpr double QMAX = (double)((1 << BITS) - 1);
    float alpha = 1.0f;
    double beta = 0.0;
    const double width = (double)hi - (double)lo;
    if (width != 0.0) {
        const float a = (float)(width / QMAX);
        if (a > 0.0f && __builtin_isfinite(a)) {
            alpha = a;
            beta = (double)lo / (double)alpha;
        }
    }
    const double zu = fmin(fmax(rint(-beta), 0.0), QMAX);
    *alpha_out = alpha;
    *zp_out = (int32_t)zu - (1 << (BITS - 1));
}

// [min, max] of the finite values of v[0..n), widened to contain 0, for the
// whole block (every thread gets the result).
__device__ inline void block_finite_range(const float* v, int64_t n, float* lo_out, float* hi_out)
{
    __shared__ float red_lo[kThreads / 64], red_hi[kThreads / 64];
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    float lo = 0.0f, hi = 0.0f;
    for (int64_t k = threadIdx.x; k < n; k += kThreads) {
        const float x = v[k];
        if (__builtin_isfinite(x)) {
            lo = fminf(lo, x);
            hi = fmaxf(hi, x);
        }
    }
    for (int o = 32; o > 0; o >>= 1) {
        lo = fminf(lo, __shfl_xor(lo, o));
        hi = fmaxf(hi, __shfl_xor(hi, o));
    }
    if (lane == 0) {
        red_lo[wave] = lo;
        red_hi[wave] = hi;
    }
    __syncthreads();
    lo = red_lo[0];
    hi = red_hi[0];
#pragma unroll
    for (int i = 1; i < kThreads / 64; ++i) {
        lo = fminf(lo, red_lo[i]);
        hi = fmaxf(hi, red_hi[i]);
    }
    *lo_out = lo;
    *hi_out = hi;
}

// Per-tensor range, step 1: each row's range into lo[n], hi[n].
__global__ __launch_bounds__(kThreads) void row_range_kernel(const float* __restrict__ w,
                                                             int64_t K, float* __restrict__ lo,
                                                             float* __restrict__ hi)
{
    float l, h;
    block_finite_range(w + (int64_t)blockIdx.x * K, K, &l, &h);
    if (threadIdx.x == 0) {
        lo[blockIdx.x] = l;
        hi[blockIdx.x] = h;
    }
}

// Per-tensor range, step 2 (one block): the rows' ranges -> the tensor's
// alpha and zero-point, written to scale[0] and zp[0].  lo/hi alias
// scale/zp (the host passes the output arrays as the scratch of step 1).
template <int BITS>
__global__ __launch_bounds__(kThreads) void tensor_format_kernel(int64_t N, float* scale,
                                                                 int32_t* zp)
{
    __shared__ float red_lo[kThreads / 64], red_hi[kThreads / 64];
    const float* lo_in = scale;
    const float* hi_in = reinterpret_cast<const float*>(zp);
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    float lo = 0.0f, hi = 0.0f;
    for (int64_t n = threadIdx.x; n < N; n += kThreads) {
        lo = fminf(lo, lo_in[n]);
        hi = fmaxf(hi, hi_in[n]);
    }
    for (int o = 32; o > 0; o >>= 1) {
        lo = fminf(lo, __shfl_xor(lo, o));
        hi = fmaxf(hi, __shfl_xor(hi, o));
    }
    if (lane == 0) {
        red_lo[wave] = lo;
        red_hi[wave] = hi;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
#pragma unroll
        for (int i = 1; i < kThreads / 64; ++i) {  // lo, hi already hold wave 0's
            lo = fminf(lo, red_lo[i]);
            hi = fmaxf(hi, red_hi[i]);
        }
        float a;
        int32_t z;
        asym_format<BITS>(lo, hi, &a, &z);
        scale[0] = a;
        zp[0] = z;
    }
}

// Codes, code sums and (per channel) the row's own format.  PER_TENSOR:
// the format comes from scale[0], zp[0] (written by tensor_format_kernel);
// row 0 leaves them in place and every other row copies them.
template <int BITS, bool PER_TENSOR>
__global__ __launch_bounds__(kThreads) void pack_weights_asym_kernel(
    const float* __restrict__ w, int64_t K, void* __restrict__ wq, float* scale_out,
    int32_t* zp_out, int32_t* __restrict__ colsum)
{
#pragma clang fp contract(off)
    constexpr int QLO = -(1 << (BITS - 1)), QHI = (1 << (BITS - 1)) - 1;
    constexpr float LIM = 1048576.0f;  // 2^20: the quotient converts to an integer
    __shared__ int32_t red_i[kThreads / 64];
    const int64_t n = blockIdx.x;
    const float* row = w + n * K;
    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;

    float alpha;
    int32_t zp;
    if constexpr (PER_TENSOR) {
        alpha = scale_out[0];
        zp = zp_out[0];
    } else {
        float lo, hi;
        block_finite_range(row, K, &lo, &hi);
        asym_format<BITS>(lo, hi, &alpha, &zp);
    }

    auto code = [&](float v) {
        const float t = fminf(fmaxf(v / alpha, -LIM), LIM);
        const int32_t q = (int32_t)rintf(t) + zp;
        return q < QLO ? QLO : (q > QHI ? QHI : q);
    };
    int32_t sum = 0;
    if constexpr (BITS == 8) {
        int8_t* dst = static_cast<int8_t*>(wq) + n * K;
        for (int64_t k = threadIdx.x; k < K; k += kThreads) {
            const int32_t v = code(row[k]);
            dst[k] = (int8_t)v;
            sum += v;
        }
    } else {
        uint8_t* dst = static_cast<uint8_t*>(wq) + n * (K / 2);
        for (int64_t j = threadIdx.x; j < K / 2; j += kThreads) {
            const int32_t v0 = code(row[2 * j]);
            const int32_t v1 = code(row[2 * j + 1]);
            dst[j] = (uint8_t)(((uint32_t)v0 & 0xFu) | (((uint32_t)v1 & 0xFu) << 4));
            sum += v0 + v1;
        }
    }
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) red_i[wave] = sum;
    __syncthreads();
    if (threadIdx.x == 0) {
        int32_t t = 0;
#pragma unroll
        for (int i = 0; i < kThreads / 64; ++i) t += red_i[i];
        colsum[n] = t;
        if (!PER_TENSOR || n != 0) {
            scale_out[n] = alpha;
            zp_out[n] = zp;
        }
    }
}

// Row sums of int8 activations, one wave per row: 16-byte loads folded with
// dot4 against ones when the rows are 16-byte aligned, bytes otherwise.
// |sum| <= 128 * K fits int32 for every accepted K.
__global__ __launch_bounds__(kThreads) void act_rowsum_kernel(const int8_t* __restrict__ a,
                                                              int64_t M, int64_t K,
                                                              int32_t* __restrict__ rowsum)
{
    const int lane = threadIdx.x & 63;
    const int64_t m = (int64_t)blockIdx.x * (kThreads / 64) + (threadIdx.x >> 6);
    if (m >= M) return;
    const int8_t* row = a + m * K;
    int32_t sum = 0;
    int64_t k0 = 0;
    if (((uintptr_t)row % 16) == 0) {
        const int64_t n16 = K / 16;
        const int4* r16 = reinterpret_cast<const int4*>(row);
        for (int64_t i = lane; i < n16; i += 64) {
            const int4 v = r16[i];
            sum = __builtin_amdgcn_sdot4(v.x, 0x01010101, sum, false);
            sum = __builtin_amdgcn_sdot4(v.y, 0x01010101, sum, false);
            sum = __builtin_amdgcn_sdot4(v.z, 0x01010101, sum, false);
            sum = __builtin_amdgcn_sdot4(v.w, 0x01010101, sum, false);
        }
        k0 = n16 * 16;
    }
    for (int64_t k = k0 + lane; k < K; k += 64) sum += row[k];
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if (lane == 0) rowsum[m] = sum;
}

}  // namespace

hipError_t launch_quantize_act(const float* x, int64_t n, float alpha, int32_t zp, int32_t bits,
                               void* q, hipStream_t st)
{
    int64_t n4 = 0;
    const uintptr_t qalign = bits == 8 ? 4 : 8;
    if (aligned(x, 16) && aligned(q, qalign)) n4 = n / 4;
    if (n4 > 0) {
        const int g = grid_for(n4, 2 * kThreads);
        // rounded reciprocal (see quotient_for_rint); for alpha >= 2^126 it
        // would be subnormal and too coarse, and NaN sends every lane to the
        // division
        const float inv = alpha < 0x1p126f ? 1.0f / alpha : __builtin_nanf("");
        if (bits == 8)
            quantize_act_vec<8><<<g, kThreads, 0, st>>>(reinterpret_cast<const float4*>(x), n4,
                                                        alpha, inv, zp, q);
        else
            quantize_act_vec<16><<<g, kThreads, 0, st>>>(reinterpret_cast<const float4*>(x), n4,
                                                         alpha, inv, zp, q);
    }
    const int64_t begin = n4 * 4;
    if (begin < n) {
        const int g = grid_for(n - begin, kThreads);
        if (bits == 8)
            quantize_act_scalar<8><<<g, kThreads, 0, st>>>(x, begin, n, alpha, zp, q);
        else
            quantize_act_scalar<16><<<g, kThreads, 0, st>>>(x, begin, n, alpha, zp, q);
    }
    return hipGetLastError();
}

hipError_t launch_dequant(const void* q, int32_t bits, int64_t n, float alpha, int32_t zp,
                          float* y, hipStream_t st)
{
    int64_t n4 = 0;
    const uintptr_t qalign = bits == 8 ? 4 : 8;
    if (aligned(y, 16) && aligned(q, qalign)) n4 = n / 4;
    if (n4 > 0) {
        const int g = grid_for(n4, 2 * kThreads);
        if (bits == 8)
            dequant_vec<8><<<g, kThreads, 0, st>>>(q, n4, alpha, zp, reinterpret_cast<float4*>(y));
        else
            dequant_vec<16><<<g, kThreads, 0, st>>>(q, n4, alpha, zp, reinterpret_cast<float4*>(y));
    }
    const int64_t begin = n4 * 4;
    if (begin < n) {
        const int g = grid_for(n - begin, kThreads);
        if (bits == 8)
            dequant_scalar<8><<<g, kThreads, 0, st>>>(q, begin, n, alpha, zp, y);
        else
            dequant_scalar<16><<<g, kThreads, 0, st>>>(q, begin, n, alpha, zp, y);
    }
    return hipGetLastError();
}

hipError_t launch_fold_weights(const float* w, const float* sv, int64_t N, int64_t K, float* out,
                               hipStream_t st)
{
    fold_kernel<false><<<grid_for(N * K, kThreads), kThreads, 0, st>>>(w, sv, N, K, out);
    return hipGetLastError();
}

hipError_t launch_fold_acts(const float* x, const float* sv, int64_t M, int64_t K, float* out,
                            hipStream_t st)
{
    fold_kernel<true><<<grid_for(M * K, kThreads), kThreads, 0, st>>>(x, sv, M, K, out);
    return hipGetLastError();
}

hipError_t launch_pack_weights(const float* w, int64_t N, int64_t K, int32_t bits, void* wq,
                               float* scale, int32_t* colsum, hipStream_t st)
{
    // one block per row; rows beyond the 2^31-1 grid limit are rejected by
    // the host validation
    if (bits == 8)
        pack_weights_kernel<8><<<(unsigned)N, kThreads, 0, st>>>(w, K, wq, scale, colsum);
    else
        pack_weights_kernel<4><<<(unsigned)N, kThreads, 0, st>>>(w, K, wq, scale, colsum);
    return hipGetLastError();
}

template <int BITS>
hipError_t pack_asym_t(const float* w, int64_t N, int64_t K, bool per_tensor, void* wq,
                       float* scale, int32_t* zp, int32_t* colsum, hipStream_t st)
{
    const unsigned g = (unsigned)N;
    if (!per_tensor) {
        pack_weights_asym_kernel<BITS, false><<<g, kThreads, 0, st>>>(w, K, wq, scale, zp, colsum);
        return hipGetLastError();
    }
    // the output arrays hold the per-row ranges between the first two steps
    row_range_kernel<<<g, kThreads, 0, st>>>(w, K, scale, reinterpret_cast<float*>(zp));
    tensor_format_kernel<BITS><<<1, kThreads, 0, st>>>(N, scale, zp);
    pack_weights_asym_kernel<BITS, true><<<g, kThreads, 0, st>>>(w, K, wq, scale, zp, colsum);
    return hipGetLastError();
}

hipError_t launch_pack_weights_asym(const float* w, int64_t N, int64_t K, int32_t bits,
                                    bool per_tensor, void* wq, float* scale, int32_t* zp,
                                    int32_t* colsum, hipStream_t st)
{
    if (bits == 8) return pack_asym_t<8>(w, N, K, per_tensor, wq, scale, zp, colsum, st);
    return pack_asym_t<4>(w, N, K, per_tensor, wq, scale, zp, colsum, st);
}

hipError_t launch_quantize_act_rowsum(const float* x, int64_t M, int64_t K, float alpha,
                                      int32_t zp, int8_t* q, int32_t* rowsum, hipStream_t st)
{
    // one block per row; M <= 2^31 - 1 (host validation)
    if (K % 4 == 0 && aligned(x, 16) && aligned(q, 4)) {
        const float inv = alpha < 0x1p126f ? 1.0f / alpha : __builtin_nanf("");
        quantize_rowsum_vec<<<(unsigned)M, kThreads, 0, st>>>(
            reinterpret_cast<const float4*>(x), K / 4, alpha, inv, zp, q, rowsum);
    } else {
        quantize_rowsum_scalar<<<(unsigned)M, kThreads, 0, st>>>(x, K, alpha, zp, q, rowsum);
    }
    return hipGetLastError();
}

hipError_t launch_act_rowsum(const int8_t* a, int64_t M, int64_t K, int32_t* rowsum,
                             hipStream_t st)
{
    // four rows per block; M <= 2^31 - 1 (host validation) keeps the grid in range
    const int64_t blocks = (M + kThreads / 64 - 1) / (kThreads / 64);
    act_rowsum_kernel<<<(unsigned)blocks, kThreads, 0, st>>>(a, M, K, rowsum);
    return hipGetLastError();
}

}  // namespace mq
