// Bandwidth-bound kernels around the integer linear layer: the static
// activation quantizer (Section 4.2, Eq.(4)), its inverse, the fold of the
// smoothing vector (Section 3.2, Eq.(1)) and the per-channel weight packer.
//
// All of them stream HBM: 16-byte vector loads, grid-stride loops sized to
// the 256 CUs, and scalar code only for ragged tails and unaligned buffers.
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
    // enough blocks for every CU several times over; the loops stride
    if (b > 256 * 16) b = 256 * 16;
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

// 8 elements per thread per step: two float4 loads, one 8- or 16-byte store.
template <int BITS>
__global__ __launch_bounds__(kThreads) void quantize_act_vec(const float4* __restrict__ x,
                                                             int64_t groups, float alpha,
                                                             int32_t zp, void* __restrict__ q)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < groups; g += stride) {
        const float4 a = x[2 * g];
        const float4 b = x[2 * g + 1];
        int32_t v[8] = {quant1<BITS>(a.x, alpha, zp), quant1<BITS>(a.y, alpha, zp),
                        quant1<BITS>(a.z, alpha, zp), quant1<BITS>(a.w, alpha, zp),
                        quant1<BITS>(b.x, alpha, zp), quant1<BITS>(b.y, alpha, zp),
                        quant1<BITS>(b.z, alpha, zp), quant1<BITS>(b.w, alpha, zp)};
        if constexpr (BITS == 8) {
            uint32_t lo = 0, hi = 0;
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                lo |= ((uint32_t)v[i] & 0xFFu) << (8 * i);
                hi |= ((uint32_t)v[4 + i] & 0xFFu) << (8 * i);
            }
            reinterpret_cast<uint2*>(q)[g] = make_uint2(lo, hi);
        } else {
            uint32_t w[4];
#pragma unroll
            for (int i = 0; i < 4; ++i)
                w[i] = ((uint32_t)v[2 * i] & 0xFFFFu) | (((uint32_t)v[2 * i + 1] & 0xFFFFu) << 16);
            reinterpret_cast<uint4*>(q)[g] = make_uint4(w[0], w[1], w[2], w[3]);
        }
    }
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

template <int BITS>
__device__ inline float deq1(int32_t q, float alpha, int32_t zp)
{
#pragma clang fp contract(off)
    return alpha * (float)(q - zp);
}

template <int BITS>
__global__ __launch_bounds__(kThreads) void dequant_vec(const void* __restrict__ q, int64_t groups,
                                                        float alpha, int32_t zp,
                                                        float4* __restrict__ y)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t g = (int64_t)blockIdx.x * kThreads + threadIdx.x; g < groups; g += stride) {
        int32_t v[8];
        if constexpr (BITS == 8) {
            const uint2 p = reinterpret_cast<const uint2*>(q)[g];
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[i] = (int32_t)(int8_t)(p.x >> (8 * i));
                v[4 + i] = (int32_t)(int8_t)(p.y >> (8 * i));
            }
        } else {
            const uint4 p = reinterpret_cast<const uint4*>(q)[g];
            const uint32_t w[4] = {p.x, p.y, p.z, p.w};
#pragma unroll
            for (int i = 0; i < 4; ++i) {
                v[2 * i] = (int32_t)(int16_t)(w[i] & 0xFFFFu);
                v[2 * i + 1] = (int32_t)(int16_t)(w[i] >> 16);
            }
        }
        y[2 * g] = make_float4(deq1<BITS>(v[0], alpha, zp), deq1<BITS>(v[1], alpha, zp),
                               deq1<BITS>(v[2], alpha, zp), deq1<BITS>(v[3], alpha, zp));
        y[2 * g + 1] = make_float4(deq1<BITS>(v[4], alpha, zp), deq1<BITS>(v[5], alpha, zp),
                                   deq1<BITS>(v[6], alpha, zp), deq1<BITS>(v[7], alpha, zp));
    }
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

}  // namespace

hipError_t launch_quantize_act(const float* x, int64_t n, float alpha, int32_t zp, int32_t bits,
                               void* q, hipStream_t st)
{
    int64_t vec_groups = 0;
    const uintptr_t qalign = bits == 8 ? 8 : 16;
    if (aligned(x, 16) && aligned(q, qalign)) vec_groups = n / 8;
    if (vec_groups > 0) {
        const int g = grid_for(vec_groups, kThreads);
        if (bits == 8)
            quantize_act_vec<8><<<g, kThreads, 0, st>>>(reinterpret_cast<const float4*>(x),
                                                        vec_groups, alpha, zp, q);
        else
            quantize_act_vec<16><<<g, kThreads, 0, st>>>(reinterpret_cast<const float4*>(x),
                                                         vec_groups, alpha, zp, q);
    }
    const int64_t begin = vec_groups * 8;
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
    int64_t vec_groups = 0;
    const uintptr_t qalign = bits == 8 ? 8 : 16;
    if (aligned(y, 16) && aligned(q, qalign)) vec_groups = n / 8;
    if (vec_groups > 0) {
        const int g = grid_for(vec_groups, kThreads);
        if (bits == 8)
            dequant_vec<8><<<g, kThreads, 0, st>>>(q, vec_groups, alpha, zp,
                                                   reinterpret_cast<float4*>(y));
        else
            dequant_vec<16><<<g, kThreads, 0, st>>>(q, vec_groups, alpha, zp,
                                                    reinterpret_cast<float4*>(y));
    }
    const int64_t begin = vec_groups * 8;
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

}  // namespace mq
