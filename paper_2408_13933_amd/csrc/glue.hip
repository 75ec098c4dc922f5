// Decoder-block glue on 16-bit integer activations: the operators between
// the quantized linear layers keep 16-bit integer activations (Section 4.1,
// Section 5.1).  Each kernel dequantizes exactly (an fp32 scale times an
// integer of at most 17 bits is exact in fp64), evaluates the operator in
// fp64 one IEEE operation at a time in a fixed order, and requantizes with
// the Eq.(4) quantizer (rint half to even, clamp).  Residual add and
// RMSNorm therefore give the same bits as any IEEE evaluation of the same
// sequence; SiLU and softmax go through exp, whose last bit IEEE does not
// fix.
#include <cmath>
#include <type_traits>

#include "mq_internal.h"

namespace mq {
namespace {

constexpr int kThreads = 256;

inline int grid_for(int64_t items, int per_block, int cap)
{
    int64_t g = (items + per_block - 1) / per_block;
    if (g < 1) g = 1;
    if (g > cap) g = cap;
    return (int)g;
}

template <int BITS>
__device__ inline int32_t requant_f64(double v, double ay, int32_t zy)
{
#pragma clang fp contract(off)
    constexpr int32_t qmin = -(1 << (BITS - 1)), qmax = (1 << (BITS - 1)) - 1;
    double t = v / ay;
    if (!(t == t)) t = -1e300;  // NaN -> the low end
    t = fmin(fmax(t, -1e18), 1e18);
    const int64_t q = (int64_t)rint(t) + zy;
    return (int32_t)(q < qmin ? qmin : (q > qmax ? qmax : q));
}

template <int BITS>
__device__ inline void store_code(void* y, int64_t i, int32_t v)
{
    if constexpr (BITS == 8) static_cast<int8_t*>(y)[i] = (int8_t)v;
    else static_cast<int16_t*>(y)[i] = (int16_t)v;
}

// ---------------------------------------------------------------------------
// Residual add: v = alpha_1 (x1 - zp_1) + alpha_2 (x2 - zp_2), requantized.
template <int BITS>
__global__ __launch_bounds__(kThreads) void add_requant_kernel(
    const int16_t* __restrict__ x1, float a1, int32_t z1, const int16_t* __restrict__ x2,
    float a2, int32_t z2, int64_t n, float ay, int32_t zy, void* __restrict__ y)
{
#pragma clang fp contract(off)
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        const double v = (double)a1 * (double)((int32_t)x1[i] - z1) +
                         (double)a2 * (double)((int32_t)x2[i] - z2);
        store_code<BITS>(y, i, requant_f64<BITS>(v, (double)ay, zy));
    }
}

// ---------------------------------------------------------------------------
// Tables of elementwise operators on int16 codes: entry i + 32768 holds the
// requantized f(alpha_x (i - zp_x)).  op 1: SiLU, v / (1 + exp(-v)).
template <int BITS>
__global__ __launch_bounds__(kThreads) void lut_build_kernel(int32_t op, float ax, int32_t zx,
                                                             float ay, int32_t zy,
                                                             void* __restrict__ lut)
{
#pragma clang fp contract(off)
    const int32_t idx = blockIdx.x * kThreads + threadIdx.x;  // 0 .. 65535
    const double v = (double)ax * (double)(idx - 32768 - zx);
    const double f = op == 1 ? v / (1.0 + exp(-v)) : v;
    store_code<BITS>(lut, idx, requant_f64<BITS>(f, (double)ay, zy));
}

// y[i] = lut[x[i] + 32768]; the table stays in the L1/L2 caches.
template <int BITS>
__global__ __launch_bounds__(kThreads) void lut_apply_kernel(const int16_t* __restrict__ x,
                                                             int64_t n,
                                                             const void* __restrict__ lut,
                                                             void* __restrict__ y)
{
    using T = typename std::conditional<BITS == 8, int8_t, int16_t>::type;
    const T* t = static_cast<const T*>(lut);
    T* out = static_cast<T*>(y);
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride)
        out[i] = t[(int32_t)x[i] + 32768];
}

// ---------------------------------------------------------------------------
// Row reductions: one block per row.
__device__ inline int64_t block_sum_i64(int64_t v, int64_t* red)
{
    for (int o = 32; o > 0; o >>= 1) v += __shfl_xor(v, o);
    if ((threadIdx.x & 63) == 0) red[threadIdx.x >> 6] = v;
    __syncthreads();
    int64_t t = 0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) t += red[w];
    __syncthreads();
    return t;
}

// RMSNorm: ss = sum (x - zp_x)^2 (exact, int64); ms = alpha^2 ss / K + eps;
// r = sqrt(ms); v = alpha (x - zp_x) [* gamma_k] / r.
template <int BITS>
__global__ __launch_bounds__(kThreads) void rmsnorm_kernel(const int16_t* __restrict__ x,
                                                           int64_t K, float ax, int32_t zx,
                                                           const float* __restrict__ gamma,
                                                           float eps, float ay, int32_t zy,
                                                           void* __restrict__ y)
{
#pragma clang fp contract(off)
    __shared__ int64_t red[kThreads / 64];
    const int64_t m = blockIdx.x;
    const int16_t* row = x + m * K;
    int64_t ss = 0;
    for (int64_t k = threadIdx.x; k < K; k += kThreads) {
        const int64_t d = (int64_t)row[k] - zx;
        ss += d * d;
    }
    ss = block_sum_i64(ss, red);
    const double a = (double)ax;
    const double ms = a * a * (double)ss / (double)K + (double)eps;
    const double r = sqrt(ms);
    for (int64_t k = threadIdx.x; k < K; k += kThreads) {
        double v = a * (double)((int64_t)row[k] - zx);
        if (gamma) v = v * (double)gamma[k];
        v = v / r;
        store_code<BITS>(y, m * K + k, requant_f64<BITS>(v, (double)ay, zy));
    }
}

// Softmax: e_k = exp(alpha (x_k - max_j x_j)), p_k = e_k / sum_j e_j.
template <int BITS>
__global__ __launch_bounds__(kThreads) void softmax_kernel(const int16_t* __restrict__ x,
                                                           int64_t K, float ax, float ay,
                                                           int32_t zy, void* __restrict__ y)
{
#pragma clang fp contract(off)
    __shared__ int32_t red_i[kThreads / 64];
    __shared__ double red_d[kThreads / 64];
    const int64_t m = blockIdx.x;
    const int16_t* row = x + m * K;
    int32_t mx = -32768;
    for (int64_t k = threadIdx.x; k < K; k += kThreads) mx = max(mx, (int32_t)row[k]);
    for (int o = 32; o > 0; o >>= 1) mx = max(mx, __shfl_xor(mx, o));
    if ((threadIdx.x & 63) == 0) red_i[threadIdx.x >> 6] = mx;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) mx = max(mx, red_i[w]);
    const double a = (double)ax;
    double sum = 0.0;
    for (int64_t k = threadIdx.x; k < K; k += kThreads)
        sum += exp(a * (double)((int32_t)row[k] - mx));
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if ((threadIdx.x & 63) == 0) red_d[threadIdx.x >> 6] = sum;
    __syncthreads();
    sum = 0.0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) sum += red_d[w];
    for (int64_t k = threadIdx.x; k < K; k += kThreads) {
        const double e = exp(a * (double)((int32_t)row[k] - mx));
        store_code<BITS>(y, m * K + k, requant_f64<BITS>(e / sum, (double)ay, zy));
    }
}

}  // namespace

hipError_t launch_add_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                              float a2, int32_t z2, int64_t n, float ay, int32_t zy,
                              int32_t bits, void* y, hipStream_t st)
{
    const int g = grid_for(n, kThreads * 4, 256 * 64);
    if (bits == 8)
        add_requant_kernel<8><<<g, kThreads, 0, st>>>(x1, a1, z1, x2, a2, z2, n, ay, zy, y);
    else
        add_requant_kernel<16><<<g, kThreads, 0, st>>>(x1, a1, z1, x2, a2, z2, n, ay, zy, y);
    return hipGetLastError();
}

hipError_t launch_lut_build(int32_t op, float ax, int32_t zx, float ay, int32_t zy, int32_t bits,
                            void* lut, hipStream_t st)
{
    if (bits == 8) lut_build_kernel<8><<<65536 / kThreads, kThreads, 0, st>>>(op, ax, zx, ay, zy, lut);
    else lut_build_kernel<16><<<65536 / kThreads, kThreads, 0, st>>>(op, ax, zx, ay, zy, lut);
    return hipGetLastError();
}

hipError_t launch_lut_apply(const int16_t* x, int64_t n, const void* lut, int32_t bits, void* y,
                            hipStream_t st)
{
    const int g = grid_for(n, kThreads * 4, 256 * 64);
    if (bits == 8) lut_apply_kernel<8><<<g, kThreads, 0, st>>>(x, n, lut, y);
    else lut_apply_kernel<16><<<g, kThreads, 0, st>>>(x, n, lut, y);
    return hipGetLastError();
}

hipError_t launch_rmsnorm(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                          const float* gamma, float eps, float ay, int32_t zy, int32_t bits,
                          void* y, hipStream_t st)
{
    if (bits == 8)
        rmsnorm_kernel<8><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, zx, gamma, eps, ay, zy, y);
    else
        rmsnorm_kernel<16><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, zx, gamma, eps, ay, zy, y);
    return hipGetLastError();
}

hipError_t launch_softmax(const int16_t* x, int64_t M, int64_t K, float ax, float ay, int32_t zy,
                          int32_t bits, void* y, hipStream_t st)
{
    if (bits == 8) softmax_kernel<8><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, ay, zy, y);
    else softmax_kernel<16><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, ay, zy, y);
    return hipGetLastError();
}

}  // namespace mq
