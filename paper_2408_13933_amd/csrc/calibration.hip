// Calibration-side kernels: SmoothQuant's closed-form scaling vector
// (Section 3.2) and the training form of activation range learning
// (Section 4.2, Eq.(2)-(4)) with straight-through gradients.  These run
// offline, before the integer-only deployment; they are HBM-bound
// elementwise/reduction kernels.
#include <cmath>

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

// ---------------------------------------------------------------------------
// Activation range learning.  Forward, every step one fp32 operation:
//   u = rint(x / alpha) - beta,  c = min(max(u, 0), q_max),
//   y = alpha * (c + beta)
// (rint rounds half to even; the straight-through estimator only changes
// the backward pass).  Backward with mask = (0 <= u <= q_max):
//   dx = g * mask
//   dalpha += g * ((c + beta) - mask * x / alpha)     (fp64 terms and sums)
//   dbeta  += g * alpha * (1 - mask)
__device__ inline float arl_u(float x, float alpha, float beta)
{
#pragma clang fp contract(off)
    return rintf(x / alpha) - beta;
}

__device__ inline float arl_y(float x, float alpha, float beta, float q_max)
{
#pragma clang fp contract(off)
    const float c = fminf(fmaxf(arl_u(x, alpha, beta), 0.0f), q_max);
    return alpha * (c + beta);
}

// 16-byte loads and stores for the aligned body (n4 float4s), elements
// [begin, n) one by one
__global__ __launch_bounds__(kThreads) void arl_forward_kernel(const float* __restrict__ x,
                                                               int64_t n4, int64_t begin,
                                                               int64_t n, float alpha,
                                                               float beta, float q_max,
                                                               float* __restrict__ y)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    const int64_t t0 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    const float4* x4 = reinterpret_cast<const float4*>(x);
    float4* y4 = reinterpret_cast<float4*>(y);
    for (int64_t i = t0; i < n4; i += stride) {
        const float4 v = x4[i];
        y4[i] = make_float4(arl_y(v.x, alpha, beta, q_max), arl_y(v.y, alpha, beta, q_max),
                            arl_y(v.z, alpha, beta, q_max), arl_y(v.w, alpha, beta, q_max));
    }
    for (int64_t i = begin + t0; i < n; i += stride) y[i] = arl_y(x[i], alpha, beta, q_max);
}

__global__ __launch_bounds__(kThreads) void arl_backward_kernel(
    const float* __restrict__ x, const float* __restrict__ g, int64_t n, float alpha, float beta,
    float q_max, float* __restrict__ gx, double* __restrict__ partials)
{
#pragma clang fp contract(off)
    __shared__ double red[2][kThreads / 64];
    double ga = 0.0, gb = 0.0;
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        const float xi = x[i], gi = g[i];
        const float t = xi / alpha;
        const float u = rintf(t) - beta;
        const float c = fminf(fmaxf(u, 0.0f), q_max);
        const bool in = u >= 0.0f && u <= q_max;
        gx[i] = in ? gi : 0.0f;
        const double da = (double)c + (double)beta - (in ? (double)t : 0.0);
        const double db = in ? 0.0 : (double)alpha;
        ga += (double)gi * da;
        gb += (double)gi * db;
    }
    for (int o = 32; o > 0; o >>= 1) {
        ga += __shfl_xor(ga, o);
        gb += __shfl_xor(gb, o);
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) {
        red[0][wave] = ga;
        red[1][wave] = gb;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double a = 0.0, b = 0.0;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) {
            a += red[0][w];
            b += red[1][w];
        }
        partials[2 * blockIdx.x] = a;
        partials[2 * blockIdx.x + 1] = b;
    }
}

// The per-block partial sums: thread t adds partials t, t + 256, ... in
// order, then a fixed tree over the threads; the order depends on nblocks
// only, so a given n always sums the same way.
__global__ __launch_bounds__(kThreads) void arl_reduce_kernel(const double* __restrict__ partials,
                                                              int nblocks,
                                                              double* __restrict__ out)
{
    __shared__ double red[2][kThreads / 64];
    double a = 0.0, b = 0.0;
    for (int i = threadIdx.x; i < nblocks; i += kThreads) {
        a += partials[2 * i];
        b += partials[2 * i + 1];
    }
    for (int o = 32; o > 0; o >>= 1) {
        a += __shfl_xor(a, o);
        b += __shfl_xor(b, o);
    }
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    if (lane == 0) {
        red[0][wave] = a;
        red[1][wave] = b;
    }
    __syncthreads();
    if (threadIdx.x == 0) {
        double sa = 0.0, sb = 0.0;
#pragma unroll
        for (int w = 0; w < kThreads / 64; ++w) {
            sa += red[0][w];
            sb += red[1][w];
        }
        out[0] = sa;
        out[1] = sb;
    }
}

// ---------------------------------------------------------------------------
// SmoothQuant scales.  Column maxima of |v| over finite entries, as float
// bit patterns (non-negative floats order like their bits, so an unsigned
// atomic max keeps the largest); one block covers 256 columns of a chunk
// of rows.
__global__ __launch_bounds__(kThreads) void fill_u32_kernel(uint32_t* __restrict__ p, int64_t n,
                                                            uint32_t v)
{
    const int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (i < n) p[i] = v;
}

__device__ inline float absmax_finite(float m, float v)
{
    const float a = fabsf(v);
    return __builtin_isfinite(a) && a > m ? a : m;
}

// A block covers 64 * COLS columns (COLS = 4: 16-byte loads, K % 4 == 0 and
// an aligned base) and a chunk of rows; its four waves take every fourth
// row, eight rows per trip in flight, meet in LDS, and wave 0 folds the
// block's maxima into `out` with one atomic per column.
template <int COLS>
__global__ __launch_bounds__(kThreads) void col_absmax_kernel(const float* __restrict__ v,
                                                              int64_t rows, int64_t K,
                                                              int64_t rows_per_block,
                                                              uint32_t* __restrict__ out)
{
    __shared__ float red[kThreads / 64][64 * COLS];
    const int lane = threadIdx.x & 63, wave = threadIdx.x >> 6;
    const int64_t col = ((int64_t)blockIdx.x * 64 + lane) * COLS;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_block;
    const int64_t r1 = r0 + rows_per_block < rows ? r0 + rows_per_block : rows;
    constexpr int NW = kThreads / 64;
    float m[COLS] = {};
    if (col < K) {
        int64_t r = r0 + wave;
        for (; r + 7 * NW < r1; r += 8 * NW) {
            if constexpr (COLS == 4) {
                float4 t[8];
#pragma unroll
                for (int u = 0; u < 8; ++u)
                    t[u] = *reinterpret_cast<const float4*>(v + (r + u * NW) * K + col);
#pragma unroll
                for (int u = 0; u < 8; ++u) {
                    m[0] = absmax_finite(m[0], t[u].x);
                    m[1] = absmax_finite(m[1], t[u].y);
                    m[2] = absmax_finite(m[2], t[u].z);
                    m[3] = absmax_finite(m[3], t[u].w);
                }
            } else {
                float t[8];
#pragma unroll
                for (int u = 0; u < 8; ++u) t[u] = v[(r + u * NW) * K + col];
#pragma unroll
                for (int u = 0; u < 8; ++u) m[0] = absmax_finite(m[0], t[u]);
            }
        }
        for (; r < r1; r += NW)
#pragma unroll
            for (int c = 0; c < COLS; ++c) m[c] = absmax_finite(m[c], v[r * K + col + c]);
    }
#pragma unroll
    for (int c = 0; c < COLS; ++c) red[wave][lane * COLS + c] = m[c];
    __syncthreads();
    if (wave == 0 && col < K) {
#pragma unroll
        for (int c = 0; c < COLS; ++c) {
            float b = red[0][lane * COLS + c];
#pragma unroll
            for (int w = 1; w < NW; ++w) b = fmaxf(b, red[w][lane * COLS + c]);
            if (b > 0.0f) atomicMax(out + col + c, __float_as_uint(b));
        }
    }
}

// s_k = max|X_k|^a / max|W_k|^(1-a) in fp64, rounded once to fp32; 1 for a
// channel whose activation or weight maximum is 0.
__global__ __launch_bounds__(kThreads) void smooth_combine_kernel(const float* __restrict__ mx,
                                                                  const float* __restrict__ mw,
                                                                  int64_t K, float a,
                                                                  float* __restrict__ s)
{
    const int64_t k = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (k >= K) return;
    const float x = mx[k], w = mw[k];
    s[k] = (x > 0.0f && w > 0.0f) ? (float)(pow((double)x, (double)a) /
                                            pow((double)w, 1.0 - (double)a))
                                  : 1.0f;
}

}  // namespace

hipError_t launch_arl_forward(const float* x, int64_t n, float alpha, float beta, int32_t bits,
                              float* y, hipStream_t st)
{
    const float q_max = (float)((1 << bits) - 1);
    const bool vec = ((uintptr_t)x % 16) == 0 && ((uintptr_t)y % 16) == 0;
    const int64_t n4 = vec ? n / 4 : 0;
    arl_forward_kernel<<<grid_for(vec ? n4 : n, kThreads, 256 * 64), kThreads, 0, st>>>(
        x, n4, n4 * 4, n, alpha, beta, q_max, y);
    return hipGetLastError();
}

hipError_t launch_arl_backward(const float* x, const float* g, int64_t n, float alpha, float beta,
                               int32_t bits, float* gx, double* grads, int32_t max_partials,
                               hipStream_t st)
{
    const float q_max = (float)((1 << bits) - 1);
    const int blocks = grid_for(n, kThreads * 4, max_partials);
    double* partials = grads + 2;
    arl_backward_kernel<<<blocks, kThreads, 0, st>>>(x, g, n, alpha, beta, q_max, gx, partials);
    arl_reduce_kernel<<<1, kThreads, 0, st>>>(partials, blocks, grads);
    return hipGetLastError();
}

hipError_t launch_smooth_scales(const float* x, int64_t M, int64_t K, const float* w, int64_t N,
                                float a, float* x_absmax, float* w_absmax, float* s,
                                hipStream_t st)
{
    const unsigned gk = (unsigned)((K + kThreads - 1) / kThreads);
    fill_u32_kernel<<<gk, kThreads, 0, st>>>(reinterpret_cast<uint32_t*>(x_absmax), K, 0u);
    fill_u32_kernel<<<gk, kThreads, 0, st>>>(reinterpret_cast<uint32_t*>(w_absmax), K, 0u);
    // 64 rows per block (so each column takes rows / 64 atomics), more when
    // the grid's y limit of 65535 row blocks needs it
    auto colmax = [&](const float* v, int64_t rows, float* out) {
        const bool vec = K % 4 == 0 && ((uintptr_t)v % 16) == 0;
        const int64_t gx = vec ? (K / 4 + 63) / 64 : (K + 63) / 64;
        int64_t rpb = 64;
        if ((rows + rpb - 1) / rpb > 65535) rpb = (rows + 65534) / 65535;
        const dim3 grid((unsigned)gx, (unsigned)((rows + rpb - 1) / rpb));
        uint32_t* o = reinterpret_cast<uint32_t*>(out);
        if (vec) col_absmax_kernel<4><<<grid, kThreads, 0, st>>>(v, rows, K, rpb, o);
        else col_absmax_kernel<1><<<grid, kThreads, 0, st>>>(v, rows, K, rpb, o);
    };
    if (M > 0) colmax(x, M, x_absmax);
    if (N > 0) colmax(w, N, w_absmax);
    smooth_combine_kernel<<<gk, kThreads, 0, st>>>(x_absmax, w_absmax, K, a, s);
    return hipGetLastError();
}

}  // namespace mq
