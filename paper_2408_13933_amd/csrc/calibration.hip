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

__global__ __launch_bounds__(kThreads) void arl_forward_kernel(const float* __restrict__ x,
                                                               int64_t n, float alpha,
                                                               float beta, float q_max,
                                                               float* __restrict__ y)
{
#pragma clang fp contract(off)
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    for (int64_t i = (int64_t)blockIdx.x * kThreads + threadIdx.x; i < n; i += stride) {
        const float c = fminf(fmaxf(arl_u(x[i], alpha, beta), 0.0f), q_max);
        y[i] = alpha * (c + beta);
    }
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

// The per-block partial sums in block order (deterministic for a given n).
__global__ __launch_bounds__(64) void arl_reduce_kernel(const double* __restrict__ partials,
                                                        int nblocks, double* __restrict__ out)
{
    if (threadIdx.x != 0) return;
    double a = 0.0, b = 0.0;
    for (int i = 0; i < nblocks; ++i) {
        a += partials[2 * i];
        b += partials[2 * i + 1];
    }
    out[0] = a;
    out[1] = b;
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

__global__ __launch_bounds__(kThreads) void col_absmax_kernel(const float* __restrict__ v,
                                                              int64_t rows, int64_t K,
                                                              int64_t rows_per_block,
                                                              uint32_t* __restrict__ out)
{
    const int64_t col = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    if (col >= K) return;
    const int64_t r0 = (int64_t)blockIdx.y * rows_per_block;
    const int64_t r1 = r0 + rows_per_block < rows ? r0 + rows_per_block : rows;
    float m = 0.0f;
    for (int64_t r = r0; r < r1; ++r) {
        const float a = fabsf(v[r * K + col]);
        if (__builtin_isfinite(a) && a > m) m = a;
    }
    if (m > 0.0f) atomicMax(out + col, __float_as_uint(m));
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
    arl_forward_kernel<<<grid_for(n, kThreads, 256 * 64), kThreads, 0, st>>>(x, n, alpha, beta,
                                                                             q_max, y);
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
    arl_reduce_kernel<<<1, 64, 0, st>>>(partials, blocks, grads);
    return hipGetLastError();
}

hipError_t launch_smooth_scales(const float* x, int64_t M, int64_t K, const float* w, int64_t N,
                                float a, float* x_absmax, float* w_absmax, float* s,
                                hipStream_t st)
{
    const unsigned gk = (unsigned)((K + kThreads - 1) / kThreads);
    fill_u32_kernel<<<gk, kThreads, 0, st>>>(reinterpret_cast<uint32_t*>(x_absmax), K, 0u);
    fill_u32_kernel<<<gk, kThreads, 0, st>>>(reinterpret_cast<uint32_t*>(w_absmax), K, 0u);
    // at least 64 rows per block, and at most 65535 row blocks (grid y limit)
    auto colmax = [&](const float* v, int64_t rows, float* out) {
        int64_t rpb = 64;
        if ((rows + rpb - 1) / rpb > 65535) rpb = (rows + 65534) / 65535;
        const unsigned gy = (unsigned)((rows + rpb - 1) / rpb);
        col_absmax_kernel<<<dim3(gk, gy), kThreads, 0, st>>>(v, rows, K, rpb,
                                                            reinterpret_cast<uint32_t*>(out));
    };
    if (M > 0) colmax(x, M, x_absmax);
    if (N > 0) colmax(w, N, w_absmax);
    smooth_combine_kernel<<<gk, kThreads, 0, st>>>(x_absmax, w_absmax, K, a, s);
    return hipGetLastError();
}

}  // namespace mq
