// Helpers of the batched attention matmuls (Section 5.6: in the W8A16
// setting the self-attention products multiply 16-bit by 8-bit activation
// codes): the zero-point sums of both operands and the transpose of the
// value codes into the [group][head dim][token] operand layout.
#include "mq_internal.h"

namespace mq {
namespace {

// Partial sum, for lane li of the LPR lanes that share one row, of the K
// codes starting at x: 16-byte loads when `vec` (x 16-byte aligned), else
// element loads; the LPR partial sums are reduced by the caller.
template <class T>
__device__ inline int64_t row_sum_part(const T* x, int64_t K, int li, int lpr, bool vec)
{
    constexpr int PER = 16 / sizeof(T);  // codes per 16-byte load
    int64_t s = 0;
    int64_t k0 = 0;
    if (vec) {
        const int64_t step = (int64_t)lpr * PER;
        const int64_t full = K / step * step;
        for (int64_t k = (int64_t)li * PER; k < full; k += step) {
            const int4 v = *reinterpret_cast<const int4*>(x + k);
            const T* e = reinterpret_cast<const T*>(&v);
            int32_t t = 0;
#pragma unroll
            for (int i = 0; i < PER; ++i) t += e[i];
            s += t;
        }
        k0 = full;
    }
    for (int64_t k = k0 + li; k < K; k += lpr) s += x[k];
    return s;
}

// LPR lanes (a power of two, at most 64) per row: rows [0, rows_a) are rows
// of A (int16; none when B's zero-point is 0), rows [rows_a, rows_a +
// rows_b) rows of B (int8), each B row once per block of tile_m rows of A
// ([group][m block][n]).  A rows give the term of B's zero-point,
// -b_zp * sum_k (A[k] - a_zp) (int64, exact); B rows give sum_k B[k] over
// k < K, or, with causal activations (in_causal >= 0), over the K range the
// tiled kernel reads for that m block: up to the tile_k stage holding the
// block's last row's boundary.
__global__ __launch_bounds__(256) void attn_sums_kernel(const int16_t* a, int64_t lda, int64_t a_bs,
                                                        int64_t rows_a, int64_t M,
                                                        const int8_t* b, int64_t ldb, int64_t b_bs,
                                                        int64_t rows_b, int64_t N, int64_t K,
                                                        int32_t a_zp, int32_t b_zp, float b_scale,
                                                        int64_t* row_off, int32_t* colsum,
                                                        float* scale_out, bool vec_a, bool vec_b,
                                                        int64_t n_mb, int64_t in_causal,
                                                        int64_t tile_m, int64_t tile_k, int lpr)
{
    const int li = threadIdx.x & (lpr - 1);
    if (blockIdx.x == 0 && threadIdx.x == 0) *scale_out = b_scale;
    const int64_t row = (int64_t)blockIdx.x * (256 / lpr) + threadIdx.x / lpr;
    // rows past the end still take part in the reduction (all lanes of a
    // group reach the shuffles) with a zero sum
    const bool live = row < rows_a + rows_b;
    // row indices below 2^32 (the host's check) divide in 32 bits
    int64_t s = 0;
    if (live && row < rows_a) {
        const uint32_t h = (uint32_t)row / (uint32_t)M, m = (uint32_t)row - h * (uint32_t)M;
        s = row_sum_part(a + (int64_t)h * a_bs + (int64_t)m * lda, K, li, lpr, vec_a);
    } else if (live) {
        const uint32_t r = (uint32_t)(row - rows_a);  // (g * n_mb + mb) * N + n
        const uint32_t q = r / (uint32_t)N, n = r - q * (uint32_t)N;
        const uint32_t g = q / (uint32_t)n_mb, mb = q - g * (uint32_t)n_mb;
        int64_t len = K;
        if (in_causal >= 0) {
            const int64_t m_end = (mb + 1) * tile_m < M ? (mb + 1) * tile_m : M;
            const int64_t need = (m_end + in_causal + tile_k - 1) / tile_k * tile_k;
            if (need < len) len = need;
        }
        s = row_sum_part(b + g * b_bs + n * ldb, len, li, lpr, vec_b);
    }
    for (int o = lpr / 2; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (li != 0 || !live) return;
    if (row < rows_a)
        row_off[row] = -(int64_t)b_zp * (s - K * (int64_t)a_zp);
    else
        colsum[row - rows_a] = (int32_t)s;  // |s| <= 128 K <= 2^23
}

// y[c][r] = x[r][c] through a 64 x 64 LDS tile (row pitch 65 bytes keeps
// the column reads on distinct banks).
__global__ __launch_bounds__(256) void transpose_i8_kernel(const int8_t* x, int64_t rows,
                                                           int64_t cols, int64_t ldx, int8_t* y)
{
    __shared__ int8_t t[64][65];
    const int64_t r0 = (int64_t)blockIdx.y * 64, c0 = (int64_t)blockIdx.x * 64;
    const int tx = threadIdx.x & 63, ty = threadIdx.x >> 6;
    for (int i = ty; i < 64; i += 4) {
        const int64_t r = r0 + i, c = c0 + tx;
        t[i][tx] = (r < rows && c < cols) ? x[r * ldx + c] : 0;
    }
    __syncthreads();
    for (int i = ty; i < 64; i += 4) {
        const int64_t c = c0 + i, r = r0 + tx;
        if (c < cols && r < rows) y[c * rows + r] = t[tx][i];
    }
}

}  // namespace

hipError_t launch_attn_sums(const int16_t* a, int64_t lda, int64_t a_bs, int32_t H, int64_t M,
                            const int8_t* b, int64_t ldb, int64_t b_bs, int32_t G, int64_t N,
                            int64_t K, int32_t a_zp, int32_t b_zp, float b_scale,
                            int64_t* row_off, int32_t* colsum, float* scale_out,
                            int64_t in_causal, int64_t tile_m, int64_t tile_k, hipStream_t s)
{
    // B's zero-point 0: the row terms vanish and A is not read
    const int64_t n_mb = in_causal >= 0 ? (M + tile_m - 1) / tile_m : 1;
    const int64_t rows_a = b_zp != 0 ? (int64_t)H * M : 0, rows_b = (int64_t)G * n_mb * N;
    // lanes per row: enough 16-byte loads of int16 codes to cover K once
    int lpr = 1;
    while (lpr < 64 && (int64_t)lpr * 8 < K) lpr *= 2;
    const int64_t rpb = 256 / lpr;
    const int64_t blocks = (rows_a + rows_b + rpb - 1) / rpb;
    if (blocks == 0) return hipSuccess;
    if (rows_a + rows_b >= ((int64_t)1 << 32) || M >= ((int64_t)1 << 32) ||
        N >= ((int64_t)1 << 32))
        return hipErrorInvalidValue;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    const bool vec_a = (uintptr_t)a % 16 == 0 && (lda * 2) % 16 == 0 && (a_bs * 2) % 16 == 0;
    const bool vec_b = (uintptr_t)b % 16 == 0 && ldb % 16 == 0 && b_bs % 16 == 0;
    attn_sums_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(
        a, lda, a_bs, rows_a, M, b, ldb, b_bs, rows_b, N, K, a_zp, b_zp, b_scale, row_off, colsum,
        scale_out, vec_a, vec_b, n_mb, in_causal, tile_m, tile_k, lpr);
    return hipGetLastError();
}

hipError_t launch_transpose_i8(const int8_t* x, int64_t rows, int64_t cols, int64_t ldx,
                               int8_t* y, hipStream_t s)
{
    if (rows == 0 || cols == 0) return hipSuccess;
    const int64_t gx = (cols + 63) / 64, gy = (rows + 63) / 64;
    if (gx > 0x7FFFFFFF || gy > 65535) return hipErrorInvalidValue;
    transpose_i8_kernel<<<dim3((unsigned)gx, (unsigned)gy), dim3(256), 0, s>>>(x, rows, cols, ldx,
                                                                              y);
    return hipGetLastError();
}

}  // namespace mq
