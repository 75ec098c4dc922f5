// Helpers of the batched attention matmuls (Section 5.6: in the W8A16
// setting the self-attention products multiply 16-bit by 8-bit activation
// codes): the zero-point sums of both operands and the transpose of the
// value codes into the [group][head dim][token] operand layout.
#include "mq_internal.h"

namespace mq {
namespace {

// One wave per row: rows [0, H*M) are rows of A (int16), rows [H*M,
// H*M + G*N) rows of B (int8).  A rows give the term of B's zero-point,
// -b_zp * sum_k (A[k] - a_zp) (int64, exact); B rows give sum_k B[k].
__global__ __launch_bounds__(256) void attn_sums_kernel(const int16_t* a, int64_t lda, int64_t a_bs,
                                                        int64_t rows_a, int64_t M,
                                                        const int8_t* b, int64_t ldb, int64_t b_bs,
                                                        int64_t rows_b, int64_t N, int64_t K,
                                                        int32_t a_zp, int32_t b_zp, float b_scale,
                                                        int64_t* row_off, int32_t* colsum,
                                                        float* scale_out)
{
    const int lane = threadIdx.x & 63;
    if (blockIdx.x == 0 && threadIdx.x == 0) *scale_out = b_scale;
    const int64_t row = (int64_t)blockIdx.x * 4 + (threadIdx.x >> 6);
    if (row >= rows_a + rows_b) return;
    int64_t s = 0;
    if (row < rows_a) {
        const int16_t* x = a + (row / M) * a_bs + (row % M) * lda;
        for (int64_t k = lane; k < K; k += 64) s += x[k];
    } else {
        const int64_t r = row - rows_a;
        const int8_t* x = b + (r / N) * b_bs + (r % N) * ldb;
        for (int64_t k = lane; k < K; k += 64) s += x[k];
    }
#pragma unroll
    for (int o = 32; o > 0; o >>= 1) s += __shfl_xor(s, o, 64);
    if (lane != 0) return;
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
                            int64_t* row_off, int32_t* colsum, float* scale_out, hipStream_t s)
{
    const int64_t rows_a = (int64_t)H * M, rows_b = (int64_t)G * N;
    const int64_t blocks = (rows_a + rows_b + 3) / 4;
    if (blocks == 0) return hipSuccess;
    if (blocks > 0x7FFFFFFF) return hipErrorInvalidValue;
    attn_sums_kernel<<<dim3((unsigned)blocks), dim3(256), 0, s>>>(
        a, lda, a_bs, rows_a, M, b, ldb, b_bs, rows_b, N, K, a_zp, b_zp, b_scale, row_off, colsum,
        scale_out);
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
