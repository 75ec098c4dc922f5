// Shape- and alignment-agnostic qlinear: one thread per output element,
// byte loads, the shared epilogue.  Slow; it serves ragged K, unaligned
// buffers and as an independent kernel path for cross-checks.
#include <type_traits>

#include "mq_internal.h"
#include "requant.h"

namespace mq {
namespace {

// ABITS = 16: 16-bit activation codes; the sum (|.| < 2^38) is kept in
// int64 and c = sat_int32(sum - a_zp * colsum + bias_q) in int64.
// blockIdx.y: batch index (one product per batch, the weights of batch b
// at b / group); row strides and batch strides as in QLinearArgs.
template <int WBITS, int OBITS, int ABITS>
__global__ __launch_bounds__(256) void qlinear_generic_kernel(QLinearArgs p)
{
    constexpr int32_t qmin = -(1 << (OBITS - 1));
    constexpr int32_t qmax = (1 << (OBITS - 1)) - 1;
    using AT = typename std::conditional<ABITS == 8, int8_t, int16_t>::type;
    using ACC = typename std::conditional<ABITS == 8, int32_t, int64_t>::type;
    const int64_t bt = blockIdx.y;
    const int64_t bg = bt / p.group;
    const int64_t lda = eff_lda(p), ldy = eff_ldy(p);
    const int64_t ldw = WBITS == 8 ? eff_ldw(p) : (p.ldw ? p.ldw : p.K / 2);  // bytes for int4
    const AT* a = reinterpret_cast<const AT*>(p.a) + bt * p.a_bs;
    const int8_t* wb = static_cast<const int8_t*>(p.w) + bg * p.w_bs;
    const int32_t* colsum = p.colsum + bg * p.cs_bs;
    const int64_t* row_off = p.row_off ? p.row_off + bt * p.ro_bs : nullptr;
    const int64_t total = p.M * p.N;
    const int64_t stride = (int64_t)gridDim.x * blockDim.x;
    for (int64_t idx = (int64_t)blockIdx.x * blockDim.x + threadIdx.x; idx < total; idx += stride) {
        const int64_t m = idx / p.N;
        const int64_t n = idx - m * p.N;
        const AT* arow = a + m * lda;
        ACC acc = 0;
        if constexpr (WBITS == 8) {
            const int8_t* wrow = wb + n * ldw;
            for (int64_t k = 0; k < p.K; ++k) acc += (ACC)arow[k] * (ACC)wrow[k];
        } else {
            const uint8_t* wrow = reinterpret_cast<const uint8_t*>(wb) + n * ldw;
            for (int64_t j = 0; j < p.K / 2; ++j) {
                const int32_t b = wrow[j];
                const int32_t lo = (int32_t)((uint32_t)b << 28) >> 28;  // sign-extend nibble
                const int32_t hi = (int32_t)((uint32_t)b << 24) >> 28;
                acc += (ACC)arow[2 * j] * lo + (ACC)arow[2 * j + 1] * hi;
            }
        }
        const ColParams cp =
            derive_col_params(p.a_scale, p.w_scale[n * p.ws_stride], p.out_scale,
                              p.bias ? p.bias + n : nullptr, colsum[n], p.a_zp);
        int32_t y;
        if (ABITS == 16 || row_off) {
            int64_t c = (int64_t)acc - (int64_t)p.a_zp * colsum[n] + cp.bq;
            if (row_off) c += row_off[m];
            y = requant_c(sat32(c), cp, p.out_zp, qmin, qmax);
        } else if (p.w_zp) {
            const int32_t rs = p.a_rowsum[m] - (int32_t)p.K * p.a_zp;
            y = requant_c(corrected_acc_asym((int32_t)acc, cp.off, -p.w_zp[n], rs), cp, p.out_zp,
                          qmin, qmax);
        } else {
            y = requant_out((int32_t)acc, cp, p.out_zp, qmin, qmax);
        }
        const int64_t yi = bt * p.y_bs + m * ldy + n;
        if (p.y) {
            if constexpr (OBITS == 8)
                static_cast<int8_t*>(p.y)[yi] = (int8_t)y;
            else
                static_cast<int16_t*>(p.y)[yi] = (int16_t)y;
        }
        if (p.y_f) p.y_f[m * p.N + n] = dequant_code(y, p.out_scale, p.out_zp);
    }
}

}  // namespace

hipError_t launch_qlinear_generic(const QLinearArgs& p, hipStream_t s)
{
    const int64_t total = p.M * p.N;
    int64_t blocks = (total + 255) / 256;
    if (blocks > 256 * 64) blocks = 256 * 64;
    if (blocks < 1) blocks = 1;
    const dim3 g((unsigned)blocks, (unsigned)p.batch), b(256);
    if (p.a_bits == 16) {
        if (p.w_bits == 8 && p.out_bits == 8) qlinear_generic_kernel<8, 8, 16><<<g, b, 0, s>>>(p);
        else if (p.w_bits == 8) qlinear_generic_kernel<8, 16, 16><<<g, b, 0, s>>>(p);
        else if (p.out_bits == 8) qlinear_generic_kernel<4, 8, 16><<<g, b, 0, s>>>(p);
        else qlinear_generic_kernel<4, 16, 16><<<g, b, 0, s>>>(p);
        return hipGetLastError();
    }
    if (p.w_bits == 8 && p.out_bits == 8) qlinear_generic_kernel<8, 8, 8><<<g, b, 0, s>>>(p);
    else if (p.w_bits == 8) qlinear_generic_kernel<8, 16, 8><<<g, b, 0, s>>>(p);
    else if (p.out_bits == 8) qlinear_generic_kernel<4, 8, 8><<<g, b, 0, s>>>(p);
    else qlinear_generic_kernel<4, 16, 8><<<g, b, 0, s>>>(p);
    return hipGetLastError();
}

}  // namespace mq
