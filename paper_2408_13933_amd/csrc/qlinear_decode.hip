// Decode-shaped qlinear (M <= 16 tokens): a weight-streaming GEMV.
//
// Generation is bound by weight traffic (the paper finds autoregressive
// decoding partly memory-bound, Section 5.6, and 4-bit weights help it most,
// appendix).  Each block owns 16 output channels; its waves split K and each
// lane streams 16 weights of one channel per step with a 16-byte (int8) or
// 8-byte (int4) load, so one wave-wide load covers 64 contiguous bytes of 16
// rows.  The 16 x 16 x 64 int8 MFMA multiplies those weights with up to 16
// token rows (rows beyond M are zero), which keeps the math far below the
// memory time for any M <= 16.  Waves combine partial int32 sums in LDS
// (exact) and wave 0 runs the shared requant epilogue.
#include "mq_internal.h"
#include "requant.h"

namespace mq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

// 16 packed int4 weights (8 bytes, two's-complement nibbles, low nibble =
// even k) -> 16 int8 lanes holding 16*w in natural k order.  Scaling by 16
// keeps every value in int8 ([-128, 112]) and is undone exactly by an
// arithmetic shift of the int32 sum.
__device__ inline v4i unpack_int4_x16(uint32_t x0, uint32_t x1)
{
    const uint32_t l0 = (x0 << 4) & 0xF0F0F0F0u, h0 = x0 & 0xF0F0F0F0u;
    const uint32_t l1 = (x1 << 4) & 0xF0F0F0F0u, h1 = x1 & 0xF0F0F0F0u;
    v4i r;
    // v_perm_b32: selector bytes 0-3 pick from the second source, 4-7 from the first
    r[0] = (int)__builtin_amdgcn_perm(h0, l0, 0x05010400u);
    r[1] = (int)__builtin_amdgcn_perm(h0, l0, 0x07030602u);
    r[2] = (int)__builtin_amdgcn_perm(h1, l1, 0x05010400u);
    r[3] = (int)__builtin_amdgcn_perm(h1, l1, 0x07030602u);
    return r;
}

template <int WBITS, int OBITS, int NWAVES>
__global__ __launch_bounds__(NWAVES * 64) void qlinear_decode_kernel(QLinearArgs p)
{
    constexpr int U = 4;  // steps in flight per wave
    constexpr int32_t qmin = -(1 << (OBITS - 1));
    constexpr int32_t qmax = (1 << (OBITS - 1)) - 1;
    __shared__ v4i red[NWAVES][64];

    const int lane = threadIdx.x & 63;
    const int wave = threadIdx.x >> 6;
    const int r16 = lane & 15;  // weight row in the group / token row
    const int kg = lane >> 4;   // 16-wide k group inside a 64-wide step
    const int64_t n0 = (int64_t)blockIdx.x * 16;
    int64_t nrow = n0 + r16;
    if (nrow >= p.N) nrow = p.N - 1;  // duplicate a valid row; never stored
    const bool has_a = r16 < p.M;
    const int8_t* arow = p.a + (has_a ? (int64_t)r16 * p.K : 0);

    const int64_t steps = (p.K + 63) / 64;
    const int64_t s_begin = steps * wave / NWAVES;
    const int64_t s_end = steps * (wave + 1) / NWAVES;

    v4i acc = {0, 0, 0, 0};
    for (int64_t s = s_begin; s < s_end; s += U) {
        v4i wv[U], av[U];
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int64_t k = (s + u) * 64 + kg * 16;
            const bool ok = (s + u < s_end) && (k < p.K);
            v4i w = {0, 0, 0, 0}, a = {0, 0, 0, 0};
            if (ok) {
                if constexpr (WBITS == 8) {
                    w = *reinterpret_cast<const v4i*>(static_cast<const int8_t*>(p.w) +
                                                       nrow * p.K + k);
                } else {
                    const uint2 pk = *reinterpret_cast<const uint2*>(
                        static_cast<const uint8_t*>(p.w) + nrow * (p.K / 2) + k / 2);
                    w = unpack_int4_x16(pk.x, pk.y);
                }
                if (has_a) a = *reinterpret_cast<const v4i*>(arow + k);
            }
            wv[u] = w;
            av[u] = a;
        }
#pragma unroll
        for (int u = 0; u < U; ++u) acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(wv[u], av[u], acc, 0, 0, 0);
    }

    if constexpr (NWAVES > 1) {
        red[wave][lane] = acc;
        __syncthreads();
        if (wave != 0) return;
#pragma unroll
        for (int w = 1; w < NWAVES; ++w) acc += red[w][lane];
    }

    // lane holds acc for token m = r16 and channels n0 + 4*kg + {0,1,2,3}
    const int64_t m = r16;
    if (m >= p.M) return;
    int32_t out[4];
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        int64_t n = n0 + 4 * kg + r;
        if (n >= p.N) n = p.N - 1;
        int32_t a32 = acc[r];
        if constexpr (WBITS == 4) a32 >>= 4;  // exact: the sum is a multiple of 16
        const ColParams cp = derive_col_params(p.a_scale, p.w_scale[n], p.out_scale,
                                               p.bias ? p.bias + n : nullptr, p.colsum[n], p.a_zp);
        out[r] = requant_out(a32, cp, p.out_zp, qmin, qmax);
    }
    const int64_t nb = n0 + 4 * kg;
    const int64_t base = m * p.N + nb;
    if (nb + 3 < p.N && (p.N % 4) == 0) {
        if constexpr (OBITS == 8) {
            const uint32_t v = ((uint32_t)out[0] & 0xFFu) | (((uint32_t)out[1] & 0xFFu) << 8) |
                               (((uint32_t)out[2] & 0xFFu) << 16) | ((uint32_t)out[3] << 24);
            *reinterpret_cast<uint32_t*>(static_cast<int8_t*>(p.y) + base) = v;
        } else {
            const uint2 v = make_uint2(((uint32_t)out[0] & 0xFFFFu) | ((uint32_t)out[1] << 16),
                                       ((uint32_t)out[2] & 0xFFFFu) | ((uint32_t)out[3] << 16));
            *reinterpret_cast<uint2*>(static_cast<int16_t*>(p.y) + base) = v;
        }
    } else {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            if (nb + r >= p.N) break;
            if constexpr (OBITS == 8)
                static_cast<int8_t*>(p.y)[base + r] = (int8_t)out[r];
            else
                static_cast<int16_t*>(p.y)[base + r] = (int16_t)out[r];
        }
    }
}

template <int WBITS, int OBITS>
hipError_t launch_t(const QLinearArgs& p, hipStream_t s)
{
    const int64_t blocks = (p.N + 15) / 16;
    const int64_t steps = (p.K + 63) / 64;
    // enough waves in flight to cover HBM latency: split K further when there
    // are few channel groups
    int nw = blocks >= 2048 ? 4 : (blocks >= 256 ? 8 : 16);
    while (nw > 1 && steps < nw) nw /= 2;
    const dim3 g((unsigned)blocks);
    switch (nw) {
    case 16: qlinear_decode_kernel<WBITS, OBITS, 16><<<g, 16 * 64, 0, s>>>(p); break;
    case 8: qlinear_decode_kernel<WBITS, OBITS, 8><<<g, 8 * 64, 0, s>>>(p); break;
    case 4: qlinear_decode_kernel<WBITS, OBITS, 4><<<g, 4 * 64, 0, s>>>(p); break;
    case 2: qlinear_decode_kernel<WBITS, OBITS, 2><<<g, 2 * 64, 0, s>>>(p); break;
    default: qlinear_decode_kernel<WBITS, OBITS, 1><<<g, 64, 0, s>>>(p); break;
    }
    return hipGetLastError();
}

}  // namespace

bool decode_supported(const QLinearArgs& p)
{
    const uintptr_t wa = p.w_bits == 8 ? 16 : 8;
    return p.M <= 16 && p.K % 16 == 0 && ((uintptr_t)p.a % 16) == 0 &&
           ((uintptr_t)p.w % wa) == 0 && ((uintptr_t)p.y % 8) == 0 &&
           (p.N + 15) / 16 <= 0x7FFFFFFF;
}

hipError_t launch_qlinear_decode(const QLinearArgs& p, hipStream_t s)
{
    if (p.w_bits == 8 && p.out_bits == 8) return launch_t<8, 8>(p, s);
    if (p.w_bits == 8) return launch_t<8, 16>(p, s);
    if (p.out_bits == 8) return launch_t<4, 8>(p, s);
    return launch_t<4, 16>(p, s);
}

}  // namespace mq
