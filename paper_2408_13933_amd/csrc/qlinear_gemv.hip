// One-token qlinear (M = 1, a generation step): a weight-streaming GEMV on
// the vector ALU.
//
// Generation is bound by weight traffic (Section 5.6; 4-bit weights help it
// most, appendix).  The MFMA decode kernel multiplies up to 16 token rows at
// once; with a single token 15 of its 16 operand columns are zero, yet
// every wave still issues an activation load per weight load.  Here the
// block stages the token's K activation codes in LDS once, and every lane of
// every weight load carries useful bytes: a block owns 8 output channels,
// and in each wave load 8 lanes read 128 contiguous bytes of one weight row
// (16 per lane: 16 int8 or 32 packed int4 weights).  Products are
// v_dot4_i32_i8 (int4 weights unpacked to 16*w in registers, removed by an
// exact shift of the sum), summed over the channel's 8 lanes with lane
// shuffles and over the waves in LDS; wave 0 runs the requant epilogue.
#include "mq_internal.h"
#include "requant.h"

namespace mq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

constexpr uint32_t kOOB = 0x80000000u;  // any offset past num_records reads zero
// cache policy of the weight loads: non-temporal (each weight byte is read
// once per call).  Measured on MI355X for the 1 x 2048 x 256000 LM head:
// 86.6 -> 78.1 us cold, and 112 -> 80 us after a layer that left 524 MB of
// dirty outputs in the Infinity Cache (the stream no longer evicts them).
constexpr int kStreamLoad = 2;
constexpr int kCPB = 8;                 // output channels per block
constexpr int kLPC = 64 / kCPB;         // lanes per channel in a wave load
constexpr int kU = 4;                   // steps (wave loads) in flight per round

// 16 packed int4 weights (8 bytes, two's-complement nibbles, low nibble =
// even k) -> 16 int8 lanes holding 16*w in k order.
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

// LDS: the K activation codes, then the per-wave channel sums.
__host__ __device__ constexpr int64_t gemv_lds_bytes(int64_t K, int nw)
{
    return K + (int64_t)nw * kCPB * 4;
}

template <int WBITS, int OBITS, int NW, bool ASYM>
__global__ __launch_bounds__(NW * 64) void qlinear_gemv_kernel(QLinearArgs p)
{
    constexpr int32_t qmin = -(1 << (OBITS - 1));
    constexpr int32_t qmax = (1 << (OBITS - 1)) - 1;
    extern __shared__ __align__(16) int8_t smem[];
    const int K32 = (int)p.K;
    int32_t* red = reinterpret_cast<int32_t*>(smem + K32);  // [NW][kCPB]
    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keep it scalar
    const int c = lane / kLPC;  // channel of this lane's weight bytes
    const int j = lane % kLPC;  // its 16-byte chunk among the channel's kLPC
    const int64_t n0 = (int64_t)blockIdx.x * kCPB;
    const int wrow = WBITS == 8 ? K32 : K32 / 2;  // bytes per weight row
    const int rows_w = (int)(p.N - n0 < kCPB ? p.N - n0 : kCPB);
    // descriptor over this block's weight rows: channels past N read zeros
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(static_cast<const int8_t*>(p.w) + n0 * wrow), (short)0, rows_w * wrow,
        0x00020000);
    const __amdgpu_buffer_rsrc_t ra =
        __builtin_amdgcn_make_buffer_rsrc((void*)p.a, (short)0, K32, 0x00020000);

    // Per-channel inputs of the epilogue (lanes 0..7 of wave 0, one channel
    // each), issued before the weight stream so both share one latency.
    const bool epi = wave == 0 && lane < kCPB;
    float col_ws = 1.0f, col_b = 0.0f;
    int32_t col_cs = 0, col_zw = 0, row_sum = 0;
    if (epi) {
        int64_t n = n0 + lane;
        if (n >= p.N) n = p.N - 1;
        col_ws = p.w_scale[n];
        col_cs = p.colsum[n];
        col_b = (p.bias ? p.bias : p.w_scale)[p.bias ? n : 0];  // branch-free
        if constexpr (ASYM) {
            col_zw = p.w_zp[n];
            row_sum = p.a_rowsum[0];
        }
    }

    // The row's 16-byte chunks in steps of kLPC (one wave load covers 128
    // bytes of each of the 8 rows); waves split the steps.
    const int steps = (wrow + kLPC * 16 - 1) / (kLPC * 16);
    const int s_begin = steps * wave / NW;
    const int s_end = steps * (wave + 1) / NW;
    v4i wv[kU];
    auto load = [&](int s) {
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int su = s + u;
            const int off = (su * kLPC + j) * 16;
            // steps past the wave's range and chunks past the row read zeros
            const uint32_t dead = (uint32_t)((su >= s_end) | (off >= wrow)) << 31;
            wv[u] = __builtin_amdgcn_raw_buffer_load_b128(rw, (uint32_t)(c * wrow + off) | dead, 0,
                                                          kStreamLoad);
        }
    };
    load(s_begin);
    // the token's activation codes into LDS, 16 bytes per lane
    for (int i = tid; i < K32 / 16; i += NW * 64) {
        const v4i v = __builtin_amdgcn_raw_buffer_load_b128(ra, (uint32_t)(i * 16), 0, 0);
        *reinterpret_cast<v4i*>(smem + i * 16) = v;
    }
    // every use of the per-channel inputs stays behind the weight loads
    asm volatile("" : "+v"(col_ws), "+v"(col_cs), "+v"(col_b));
    if constexpr (ASYM) asm volatile("" : "+v"(col_zw), "+v"(row_sum));
    ColParams cp = {};
    EpiInt ei = {};
    if (epi) {
        cp = derive_col_params_v(p.a_scale, col_ws, p.out_scale, p.bias != nullptr, col_b,
                                 col_cs, p.a_zp);
        ei = epi_int_params(cp);  // the integer (mul_hi) form of the requant
    }
    __syncthreads();

    // |acc| <= K * 128 * 128 = K * 2^14 <= 2^30 (K <= 65536; int4 as 16*w
    // stays within [-128, 112]): the int32 sums are exact
    int32_t acc = 0;
    for (int s = s_begin; s < s_end; s += kU) {
        if (s != s_begin) load(s);
#pragma unroll
        for (int u = 0; u < kU; ++u) {
            const int off = ((s + u) * kLPC + j) * 16;  // byte in the weight row
            if constexpr (WBITS == 8) {
                const int kk = off < wrow ? off : 0;  // dead chunks hold zeros
                const v4i a = *reinterpret_cast<const v4i*>(smem + kk);
#pragma unroll
                for (int q = 0; q < 4; ++q) acc = __builtin_amdgcn_sdot4(wv[u][q], a[q], acc, false);
            } else {
                const int kk = off < wrow ? 2 * off : 0;
                const v4i w0 = unpack_int4_x16((uint32_t)wv[u][0], (uint32_t)wv[u][1]);
                const v4i w1 = unpack_int4_x16((uint32_t)wv[u][2], (uint32_t)wv[u][3]);
                const v4i a0 = *reinterpret_cast<const v4i*>(smem + kk);
                const v4i a1 = *reinterpret_cast<const v4i*>(smem + kk + 16);
#pragma unroll
                for (int q = 0; q < 4; ++q) acc = __builtin_amdgcn_sdot4(w0[q], a0[q], acc, false);
#pragma unroll
                for (int q = 0; q < 4; ++q) acc = __builtin_amdgcn_sdot4(w1[q], a1[q], acc, false);
            }
        }
    }
    // the channel's kLPC lanes (aligned groups of 8), then the waves
    acc += __shfl_xor(acc, 1);
    acc += __shfl_xor(acc, 2);
    acc += __shfl_xor(acc, 4);
    if (j == 0) red[wave * kCPB + c] = acc;
    __syncthreads();
    if (!epi || n0 + lane >= p.N) return;
    int32_t sum = 0;
#pragma unroll
    for (int w = 0; w < NW; ++w) sum += red[w * kCPB + lane];
    if constexpr (WBITS == 4) sum >>= 4;  // exact: the sum is a multiple of 16
    int32_t y;
    if constexpr (ASYM)
        y = requant_int(corrected_acc_asym(sum, cp.off, -col_zw, row_sum - K32 * p.a_zp), 0, ei,
                        p.out_zp, qmin, qmax);
    else
        y = requant_int(sum, cp.off, ei, p.out_zp, qmin, qmax);
    if (p.y) {
        if constexpr (OBITS == 8)
            static_cast<int8_t*>(p.y)[n0 + lane] = (int8_t)y;
        else
            static_cast<int16_t*>(p.y)[n0 + lane] = (int16_t)y;
    }
    if (p.y_f) p.y_f[n0 + lane] = dequant_code(y, p.out_scale, p.out_zp);
}

template <int WBITS, int OBITS, int NW, bool ASYM>
hipError_t launch_nw(const QLinearArgs& p, hipStream_t s)
{
    const int64_t lds = gemv_lds_bytes(p.K, NW);
    // more than 64 KiB of dynamic LDS (K > 65536 - 256) must be opted into
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&qlinear_gemv_kernel<WBITS, OBITS, NW, ASYM>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)gemv_lds_bytes(65536, NW));
    if (attr != hipSuccess) return attr;
    const dim3 g((unsigned)((p.N + kCPB - 1) / kCPB));
    qlinear_gemv_kernel<WBITS, OBITS, NW, ASYM><<<g, NW * 64, (size_t)lds, s>>>(p);
    return hipGetLastError();
}

template <int WBITS, int OBITS, bool ASYM>
hipError_t launch_a(const QLinearArgs& p, hipStream_t s)
{
    // Waves: enough that one round of kU loads covers each wave's share of
    // the row (all of the block's weight bytes requested at once), at most
    // eight (longer rows take several rounds).  Measured on MI355X, cold
    // weights: 1 x 5632 x 2048 int4 4.2 us on eight waves (the MFMA decode
    // kernel: 6.3), 1 x 2048 x 2048 int8 3.6 us on four (3.9).
    const int64_t wrow = p.w_bits == 8 ? p.K : p.K / 2;
    const int64_t steps = (wrow + kLPC * 16 - 1) / (kLPC * 16);
    int nw = 1;
    while (nw < 8 && nw * kU < steps) nw *= 2;
    switch (nw) {
    case 8: return launch_nw<WBITS, OBITS, 8, ASYM>(p, s);
    case 4: return launch_nw<WBITS, OBITS, 4, ASYM>(p, s);
    case 2: return launch_nw<WBITS, OBITS, 2, ASYM>(p, s);
    default: return launch_nw<WBITS, OBITS, 1, ASYM>(p, s);
    }
}

template <int WBITS, int OBITS>
hipError_t launch_t(const QLinearArgs& p, hipStream_t s)
{
    return p.w_zp ? launch_a<WBITS, OBITS, true>(p, s) : launch_a<WBITS, OBITS, false>(p, s);
}

}  // namespace

bool gemv_supported(const QLinearArgs& p)
{
    // one token of 8-bit codes, dense; whole 16-byte chunks per weight row
    // (packed int4 rows too), so no chunk spans two rows; the codes fit LDS
    const bool dense = p.lda == 0 && p.ldw == 0 && p.ldy == 0 && p.batch == 1 &&
                       p.row_off == nullptr && p.ws_stride == 1;
    const bool kok = p.w_bits == 8 ? (p.K % 16 == 0) : (p.K % 32 == 0);
    return dense && p.M == 1 && p.a_bits == 8 && kok && p.K <= 65536 &&
           ((uintptr_t)p.a % 16) == 0 && ((uintptr_t)p.w % 16) == 0 &&
           (p.N + kCPB - 1) / kCPB <= 0x7FFFFFFF;
}

hipError_t launch_qlinear_gemv(const QLinearArgs& p, hipStream_t s)
{
    if (p.w_bits == 8 && p.out_bits == 8) return launch_t<8, 8>(p, s);
    if (p.w_bits == 8) return launch_t<8, 16>(p, s);
    if (p.out_bits == 8) return launch_t<4, 8>(p, s);
    return launch_t<4, 16>(p, s);
}

}  // namespace mq
