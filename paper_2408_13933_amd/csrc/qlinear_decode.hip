// Decode-shaped qlinear (2 <= M <= 16 tokens; a single token takes the
// vector-ALU GEMV of qlinear_gemv.hip): a weight-streaming GEMV.
//
// Generation is bound by weight traffic (the paper finds autoregressive
// decoding partly memory-bound, Section 5.6, and 4-bit weights help it most,
// appendix).  Each block owns 16 (or 8) output channels; its waves split K and each
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

// R output channels per block (16, or 8 for narrow layers so the weight
// stream spreads over more CUs; rows R..15 of the MFMA then load nothing).
// ASYM: asymmetric weights, the zero-point term is added in the epilogue
// (exact int64 form, four outputs per lane).  A16: 16-bit activation codes,
// each 64-deep step loads 32 bytes of a token row per lane and runs two
// MFMAs on its high and offset-low byte planes (split_a16), combined
// exactly in int64 in the epilogue.
template <int WBITS, int OBITS, int NWAVES, int R, bool ASYM, bool A16>
__global__ __launch_bounds__(NWAVES * 64) void qlinear_decode_kernel(QLinearArgs p)
{
    constexpr int U = 8;  // 64-wide k steps per load round (one round covers most layers)
    constexpr int32_t qmin = -(1 << (OBITS - 1));
    constexpr int32_t qmax = (1 << (OBITS - 1)) - 1;
    constexpr int AB = A16 ? 2 : 1;  // activation bytes per code
    __shared__ v4i red[NWAVES][64 * AB];

    const int lane = threadIdx.x & 63;
    const int wave = __builtin_amdgcn_readfirstlane(threadIdx.x >> 6);  // uniform: scalar loop
    const int r16 = lane & 15;  // weight row in the group / token row
    const int kg = lane >> 4;   // 16-wide k group inside a 64-wide step
    const int64_t n0 = (int64_t)blockIdx.x * R;
    // Buffer descriptors over this block's weight rows and the M token rows:
    // a load past a valid row (channel >= N, token >= M, k >= K, or a step
    // beyond this wave's range) returns zeros without touching memory, so
    // every load is unconditional.
    constexpr uint32_t kOOB = 0x80000000u;
    constexpr int kStreamLoad = 2;  // weights: non-temporal cache policy (read once per call)
    const int64_t wrow_bytes = WBITS == 8 ? p.K : p.K / 2;
    const int rows_w = (int)(p.N - n0 < R ? p.N - n0 : R);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(static_cast<const int8_t*>(p.w) + n0 * wrow_bytes), (short)0,
        (int)(rows_w * wrow_bytes), 0x00020000);
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        (void*)p.a, (short)0, (int)(p.M * p.K * AB), 0x00020000);
    const bool has_a = r16 < p.M;

    // Per-channel inputs of the epilogue (channels n0 + 4*kg + r), loaded by
    // the epilogue wave before the weight stream so both share one memory
    // latency.
    float col_ws[4] = {1.0f, 1.0f, 1.0f, 1.0f}, col_b[4] = {0.0f, 0.0f, 0.0f, 0.0f};
    int32_t col_cs[4] = {0, 0, 0, 0}, col_zw[4] = {0, 0, 0, 0}, row_sum = 0;
    if (wave == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            int64_t n = n0 + 4 * kg + r;
            if (n >= p.N) n = p.N - 1;
            col_ws[r] = p.w_scale[n];
            col_cs[r] = p.colsum[n];
            col_b[r] = (p.bias ? p.bias : p.w_scale)[n];  // branch-free; unused without bias
            if constexpr (ASYM) col_zw[r] = p.w_zp[n];
        }
        if constexpr (ASYM) row_sum = p.a_rowsum[r16 < p.M ? r16 : p.M - 1];
    }

    const int64_t steps = (p.K + 63) / 64;
    const int64_t s_begin = steps * wave / NWAVES;
    const int64_t s_end = steps * (wave + 1) / NWAVES;

    // offsets stay below 2^22 (16 rows of at most 131072 bytes), so setting
    // bit 31 pushes a load out of range without a branch
    const int K32 = (int)p.K;
    const int s_end32 = (int)s_end;
    const uint32_t a_dead = has_a ? 0u : kOOB;
    auto load = [&](int64_t s, v4i* wv, v4i* av, v4i* av2) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            const int su = (int)s + u;
            const int k = su * 64 + kg * 16;
            const uint32_t dead = (uint32_t)((su >= s_end32) | (k >= K32)) << 31;
            if constexpr (WBITS == 8) {
                wv[u] = __builtin_amdgcn_raw_buffer_load_b128(rw, (uint32_t)(r16 * K32 + k) | dead,
                                                              0, kStreamLoad);
            } else {
                // packed nibbles stay packed until the MFMA needs them, so
                // the next load round is issued before this one lands
                typedef unsigned v2u __attribute__((ext_vector_type(2)));
                const v2u pk = __builtin_amdgcn_raw_buffer_load_b64(
                    rw, (uint32_t)(r16 * (K32 / 2) + k / 2) | dead, 0, kStreamLoad);
                wv[u] = v4i{(int)pk[0], (int)pk[1], 0, 0};
            }
            if constexpr (A16) {
                const uint32_t off = (uint32_t)(r16 * K32 + k) * 2;
                av[u] = __builtin_amdgcn_raw_buffer_load_b128(ra, off | dead | a_dead, 0, 0);
                av2[u] = __builtin_amdgcn_raw_buffer_load_b128(ra, (off + 16) | dead | a_dead,
                                                               0, 0);
            } else {
                av[u] = __builtin_amdgcn_raw_buffer_load_b128(
                    ra, (uint32_t)(r16 * K32 + k) | dead | a_dead, 0, 0);
            }
        }
    };
    v4i acc = {0, 0, 0, 0}, acc2 = {0, 0, 0, 0};  // acc2: A16 low-byte plane
    auto mfma = [&](const v4i* wv, const v4i* av, const v4i* av2) {
#pragma unroll
        for (int u = 0; u < U; ++u) {
            v4i w = wv[u];
            if constexpr (WBITS == 4) w = unpack_int4_x16((uint32_t)w[0], (uint32_t)w[1]);
            if constexpr (A16) {
                v4i h, l;
                split_a16(av[u], av2[u], h, l);
                acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(w, h, acc, 0, 0, 0);
                acc2 = __builtin_amdgcn_mfma_i32_16x16x64_i8(w, l, acc2, 0, 0, 0);
            } else {
                acc = __builtin_amdgcn_mfma_i32_16x16x64_i8(w, av[u], acc, 0, 0, 0);
            }
        }
    };
    // The launch picks the wave count so one round covers a wave's K range
    // whenever K <= 16 * 8 * 64; longer rows take several rounds.  Steps
    // past the range load zeros and touch no memory.  The epilogue wave
    // derives its fixed-point constants while the first round is in flight
    // (the per-channel loads were issued before it and return first).
    v4i wv[U], av[U], av2[A16 ? U : 1];
    load(s_begin, wv, av, av2);
    // every use of the per-channel inputs stays behind the weight loads
    asm volatile("" : "+v"(col_ws[0]), "+v"(col_ws[1]), "+v"(col_ws[2]), "+v"(col_ws[3]),
                 "+v"(col_cs[0]), "+v"(col_cs[1]), "+v"(col_cs[2]), "+v"(col_cs[3]),
                 "+v"(col_b[0]), "+v"(col_b[1]), "+v"(col_b[2]), "+v"(col_b[3]));
    if constexpr (ASYM)
        asm volatile("" : "+v"(col_zw[0]), "+v"(col_zw[1]), "+v"(col_zw[2]), "+v"(col_zw[3]),
                     "+v"(row_sum));
    // the fixed-point constants and their integer (mul_hi) form, off the
    // critical path: the weight stream is still in flight
    ColParams cps[4] = {};
    EpiInt eis[4] = {};
    if (wave == 0) {
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            cps[r] = derive_col_params_v(p.a_scale, col_ws[r], p.out_scale, p.bias != nullptr,
                                         col_b[r], col_cs[r], p.a_zp);
            eis[r] = epi_int_params(cps[r]);
        }
    }
    __builtin_amdgcn_sched_barrier(0);
    for (int64_t s = s_begin; s < s_end; s += U) {
        if (s != s_begin) load(s, wv, av, av2);
        mfma(wv, av, av2);
    }

    if constexpr (NWAVES > 1) {
        red[wave][lane] = acc;
        if constexpr (A16) red[wave][64 + lane] = acc2;
        __syncthreads();
        if (wave != 0) return;
#pragma unroll
        for (int w = 1; w < NWAVES; ++w) {
            acc += red[w][lane];
            if constexpr (A16) acc2 += red[w][64 + lane];
        }
    }

    // lane holds acc for token m = r16 and channels n0 + 4*kg + {0,1,2,3}
    const int64_t m = r16;
    if (m >= p.M || 4 * kg >= R) return;
    int32_t out[4];
    const int32_t rs = row_sum - (int32_t)p.K * p.a_zp;  // sum_k (a - a_zp), ASYM only
#pragma unroll
    for (int r = 0; r < 4; ++r) {
        if constexpr (A16) {
            int64_t sum = ((int64_t)acc[r] << 8) + acc2[r];
            if constexpr (WBITS == 4) sum >>= 4;  // exact: a multiple of 16
            const int64_t c = sum + a16_offset(cps[r], p.a_zp, col_cs[r]);
            out[r] = requant_int(sat32(c), 0, eis[r], p.out_zp, qmin, qmax);
            continue;
        }
        int32_t a32 = acc[r];
        if constexpr (WBITS == 4) a32 >>= 4;  // exact: the sum is a multiple of 16
        // the integer form of the requant (requant_int, as the prefill
        // epilogue): one mul_hi, no int64 arithmetic, no branches
        if constexpr (ASYM)
            out[r] = requant_int(corrected_acc_asym(a32, cps[r].off, -col_zw[r], rs), 0, eis[r],
                                 p.out_zp, qmin, qmax);
        else
            out[r] = requant_int(a32, cps[r].off, eis[r], p.out_zp, qmin, qmax);
    }
    const int64_t nb = n0 + 4 * kg;
    const int64_t base = m * p.N + nb;
    if (p.y_f) {
        if (nb + 3 < p.N && (p.N % 4) == 0) {
            *reinterpret_cast<float4*>(p.y_f + base) =
                make_float4(dequant_code(out[0], p.out_scale, p.out_zp),
                            dequant_code(out[1], p.out_scale, p.out_zp),
                            dequant_code(out[2], p.out_scale, p.out_zp),
                            dequant_code(out[3], p.out_scale, p.out_zp));
        } else {
#pragma unroll
            for (int r = 0; r < 4; ++r)
                if (nb + r < p.N) p.y_f[base + r] = dequant_code(out[r], p.out_scale, p.out_zp);
        }
    }
    if (!p.y) return;
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

template <int WBITS, int OBITS, int R, bool ASYM, bool A16>
hipError_t launch_r(const QLinearArgs& p, hipStream_t s)
{
    const int64_t blocks = (p.N + R - 1) / R;
    const int64_t steps = (p.K + 63) / 64;
    // Waves per block: enough that one 8-step load round covers each wave's
    // share of K (every weight byte of the block is requested at once), at
    // least 4 when there are few channel groups so more loads are in flight.
    // 16-bit codes double the activation registers: at most 8 waves (two per
    // SIMD) so they fit without spilling
    constexpr int NWMAX = A16 ? 8 : 16;
    int nw = 1;
    while (nw < NWMAX && nw * 8 < steps) nw *= 2;
    if (blocks < 2048) {
        while (nw < 4 && nw < steps) nw *= 2;
    }
    const dim3 g((unsigned)blocks);
    switch (nw) {
    case 16:
        if constexpr (NWMAX >= 16)
            qlinear_decode_kernel<WBITS, OBITS, 16, R, ASYM, A16><<<g, 16 * 64, 0, s>>>(p);
        break;
    case 8: qlinear_decode_kernel<WBITS, OBITS, 8, R, ASYM, A16><<<g, 8 * 64, 0, s>>>(p); break;
    case 4: qlinear_decode_kernel<WBITS, OBITS, 4, R, ASYM, A16><<<g, 4 * 64, 0, s>>>(p); break;
    case 2: qlinear_decode_kernel<WBITS, OBITS, 2, R, ASYM, A16><<<g, 2 * 64, 0, s>>>(p); break;
    default: qlinear_decode_kernel<WBITS, OBITS, 1, R, ASYM, A16><<<g, 64, 0, s>>>(p); break;
    }
    return hipGetLastError();
}

template <int WBITS, int OBITS, bool ASYM, bool A16>
hipError_t launch_a(const QLinearArgs& p, hipStream_t s)
{
    // narrow layers: 8 channels per block so at least 256 blocks stream
    if ((p.N + 15) / 16 < 256) return launch_r<WBITS, OBITS, 8, ASYM, A16>(p, s);
    return launch_r<WBITS, OBITS, 16, ASYM, A16>(p, s);
}

template <int WBITS, int OBITS>
hipError_t launch_t(const QLinearArgs& p, hipStream_t s)
{
    if (p.a_bits == 16) return launch_a<WBITS, OBITS, false, true>(p, s);
    return p.w_zp ? launch_a<WBITS, OBITS, true, false>(p, s)
                  : launch_a<WBITS, OBITS, false, false>(p, s);
}

}  // namespace

bool decode_supported(const QLinearArgs& p)
{
    const uintptr_t wa = p.w_bits == 8 ? 16 : 8;
    // dense, single products only (no strides, batches, row terms or
    // broadcast scales)
    const bool dense = p.lda == 0 && p.ldw == 0 && p.ldy == 0 && p.batch == 1 &&
                       p.row_off == nullptr && p.ws_stride == 1;
    return dense && p.M <= 16 && p.K % 16 == 0 && ((uintptr_t)p.a % 16) == 0 &&
           ((uintptr_t)p.w % wa) == 0 && ((uintptr_t)p.y % 8) == 0 &&
           ((uintptr_t)p.y_f % 16) == 0 &&
           (p.N + 15) / 16 <= 0x7FFFFFFF;
}

hipError_t launch_qlinear_decode(const QLinearArgs& p, hipStream_t s)
{
    // a single token: the GEMV whose every load lane carries weight bytes
    if (gemv_supported(p)) return launch_qlinear_gemv(p, s);
    if (p.w_bits == 8 && p.out_bits == 8) return launch_t<8, 8>(p, s);
    if (p.w_bits == 8) return launch_t<8, 16>(p, s);
    if (p.out_bits == 8) return launch_t<4, 8>(p, s);
    return launch_t<4, 16>(p, s);
}

}  // namespace mq
