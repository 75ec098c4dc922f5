// Prefill-shaped qlinear: an LDS-tiled int8 MFMA GEMM with the requant
// epilogue fused in registers.
//
// Prompt encoding is compute-bound (Section 5.6) and int8 x int8 is the
// fastest integer product (Section 3.1), so the inner loop is
// v_mfma_i32_16x16x64_i8.  The weight matrix is the MFMA "A" operand (rows =
// output channels) and the activations the "B" operand (columns = tokens):
// every lane then ends with four consecutive output channels of one token,
// which become one 4-byte (int8) or 8-byte (int16) store.
//
// Tiles of both operands are staged through LDS (double buffered, one
// barrier per K tile); rows are padded so the 16-row operand reads hit
// distinct banks.  int4 weights stay packed in LDS (half the bytes) and
// are unpacked into registers right before the MFMA as 16*w, which the
// epilogue removes with an exact shift.  Block ids are remapped so the
// blocks that share weight tiles run on the same XCD (each XCD has its
// own L2).
#include "mq_internal.h"
#include "requant.h"

namespace mq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));

__device__ inline v4i unpack_int4_x16(uint32_t x0, uint32_t x1)
{
    const uint32_t l0 = (x0 << 4) & 0xF0F0F0F0u, h0 = x0 & 0xF0F0F0F0u;
    const uint32_t l1 = (x1 << 4) & 0xF0F0F0F0u, h1 = x1 & 0xF0F0F0F0u;
    v4i r;
    r[0] = (int)__builtin_amdgcn_perm(h0, l0, 0x05010400u);
    r[1] = (int)__builtin_amdgcn_perm(h0, l0, 0x07030602u);
    r[2] = (int)__builtin_amdgcn_perm(h1, l1, 0x05010400u);
    r[3] = (int)__builtin_amdgcn_perm(h1, l1, 0x07030602u);
    return r;
}

template <int WBITS_, int OBITS_, int TN_, int TM_, int WN_, int WM_, int BK_>
struct Cfg {
    static constexpr int WBITS = WBITS_, OBITS = OBITS_;
    static constexpr int TN = TN_, TM = TM_, WN = WN_, WM = WM_, BK = BK_;
    static constexpr int THREADS = 64 * WN * WM;
    static constexpr int FN = TN / (WN * 16);        // 16-row fragments per wave (channels)
    static constexpr int FM = TM / (WM * 16);        // 16-col fragments per wave (tokens)
    static constexpr int BKW = WBITS == 8 ? BK : BK / 2;  // weight bytes per row per stage
    static constexpr int PADW = WBITS == 8 ? 16 : 8;
    static constexpr int LDW = BKW + PADW;           // LDS row stride, weights
    static constexpr int LDA = BK + 16;              // LDS row stride, activations
    static constexpr int W_STAGE = TN * LDW;
    static constexpr int A_STAGE = TM * LDA;
    static constexpr int STAGE = W_STAGE + A_STAGE;
    static constexpr int W_CHUNKS = TN * BKW / 16;   // 16-byte global chunks per stage
    static constexpr int A_CHUNKS = TM * BK / 16;
    static constexpr int W_PER_T = W_CHUNKS / THREADS;
    static constexpr int A_PER_T = A_CHUNKS / THREADS;
    static_assert(W_CHUNKS % THREADS == 0 && A_CHUNKS % THREADS == 0, "staging split");
    static_assert(BK % 64 == 0, "BK is a multiple of the MFMA depth");
    static_assert(FN >= 1 && FM >= 1, "tile too small for the wave grid");
};

template <class C>
__global__ __launch_bounds__(C::THREADS) void qlinear_prefill_kernel(QLinearArgs p, int tiles_n,
                                                                    int tiles_m)
{
    constexpr int32_t qmin = -(1 << (C::OBITS - 1));
    constexpr int32_t qmax = (1 << (C::OBITS - 1)) - 1;
    extern __shared__ __align__(16) int8_t smem[];
    ColParams* params = reinterpret_cast<ColParams*>(smem + 2 * C::STAGE);

    // ---- tile id: blocks that land on one XCD (block id mod 8) get a
    // contiguous run of tiles, so they share weight tiles in that XCD's L2
    const int total = tiles_n * tiles_m;
    int b = blockIdx.x;
    {
        const int per = total / 8, rem = total % 8;
        const int xcd = b % 8, idx = b / 8;
        // xcd x owns tiles [start(x), start(x) + per + (x < rem))
        const int start = xcd * per + (xcd < rem ? xcd : rem);
        b = start + idx;
    }
    const int tn = b / tiles_m;
    const int tm = b % tiles_m;
    const int64_t n_tile = (int64_t)tn * C::TN;
    const int64_t m_tile = (int64_t)tm * C::TM;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = tid >> 6;
    const int wn = wave / C::WM;
    const int wm = wave % C::WM;
    const int r16 = lane & 15;
    const int kg = lane >> 4;

    // ---- per-column requant parameters of this tile
    if (tid < C::TN) {
        int64_t n = n_tile + tid;
        if (n >= p.N) n = p.N - 1;
        params[tid] = derive_col_params(p.a_scale, p.w_scale[n], p.out_scale,
                                        p.bias ? p.bias + n : nullptr, p.colsum[n], p.a_zp);
    }

    const int64_t wrow_bytes = C::WBITS == 8 ? p.K : p.K / 2;
    const int8_t* wbase = static_cast<const int8_t*>(p.w);
    const int KT = (int)((p.K + C::BK - 1) / C::BK);

    // ---- global -> register staging
    v4i wreg[C::W_PER_T], areg[C::A_PER_T];
    auto load_tile = [&](int kt) {
#pragma unroll
        for (int i = 0; i < C::W_PER_T; ++i) {
            const int c = tid + i * C::THREADS;
            const int row = c / (C::BKW / 16), col = c % (C::BKW / 16);
            int64_t n = n_tile + row;
            if (n >= p.N) n = p.N - 1;
            const int64_t kb = (int64_t)kt * C::BKW + col * 16;
            v4i v = {0, 0, 0, 0};
            if (kb < wrow_bytes) v = *reinterpret_cast<const v4i*>(wbase + n * wrow_bytes + kb);
            wreg[i] = v;
        }
#pragma unroll
        for (int i = 0; i < C::A_PER_T; ++i) {
            const int c = tid + i * C::THREADS;
            const int row = c / (C::BK / 16), col = c % (C::BK / 16);
            int64_t m = m_tile + row;
            if (m >= p.M) m = p.M - 1;
            const int64_t kb = (int64_t)kt * C::BK + col * 16;
            v4i v = {0, 0, 0, 0};
            if (kb < p.K) v = *reinterpret_cast<const v4i*>(p.a + m * p.K + kb);
            areg[i] = v;
        }
    };
    auto store_tile = [&](int buf) {
        int8_t* sw = smem + buf * C::STAGE;
        int8_t* sa = sw + C::W_STAGE;
#pragma unroll
        for (int i = 0; i < C::W_PER_T; ++i) {
            const int c = tid + i * C::THREADS;
            const int row = c / (C::BKW / 16), col = c % (C::BKW / 16);
            int8_t* dst = sw + row * C::LDW + col * 16;
            if constexpr (C::WBITS == 8) {
                *reinterpret_cast<v4i*>(dst) = wreg[i];
            } else {
                // 72-byte rows are only 8-byte aligned
                reinterpret_cast<int2*>(dst)[0] = make_int2(wreg[i][0], wreg[i][1]);
                reinterpret_cast<int2*>(dst)[1] = make_int2(wreg[i][2], wreg[i][3]);
            }
        }
#pragma unroll
        for (int i = 0; i < C::A_PER_T; ++i) {
            const int c = tid + i * C::THREADS;
            const int row = c / (C::BK / 16), col = c % (C::BK / 16);
            *reinterpret_cast<v4i*>(sa + row * C::LDA + col * 16) = areg[i];
        }
    };

    v4i acc[C::FN][C::FM];
#pragma unroll
    for (int i = 0; i < C::FN; ++i)
#pragma unroll
        for (int j = 0; j < C::FM; ++j) acc[i][j] = v4i{0, 0, 0, 0};

    load_tile(0);
    store_tile(0);
    __syncthreads();

    for (int kt = 0; kt < KT; ++kt) {
        const int buf = kt & 1;
        if (kt + 1 < KT) load_tile(kt + 1);
        const int8_t* sw = smem + buf * C::STAGE;
        const int8_t* sa = sw + C::W_STAGE;
#pragma unroll
        for (int ks = 0; ks < C::BK / 64; ++ks) {
            v4i wf[C::FN], af[C::FM];
#pragma unroll
            for (int i = 0; i < C::FN; ++i) {
                const int row = wn * (C::TN / C::WN) + i * 16 + r16;
                if constexpr (C::WBITS == 8) {
                    wf[i] = *reinterpret_cast<const v4i*>(sw + row * C::LDW + ks * 64 + kg * 16);
                } else {
                    const uint2 pk =
                        *reinterpret_cast<const uint2*>(sw + row * C::LDW + ks * 32 + kg * 8);
                    wf[i] = unpack_int4_x16(pk.x, pk.y);
                }
            }
#pragma unroll
            for (int j = 0; j < C::FM; ++j) {
                const int row = wm * (C::TM / C::WM) + j * 16 + r16;
                af[j] = *reinterpret_cast<const v4i*>(sa + row * C::LDA + ks * 64 + kg * 16);
            }
#pragma unroll
            for (int i = 0; i < C::FN; ++i)
#pragma unroll
                for (int j = 0; j < C::FM; ++j)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_16x16x64_i8(wf[i], af[j], acc[i][j], 0, 0, 0);
        }
        if (kt + 1 < KT) store_tile(buf ^ 1);
        __syncthreads();
    }

    // ---- epilogue: lane holds channels 4*kg + {0..3} of token r16 in each fragment
#pragma unroll
    for (int i = 0; i < C::FN; ++i) {
        const int nl = wn * (C::TN / C::WN) + i * 16 + 4 * kg;
        const int64_t nb = n_tile + nl;
        ColParams cp[4];
#pragma unroll
        for (int r = 0; r < 4; ++r) cp[r] = params[nl + r];
#pragma unroll
        for (int j = 0; j < C::FM; ++j) {
            const int64_t m = m_tile + wm * (C::TM / C::WM) + j * 16 + r16;
            if (m >= p.M || nb >= p.N) continue;
            int32_t out[4];
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                int32_t a32 = acc[i][j][r];
                if constexpr (C::WBITS == 4) a32 >>= 4;
                out[r] = requant_out(a32, cp[r], p.out_zp, qmin, qmax);
            }
            const int64_t base = m * p.N + nb;
            if (nb + 3 < p.N && (p.N % 4) == 0) {
                if constexpr (C::OBITS == 8) {
                    const uint32_t v = ((uint32_t)out[0] & 0xFFu) |
                                       (((uint32_t)out[1] & 0xFFu) << 8) |
                                       (((uint32_t)out[2] & 0xFFu) << 16) |
                                       ((uint32_t)out[3] << 24);
                    *reinterpret_cast<uint32_t*>(static_cast<int8_t*>(p.y) + base) = v;
                } else {
                    const uint2 v =
                        make_uint2(((uint32_t)out[0] & 0xFFFFu) | ((uint32_t)out[1] << 16),
                                   ((uint32_t)out[2] & 0xFFFFu) | ((uint32_t)out[3] << 16));
                    *reinterpret_cast<uint2*>(static_cast<int16_t*>(p.y) + base) = v;
                }
            } else {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    if (nb + r >= p.N) break;
                    if constexpr (C::OBITS == 8)
                        static_cast<int8_t*>(p.y)[base + r] = (int8_t)out[r];
                    else
                        static_cast<int16_t*>(p.y)[base + r] = (int16_t)out[r];
                }
            }
        }
    }
}

template <class C>
hipError_t launch_cfg(const QLinearArgs& p, hipStream_t s)
{
    const int64_t tiles_n = (p.N + C::TN - 1) / C::TN;
    const int64_t tiles_m = (p.M + C::TM - 1) / C::TM;
    const int64_t total = tiles_n * tiles_m;
    if (total > 0x7FFFFFFF) return hipErrorInvalidValue;
    const size_t lds = 2 * C::STAGE + C::TN * sizeof(ColParams);
    // more than 64 KiB of dynamic LDS must be opted into once per kernel
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&qlinear_prefill_kernel<C>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (attr != hipSuccess) return attr;
    qlinear_prefill_kernel<C><<<dim3((unsigned)total), dim3(C::THREADS), lds, s>>>(
        p, (int)tiles_n, (int)tiles_m);
    return hipGetLastError();
}

template <int WB, int OB>
hipError_t launch_t(const QLinearArgs& p, hipStream_t s)
{
    return launch_cfg<Cfg<WB, OB, 128, 128, 2, 2, 128>>(p, s);
}

}  // namespace

bool prefill_supported(const QLinearArgs& p)
{
    const bool kok = p.w_bits == 8 ? (p.K % 16 == 0) : (p.K % 32 == 0);
    return kok && ((uintptr_t)p.a % 16) == 0 && ((uintptr_t)p.w % 16) == 0 &&
           ((uintptr_t)p.y % 8) == 0;
}

hipError_t launch_qlinear_prefill(const QLinearArgs& p, hipStream_t s)
{
    if (p.w_bits == 8 && p.out_bits == 8) return launch_t<8, 8>(p, s);
    if (p.w_bits == 8) return launch_t<8, 16>(p, s);
    if (p.out_bits == 8) return launch_t<4, 8>(p, s);
    return launch_t<4, 16>(p, s);
}

}  // namespace mq
