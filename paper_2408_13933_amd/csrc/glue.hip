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

// requant_f64 with the division by ay replaced by a product with its
// reciprocal ri (one extra rounding)
template <int BITS>
__device__ inline int32_t requant_mul(double v, double ri, int32_t zy)
{
#pragma clang fp contract(off)
    constexpr int32_t qmin = -(1 << (BITS - 1)), qmax = (1 << (BITS - 1)) - 1;
    double t = v * ri;
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
__device__ inline int32_t add_one(int32_t u, int32_t v, float a1, int32_t z1, float a2,
                                  int32_t z2, float ay, int32_t zy)
{
#pragma clang fp contract(off)
    const double s = (double)a1 * (double)(u - z1) + (double)a2 * (double)(v - z2);
    return requant_f64<BITS>(s, (double)ay, zy);
}

// Product of the two dequantized codes (each factor exact in fp64, the
// product one rounding): the gated unit SiLU(gate) * up.
template <int BITS>
__device__ inline int32_t mul_one(int32_t u, int32_t v, float a1, int32_t z1, float a2,
                                  int32_t z2, float ay, int32_t zy)
{
#pragma clang fp contract(off)
    const double f1 = (double)a1 * (double)(u - z1);
    const double f2 = (double)a2 * (double)(v - z2);
    return requant_f64<BITS>(f1 * f2, (double)ay, zy);
}

template <int BITS, int OP>
__device__ inline int32_t binary_one(int32_t u, int32_t v, float a1, int32_t z1, float a2,
                                     int32_t z2, float ay, int32_t zy)
{
    if constexpr (OP == 0) return add_one<BITS>(u, v, a1, z1, a2, z2, ay, zy);
    else return mul_one<BITS>(u, v, a1, z1, a2, z2, ay, zy);
}

// n4 groups of four codes through 8-byte loads (aligned buffers), the
// codes [begin, n) one by one
// OP 0: sum, OP 1: product of the dequantized codes.
template <int BITS, int OP>
__global__ __launch_bounds__(kThreads) void add_requant_kernel(
    const int16_t* __restrict__ x1, float a1, int32_t z1, const int16_t* __restrict__ x2,
    float a2, int32_t z2, int64_t n4, int64_t begin, int64_t n, float ay, int32_t zy,
    void* __restrict__ y)
{
    const int64_t stride = (int64_t)gridDim.x * kThreads;
    const int64_t t0 = (int64_t)blockIdx.x * kThreads + threadIdx.x;
    for (int64_t i = t0; i < n4; i += stride) {
        const short4 u = reinterpret_cast<const short4*>(x1)[i];
        const short4 v = reinterpret_cast<const short4*>(x2)[i];
        const int32_t r0 = binary_one<BITS, OP>(u.x, v.x, a1, z1, a2, z2, ay, zy);
        const int32_t r1 = binary_one<BITS, OP>(u.y, v.y, a1, z1, a2, z2, ay, zy);
        const int32_t r2 = binary_one<BITS, OP>(u.z, v.z, a1, z1, a2, z2, ay, zy);
        const int32_t r3 = binary_one<BITS, OP>(u.w, v.w, a1, z1, a2, z2, ay, zy);
        if constexpr (BITS == 8)
            reinterpret_cast<char4*>(y)[i] = make_char4((char)r0, (char)r1, (char)r2, (char)r3);
        else
            reinterpret_cast<short4*>(y)[i] =
                make_short4((short)r0, (short)r1, (short)r2, (short)r3);
    }
    for (int64_t i = begin + t0; i < n; i += stride)
        store_code<BITS>(y, i, binary_one<BITS, OP>(x1[i], x2[i], a1, z1, a2, z2, ay, zy));
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

// y[i] = lut[x[i] + 32768].  The table (64 or 128 KiB) is copied into LDS
// once per block, and each block then streams many codes: 8 per thread
// per trip through 16-byte loads when the buffers are aligned.
constexpr int kLutThreads = 1024;

template <int BITS>
__global__ __launch_bounds__(kLutThreads) void lut_apply_kernel(const int16_t* __restrict__ x,
                                                                int64_t n8, int64_t begin,
                                                                int64_t n,
                                                                const void* __restrict__ lut,
                                                                void* __restrict__ y)
{
    using T = typename std::conditional<BITS == 8, int8_t, int16_t>::type;
    extern __shared__ __align__(16) int8_t lds_table[];
    T* tab = reinterpret_cast<T*>(lds_table);
    {
        const int4* src = static_cast<const int4*>(lut);
        int4* dst = reinterpret_cast<int4*>(lds_table);
        constexpr int chunks = 65536 * sizeof(T) / 16;
        for (int i = threadIdx.x; i < chunks; i += kLutThreads) dst[i] = src[i];
    }
    __syncthreads();
    T* out = static_cast<T*>(y);
    const int64_t stride = (int64_t)gridDim.x * kLutThreads;
    const int64_t t0 = (int64_t)blockIdx.x * kLutThreads + threadIdx.x;
    for (int64_t i = t0; i < n8; i += stride) {
        const int4 v = reinterpret_cast<const int4*>(x)[i];
        const int16_t* c = reinterpret_cast<const int16_t*>(&v);
        T r[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) r[u] = tab[(int32_t)c[u] + 32768];
        if constexpr (BITS == 8) {
            uint2 o;
            o.x = ((uint32_t)(uint8_t)r[0]) | ((uint32_t)(uint8_t)r[1] << 8) |
                  ((uint32_t)(uint8_t)r[2] << 16) | ((uint32_t)(uint8_t)r[3] << 24);
            o.y = ((uint32_t)(uint8_t)r[4]) | ((uint32_t)(uint8_t)r[5] << 8) |
                  ((uint32_t)(uint8_t)r[6] << 16) | ((uint32_t)(uint8_t)r[7] << 24);
            reinterpret_cast<uint2*>(out)[i] = o;
        } else {
            int4 o;
            o.x = (int)(((uint32_t)(uint16_t)r[0]) | ((uint32_t)(uint16_t)r[1] << 16));
            o.y = (int)(((uint32_t)(uint16_t)r[2]) | ((uint32_t)(uint16_t)r[3] << 16));
            o.z = (int)(((uint32_t)(uint16_t)r[4]) | ((uint32_t)(uint16_t)r[5] << 16));
            o.w = (int)(((uint32_t)(uint16_t)r[6]) | ((uint32_t)(uint16_t)r[7] << 16));
            reinterpret_cast<int4*>(out)[i] = o;
        }
    }
    for (int64_t i = begin + t0; i < n; i += stride) out[i] = tab[(int32_t)x[i] + 32768];
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

// Rows of at most 8 * 256 * NCH codes with K % 8 == 0 and 16-byte aligned
// rows stay in registers: chunk c of thread t holds codes
// 8 (t + 256 c) .. +7, read once with a 16-byte load.
// Eight codes to y[i .. i+7] with one 8-byte (int8) or 16-byte (int16)
// store; i is a multiple of 8 and y is 16-byte aligned.
template <int BITS>
__device__ inline void store8(void* y, int64_t i, const int32_t* q)
{
    if constexpr (BITS == 8) {
        uint2 o;
        o.x = ((uint32_t)(uint8_t)q[0]) | ((uint32_t)(uint8_t)q[1] << 8) |
              ((uint32_t)(uint8_t)q[2] << 16) | ((uint32_t)(uint8_t)q[3] << 24);
        o.y = ((uint32_t)(uint8_t)q[4]) | ((uint32_t)(uint8_t)q[5] << 8) |
              ((uint32_t)(uint8_t)q[6] << 16) | ((uint32_t)(uint8_t)q[7] << 24);
        *reinterpret_cast<uint2*>(static_cast<int8_t*>(y) + i) = o;
    } else {
        int4 o;
        o.x = (int)(((uint32_t)(uint16_t)q[0]) | ((uint32_t)(uint16_t)q[1] << 16));
        o.y = (int)(((uint32_t)(uint16_t)q[2]) | ((uint32_t)(uint16_t)q[3] << 16));
        o.z = (int)(((uint32_t)(uint16_t)q[4]) | ((uint32_t)(uint16_t)q[5] << 16));
        o.w = (int)(((uint32_t)(uint16_t)q[6]) | ((uint32_t)(uint16_t)q[7] << 16));
        *reinterpret_cast<int4*>(static_cast<int16_t*>(y) + i) = o;
    }
}

// Table lookup fused with the product of two dequantized codes: the gated
// unit SiLU(gate) * up without the SiLU codes going through memory.
// u = lut[x1 + 32768] (LB-bit entries in format (a1, z1)), then the product
// of mul_one with x2: the same two steps as mq_lut_apply and
// mq_mul_requant, so the same bits.
template <int LB, int OB>
__global__ __launch_bounds__(kLutThreads) void lut_mul_kernel(
    const int16_t* __restrict__ x1, const void* __restrict__ lut, float a1, int32_t z1,
    const int16_t* __restrict__ x2, float a2, int32_t z2, int64_t n8, int64_t begin, int64_t n,
    float ay, int32_t zy, void* __restrict__ y)
{
    using T = typename std::conditional<LB == 8, int8_t, int16_t>::type;
    extern __shared__ __align__(16) int8_t lds_table[];
    const T* tab = reinterpret_cast<const T*>(lds_table);
    {
        const int4* src = static_cast<const int4*>(lut);
        int4* dst = reinterpret_cast<int4*>(lds_table);
        constexpr int chunks = 65536 * sizeof(T) / 16;
        for (int i = threadIdx.x; i < chunks; i += kLutThreads) dst[i] = src[i];
    }
    __syncthreads();
    const int64_t stride = (int64_t)gridDim.x * kLutThreads;
    const int64_t t0 = (int64_t)blockIdx.x * kLutThreads + threadIdx.x;
    for (int64_t i = t0; i < n8; i += stride) {
        const int4 g = reinterpret_cast<const int4*>(x1)[i];
        const int4 v = reinterpret_cast<const int4*>(x2)[i];
        const int16_t* gc = reinterpret_cast<const int16_t*>(&g);
        const int16_t* vc = reinterpret_cast<const int16_t*>(&v);
        int32_t q[8];
#pragma unroll
        for (int u = 0; u < 8; ++u)
            q[u] = mul_one<OB>(tab[(int32_t)gc[u] + 32768], vc[u], a1, z1, a2, z2, ay, zy);
        store8<OB>(y, 8 * i, q);
    }
    for (int64_t i = begin + t0; i < n; i += stride)
        store_code<OB>(y, i, mul_one<OB>(tab[(int32_t)x1[i] + 32768], x2[i], a1, z1, a2, z2, ay,
                                         zy));
}

template <int NCH>
struct RowRegs {
    int16_t v[NCH][8];
    bool live[NCH];
    __device__ void load(const int16_t* row, int64_t K)
    {
#pragma unroll
        for (int c = 0; c < NCH; ++c) {
            const int64_t k0 = 8 * ((int64_t)threadIdx.x + kThreads * c);
            live[c] = k0 < K;
            int4 q = {0, 0, 0, 0};
            if (live[c]) q = *reinterpret_cast<const int4*>(row + k0);
            const int16_t* e = reinterpret_cast<const int16_t*>(&q);
#pragma unroll
            for (int u = 0; u < 8; ++u) v[c][u] = e[u];
        }
    }
};

template <int BITS, int NCH>
__global__ __launch_bounds__(kThreads) void rmsnorm_regs_kernel(const int16_t* __restrict__ x,
                                                                int64_t K, float ax, int32_t zx,
                                                                const float* __restrict__ gamma,
                                                                float eps, float ay, int32_t zy,
                                                                void* __restrict__ y)
{
#pragma clang fp contract(off)
    __shared__ int64_t red[kThreads / 64];
    const int64_t m = blockIdx.x;
    RowRegs<NCH> r;
    r.load(x + m * K, K);
    int64_t ss = 0;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        if (r.live[c])
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                const int64_t d = (int64_t)r.v[c][u] - zx;
                ss += d * d;
            }
    ss = block_sum_i64(ss, red);
    const double a = (double)ax;
    const double ms = a * a * (double)ss / (double)K + (double)eps;
    const double rt = sqrt(ms);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!r.live[c]) continue;
        const int64_t k0 = 8 * ((int64_t)threadIdx.x + kThreads * c);
        int32_t q[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            double v = a * (double)((int64_t)r.v[c][u] - zx);
            if (gamma) v = v * (double)gamma[k0 + u];
            v = v / rt;
            q[u] = requant_f64<BITS>(v, (double)ay, zy);
        }
        store8<BITS>(y, m * K + k0, q);
    }
}

// Residual add fused with the RMSNorm that reads its result: per row, the
// sum codes h = code_h(a1 (x1 - z1) + a2 (x2 - z2)) (add_one) are written
// and, still in registers, normalized as rmsnorm_regs_kernel normalizes its
// input.  The same operations as mq_add_requant then mq_rmsnorm, so the
// same bits, with one read of h less and one launch less.
template <int BITS, int NCH>
__global__ __launch_bounds__(kThreads) void add_rmsnorm_kernel(
    const int16_t* __restrict__ x1, float a1, int32_t z1, const int16_t* __restrict__ x2,
    float a2, int32_t z2, int64_t K, float ah, int32_t zh, int16_t* __restrict__ h,
    const float* __restrict__ gamma, float eps, float ay, int32_t zy, void* __restrict__ y)
{
#pragma clang fp contract(off)
    __shared__ int64_t red[kThreads / 64];
    const int64_t m = blockIdx.x;
    RowRegs<NCH> r1, r2;
    r1.load(x1 + m * K, K);
    r2.load(x2 + m * K, K);
    int32_t hc[NCH][8];
    int64_t ss = 0;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!r1.live[c]) continue;
        const int64_t k0 = 8 * ((int64_t)threadIdx.x + kThreads * c);
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            hc[c][u] = add_one<16>(r1.v[c][u], r2.v[c][u], a1, z1, a2, z2, ah, zh);
            const int64_t d = (int64_t)hc[c][u] - zh;
            ss += d * d;
        }
        store8<16>(h, m * K + k0, hc[c]);
    }
    ss = block_sum_i64(ss, red);
    const double a = (double)ah;
    const double ms = a * a * (double)ss / (double)K + (double)eps;
    const double rt = sqrt(ms);
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!r1.live[c]) continue;
        const int64_t k0 = 8 * ((int64_t)threadIdx.x + kThreads * c);
        int32_t q[8];
#pragma unroll
        for (int u = 0; u < 8; ++u) {
            double v = a * (double)((int64_t)hc[c][u] - zh);
            if (gamma) v = v * (double)gamma[k0 + u];
            v = v / rt;
            q[u] = requant_f64<BITS>(v, (double)ay, zy);
        }
        store8<BITS>(y, m * K + k0, q);
    }
}

// Keys row m of a causal softmax sees: (m mod period) + offset + 1, at most
// K (period 0: all K).
__device__ inline int64_t causal_keys(int64_t m, int64_t K, int64_t period, int64_t offset)
{
    if (period <= 0) return K;
    const int64_t n = m % period + offset + 1;
    return n < K ? n : K;
}

// Rows of at most 2048 codes (K % 8 == 0, 16-byte aligned), one wave per
// row, NC chunks of eight codes per lane (chunk c of lane t holds keys
// 8 (t + 64 c) .. +7).  The exponent alpha (x_k - max) is -alpha d with
// d = max - x_k an integer in [0, 65535] and alpha an fp32 scale, so
// alpha d is exact in fp64 and, for d = 256 h + l,
//   exp(-alpha d) = exp(-256 alpha h) exp(-alpha l).
// Each block evaluates the two 256-entry factor tables once (one exp per
// entry, in LDS); a key then costs two table reads and one fp64 product,
// within three ulp of the direct exp.  The code is rint(e * s) + zy with
// s = (1 / sum) (1 / ay) (two roundings where the oracle divides twice);
// the codes can differ from the oracle's only where the fp64 value sits
// within a few ulp of a rounding tie.  Hidden keys are written as zy.
// Each wave takes kSmRows rows in snake order (m, 2G - 1 - m, 2G + m, ...
// for G waves in the grid): under a causal mask whose period divides 2G
// the key counts of each pair sum to the period plus one.
constexpr int kSmWaves = 8, kSmRows = 4;

typedef short s16x2 __attribute__((ext_vector_type(2)));
typedef unsigned short u16x2 __attribute__((ext_vector_type(2)));

__device__ inline s16x2 as_s16x2(int v) { return __builtin_bit_cast(s16x2, v); }

// DPP lane moves within rows of 16 lanes (all 64 lanes active)
template <int CTRL>
__device__ inline int dpp_mov(int v)
{
    return __builtin_amdgcn_update_dpp(0, v, CTRL, 0xF, 0xF, false);
}
constexpr int kDppXor1 = 0xB1, kDppXor2 = 0x4E, kDppHalfMirror = 0x141, kDppMirror = 0x140;

template <int CTRL>
__device__ inline double dpp_f64(double v)
{
    const long long b = __double_as_longlong(v);
    const int lo = dpp_mov<CTRL>((int)b), hi = dpp_mov<CTRL>((int)(b >> 32));
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

__device__ inline double readlane_f64(double v, int l)
{
    const long long b = __double_as_longlong(v);
    const int lo = __builtin_amdgcn_readlane((int)b, l);
    const int hi = __builtin_amdgcn_readlane((int)(b >> 32), l);
    return __longlong_as_double(((long long)hi << 32) | (unsigned)lo);
}

// wave-wide max and fp64 sum: butterfly within each 16-lane row, then the
// four row results; every lane gets the same value
__device__ inline int32_t wave_max_i32(int32_t v)
{
    v = max(v, dpp_mov<kDppXor1>(v));
    v = max(v, dpp_mov<kDppXor2>(v));
    v = max(v, dpp_mov<kDppHalfMirror>(v));
    v = max(v, dpp_mov<kDppMirror>(v));
    const int a = __builtin_amdgcn_readlane(v, 0), b = __builtin_amdgcn_readlane(v, 16);
    const int c = __builtin_amdgcn_readlane(v, 32), d = __builtin_amdgcn_readlane(v, 48);
    return max(max(a, b), max(c, d));
}

__device__ inline double wave_sum_f64(double v)
{
#pragma clang fp contract(off)
    v = v + dpp_f64<kDppXor1>(v);
    v = v + dpp_f64<kDppXor2>(v);
    v = v + dpp_f64<kDppHalfMirror>(v);
    v = v + dpp_f64<kDppMirror>(v);
    return (readlane_f64(v, 0) + readlane_f64(v, 16)) + (readlane_f64(v, 32) + readlane_f64(v, 48));
}

// the factor products of the two keys of one packed word
__device__ inline void exp_pair(int w, s16x2 mx2, const double* tab, double& e0, double& e1)
{
#pragma clang fp contract(off)
    const uint32_t D = __builtin_bit_cast(uint32_t, __builtin_bit_cast(u16x2, mx2 - as_s16x2(w)));
    const char* tb = reinterpret_cast<const char*>(tab);
    e0 = *reinterpret_cast<const double*>(tb + (((D >> 8) & 255u) << 3)) *
         *reinterpret_cast<const double*>(tb + 2048 + ((D & 255u) << 3));
    e1 = *reinterpret_cast<const double*>(tb + ((D >> 24) << 3)) *
         *reinterpret_cast<const double*>(tb + 2048 + (((D >> 16) & 255u) << 3));
}

// rint(e s) + zy, clamped.  Adding 1.5 * 2^52 rounds t in [0, 2^31) to an
// integer (to nearest, ties to even) held in the low word; CLAMP caps t
// when s (an upper bound of t, e <= 1) exceeds 1e9.
template <int BITS, bool CLAMP>
__device__ inline int32_t requant_prob(double e, double s, int32_t zy)
{
#pragma clang fp contract(off)
    constexpr int32_t qmax = (1 << (BITS - 1)) - 1, qmin = -(1 << (BITS - 1));
    double t = e * s;
    if (CLAMP) t = fmin(t, 1e9);
    t = t + 6755399441055744.0;
    const int32_t r = (int32_t)(uint32_t)__double_as_longlong(t) + zy;
    return min(max(r, qmin), qmax);
}

template <int BITS, bool CLAMP>
__device__ inline void requant_chunk(const double* e, int k0, int n, double s, int32_t zy,
                                     void* y, int64_t base)
{
    int32_t o[8];
    if (k0 + 8 <= n) {
#pragma unroll
        for (int u = 0; u < 8; ++u) o[u] = requant_prob<BITS, CLAMP>(e[u], s, zy);
    } else if (k0 < n) {
#pragma unroll
        for (int u = 0; u < 8; ++u) o[u] = k0 + u < n ? requant_prob<BITS, CLAMP>(e[u], s, zy) : zy;
    } else {
#pragma unroll
        for (int u = 0; u < 8; ++u) o[u] = zy;
    }
    store8<BITS>(y, base + k0, o);
}

// one row: m and n (keys visible, 1 <= n <= K <= 512 NC) are wave-uniform
template <int BITS, int NC>
__device__ inline void softmax_table_row(int64_t m, int K, int n, const int4* q,
                                         const double* tab, double ri, int32_t zy,
                                         void* __restrict__ y)
{
#pragma clang fp contract(off)
    const int lane = threadIdx.x & 63;
    int32_t mx = -32768;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int k0 = 8 * (lane + 64 * c);
        const int4 w = q[c];
        if (k0 + 8 <= n) {
            const s16x2 a = __builtin_elementwise_max(as_s16x2(w.x), as_s16x2(w.y));
            const s16x2 b = __builtin_elementwise_max(as_s16x2(w.z), as_s16x2(w.w));
            const s16x2 h = __builtin_elementwise_max(a, b);
            mx = max(mx, max((int32_t)h.x, (int32_t)h.y));
        } else if (k0 < n) {
            const int16_t* v = reinterpret_cast<const int16_t*>(&q[c]);
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (k0 + u < n) mx = max(mx, (int32_t)v[u]);
        }
    }
    mx = wave_max_i32(mx);
    const s16x2 mx2 = {(short)mx, (short)mx};
    double e[NC][8];
    double sum = 0.0;
#pragma unroll
    for (int c = 0; c < NC; ++c) {
        const int k0 = 8 * (lane + 64 * c);
        if (k0 < n) {
            // hidden keys of a partial chunk read valid entries (their
            // codes are zero or real scores) and are zeroed below
            exp_pair(q[c].x, mx2, tab, e[c][0], e[c][1]);
            exp_pair(q[c].y, mx2, tab, e[c][2], e[c][3]);
            exp_pair(q[c].z, mx2, tab, e[c][4], e[c][5]);
            exp_pair(q[c].w, mx2, tab, e[c][6], e[c][7]);
            if (k0 + 8 > n) {
#pragma unroll
                for (int u = 0; u < 8; ++u) e[c][u] = k0 + u < n ? e[c][u] : 0.0;
            }
        } else {
#pragma unroll
            for (int u = 0; u < 8; ++u) e[c][u] = 0.0;
        }
#pragma unroll
        for (int u = 0; u < 8; ++u) sum += e[c][u];
    }
    sum = wave_sum_f64(sum);  // >= 1: the maximum key contributes exp(0)
    const double s = (1.0 / sum) * ri;
    const int64_t base = m * K;
    if (s <= 1e9) {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int k0 = 8 * (lane + 64 * c);
            if (k0 < K) requant_chunk<BITS, false>(e[c], k0, n, s, zy, y, base);
        }
    } else {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const int k0 = 8 * (lane + 64 * c);
            if (k0 < K) requant_chunk<BITS, true>(e[c], k0, n, s, zy, y, base);
        }
    }
}

template <int BITS, int NC>
__global__ __launch_bounds__(kSmWaves * 64) void softmax_table_kernel(
    const int16_t* __restrict__ x, int64_t M, int64_t K, float ax, float ay, int32_t zy,
    int64_t period, int64_t offset, void* __restrict__ y)
{
#pragma clang fp contract(off)
    __shared__ double tab[512];  // [0, 256): exp(-256 alpha h); [256, 512): exp(-alpha l)
    const int t = threadIdx.x, lane = t & 63;
    const double a = (double)ax;
    for (int i = t; i < 512; i += kSmWaves * 64)
        tab[i] = i < 256 ? exp(-(a * (double)(256 * i))) : exp(-(a * (double)(i - 256)));
    const int64_t G = (int64_t)gridDim.x * kSmWaves;
    const int64_t g = (int64_t)blockIdx.x * kSmWaves + __builtin_amdgcn_readfirstlane(t >> 6);
    auto row_of = [&](int r) -> int64_t {
        return (r & 1) ? (int64_t)(r + 1) * G - 1 - g : (int64_t)r * G + g;
    };
    // keys row m sees (0 past M); M < 2^31, so m % period fits 32 bits
    auto keys_of = [&](int64_t m) -> int {
        if (m >= M) return 0;
        if (period <= 0) return (int)K;
        const int64_t r = period > m ? m : (int64_t)((uint32_t)m % (uint32_t)period);
        const int64_t n = r + offset + 1;
        return (int)(n < K ? n : K);
    };
    // chunks from ceil(n / 8) on lie outside the row's descriptor and read
    // as zeros without a memory access
    int4 q[2][NC];
    int n[2];
    auto load = [&](int slot, int r) {
        const int64_t m = row_of(r);
        n[slot] = keys_of(m);
        const __amdgpu_buffer_rsrc_t rx = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(x + (m < M ? m : 0) * K), (short)0, (n[slot] + 7) / 8 * 16, 0x00020000);
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const auto v = __builtin_amdgcn_raw_buffer_load_b128(rx, 16 * (lane + 64 * c), 0, 0);
            q[slot][c] = make_int4((int)v[0], (int)v[1], (int)v[2], (int)v[3]);
        }
    };
    load(0, 0);
    load(1, 1);
    __syncthreads();
    const double ri = 1.0 / (double)ay;
#pragma unroll
    for (int r = 0; r < kSmRows; ++r) {
        const int slot = r & 1;
        const int64_t m = row_of(r);
        if (m < M) softmax_table_row<BITS, NC>(m, (int)K, n[slot], q[slot], tab, ri, zy, y);
        if (r + 2 < kSmRows) load(slot, r + 2);
    }
}

template <int BITS, int NCH>
__global__ __launch_bounds__(kThreads) void softmax_regs_kernel(const int16_t* __restrict__ x,
                                                                int64_t K, float ax, float ay,
                                                                int32_t zy, int64_t period,
                                                                int64_t offset,
                                                                void* __restrict__ y)
{
#pragma clang fp contract(off)
    __shared__ int32_t red_i[kThreads / 64];
    __shared__ double red_d[kThreads / 64];
    const int64_t m = blockIdx.x;
    const int64_t n = causal_keys(m, K, period, offset);  // keys this row sees
    RowRegs<NCH> r;
    r.load(x + m * K, K);
    int32_t mx = -32768;
#pragma unroll
    for (int c = 0; c < NCH; ++c)
        if (r.live[c])
#pragma unroll
            for (int u = 0; u < 8; ++u)
                if (8 * ((int64_t)threadIdx.x + kThreads * c) + u < n)
                    mx = max(mx, (int32_t)r.v[c][u]);
    for (int o = 32; o > 0; o >>= 1) mx = max(mx, __shfl_xor(mx, o));
    if ((threadIdx.x & 63) == 0) red_i[threadIdx.x >> 6] = mx;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) mx = max(mx, red_i[w]);
    const double a = (double)ax;
    double e[NCH][8];
    double sum = 0.0;
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        const int64_t k0 = 8 * ((int64_t)threadIdx.x + kThreads * c);
        if (r.live[c] && k0 < n) {
#pragma unroll
            for (int u = 0; u < 8; ++u) {
                e[c][u] = k0 + u < n ? exp(a * (double)((int32_t)r.v[c][u] - mx)) : 0.0;
                sum += e[c][u];
            }
        } else {  // past the causal boundary (or past K): no exponentials
#pragma unroll
            for (int u = 0; u < 8; ++u) e[c][u] = 0.0;
        }
    }
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if ((threadIdx.x & 63) == 0) red_d[threadIdx.x >> 6] = sum;
    __syncthreads();
    sum = 0.0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) sum += red_d[w];
#pragma unroll
    for (int c = 0; c < NCH; ++c) {
        if (!r.live[c]) continue;
        const int64_t k0 = 8 * ((int64_t)threadIdx.x + kThreads * c);
        int32_t q[8];
        if (k0 < n) {
#pragma unroll
            for (int u = 0; u < 8; ++u)
                q[u] = k0 + u < n ? requant_f64<BITS>(e[c][u] / sum, (double)ay, zy) : zy;
        } else {  // keys past the causal boundary: probability 0, no arithmetic
#pragma unroll
            for (int u = 0; u < 8; ++u) q[u] = zy;
        }
        store8<BITS>(y, m * K + k0, q);
    }
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
                                                           int32_t zy, int64_t period,
                                                           int64_t offset, void* __restrict__ y)
{
#pragma clang fp contract(off)
    __shared__ int32_t red_i[kThreads / 64];
    __shared__ double red_d[kThreads / 64];
    const int64_t m = blockIdx.x;
    const int64_t n = causal_keys(m, K, period, offset);  // keys this row sees
    const int16_t* row = x + m * K;
    int32_t mx = -32768;
    for (int64_t k = threadIdx.x; k < n; k += kThreads) mx = max(mx, (int32_t)row[k]);
    for (int o = 32; o > 0; o >>= 1) mx = max(mx, __shfl_xor(mx, o));
    if ((threadIdx.x & 63) == 0) red_i[threadIdx.x >> 6] = mx;
    __syncthreads();
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) mx = max(mx, red_i[w]);
    const double a = (double)ax;
    double sum = 0.0;
    for (int64_t k = threadIdx.x; k < n; k += kThreads)
        sum += exp(a * (double)((int32_t)row[k] - mx));
    for (int o = 32; o > 0; o >>= 1) sum += __shfl_xor(sum, o);
    if ((threadIdx.x & 63) == 0) red_d[threadIdx.x >> 6] = sum;
    __syncthreads();
    sum = 0.0;
#pragma unroll
    for (int w = 0; w < kThreads / 64; ++w) sum += red_d[w];
    for (int64_t k = threadIdx.x; k < K; k += kThreads) {
        if (k >= n) {  // past the causal boundary: probability 0
            store_code<BITS>(y, m * K + k, zy);
            continue;
        }
        const double e = exp(a * (double)((int32_t)row[k] - mx));
        store_code<BITS>(y, m * K + k, requant_f64<BITS>(e / sum, (double)ay, zy));
    }
}

}  // namespace

template <int OP>
static hipError_t launch_binary(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                                float a2, int32_t z2, int64_t n, float ay, int32_t zy,
                                int32_t bits, void* y, hipStream_t st)
{
    const uintptr_t ya = bits == 8 ? 4 : 8;
    const bool vec = ((uintptr_t)x1 % 8) == 0 && ((uintptr_t)x2 % 8) == 0 &&
                     ((uintptr_t)y % ya) == 0;
    const int64_t n4 = vec ? n / 4 : 0;
    const int g = grid_for(vec ? n4 : n, kThreads * 2, 256 * 64);
    if (bits == 8)
        add_requant_kernel<8, OP><<<g, kThreads, 0, st>>>(x1, a1, z1, x2, a2, z2, n4, n4 * 4, n,
                                                          ay, zy, y);
    else
        add_requant_kernel<16, OP><<<g, kThreads, 0, st>>>(x1, a1, z1, x2, a2, z2, n4, n4 * 4, n,
                                                           ay, zy, y);
    return hipGetLastError();
}

hipError_t launch_add_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                              float a2, int32_t z2, int64_t n, float ay, int32_t zy,
                              int32_t bits, void* y, hipStream_t st)
{
    return launch_binary<0>(x1, a1, z1, x2, a2, z2, n, ay, zy, bits, y, st);
}

hipError_t launch_mul_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                              float a2, int32_t z2, int64_t n, float ay, int32_t zy,
                              int32_t bits, void* y, hipStream_t st)
{
    return launch_binary<1>(x1, a1, z1, x2, a2, z2, n, ay, zy, bits, y, st);
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
    // one or two blocks per CU (the table fills 64 or 128 KiB of LDS), each
    // streaming at least 16 codes per thread (the 1024 x 5632 SiLU input
    // then fills all 256 CUs)
    const uintptr_t ya = bits == 8 ? 8 : 16;
    const bool vec = ((uintptr_t)x % 16) == 0 && ((uintptr_t)y % ya) == 0 &&
                     ((uintptr_t)lut % 16) == 0;
    const int64_t n8 = vec ? n / 8 : 0;
    const int cap = bits == 8 ? 512 : 256;
    const int g = grid_for(n, kLutThreads * 16, cap);
    const size_t lds = 65536 * (bits / 8);
    if (bits == 8) {
        static const hipError_t a8 = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&lut_apply_kernel<8>),
            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (a8 != hipSuccess) return a8;
        lut_apply_kernel<8><<<g, kLutThreads, lds, st>>>(x, n8, n8 * 8, n, lut, y);
    } else {
        static const hipError_t a16 = hipFuncSetAttribute(
            reinterpret_cast<const void*>(&lut_apply_kernel<16>),
            hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
        if (a16 != hipSuccess) return a16;
        lut_apply_kernel<16><<<g, kLutThreads, lds, st>>>(x, n8, n8 * 8, n, lut, y);
    }
    return hipGetLastError();
}

template <int LB, int OB>
static hipError_t lut_mul_launch(const int16_t* x1, const void* lut, float a1, int32_t z1,
                                 const int16_t* x2, float a2, int32_t z2, int64_t n, float ay,
                                 int32_t zy, void* y, hipStream_t st)
{
    const uintptr_t ya = OB == 8 ? 8 : 16;
    const bool vec = ((uintptr_t)x1 % 16) == 0 && ((uintptr_t)x2 % 16) == 0 &&
                     ((uintptr_t)y % ya) == 0 && ((uintptr_t)lut % 16) == 0;
    const int64_t n8 = vec ? n / 8 : 0;
    const int g = grid_for(n, kLutThreads * 16, LB == 8 ? 512 : 256);
    const size_t lds = 65536 * (LB / 8);
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&lut_mul_kernel<LB, OB>),
        hipFuncAttributeMaxDynamicSharedMemorySize, (int)lds);
    if (attr != hipSuccess) return attr;
    lut_mul_kernel<LB, OB><<<g, kLutThreads, lds, st>>>(x1, lut, a1, z1, x2, a2, z2, n8, n8 * 8,
                                                       n, ay, zy, y);
    return hipGetLastError();
}

hipError_t launch_lut_mul(const int16_t* x1, const void* lut, int32_t lut_bits, float a1,
                          int32_t z1, const int16_t* x2, float a2, int32_t z2, int64_t n,
                          float ay, int32_t zy, int32_t bits, void* y, hipStream_t st)
{
    if (n == 0) return hipSuccess;
    if (lut_bits == 8)
        return bits == 8 ? lut_mul_launch<8, 8>(x1, lut, a1, z1, x2, a2, z2, n, ay, zy, y, st)
                         : lut_mul_launch<8, 16>(x1, lut, a1, z1, x2, a2, z2, n, ay, zy, y, st);
    return bits == 8 ? lut_mul_launch<16, 8>(x1, lut, a1, z1, x2, a2, z2, n, ay, zy, y, st)
                     : lut_mul_launch<16, 16>(x1, lut, a1, z1, x2, a2, z2, n, ay, zy, y, st);
}

template <int BITS, int NCH>
void rmsnorm_regs(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                  const float* gamma, float eps, float ay, int32_t zy, void* y, hipStream_t st)
{
    rmsnorm_regs_kernel<BITS, NCH><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, zx, gamma, eps, ay,
                                                                    zy, y);
}

template <int BITS, int NCH>
void softmax_regs(const int16_t* x, int64_t M, int64_t K, float ax, float ay, int32_t zy,
                  int64_t period, int64_t offset, void* y, hipStream_t st)
{
    softmax_regs_kernel<BITS, NCH><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, ay, zy, period,
                                                                    offset, y);
}

// register-resident rows: K % 8 == 0, 16-byte aligned x and y, chunks per
// thread (0: the strided kernel)
static int row_chunks(const int16_t* x, const void* y, int64_t K)
{
    if (K % 8 != 0 || ((uintptr_t)x % 16) != 0 || ((uintptr_t)y % 16) != 0) return 0;
    const int64_t ch = (K / 8 + kThreads - 1) / kThreads;
    return ch <= 1 ? 1 : ch <= 2 ? 2 : ch <= 4 ? 4 : 0;
}

hipError_t launch_rmsnorm(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                          const float* gamma, float eps, float ay, int32_t zy, int32_t bits,
                          void* y, hipStream_t st)
{
    const int ch = row_chunks(x, y, K);
    if (ch > 0) {
        if (bits == 8) {
            if (ch == 1) rmsnorm_regs<8, 1>(x, M, K, ax, zx, gamma, eps, ay, zy, y, st);
            else if (ch == 2) rmsnorm_regs<8, 2>(x, M, K, ax, zx, gamma, eps, ay, zy, y, st);
            else rmsnorm_regs<8, 4>(x, M, K, ax, zx, gamma, eps, ay, zy, y, st);
        } else {
            if (ch == 1) rmsnorm_regs<16, 1>(x, M, K, ax, zx, gamma, eps, ay, zy, y, st);
            else if (ch == 2) rmsnorm_regs<16, 2>(x, M, K, ax, zx, gamma, eps, ay, zy, y, st);
            else rmsnorm_regs<16, 4>(x, M, K, ax, zx, gamma, eps, ay, zy, y, st);
        }
        return hipGetLastError();
    }
    if (bits == 8)
        rmsnorm_kernel<8><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, zx, gamma, eps, ay, zy, y);
    else
        rmsnorm_kernel<16><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, zx, gamma, eps, ay, zy, y);
    return hipGetLastError();
}

hipError_t launch_add_rmsnorm(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                             float a2, int32_t z2, int64_t M, int64_t K, float ah, int32_t zh,
                             int16_t* h, const float* gamma, float eps, float ay, int32_t zy,
                             int32_t bits, void* y, hipStream_t st)
{
    if (M == 0) return hipSuccess;
    const int ch = row_chunks(x1, y, K);
    if (ch > 0 && row_chunks(x2, h, K) > 0) {
        const dim3 g((unsigned)M), b(kThreads);
        if (bits == 8) {
            if (ch == 1) add_rmsnorm_kernel<8, 1><<<g, b, 0, st>>>(x1, a1, z1, x2, a2, z2, K, ah, zh, h, gamma, eps, ay, zy, y);
            else if (ch == 2) add_rmsnorm_kernel<8, 2><<<g, b, 0, st>>>(x1, a1, z1, x2, a2, z2, K, ah, zh, h, gamma, eps, ay, zy, y);
            else add_rmsnorm_kernel<8, 4><<<g, b, 0, st>>>(x1, a1, z1, x2, a2, z2, K, ah, zh, h, gamma, eps, ay, zy, y);
        } else {
            if (ch == 1) add_rmsnorm_kernel<16, 1><<<g, b, 0, st>>>(x1, a1, z1, x2, a2, z2, K, ah, zh, h, gamma, eps, ay, zy, y);
            else if (ch == 2) add_rmsnorm_kernel<16, 2><<<g, b, 0, st>>>(x1, a1, z1, x2, a2, z2, K, ah, zh, h, gamma, eps, ay, zy, y);
            else add_rmsnorm_kernel<16, 4><<<g, b, 0, st>>>(x1, a1, z1, x2, a2, z2, K, ah, zh, h, gamma, eps, ay, zy, y);
        }
        return hipGetLastError();
    }
    // rows that do not fit the register kernel: the two steps
    const hipError_t e = launch_add_requant(x1, a1, z1, x2, a2, z2, M * K, ah, zh, 16, h, st);
    if (e != hipSuccess) return e;
    return launch_rmsnorm(h, M, K, ah, zh, gamma, eps, ay, zy, bits, y, st);
}

template <int BITS, int NC>
static void softmax_table(const int16_t* x, int64_t M, int64_t K, float ax, float ay, int32_t zy,
                          int64_t period, int64_t offset, void* y, hipStream_t st)
{
    constexpr int RPB = kSmRows * kSmWaves;
    softmax_table_kernel<BITS, NC><<<(unsigned)((M + RPB - 1) / RPB), kSmWaves * 64, 0, st>>>(
        x, M, K, ax, ay, zy, period, offset, y);
}

hipError_t launch_softmax(const int16_t* x, int64_t M, int64_t K, float ax, float ay, int32_t zy,
                          int32_t bits, int64_t period, int64_t offset, void* y, hipStream_t st)
{
    const int ch = row_chunks(x, y, K);
    const int64_t P = period, O = offset;
    if (ch == 1 && K <= 2048) {  // one wave per row, 8 NC codes per lane
        const int nc = K <= 512 ? 1 : K <= 1024 ? 2 : 4;
        if (bits == 8) {
            if (nc == 1) softmax_table<8, 1>(x, M, K, ax, ay, zy, P, O, y, st);
            else if (nc == 2) softmax_table<8, 2>(x, M, K, ax, ay, zy, P, O, y, st);
            else softmax_table<8, 4>(x, M, K, ax, ay, zy, P, O, y, st);
        } else {
            if (nc == 1) softmax_table<16, 1>(x, M, K, ax, ay, zy, P, O, y, st);
            else if (nc == 2) softmax_table<16, 2>(x, M, K, ax, ay, zy, P, O, y, st);
            else softmax_table<16, 4>(x, M, K, ax, ay, zy, P, O, y, st);
        }
        return hipGetLastError();
    }
    if (ch > 0) {
        if (bits == 8) {
            if (ch == 1) softmax_regs<8, 1>(x, M, K, ax, ay, zy, P, O, y, st);
            else if (ch == 2) softmax_regs<8, 2>(x, M, K, ax, ay, zy, P, O, y, st);
            else softmax_regs<8, 4>(x, M, K, ax, ay, zy, P, O, y, st);
        } else {
            if (ch == 1) softmax_regs<16, 1>(x, M, K, ax, ay, zy, P, O, y, st);
            else if (ch == 2) softmax_regs<16, 2>(x, M, K, ax, ay, zy, P, O, y, st);
            else softmax_regs<16, 4>(x, M, K, ax, ay, zy, P, O, y, st);
        }
        return hipGetLastError();
    }
    if (bits == 8) softmax_kernel<8><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, ay, zy, P, O, y);
    else softmax_kernel<16><<<(unsigned)M, kThreads, 0, st>>>(x, K, ax, ay, zy, P, O, y);
    return hipGetLastError();
}

}  // namespace mq

namespace mq {
namespace {

// Rotary position embedding.  The angle table holds cos and sin of
// (t + pos0) * base^(-2i/D) for every token t and pair i (fp64: inverse
// frequency by pow, one product, cos, sin); the main kernel rotates each
// pair (i, i + D/2) of every head of x [T][H * D] and requantizes.
__global__ __launch_bounds__(256) void rope_table_kernel(int64_t T, int64_t half, int64_t D,
                                                         double base, int64_t pos0,
                                                         double* __restrict__ cs)
{
#pragma clang fp contract(off)
    const int64_t idx = (int64_t)blockIdx.x * 256 + threadIdx.x;
    if (idx >= T * half) return;
    const int64_t t = idx / half, i = idx - t * half;
    const double inv = pow(base, -(double)(2 * i) / (double)D);
    const double ang = (double)(t + pos0) * inv;
    cs[2 * idx] = cos(ang);
    cs[2 * idx + 1] = sin(ang);
}

// grid (ceil(H * D/2 / 256), min(T, 65535)): block row t holds the pairs
// (h, i) of tokens t, t + gridDim.y, ..., one per thread
template <int BITS>
__global__ __launch_bounds__(256) void rope_kernel(const int16_t* __restrict__ x, int64_t T,
                                                   int32_t H,
                                                   int32_t half, float ax, int32_t zx,
                                                   const double* __restrict__ cs, float ay,
                                                   int32_t zy, void* __restrict__ y)
{
#pragma clang fp contract(off)
    const int32_t q = (int32_t)blockIdx.x * 256 + (int32_t)threadIdx.x;
    if (q >= H * half) return;
    const int32_t h = q / half, i = q - h * half;
    for (int64_t t = blockIdx.y; t < T; t += gridDim.y) {
        const int64_t j0 = (t * H + h) * (int64_t)(2 * half) + i, j1 = j0 + half;
        const double c = cs[2 * (t * half + i)], sn = cs[2 * (t * half + i) + 1];
        const double u = (double)ax * (double)((int32_t)x[j0] - zx);
        const double w = (double)ax * (double)((int32_t)x[j1] - zx);
        store_code<BITS>(y, j0, requant_f64<BITS>(u * c - w * sn, (double)ay, zy));
        store_code<BITS>(y, j1, requant_f64<BITS>(w * c + u * sn, (double)ay, zy));
    }
}

}  // namespace

hipError_t launch_rope_table(int64_t T, int64_t D, double base, int64_t pos0, double* table,
                             hipStream_t st)
{
    const int64_t half = D / 2;
    const int64_t entries = T * half;
    if (entries == 0) return hipSuccess;
    rope_table_kernel<<<(unsigned)((entries + 255) / 256), 256, 0, st>>>(T, half, D, base, pos0,
                                                                         table);
    return hipGetLastError();
}

hipError_t launch_rope_apply(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax,
                             int32_t zx, const double* table, float ay, int32_t zy, int32_t bits,
                             void* y, hipStream_t st)
{
    const int64_t half = D / 2;
    if (T == 0) return hipSuccess;
    if (H * half > 0x7FFFFFFF - 256) return hipErrorInvalidValue;
    const dim3 g((unsigned)((H * half + 255) / 256), (unsigned)(T < 65535 ? T : 65535));
    if (bits == 8)
        rope_kernel<8><<<g, 256, 0, st>>>(x, T, (int32_t)H, (int32_t)half, ax, zx, table, ay, zy,
                                          y);
    else
        rope_kernel<16><<<g, 256, 0, st>>>(x, T, (int32_t)H, (int32_t)half, ax, zx, table, ay,
                                           zy, y);
    return hipGetLastError();
}

hipError_t launch_rope(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax, int32_t zx,
                       double base, int64_t pos0, float ay, int32_t zy, int32_t bits,
                       double* table, void* y, hipStream_t st)
{
    const hipError_t e = launch_rope_table(T, D, base, pos0, table, st);
    if (e != hipSuccess) return e;
    return launch_rope_apply(x, T, H, D, ax, zx, table, ay, zy, bits, y, st);
}

}  // namespace mq
