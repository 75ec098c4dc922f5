// Host side of the C ABI declared in include/mq.h: argument validation,
// the Eq.(2)-(3) activation-format derivation, kernel-path dispatch and HIP
// error mapping.  Nothing here allocates or synchronises.
#include <cmath>
#include <cstdint>

#include "mq.h"
#include "mq_internal.h"

namespace {

constexpr int32_t kAbiVersion = 1;

bool finite_pos(float v) { return std::isfinite(v) && v > 0.0f; }

bool zp_ok(int32_t zp, int32_t bits)
{
    const int32_t lo = -(1 << (bits - 1)), hi = (1 << (bits - 1)) - 1;
    return zp >= lo && zp <= hi;
}

bool act_bits_ok(int32_t bits) { return bits == 8 || bits == 16; }

mq_status from_hip(hipError_t e) { return e == hipSuccess ? MQ_OK : MQ_ERR_HIP; }

hipStream_t as_stream(void* s) { return reinterpret_cast<hipStream_t>(s); }

// largest element count the grid-stride kernels index with int64 safely
constexpr int64_t kMaxElems = (int64_t)1 << 46;

}  // namespace

extern "C" {

const char* mq_status_string(mq_status status)
{
    switch (status) {
    case MQ_OK: return "MQ_OK";
    case MQ_ERR_INVALID_ARG: return "MQ_ERR_INVALID_ARG: argument rejected by validation";
    case MQ_ERR_UNSUPPORTED: return "MQ_ERR_UNSUPPORTED: valid but not supported";
    case MQ_ERR_HIP: return "MQ_ERR_HIP: a HIP launch failed";
    }
    return "unknown mq_status";
}

int32_t mq_version(void) { return kAbiVersion; }

mq_status mq_act_params(float f_min, float f_max, int32_t bits, float* alpha, int32_t* zp)
{
    if (!alpha || !zp || !act_bits_ok(bits)) return MQ_ERR_INVALID_ARG;
    if (!std::isfinite(f_min) || !std::isfinite(f_max) || f_min > f_max) return MQ_ERR_INVALID_ARG;
    // widen to contain zero, then Eq.(2) q_max and Eq.(3) alpha, beta
    const double lo = std::fmin((double)f_min, 0.0);
    const double hi = std::fmax((double)f_max, 0.0);
    const double qmax = std::ldexp(1.0, bits) - 1.0;
    const double width = hi - lo;
    float a = 1.0f;
    double beta = 0.0;
    if (width != 0.0) {
        a = (float)(width / qmax);
        if (!(a > 0.0f) || !std::isfinite(a)) return MQ_ERR_INVALID_ARG;
        beta = lo / (double)a;
    }
    double z = std::rint(-beta);
    z = std::fmin(std::fmax(z, 0.0), qmax);
    *alpha = a;
    *zp = (int32_t)z - (1 << (bits - 1));
    return MQ_OK;
}

mq_status mq_fold_weights(const float* w, const float* s, int64_t N, int64_t K, float* w_hat,
                          void* stream)
{
    if (N < 0 || K < 0 || N > kMaxElems || K > kMaxElems || (K > 0 && N > kMaxElems / K))
        return MQ_ERR_INVALID_ARG;
    if (N == 0 || K == 0) return MQ_OK;
    if (!w || !s || !w_hat) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_fold_weights(w, s, N, K, w_hat, as_stream(stream)));
}

mq_status mq_fold_acts(const float* x, const float* s, int64_t M, int64_t K, float* x_hat,
                       void* stream)
{
    if (M < 0 || K < 0 || M > kMaxElems || K > kMaxElems || (K > 0 && M > kMaxElems / K))
        return MQ_ERR_INVALID_ARG;
    if (M == 0 || K == 0) return MQ_OK;
    if (!x || !s || !x_hat) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_fold_acts(x, s, M, K, x_hat, as_stream(stream)));
}

mq_status mq_quantize_act(const float* x, int64_t numel, float alpha, int32_t zp, int32_t bits,
                          void* x_q, void* stream)
{
    if (numel < 0 || numel > kMaxElems || !act_bits_ok(bits) || !finite_pos(alpha) ||
        !zp_ok(zp, bits))
        return MQ_ERR_INVALID_ARG;
    if (numel == 0) return MQ_OK;
    if (!x || !x_q) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_quantize_act(x, numel, alpha, zp, bits, x_q, as_stream(stream)));
}

mq_status mq_dequant(const void* q, int32_t bits, int64_t numel, float alpha, int32_t zp,
                     float* y, void* stream)
{
    if (numel < 0 || numel > kMaxElems || !act_bits_ok(bits) || !finite_pos(alpha) ||
        !zp_ok(zp, bits))
        return MQ_ERR_INVALID_ARG;
    if (numel == 0) return MQ_OK;
    if (!q || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_dequant(q, bits, numel, alpha, zp, y, as_stream(stream)));
}

mq_status mq_pack_weights(const float* w, int64_t N, int64_t K, int32_t bits, void* w_q,
                          float* w_scale, int32_t* w_colsum, void* stream)
{
    if (bits != 8 && bits != 4) return MQ_ERR_INVALID_ARG;
    if (N < 0 || N > 0x7FFFFFFF || K < 1 || K > MQ_MAX_K) return MQ_ERR_INVALID_ARG;
    if (bits == 4 && (K % 2) != 0) return MQ_ERR_INVALID_ARG;
    if (N == 0) return MQ_OK;
    if (!w || !w_q || !w_scale || !w_colsum) return MQ_ERR_INVALID_ARG;
    return from_hip(
        mq::launch_pack_weights(w, N, K, bits, w_q, w_scale, w_colsum, as_stream(stream)));
}

mq_status mq_pack_weights_asym(const float* w, int64_t N, int64_t K, int32_t bits,
                               int32_t per_tensor, void* w_q, float* w_scale, int32_t* w_zp,
                               int32_t* w_colsum, void* stream)
{
    if (bits != 8 && bits != 4) return MQ_ERR_INVALID_ARG;
    if (per_tensor != 0 && per_tensor != 1) return MQ_ERR_INVALID_ARG;
    if (N < 0 || N > 0x7FFFFFFF || K < 1 || K > MQ_MAX_K) return MQ_ERR_INVALID_ARG;
    if (bits == 4 && (K % 2) != 0) return MQ_ERR_INVALID_ARG;
    if (N == 0) return MQ_OK;
    if (!w || !w_q || !w_scale || !w_zp || !w_colsum) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_pack_weights_asym(w, N, K, bits, per_tensor != 0, w_q, w_scale,
                                                 w_zp, w_colsum, as_stream(stream)));
}

mq_status mq_add_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2, float a2,
                         int32_t z2, int64_t numel, float ay, int32_t zy, int32_t out_bits,
                         void* y, void* stream)
{
    if (numel < 0 || numel > kMaxElems || !act_bits_ok(out_bits)) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(a1) || !finite_pos(a2) || !finite_pos(ay)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(z1, 16) || !zp_ok(z2, 16) || !zp_ok(zy, out_bits)) return MQ_ERR_INVALID_ARG;
    if (numel == 0) return MQ_OK;
    if (!x1 || !x2 || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_add_requant(x1, a1, z1, x2, a2, z2, numel, ay, zy, out_bits, y,
                                           as_stream(stream)));
}

mq_status mq_mul_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2, float a2,
                         int32_t z2, int64_t numel, float ay, int32_t zy, int32_t out_bits,
                         void* y, void* stream)
{
    if (numel < 0 || numel > kMaxElems || !act_bits_ok(out_bits)) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(a1) || !finite_pos(a2) || !finite_pos(ay)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(z1, 16) || !zp_ok(z2, 16) || !zp_ok(zy, out_bits)) return MQ_ERR_INVALID_ARG;
    if (numel == 0) return MQ_OK;
    if (!x1 || !x2 || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_mul_requant(x1, a1, z1, x2, a2, z2, numel, ay, zy, out_bits, y,
                                           as_stream(stream)));
}

mq_status mq_add_rmsnorm(const int16_t* x1, float a1, int32_t z1, const int16_t* x2, float a2,
                         int32_t z2, int64_t M, int64_t K, float ah, int32_t zh, int16_t* h,
                         const float* gamma, float eps, float ay, int32_t zy, int32_t out_bits,
                         void* y, void* stream)
{
    if (M < 0 || M > 0x7FFFFFFF || K < 1 || K > (1 << 20) || !act_bits_ok(out_bits))
        return MQ_ERR_INVALID_ARG;
    if (M > 0 && M > kMaxElems / K) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(a1) || !finite_pos(a2) || !finite_pos(ah) || !finite_pos(ay))
        return MQ_ERR_INVALID_ARG;
    if (!std::isfinite(eps) || eps < 0.0f) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(z1, 16) || !zp_ok(z2, 16) || !zp_ok(zh, 16) || !zp_ok(zy, out_bits))
        return MQ_ERR_INVALID_ARG;
    if (M == 0) return MQ_OK;
    if (!x1 || !x2 || !h || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_add_rmsnorm(x1, a1, z1, x2, a2, z2, M, K, ah, zh, h, gamma, eps, ay,
                                           zy, out_bits, y, as_stream(stream)));
}

mq_status mq_lut_mul(const int16_t* x1, const void* lut, int32_t lut_bits, float a1, int32_t z1,
                     const int16_t* x2, float a2, int32_t z2, int64_t numel, float ay,
                     int32_t zy, int32_t out_bits, void* y, void* stream)
{
    if (numel < 0 || numel > kMaxElems || !act_bits_ok(out_bits) || !act_bits_ok(lut_bits))
        return MQ_ERR_INVALID_ARG;
    if (!finite_pos(a1) || !finite_pos(a2) || !finite_pos(ay)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(z1, lut_bits) || !zp_ok(z2, 16) || !zp_ok(zy, out_bits)) return MQ_ERR_INVALID_ARG;
    if (numel == 0) return MQ_OK;
    if (!x1 || !lut || !x2 || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_lut_mul(x1, lut, lut_bits, a1, z1, x2, a2, z2, numel, ay, zy,
                                       out_bits, y, as_stream(stream)));
}

mq_status mq_rope(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax, int32_t zx,
                  double base, int64_t pos0, float ay, int32_t zy, int32_t out_bits,
                  double* table, void* y, void* stream)
{
    if (T < 0 || H < 1 || D < 2 || D % 2 != 0 || !act_bits_ok(out_bits)) return MQ_ERR_INVALID_ARG;
    if (H > kMaxElems / D || (T > 0 && T > kMaxElems / (H * D))) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(ax) || !finite_pos(ay) || !std::isfinite(base) || !(base > 1.0))
        return MQ_ERR_INVALID_ARG;
    if (pos0 < 0 || pos0 > ((int64_t)1 << 40)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(zx, 16) || !zp_ok(zy, out_bits)) return MQ_ERR_INVALID_ARG;
    if (T == 0) return MQ_OK;
    if (!x || !y || !table) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_rope(x, T, H, D, ax, zx, base, pos0, ay, zy, out_bits, table, y,
                                    as_stream(stream)));
}

mq_status mq_rope_table(int64_t T, int64_t D, double base, int64_t pos0, double* table,
                        void* stream)
{
    if (T < 0 || D < 2 || D % 2 != 0 || D > kMaxElems) return MQ_ERR_INVALID_ARG;
    if (T > 0 && T > kMaxElems / D) return MQ_ERR_INVALID_ARG;
    if (!std::isfinite(base) || !(base > 1.0)) return MQ_ERR_INVALID_ARG;
    if (pos0 < 0 || pos0 > ((int64_t)1 << 40)) return MQ_ERR_INVALID_ARG;
    if (T == 0) return MQ_OK;
    if (!table) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_rope_table(T, D, base, pos0, table, as_stream(stream)));
}

mq_status mq_rope_apply(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax, int32_t zx,
                        const double* table, float ay, int32_t zy, int32_t out_bits, void* y,
                        void* stream)
{
    if (T < 0 || H < 1 || D < 2 || D % 2 != 0 || !act_bits_ok(out_bits)) return MQ_ERR_INVALID_ARG;
    if (H > kMaxElems / D || (T > 0 && T > kMaxElems / (H * D))) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(ax) || !finite_pos(ay)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(zx, 16) || !zp_ok(zy, out_bits)) return MQ_ERR_INVALID_ARG;
    if (T == 0) return MQ_OK;
    if (!x || !y || !table) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_rope_apply(x, T, H, D, ax, zx, table, ay, zy, out_bits, y,
                                          as_stream(stream)));
}

mq_status mq_lut_build(int32_t op, float ax, int32_t zx, float ay, int32_t zy, int32_t out_bits,
                       void* lut, void* stream)
{
    if (op != MQ_LUT_SILU || !act_bits_ok(out_bits)) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(ax) || !finite_pos(ay)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(zx, 16) || !zp_ok(zy, out_bits) || !lut) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_lut_build(op, ax, zx, ay, zy, out_bits, lut, as_stream(stream)));
}

mq_status mq_lut_apply(const int16_t* x, int64_t numel, const void* lut, int32_t out_bits,
                       void* y, void* stream)
{
    if (numel < 0 || numel > kMaxElems || !act_bits_ok(out_bits)) return MQ_ERR_INVALID_ARG;
    if (numel == 0) return MQ_OK;
    if (!x || !lut || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_lut_apply(x, numel, lut, out_bits, y, as_stream(stream)));
}

mq_status mq_rmsnorm(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                     const float* gamma, float eps, float ay, int32_t zy, int32_t out_bits,
                     void* y, void* stream)
{
    if (M < 0 || M > 0x7FFFFFFF || K < 1 || K > (1 << 20) || !act_bits_ok(out_bits))
        return MQ_ERR_INVALID_ARG;
    if (!finite_pos(ax) || !finite_pos(ay) || !std::isfinite(eps) || eps < 0.0f)
        return MQ_ERR_INVALID_ARG;
    if (!zp_ok(zx, 16) || !zp_ok(zy, out_bits)) return MQ_ERR_INVALID_ARG;
    if (M == 0) return MQ_OK;
    if (!x || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_rmsnorm(x, M, K, ax, zx, gamma, eps, ay, zy, out_bits, y,
                                       as_stream(stream)));
}

mq_status mq_softmax(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx, float ay,
                     int32_t zy, int32_t out_bits, void* y, void* stream)
{
    if (M < 0 || M > 0x7FFFFFFF || K < 1 || K > (1 << 20) || !act_bits_ok(out_bits))
        return MQ_ERR_INVALID_ARG;
    if (!finite_pos(ax) || !finite_pos(ay)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(zx, 16) || !zp_ok(zy, out_bits)) return MQ_ERR_INVALID_ARG;
    if (M == 0) return MQ_OK;
    if (!x || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_softmax(x, M, K, ax, ay, zy, out_bits, 0, 0, y, as_stream(stream)));
}

mq_status mq_softmax_causal(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                            float ay, int32_t zy, int32_t out_bits, int64_t period,
                            int64_t offset, void* y, void* stream)
{
    if (M < 0 || M > 0x7FFFFFFF || K < 1 || K > (1 << 20) || !act_bits_ok(out_bits))
        return MQ_ERR_INVALID_ARG;
    if (!finite_pos(ax) || !finite_pos(ay)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(zx, 16) || !zp_ok(zy, out_bits)) return MQ_ERR_INVALID_ARG;
    if (period < 1 || offset < 0 || offset > ((int64_t)1 << 40)) return MQ_ERR_INVALID_ARG;
    if (M == 0) return MQ_OK;
    if (!x || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_softmax(x, M, K, ax, ay, zy, out_bits, period, offset, y,
                                       as_stream(stream)));
}

mq_status mq_smooth_scales(const float* x, int64_t M, int64_t K, const float* w, int64_t N,
                           float a, float* x_absmax, float* w_absmax, float* s, void* stream)
{
    if (M < 0 || N < 0 || K < 0 || M > kMaxElems || N > kMaxElems || K > 0x7FFFFFFF)
        return MQ_ERR_INVALID_ARG;
    if ((K > 0 && (M > kMaxElems / K || N > kMaxElems / K))) return MQ_ERR_INVALID_ARG;
    if (!(a >= 0.0f && a <= 1.0f)) return MQ_ERR_INVALID_ARG;
    if (K == 0) return MQ_OK;
    if (!x_absmax || !w_absmax || !s || (M > 0 && !x) || (N > 0 && !w)) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_smooth_scales(x, M, K, w, N, a, x_absmax, w_absmax, s,
                                             as_stream(stream)));
}

mq_status mq_arl_forward(const float* x, int64_t numel, float alpha, float beta, int32_t bits,
                         float* y, void* stream)
{
    if (numel < 0 || numel > kMaxElems || bits < 2 || bits > 16) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(alpha) || !std::isfinite(beta)) return MQ_ERR_INVALID_ARG;
    if (numel == 0) return MQ_OK;
    if (!x || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_arl_forward(x, numel, alpha, beta, bits, y, as_stream(stream)));
}

mq_status mq_arl_backward(const float* x, const float* g, int64_t numel, float alpha, float beta,
                          int32_t bits, float* gx, double* grads, void* stream)
{
    if (numel < 0 || numel > kMaxElems || bits < 2 || bits > 16) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(alpha) || !std::isfinite(beta)) return MQ_ERR_INVALID_ARG;
    if (!grads || (numel > 0 && (!x || !g || !gx))) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_arl_backward(x, g, numel, alpha, beta, bits, gx, grads,
                                            MQ_ARL_PARTIALS, as_stream(stream)));
}

mq_status mq_quantize_act_rowsum(const float* x, int64_t M, int64_t K, float alpha, int32_t zp,
                                 int8_t* x_q, int32_t* rowsum, void* stream)
{
    if (M < 0 || M > 0x7FFFFFFF || K < 1 || K > MQ_MAX_K) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(alpha) || !zp_ok(zp, 8)) return MQ_ERR_INVALID_ARG;
    if (M == 0) return MQ_OK;
    if (!x || !x_q || !rowsum) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_quantize_act_rowsum(x, M, K, alpha, zp, x_q, rowsum,
                                                   as_stream(stream)));
}

mq_status mq_act_rowsum(const int8_t* a_q, int64_t M, int64_t K, int32_t* rowsum, void* stream)
{
    if (M < 0 || M > 0x7FFFFFFF || K < 1 || K > MQ_MAX_K) return MQ_ERR_INVALID_ARG;
    if (M == 0) return MQ_OK;
    if (!a_q || !rowsum) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_act_rowsum(a_q, M, K, rowsum, as_stream(stream)));
}

int64_t mq_qlinear_workspace_bytes(int64_t M, int64_t K, int64_t N, int32_t w_bits,
                                   int32_t out_bits)
{
    if (w_bits != 8 && w_bits != 4) return -1;
    if (!act_bits_ok(out_bits)) return -1;
    if (M < 0 || N < 0 || K < 1 || K > MQ_MAX_K) return -1;
    if (M > 0x7FFFFFFF || N > 0x7FFFFFFF || (M > 0 && N > kMaxElems / M)) return -1;
    if (M <= 16 || N == 0) return 0;  // decode path or nothing to do
    mq::QLinearArgs p;
    p.M = M;
    p.K = K;
    p.N = N;
    p.w_bits = w_bits;
    p.out_bits = out_bits;
    return mq::prefill_workspace_bytes(p);
}

mq_status mq_qlinear_ex(const int8_t* a_q, int64_t M, int64_t K, int64_t N, const void* w_q,
                        int32_t w_bits, const float* w_scale, const int32_t* w_colsum,
                        float a_scale, int32_t a_zp, float out_scale, int32_t out_zp,
                        int32_t out_bits, const float* bias, void* y_q, int32_t path,
                        void* stream)
{
    return mq_qlinear_ws(a_q, M, K, N, w_q, w_bits, w_scale, w_colsum, a_scale, a_zp, out_scale,
                         out_zp, out_bits, bias, y_q, nullptr, 0, path, stream);
}

}  // extern "C"

namespace mq {

// Validation shared by the qlinear entry points (w_zp and a_rowsum are both
// null, symmetric, or both set); fills the kernel arguments and resolves
// the path.  MQ_OK with M == 0 or N == 0: nothing to launch.
mq_status qlinear_validate(const void* a_q, int32_t a_bits, const int32_t* a_rowsum, int64_t M,
                           int64_t K, int64_t N, const void* w_q, int32_t w_bits,
                           const float* w_scale, const int32_t* w_zp, const int32_t* w_colsum,
                           float a_scale, int32_t a_zp, float out_scale, int32_t out_zp,
                           int32_t out_bits, const float* bias, void* y_q, void* workspace,
                           int64_t workspace_bytes, int32_t path, QLinearArgs* out,
                           int32_t* path_out, float* y_f)
{
    if (workspace_bytes < 0) return MQ_ERR_INVALID_ARG;
    if (workspace && ((uintptr_t)workspace % 256) != 0) return MQ_ERR_INVALID_ARG;
    if (w_bits != 8 && w_bits != 4) return MQ_ERR_INVALID_ARG;
    if (!act_bits_ok(out_bits)) return MQ_ERR_INVALID_ARG;
    if (M < 0 || N < 0 || K < 1 || K > MQ_MAX_K) return MQ_ERR_INVALID_ARG;
    if (M > 0x7FFFFFFF || N > 0x7FFFFFFF || (M > 0 && N > kMaxElems / M)) return MQ_ERR_INVALID_ARG;
    if (w_bits == 4 && (K % 2) != 0) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(a_scale) || !finite_pos(out_scale)) return MQ_ERR_INVALID_ARG;
    if (!zp_ok(a_zp, a_bits) || !zp_ok(out_zp, out_bits)) return MQ_ERR_INVALID_ARG;
    int32_t force_tile = -1;
    if (path >= MQ_PATH_PREFILL_TILE0 && path < MQ_PATH_PREFILL_TILE0 + MQ_PREFILL_TILES) {
        force_tile = path - MQ_PATH_PREFILL_TILE0;
        path = MQ_PATH_PREFILL;
    }
    if (path < MQ_PATH_AUTO || path > MQ_PATH_GENERIC) return MQ_ERR_INVALID_ARG;
    if (path == MQ_PATH_DECODE && M > 16) return MQ_ERR_INVALID_ARG;
    QLinearArgs& p = *out;
    p.M = M;
    p.K = K;
    p.N = N;
    if (M == 0 || N == 0) return MQ_OK;
    if (!a_q || !w_q || !w_scale || !w_colsum || (!y_q && !y_f)) return MQ_ERR_INVALID_ARG;
    if ((w_zp == nullptr) != (a_rowsum == nullptr)) return MQ_ERR_INVALID_ARG;
    if (y_f && a_bits != 8) return MQ_ERR_INVALID_ARG;

    p.a = static_cast<const int8_t*>(a_q);
    p.a_bits = a_bits;
    p.w = w_q;
    p.w_scale = w_scale;
    p.colsum = w_colsum;
    p.bias = bias;
    p.y = y_q;
    p.y_f = y_f;
    p.a_scale = a_scale;
    p.out_scale = out_scale;
    p.a_zp = a_zp;
    p.out_zp = out_zp;
    p.w_bits = w_bits;
    p.out_bits = out_bits;
    p.ws = workspace;
    p.ws_bytes = workspace ? workspace_bytes : 0;
    p.w_zp = w_zp;
    p.a_rowsum = a_rowsum;
    p.force_tile = force_tile;
    *path_out = path == MQ_PATH_AUTO ? (M <= 16 ? MQ_PATH_DECODE : MQ_PATH_PREFILL) : path;
    return MQ_OK;
}

// Launch of a validated call on the resolved path; the tuned kernels fall
// back to the generic one when the shape or alignment rules are not met.
mq_status qlinear_dispatch(const QLinearArgs& p, int32_t path, hipStream_t s)
{
    if (p.M == 0 || p.N == 0) return MQ_OK;
    if (path == MQ_PATH_DECODE && decode_supported(p)) return from_hip(launch_qlinear_decode(p, s));
    if (path == MQ_PATH_PREFILL && prefill_supported(p))
        return from_hip(launch_qlinear_prefill(p, s));
    return from_hip(launch_qlinear_generic(p, s));
}

}  // namespace mq

namespace {

mq_status qlinear_impl(const void* a_q, int32_t a_bits, const int32_t* a_rowsum, int64_t M,
                       int64_t K, int64_t N, const void* w_q, int32_t w_bits,
                       const float* w_scale, const int32_t* w_zp, const int32_t* w_colsum,
                       float a_scale, int32_t a_zp, float out_scale, int32_t out_zp,
                       int32_t out_bits, const float* bias, void* y_q, void* workspace,
                       int64_t workspace_bytes, int32_t path, void* stream)
{
    mq::QLinearArgs p;
    int32_t resolved = MQ_PATH_AUTO;
    const mq_status st = mq::qlinear_validate(
        a_q, a_bits, a_rowsum, M, K, N, w_q, w_bits, w_scale, w_zp, w_colsum, a_scale, a_zp,
        out_scale, out_zp, out_bits, bias, y_q, workspace, workspace_bytes, path, &p, &resolved);
    if (st != MQ_OK) return st;
    return mq::qlinear_dispatch(p, resolved, as_stream(stream));
}

}  // namespace

extern "C" {

mq_status mq_qlinear_ws(const int8_t* a_q, int64_t M, int64_t K, int64_t N, const void* w_q,
                        int32_t w_bits, const float* w_scale, const int32_t* w_colsum,
                        float a_scale, int32_t a_zp, float out_scale, int32_t out_zp,
                        int32_t out_bits, const float* bias, void* y_q, void* workspace,
                        int64_t workspace_bytes, int32_t path, void* stream)
{
    return qlinear_impl(a_q, 8, nullptr, M, K, N, w_q, w_bits, w_scale, nullptr, w_colsum,
                        a_scale, a_zp, out_scale, out_zp, out_bits, bias, y_q, workspace,
                        workspace_bytes, path, stream);
}

mq_status mq_qlinear_a16(const int16_t* a_q, int64_t M, int64_t K, int64_t N, const void* w_q,
                         int32_t w_bits, const float* w_scale, const int32_t* w_colsum,
                         float a_scale, int32_t a_zp, float out_scale, int32_t out_zp,
                         int32_t out_bits, const float* bias, void* y_q, int32_t path,
                         void* stream)
{
    return qlinear_impl(a_q, 16, nullptr, M, K, N, w_q, w_bits, w_scale, nullptr, w_colsum,
                        a_scale, a_zp, out_scale, out_zp, out_bits, bias, y_q, nullptr, 0, path,
                        stream);
}

mq_status mq_qlinear_asym(const int8_t* a_q, const int32_t* a_rowsum, int64_t M, int64_t K,
                          int64_t N, const void* w_q, int32_t w_bits, const float* w_scale,
                          const int32_t* w_zp, const int32_t* w_colsum, float a_scale,
                          int32_t a_zp, float out_scale, int32_t out_zp, int32_t out_bits,
                          const float* bias, void* y_q, void* workspace, int64_t workspace_bytes,
                          int32_t path, void* stream)
{
    if (M > 0 && N > 0 && (!a_rowsum || !w_zp)) return MQ_ERR_INVALID_ARG;
    return qlinear_impl(a_q, 8, a_rowsum, M, K, N, w_q, w_bits, w_scale, w_zp, w_colsum,
                        a_scale, a_zp, out_scale, out_zp, out_bits, bias, y_q, workspace,
                        workspace_bytes, path, stream);
}

mq_status mq_qlinear_dequant(const int8_t* a_q, const int32_t* a_rowsum, int64_t M, int64_t K,
                             int64_t N, const void* w_q, int32_t w_bits, const float* w_scale,
                             const int32_t* w_zp, const int32_t* w_colsum, float a_scale,
                             int32_t a_zp, float out_scale, int32_t out_zp, int32_t out_bits,
                             const float* bias, void* y_q, float* y, void* workspace,
                             int64_t workspace_bytes, int32_t path, void* stream)
{
    if (M > 0 && N > 0 && !y) return MQ_ERR_INVALID_ARG;
    mq::QLinearArgs p;
    int32_t resolved = MQ_PATH_AUTO;
    const mq_status st = mq::qlinear_validate(
        a_q, 8, a_rowsum, M, K, N, w_q, w_bits, w_scale, w_zp, w_colsum, a_scale, a_zp,
        out_scale, out_zp, out_bits, bias, y_q, workspace, workspace_bytes, path, &p, &resolved,
        y);
    if (st != MQ_OK) return st;
    return mq::qlinear_dispatch(p, resolved, as_stream(stream));
}

mq_status mq_qlinear_group(const int8_t* a_q, const int32_t* a_rowsum, int64_t M, int64_t K,
                           int32_t w_bits, float a_scale, int32_t a_zp, int32_t out_bits,
                           const mq_qlinear_out* outs, int32_t n_outs, int32_t path,
                           void* stream)
{
    if (!outs || n_outs < 1 || n_outs > MQ_MAX_GROUP) return MQ_ERR_INVALID_ARG;
    const bool asym = outs[0].w_zp != nullptr;
    mq::QLinearArgs ps[MQ_MAX_GROUP];
    int32_t resolved[MQ_MAX_GROUP];
    // every linear is checked before anything is launched
    for (int i = 0; i < n_outs; ++i) {
        const mq_qlinear_out& o = outs[i];
        if ((o.w_zp != nullptr) != asym) return MQ_ERR_INVALID_ARG;
        const mq_status st = mq::qlinear_validate(
            a_q, 8, a_rowsum, M, K, o.N, o.w_q, w_bits, o.w_scale, o.w_zp, o.w_colsum, a_scale,
            a_zp, o.out_scale, o.out_zp, out_bits, o.bias, o.y_q, nullptr, 0, path, &ps[i],
            &resolved[i]);
        if (st != MQ_OK) return st;
    }
    const hipStream_t s = as_stream(stream);
    // the linears with work; one launch when each of them would take the
    // prefill kernel on its own
    mq::GroupArgs g{};
    int first = -1;
    bool one_launch = true;
    for (int i = 0; i < n_outs; ++i) {
        const mq::QLinearArgs& p = ps[i];
        if (p.M == 0 || p.N == 0) continue;
        if (first < 0) first = i;
        one_launch = one_launch && resolved[i] == MQ_PATH_PREFILL && mq::prefill_supported(p);
        mq::GroupPart& gp = g.part[g.n++];
        gp.w = p.w;
        gp.w_scale = p.w_scale;
        gp.colsum = p.colsum;
        gp.bias = p.bias;
        gp.w_zp = p.w_zp;
        gp.y = p.y;
        gp.N = p.N;
        gp.out_scale = p.out_scale;
        gp.out_zp = p.out_zp;
    }
    if (g.n == 0) return MQ_OK;
    if (one_launch && g.n > 1) return from_hip(mq::launch_qlinear_prefill_group(ps[first], g, s));
    for (int i = 0; i < n_outs; ++i) {
        const mq_status st = mq::qlinear_dispatch(ps[i], resolved[i], s);
        if (st != MQ_OK) return st;
    }
    return MQ_OK;
}

mq_status mq_qlinear(const int8_t* a_q, int64_t M, int64_t K, int64_t N, const void* w_q,
                     int32_t w_bits, const float* w_scale, const int32_t* w_colsum,
                     float a_scale, int32_t a_zp, float out_scale, int32_t out_zp,
                     int32_t out_bits, const float* bias, void* y_q, void* stream)
{
    return mq_qlinear_ex(a_q, M, K, N, w_q, w_bits, w_scale, w_colsum, a_scale, a_zp, out_scale,
                         out_zp, out_bits, bias, y_q, MQ_PATH_AUTO, stream);
}

// Batched attention matmuls: workspace = [row terms: H*M int64][colsum:
// G * (M / 128 rounded up) * N int32][b_scale: float], each part 256-byte
// aligned (the column sums per block of 128 rows serve causal activations).
static int64_t attn_ws_parts(int32_t H, int32_t G, int64_t M, int64_t N, int64_t* off_cs,
                             int64_t* off_sc)
{
    auto up = [](int64_t v) { return (v + 255) / 256 * 256; };
    const int64_t ro = up((int64_t)H * M * 8);
    const int64_t n_mb = (M + mq::kA16TileM - 1) / mq::kA16TileM;
    const int64_t cs = up((int64_t)G * (n_mb > 0 ? n_mb : 1) * N * 4);
    *off_cs = ro;
    *off_sc = ro + cs;
    return ro + cs + 256;
}

int64_t mq_attn_matmul_workspace_bytes(int32_t H, int32_t G, int64_t M, int64_t N)
{
    if (H < 1 || G < 1 || H % G != 0 || M < 0 || N < 0) return -1;
    if (M > kMaxElems / H || N > kMaxElems / G) return -1;
    int64_t a, b;
    return attn_ws_parts(H, G, M, N, &a, &b);
}

mq_status mq_attn_matmul(const int16_t* a, int64_t lda, int64_t a_hs, int32_t H, const int8_t* b,
                         int64_t ldb, int64_t b_hs, int32_t G, int64_t M, int64_t N, int64_t K,
                         float a_scale, int32_t a_zp, float b_scale, int32_t b_zp,
                         float out_scale, int32_t out_zp, int32_t out_bits, void* y, int64_t ldy,
                         int64_t y_hs, int64_t out_causal, int64_t in_causal, void* workspace,
                         int64_t workspace_bytes, int32_t path, void* stream)
{
    const int64_t kCausalMax = (int64_t)1 << 40;
    if (out_causal < -1 || out_causal > kCausalMax || in_causal < -1 || in_causal > kCausalMax)
        return MQ_ERR_INVALID_ARG;
    if (H < 1 || G < 1 || H % G != 0) return MQ_ERR_INVALID_ARG;
    if (M < 0 || N < 0 || K < 1 || K > MQ_MAX_K) return MQ_ERR_INVALID_ARG;
    if (M > 0x7FFFFFFF || N > 0x7FFFFFFF || (M > 0 && N > kMaxElems / M)) return MQ_ERR_INVALID_ARG;
    if (lda < K || ldb < K || ldy < N || a_hs < 0 || b_hs < 0 || y_hs < 0)
        return MQ_ERR_INVALID_ARG;
    if (!act_bits_ok(out_bits)) return MQ_ERR_INVALID_ARG;
    if (!finite_pos(a_scale) || !finite_pos(b_scale) || !finite_pos(out_scale))
        return MQ_ERR_INVALID_ARG;
    if (!zp_ok(a_zp, 16) || !zp_ok(b_zp, 8) || !zp_ok(out_zp, out_bits)) return MQ_ERR_INVALID_ARG;
    if (path != MQ_PATH_AUTO && path != MQ_PATH_PREFILL && path != MQ_PATH_GENERIC)
        return MQ_ERR_INVALID_ARG;
    int64_t off_cs, off_sc;
    const int64_t need = mq_attn_matmul_workspace_bytes(H, G, M, N);
    if (need < 0) return MQ_ERR_INVALID_ARG;
    attn_ws_parts(H, G, M, N, &off_cs, &off_sc);
    if (M == 0 || N == 0) return MQ_OK;
    if (!a || !b || !y || !workspace) return MQ_ERR_INVALID_ARG;
    if (workspace_bytes < need || ((uintptr_t)workspace % 256) != 0) return MQ_ERR_INVALID_ARG;

    hipStream_t s = as_stream(stream);
    int8_t* ws = static_cast<int8_t*>(workspace);
    int64_t* row_off = reinterpret_cast<int64_t*>(ws);
    int32_t* colsum = reinterpret_cast<int32_t*>(ws + off_cs);
    float* scale = reinterpret_cast<float*>(ws + off_sc);

    mq::QLinearArgs p;
    p.a = reinterpret_cast<const int8_t*>(a);
    p.a_bits = 16;
    p.w = b;
    p.w_scale = scale;
    p.ws_stride = 0;
    p.colsum = colsum;
    p.bias = nullptr;
    p.y = y;
    p.M = M;
    p.K = K;
    p.N = N;
    p.a_scale = a_scale;
    p.out_scale = out_scale;
    p.a_zp = a_zp;
    p.out_zp = out_zp;
    p.w_bits = 8;
    p.out_bits = out_bits;
    p.lda = lda;
    p.ldw = ldb;
    p.ldy = ldy;
    p.batch = H;
    p.group = H / G;
    p.a_bs = a_hs;
    p.w_bs = b_hs;
    p.y_bs = y_hs;
    p.cs_bs = N;
    p.ro_bs = M;
    p.row_off = b_zp != 0 ? row_off : nullptr;  // b_zp = 0: no row terms
    if (path == MQ_PATH_AUTO) path = M <= 16 ? MQ_PATH_GENERIC : MQ_PATH_PREFILL;
    const bool tiled = path == MQ_PATH_PREFILL && mq::prefill_supported(p);
    // the causal promises shorten the tiled kernel's work; the generic
    // kernel computes every output over all of K, which they also allow
    if (tiled) {
        p.out_causal = out_causal;
        p.in_causal = in_causal;
        if (in_causal >= 0) {
            p.cs_mt = N;
            p.cs_bs = ((M + mq::kA16TileM - 1) / mq::kA16TileM) * N;
        }
    }
    hipError_t e = mq::launch_attn_sums(a, lda, a_hs, H, M, b, ldb, b_hs, G, N, K, a_zp, b_zp,
                                        b_scale, row_off, colsum, scale, p.in_causal,
                                        mq::kA16TileM, mq::kA16TileK, s);
    if (e != hipSuccess) return MQ_ERR_HIP;
    return from_hip(tiled ? mq::launch_qlinear_prefill(p, s) : mq::launch_qlinear_generic(p, s));
}

mq_status mq_transpose_i8(const int8_t* x, int64_t rows, int64_t cols, int64_t ldx, int8_t* y,
                          void* stream)
{
    if (rows < 0 || cols < 0 || ldx < cols) return MQ_ERR_INVALID_ARG;
    if (rows > (int64_t)65535 * 64 || cols > kMaxElems || (rows > 0 && cols > kMaxElems / rows))
        return MQ_ERR_INVALID_ARG;
    if (rows == 0 || cols == 0) return MQ_OK;
    if (!x || !y) return MQ_ERR_INVALID_ARG;
    return from_hip(mq::launch_transpose_i8(x, rows, cols, ldx, y, as_stream(stream)));
}

}  // extern "C"
