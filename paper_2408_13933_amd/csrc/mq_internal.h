// Internal declarations shared by the host entry points and the kernel
// translation units of libmq.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

namespace mq {

// Scalars every qlinear kernel needs besides its buffers.
struct QLinearArgs {
    const int8_t* a;        // [M][K] int8, or int16 when a_bits == 16 (byte pointer)
    const void* w;          // [N][K] int8 or [N][K/2] packed int4
    const float* w_scale;   // [N]
    const int32_t* colsum;  // [N]
    const float* bias;      // [N] or nullptr
    void* y;                // [M][N] int8 or int16
    int64_t M, K, N;
    float a_scale;
    float out_scale;
    int32_t a_zp;
    int32_t out_zp;
    int32_t w_bits;         // 8 or 4
    int32_t out_bits;       // 8 or 16
    void* ws = nullptr;     // split-K workspace (zero-filled once by its owner) or nullptr
    int64_t ws_bytes = 0;
    // asymmetric per-channel weights: zero-points [N] and the activation
    // row sums [M] (sum_k a[m][k]); both nullptr for symmetric weights
    const int32_t* w_zp = nullptr;
    const int32_t* a_rowsum = nullptr;
    int32_t a_bits = 8;     // 8, or 16 (W8A16: 16-bit activation codes)
};

hipError_t launch_quantize_act(const float* x, int64_t n, float alpha, int32_t zp,
                               int32_t bits, void* q, hipStream_t s);
hipError_t launch_dequant(const void* q, int32_t bits, int64_t n, float alpha,
                          int32_t zp, float* y, hipStream_t s);
hipError_t launch_fold_weights(const float* w, const float* sv, int64_t N, int64_t K,
                               float* out, hipStream_t s);
hipError_t launch_fold_acts(const float* x, const float* sv, int64_t M, int64_t K,
                            float* out, hipStream_t s);
hipError_t launch_pack_weights(const float* w, int64_t N, int64_t K, int32_t bits,
                               void* wq, float* scale, int32_t* colsum, hipStream_t s);
hipError_t launch_pack_weights_asym(const float* w, int64_t N, int64_t K, int32_t bits,
                                    bool per_tensor, void* wq, float* scale, int32_t* zp,
                                    int32_t* colsum, hipStream_t s);
hipError_t launch_quantize_act_rowsum(const float* x, int64_t M, int64_t K, float alpha,
                                      int32_t zp, int8_t* q, int32_t* rowsum, hipStream_t s);
hipError_t launch_act_rowsum(const int8_t* a, int64_t M, int64_t K, int32_t* rowsum,
                             hipStream_t s);

hipError_t launch_arl_forward(const float* x, int64_t n, float alpha, float beta, int32_t bits,
                              float* y, hipStream_t s);
hipError_t launch_arl_backward(const float* x, const float* g, int64_t n, float alpha, float beta,
                               int32_t bits, float* gx, double* grads, int32_t max_partials,
                               hipStream_t s);
hipError_t launch_smooth_scales(const float* x, int64_t M, int64_t K, const float* w, int64_t N,
                                float a, float* x_absmax, float* w_absmax, float* s,
                                hipStream_t st);

hipError_t launch_add_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                              float a2, int32_t z2, int64_t n, float ay, int32_t zy,
                              int32_t bits, void* y, hipStream_t st);
hipError_t launch_lut_build(int32_t op, float ax, int32_t zx, float ay, int32_t zy, int32_t bits,
                            void* lut, hipStream_t st);
hipError_t launch_lut_apply(const int16_t* x, int64_t n, const void* lut, int32_t bits, void* y,
                            hipStream_t st);
hipError_t launch_rmsnorm(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                          const float* gamma, float eps, float ay, int32_t zy, int32_t bits,
                          void* y, hipStream_t st);
hipError_t launch_softmax(const int16_t* x, int64_t M, int64_t K, float ax, float ay, int32_t zy,
                          int32_t bits, void* y, hipStream_t st);

hipError_t launch_qlinear_generic(const QLinearArgs& p, hipStream_t s);
hipError_t launch_qlinear_decode(const QLinearArgs& p, hipStream_t s);
hipError_t launch_qlinear_prefill(const QLinearArgs& p, hipStream_t s);

// Workspace bytes the prefill kernel would use to split K for this shape
// (0 when it would not split).
int64_t prefill_workspace_bytes(const QLinearArgs& p);

// Shape/alignment rules of the tuned kernels.
bool decode_supported(const QLinearArgs& p);
bool prefill_supported(const QLinearArgs& p);

}  // namespace mq
