// Internal declarations shared by the host entry points and the kernel
// translation units of libmq.  Not part of the public ABI.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>

#include "mq.h"

namespace mq {

// Scalars every qlinear kernel needs besides its buffers.
struct QLinearArgs {
    const int8_t* a;        // [M][K] int8, or int16 when a_bits == 16 (byte pointer)
    const void* w;          // [N][K] int8 or [N][K/2] packed int4
    const float* w_scale;   // [N]
    const int32_t* colsum;  // [N]
    const float* bias;      // [N] or nullptr
    void* y;                // [M][N] int8 or int16, or nullptr when y_f is set
    // [M][N] fp32, out_scale * (y - out_zp) written by the same pass (the
    // dequantized outputs), or nullptr; dense 8-bit-activation products only
    float* y_f = nullptr;
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
    // Row strides in elements (0: dense, K for a and w, N for y).
    int64_t lda = 0, ldw = 0, ldy = 0;
    // Batched products (the attention matmuls): batch b reads a, y, row_off
    // at b times their batch strides and w, colsum at (b / group) times
    // theirs; w_scale[n * ws_stride] (0: one scale for every n).
    int32_t batch = 1, group = 1;
    int64_t a_bs = 0, w_bs = 0, y_bs = 0, cs_bs = 0, ro_bs = 0;
    int32_t ws_stride = 1;
    // per-row int64 term added to the exact sum before the saturation (the
    // zero-point term of a per-tensor asymmetric "weight" operand), or nullptr
    const int64_t* row_off = nullptr;
    // Causal structure of self-attention (16-bit tile only; the other
    // kernels compute everything, which these promises allow):
    // out_causal >= 0: outputs y[m][n] with n > m + out_causal are not
    //   needed (tiles wholly beyond that boundary are skipped);
    // in_causal >= 0: a[m][k] == a_zp for k > m + in_causal, so a tile's K
    //   range stops at the stage holding its last row's boundary, and
    //   colsum holds, per 128-row tile (stride cs_mt), the column sums over
    //   that range.
    int64_t out_causal = -1, in_causal = -1, cs_mt = 0;
    // prefill tile requested explicitly (0..MQ_PREFILL_TILES-1), or -1: chosen by
    // the cost model
    int32_t force_tile = -1;
};

// Several linears on one activation input in one prefill launch: the
// fields of each that differ (the shared ones stay in QLinearArgs).  tile0
// and tiles_n are set by the launch: the linear's first tile index and its
// tile columns.
constexpr int kMaxGroup = MQ_MAX_GROUP;
struct GroupPart {
    const void* w;
    const float* w_scale;
    const int32_t* colsum;
    const float* bias;
    const int32_t* w_zp;
    void* y;
    int64_t N;
    float out_scale;
    int32_t out_zp;
    int32_t tile0;
    int32_t tiles_n;
};
struct GroupArgs {
    GroupPart part[kMaxGroup];
    int32_t n;
};

// Dense defaults of the stride fields.
__host__ __device__ inline int64_t eff_lda(const QLinearArgs& p) { return p.lda ? p.lda : p.K; }
__host__ __device__ inline int64_t eff_ldw(const QLinearArgs& p) { return p.ldw ? p.ldw : p.K; }
__host__ __device__ inline int64_t eff_ldy(const QLinearArgs& p) { return p.ldy ? p.ldy : p.N; }

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
hipError_t launch_lut_mul(const int16_t* x1, const void* lut, int32_t lut_bits, float a1,
                          int32_t z1, const int16_t* x2, float a2, int32_t z2, int64_t n,
                          float ay, int32_t zy, int32_t bits, void* y, hipStream_t st);
hipError_t launch_add_rmsnorm(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                             float a2, int32_t z2, int64_t M, int64_t K, float ah, int32_t zh,
                             int16_t* h, const float* gamma, float eps, float ay, int32_t zy,
                             int32_t bits, void* y, hipStream_t st);
hipError_t launch_mul_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                              float a2, int32_t z2, int64_t n, float ay, int32_t zy,
                              int32_t bits, void* y, hipStream_t st);
hipError_t launch_rope_table(int64_t T, int64_t D, double base, int64_t pos0, double* table,
                             hipStream_t st);
hipError_t launch_rope_apply(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax,
                             int32_t zx, const double* table, float ay, int32_t zy, int32_t bits,
                             void* y, hipStream_t st);
hipError_t launch_rope(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax, int32_t zx,
                       double base, int64_t pos0, float ay, int32_t zy, int32_t bits,
                       double* table, void* y, hipStream_t st);
hipError_t launch_lut_build(int32_t op, float ax, int32_t zx, float ay, int32_t zy, int32_t bits,
                            void* lut, hipStream_t st);
hipError_t launch_lut_apply(const int16_t* x, int64_t n, const void* lut, int32_t bits, void* y,
                            hipStream_t st);
hipError_t launch_rmsnorm(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                          const float* gamma, float eps, float ay, int32_t zy, int32_t bits,
                          void* y, hipStream_t st);
hipError_t launch_softmax(const int16_t* x, int64_t M, int64_t K, float ax, float ay, int32_t zy,
                          int32_t bits, int64_t period, int64_t offset, void* y, hipStream_t st);

hipError_t launch_attn_sums(const int16_t* a, int64_t lda, int64_t a_bs, int32_t H, int64_t M,
                            const int8_t* b, int64_t ldb, int64_t b_bs, int32_t G, int64_t N,
                            int64_t K, int32_t a_zp, int32_t b_zp, float b_scale,
                            int64_t* row_off, int32_t* colsum, float* scale_out,
                            int64_t in_causal, int64_t tile_m, int64_t tile_k, hipStream_t s);

// Token rows and K codes per stage of the 16-bit prefill tiles (the causal
// K range and the per-block column sums of the attention products follow
// them).
constexpr int kA16TileM = 128, kA16TileK = 64;
hipError_t launch_transpose_i8(const int8_t* x, int64_t rows, int64_t cols, int64_t ldx,
                               int8_t* y, hipStream_t s);

hipError_t launch_qlinear_generic(const QLinearArgs& p, hipStream_t s);
hipError_t launch_qlinear_decode(const QLinearArgs& p, hipStream_t s);
// one token (M = 1, 8-bit codes): the vector-ALU GEMV the decode path takes
hipError_t launch_qlinear_gemv(const QLinearArgs& p, hipStream_t s);
bool gemv_supported(const QLinearArgs& p);
hipError_t launch_qlinear_prefill(const QLinearArgs& p, hipStream_t s);
// the linears of g on p's input (8-bit codes, dense, every part meeting
// prefill_supported), one launch, no K split
hipError_t launch_qlinear_prefill_group(const QLinearArgs& p, GroupArgs g, hipStream_t s);

// Workspace bytes the prefill kernel would use to split K for this shape
// (0 when it would not split).
int64_t prefill_workspace_bytes(const QLinearArgs& p);

// Bytes at the start of the split-K workspace that hold the per-tile
// arrival counters for this shape (0 when it would not split).
int64_t prefill_counter_bytes(const QLinearArgs& p);

// Shape/alignment rules of the tuned kernels.
bool decode_supported(const QLinearArgs& p);
bool prefill_supported(const QLinearArgs& p);

// Host side of the qlinear entry points: validation (fills the kernel
// arguments and resolves MQ_PATH_AUTO and the tile paths) and the launch.
mq_status qlinear_validate(const void* a_q, int32_t a_bits, const int32_t* a_rowsum, int64_t M,
                           int64_t K, int64_t N, const void* w_q, int32_t w_bits,
                           const float* w_scale, const int32_t* w_zp, const int32_t* w_colsum,
                           float a_scale, int32_t a_zp, float out_scale, int32_t out_zp,
                           int32_t out_bits, const float* bias, void* y_q, void* workspace,
                           int64_t workspace_bytes, int32_t path, QLinearArgs* out,
                           int32_t* path_out, float* y_f = nullptr);
mq_status qlinear_dispatch(const QLinearArgs& p, int32_t path, hipStream_t s);

}  // namespace mq
