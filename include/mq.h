/*
 * mq.h -- C ABI of the MI355X (gfx950) integer-only quantized linear layer
 * of MobileQuant (arXiv 2408.13933).
 *
 * The layer maps static per-tensor int8 activations and per-output-channel
 * symmetric int8 (or packed int4) weights to int8/int16 activations of the
 * next layer with integer arithmetic only: int32 accumulation, zero-point
 * and bias correction, a fixed-point multiplier and shift, saturation.
 *
 * Conventions shared by every entry point
 * ---------------------------------------
 * - Layout: row-major, the reduction (input-channel) dimension K contiguous.
 *     activations  A_q  int8          [M][K]
 *     weights      W_q  int8          [N][K]      (w_bits = 8)
 *                       uint8         [N][K/2]    (w_bits = 4): byte j of a
 *                       row holds the weight of input channel 2j in its low
 *                       nibble and of channel 2j+1 in its high nibble, as
 *                       two's-complement 4-bit integers
 *     outputs      Y_q  int8 / int16  [M][N]
 *   The paper writes Y = XW with W of shape [in][out]; here tokens are rows
 *   and each output channel owns one contiguous weight row.
 * - Pointers named as device pointers are HIP device memory (or memory the
 *   device can address) owned by the caller; the library never keeps,
 *   frees or allocates memory.  A pointer may be NULL only where its
 *   element count is 0 or where the comment says so.
 * - `stream` is a hipStream_t passed as void* (NULL = the null stream).  Device
 *   work is enqueued on it and the call returns without synchronising;
 *   errors raised while the kernels run surface at the caller's next
 *   synchronisation on that stream.
 * - Arguments are validated on the host before anything is enqueued; an
 *   invalid call returns MQ_ERR_INVALID_ARG and touches no memory.  A failed
 *   kernel launch returns MQ_ERR_HIP.  No C++ exception crosses this ABI.
 * - Activation formats are signed: bits = 8 stores [-128, 127], bits = 16
 *   stores [-32768, 32767].  The paper's unsigned code X_int in
 *   [0, 2^bw - 1] (Section 4.2, Eq.(4)) equals the stored value plus
 *   2^(bw-1); the zero-point carries the same shift.
 */
#ifndef MQ_H
#define MQ_H

#include <stdint.h>

#ifdef __cplusplus
extern "C" {
#endif

typedef enum {
    MQ_OK = 0,
    MQ_ERR_INVALID_ARG = 1,
    MQ_ERR_UNSUPPORTED = 2,
    MQ_ERR_HIP = 3
} mq_status;

/* Kernel path selection for mq_qlinear_ex (cross-checks and timing). */
typedef enum {
    MQ_PATH_AUTO = 0,     /* M <= 16 -> decode, otherwise prefill          */
    MQ_PATH_DECODE = 1,   /* wavefront GEMV kernel, any M <= 16            */
    MQ_PATH_PREFILL = 2,  /* LDS-tiled MFMA GEMM kernel, any M             */
    MQ_PATH_GENERIC = 3,  /* one thread per output, any shape or alignment */
    /* MQ_PATH_PREFILL_TILE0 + t, t = 0..MQ_PREFILL_TILES-1: the prefill
     * kernel with output tile t (0: 256x128, 1: 128x128, 2: 192x256,
     * 3: 64x64, 4: 256x256 on eight waves, 5: 128x64; tokens x channels)
     * instead of the one its cost model picks -- a hook for tests and
     * measurements;
     * the results are the same bits.  With a workspace the K split is the
     * cost model's best for that tile and may need more bytes than
     * mq_qlinear_workspace_bytes reports (at most 256*ceil(T/64) +
     * 8*T*tm*tn*4 bytes for T tiles of tm x tn); with fewer bytes it does
     * not split. */
    MQ_PATH_PREFILL_TILE0 = 16
} mq_path;
#define MQ_PREFILL_TILES 6

/* Largest K accepted: keeps |sum_k A_q W_q| below 2^30 so the int32
 * accumulator cannot overflow. */
#define MQ_MAX_K 65536

/* Human-readable name of a status code (static storage). */
const char* mq_status_string(mq_status status);

/* ABI version; bumped on any incompatible change. */
int32_t mq_version(void);

/*
 * mq_act_params -- static per-tensor activation format from a range.
 * Section 4.2, Eq.(2)-(3): q_max = 2^bw - 1, alpha = (f_max - f_min)/q_max,
 * beta = f_min/alpha.  The range is first widened to contain 0; alpha is
 * computed in fp64 and rounded once to fp32; the offset -beta is rounded
 * half-to-even to an integer and clamped to [0, q_max]; the signed
 * zero-point returned is round(-beta) - 2^(bw-1).  A zero-width range
 * gives alpha = 1 and zero-point -2^(bw-1).
 *   f_min, f_max  finite, f_min <= f_max
 *   bits          8 or 16
 *   alpha, zp     host pointers receiving the scale and signed zero-point
 * Host-only arithmetic; touches no device.
 */
mq_status mq_act_params(float f_min, float f_max, int32_t bits,
                        float* alpha, int32_t* zp);

/*
 * mq_fold_weights -- equivalent transformation of Section 3.2, Eq.(1):
 * Y = XW = (X S^-1)(S W).  With S = diag(s) on the input channels,
 *   w_hat[n][k] = w[n][k] * s[k]      (one fp32 multiply)
 *   w, w_hat  device fp32 [N][K] (may alias)   s  device fp32 [K]
 */
mq_status mq_fold_weights(const float* w, const float* s, int64_t N, int64_t K,
                          float* w_hat, void* stream);

/*
 * mq_fold_acts -- the activation side of Eq.(1):
 *   x_hat[m][k] = x[m][k] / s[k]      (one IEEE fp32 division)
 *   x, x_hat  device fp32 [M][K] (may alias)   s  device fp32 [K]
 */
mq_status mq_fold_acts(const float* x, const float* s, int64_t M, int64_t K,
                       float* x_hat, void* stream);

/*
 * mq_quantize_act -- static per-tensor activation quantizer, Section 4.2
 * Eq.(4) in signed storage:
 *   q = clamp(rint(x / alpha) + zp, -2^(bits-1), 2^(bits-1) - 1)
 * x/alpha is one IEEE fp32 division, rint rounds half to even; the
 * quotient is limited to +-2^20 first (NaN ends at the low end).
 *   x      device fp32 [numel]
 *   alpha  finite, > 0        zp  within the signed range of `bits`
 *   bits   8 (x_q is int8) or 16 (x_q is int16)
 *   x_q    device [numel]
 */
mq_status mq_quantize_act(const float* x, int64_t numel, float alpha, int32_t zp,
                          int32_t bits, void* x_q, void* stream);

/*
 * mq_pack_weights -- symmetric per-output-channel weight quantizer and
 * packer (Section 5.1 W8A8/W4A8 settings; appendix: symmetric per-channel
 * W4).  For each row n, with Q = 127 (bits 8) or 7 (bits 4):
 *   w_scale[n] = max_k |w[n][k]| / Q  (fp32; 1 when that is not > 0)
 *   q[n][k]    = rint(clamp(w[n][k] / w_scale[n], -Q, Q))
 *   w_colsum[n] = sum_k q[n][k]      (used for the zero-point correction)
 *   w        device fp32 [N][K], smoothing already folded (mq_fold_weights)
 *   bits     8 -> w_q int8 [N][K];  4 -> w_q uint8 [N][K/2] (K even)
 *   w_scale  device fp32 [N]          w_colsum  device int32 [N]
 *   1 <= K <= MQ_MAX_K.
 */
mq_status mq_pack_weights(const float* w, int64_t N, int64_t K, int32_t bits,
                          void* w_q, float* w_scale, int32_t* w_colsum,
                          void* stream);

/*
 * mq_qlinear -- integer-only linear layer (the hot path).  For every
 * token m and output channel n:
 *   acc      = sum_k A_q[m][k] * W_q[n][k]                     (int32)
 *   c        = sat_int32(acc - a_zp * w_colsum[n] + bias_q[n])
 *   M_n      = (a_scale * w_scale[n]) / out_scale   (fp64)  = M0 * 2^-sh,
 *              M0 = rint(f * 2^31) in [2^30, 2^31) for M_n = f * 2^e,
 *              f in [0.5, 1), sh = 31 - e
 *   r        = floor((c * M0 + 2^(sh-1)) / 2^sh)   (exact; 0 if sh >= 63;
 *              sh <= 0 saturates every non-zero c)
 *   Y_q[m][n] = clamp(r + out_zp, -2^(out_bits-1), 2^(out_bits-1) - 1)
 *   bias_q[n] = rint(clamp(bias[n] / (a_scale * w_scale[n]), -2^30, 2^30))
 *              in fp64, or 0 when bias is NULL.
 * The paper fixes integer-only execution with static per-tensor
 * activations and per-channel weights (Section 3.1, Section 5.1) but not
 * the rescale; this Q31 single-rounding form is the reading implemented.
 *   a_q       device int8 [M][K]
 *   w_q       device, layout of mq_pack_weights for w_bits (8 or 4)
 *   w_scale   device fp32 [N]     w_colsum  device int32 [N], equal to
 *             sum_k W_q[n][k] (as written by mq_pack_weights)
 *   a_scale, out_scale  finite, > 0
 *   a_zp      in [-128, 127]      out_zp within the range of out_bits
 *   out_bits  8 (y_q int8) or 16 (y_q int16)
 *   bias      device fp32 [N], or NULL
 *   y_q       device [M][N]; must not overlap the inputs
 *   M >= 0, N >= 0 (0 -> nothing to do), 1 <= K <= MQ_MAX_K, K even for
 *   w_bits = 4.  Any shape and alignment is accepted; 16-byte-aligned
 *   buffers with K % 16 == 0 (int8) or K % 32 == 0 (int4) take the tuned
 *   kernels.
 */
mq_status mq_qlinear(const int8_t* a_q, int64_t M, int64_t K, int64_t N,
                     const void* w_q, int32_t w_bits, const float* w_scale,
                     const int32_t* w_colsum, float a_scale, int32_t a_zp,
                     float out_scale, int32_t out_zp, int32_t out_bits,
                     const float* bias, void* y_q, void* stream);

/*
 * mq_qlinear_ex -- mq_qlinear with an explicit kernel path; every path
 * computes the same bits.  MQ_PATH_DECODE requires M <= 16; the tuned
 * paths fall back to MQ_PATH_GENERIC when the shape or alignment rules
 * above are not met.
 */
mq_status mq_qlinear_ex(const int8_t* a_q, int64_t M, int64_t K, int64_t N,
                        const void* w_q, int32_t w_bits, const float* w_scale,
                        const int32_t* w_colsum, float a_scale, int32_t a_zp,
                        float out_scale, int32_t out_zp, int32_t out_bits,
                        const float* bias, void* y_q, int32_t path, void* stream);

/*
 * mq_qlinear_workspace_bytes -- device workspace mq_qlinear_ws can use for
 * this shape to split the reduction over K across several work-groups per
 * output tile (for layers with few output tiles and a long K, e.g. the
 * down projections).  0: the shape is not split.  -1: invalid arguments
 * (negative sizes, K outside [1, MQ_MAX_K], bits other than 8/4 and 8/16).
 * The result depends only on the shape and bit widths.
 */
int64_t mq_qlinear_workspace_bytes(int64_t M, int64_t K, int64_t N, int32_t w_bits,
                                   int32_t out_bits);

/*
 * mq_qlinear_ws -- mq_qlinear_ex with a workspace for the K split.  Results
 * are bit-identical to mq_qlinear_ex: the slices' int32 partial sums are
 * added exactly before the requant.
 *   workspace        device memory owned by the caller, 256-byte aligned,
 *                    zero-filled once before its first use with this
 *                    library; every call leaves its counters at zero again.
 *                    NULL (or workspace_bytes below
 *                    mq_qlinear_workspace_bytes) -> no split.  Calls that may
 *                    run concurrently must not share a workspace.
 *   workspace_bytes  >= 0
 */
mq_status mq_qlinear_ws(const int8_t* a_q, int64_t M, int64_t K, int64_t N,
                        const void* w_q, int32_t w_bits, const float* w_scale,
                        const int32_t* w_colsum, float a_scale, int32_t a_zp,
                        float out_scale, int32_t out_zp, int32_t out_bits,
                        const float* bias, void* y_q, void* workspace,
                        int64_t workspace_bytes, int32_t path, void* stream);

/*
 * mq_qlinear_noalloc -- mq_qlinear for callers that cannot allocate device
 * memory: code under HIP graph capture, serving loops and harnesses that
 * forbid hipMalloc.  It allocates nothing (no hipMalloc, hipFree or
 * allocating library call).  Arguments and results are those of mq_qlinear;
 * the results are the bits mq_qlinear_ws gives with a workspace of
 * mq_qlinear_workspace_bytes(M, K, N, w_bits, out_bits) bytes, because that
 * K split runs here too, with its workspace in a static device array of
 * MQ_NOALLOC_SCRATCH_BYTES on each GPU (held from the library's load until
 * the process ends; the first call on a device looks up that device's copy).
 *   Returns MQ_ERR_UNSUPPORTED, launching nothing, when the shape's K split
 *   needs more than MQ_NOALLOC_SCRATCH_BYTES; other errors as mq_qlinear.
 *   Each call clears the arrival counters it uses with a fill kernel on
 *   `stream` (no memset node, so the call can be captured).  All calls on
 *   one GPU share that GPU's array and it keeps the last call's contents:
 *   calls that may overlap on one GPU (unordered streams, concurrent graph
 *   branches) race and give wrong results.
 */
#define MQ_NOALLOC_SCRATCH_BYTES (32 << 20)
mq_status mq_qlinear_noalloc(const int8_t* a_q, int64_t M, int64_t K, int64_t N,
                             const void* w_q, int32_t w_bits, const float* w_scale,
                             const int32_t* w_colsum, float a_scale, int32_t a_zp,
                             float out_scale, int32_t out_zp, int32_t out_bits,
                             const float* bias, void* y_q, void* stream);

/*
 * mq_pack_weights_asym -- asymmetric weight quantizer and packer (Section
 * 5.1: the W8A8 and W4A8 settings quantize weights asymmetrically over the
 * full integer range; W8A8 with one range per tensor except the MLP down
 * projection, W4A8 per output channel).  The Eq.(2)-(4) quantizer runs
 * over the range lo = min(0, min w), hi = max(0, max w) of the finite
 * entries of row n (per_tensor = 0) or of the whole matrix (per_tensor = 1):
 *   w_scale[n] = (float)((hi - lo) / (2^bits - 1))       (fp64, then fp32)
 *   w_zp[n]    = clamp(rint(-lo / w_scale[n]), 0, 2^bits - 1) - 2^(bits-1)
 *   q[n][k]    = clamp(rint(w[n][k] / w_scale[n]) + w_zp[n],
 *                      -2^(bits-1), 2^(bits-1) - 1)
 * with one IEEE fp32 division limited to +-2^20 (NaN ends at the low end).
 * A zero-width range gives w_scale 1 and w_zp -2^(bits-1).  Per tensor,
 * every row repeats the tensor's scale and zero-point, so the layer call
 * is the same for both granularities.
 *   w         device fp32 [N][K]
 *   bits      8 -> w_q int8 [N][K];  4 -> w_q uint8 [N][K/2] (K even,
 *             low nibble = even k)
 *   per_tensor  0 or 1
 *   w_scale   device fp32 [N]     w_zp  device int32 [N] (per tensor both
 *             also hold the per-row ranges between the launches of the call)
 *   w_colsum  device int32 [N], sum_k q[n][k]
 *   1 <= K <= MQ_MAX_K.
 */
mq_status mq_pack_weights_asym(const float* w, int64_t N, int64_t K, int32_t bits,
                               int32_t per_tensor, void* w_q, float* w_scale,
                               int32_t* w_zp, int32_t* w_colsum, void* stream);

/*
 * mq_act_rowsum -- rowsum[m] = sum_k a_q[m][k] (int32), the per-token
 * term the weight zero-points of mq_qlinear_asym multiply.  Compute it once
 * per quantized activation and share it among the layers that read it.
 *   a_q     device int8 [M][K]     rowsum  device int32 [M]
 *   M >= 0 (0 -> nothing to do), 1 <= K <= MQ_MAX_K.
 */
mq_status mq_act_rowsum(const int8_t* a_q, int64_t M, int64_t K, int32_t* rowsum,
                        void* stream);

/*
 * mq_quantize_act_rowsum -- mq_quantize_act at 8 bits on x [M][K] fused
 * with mq_act_rowsum of the codes it writes (one pass; the codes are those
 * of mq_quantize_act bit for bit).  For the activations that feed layers
 * with asymmetric weights.
 *   x       device fp32 [M][K]       x_q  device int8 [M][K]
 *   alpha   finite, > 0              zp   in [-128, 127]
 *   rowsum  device int32 [M]
 *   M >= 0 (0 -> nothing to do), 1 <= K <= MQ_MAX_K.
 */
mq_status mq_quantize_act_rowsum(const float* x, int64_t M, int64_t K, float alpha,
                                 int32_t zp, int8_t* x_q, int32_t* rowsum, void* stream);

/*
 * mq_qlinear_asym -- mq_qlinear_ws for asymmetric per-channel weights
 * (Section 5.1).  For every token m and output channel n:
 *   c = sat_int32( sum_k (A_q[m][k] - a_zp) * (W_q[n][k] - w_zp[n])
 *                  + bias_q[n] )
 * (the sum exact), then the requant of mq_qlinear.  The kernels evaluate
 * it as acc - a_zp * w_colsum[n] - w_zp[n] * (a_rowsum[m] - K * a_zp)
 * + bias_q[n].
 *   a_rowsum  device int32 [M], sum_k A_q[m][k] as written by
 *             mq_act_rowsum or mq_quantize_act_rowsum for this a_q (not
 *             checked: other values give other results)
 *   w_q, w_scale, w_zp, w_colsum  as written by mq_pack_weights_asym
 *             (w_zp device int32 [N], within the signed range of w_bits)
 *   everything else as in mq_qlinear_ws (same workspace rules; the split
 *   decision does not depend on the zero-points).
 */
mq_status mq_qlinear_asym(const int8_t* a_q, const int32_t* a_rowsum, int64_t M,
                          int64_t K, int64_t N, const void* w_q, int32_t w_bits,
                          const float* w_scale, const int32_t* w_zp,
                          const int32_t* w_colsum, float a_scale, int32_t a_zp,
                          float out_scale, int32_t out_zp, int32_t out_bits,
                          const float* bias, void* y_q, void* workspace,
                          int64_t workspace_bytes, int32_t path, void* stream);

/*
 * mq_qlinear_dequant -- mq_qlinear_ws (mq_qlinear_asym when w_zp and
 * a_rowsum are set) whose epilogue also writes the dequantized outputs,
 *   y[m][n] = out_scale * (float)(Y_q[m][n] - out_zp)
 * (the inverse of Eq.(4): mq_dequant of the codes, bit for bit), and the
 * codes Y_q themselves only when y_q is not NULL: for a layer whose codes
 * only feed the dequantization (the logits of the LM head), one pass
 * instead of a qlinear, a store of the codes and a dequantization pass
 * reading them back.
 *   y         device fp32 [M][N] (16-byte aligned with N % 4 == 0 for the
 *             tuned kernels); must not overlap the inputs or y_q
 *   y_q       device [M][N] codes (out_bits), or NULL
 *   a_rowsum, w_zp  both NULL (symmetric weights) or as for mq_qlinear_asym
 *   everything else as in mq_qlinear_ws.
 */
mq_status mq_qlinear_dequant(const int8_t* a_q, const int32_t* a_rowsum, int64_t M, int64_t K,
                             int64_t N, const void* w_q, int32_t w_bits, const float* w_scale,
                             const int32_t* w_zp, const int32_t* w_colsum, float a_scale,
                             int32_t a_zp, float out_scale, int32_t out_zp, int32_t out_bits,
                             const float* bias, void* y_q, float* y, void* workspace,
                             int64_t workspace_bytes, int32_t path, void* stream);

/* Most linears one mq_qlinear_group call takes. */
#define MQ_MAX_GROUP 4

/*
 * mq_qlinear_out -- one linear of an mq_qlinear_group call: what differs
 * between linears that read the same activations.
 */
typedef struct mq_qlinear_out {
    const void* w_q;          /* device, layout of mq_pack_weights for the call's w_bits */
    const float* w_scale;     /* device fp32 [N] */
    const int32_t* w_zp;      /* device int32 [N] (asymmetric weights), or NULL */
    const int32_t* w_colsum;  /* device int32 [N] */
    const float* bias;        /* device fp32 [N], or NULL */
    int64_t N;                /* output channels, >= 0 */
    float out_scale;          /* finite, > 0 */
    int32_t out_zp;           /* within the range of the call's out_bits */
    void* y_q;                /* device [M][N] int8 or int16 (out_bits); must not overlap
                                 the inputs or another linear's output */
} mq_qlinear_out;

/*
 * mq_qlinear_group -- the linears that read one activation input (the
 * query, key and value projections of an attention layer; the gate and
 * up projections of a gated MLP; Section 4.1's block), each the operation
 * of mq_qlinear (symmetric weights: every w_zp NULL) or mq_qlinear_asym
 * (every w_zp set, a_rowsum set) on a_q, bit for bit, in one call.  On the
 * prefill path (M > 16 with MQ_PATH_AUTO) with K % 16 == 0 (int8) or
 * K % 32 == 0 (int4) and 16-byte-aligned buffers, one launch takes the
 * output tiles of all the linears, so a set of small layers fills the chip
 * as one large one would; otherwise each linear runs on the path
 * mq_qlinear_ex would take with the same path argument.  No K split.
 *   a_q       device int8 [M][K]   a_rowsum  device int32 [M] or NULL (as
 *             for mq_qlinear_asym)
 *   w_bits, a_scale, a_zp, out_bits  as for mq_qlinear, shared
 *   outs      host array of n_outs linears, 1 <= n_outs <= MQ_MAX_GROUP;
 *             each N may differ (N = 0: that linear has nothing to do)
 *   path      as for mq_qlinear_ex; MQ_PATH_PREFILL_TILE0 + t forces tile
 *             t for the whole launch
 *   M >= 0, 1 <= K <= MQ_MAX_K.  Errors: MQ_ERR_INVALID_ARG when any
 *   linear's arguments are invalid (nothing is launched).
 */
mq_status mq_qlinear_group(const int8_t* a_q, const int32_t* a_rowsum, int64_t M, int64_t K,
                           int32_t w_bits, float a_scale, int32_t a_zp, int32_t out_bits,
                           const mq_qlinear_out* outs, int32_t n_outs, int32_t path,
                           void* stream);

/*
 * mq_qlinear_a16 -- mq_qlinear_ex with 16-bit activation codes (the W8A16
 * setting of Section 5.6: activations kept at 16 bits, 8-bit weights):
 *   c = sat_int32( sum_k (A_q[m][k] - a_zp) * W_q[n][k] + bias_q[n] )
 * with the sum exact, then the requant of mq_qlinear.  The kernels split
 * each code into its high byte and its low byte - 128 and run two int8
 * products (exact).
 *   a_q    device int16 [M][K] (as written by mq_quantize_act with bits 16)
 *   a_zp   in [-32768, 32767]
 *   w_q, w_bits, w_scale, w_colsum: symmetric weights as in mq_qlinear
 *   (the tuned prefill kernel takes w_bits 8; w_bits 4 runs on the decode
 *   kernel for M <= 16 and on the generic kernel otherwise).
 *   Everything else as in mq_qlinear_ex.
 */
mq_status mq_qlinear_a16(const int16_t* a_q, int64_t M, int64_t K, int64_t N,
                         const void* w_q, int32_t w_bits, const float* w_scale,
                         const int32_t* w_colsum, float a_scale, int32_t a_zp,
                         float out_scale, int32_t out_zp, int32_t out_bits,
                         const float* bias, void* y_q, int32_t path, void* stream);

/*
 * Decoder-block glue on 16-bit integer activations (Section 4.1 and 5.1:
 * the operators between the quantized linears keep 16-bit integer
 * activations).  The paper fixes the formats, not the arithmetic inside
 * the operators; here every operator dequantizes exactly, evaluates in
 * fp64 one IEEE operation at a time in the order written, and requantizes
 * with Eq.(4): code = clamp(rint(v / ay) + zy) over out_bits (8 or 16).
 * x codes are int16 with zero-points in the int16 range; all scales finite
 * and > 0.
 *
 * mq_add_requant -- residual add:
 *   v = a1 * (x1 - z1) + a2 * (x2 - z2)          x1, x2 device int16 [numel]
 */
mq_status mq_add_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                         float a2, int32_t z2, int64_t numel, float ay, int32_t zy,
                         int32_t out_bits, void* y, void* stream);

/*
 * mq_mul_requant -- product of two code tensors (the gated unit of the
 * feed-forward block, SiLU(gate) * up):
 *   v = (a1 * (x1 - z1)) * (a2 * (x2 - z2))      x1, x2 device int16 [numel]
 * each factor exact in fp64, the product one rounding.
 */
mq_status mq_mul_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                         float a2, int32_t z2, int64_t numel, float ay, int32_t zy,
                         int32_t out_bits, void* y, void* stream);

/*
 * mq_add_rmsnorm -- the residual add and the RMSNorm of its result in one
 * pass: h = mq_add_requant(x1, x2) as int16 codes in format (ah, zh),
 * written to h, and y = mq_rmsnorm(h) (gamma, eps, ay, zy, out_bits), with
 * the arithmetic of those two calls, so the same bits (rows that do not
 * fit the one-pass kernel run the two steps).
 *   x1, x2 device int16 [M][K]; h device int16 [M][K], written;
 *   y device int8 or int16 [M][K]; gamma device fp32 [K] or NULL
 *   1 <= K <= 2^20; scales finite and > 0; eps finite and >= 0.
 */
mq_status mq_add_rmsnorm(const int16_t* x1, float a1, int32_t z1, const int16_t* x2, float a2,
                         int32_t z2, int64_t M, int64_t K, float ah, int32_t zh, int16_t* h,
                         const float* gamma, float eps, float ay, int32_t zy, int32_t out_bits,
                         void* y, void* stream);

/*
 * mq_lut_mul -- a table lookup and the product of mq_mul_requant in one
 * pass (the gated unit SiLU(gate) * up with the SiLU codes kept out of
 * memory): u = lut[x1[i] + 32768], a code of the table's format (a1, z1),
 *   y[i] = code(a1 (u - z1) * a2 (x2[i] - z2))
 * with the arithmetic of mq_mul_requant, so y equals mq_lut_apply followed
 * by mq_mul_requant bit for bit.
 *   x1, x2 device int16 [numel]; lut device table of mq_lut_build,
 *   lut_bits 8 or 16 (its entries); y device int8 or int16 [numel]
 *   a1, a2, ay finite and > 0; z1 in the lut_bits range, z2 in int16,
 *   zy in the out_bits range.
 */
mq_status mq_lut_mul(const int16_t* x1, const void* lut, int32_t lut_bits, float a1, int32_t z1,
                     const int16_t* x2, float a2, int32_t z2, int64_t numel, float ay,
                     int32_t zy, int32_t out_bits, void* y, void* stream);

/*
 * mq_rope -- rotary position embedding on the query or key codes of a
 * Llama-family block (the paper's models; a non-linear operator kept at 16
 * bits): for token t, head h and pair i < D/2 (dimensions i and i + D/2 of
 * the head), with the angle (t + pos0) * base^(-2i/D):
 *   u = ax * (x[t][h*D + i] - zx),  w = ax * (x[t][h*D + i + D/2] - zx)
 *   y[t][h*D + i] = u cos - w sin,  y[t][h*D + i + D/2] = w cos + u sin
 * (fp64: inverse frequency by pow, the angle one product, cos and sin).
 *   x      device int16 [T][H * D]; y device int8 or int16 [T][H * D]
 *   table  device fp64 scratch of T * D values (the cos/sin table)
 *   T >= 0, H >= 1, D >= 2 even, base finite and > 1, 0 <= pos0 <= 2^40.
 */
mq_status mq_rope(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax, int32_t zx,
                  double base, int64_t pos0, float ay, int32_t zy, int32_t out_bits,
                  double* table, void* y, void* stream);

/*
 * mq_rope_table -- the angle table of mq_rope alone: table[2 (t D/2 + i)]
 * and table[2 (t D/2 + i) + 1] get cos and sin of (t + pos0) *
 * base^(-2i/D) for t < T, i < D/2 (the same fp64 evaluation as mq_rope).
 * The table depends only on T, D, base and pos0, so one table serves the
 * queries and keys of every layer.
 *   table  device fp64 [T * D], written
 *   T >= 0, D >= 2 even, base finite and > 1, 0 <= pos0 <= 2^40.
 */
mq_status mq_rope_table(int64_t T, int64_t D, double base, int64_t pos0, double* table,
                        void* stream);

/*
 * mq_rope_apply -- mq_rope's rotation and requantization with an angle
 * table made by mq_rope_table (same T and D); mq_rope equals
 * mq_rope_table followed by mq_rope_apply.
 *   x      device int16 [T][H * D]; y device int8 or int16 [T][H * D]
 *   table  device fp64 [T * D], read only
 */
mq_status mq_rope_apply(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax, int32_t zx,
                        const double* table, float ay, int32_t zy, int32_t out_bits, void* y,
                        void* stream);

/* Table operators of mq_lut_build. */
#define MQ_LUT_SILU 1

/*
 * mq_lut_build -- a 65536-entry table of an elementwise operator on int16
 * codes: lut[i + 32768] = code of f(ax * (i - zx)); op MQ_LUT_SILU:
 * f(v) = v / (1 + exp(-v)).  lut: device int8 or int16 [65536] (out_bits).
 * mq_lut_apply -- y[i] = lut[x[i] + 32768].
 */
mq_status mq_lut_build(int32_t op, float ax, int32_t zx, float ay, int32_t zy,
                       int32_t out_bits, void* lut, void* stream);
mq_status mq_lut_apply(const int16_t* x, int64_t numel, const void* lut, int32_t out_bits,
                       void* y, void* stream);

/*
 * mq_rmsnorm -- RMSNorm over each row of K codes:
 *   ss = sum_k (x - zx)^2 (exact),  ms = ax^2 * ss / K + eps,  r = sqrt(ms),
 *   v = ax * (x - zx) [* gamma[k]] / r
 *   x device int16 [M][K]; gamma device fp32 [K] or NULL; eps >= 0;
 *   1 <= K <= 2^20.
 */
mq_status mq_rmsnorm(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                     const float* gamma, float eps, float ay, int32_t zy, int32_t out_bits,
                     void* y, void* stream);

/*
 * mq_softmax -- softmax over each row of K score codes:
 *   e_k = exp(ax * (x_k - max_j x_j)),  p_k = e_k / sum_j e_j
 *   x device int16 [M][K]; 1 <= K <= 2^20.  For 16-bit probabilities over
 *   the unsigned range take ay = 1/65535, zy = -32768.
 */
mq_status mq_softmax(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx, float ay,
                     int32_t zy, int32_t out_bits, void* y, void* stream);

/*
 * mq_softmax_causal -- mq_softmax over the keys a decoder's causal
 * self-attention lets each query see: row m covers the keys
 * k <= (m mod period) + offset (the rows of one head are `period`
 * consecutive queries, `offset` the keys before the first of them); the
 * softmax runs over those keys and the others get probability 0 (code zy).
 *   period >= 1, offset >= 0; everything else as in mq_softmax.
 */
mq_status mq_softmax_causal(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                            float ay, int32_t zy, int32_t out_bits, int64_t period,
                            int64_t offset, void* y, void* stream);

/*
 * mq_smooth_scales -- SmoothQuant's closed-form scaling vector as the
 * paper restates it (Section 3.2), for calibration:
 *   x_absmax[k] = max_m |x[m][k]|,  w_absmax[k] = max_n |w[n][k]|
 *   s[k] = x_absmax[k]^a / w_absmax[k]^(1-a)   (fp64 pow, rounded to fp32)
 * over finite entries; s[k] = 1 where either maximum is 0.  Fold s with
 * mq_fold_weights / mq_fold_acts (Eq.(1)).
 *   x  device fp32 [M][K]   w  device fp32 [N][K]   a  in [0, 1]
 *   x_absmax, w_absmax, s  device fp32 [K]
 *   M, N >= 0 (0 rows give a maximum of 0), K >= 0 (0 -> nothing to do).
 */
mq_status mq_smooth_scales(const float* x, int64_t M, int64_t K, const float* w,
                           int64_t N, float a, float* x_absmax, float* w_absmax,
                           float* s, void* stream);

/*
 * mq_arl_forward -- activation range learning, the training form of
 * Section 4.2, Eq.(2)-(4) with learnable scale alpha and offset beta:
 *   y = alpha * (min(max(rint(x/alpha) - beta, 0), 2^bits - 1) + beta)
 * each step one fp32 operation, rint half to even (the straight-through
 * estimator only changes the backward pass).
 *   x, y   device fp32 [numel] (may alias)
 *   alpha  finite, > 0     beta  finite     bits in [2, 16]
 */
mq_status mq_arl_forward(const float* x, int64_t numel, float alpha, float beta,
                         int32_t bits, float* y, void* stream);

/* Partial sums mq_arl_backward keeps after its two results. */
#define MQ_ARL_PARTIALS 1024

/*
 * mq_arl_backward -- straight-through gradients of mq_arl_forward.  With
 * u = rint(x/alpha) - beta and mask = (0 <= u <= 2^bits - 1):
 *   gx[i]    = g[i] * mask
 *   grads[0] = sum_i g[i] * ((clamp(u) + beta) - mask * x[i]/alpha)   (dL/dalpha)
 *   grads[1] = sum_i g[i] * alpha * (1 - mask)                        (dL/dbeta)
 * per-element terms and sums in fp64; the sum runs over fixed per-block
 * partials in block order, so a given numel always sums in the same order.
 *   x, g, gx  device fp32 [numel]
 *   grads     device fp64 [2 + 2 * MQ_ARL_PARTIALS]: the two results, then
 *             scratch for the partial sums
 */
mq_status mq_arl_backward(const float* x, const float* g, int64_t numel, float alpha,
                          float beta, int32_t bits, float* gx, double* grads,
                          void* stream);

/*
 * mq_attn_matmul -- the batched integer matmuls of self-attention.  In the
 * W8A16 setting (Section 5.6) the attention products multiply 16-bit by
 * 8-bit activation codes; both operands are per-tensor quantized
 * activations (Eq.(2)-(4)) with their own zero-points.  For every head h
 * in [0, H), with group g = h / (H / G) (grouped-query attention: G heads
 * of keys and values):
 *   c[h][m][n] = sat_int32( sum_k (A[h][m][k] - a_zp) * (B[g][n][k] - b_zp) )
 * (the sum exact), then the requant of mq_qlinear with
 * M = a_scale * b_scale / out_scale and no bias.
 *   Q K^T: A = query codes (m = query token, k = head dimension), B = key
 *          codes (n = key token).
 *   P V:   A = probability codes (k = key token), B = value codes in the
 *          [group][head dimension][token] layout (mq_transpose_i8 of the
 *          [token][G * head dimension] value matrix).
 *   a         device int16; element (h, m, k) at a[h * a_hs + m * lda + k]
 *   b         device int8;  element (g, n, k) at b[g * b_hs + n * ldb + k]
 *   y         device int8 (out_bits 8) or int16 (16); element (h, m, n) at
 *             y[h * y_hs + m * ldy + n]
 *   H >= 1, G >= 1, H % G == 0; M, N >= 0 (0 -> nothing to do);
 *   1 <= K <= MQ_MAX_K; lda, ldb >= K; ldy >= N; strides >= 0, in elements
 *   a_zp in [-32768, 32767], b_zp in [-128, 127], out_zp in the range of
 *   out_bits; scales finite and > 0
 *   out_causal >= 0: outputs y[h][m][n] with n > m + out_causal are not
 *              needed and may be left unwritten (Q K^T of a causal decoder,
 *              out_causal = keys before the first query); -1: all
 *   in_causal  >= 0: the caller promises A[h][m][k] == a_zp for
 *              k > m + in_causal (P V with causal probabilities, whose
 *              hidden keys hold the probability-0 code), so they may be
 *              skipped; -1: none
 *   workspace  device, 256-byte aligned, >= mq_attn_matmul_workspace_bytes
 *              bytes; overwritten with the per-row zero-point terms, the
 *              per-row sums of B and b_scale (calls that may run
 *              concurrently must not share it)
 *   path       MQ_PATH_AUTO (tiled MFMA kernel for M > 16 when the strides
 *              keep 16-byte aligned rows, else the generic kernel),
 *              MQ_PATH_PREFILL or MQ_PATH_GENERIC
 *   out_causal, in_causal in [-1, 2^40]
 * Errors: MQ_ERR_INVALID_ARG for any violation above.
 */
int64_t mq_attn_matmul_workspace_bytes(int32_t H, int32_t G, int64_t M, int64_t N);
mq_status mq_attn_matmul(const int16_t* a, int64_t lda, int64_t a_hs, int32_t H,
                         const int8_t* b, int64_t ldb, int64_t b_hs, int32_t G, int64_t M,
                         int64_t N, int64_t K, float a_scale, int32_t a_zp, float b_scale,
                         int32_t b_zp, float out_scale, int32_t out_zp, int32_t out_bits,
                         void* y, int64_t ldy, int64_t y_hs, int64_t out_causal,
                         int64_t in_causal, void* workspace, int64_t workspace_bytes,
                         int32_t path, void* stream);

/*
 * mq_transpose_i8 -- y[c][r] = x[r][c] for an int8 [rows][cols] matrix with
 * row stride ldx (elements); y is dense [cols][rows].  Lays the value codes
 * out as the B operand of the P V product in mq_attn_matmul.
 *   0 <= rows <= 65535 * 64, cols >= 0, ldx >= cols; x, y device.
 */
mq_status mq_transpose_i8(const int8_t* x, int64_t rows, int64_t cols, int64_t ldx,
                          int8_t* y, void* stream);

/*
 * mq_dequant -- inverse of Eq.(4): y = alpha * (float)(q - zp), one exact
 * integer subtraction and one fp32 multiply.
 *   q      device int8 (bits 8) or int16 (bits 16) [numel]
 *   alpha  finite, > 0     zp  within the signed range of `bits`
 *   y      device fp32 [numel]
 */
mq_status mq_dequant(const void* q, int32_t bits, int64_t numel, float alpha,
                     int32_t zp, float* y, void* stream);

/*
 * mq_probe_read -- a measurement helper, not a step of the method: reads
 * `bytes` bytes of device memory at `src` with `blocks` work-groups of
 * `waves` wavefronts (the grid of the kernel whose memory floor is being
 * measured).  Block b reads bytes [b*per, (b+1)*per), per = bytes/blocks
 * rounded up to 1 KiB, as 1 KiB wave loads (16 bytes per lane, the
 * non-temporal cache policy of the decode kernels' weight loads) with
 * `unroll` loads per lane in flight per round.  Each wave writes the XOR of
 * what it read to sink[b*waves + w], so no load can be dropped.
 *   src    device, any alignment of 16 bytes or more (null when bytes == 0)
 *   bytes  >= 0, bytes/blocks < 2^31    blocks > 0    waves in [1, 16]
 *   unroll 1, 2, 4, 8 or 16
 *   sink   device int32 [blocks * waves], written
 * Errors: MQ_ERR_INVALID_ARG for a violation above, MQ_ERR_UNSUPPORTED for
 * a per-block range of 2 GiB or more, MQ_ERR_HIP for a failed launch.
 */
mq_status mq_probe_read(const void* src, int64_t bytes, int32_t blocks, int32_t waves,
                        int32_t unroll, int32_t* sink, void* stream);

#ifdef __cplusplus
}
#endif

#endif /* MQ_H */
