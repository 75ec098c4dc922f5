/*
 * mq_oracle.c -- plain, slow CPU oracle of MobileQuant's integer-only
 * quantized linear layer (arXiv 2408.13933).
 *
 * TEST INFRASTRUCTURE ONLY.  This file exists to check the HIP library
 * against the paper.  Only the test suite, the smoke check and the CPU
 * baseline leg of the benchmark may load it.  The product never calls it
 * and it shares no code, header, table or helper with the HIP sources.
 *
 * Every function below is the definition written out with plain loops,
 * int64 accumulation and IEEE fp32/fp64 (compile with -O2, no fast-math,
 * -ffp-contract=off).  Where the paper is silent the reading used is named
 * in the comment (the same readings are listed in the design notes).
 *
 * Storage conventions (the paper writes Y = XW with W of shape
 * [in, out]; here tokens are rows):
 *   A_q  int8   [M][K]   activations, K contiguous
 *   W_q  int8   [N][K]   weights, K contiguous  (bits = 8)
 *        uint8  [N][K/2] two int4 weights per byte (bits = 4):
 *                        low nibble = even k, high nibble = odd k,
 *                        two's-complement nibbles
 *   Y_q  int8 / int16 [M][N]
 */
#include <math.h>
#include <pthread.h>
#include <stdint.h>
#include <stdlib.h>
#include <string.h>

/* ------------------------------------------------------------------ */
/* integer helpers                                                     */
/* ------------------------------------------------------------------ */
static int64_t clamp_i64(int64_t v, int64_t lo, int64_t hi)
{
    return v < lo ? lo : (v > hi ? hi : v);
}

static int64_t qmin_of(int bits) { return -((int64_t)1 << (bits - 1)); }
static int64_t qmax_of(int bits) { return ((int64_t)1 << (bits - 1)) - 1; }

static void store_q(void* dst, int bits, int64_t i, int64_t v)
{
    if (bits == 8)
        ((int8_t*)dst)[i] = (int8_t)v;
    else
        ((int16_t*)dst)[i] = (int16_t)v;
}

static int64_t load_q(const void* src, int bits, int64_t i)
{
    return bits == 8 ? ((const int8_t*)src)[i] : ((const int16_t*)src)[i];
}

/* ------------------------------------------------------------------ */
/* Activation range -> (alpha, zero-point)                             */
/* Section 4.2, Eq.(2)-(3): q_max = 2^bw - 1, alpha = (f_max-f_min)/q_max,
 * beta = f_min/alpha.
 * Readings: the range is widened to contain 0; the offset -beta is
 * rounded half-to-even to an integer zero-point and clamped to
 * [0, q_max]; values are stored signed, shifted by 2^(bw-1), so the
 * signed zero-point is round(-beta) - 2^(bw-1).  alpha is computed in
 * fp64 and rounded once to fp32.  A zero-width range gives alpha = 1,
 * beta = 0.                                                            */
/* ------------------------------------------------------------------ */
int oracle_act_params(float f_min, float f_max, int bits,
                      float* alpha_out, int32_t* zp_out)
{
    if (bits != 8 && bits != 16) return 1;
    if (!isfinite(f_min) || !isfinite(f_max) || f_min > f_max) return 1;
    double lo = f_min < 0.0f ? (double)f_min : 0.0;
    double hi = f_max > 0.0f ? (double)f_max : 0.0;
    double q_max = (double)(((int64_t)1 << bits) - 1);     /* Eq.(2) */
    float alpha;
    double beta;
    if (hi - lo == 0.0) {
        alpha = 1.0f;
        beta = 0.0;
    } else {
        alpha = (float)((hi - lo) / q_max);                /* Eq.(3) */
        if (!(alpha > 0.0f) || !isfinite(alpha)) return 1;
        beta = lo / (double)alpha;                         /* Eq.(3) */
    }
    double zu = rint(-beta);
    if (zu < 0.0) zu = 0.0;
    if (zu > q_max) zu = q_max;
    *alpha_out = alpha;
    *zp_out = (int32_t)((int64_t)zu - ((int64_t)1 << (bits - 1)));
    return 0;
}

/* ------------------------------------------------------------------ */
/* Activation quantizer, Section 4.2 Eq.(4):
 *   X_int = min(max(round(X/alpha) - beta, 0), q_max)
 * in signed storage: q = clamp(rint(x/alpha) + zp, -2^(bw-1), 2^(bw-1)-1).
 * x/alpha is one IEEE fp32 division, rint is half-to-even.  The quotient
 * is first limited to +-2^20 so that it converts to an integer; NaN takes
 * the fmaxf/fminf convention (the non-NaN bound) and ends at the low end.  */
/* ------------------------------------------------------------------ */
void oracle_quantize_act(const float* x, int64_t n, float alpha, int32_t zp,
                         int bits, void* q)
{
    const float lim = 1048576.0f; /* 2^20 */
    for (int64_t i = 0; i < n; ++i) {
        float t = x[i] / alpha;
        t = fminf(fmaxf(t, -lim), lim);
        int64_t v = (int64_t)rintf(t) + zp;
        store_q(q, bits, i, clamp_i64(v, qmin_of(bits), qmax_of(bits)));
    }
}

/* ------------------------------------------------------------------ */
/* Dequantization: the inverse map of Eq.(4), y = alpha * (q - zp), one
 * exact integer subtraction and one fp32 multiply.                    */
/* ------------------------------------------------------------------ */
void oracle_dequant(const void* q, int bits, int64_t n, float alpha,
                    int32_t zp, float* y)
{
    for (int64_t i = 0; i < n; ++i) {
        int64_t d = load_q(q, bits, i) - zp;
        y[i] = alpha * (float)d;
    }
}

/* ------------------------------------------------------------------ */
/* Equivalent transformation, Section 3.2 Eq.(1): Y = X W = (X S^-1)(S W).
 * With S = diag(s) on the input channels: W_hat[n][k] = W[n][k] * s[k]
 * and X_hat[m][k] = X[m][k] / s[k], one fp32 rounding each.            */
/* ------------------------------------------------------------------ */
void oracle_fold_weights(const float* w, const float* s, int64_t N, int64_t K,
                         float* w_hat)
{
    for (int64_t n = 0; n < N; ++n)
        for (int64_t k = 0; k < K; ++k)
            w_hat[n * K + k] = w[n * K + k] * s[k];
}

void oracle_fold_acts(const float* x, const float* s, int64_t M, int64_t K,
                      float* x_hat)
{
    for (int64_t m = 0; m < M; ++m)
        for (int64_t k = 0; k < K; ++k)
            x_hat[m * K + k] = x[m * K + k] / s[k];
}

/* ------------------------------------------------------------------ */
/* SmoothQuant's closed-form scaling vector, as the paper restates it in
 * Section 3.2: s_k = max_m |X[m][k]|^a / max_n |W[n][k]|^(1-a) for each
 * input channel k, a the migration strength in [0, 1].  Readings: the
 * maxima run over finite entries; in fp64 with pow, rounded once to
 * fp32; a channel whose activation or weight maximum is 0 gets s = 1.
 * The column maxima are returned as well.                              */
/* ------------------------------------------------------------------ */
void oracle_smooth_scales(const float* x, int64_t M, int64_t K, const float* w,
                          int64_t N, float a, float* x_absmax, float* w_absmax,
                          float* s)
{
    for (int64_t k = 0; k < K; ++k) {
        float mx = 0.0f, mw = 0.0f;
        for (int64_t m = 0; m < M; ++m) {
            const float v = fabsf(x[m * K + k]);
            if (isfinite(v) && v > mx) mx = v;
        }
        for (int64_t n = 0; n < N; ++n) {
            const float v = fabsf(w[n * K + k]);
            if (isfinite(v) && v > mw) mw = v;
        }
        x_absmax[k] = mx;
        w_absmax[k] = mw;
        s[k] = (mx > 0.0f && mw > 0.0f)
                   ? (float)(pow((double)mx, (double)a) / pow((double)mw, 1.0 - (double)a))
                   : 1.0f;
    }
}

/* ------------------------------------------------------------------ */
/* Activation range learning (Section 4.2, Eq.(2)-(4)), the training-time
 * form with learnable scale alpha and offset beta (both real):
 *   X_int = min(max(ste(X/alpha) - beta, 0), q_max),  q_max = 2^bw - 1
 * Readings: ste rounds half to even in the forward pass and has
 * derivative 1 in the backward pass; the simulated (fake-quantized)
 * value is the inverse map X_hat = alpha * (X_int + beta); every forward
 * step is one fp32 operation.  Backward, with mask = (0 <= u <= q_max),
 * u = rint(X/alpha) - beta (the clamp passes the gradient at its ends):
 *   dX_hat/dX     = mask
 *   dX_hat/dalpha = (X_int + beta) - mask * X/alpha
 *   dX_hat/dbeta  = alpha * (1 - mask)
 * so outside the range X_hat is f_min = alpha beta or f_max = alpha q_max
 * + alpha beta, the two ends the paper learns through alpha and beta.
 * The parameter gradients are sums over the tensor, per-element terms in
 * fp64 from the fp32 values, accumulated in fp64.                      */
/* ------------------------------------------------------------------ */
void oracle_arl_forward(const float* x, int64_t n, float alpha, float beta, int bits,
                        float* y)
{
    const float q_max = (float)(((int64_t)1 << bits) - 1);      /* Eq.(2) */
    for (int64_t i = 0; i < n; ++i) {
        const float t = x[i] / alpha;
        const float u = rintf(t) - beta;                         /* Eq.(4) */
        const float c = fminf(fmaxf(u, 0.0f), q_max);
        y[i] = alpha * (c + beta);
    }
}

void oracle_arl_backward(const float* x, const float* g, int64_t n, float alpha,
                         float beta, int bits, float* gx, double* g_alpha,
                         double* g_beta)
{
    const float q_max = (float)(((int64_t)1 << bits) - 1);
    double ga = 0.0, gb = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        const float t = x[i] / alpha;
        const float u = rintf(t) - beta;
        const float c = fminf(fmaxf(u, 0.0f), q_max);
        const int in = u >= 0.0f && u <= q_max;
        gx[i] = in ? g[i] : 0.0f;
        const double da = (double)c + (double)beta - (in ? (double)t : 0.0);
        const double db = in ? 0.0 : (double)alpha;
        ga += (double)g[i] * da;
        gb += (double)g[i] * db;
    }
    *g_alpha = ga;
    *g_beta = gb;
}

/* ------------------------------------------------------------------ */
/* Decoder-block glue on integer activations (Section 4.1: the
 * non-linear operators keep 16-bit integer activations; Section 5.1).
 * The paper fixes the formats, not the arithmetic inside the operators.
 * Readings: inputs are dequantized exactly (an fp32 scale times an
 * integer of at most 17 bits is exact in fp64), each operator is
 * evaluated in fp64 one IEEE operation at a time in the order written
 * below, and the result is requantized with the Eq.(4) quantizer:
 * code = clamp(rint(v / alpha_y) + zp_y) (rint half to even).          */
/* ------------------------------------------------------------------ */
static int64_t requant_f64(double v, float alpha_y, int32_t zp_y, int bits_y)
{
    double t = v / (double)alpha_y;
    if (!(t == t)) t = -1e300;                         /* NaN -> low end */
    if (t > 1e18) t = 1e18;
    if (t < -1e18) t = -1e18;
    return clamp_i64((int64_t)rint(t) + zp_y, qmin_of(bits_y), qmax_of(bits_y));
}

/* residual add: v = alpha_1 (x1 - zp_1) + alpha_2 (x2 - zp_2)          */
void oracle_add_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                        float a2, int32_t z2, int64_t n, float ay, int32_t zy, int bits_y,
                        void* y)
{
    for (int64_t i = 0; i < n; ++i) {
        const double v = (double)a1 * (double)((int64_t)x1[i] - z1) +
                         (double)a2 * (double)((int64_t)x2[i] - z2);
        store_q(y, bits_y, i, requant_f64(v, ay, zy, bits_y));
    }
}

/* Elementwise product of two int16 code tensors (the gated unit of the
 * feed-forward block, SiLU(gate) * up), requantized:
 *   v = (a1 (x1 - z1)) * (a2 (x2 - z2)), each factor exact in fp64, the
 * product one rounding.                                                */
void oracle_mul_requant(const int16_t* x1, float a1, int32_t z1, const int16_t* x2,
                        float a2, int32_t z2, int64_t n, float ay, int32_t zy, int bits_y,
                        void* y)
{
    for (int64_t i = 0; i < n; ++i) {
        const double f1 = (double)a1 * (double)((int64_t)x1[i] - z1);
        const double f2 = (double)a2 * (double)((int64_t)x2[i] - z2);
        store_q(y, bits_y, i, requant_f64(f1 * f2, ay, zy, bits_y));
    }
}

/* Rotary position embedding on int16 codes [T][H * D] (the query and key
 * projections of a Llama-family block; the paper's models use it, the
 * paper leaves it in higher precision like the other non-linear operators,
 * Section 4.1).  Pairs (i, i + D/2) of every head rotate by the angle
 * (t + pos0) * base^(-2i/D) of token t:
 *   u = ax (x_i - zx), w = ax (x_{i+D/2} - zx)
 *   y_i = u cos - w sin,   y_{i+D/2} = w cos + u sin
 * in fp64 (inverse frequency by pow, angle one product, then cos and sin),
 * requantized.                                                         */
void oracle_rope(const int16_t* x, int64_t T, int64_t H, int64_t D, float ax, int32_t zx,
                 double base, int64_t pos0, float ay, int32_t zy, int bits_y, void* y)
{
    const int64_t half = D / 2;
    for (int64_t t = 0; t < T; ++t)
        for (int64_t h = 0; h < H; ++h)
            for (int64_t i = 0; i < half; ++i) {
                const double inv = pow(base, -(double)(2 * i) / (double)D);
                const double ang = (double)(t + pos0) * inv;
                const double c = cos(ang), sn = sin(ang);
                const int64_t j0 = t * H * D + h * D + i, j1 = j0 + half;
                const double u = (double)ax * (double)((int64_t)x[j0] - zx);
                const double w = (double)ax * (double)((int64_t)x[j1] - zx);
                store_q(y, bits_y, j0, requant_f64(u * c - w * sn, ay, zy, bits_y));
                store_q(y, bits_y, j1, requant_f64(w * c + u * sn, ay, zy, bits_y));
            }
}

/* Elementwise non-linear operator on int16 codes as a 65536-entry table,
 * entry i + 32768 for code i: f(alpha_x (i - zp_x)) requantized.
 * op 1: SiLU, f(v) = v / (1 + exp(-v)).                                */
static double glue_f(int op, double v)
{
    if (op == 1) return v / (1.0 + exp(-v));
    return v;
}

void oracle_lut_build(int op, float ax, int32_t zx, float ay, int32_t zy, int bits_y,
                      void* lut)
{
    for (int64_t i = -32768; i <= 32767; ++i) {
        const double v = (double)ax * (double)(i - zx);
        store_q(lut, bits_y, i + 32768, requant_f64(glue_f(op, v), ay, zy, bits_y));
    }
}

/* RMSNorm over each row of K codes (gamma optional):
 *   ss = sum_k (x - zp_x)^2 (exact, int64),  ms = alpha_x^2 ss / K + eps,
 *   r = sqrt(ms),  v = alpha_x (x - zp_x) * gamma[k] / r                */
void oracle_rmsnorm(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                    const float* gamma, float eps, float ay, int32_t zy, int bits_y, void* y)
{
    for (int64_t m = 0; m < M; ++m) {
        int64_t ss = 0;
        for (int64_t k = 0; k < K; ++k) {
            const int64_t d = (int64_t)x[m * K + k] - zx;
            ss += d * d;
        }
        const double a = (double)ax;
        const double ms = a * a * (double)ss / (double)K + (double)eps;
        const double r = sqrt(ms);
        for (int64_t k = 0; k < K; ++k) {
            double v = a * (double)((int64_t)x[m * K + k] - zx);
            if (gamma) v = v * (double)gamma[k];
            v = v / r;
            store_q(y, bits_y, m * K + k, requant_f64(v, ay, zy, bits_y));
        }
    }
}

/* Softmax over each row of K codes (scores):
 *   e_k = exp(alpha_x (x_k - max_j x_j)),  p_k = e_k / sum_j e_j
 * the sum in index order; the probabilities requantized.               */
/* Causal form (self-attention scores of a decoder): row m sees the keys
 * k <= (m mod period) + offset, the rows of one head being the period
 * consecutive queries and offset the keys before the first query; the
 * softmax runs over those keys and the others get probability 0 (code
 * zp_y).  period = 0: every key. */
void oracle_softmax_causal(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                           float ay, int32_t zy, int bits_y, int64_t period, int64_t offset,
                           void* y)
{
    (void)zx;  /* the zero-point cancels in x_k - max_j x_j */
    double* e = (double*)malloc(sizeof(double) * (size_t)(K > 0 ? K : 1));
    for (int64_t m = 0; m < M; ++m) {
        int64_t n = K;  /* keys seen by this row */
        if (period > 0 && (m % period) + offset + 1 < K) n = (m % period) + offset + 1;
        int64_t mx = x[m * K];
        for (int64_t k = 1; k < n; ++k)
            if (x[m * K + k] > mx) mx = x[m * K + k];
        double sum = 0.0;
        for (int64_t k = 0; k < n; ++k) {
            e[k] = exp((double)ax * (double)((int64_t)x[m * K + k] - mx));
            sum += e[k];
        }
        for (int64_t k = 0; k < K; ++k)
            store_q(y, bits_y, m * K + k, requant_f64(k < n ? e[k] / sum : 0.0, ay, zy, bits_y));
    }
    free(e);
}

void oracle_softmax(const int16_t* x, int64_t M, int64_t K, float ax, int32_t zx,
                    float ay, int32_t zy, int bits_y, void* y)
{
    oracle_softmax_causal(x, M, K, ax, zx, ay, zy, bits_y, 0, 0, y);
}

/* ------------------------------------------------------------------ */
/* Symmetric per-output-channel weight quantizer (Section 5.1 W8A8/W4A8
 * settings and the appendix's symmetric per-channel W4).
 * Readings: narrow range +-Q with Q = 2^(b-1)-1; scale = absmax/Q in fp32
 * (1 when that is not positive); q = rint(w/scale) limited to [-Q, Q]
 * (NaN -> -Q by the fmaxf/fminf convention).  colsum[n] = sum_k q[n][k].
 * bits = 4 packs two weights per byte, low nibble = even k.           */
/* ------------------------------------------------------------------ */
void oracle_pack_weights(const float* w, int64_t N, int64_t K, int bits,
                         void* w_q, float* w_scale, int32_t* colsum)
{
    const float Q = bits == 8 ? 127.0f : 7.0f;
    int8_t* tmp = (int8_t*)malloc((size_t)K);
    for (int64_t n = 0; n < N; ++n) {
        const float* row = w + n * K;
        float m = 0.0f;
        for (int64_t k = 0; k < K; ++k) m = fmaxf(m, fabsf(row[k]));
        float s = m / Q;
        if (!(s > 0.0f)) s = 1.0f;
        int64_t sum = 0;
        for (int64_t k = 0; k < K; ++k) {
            float t = row[k] / s;
            t = fminf(fmaxf(t, -Q), Q);
            tmp[k] = (int8_t)rintf(t);
            sum += tmp[k];
        }
        w_scale[n] = s;
        colsum[n] = (int32_t)sum;
        if (bits == 8) {
            memcpy((int8_t*)w_q + n * K, tmp, (size_t)K);
        } else {
            uint8_t* dst = (uint8_t*)w_q + n * (K / 2);
            for (int64_t j = 0; j < K / 2; ++j)
                dst[j] = (uint8_t)(((unsigned)tmp[2 * j] & 0xFu) |
                                   (((unsigned)tmp[2 * j + 1] & 0xFu) << 4));
        }
    }
    free(tmp);
}

/* ------------------------------------------------------------------ */
/* Asymmetric weights (Section 5.1: both the W8A8 and the W4A8 settings
 * quantize weights asymmetrically, using the full range of the format;
 * W8A8 takes one range per tensor except for the MLP down projection,
 * W4A8 one range per output channel).  The weights are quantized like an
 * activation tensor with the quantizer of Eq.(2)-(4) at bits 8 or 4, over
 * the range [min, max] of the finite values of a row (per channel) or of
 * the whole matrix (per tensor), widened to contain 0:
 *   alpha = (hi - lo) / (2^bits - 1)   (in fp64, then to fp32)
 *   beta  = lo / alpha,  zp = clamp(rint(-beta), 0, 2^bits - 1)
 *                             - 2^(bits-1)                     (signed)
 *   q = clamp(rint(w / alpha) + zp, -2^(bits-1), 2^(bits-1) - 1)
 * with w / alpha one fp32 division limited to +-2^20 (NaN -> the low
 * end) as in the activation quantizer.  A zero-width range (or one whose
 * alpha would not be a positive finite fp32) takes alpha = 1 and beta = 0,
 * so an all-zero range stores zp = -2^(bits-1) everywhere.  The per-row
 * outputs w_scale[n], w_zp[n] repeat the tensor's values per tensor.
 * colsum[n] = sum_k q[n][k]; int4 packs two codes per byte, low nibble =
 * even k.                                                              */
/* ------------------------------------------------------------------ */
static void finite_range(const float* v, int64_t n, double* lo, double* hi)
{
    *lo = 0.0;
    *hi = 0.0;
    for (int64_t i = 0; i < n; ++i) {
        if (!isfinite(v[i])) continue;
        if (v[i] < *lo) *lo = v[i];
        if (v[i] > *hi) *hi = v[i];
    }
}

static void asym_format(double lo, double hi, int bits, float* alpha_out, int32_t* zp_out)
{
    const double q_max = (double)(((int64_t)1 << bits) - 1);   /* Eq.(2) */
    float alpha = 1.0f;
    double beta = 0.0;
    if (hi - lo != 0.0) {
        float a = (float)((hi - lo) / q_max);                  /* Eq.(3) */
        if (a > 0.0f && isfinite(a)) {
            alpha = a;
            beta = lo / (double)alpha;                         /* Eq.(3) */
        }
    }
    double zu = rint(-beta);
    if (zu < 0.0) zu = 0.0;
    if (zu > q_max) zu = q_max;
    *alpha_out = alpha;
    *zp_out = (int32_t)((int64_t)zu - ((int64_t)1 << (bits - 1)));
}

void oracle_pack_weights_asym(const float* w, int64_t N, int64_t K, int bits,
                              int per_tensor, void* w_q, float* w_scale,
                              int32_t* w_zp, int32_t* colsum)
{
    const int64_t qlo = qmin_of(bits), qhi = qmax_of(bits);
    const float lim = 1048576.0f; /* 2^20 */
    double lo, hi;
    float alpha = 1.0f;
    int32_t zp = 0;
    if (per_tensor) {
        finite_range(w, N * K, &lo, &hi);
        asym_format(lo, hi, bits, &alpha, &zp);
    }
    int8_t* tmp = (int8_t*)malloc((size_t)K);
    for (int64_t n = 0; n < N; ++n) {
        const float* row = w + n * K;
        if (!per_tensor) {
            finite_range(row, K, &lo, &hi);
            asym_format(lo, hi, bits, &alpha, &zp);
        }
        int64_t sum = 0;
        for (int64_t k = 0; k < K; ++k) {
            float t = row[k] / alpha;                              /* Eq.(4) */
            t = fminf(fmaxf(t, -lim), lim);
            tmp[k] = (int8_t)clamp_i64((int64_t)rintf(t) + zp, qlo, qhi);
            sum += tmp[k];
        }
        w_scale[n] = alpha;
        w_zp[n] = zp;
        colsum[n] = (int32_t)sum;
        if (bits == 8) {
            memcpy((int8_t*)w_q + n * K, tmp, (size_t)K);
        } else {
            uint8_t* dst = (uint8_t*)w_q + n * (K / 2);
            for (int64_t j = 0; j < K / 2; ++j)
                dst[j] = (uint8_t)(((unsigned)tmp[2 * j] & 0xFu) |
                                   (((unsigned)tmp[2 * j + 1] & 0xFu) << 4));
        }
    }
    free(tmp);
}

/* Row sums of the quantized activations, sum_k A_q[m][k].              */
void oracle_act_rowsum(const int8_t* a_q, int64_t M, int64_t K, int32_t* rowsum)
{
    for (int64_t m = 0; m < M; ++m) {
        int64_t s = 0;
        for (int64_t k = 0; k < K; ++k) s += a_q[m * K + k];
        rowsum[m] = (int32_t)s;
    }
}

/* Weight code of row n, input channel k, read from the stored layout.
 * int4: the nibble is a two's-complement 4-bit integer.               */
static int64_t weight_at(const void* w_q, int bits, int64_t K, int64_t n,
                         int64_t k)
{
    if (bits == 8) return ((const int8_t*)w_q)[n * K + k];
    unsigned byte = ((const uint8_t*)w_q)[n * (K / 2) + k / 2];
    unsigned nib = (k & 1) ? (byte >> 4) : (byte & 0xFu);
    return nib >= 8 ? (int64_t)nib - 16 : (int64_t)nib;
}

/* ------------------------------------------------------------------ */
/* Fixed-point requantization parameters for output channel n.
 * The paper only states that every operation runs on fixed-point integers
 * (Section 1 and the design choices of Section 3.1).  Reading: the real
 * rescale M = (alpha_a * w_scale[n]) / alpha_y is computed in fp64 and
 * written M = M0 * 2^-sh with a 31-bit integer M0 in [2^30, 2^31): with
 * M = f * 2^e, f in [0.5, 1), M0 = rint(f * 2^31) (2^31 is renormalised
 * to 2^30 with e + 1), sh = 31 - e.
 * The bias enters in accumulator units: bias_q = rint(b / (alpha_a *
 * w_scale)) in fp64, limited to +-2^30 (0 without bias).               */
/* ------------------------------------------------------------------ */
void oracle_requant_params(float alpha_a, float w_scale, float alpha_y,
                           const float* bias_n, int64_t* M0_out,
                           int32_t* sh_out, int64_t* bias_q_out)
{
    double M = ((double)alpha_a * (double)w_scale) / (double)alpha_y;
    if (!(M > 0.0)) {
        /* not a usable scale (w_scale <= 0 or NaN): the rescaled value is 0 */
        *M0_out = 0;
        *sh_out = 31;
    } else if (isinf(M)) {
        /* infinite rescale: every non-zero accumulator saturates */
        *M0_out = (int64_t)1 << 30;
        *sh_out = 0;
    } else {
        int e = 0;
        double f = frexp(M, &e);
        int64_t M0 = (int64_t)rint(ldexp(f, 31));
        if (M0 == ((int64_t)1 << 31)) {
            M0 = (int64_t)1 << 30;
            e += 1;
        }
        *M0_out = M0;
        *sh_out = 31 - e;
    }
    int64_t bq = 0;
    if (bias_n) {
        double t = (double)*bias_n / ((double)alpha_a * (double)w_scale);
        t = fmin(fmax(t, -1073741824.0), 1073741824.0);
        bq = (int64_t)rint(t);
    }
    *bias_q_out = bq;
}

/* ------------------------------------------------------------------ */
/* One requantized output value from its corrected accumulator c:
 *   r = floor((c * M0 + 2^(sh-1)) / 2^sh)   (one rounding, ties up)
 *   y = clamp(r + zp_y, qmin, qmax)
 * c has already been limited to int32, so |c * M0| < 2^62 and the int64
 * arithmetic below is exact.  sh >= 63 gives r = 0 exactly.  sh <= 0
 * means M >= 2^30, so |r| >= 2^30 * |c| and any non-zero c saturates.  */
/* ------------------------------------------------------------------ */
int64_t oracle_requant_round(int64_t c, int64_t M0, int32_t sh)
{
    if (sh >= 63) return 0;
    if (sh >= 1) {
        int64_t p = c * M0 + ((int64_t)1 << (sh - 1));
        /* floor division by 2^sh, written without shifting a negative value */
        return p >= 0 ? p >> sh : -((-p + ((int64_t)1 << sh) - 1) >> sh);
    }
    /* sh <= 0: |r| >= 2^30 |c|; any value beyond the int16 range will do */
    return c > 0 ? ((int64_t)1 << 40) : (c < 0 ? -((int64_t)1 << 40) : 0);
}

int64_t oracle_requant_value(int64_t c, int64_t M0, int32_t sh, int32_t zp_y,
                             int bits_y)
{
    int64_t r = oracle_requant_round(c, M0, sh);
    return clamp_i64(r + zp_y, qmin_of(bits_y), qmax_of(bits_y));
}

/* ------------------------------------------------------------------ */
/* Integer-only linear layer (the hot path):
 *   c[m][n] = sat_int32( sum_k (A_q[m][k] - zp_a) * (W_q[n][k] - zp_w[n])
 *                        + bias_q[n] )
 *   Y_q[m][n] = requant(c[m][n])
 * zp_w = 0 for symmetric weights.  A_q holds 8-bit codes, or 16-bit codes
 * for the W8A16 setting (Section 5.6: 16-bit activations into 8-bit-weight
 * matmuls).  The sum is the plain definition, accumulated exactly in int64
 * (integer MACs with a wide accumulator: Section 1, Section 3.1).       */
/* ------------------------------------------------------------------ */
typedef struct {
    const void* a;
    int a_bits;
    int64_t M, K, N;
    const void* w_q;
    int bits;
    const float* w_scale;
    const int32_t* w_zp;
    float alpha_a;
    int32_t zp_a;
    float alpha_y;
    int32_t zp_y;
    int bits_y;
    const float* bias;
    void* y;
    int64_t row_begin, row_end;
    int64_t* M0;
    int32_t* sh;
    int64_t* bq;
} qlinear_job;

static void* qlinear_rows(void* arg)
{
    qlinear_job* j = (qlinear_job*)arg;
    for (int64_t m = j->row_begin; m < j->row_end; ++m) {
        const int8_t* arow8 = (const int8_t*)j->a + m * j->K;
        const int16_t* arow16 = (const int16_t*)j->a + m * j->K;
        for (int64_t n = 0; n < j->N; ++n) {
            const int64_t zw = j->w_zp ? j->w_zp[n] : 0;
            int64_t acc = 0;
            for (int64_t k = 0; k < j->K; ++k) {
                const int64_t a = j->a_bits == 8 ? (int64_t)arow8[k] : (int64_t)arow16[k];
                acc += (a - j->zp_a) * (weight_at(j->w_q, j->bits, j->K, n, k) - zw);
            }
            int64_t c = clamp_i64(acc + j->bq[n], INT32_MIN, INT32_MAX);
            int64_t v = oracle_requant_value(c, j->M0[n], j->sh[n], j->zp_y,
                                             j->bits_y);
            store_q(j->y, j->bits_y, m * j->N + n, v);
        }
    }
    return NULL;
}

void oracle_qlinear_gen(const void* a_q, int a_bits, int64_t M, int64_t K, int64_t N,
                        const void* w_q, int bits, const float* w_scale,
                        const int32_t* w_zp, float alpha_a, int32_t zp_a,
                        float alpha_y, int32_t zp_y, int bits_y,
                        const float* bias, void* y_q, int nthreads)
{
    int64_t* M0 = (int64_t*)malloc(sizeof(int64_t) * (size_t)N);
    int32_t* sh = (int32_t*)malloc(sizeof(int32_t) * (size_t)N);
    int64_t* bq = (int64_t*)malloc(sizeof(int64_t) * (size_t)N);
    for (int64_t n = 0; n < N; ++n)
        oracle_requant_params(alpha_a, w_scale[n], alpha_y,
                              bias ? bias + n : NULL, &M0[n], &sh[n], &bq[n]);
    if (nthreads < 1) nthreads = 1;
    if (nthreads > M) nthreads = (int)(M > 0 ? M : 1);
    pthread_t* th = (pthread_t*)malloc(sizeof(pthread_t) * (size_t)nthreads);
    qlinear_job* jobs = (qlinear_job*)malloc(sizeof(qlinear_job) * (size_t)nthreads);
    for (int t = 0; t < nthreads; ++t) {
        qlinear_job j = {a_q, a_bits, M, K, N, w_q, bits, w_scale, w_zp, alpha_a, zp_a,
                         alpha_y, zp_y, bits_y, bias, y_q,
                         M * t / nthreads, M * (t + 1) / nthreads, M0, sh, bq};
        jobs[t] = j;
        pthread_create(&th[t], NULL, qlinear_rows, &jobs[t]);
    }
    for (int t = 0; t < nthreads; ++t) pthread_join(th[t], NULL);
    free(jobs);
    free(th);
    free(M0);
    free(sh);
    free(bq);
}

/* 8-bit activations.                                                   */
void oracle_qlinear_asym(const int8_t* a_q, int64_t M, int64_t K, int64_t N,
                         const void* w_q, int bits, const float* w_scale,
                         const int32_t* w_zp, float alpha_a, int32_t zp_a,
                         float alpha_y, int32_t zp_y, int bits_y,
                         const float* bias, void* y_q, int nthreads)
{
    oracle_qlinear_gen(a_q, 8, M, K, N, w_q, bits, w_scale, w_zp, alpha_a, zp_a,
                       alpha_y, zp_y, bits_y, bias, y_q, nthreads);
}

/* Symmetric weights: zp_w = 0.                                         */
void oracle_qlinear(const int8_t* a_q, int64_t M, int64_t K, int64_t N,
                    const void* w_q, int bits, const float* w_scale,
                    float alpha_a, int32_t zp_a, float alpha_y, int32_t zp_y,
                    int bits_y, const float* bias, void* y_q, int nthreads)
{
    oracle_qlinear_asym(a_q, M, K, N, w_q, bits, w_scale, NULL, alpha_a, zp_a,
                        alpha_y, zp_y, bits_y, bias, y_q, nthreads);
}

/* The raw integer product sum_k A_q[m][k] * W_q[n][k] (no zero-point, no
 * bias, no rescale), exposed so tests can pin the accumulation alone.  */
void oracle_int_matmul(const int8_t* a_q, int64_t M, int64_t K, int64_t N,
                       const void* w_q, int bits, int64_t* acc)
{
    for (int64_t m = 0; m < M; ++m)
        for (int64_t n = 0; n < N; ++n) {
            int64_t s = 0;
            for (int64_t k = 0; k < K; ++k)
                s += (int64_t)a_q[m * K + k] * weight_at(w_q, bits, K, n, k);
            acc[m * N + n] = s;
        }
}
