// Prefill-shaped qlinear: an LDS-tiled int8 MFMA GEMM with the requant
// epilogue fused in registers.
//
// Prompt encoding is compute-bound (Section 5.6) and int8 x int8 is the
// fastest integer product (Section 3.1), so the inner loop is
// v_mfma_i32_32x32x32_i8 (measured on MI355X: one wave per SIMD issuing it
// back to back reaches ~92% of the int8 peak, the 16x16x64 form ~52%).  The
// weight matrix is the MFMA "A" operand (rows = output channels) and the
// activations the "B" operand (columns = tokens): every lane then ends with
// runs of four consecutive output channels of one token, which become one
// 4-byte (int8) or 8-byte (int16) store.
//
// Data movement (gfx950):
// - Operand tiles go HBM/L2 -> LDS with buffer_load_dwordx4 ... lds (LDS DMA:
//   no VGPR staging, no ds_write).  A wave's load fills 1 KiB of LDS; which
//   16-byte chunk each lane fetches decides the LDS layout, so 16-byte chunks
//   are XOR-swizzled per row to keep the 16-row MFMA operand reads on
//   distinct banks.
// - The buffer descriptor of each tile covers only its valid rows, and a
//   K-tail chunk gets an out-of-range offset: the hardware returns zeros, so
//   ragged M, N and K need no branches in the inner loop.
// - STAGES-deep ring of LDS buffers, one barrier per K step, waits on the
//   vector-memory counter so STAGES-1 tiles stay in flight.
// - int4 weights stay packed in LDS (half the bytes) and are unpacked into
//   registers right before the MFMA as 16*w; the epilogue removes the 16 with
//   an exact shift.
// - Block ids are remapped so blocks that share weight tiles run on the same
//   XCD (each XCD has its own L2).
#include <type_traits>

#include "mq_internal.h"
#include "requant.h"

#define MQ_LDS __attribute__((address_space(3)))

namespace mq {
namespace {

typedef int v4i __attribute__((ext_vector_type(4)));
typedef int v16i __attribute__((ext_vector_type(16)));

constexpr uint32_t kOOB = 0x80000000u;  // any offset past num_records reads zero

// Split-K workspace: one int32 arrival counter per tile (rounded up to 256
// bytes), then the int32 partial sums of every (tile, slice) block.
__host__ __device__ inline int64_t split_counter_bytes(int64_t tiles)
{
    return (tiles * 4 + 255) / 256 * 256;
}

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

// v_med3_i32: x clamped to [lo, hi] (lo <= hi) in one instruction; the
// compiler emits two (v_min, v_max) when the bounds are not constants
__device__ __forceinline__ int32_t med3_i32(int32_t x, int32_t lo, int32_t hi)
{
    int32_t r;
    asm("v_med3_i32 %0, %1, %2, %3" : "=v"(r) : "v"(x), "v"(lo), "v"(hi));
    return r;
}

// v_cvt_pk_i16_i32: two int32 saturated to the int16 range and packed, the
// first in the low half (one instruction for what two clamps and a byte
// permute do; saturation checked on MI355X at the int16 and int32 ends)
__device__ __forceinline__ uint32_t pack_sat_i16(int32_t lo, int32_t hi)
{
    typedef short v2s __attribute__((ext_vector_type(2)));
    return __builtin_bit_cast(uint32_t, __builtin_amdgcn_cvt_pk_i16(lo, hi));
}

// s_waitcnt vmcnt(N) with the other counters left alone (gfx9 encoding:
// vmcnt bits [3:0] and [15:14], expcnt [6:4], lgkmcnt [11:8]).
template <int N>
__device__ inline void wait_vmcnt()
{
    static_assert(N >= 0 && N < 64, "vmcnt is 6 bits");
    __builtin_amdgcn_s_waitcnt((N & 15) | ((N >> 4) << 14) | (7 << 4) | (15 << 8));
}

template <int WBITS_, int OBITS_, int TM_, int TN_, int WM_, int WN_, int BK_, int STAGES_,
          int SWZ_, int SPREAD_, int ABITS_ = 8>
struct Cfg {
    static constexpr int WBITS = WBITS_, OBITS = OBITS_;
    // 16-bit activation codes (W8A16): two byte planes per code, two MFMAs
    // per fragment pair, a second accumulator set
    static constexpr int ABITS = ABITS_;
    static constexpr bool A16 = ABITS == 16;
    static constexpr int AB = ABITS / 8;  // activation bytes per code
    static constexpr int TM = TM_, TN = TN_, WM = WM_, WN = WN_, BK = BK_;
    static constexpr int STAGES = STAGES_, SWZ = SWZ_;
    static constexpr int NWAVES = WM * WN;
    // work-groups per CU the register budget is sized for: the short-K
    // 16-bit tile (two stages) shares a CU between two
    static constexpr int OCC = (ABITS_ == 16 && STAGES_ == 2) ? 2 : 1;
    // the short-K 16-bit tile (two stages) serves K <= 128 without bias
    // only: then |c| = |sum_k (a - a_zp)(b - b_zp)| <= 128 * 65535 * 255 <
    // 2^31, the saturation is the identity and its terms sum in int32
    // (wrapping to the exact value)
    static constexpr bool A16_I32 = ABITS_ == 16 && STAGES_ == 2;
    static constexpr int A16_I32_MAX_K = 128;
    static constexpr int THREADS = 64 * NWAVES;
    static constexpr int FM = TM / (WM * 32);   // 32-token fragments per wave
    static constexpr int FN = TN / (WN * 32);   // 32-channel fragments per wave
    static constexpr int BKW = WBITS == 8 ? BK : BK / 2;  // weight bytes per row per stage
    static constexpr int BKA = BK * AB;         // activation bytes per row per stage
    static constexpr int CA = BKA / 16;         // 16-byte chunks per activation row
    static constexpr int CW = BKW / 16;         // 16-byte chunks per weight row
    static constexpr int A_WLOADS = TM * CA / 64;  // 1 KiB wave loads per stage
    static constexpr int W_WLOADS = TN * CW / 64;
    static constexpr int A_PER_WAVE = (A_WLOADS + NWAVES - 1) / NWAVES;
    static constexpr int W_PER_WAVE = (W_WLOADS + NWAVES - 1) / NWAVES;
    static constexpr int LOADS = A_PER_WAVE + W_PER_WAVE;  // per thread per stage
    static constexpr int KS = BK / 32;                       // 32-deep steps per stage
    static constexpr int NRD = FN + FM * AB;                 // fragment reads per step
    // DMA of a stage spread over the groups of SPREAD steps after its switch
    static constexpr int SPREAD = SPREAD_;
    // group slot of DMA d of a stage among the SPREAD*NRD groups after its switch
    static constexpr int dma_slot(int d) { return d * SPREAD * NRD / LOADS; }
    // DMAs issued in the stage switch step itself
    static constexpr int nsw()
    {
        int n = 0;
        for (int d = 0; d < LOADS; ++d) n += dma_slot(d) < NRD ? 1 : 0;
        return n;
    }
    static constexpr int NSW = nsw();
    // K slices (split-K) for the 8-bit activation tiles
    static constexpr bool SPLITK = !A16;
    // at most 12 accumulator fragments per wave leave registers for the
    // slice bookkeeping of a K split and the pre-shift epilogue forms
    static_assert(FM * FN <= 12, "accumulator registers");
    // split-K merge: fragment rows of the other slices' partial sums loaded
    // per batch (16 chunks, 64 registers in flight), never more than the
    // wave has, and a whole number of batches per wave
    static constexpr int MERGE_IB = 16 / (FM * 4) < 1 ? 1 : (16 / (FM * 4) > FN ? FN : 16 / (FM * 4));
    static_assert(FN % MERGE_IB == 0, "whole merge batches per wave");
    static constexpr int A_BYTES = A_PER_WAVE * NWAVES * 1024;
    static constexpr int W_BYTES = W_PER_WAVE * NWAVES * 1024;
    static constexpr int STAGE = A_BYTES + W_BYTES;
    // + per-column epilogue constants + one flag word per wave
    static constexpr int LDS = STAGES * STAGE + TN * 16 + NWAVES * 4;
    // asymmetric weights add per channel -w_zp and per token row sum; 16-bit
    // activations use the channel array for the low part of the offset and
    // two words per token row for an int64 row term
    static constexpr int LDS_ASYM = LDS + (TN + 2 * TM) * 4;
    static_assert(!A16 || (WBITS == 8 && !SPLITK), "16-bit activations: int8 weights, no split");
    static_assert(TM % (WM * 32) == 0 && TN % (WN * 32) == 0, "wave grid");
    static_assert((TM * CA) % 64 == 0 && (TN * CW) % 64 == 0, "whole wave loads");
    static_assert(BK % 64 == 0, "BK is a multiple of the MFMA depth");
    static_assert(STAGES >= 2 && STAGES <= 4, "pipeline depth");
    static_assert((BK / 32) % 2 == 0, "even number of 32-deep steps per stage");
    static_assert(LOADS * (STAGES - 1) < 64, "vmcnt range");
    static_assert(SPREAD >= 1 && SPREAD <= KS, "the DMA spread stays within one stage");
    static_assert(LDS_ASYM <= 160 * 1024, "LDS per CU");
};

template <int SWZ>
__device__ inline int swz(int row, int nchunks)
{
    if constexpr (SWZ == 0) return row & (nchunks - 1);
    else if constexpr (SWZ == 1) return (row >> 1) & (nchunks - 1);
    else if constexpr (SWZ == 2) {
        // 64 banks x 4 bytes: 256 / (16 * nchunks) rows share one bank row,
        // so the row index above that is the XOR key; 16 consecutive rows
        // then cover all 16 groups of four banks
        const int per = 16 / nchunks;  // rows per 256 bytes
        return (row / per) & (nchunks - 1);
    } else return 0;
}

struct EpiCtx {
    const int32_t* e_nzw;  // asymmetric weights: -w_zp per tile channel
    const int32_t* e_rs;   // asymmetric weights: sum_k (a - a_zp) per tile token row;
                           // 16-bit codes: low words of the int64 row terms
    const int32_t* e_rhi;  // 16-bit codes: high words of the int64 row terms
    const int32_t* e_off;
    const int32_t* e_m0;
    const int32_t* e_rnd;
    const int32_t* e_sp;
    int32_t row_bytes;     // bytes per output row
    int32_t lane_row_off;  // byte offset of this lane's first token row in the tile
    int32_t col0;          // this lane's first channel inside the tile
    int32_t n_left;        // channels of the tile that exist (N - n_tile)
    int32_t n_tile;
    int32_t out_zp;        // 0 when folded into the rounding constants
    int32_t r32;           // this lane's token row within a 32-row fragment
    int32_t wave_row0;     // first token row of this wave's sub-tile (tile-local)
    int32_t wave_col0;     // first channel of this wave's sub-tile (tile-local)
    MQ_LDS int8_t* stage;  // this wave's LDS staging area (staged stores)
    __amdgpu_buffer_rsrc_t ry;  // output rows of this tile
    // dequantized outputs (fp32): the layer's output format, this tile's
    // fp32 rows, whether the codes are stored as well
    float out_scale;
    int32_t out_zp_code;   // the output zero-point (out_zp may be folded away)
    int32_t row_bytes_f;
    int32_t lane_row_off_f;
    bool has_codes;
    __amdgpu_buffer_rsrc_t ryf;
};

// Staged stores: a wave's outputs go through its own LDS area, PB bytes of
// each sub-tile row per pass, and leave as 16-byte stores that cover whole
// row segments.  Direct stores from the accumulator layout write 4 or 8
// bytes into each of 32 rows per instruction, which measured ~2x slower
// for the whole epilogue on MI355X.
template <class C>
struct Staging {
    static constexpr int OB = C::OBITS / 8;
    static constexpr int WR = C::TM / C::WM;  // sub-tile rows
    static constexpr int WC = C::TN / C::WN;  // sub-tile channels
    // channels staged per pass: at most 128 bytes of a row, and few enough
    // that every wave's staging area fits the stage ring (the eight-wave
    // 256x256 tile with int16 outputs stages 32 channels at a time)
    static constexpr int pass_cols()
    {
        int c = WC * OB > 128 ? 128 / OB : WC;
        while (c > 32 && C::NWAVES * WR * (c * OB + 16) > C::STAGES * C::STAGE) c /= 2;
        return c;
    }
    static constexpr int PASS_COLS = pass_cols();
    static constexpr int PASSES = WC / PASS_COLS;
    static constexpr int FNP = C::FN / PASSES;  // 32-channel fragments per pass
    static constexpr int PB = PASS_COLS * OB;   // staged bytes per row
    static constexpr int PITCH = PB + 16;       // padding spreads rows over banks
    static constexpr int CPR = PB / 16;         // 16-byte chunks per row
    static constexpr int RPI = 64 / CPR;        // rows per wave-wide 16-byte store
    static constexpr int BYTES = WR * PITCH;    // per wave
    static_assert(PASS_COLS % 32 == 0 && C::FN % PASSES == 0, "whole fragments per pass");
    static_assert(WR % RPI == 0, "whole stores per sub-tile");
    static_assert(C::NWAVES * BYTES <= C::STAGES * C::STAGE, "staging fits the stage ring");
};

// Requant and store one tile's accumulators.  32x32 accumulator layout:
// lane holds token r32 and, in register group g, the four consecutive
// channels 8g + 4hk + {0..3}: one 4-byte (int8) or 8-byte (int16) store.
// Rows past M fall outside the descriptor and are dropped by the hardware;
// channel groups past N get an out-of-range offset.  The requant is the
// integer form with one mul_hi per output (cheaper on gfx950 than fp64
// conversions).  FAST: off is in the accumulator's start value, the output
// zero-point is folded into the rounding constants and N % 4 == 0, leaving
// mul_hi, add, shift, clamp per output; PRE adds the clamp and left shift
// of the columns whose shift is below 33 (large rescale factors, typical of
// int16 outputs), which the plain FAST form leaves out when no column of
// the tile needs them.
// ASYM (asymmetric weights) adds -w_zp[n] * rs[m]: the fast form has it in
// the accumulator's start value already, the other adds it exactly in
// int64 before the saturation.  With 16-bit codes ASYM instead adds an
// int64 term per token row (a per-tensor zero-point of the other operand),
// also before the saturation.
// YF: also (or, without codes, only) the dequantized outputs in fp32.  The
// staged form converts each 16-byte chunk of codes it reads back from LDS
// (whole 128-byte row segments per four lanes); the other forms store four
// channels of one token per lane from the accumulator layout.
template <class C, bool ASYM, bool FAST, bool PRE, bool STAGED, bool YF, class Acc, class Acc2>
__device__ __forceinline__ void prefill_epilogue(Acc& acc, Acc2& acc2, const EpiCtx& x)
{
    constexpr int32_t qmin = -(1 << (C::OBITS - 1));
    constexpr int32_t qmax = (1 << (C::OBITS - 1)) - 1;
    constexpr int OB = C::OBITS / 8;
    using S = Staging<C>;
    static_assert(!STAGED || FAST, "staged stores assume whole 4-channel groups");
    constexpr int PASSES = STAGED ? S::PASSES : 1;
    constexpr int FNP = C::FN / PASSES;
    constexpr bool CASYM = ASYM && !C::A16;  // per-channel weight zero-points
    constexpr bool ROFF = ASYM && C::A16;    // int64 row terms
    int32_t rs[C::FM];  // this lane's token rows
    int64_t roff[C::FM];
    uint32_t roff32[C::FM];  // the int32 form: low words
#pragma unroll
    for (int j = 0; j < C::FM; ++j) {
        const int row = x.wave_row0 + j * 32 + x.r32;
        rs[j] = CASYM && !FAST ? x.e_rs[row] : 0;
        roff[j] = ROFF && !C::A16_I32 ? (int64_t)(((uint64_t)(uint32_t)x.e_rhi[row] << 32) |
                                                  (uint64_t)(uint32_t)x.e_rs[row])
                                      : 0;
        roff32[j] = ROFF && C::A16_I32 ? (uint32_t)x.e_rs[row] : 0u;
    }
#pragma unroll
    for (int pass = 0; pass < PASSES; ++pass) {
#pragma unroll
    for (int i = pass * FNP; i < (pass + 1) * FNP; ++i) {
#pragma unroll
        for (int g = 0; g < 4; ++g) {
            const int nl = x.col0 + i * 32 + 8 * g;  // tile-local channel
            v4i off = {0, 0, 0, 0}, nzw = {0, 0, 0, 0};
            if constexpr (!FAST) off = *reinterpret_cast<const v4i*>(x.e_off + nl);
            if constexpr ((CASYM || C::A16) && !FAST)
                nzw = *reinterpret_cast<const v4i*>(x.e_nzw + nl);  // A16: offset low part
            const v4i m0 = *reinterpret_cast<const v4i*>(x.e_m0 + nl);
            const v4i rnd = *reinterpret_cast<const v4i*>(x.e_rnd + nl);
            const v4i sp = *reinterpret_cast<const v4i*>(x.e_sp + nl);
            const int32_t col_off = (x.n_tile + nl) * OB;
            const bool col_ok = nl < x.n_left;
            int32_t shr[4], pre[4], bnd[4], nbnd[4];  // per column, hoisted out of the token loop
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                shr[r] = sp[r] & 0xFF;
                pre[r] = sp[r] >> 8;
                bnd[r] = pre[r] ? (1 << (30 - pre[r])) : 0x7FFFFFFF;
                nbnd[r] = -bnd[r];
            }
#pragma unroll
            for (int j = 0; j < C::FM; ++j) {
                // int8 outputs: clamped codes; int16 outputs: the unclamped
                // values, saturated by the pack (pack_sat_i16) or per element
                int32_t y[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    int32_t a32 = acc[i][j][4 * g + r];
                    if constexpr (C::WBITS == 4) a32 >>= 4;  // exact: a multiple of 16
                    int32_t c = a32;  // fast form: off is already in the accumulator
                    if constexpr (C::A16_I32) {
                        // the same sum modulo 2^32, whose exact value fits
                        uint32_t u = ((uint32_t)a32 << 8) + (uint32_t)acc2[i][j][4 * g + r];
                        if constexpr (!FAST) u += ((uint32_t)off[r] << 8) + (uint32_t)nzw[r];
                        if constexpr (ROFF) u += roff32[j];
                        c = (int32_t)u;
                    } else if constexpr (C::A16) {
                        // high plane * 256 + low plane (+ the offset, split
                        // the same way, when it is not in the start values)
                        int64_t c64 = ((int64_t)a32 << 8) + acc2[i][j][4 * g + r];
                        if constexpr (!FAST) c64 += ((int64_t)off[r] << 8) + nzw[r];
                        if constexpr (ROFF) c64 += roff[j];
                        c = sat32(c64);
                    } else if constexpr (!FAST) {
                        if constexpr (CASYM)
                            c = corrected_acc_asym(a32, off[r], nzw[r], rs[j]);
                        else
                            c = __builtin_elementwise_add_sat(a32, off[r]);
                    }
                    // (no column of the tile with a pre-shift: bnd = 2^31 - 1 and
                    // pre = 0, both the identity)
                    if constexpr (!FAST || PRE) {
                        c = med3_i32(c, nbnd[r], bnd[r]);
                        c = (int32_t)((uint32_t)c << pre[r]);
                    }
                    int32_t v = (__mulhi(c, m0[r]) + rnd[r]) >> shr[r];
                    if constexpr (!FAST) v += x.out_zp;
                    y[r] = C::OBITS == 16 ? v : max(min(v, qmax), qmin);
                }
                if constexpr (STAGED) {
                    // tile-local row j*32 + r32, pass-local channel nl - first
                    const int lrow = j * 32 + x.r32;
                    MQ_LDS int8_t* dst = x.stage + lrow * S::PITCH +
                                         (nl - x.wave_col0 - pass * S::PASS_COLS) * OB;
                    if constexpr (C::OBITS == 8) {
                        const uint32_t lo =
                            __builtin_amdgcn_perm((uint32_t)y[1], (uint32_t)y[0], 0x0c0c0400u);
                        const uint32_t hi =
                            __builtin_amdgcn_perm((uint32_t)y[3], (uint32_t)y[2], 0x04000c0cu);
                        *reinterpret_cast<MQ_LDS uint32_t*>(dst) = lo | hi;
                    } else {
                        typedef unsigned v2u __attribute__((ext_vector_type(2)));
                        v2u v;
                        v[0] = pack_sat_i16(y[0], y[1]);
                        v[1] = pack_sat_i16(y[2], y[3]);
                        *reinterpret_cast<MQ_LDS v2u*>(dst) = v;
                    }
                    continue;
                }
                const int32_t row_off = x.lane_row_off + j * 32 * x.row_bytes;
                if constexpr (YF) {
                    float f[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r)
                        f[r] = dequant_code(max(min(y[r], qmax), qmin), x.out_scale,
                                            x.out_zp_code);
                    const int32_t row_f = x.lane_row_off_f + j * 32 * x.row_bytes_f;
                    const int32_t col_f = (x.n_tile + nl) * 4;
                    if (FAST || (x.n_left & 3) == 0 || nl + 3 < x.n_left) {
                        const v4i v = {__builtin_bit_cast(int, f[0]), __builtin_bit_cast(int, f[1]),
                                       __builtin_bit_cast(int, f[2]), __builtin_bit_cast(int, f[3])};
                        __builtin_amdgcn_raw_buffer_store_b128(
                            v, x.ryf, col_ok ? (uint32_t)(row_f + col_f) : kOOB, 0, 0);
                    } else {
#pragma unroll
                        for (int r = 0; r < 4; ++r)
                            __builtin_amdgcn_raw_buffer_store_b32(
                                __builtin_bit_cast(int, f[r]), x.ryf,
                                nl + r < x.n_left ? (uint32_t)(row_f + col_f + 4 * r) : kOOB, 0,
                                0);
                    }
                    if (!x.has_codes) continue;
                }
                if (FAST || (x.n_left & 3) == 0 || nl + 3 < x.n_left) {
                    const uint32_t voff = col_ok ? (uint32_t)(row_off + col_off) : kOOB;
                    if constexpr (C::OBITS == 8) {
                        const uint32_t lo =
                            __builtin_amdgcn_perm((uint32_t)y[1], (uint32_t)y[0], 0x0c0c0400u);
                        const uint32_t hi =
                            __builtin_amdgcn_perm((uint32_t)y[3], (uint32_t)y[2], 0x04000c0cu);
                        __builtin_amdgcn_raw_buffer_store_b32(lo | hi, x.ry, voff, 0, 0);
                    } else {
                        typedef unsigned v2u __attribute__((ext_vector_type(2)));
                        v2u v;
                        v[0] = pack_sat_i16(y[0], y[1]);
                        v[1] = pack_sat_i16(y[2], y[3]);
                        __builtin_amdgcn_raw_buffer_store_b64(v, x.ry, voff, 0, 0);
                    }
                } else {
                    // a channel group straddling N (N % 4 != 0): element stores
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const uint32_t voff =
                            nl + r < x.n_left ? (uint32_t)(row_off + col_off + r * OB) : kOOB;
                        if constexpr (C::OBITS == 8)
                            __builtin_amdgcn_raw_buffer_store_b8((unsigned char)y[r], x.ry, voff, 0, 0);
                        else
                            __builtin_amdgcn_raw_buffer_store_b16(
                                (unsigned short)max(min(y[r], qmax), qmin), x.ry, voff, 0, 0);
                    }
                }
            }
        }
    }
    if constexpr (STAGED) {
        // read back whole 16-byte row chunks and store them
        const int lane = threadIdx.x & 63;
        const int ch = lane % S::CPR;
        const int32_t col_byte = (x.n_tile + x.wave_col0 + pass * S::PASS_COLS) * OB + ch * 16;
#pragma unroll
        for (int t = 0; t < S::WR / S::RPI; ++t) {
            const int lrow = t * S::RPI + lane / S::CPR;
            const v4i v = *reinterpret_cast<MQ_LDS const v4i*>(x.stage + lrow * S::PITCH + ch * 16);
            if (!YF || x.has_codes) {
                const uint32_t voff = (uint32_t)((x.wave_row0 + lrow) * x.row_bytes + col_byte);
                __builtin_amdgcn_raw_buffer_store_b128(v, x.ry, voff, 0, 0);
            }
            if constexpr (YF) {
                // the chunk's 16 / OB codes (clamped already), four per store
                const int32_t off_f = (x.wave_row0 + lrow) * x.row_bytes_f +
                                      (x.n_tile + x.wave_col0 + pass * S::PASS_COLS) * 4 +
                                      ch * (16 / OB) * 4;
#pragma unroll
                for (int q = 0; q < 4 / OB; ++q) {
                    int32_t c[4];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int e = 4 * q + r;  // code index in the chunk
                        const uint32_t d = (uint32_t)v[e * OB / 4];
                        c[r] = OB == 2 ? (int32_t)(int16_t)(d >> (16 * (e & 1)))
                                       : (int32_t)(int8_t)(d >> (8 * (e & 3)));
                    }
                    const v4i fv = {
                        __builtin_bit_cast(int, dequant_code(c[0], x.out_scale, x.out_zp_code)),
                        __builtin_bit_cast(int, dequant_code(c[1], x.out_scale, x.out_zp_code)),
                        __builtin_bit_cast(int, dequant_code(c[2], x.out_scale, x.out_zp_code)),
                        __builtin_bit_cast(int, dequant_code(c[3], x.out_scale, x.out_zp_code))};
                    __builtin_amdgcn_raw_buffer_store_b128(fv, x.ryf, (uint32_t)(off_f + 16 * q),
                                                           0, 0);
                }
            }
        }
    }
    }
}

// One work-group's tile of the product.  GROUP: tiles of several linears
// that share the activation input, one block per tile of any of them (g
// holds each linear's weights, per-channel inputs, output and requant
// constants, tiles_n the tile columns of all of them); p carries the shared
// fields and takes those of the block's linear.
template <class C, bool ASYM, bool GROUP, bool YF = false>
__device__ __forceinline__ void prefill_body(QLinearArgs& p, const GroupArgs* g, int tiles_n,
                                             int tiles_m, int splits, int kt_per_split)
{
    constexpr int32_t qmin = -(1 << (C::OBITS - 1));
    constexpr int32_t qmax = (1 << (C::OBITS - 1)) - 1;
    constexpr int KS = C::BK / 32;  // 32-deep MFMA steps per stage
    extern __shared__ __align__(1024) int8_t smem[];
    // per-column epilogue constants, structure of arrays after the stages
    int32_t* e_off = reinterpret_cast<int32_t*>(smem + C::STAGES * C::STAGE);
    int32_t* e_m0 = e_off + C::TN;
    int32_t* e_rnd = e_m0 + C::TN;
    int32_t* e_sp = e_rnd + C::TN;  // shr | pre << 8
    int32_t* e_flag = e_sp + C::TN;  // per wave: bit 0 all pre == 0, bit 1 zp foldable
    int32_t* e_nzw = e_flag + C::NWAVES;  // asymmetric weights only
    int32_t* e_rs = e_nzw + C::TN;
    int32_t* e_rhi = e_rs + C::TM;        // 16-bit codes with row terms
    constexpr bool CASYM = ASYM && !C::A16;  // per-channel weight zero-points
    constexpr bool ROFF = ASYM && C::A16;    // int64 row terms

    // ---- tile and K slice: the blocks of one XCD (block id mod 8) take a
    // contiguous run of work items, so they share operand tiles in that
    // XCD's L2; item = slice * tiles + tile
    const int total = tiles_n * tiles_m;
    int b = blockIdx.x;
    {
        const int items = total * splits;
        const int per = items / 8, rem = items % 8;
        const int xcd = b % 8, idx = b / 8;
        b = xcd * per + (xcd < rem ? xcd : rem) + idx;
        // causal products skip the tiles past the diagonal (or the K past
        // it), which leaves the XCDs holding some tile columns (rows) with
        // most of the work: batch b starts its XCD runs (b mod 8) runs
        // later, so over eight batches every XCD gets each of them once
        if (C::A16 && (p.out_causal >= 0 || p.in_causal >= 0) && per > 0)
            b = (int)((b + (int64_t)(blockIdx.y % 8) * per) % items);
    }
    const int split = C::SPLITK ? b / total : 0;
    int tile = C::SPLITK ? b % total : b;
    if constexpr (GROUP) {
        // the linear whose tile columns hold this tile (block-uniform)
        int k = 0;
#pragma unroll
        for (int i = 1; i < kMaxGroup; ++i)
            if (i < g->n && tile >= g->part[i].tile0) k = i;
        const GroupPart& gp = g->part[k];
        p.w = gp.w;
        p.w_scale = gp.w_scale;
        p.colsum = gp.colsum;
        p.bias = gp.bias;
        p.w_zp = gp.w_zp;
        p.y = gp.y;
        p.N = gp.N;
        p.out_scale = gp.out_scale;
        p.out_zp = gp.out_zp;
        tile -= gp.tile0;
    }
    const int tn = tile / tiles_m;
    const int tm = tile % tiles_m;
    const int64_t n_tile = (int64_t)tn * C::TN;
    const int64_t m_tile = (int64_t)tm * C::TM;
    // batched, strided products (the attention matmuls) run on the 16-bit
    // tile only: this block's batch and the group whose weights it reads
    constexpr bool STR = C::A16;
    const int64_t bt = STR ? (int64_t)blockIdx.y : 0, bg = STR ? bt / p.group : 0;
    // causal outputs: a tile wholly past the boundary has nothing to compute
    if (STR && p.out_causal >= 0 && n_tile > m_tile + C::TM - 1 + p.out_causal) return;

    const int tid = threadIdx.x;
    const int lane = tid & 63;
    const int wave = __builtin_amdgcn_readfirstlane(tid >> 6);  // uniform: keep it scalar
    const int wn = wave / C::WM;
    const int wm = wave % C::WM;
    const int r32 = lane & 31;  // operand row / output token within a fragment
    const int hk = lane >> 5;   // which 16-byte half of a 32-byte k step

    // ---- buffer descriptors covering only this tile's valid rows, from the
    // first K byte of this block's slice; KL = the slice's length in K
    const int64_t K = p.K;
    const int64_t lda = STR ? eff_lda(p) : K;  // activation row stride, elements
    const int64_t wrow = C::WBITS == 8 ? (STR ? eff_ldw(p) : K) : K / 2;  // bytes
    const int rows_a = (int)((p.M - m_tile) < C::TM ? (p.M - m_tile) : C::TM);
    const int rows_w = (int)((p.N - n_tile) < C::TN ? (p.N - n_tile) : C::TN);
    const int64_t k_begin = C::SPLITK ? (int64_t)split * kt_per_split * C::BK : 0;
    int64_t KL = !C::SPLITK ? K
                 : (K - k_begin) < (int64_t)kt_per_split * C::BK
                     ? (K - k_begin) : (int64_t)kt_per_split * C::BK;
    // causal activations: the column sums come per block of kA16TileM rows
    // (a tile of fewer rows uses its enclosing block's), each over the K
    // range up to the stage that holds that block's last row's boundary
    const int64_t m_blk = m_tile / kA16TileM;
    if (STR && p.in_causal >= 0) {
        // the activations past the boundary are zero-point codes (no
        // contribution), so the tile stops at the same stage
        const int64_t m_end = (m_blk + 1) * kA16TileM < p.M ? (m_blk + 1) * kA16TileM : p.M;
        const int64_t need = (m_end + p.in_causal + C::BK - 1) / C::BK * C::BK;
        if (need < KL) KL = need;
    }
    const int64_t k_begin_w = C::WBITS == 8 ? k_begin : k_begin / 2;
    const int64_t KLw = C::WBITS == 8 ? KL : KL / 2;
    const __amdgpu_buffer_rsrc_t ra = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(p.a + (bt * p.a_bs + m_tile * lda + k_begin) * C::AB), (short)0,
        (int)(((rows_a - 1) * lda + K - k_begin) * C::AB), 0x00020000);
    const __amdgpu_buffer_rsrc_t rw = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(static_cast<const int8_t*>(p.w) + bg * p.w_bs + n_tile * wrow + k_begin_w),
        (short)0, (int)((rows_w - 1) * wrow + (C::WBITS == 8 ? K : K / 2) - k_begin_w),
        0x00020000);

    // Source offsets of this lane's chunks at k = 0; a stage adds kt*BK.  A
    // chunk past the end of its row (K tail) is pushed out of range.
    // Source offset of each of this lane's chunks at k = 0 (a stage adds
    // kt*BK).  Chunks of padding wave loads get an out-of-range offset.
    uint32_t a_off[C::A_PER_WAVE], w_off[C::W_PER_WAVE];
    auto a_kb = [&](int i) {  // k byte of the chunk within a stage
        const int q = (wave + i * C::NWAVES) * 64 + lane;
        return ((q % C::CA) ^ swz<C::SWZ>(q / C::CA, C::CA)) * 16;
    };
    auto w_kb = [&](int i) {
        const int q = (wave + i * C::NWAVES) * 64 + lane;
        return ((q % C::CW) ^ swz<C::SWZ>(q / C::CW, C::CW)) * 16;
    };
#pragma unroll
    for (int i = 0; i < C::A_PER_WAVE; ++i) {
        const int row = ((wave + i * C::NWAVES) * 64 + lane) / C::CA;
        a_off[i] = wave + i * C::NWAVES < C::A_WLOADS
                       ? (uint32_t)(row * (int)lda * C::AB + a_kb(i)) : kOOB;
    }
#pragma unroll
    for (int i = 0; i < C::W_PER_WAVE; ++i) {
        const int row = ((wave + i * C::NWAVES) * 64 + lane) / C::CW;
        w_off[i] = wave + i * C::NWAVES < C::W_WLOADS ? (uint32_t)(row * (int)wrow + w_kb(i))
                                                      : kOOB;
    }
    const int KT = (int)((KL + C::BK - 1) / C::BK);  // stages of this slice
    // DMA of stage kt into LDS buffer buf.  Every call issues the same number
    // of loads; a stage past the end (or a chunk past K) reads out of range,
    // which writes zeros and touches no memory, so the vector-memory counter
    // advances identically every step.
    auto issue_one = [&](int kt, int buf, int idx) {  // idx < LOADS, compile-time
        MQ_LDS int8_t* base = (MQ_LDS int8_t*)smem + buf * C::STAGE;
        if (idx < C::A_PER_WAVE) {
            const int i = idx, k0 = kt * C::BKA;  // bytes
            const int wl = wave + i * C::NWAVES;
            // the stage's bytes left in the row (uniform): one compare per
            // chunk against a lane constant, no per-lane sum
            const int left = __builtin_amdgcn_readfirstlane((int)KL * C::AB - k0);
            // the stage's K offset goes in the scalar offset: the lane's
            // offset is its constant one, or out of range (which the
            // hardware's range check turns into zeros whatever the scalar
            // part adds)
            const uint32_t voff = a_kb(i) < left ? a_off[i] : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(ra, (MQ_LDS void*)(base + wl * 1024), 16,
                                                     voff, (uint32_t)k0, 0, 0);
        } else {
            const int i = idx - C::A_PER_WAVE, k0w = kt * C::BKW;
            const int wl = wave + i * C::NWAVES;
            const int left = __builtin_amdgcn_readfirstlane((int)KLw - k0w);
            const uint32_t voff = w_kb(i) < left ? w_off[i] : kOOB;
            __builtin_amdgcn_raw_ptr_buffer_load_lds(
                rw, (MQ_LDS void*)(base + C::A_BYTES + wl * 1024), 16, voff, (uint32_t)k0w, 0, 0);
        }
    };
    auto issue = [&](int kt, int buf) {
#pragma unroll
        for (int idx = 0; idx < C::LOADS; ++idx) issue_one(kt, buf, idx);
    };

    // ---- per-column inputs first: the vector-memory counter retires in
    // issue order, so these loads are back before the stage DMA behind them
    // and the constants are derived while the first tiles are in flight
    float col_ws = 1.0f, col_bias = 0.0f;
    int32_t col_cs = 0, col_zw = 0, row_sum = 0;
    if (tid < C::TN) {
        int64_t n = n_tile + tid;
        if (n >= p.N) n = p.N - 1;
        col_ws = p.w_scale[STR ? n * p.ws_stride : n];
        col_cs = p.colsum[STR ? bg * p.cs_bs + (p.in_causal >= 0 ? m_blk * p.cs_mt : 0) + n : n];
        // branch-free; without bias the (unused) load reads w_scale[0]
        col_bias = (p.bias ? p.bias : p.w_scale)[p.bias ? n : 0];
        if constexpr (CASYM) col_zw = p.w_zp[n];
    }
    int32_t row_hi = 0;
    if (CASYM && tid < C::TM) row_sum = p.a_rowsum[tid < rows_a ? m_tile + tid : m_tile];
    if (ROFF && tid < C::TM) {
        const int64_t v = p.row_off[bt * p.ro_bs + (tid < rows_a ? m_tile + tid : m_tile)];
        row_sum = (int32_t)(uint32_t)(uint64_t)v;
        row_hi = (int32_t)(v >> 32);
    }
#pragma unroll
    for (int s = 0; s < C::STAGES - 1; ++s) issue(s, s);
    // keep every use of the loaded values behind the DMA issue
    asm volatile("" : "+v"(col_ws), "+v"(col_cs), "+v"(col_bias));
    if constexpr (CASYM) asm volatile("" : "+v"(col_zw), "+v"(row_sum));
    if constexpr (ROFF) asm volatile("" : "+v"(row_sum), "+v"(row_hi));
    if (CASYM && tid < C::TM) e_rs[tid] = row_sum - (int32_t)K * p.a_zp;
    if (ROFF && tid < C::TM) {
        e_rs[tid] = row_sum;
        e_rhi[tid] = row_hi;
    }

    int col_pre0 = 1, col_fold = 1, col_offin = 1;
    if (tid < C::TN) {
        const ColParams cp = derive_col_params_v(p.a_scale, col_ws, p.out_scale, p.bias != nullptr,
                                                 col_bias, col_cs, p.a_zp);
        const EpiInt ei = epi_int_params(cp);
        e_off[tid] = cp.off;
        e_m0[tid] = ei.m0;
        e_rnd[tid] = ei.rnd;
        e_sp[tid] = ei.shr | (ei.pre << 8);
        col_pre0 = ei.pre == 0;
        // out_zp * 2^shr can join the rounding constant when the sum stays
        // at most 2^30 (then mul_hi + it cannot overflow int32)
        const int64_t zabs = p.out_zp < 0 ? -(int64_t)p.out_zp : (int64_t)p.out_zp;
        col_fold = (int64_t)ei.rnd + (zabs << ei.shr) <= ((int64_t)1 << 30);
        // off can start the accumulator (scaled by 16 for int4 weights)
        // when no partial sum can leave int32: |acc| <= K * 128 * 128 =
        // K * 2^14, so the saturating add of the epilogue never saturates.
        // With asymmetric weights the start value also holds the zero-point
        // term -w_zp * rs, |rs| <= 255 K, formed by a 24-bit multiply
        // (|rs| < 2^23).
        int64_t offa = cp.off < 0 ? -(int64_t)cp.off : (int64_t)cp.off;
        if constexpr (CASYM) {
            e_nzw[tid] = -col_zw;
            offa += (col_zw < 0 ? -(int64_t)col_zw : (int64_t)col_zw) * 255 * K;
        }
        offa *= C::WBITS == 4 ? 16 : 1;
        col_offin = offa + (K << 14) < ((int64_t)1 << 31) &&
                    (!CASYM || 255 * K < ((int64_t)1 << 23));
        if constexpr (C::A16) {
            // the offset bias_q + (128 - a_zp) colsum (int64) split as
            // 256 hi + lo, lo in [0, 255]; hi starts the high-plane sums
            // when hi + K * 2^14 stays in int32
            const int64_t off = a16_offset(cp, p.a_zp, col_cs);
            const int64_t hi = off >> 8;  // floor
            e_off[tid] = (int32_t)hi;
            e_nzw[tid] = (int32_t)(off - hi * 256);
            col_offin = (hi < 0 ? -hi : hi) + (K << 14) < ((int64_t)1 << 31);
        }
    }
    // Whole-tile epilogue form: AND of the column flags over the block, by
    // ballot per wave and one LDS word per wave.  A raw barrier, since
    // __syncthreads() would also drain the stage DMA.
    {
        const bool w_pre0 = __ballot(col_pre0) == ~0ull;
        const bool w_fold = __ballot(col_fold) == ~0ull;
        const bool w_offin = __ballot(col_offin) == ~0ull;
        if (lane == 0) e_flag[wave] = (w_pre0 ? 1 : 0) | (w_fold ? 2 : 0) | (w_offin ? 4 : 0);
    }
    __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14));  // lgkmcnt(0)
    __builtin_amdgcn_s_barrier();
    int flags = 7;
#pragma unroll
    for (int w = 0; w < C::NWAVES; ++w) flags &= e_flag[w];
    flags = __builtin_amdgcn_readfirstlane(flags);
    const bool zp_fold = (flags & 2) != 0;
    // the fast epilogue form: one mul_hi per output, zero-point in the
    // rounding constant, off in the accumulator's start value; pre0: no
    // column of the tile needs the pre-shift
    const bool pre0 = (flags & 1) != 0;
    const bool fast = (flags & 6) == 6 && (p.N % 4) == 0;
    if (zp_fold && tid < C::TN) e_rnd[tid] += p.out_zp * (1 << (e_sp[tid] & 0xFF));
    // stage STAGES-1: the part the stage switch step would issue; the rest
    // goes out during the first stage's steps, as for every later stage
#pragma unroll
    for (int d = 0; d < C::LOADS; ++d)
        if (C::dma_slot(d) < C::NRD) issue_one(C::STAGES - 1, C::STAGES - 1, d);
    // stage 0 is complete when only the loads issued after it are in
    // flight, in every wave
    wait_vmcnt<(C::STAGES - 2) * C::LOADS + C::NSW>();
    __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14));
    __builtin_amdgcn_s_barrier();

    // ---- accumulators.  Layout:
    // lane holds channels col0 + 32i + 8g + 4hk + r (register 4g + r) of
    // tokens 32j + r32.  In the fast form each starts at its channel's off
    // (plus, for asymmetric weights, -w_zp[n] * rs[m]), scaled by 16 for
    // int4 weights like the products.
    // 16-bit activations: acc holds the high-byte plane, acc2 the low one
    // (each starting at its part of the offset in the fast form)
    v16i acc[C::FN][C::FM];
    v16i acc2[C::A16 ? C::FN : 1][C::A16 ? C::FM : 1];
#pragma unroll
    for (int i = 0; i < C::FN; ++i)
#pragma unroll
        for (int j = 0; j < C::FM; ++j)
#pragma unroll
            for (int r = 0; r < 16; ++r) acc[i][j][r] = 0;
    if constexpr (C::A16) {
#pragma unroll
        for (int i = 0; i < C::FN; ++i)
#pragma unroll
            for (int j = 0; j < C::FM; ++j)
#pragma unroll
                for (int r = 0; r < 16; ++r) acc2[i][j][r] = 0;
    }
    if (fast && split == 0) {  // block-uniform; off joins the sum once
        const int col0 = wn * (C::TN / C::WN) + 4 * hk;
        int32_t rs[C::FM];
#pragma unroll
        for (int j = 0; j < C::FM; ++j)
            rs[j] = CASYM ? e_rs[wm * (C::TM / C::WM) + j * 32 + r32] : 0;
#pragma unroll
        for (int i = 0; i < C::FN; ++i)
#pragma unroll
            for (int g = 0; g < 4; ++g) {
                const v4i o = *reinterpret_cast<const v4i*>(e_off + col0 + i * 32 + 8 * g);
                v4i z = {0, 0, 0, 0};
                if constexpr (CASYM || C::A16)
                    z = *reinterpret_cast<const v4i*>(e_nzw + col0 + i * 32 + 8 * g);
#pragma unroll
                for (int j = 0; j < C::FM; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        int32_t v = o[r];
                        if constexpr (CASYM) v += __mul24(z[r], rs[j]);
                        if constexpr (C::WBITS == 4) v *= 16;
                        acc[i][j][4 * g + r] = v;
                        if constexpr (C::A16) acc2[i][j][4 * g + r] = z[r];
                    }
            }
    }

    // ---- main loop.  Fragments of the next 32-deep step are read from LDS
    // while the MFMAs of the current one run; at the last step of a stage
    // the stage switch (wait, barrier, next DMA, first fragments of the next
    // stage) sits between the two halves of the step's MFMAs.  The steady
    // state has no branches, so every wait count is a compile-time constant.

    // fragment read g of a 32-deep step: g < FM*AB activation rows (16-bit
    // codes: two 16-byte halves per fragment, af[2j] and af[2j+1]), then
    // weight rows
    auto load_frag = [&](int buf, int ks, int g, v4i* wf, v4i* af) {
        const int8_t* sa = smem + buf * C::STAGE;
        const int8_t* sw = sa + C::A_BYTES;
        if (g < C::FM * C::AB) {
            const int row = wm * (C::TM / C::WM) + (g / C::AB) * 32 + r32;
            const int chunk = C::A16 ? ks * 4 + hk * 2 + (g % 2) : ks * 2 + hk;
            const int phys = chunk ^ swz<C::SWZ>(row, C::CA);
            af[g] = *reinterpret_cast<const v4i*>(sa + row * C::BKA + phys * 16);
        } else {
            const int i = g - C::FM * C::AB;
            const int row = wn * (C::TN / C::WN) + i * 32 + r32;
            if constexpr (C::WBITS == 8) {
                const int phys = (ks * 2 + hk) ^ swz<C::SWZ>(row, C::CW);
                wf[i] = *reinterpret_cast<const v4i*>(sw + row * C::BKW + phys * 16);
            } else {
                // the 32 weights of this k step are one packed 16-byte chunk;
                // they stay packed until the step that multiplies them, so the
                // read's latency is hidden behind a whole step as for int8
                const int phys = ks ^ swz<C::SWZ>(row, C::CW);
                typedef unsigned v2u __attribute__((ext_vector_type(2)));
                const v2u pk =
                    *reinterpret_cast<const v2u*>(sw + row * C::BKW + phys * 16 + hk * 8);
                wf[i] = v4i{(int)pk[0], (int)pk[1], 0, 0};
            }
        }
    };
    // MFMA t of a step: channel fragment t / FM, token fragment t % FM; with
    // 16-bit codes (af = the split planes, high at 2j, low at 2j+1) the
    // plane is t % 2 and the pair index t / 2
    auto mfma_range = [&](const v4i* wf, const v4i* af, int t0, int t1) {
        v4i wu = {0, 0, 0, 0};  // the unpacked int4 channel fragment
#pragma unroll
        for (int t = t0; t < t1; ++t) {
            if constexpr (C::A16) {
                const int q = t / 2, i = q / C::FM, j = q % C::FM;
                if (t % 2 == 0)
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wf[i], af[2 * j], acc[i][j],
                                                                      0, 0, 0);
                else
                    acc2[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wf[i], af[2 * j + 1],
                                                                       acc2[i][j], 0, 0, 0);
            } else {
                const int i = t / C::FM, j = t % C::FM;
                if constexpr (C::WBITS == 4) {
                    // packed int4: unpacked to 16*w where the group first
                    // multiplies this channel fragment (t is a compile-time
                    // constant, so the test folds away)
                    if (t == t0 || j == 0)
                        wu = unpack_int4_x16((uint32_t)wf[i][0], (uint32_t)wf[i][1]);
                    acc[i][j] = __builtin_amdgcn_mfma_i32_32x32x32_i8(wu, af[j], acc[i][j], 0, 0, 0);
                } else {
                    acc[i][j] =
                        __builtin_amdgcn_mfma_i32_32x32x32_i8(wf[i], af[j], acc[i][j], 0, 0, 0);
                }
            }
        }
    };

    // One 32-deep step in NRD groups, each: one LDS read of the next step's
    // fragments, this step's share of MFMAs, and (at a stage switch) one DMA
    // of a later stage.  sched_barrier fences keep the groups in this order:
    // a wave stalled on a full load queue (DMA issue) or on an LDS read
    // would otherwise stop feeding its MFMA pipe for the whole bunch.
    // Measured on MI355X: one wave per SIMD reaches ~83% of the int8 MFMA
    // peak with one LDS read per two MFMAs, against ~60-77% with the reads
    // bunched.
    // The DMA of a stage is spread evenly over the KS*NRD groups that follow
    // the barrier which frees its buffer: the stage switch step (slots
    // 0..NRD-1) and the first KS-1 steps of the next stage.
    constexpr int NRD = C::NRD;                  // LDS fragment reads per step
    constexpr int NMF = C::FN * C::FM * C::AB;   // MFMAs per step
    auto step = [&](const v4i* wc, const v4i* ac, bool read, int rbuf, int rks, v4i* wx,
                    v4i* ax, bool dma, int dkt, int dbuf, int slot_step) {
        // 16-bit codes: this step's byte planes (its fragments were read
        // during the previous step)
        v4i planes[C::A16 ? 2 * C::FM : 1];
        if constexpr (C::A16) {
#pragma unroll
            for (int j = 0; j < C::FM; ++j)
                split_a16(ac[2 * j], ac[2 * j + 1], planes[2 * j], planes[2 * j + 1]);
        }
        const v4i* aop = C::A16 ? planes : ac;
#pragma unroll
        for (int g = 0; g < NRD; ++g) {
            if (read) load_frag(rbuf, rks, g, wx, ax);
            mfma_range(wc, aop, g * NMF / NRD, (g + 1) * NMF / NRD);
            if (dma) {
#pragma unroll
                for (int d = 0; d < C::LOADS; ++d)
                    if (C::dma_slot(d) == slot_step * NRD + g) issue_one(dkt, dbuf, d);
            }
            __builtin_amdgcn_sched_barrier(0);
        }
    };

    v4i wf0[C::FN], af0[C::FM * C::AB], wf1[C::FN], af1[C::FM * C::AB];
#pragma unroll
    for (int g = 0; g < NRD; ++g) load_frag(0, 0, g, wf0, af0);
    // One stage kt (followed by a stage switch) held in LDS buffer bufv.  The
    // main loop passes the buffer as a compile-time constant (its stages
    // unrolled by STAGES), so a fragment read's LDS address is a lane offset
    // held across the loop plus an immediate: no address arithmetic per read.
    auto run_stage = [&](int kt, auto bufv) {
        const int buf = (int)bufv;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            v4i* wc = (ks & 1) ? wf1 : wf0;
            v4i* ac = (ks & 1) ? af1 : af0;
            v4i* wx = (ks & 1) ? wf0 : wf1;
            v4i* ax = (ks & 1) ? af0 : af1;
            if (ks + 1 < KS) {
                // the rest of the DMA of stage kt+STAGES-1 (its buffer was
                // freed by the previous stage switch)
                step(wc, ac, true, buf, ks + 1, wx, ax, true, kt + C::STAGES - 1,
                     (buf + C::STAGES - 1) % C::STAGES, ks + 1);
            } else {
                // Stage switch at the start of the stage's last step: this
                // step's fragments are already in registers, so buffer `buf`
                // is no longer read by this wave once lgkmcnt reaches 0.
                // Stage kt+1 is complete when only the STAGES-2 stages
                // issued after it are in flight.
                wait_vmcnt<(C::STAGES - 2) * C::LOADS>();
                // Raw barrier: __syncthreads() adds a workgroup release
                // fence that drains every outstanding load.
                __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14));
                __builtin_amdgcn_s_barrier();
                __builtin_amdgcn_sched_barrier(0);
                step(wc, ac, true, (buf + 1) % C::STAGES, 0, wx, ax, true, kt + C::STAGES, buf, 0);
            }
        }
    };
    using B0 = std::integral_constant<int, 0>;
    using B1 = std::integral_constant<int, 1>;
    using B2 = std::integral_constant<int, 2>;
    using B3 = std::integral_constant<int, 3>;
    int kt0 = 0;  // a multiple of STAGES: stage kt0 + b sits in buffer b
    for (; kt0 + C::STAGES <= KT - 1; kt0 += C::STAGES) {
        run_stage(kt0, B0{});
        run_stage(kt0 + 1, B1{});
        if constexpr (C::STAGES > 2) run_stage(kt0 + 2, B2{});
        if constexpr (C::STAGES > 3) run_stage(kt0 + 3, B3{});
    }
    // the fewer than STAGES stages with a switch that remain
    if (kt0 < KT - 1) run_stage(kt0, B0{});
    if constexpr (C::STAGES > 2)
        if (kt0 + 1 < KT - 1) run_stage(kt0 + 1, B1{});
    if constexpr (C::STAGES > 3)
        if (kt0 + 2 < KT - 1) run_stage(kt0 + 2, B2{});
    {  // last stage: no switch
        const int buf = (KT - 1) % C::STAGES;
#pragma unroll
        for (int ks = 0; ks < KS; ++ks) {
            v4i* wc = (ks & 1) ? wf1 : wf0;
            v4i* ac = (ks & 1) ? af1 : af0;
            v4i* wx = (ks & 1) ? wf0 : wf1;
            v4i* ax = (ks & 1) ? af0 : af1;
            step(wc, ac, ks + 1 < KS, buf, ks + 1, wx, ax, false, 0, 0, 0);
        }
    }

    // ---- K slices: every block stores its partial sums (int32, in the
    // accumulator register layout, so each lane's 16-byte chunks are
    // contiguous across the block) and counts itself in at its tile's
    // counter; the last block to arrive adds the other slices (exact integer
    // sums), returns the counter to zero for the next call and runs the
    // epilogue.  Nobody waits for anybody, so no schedule can deadlock.
    // The slices of a tile may run on different XCDs (separate L2s): the
    // partial sums are written through to memory and read around the caches
    // (sc0 sc1), and the counter is a system-scope atomic, which keeps the
    // exchange coherent without writing back or invalidating whole L2s.
    wait_vmcnt<0>();  // the out-of-range DMA of the last steps is retired
    if (C::SPLITK && splits > 1) {
        constexpr int CHUNKS = C::FN * C::FM * 4;  // 16-byte chunks per lane
        constexpr int kCoherent = 1 | 16;          // cache policy sc0 | sc1
        int32_t* counters = static_cast<int32_t*>(p.ws);
        const int64_t part_bytes = (int64_t)CHUNKS * C::THREADS * 16;  // one block's slice
        const __amdgpu_buffer_rsrc_t rp = __builtin_amdgcn_make_buffer_rsrc(
            static_cast<int8_t*>(p.ws) + split_counter_bytes(total) +
                (int64_t)tile * splits * part_bytes,
            (short)0, (int)(splits * part_bytes), 0x00020000);
        auto chunk_off = [&](int s, int i, int j, int g) {
            return (uint32_t)(s * part_bytes +
                              ((int64_t)((i * C::FM + j) * 4 + g) * C::THREADS + tid) * 16);
        };
#pragma unroll
        for (int i = 0; i < C::FN; ++i)
#pragma unroll
            for (int j = 0; j < C::FM; ++j) {
#pragma unroll
                for (int g = 0; g < 4; ++g) {
                    const v4i v = {acc[i][j][4 * g], acc[i][j][4 * g + 1], acc[i][j][4 * g + 2],
                                   acc[i][j][4 * g + 3]};
                    __builtin_amdgcn_raw_buffer_store_b128(v, rp, chunk_off(split, i, j, g), 0,
                                                           kCoherent);
                }
                __builtin_amdgcn_sched_barrier(0);  // one fragment at a time: bounded registers
            }
        wait_vmcnt<0>();  // this wave's partial sums have reached memory
        __syncthreads();
        if (tid == 0)
            e_flag[0] = __hip_atomic_fetch_add(counters + tile, 1, __ATOMIC_RELAXED,
                                               __HIP_MEMORY_SCOPE_SYSTEM);
        __syncthreads();
        const int arrived = e_flag[0];
        __syncthreads();  // everybody has read the count before e_flag is reused
        if (arrived != splits - 1) return;
        // the other slices, 16 chunks (64 registers) in flight per batch: each
        // batch costs one memory round trip, not one per chunk
        constexpr int IB = C::MERGE_IB;  // fragment rows per batch
        for (int s = 0; s < splits; ++s) {
            if (s == split) continue;
#pragma unroll
            for (int i0 = 0; i0 < C::FN; i0 += IB) {
                v4i tmp[IB][C::FM][4];
#pragma unroll
                for (int i = 0; i < IB; ++i)
#pragma unroll
                    for (int j = 0; j < C::FM; ++j)
#pragma unroll
                        for (int g = 0; g < 4; ++g)
                            tmp[i][j][g] = __builtin_amdgcn_raw_buffer_load_b128(
                                rp, chunk_off(s, i0 + i, j, g), 0, kCoherent);
#pragma unroll
                for (int i = 0; i < IB; ++i)
#pragma unroll
                    for (int j = 0; j < C::FM; ++j)
#pragma unroll
                        for (int g = 0; g < 4; ++g)
#pragma unroll
                            for (int r = 0; r < 4; ++r) acc[i0 + i][j][4 * g + r] += tmp[i][j][g][r];
                __builtin_amdgcn_sched_barrier(0);
            }
        }
        if (tid == 0)
            __hip_atomic_exchange(counters + tile, 0, __ATOMIC_RELAXED, __HIP_MEMORY_SCOPE_SYSTEM);
    }

    // ---- epilogue, straight from the accumulators (see prefill_epilogue)
    __builtin_amdgcn_s_waitcnt((0 << 8) | (7 << 4) | 15 | (3 << 14));
    __builtin_amdgcn_s_barrier();  // e_rnd update visible even when KT == 1
    EpiCtx ctx;
    ctx.e_nzw = e_nzw;
    ctx.e_rs = e_rs;
    ctx.e_rhi = e_rhi;
    ctx.e_off = e_off;
    ctx.e_m0 = e_m0;
    ctx.e_rnd = e_rnd;
    ctx.e_sp = e_sp;
    ctx.row_bytes = (int32_t)((STR ? eff_ldy(p) : p.N) * (C::OBITS / 8));
    ctx.lane_row_off = (wm * (C::TM / C::WM) + r32) * ctx.row_bytes;
    ctx.col0 = wn * (C::TN / C::WN) + 4 * hk;
    ctx.n_left = (int32_t)(p.N - n_tile);
    ctx.n_tile = (int32_t)n_tile;
    ctx.out_zp = zp_fold ? 0 : p.out_zp;
    ctx.r32 = r32;
    ctx.wave_row0 = wm * (C::TM / C::WM);
    ctx.wave_col0 = wn * (C::TN / C::WN);
    ctx.stage = (MQ_LDS int8_t*)smem + wave * Staging<C>::BYTES;
    int8_t* const y_batch =
        static_cast<int8_t*>(p.y) + (STR ? bt * p.y_bs * (C::OBITS / 8) : 0);
    ctx.ry = __builtin_amdgcn_make_buffer_rsrc(
        (void*)(y_batch + m_tile * (int64_t)ctx.row_bytes), (short)0,
        (int)(rows_a * ctx.row_bytes), 0x00020000);
    // staged stores need the tile's channels inside N and 16-byte row chunks
    const bool staged = fast && n_tile + C::TN <= p.N && (ctx.row_bytes % 16) == 0 &&
                        ((uintptr_t)y_batch % 16) == 0;
    if constexpr (YF) {
        ctx.out_scale = p.out_scale;
        ctx.out_zp_code = p.out_zp;
        ctx.row_bytes_f = (int32_t)(p.N * 4);
        ctx.lane_row_off_f = (wm * (C::TM / C::WM) + r32) * ctx.row_bytes_f;
        ctx.has_codes = p.y != nullptr;
        ctx.ryf = __builtin_amdgcn_make_buffer_rsrc(
            (void*)(p.y_f + m_tile * p.N), (short)0, (int)(rows_a * ctx.row_bytes_f),
            0x00020000);
        // staged: the tile's channels inside N, 16-byte fp32 row chunks, and
        // the codes' own rules when they are stored too
        const bool staged_f = fast && n_tile + C::TN <= p.N && (p.N % 4) == 0 &&
                              (!ctx.has_codes || staged);
        if (staged_f && pre0)
            prefill_epilogue<C, ASYM, true, false, true, true>(acc, acc2, ctx);
        else if (staged_f) prefill_epilogue<C, ASYM, true, true, true, true>(acc, acc2, ctx);
        else if (fast && pre0) prefill_epilogue<C, ASYM, true, false, false, true>(acc, acc2, ctx);
        else if (fast) prefill_epilogue<C, ASYM, true, true, false, true>(acc, acc2, ctx);
        else prefill_epilogue<C, ASYM, false, false, false, true>(acc, acc2, ctx);
        return;
    }
    if (staged && pre0) prefill_epilogue<C, ASYM, true, false, true, false>(acc, acc2, ctx);
    else if (staged) prefill_epilogue<C, ASYM, true, true, true, false>(acc, acc2, ctx);
    else if (fast) prefill_epilogue<C, ASYM, true, true, false, false>(acc, acc2, ctx);
    else prefill_epilogue<C, ASYM, false, false, false, false>(acc, acc2, ctx);
}

template <class C, bool ASYM>
__global__ __launch_bounds__(C::THREADS, C::OCC) void qlinear_prefill_kernel(QLinearArgs p,
                                                                       int tiles_n, int tiles_m,
                                                                       int splits,
                                                                       int kt_per_split)
{
    prefill_body<C, ASYM, false>(p, nullptr, tiles_n, tiles_m, splits, kt_per_split);
}

// the dequantized outputs (fp32) written by the epilogue, the codes too
// when p.y is set
template <class C, bool ASYM>
__global__ __launch_bounds__(C::THREADS, C::OCC) void qlinear_prefill_dequant_kernel(
    QLinearArgs p, int tiles_n, int tiles_m, int splits, int kt_per_split)
{
    prefill_body<C, ASYM, false, true>(p, nullptr, tiles_n, tiles_m, splits, kt_per_split);
}

// several linears on one input, without a K split (kt: K stages)
template <class C, bool ASYM>
__global__ __launch_bounds__(C::THREADS, C::OCC) void qlinear_prefill_group_kernel(
    QLinearArgs p, GroupArgs g, int tiles_n, int tiles_m, int kt)
{
    prefill_body<C, ASYM, true>(p, &g, tiles_n, tiles_m, 1, kt);
}

template <class C, bool ASYM>
hipError_t launch_cfg(const QLinearArgs& p, int splits, hipStream_t s)
{
    const int64_t tiles_n = (p.N + C::TN - 1) / C::TN;
    const int64_t tiles_m = (p.M + C::TM - 1) / C::TM;
    const int64_t total = tiles_n * tiles_m;
    const int64_t kt = (p.K + C::BK - 1) / C::BK;
    const int64_t kt_per_split = (kt + splits - 1) / splits;
    splits = (int)((kt + kt_per_split - 1) / kt_per_split);  // every slice non-empty
    if (total * splits > 0x7FFFFFFF || p.batch > 65535) return hipErrorInvalidValue;
    // more than 64 KiB of dynamic LDS must be opted into once per kernel
    constexpr int lds = ASYM || C::A16 ? C::LDS_ASYM : C::LDS;
    const dim3 grid((unsigned)(total * splits), (unsigned)p.batch);
    if constexpr (!C::A16) {
        if (p.y_f) {
            static const hipError_t attr_f = hipFuncSetAttribute(
                reinterpret_cast<const void*>(&qlinear_prefill_dequant_kernel<C, ASYM>),
                hipFuncAttributeMaxDynamicSharedMemorySize, lds);
            if (attr_f != hipSuccess) return attr_f;
            qlinear_prefill_dequant_kernel<C, ASYM><<<grid, dim3(C::THREADS), lds, s>>>(
                p, (int)tiles_n, (int)tiles_m, splits, (int)kt_per_split);
            return hipGetLastError();
        }
    }
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&qlinear_prefill_kernel<C, ASYM>),
        hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (attr != hipSuccess) return attr;
    qlinear_prefill_kernel<C, ASYM><<<grid, dim3(C::THREADS), lds, s>>>(
        p, (int)tiles_n, (int)tiles_m, splits, (int)kt_per_split);
    return hipGetLastError();
}

template <class C, bool ASYM>
hipError_t launch_group_cfg(const QLinearArgs& p, GroupArgs g, hipStream_t s)
{
    const int64_t tiles_m = (p.M + C::TM - 1) / C::TM;
    int64_t cols = 0;
    for (int i = 0; i < g.n; ++i) {
        g.part[i].tile0 = (int32_t)(cols * tiles_m);
        g.part[i].tiles_n = (int32_t)((g.part[i].N + C::TN - 1) / C::TN);
        cols += g.part[i].tiles_n;
        if (cols * tiles_m > 0x7FFFFFFF) return hipErrorInvalidValue;
    }
    const int64_t kt = (p.K + C::BK - 1) / C::BK;
    constexpr int lds = ASYM ? C::LDS_ASYM : C::LDS;
    static const hipError_t attr = hipFuncSetAttribute(
        reinterpret_cast<const void*>(&qlinear_prefill_group_kernel<C, ASYM>),
        hipFuncAttributeMaxDynamicSharedMemorySize, lds);
    if (attr != hipSuccess) return attr;
    qlinear_prefill_group_kernel<C, ASYM><<<dim3((unsigned)(cols * tiles_m)), dim3(C::THREADS),
                                            lds, s>>>(p, g, (int)cols, (int)tiles_m, (int)kt);
    return hipGetLastError();
}

// Tile shapes.  (tokens x channels, wave grid, K bytes per stage, stages,
// swizzle, steps the DMA of a stage is spread over; measured: the
// 128-deep four-wave tiles are fastest with the DMA spread over the whole
// stage.)  A four-wave 256x256 tile (4x4 fragments per wave, 256
// accumulator registers, no K split) was slower than the eight-wave one on
// every measured shape and is gone.
template <int WB, int OB> using T256x128 = Cfg<WB, OB, 256, 128, 2, 2, 128, 3, 2, 4>;
constexpr int kTile256x128 = 0;
template <int WB, int OB> using T128x128 = Cfg<WB, OB, 128, 128, 2, 2, 128, 4, 2, 4>;
constexpr int kTile128x128 = 1;
// 64x64: layers with few output tiles (1024 tokens x 256 channels: 64
// tiles instead of 16), four waves of 32x32
template <int WB, int OB> using T64x64 = Cfg<WB, OB, 64, 64, 2, 2, 128, 4, 2, 4>;
constexpr int kTile64x64 = 3;
// 192 tokens x 256 channels: 3/4 of the 256x256 tile's work per block, so a
// layer whose 256x256 tiles leave CUs idle (2048 x 5632: 176 tiles on 256
// CUs) fills more of the chip (242 tiles).  Eight waves, two per SIMD, each
// 96 tokens x 64 channels: while one wave of a SIMD waits (stage barrier,
// LDS reads, DMA issue) the other keeps the matrix core busy, and the two
// interleave their epilogues (measured on MI355X: ~9% faster than four
// waves of 96 x 128).  Two stages of 128 k (one in flight while the other
// is read, its DMA spread over two steps) beat four of 64: half the stage
// barriers, 27.2-28.0 against 29.1-29.2 us on the 2048x2048x5632 layer.
// int4 weights keep four waves: their smaller stages leave no room for
// eight waves' staged stores.
template <int WB, int OB>
using T192x256 = std::conditional_t<WB == 8, Cfg<WB, OB, 192, 256, 2, 4, 128, 2, 2, 2>,
                                    Cfg<WB, OB, 192, 256, 2, 2, 64, 4, 2, 1>>;
constexpr int kTile192x256 = 2;
// 256x256 with eight waves, two per SIMD, each 128 tokens x 64 channels (4x2
// fragments: 8 MFMAs per 6 fragment reads from LDS, against 6 per 5 for the
// 192x256 tile's 3x2), two 128-deep stages.  128 accumulator registers per
// wave leave room for the K split and the pre-shift epilogue forms.
template <int WB, int OB> using T256x256W8 = Cfg<WB, OB, 256, 256, 2, 4, 128, 2, 2, 2>;
constexpr int kTile256x256W8 = 4;
// 128 tokens x 64 channels, four waves of 64 x 32 (two fragments each: one
// weight fragment read per two MFMAs, where 64x64 has one per MFMA), four
// 128-deep stages, one work-group per CU: the layers at 1024 tokens with a
// long K and 256 such tiles (1024 x 5632 -> 2048: 18.5 against 21.8 us on
// 64x64, measured).  The cost model offers it for int8 weights with
// K >= 4096 and no K split only (int4 weights: 64x64 stays ahead).
template <int WB, int OB> using T128x64 = Cfg<WB, OB, 128, 64, 2, 2, 128, 4, 2, 4>;
constexpr int kTile128x64 = 5;
// 16-bit activation codes: 128x128 tokens x channels, 64 k per stage (128
// bytes of each activation row), DMA spread over both steps of a stage
template <int OB> using T128x128A16 = Cfg<8, OB, 128, 128, 2, 2, 64, 4, 2, 2, 16>;
// short K (<= 128 codes, e.g. the attention scores over a 64-dimensional
// head): two stages are all the pipeline needs, and half the LDS lets two
// work-groups share a CU, so one's prologue and epilogue overlap the
// other's products
template <int OB> using T128x128A16S2 = Cfg<8, OB, 128, 128, 2, 2, 64, 2, 2, 1, 16>;
// at most 64 channels (P V over a 64-dimensional head): a 128x128 tile
// would leave half of its products and weight loads idle, and 64-row tiles
// double the work-groups (P V at 1024 tokens: 512 instead of 256; the
// causal form's longest tile has half the rows)
template <int OB> using T64x64A16 = Cfg<8, OB, 64, 64, 2, 2, 64, 4, 2, 2, 16>;
static_assert(T128x128A16S2<8>::A16_I32 && !T128x128A16<8>::A16_I32 &&
                  !T64x64A16<8>::A16_I32,
              "the int32 epilogue belongs to the short-K tile");
static_assert(T128x128A16<8>::TM == kA16TileM && T128x128A16<8>::BK == kA16TileK &&
                  T128x128A16S2<8>::TM == kA16TileM && T128x128A16S2<8>::BK == kA16TileK &&
                  kA16TileM % T64x64A16<8>::TM == 0 && T64x64A16<8>::BK == kA16TileK,
              "the causal column sums assume these 16-bit tile sizes");

// Time model of each tile shape on MI355X, fitted to forced-tile
// measurements of the workload layers (graph replay, one box; every tile on
// M = 512..2048, K = 2048..16384, N = 256..256000, int8 and int4 weights).
// A block costs a fixed part (the first memory round trip, the epilogue and
// its stores) plus a time per K stage; with more CUs busy a stage takes
// longer (the chip clocks down under the MFMA load and the blocks share the
// memory system): stage * (1 + kBusySlowdown * busy fraction).  occ blocks
// share a CU within one round.  Units: microseconds.  Over the 60 measured
// (shape, tile) points the model is within about 20%, and it picks the
// measured fastest tile on every one of the ten unsplit shapes.
struct TileModel {
    int tm, tn, bk;
    double fixed_us, stage_us;
    int occ = 1;
    bool splits = true;  // whether the tile takes a K split
};
constexpr TileModel kTiles[] = {
    {256, 128, 128, 8.05, 0.593},
    {128, 128, 128, 5.58, 0.348},
    {192, 256, 128, 6.98, 0.845},  // eight waves, two 128-deep stages (int8 weights)
    {64, 64, 128, 3.63, 0.232, 2},  // 64 KiB of stage ring: two blocks per CU
    {256, 256, 128, 10.5, 0.912},   // eight waves of 128x64, two 128-deep stages
    {128, 64, 128, 5.0, 0.192, 1, false},  // int8 weights, K >= 4096 (see choose)
};
// the 192x256 tile with int4 weights runs four waves on 64-deep stages
constexpr TileModel kTile192x256W4 = {192, 256, 64, 8.0, 0.45};
constexpr int kNumTiles = sizeof(kTiles) / sizeof(kTiles[0]);
static_assert(kNumTiles == MQ_PREFILL_TILES, "one explicit path per tile");
static_assert(kTiles[kTile256x128].tn == T256x128<8, 8>::TN &&
                  kTiles[kTile128x128].tm == T128x128<8, 8>::TM &&
                  kTiles[kTile192x256].tm == T192x256<8, 8>::TM &&
                  kTiles[kTile64x64].tm == T64x64<8, 8>::TM &&
                  kTiles[kTile256x256W8].tn == T256x256W8<8, 8>::TN &&
                  kTiles[kTile256x256W8].bk == T256x256W8<8, 8>::BK &&
                  kTiles[kTile128x64].tm == T128x64<8, 8>::TM &&
                  kTiles[kTile128x64].tn == T128x64<8, 8>::TN,
              "the time model's rows follow the tile indices");
constexpr double kBusySlowdown = 0.60;
// int4 weights: the in-register unpack makes a K-loop stage ~1.35x longer
constexpr double kInt4StageFactor = 1.35;
// A K split adds round trips to memory (partial stores, the counter, the
// partial loads) and moves every slice's int32 tile through memory and back
// (written through, read around the caches): fitted, 5.2 us plus 0.24 us
// per MB of partial sums stored and loaded.
constexpr double kSplitFixedUs = 5.2;
constexpr double kSplitUsPerMB = 0.24;
constexpr int kCUs = 256;
constexpr int kMaxSplits = 8;

struct Choice {
    int tile, splits;
};

// Ns: the output channels of each linear sharing the launch (one group of
// tiles per linear), or nullptr for p.N alone
Choice choose(const QLinearArgs& p, bool can_split, const int64_t* Ns = nullptr, int nN = 1)
{
    Choice best{0, 1};
    double best_t = 1e300;
    // an explicitly requested tile (measurement and test hook of the ABI)
    const int only = p.force_tile >= 0 && p.force_tile < kNumTiles ? p.force_tile : -1;
    for (int c = 0; c < kNumTiles; ++c) {
        if (only >= 0 && c != only) continue;
        // the 128x64 tile (below) only where it was measured ahead
        if (c == kTile128x64 && only < 0 && (p.w_bits != 8 || p.K < 4096)) continue;
        const TileModel& t = c == kTile192x256 && p.w_bits == 4 ? kTile192x256W4 : kTiles[c];
        int64_t cols = 0;
        for (int i = 0; i < nN; ++i) cols += ((Ns ? Ns[i] : p.N) + t.tn - 1) / t.tn;
        const int64_t tiles = ((p.M + t.tm - 1) / t.tm) * cols;
        // ... and with a tile for every CU (with fewer, 64x64 at one
        // work-group per CU is ahead: 512 x 16384 -> 2048 28.2 against
        // 36.9 us, which the 64x64 row of the model does not capture)
        if (c == kTile128x64 && only < 0 && tiles < kCUs) continue;
        const int64_t kt = (p.K + t.bk - 1) / t.bk;
        const int64_t slots = (int64_t)kCUs * t.occ;
        for (int sp = 1; sp <= (can_split && t.splits ? kMaxSplits : 1); sp *= 2) {
            const int64_t per = (kt + sp - 1) / sp;
            if (sp > 1 && per < 4) break;  // slices too thin to pipeline
            const int64_t items = tiles * sp;
            const int64_t rounds = (items + slots - 1) / slots;
            const double busy = (double)(items < slots ? items : slots) / (double)slots;
            const double stage = t.stage_us * (p.w_bits == 4 ? kInt4StageFactor : 1.0) *
                                 (1.0 + kBusySlowdown * busy);
            const double t_blk = t.fixed_us + stage * (double)per;
            const double exchange =
                sp > 1 ? kSplitFixedUs + kSplitUsPerMB * (double)tiles * (2 * sp - 1) * t.tm *
                                             t.tn * 4 * 1e-6
                       : 0.0;
            const double tt = (double)rounds * t_blk + exchange;
            if (tt < best_t * 0.97) {  // a split has to win clearly
                best_t = tt;
                best = {c, sp};
            }
        }
    }
    return best;
}

int64_t workspace_for(const QLinearArgs& p, const Choice& ch)
{
    if (ch.splits <= 1) return 0;
    const TileModel& t = kTiles[ch.tile];
    const int64_t tiles = ((p.M + t.tm - 1) / t.tm) * ((p.N + t.tn - 1) / t.tn);
    return split_counter_bytes(tiles) + tiles * ch.splits * (int64_t)t.tm * t.tn * 4;
}

template <int WB, int OB, bool ASYM>
hipError_t launch_a(const QLinearArgs& p, hipStream_t s)
{
    Choice ch = choose(p, p.ws != nullptr);
    if (ch.splits > 1 && workspace_for(p, ch) > p.ws_bytes) ch = choose(p, false);
    switch (ch.tile) {
    case kTile256x128: return launch_cfg<T256x128<WB, OB>, ASYM>(p, ch.splits, s);
    case kTile192x256: return launch_cfg<T192x256<WB, OB>, ASYM>(p, ch.splits, s);
    case kTile64x64: return launch_cfg<T64x64<WB, OB>, ASYM>(p, ch.splits, s);
    case kTile256x256W8: return launch_cfg<T256x256W8<WB, OB>, ASYM>(p, ch.splits, s);
    case kTile128x64: return launch_cfg<T128x64<WB, OB>, ASYM>(p, ch.splits, s);
    default: return launch_cfg<T128x128<WB, OB>, ASYM>(p, ch.splits, s);
    }
}

template <int WB, int OB>
hipError_t launch_t(const QLinearArgs& p, hipStream_t s)
{
    return p.w_zp ? launch_a<WB, OB, true>(p, s) : launch_a<WB, OB, false>(p, s);
}

template <int WB, int OB, bool ASYM>
hipError_t launch_group_a(const QLinearArgs& p, const GroupArgs& g, hipStream_t s)
{
    int64_t Ns[kMaxGroup];
    for (int i = 0; i < g.n; ++i) Ns[i] = g.part[i].N;
    const Choice ch = choose(p, false, Ns, g.n);
    switch (ch.tile) {
    case kTile256x128: return launch_group_cfg<T256x128<WB, OB>, ASYM>(p, g, s);
    case kTile192x256: return launch_group_cfg<T192x256<WB, OB>, ASYM>(p, g, s);
    case kTile64x64: return launch_group_cfg<T64x64<WB, OB>, ASYM>(p, g, s);
    case kTile256x256W8: return launch_group_cfg<T256x256W8<WB, OB>, ASYM>(p, g, s);
    case kTile128x64: return launch_group_cfg<T128x64<WB, OB>, ASYM>(p, g, s);
    default: return launch_group_cfg<T128x128<WB, OB>, ASYM>(p, g, s);
    }
}

template <int WB, int OB>
hipError_t launch_group_t(const QLinearArgs& p, const GroupArgs& g, hipStream_t s)
{
    return p.w_zp ? launch_group_a<WB, OB, true>(p, g, s)
                  : launch_group_a<WB, OB, false>(p, g, s);
}

}  // namespace

bool prefill_supported(const QLinearArgs& p)
{
    const int64_t ab = p.a_bits / 8, ob = p.out_bits / 8;
    const int64_t lda = eff_lda(p) * ab, ldy = eff_ldy(p) * ob;
    const int64_t ldw = p.w_bits == 8 ? eff_ldw(p) : (p.ldw ? p.ldw : p.K / 2);
    // whole 16-byte chunks per row (packed int4 rows too), 16-byte aligned
    // rows and batches; output rows and batches aligned to one store of four
    // channels (4 bytes of int8, 8 of int16), so every channel group of the
    // epilogue is one aligned store
    const int64_t og = 4 * ob;
    const bool kok = p.w_bits == 8 ? (p.K % 16 == 0) : (p.K % 32 == 0);
    const bool align = ((uintptr_t)p.a % 16) == 0 && ((uintptr_t)p.w % 16) == 0 &&
                       ((uintptr_t)p.y % og) == 0 && lda % 16 == 0 && ldw % 16 == 0 &&
                       ldy % og == 0 && (p.a_bs * ab) % 16 == 0 && p.w_bs % 16 == 0 &&
                       (p.y_bs * ob) % og == 0;
    // byte offsets inside one 256-row tile must fit the 32-bit buffer offset
    const int64_t lim = (int64_t)1 << 31;
    const bool nok = 256 * ldy < lim && 256 * lda < lim && 256 * ldw < lim &&
                     (!p.y_f || 256 * p.N * 4 < lim);
    // fp32 outputs: 16-byte stores of four channels
    const bool fok = !p.y_f || (((uintptr_t)p.y_f % 16) == 0 && p.N % 4 == 0);
    // 16-bit activation codes: int8 weights only (the W8A16 tile), which
    // also takes strides, batches and int64 row terms; the 8-bit tiles take
    // dense single products
    const bool dense = p.lda == 0 && p.ldw == 0 && p.ldy == 0 && p.batch == 1 &&
                       p.row_off == nullptr && p.ws_stride == 1;
    const bool aok = p.a_bits == 8 ? dense : (p.w_bits == 8 && p.w_zp == nullptr);
    return kok && align && nok && aok && fok && p.batch >= 1 && p.batch <= 65535;
}

int64_t prefill_workspace_bytes(const QLinearArgs& p)
{
    return workspace_for(p, choose(p, true));
}

int64_t prefill_counter_bytes(const QLinearArgs& p)
{
    const Choice ch = choose(p, true);
    if (ch.splits <= 1) return 0;
    const TileModel& t = kTiles[ch.tile];
    return split_counter_bytes(((p.M + t.tm - 1) / t.tm) * ((p.N + t.tn - 1) / t.tn));
}

// 16-bit activation codes: no K split; ASYM: int64 row terms
template <int>
hipError_t launch_a16(const QLinearArgs& p, hipStream_t s)
{
    const bool ro = p.row_off != nullptr, o8 = p.out_bits == 8;
    if (p.K <= T128x128A16S2<8>::A16_I32_MAX_K && p.bias == nullptr) {
        if (ro) return o8 ? launch_cfg<T128x128A16S2<8>, true>(p, 1, s)
                          : launch_cfg<T128x128A16S2<16>, true>(p, 1, s);
        return o8 ? launch_cfg<T128x128A16S2<8>, false>(p, 1, s)
                  : launch_cfg<T128x128A16S2<16>, false>(p, 1, s);
    }
    if (p.N <= 64) {
        if (ro) return o8 ? launch_cfg<T64x64A16<8>, true>(p, 1, s)
                          : launch_cfg<T64x64A16<16>, true>(p, 1, s);
        return o8 ? launch_cfg<T64x64A16<8>, false>(p, 1, s)
                  : launch_cfg<T64x64A16<16>, false>(p, 1, s);
    }
    if (ro) return o8 ? launch_cfg<T128x128A16<8>, true>(p, 1, s)
                      : launch_cfg<T128x128A16<16>, true>(p, 1, s);
    return o8 ? launch_cfg<T128x128A16<8>, false>(p, 1, s)
              : launch_cfg<T128x128A16<16>, false>(p, 1, s);
}

hipError_t launch_qlinear_prefill_group(const QLinearArgs& p, GroupArgs g, hipStream_t s)
{
    if (p.a_bits != 8 || g.n < 1 || g.n > kMaxGroup) return hipErrorInvalidValue;
    if (p.w_bits == 8 && p.out_bits == 8) return launch_group_t<8, 8>(p, g, s);
    if (p.w_bits == 8) return launch_group_t<8, 16>(p, g, s);
    if (p.out_bits == 8) return launch_group_t<4, 8>(p, g, s);
    return launch_group_t<4, 16>(p, g, s);
}

hipError_t launch_qlinear_prefill(const QLinearArgs& p, hipStream_t s)
{
    if (p.a_bits == 16) return launch_a16<8>(p, s);
    if (p.w_bits == 8 && p.out_bits == 8) return launch_t<8, 8>(p, s);
    if (p.w_bits == 8) return launch_t<8, 16>(p, s);
    if (p.out_bits == 8) return launch_t<4, 8>(p, s);
    return launch_t<4, 16>(p, s);
}

}  // namespace mq
