// MonarchAttention forward kernels for CDNA4 (gfx950).
//
// One kernel per half-step of the alternating maximisation (Sec. 3 of the
// paper, eqs. R_update / L_update with beta_r / beta_l), organised as in the
// paper's Implementation paragraph: the factors L and R live only in
// registers and LDS; between launches only the states alpha_R, c_R, alpha_L,
// c_L and Y cross global memory.
//
//   r_half_step<FIRST, FINAL>  one workgroup per (head, key block k):
//        S'[i][j] = Kbar[k][i] . alpha_R[k][j]                (beta_R, MFMA)
//        R[k][j][:] = softmax_i(s * S'[:, j] / c_R[k][j])      (eq. R_update)
//        c_L[j][k] = sum_i R log R,  alpha_L[j][k] = R Kbar[k] (eq. beta_l, MFMA)
//        FINAL: Y[j][k] = R Vbar[k]                            (eq. monarch_multiply)
//   l_half_step                one workgroup per (head, residue class j):
//        S'[k][l] = alpha_L[j][k] . Qbar[j][l]                 (beta_L, MFMA)
//        L[j][:][l] = softmax_k(s * S'[:, l] - c_L[j][:])      (eq. L_update)
//        c_R[k][j] = sum_l L,  alpha_R[k][j] = sum_l L Qbar[j][l]   (eq. beta_r, MFMA)
//   monarch_apply              one workgroup per (head, j): the last L half-step
//        fused with O[l*b + j] = sum_k L[j][k][l] Y[j][k]     (eq. monarch_multiply)
//
// The permutation P is never materialised: Qbar[j][l] is row l*b + j of Q, so
// the L half-step and the apply read (and the apply writes) rows at a stride of
// b rows, each row one contiguous d-element segment.
//
// MFMA use.  Every product is a 16x16 output tile of v_mfma_f32_16x16x{32,16}
// (bf16/fp16) or 16x16x4 (fp32) with fp32 accumulation.  Lane l of a wave owns
// output rows 4*(l/16)+q (q = 0..3) of column l%16.  Scores are formed
// transposed (softmax index along the rows of the MFMA tile), so each lane
// holds a whole column slice of one softmax row: the max and sum are an
// in-lane reduction plus two cross-lane steps.  The probabilities left in
// registers feed the second product directly as its B operand: for a chunk of
// 32 contraction indices made of two 16-wide score tiles, lane l's 8 operand
// slots are the 4 rows it holds of each tile.  The A operand of that product
// (a row-major LDS tile whose rows are the contraction index) is read with
// the gfx950 LDS transpose load ds_read_b64_tr_b16, which hands lane 16g + c
// the column c of rows 4g..4g+3 of a 16-row group, i.e. the same slot order.
#pragma once

#include <hip/hip_runtime.h>
#include <stdint.h>
#include <type_traits>

namespace ma {

typedef float f32x4 __attribute__((ext_vector_type(4)));
typedef __bf16 bf16x8 __attribute__((ext_vector_type(8)));
typedef __bf16 bf16x4 __attribute__((ext_vector_type(4)));
typedef _Float16 f16x8 __attribute__((ext_vector_type(8)));
typedef _Float16 f16x4 __attribute__((ext_vector_type(4)));
typedef short s16x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));
typedef s16x4 __attribute__((address_space(3))) lds_s16x4;

constexpr float kLog2e = 1.4426950408889634f;
constexpr float kLn2 = 0.6931471805599453f;
constexpr float kMasked = -1.0e30f;  // finite "minus infinity": exp2 gives 0 and 0 * kMasked stays 0
constexpr float kTiny = 1.17549435e-38f;

template <typename T> struct Mma;

template <> struct Mma<float> {
    static constexpr int KC = 4;   // contraction length of one instruction
    static constexpr int KPL = 1;  // contraction elements per lane
    using frag = float;
    __device__ static f32x4 mma(frag a, frag b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x4f32(a, b, c, 0, 0, 0);
    }
};

template <> struct Mma<__bf16> {
    static constexpr int KC = 32;
    static constexpr int KPL = 8;
    using frag = bf16x8;
    using frag4 = bf16x4;
    __device__ static f32x4 mma(frag a, frag b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x32_bf16(a, b, c, 0, 0, 0);
    }
    __device__ static f32x4 mma4(frag4 a, frag4 b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
    }
};

template <> struct Mma<_Float16> {
    static constexpr int KC = 32;
    static constexpr int KPL = 8;
    using frag = f16x8;
    using frag4 = f16x4;
    __device__ static f32x4 mma(frag a, frag b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x32_f16(a, b, c, 0, 0, 0);
    }
    __device__ static f32x4 mma4(frag4 a, frag4 b, f32x4 c)
    {
        return __builtin_amdgcn_mfma_f32_16x16x16f16(a, b, c, 0, 0, 0);
    }
};

// Row stride (elements) of a row-major LDS tile with C columns: pad by
// MA_LDS_PAD bytes (32 measured fastest of 0, 16 and 32 on the half-steps).
#ifndef MA_LDS_PAD
#define MA_LDS_PAD 32
#endif
template <typename T, int C> struct Ld {
    static constexpr int row = C + MA_LDS_PAD / (int)sizeof(T);
};

// gfx950's v_permlane16_swap / v_permlane32_swap applied to (x, x) return
// x[lane] and x[lane ^ 16] (resp. x[lane ^ 32]), in an order that depends on
// the lane: a VALU exchange with no LDS round trip.  The pair feeds
// commutative operations only, except in xor16_value.
template <int MASK> __device__ inline void xor_pair(uint32_t x, uint32_t &a, uint32_t &b)
{
    static_assert(MASK == 16 || MASK == 32, "lane distance 16 or 32");
    if constexpr (MASK == 16) {
        const auto r = __builtin_amdgcn_permlane16_swap(x, x, false, false);
        a = r[0];
        b = r[1];
    } else {
        const auto r = __builtin_amdgcn_permlane32_swap(x, x, false, false);
        a = r[0];
        b = r[1];
    }
}

// max(a, b) that propagates NaN (IEEE 754-2019 maximum): one v_maximum3_f32
// on gfx950, where fmaxf first canonicalises each operand with a v_max_f32
// of its own.  The scores are finite or NaN from arithmetic, so the two agree
// wherever neither is NaN, and a NaN reaches the row's maximum either way.
__device__ inline float max_nan(float a, float b) { return __builtin_elementwise_maximum(a, b); }

template <int MASK> __device__ inline float wave_xor_max(float x)
{
    uint32_t a, b;
    xor_pair<MASK>(__float_as_uint(x), a, b);
    return max_nan(__uint_as_float(a), __uint_as_float(b));
}

template <int MASK> __device__ inline float wave_xor_sum(float x)
{
    uint32_t a, b;
    xor_pair<MASK>(__float_as_uint(x), a, b);
    return __uint_as_float(a) + __uint_as_float(b);
}

// x[lane ^ 16]; odd_row = bit 4 of the lane.  The first result of
// permlane16_swap holds the partner in odd rows of 16 lanes, the second in
// even rows.
__device__ inline uint32_t xor16_value(uint32_t x, bool odd_row)
{
    uint32_t a, b;
    xor_pair<16>(x, a, b);
    return odd_row ? a : b;
}

template <typename T> __device__ inline T to_elem(float x) { return static_cast<T>(x); }

// Store 4 consecutive output elements.
template <typename T> __device__ inline void store4(T *dst, f32x4 v)
{
    if constexpr (std::is_same<T, float>::value) {
        *reinterpret_cast<f32x4 *>(dst) = v;
    } else {
        T e[4] = {to_elem<T>(v[0]), to_elem<T>(v[1]), to_elem<T>(v[2]), to_elem<T>(v[3])};
        u32x2 raw;
        __builtin_memcpy(&raw, e, 8);
        *reinterpret_cast<u32x2 *>(dst) = raw;
    }
}

// A [NR][D] tile split into 16-byte chunks over NTH threads (chunk idx =
// tid + h * NTH is row idx / CPR), fetched from global memory into registers
// and later staged into a row-major LDS tile.  Rows r >= `valid` are zero.
template <typename T, int NR, int D, int NTH> struct TileChunks {
    static constexpr int V = 16 / (int)sizeof(T), CPR = D / V, CH = NR * CPR / NTH;
    static_assert(NR * CPR % NTH == 0, "whole chunks per thread");
    u32x4 c[CH];

    // (columns >= dcols, a multiple of V, are zero as well)
    template <typename RowPtr> __device__ inline void fetch(RowPtr rowptr, int valid, int tid, int dcols = D)
    {
#pragma unroll
        for (int h = 0; h < CH; ++h) {
            const int idx = tid + h * NTH, r = idx / CPR, col = (idx % CPR) * V;
            c[h] = u32x4{0u, 0u, 0u, 0u};
            if (r < valid && col < dcols) c[h] = *reinterpret_cast<const u32x4 *>(rowptr(r) + col);
        }
    }

    template <int LDR> __device__ inline void stage(T *sRow, int tid) const
    {
#pragma unroll
        for (int h = 0; h < CH; ++h) {
            const int idx = tid + h * NTH, r = idx / CPR, col = (idx % CPR) * V;
            *reinterpret_cast<u32x4 *>(sRow + r * LDR + col) = c[h];
        }
    }

    // stage(), with rows >= valid written as zero whatever was fetched
    template <int LDR> __device__ inline void stage(T *sRow, int tid, int valid) const
    {
#pragma unroll
        for (int h = 0; h < CH; ++h) {
            const int idx = tid + h * NTH, r = idx / CPR, col = (idx % CPR) * V;
            *reinterpret_cast<u32x4 *>(sRow + r * LDR + col) = r < valid ? c[h] : u32x4{0u, 0u, 0u, 0u};
        }
    }
};

// Lane 16g + c receives X[x0 + 4g + q][c0 + c], q = 0..3, from the row-major
// LDS matrix X (row stride ld elements): the MFMA operand of a product that
// contracts over the rows of X, in the score tiles' slot order.
template <typename T>
__device__ inline typename Mma<T>::frag4 rows4(const T *X, int ld, int x0, int c0, int lane)
{
    const int g = lane >> 4, p = lane & 15;
    const T *src = X + (x0 + 4 * g + (p >> 2)) * ld + c0 + 4 * (p & 3);
    const s16x4 raw = __builtin_amdgcn_ds_read_tr16_b64_v4i16((lds_s16x4 *)(src));
    typename Mma<T>::frag4 out;
    __builtin_memcpy(&out, &raw, 8);
    return out;
}

// B-operand fragments of one 16-row block of a row-major [*, D] matrix:
// lane 16g + c holds row c's elements [KC*cc + KPL*g, +KPL) for every chunk cc.
template <typename T, int D> struct RowFrags {
    using M = Mma<T>;
    typename M::frag f[D / M::KC];
    // from global memory (row == nullptr: a zero row)
    // (columns >= dcols: zero; dcols is a multiple of KPL)
    __device__ inline void load(const T *row, int g, int dcols = D)
    {
#pragma unroll
        for (int c = 0; c < D / M::KC; ++c) {
            if (row && c * M::KC + g * M::KPL < dcols) {
                f[c] = *reinterpret_cast<const typename M::frag *>(row + c * M::KC + g * M::KPL);
            } else {
                f[c] = typename M::frag{};
            }
        }
    }

    // Zero the row when `drop` (a register select: no wait on anything else).
    __device__ inline void clear_if(bool drop)
    {
#pragma unroll
        for (int c = 0; c < D / M::KC; ++c) f[c] = drop ? typename M::frag{} : f[c];
    }
};

// acc = A[r0 + 0..15][0..D) * B-fragments^T : one 16x16 tile of a score product.
// sA_row points to row (r0 + lane%16) of the row-major LDS copy of A.
template <typename T, int D>
__device__ inline f32x4 gemm_scores(const T *sA_row, const RowFrags<T, D> &bf, int g)
{
    using M = Mma<T>;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < D / M::KC; ++c) {
        const typename M::frag a = *reinterpret_cast<const typename M::frag *>(sA_row + c * M::KC + g * M::KPL);
        acc = M::mma(a, bf.f[c], acc);
    }
    return acc;
}

// Operand fragments covering NT 16-wide tiles of a contraction index, in the
// tile-pair slot order: chunk c holds tiles 2c (slots 0..3) and 2c+1 (slots
// 4..7); an odd last tile is a 4-slot fragment.  fp32 keeps one value per
// (tile, slot) for the 16x16x4 instruction.
template <typename T, int NT, bool IS_F32 = std::is_same<T, float>::value> struct ProbFrags;

template <typename T, int NT> struct ProbFrags<T, NT, false> {
    using M = Mma<T>;
    static constexpr int NC = NT / 2;
    typename M::frag f[NC > 0 ? NC : 1];
    typename M::frag4 f4;
    // from score tiles in registers (lane holds 4 rows of each tile)
    __device__ inline void pack(const f32x4 *p)
    {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                f[c][q] = to_elem<T>(p[2 * c][q]);
                f[c][4 + q] = to_elem<T>(p[2 * c + 1][q]);
            }
        }
        if constexpr (NT % 2 == 1) {
#pragma unroll
            for (int q = 0; q < 4; ++q) f4[q] = to_elem<T>(p[NT - 1][q]);
        }
    }
    // from a row-major LDS matrix X whose rows are the contraction index
    __device__ inline void gather(const T *X, int ld, int c0, int lane)
    {
#pragma unroll
        for (int c = 0; c < NC; ++c) {
            const typename M::frag4 lo = rows4<T>(X, ld, 32 * c, c0, lane);
            const typename M::frag4 hi = rows4<T>(X, ld, 32 * c + 16, c0, lane);
            f[c] = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
        }
        if constexpr (NT % 2 == 1) f4 = rows4<T>(X, ld, 16 * (NT - 1), c0, lane);
    }
};

template <typename T, int NT> struct ProbFrags<T, NT, true> {
    f32x4 p[NT];
    __device__ inline void pack(const f32x4 *src)
    {
#pragma unroll
        for (int t = 0; t < NT; ++t) p[t] = src[t];
    }
    __device__ inline void gather(const float *X, int ld, int c0, int lane)
    {
        const int g = lane >> 4, c = lane & 15;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int q = 0; q < 4; ++q) p[t][q] = X[(16 * t + 4 * g + q) * ld + c0 + c];
        }
    }
};

// acc[r][col] = sum_x X[x][c0 + r] * B[x][col] over NT 16-wide tiles of x, for
// r = 0..15: one 16x16 tile of an aggregation product.  X is a row-major LDS
// matrix whose rows are the contraction index; B is given as fragments.
template <typename T, int NT>
__device__ inline f32x4 gemm_aggregate(const T *X, int ld, int c0, const ProbFrags<T, NT> &pf, int lane)
{
    using M = Mma<T>;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if constexpr (std::is_same<T, float>::value) {
        const int g = lane >> 4, c = lane & 15;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int q = 0; q < 4; ++q) acc = M::mma(X[(16 * t + 4 * g + q) * ld + c0 + c], pf.p[t][q], acc);
        }
    } else {
#pragma unroll
        for (int c = 0; c < NT / 2; ++c) {
            const typename M::frag4 lo = rows4<T>(X, ld, 32 * c, c0, lane);
            const typename M::frag4 hi = rows4<T>(X, ld, 32 * c + 16, c0, lane);
            acc = M::mma(__builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7), pf.f[c], acc);
        }
        if constexpr (NT % 2 == 1) acc = M::mma4(rows4<T>(X, ld, 16 * (NT - 1), c0, lane), pf.f4, acc);
    }
    return acc;
}

// acc[r][col] = sum_x B[x][col] for every r: the column sums of the operand
// given as fragments (an all-ones A operand).
template <typename T, int NT>
__device__ inline f32x4 gemm_colsum(const ProbFrags<T, NT> &pf)
{
    using M = Mma<T>;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if constexpr (std::is_same<T, float>::value) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int q = 0; q < 4; ++q) acc = M::mma(1.0f, pf.p[t][q], acc);
        }
    } else {
        typename M::frag ones;
        typename M::frag4 ones4;
#pragma unroll
        for (int q = 0; q < 8; ++q) ones[q] = to_elem<T>(1.0f);
#pragma unroll
        for (int q = 0; q < 4; ++q) ones4[q] = to_elem<T>(1.0f);
#pragma unroll
        for (int c = 0; c < NT / 2; ++c) acc = M::mma(ones, pf.f[c], acc);
        if constexpr (NT % 2 == 1) acc = M::mma4(ones4, pf.f4, acc);
    }
    return acc;
}

// Row tiles per wave and waves per workgroup for a block of NT 16-row tiles:
// two tiles per wave from 4 tiles up, so that every operand fragment read
// from LDS feeds two MFMAs.
#ifndef MA_ROW_TILES
#define MA_ROW_TILES 1
#endif
template <int NT> struct Split {
    static constexpr int RT = (NT >= 4 && MA_ROW_TILES >= 2) ? 2 : 1;
    static constexpr int W = NT / RT;
};

// acc[r] = A[r0 + 0..15][0..D) * bf[r]^T for RT row blocks sharing the A
// fragments (read once from LDS).  sA_row points to row (r0 + lane%16).
template <typename T, int D, int RT>
__device__ inline void gemm_scores_rt(const T *sA_row, const RowFrags<T, D> *bf, f32x4 *acc, int g)
{
    using M = Mma<T>;
#pragma unroll
    for (int r = 0; r < RT; ++r) acc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int c = 0; c < D / M::KC; ++c) {
        const typename M::frag a = *reinterpret_cast<const typename M::frag *>(sA_row + c * M::KC + g * M::KPL);
#pragma unroll
        for (int r = 0; r < RT; ++r) acc[r] = M::mma(a, bf[r].f[c], acc[r]);
    }
}

// acc[r][row][col] = sum_x X[x][c0 + row] * B_r[x][col] for RT operands B_r
// given as fragments, sharing the A fragments read from LDS.
template <typename T, int NT, int RT>
__device__ inline void gemm_aggregate_rt(const T *X, int ld, int c0, const ProbFrags<T, NT> *pf, f32x4 *acc,
                                         int lane)
{
    using M = Mma<T>;
#pragma unroll
    for (int r = 0; r < RT; ++r) acc[r] = f32x4{0.f, 0.f, 0.f, 0.f};
    if constexpr (std::is_same<T, float>::value) {
        const int g = lane >> 4, c = lane & 15;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float a = X[(16 * t + 4 * g + q) * ld + c0 + c];
#pragma unroll
                for (int r = 0; r < RT; ++r) acc[r] = M::mma(a, pf[r].p[t][q], acc[r]);
            }
        }
    } else {
#pragma unroll
        for (int c = 0; c < NT / 2; ++c) {
            const typename M::frag4 lo = rows4<T>(X, ld, 32 * c, c0, lane);
            const typename M::frag4 hi = rows4<T>(X, ld, 32 * c + 16, c0, lane);
            const typename M::frag a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
#pragma unroll
            for (int r = 0; r < RT; ++r) acc[r] = M::mma(a, pf[r].f[c], acc[r]);
        }
        if constexpr (NT % 2 == 1) {
            const typename M::frag4 a = rows4<T>(X, ld, 16 * (NT - 1), c0, lane);
#pragma unroll
            for (int r = 0; r < RT; ++r) acc[r] = M::mma4(a, pf[r].f4, acc[r]);
        }
    }
}

// Maximum over the softmax index of transposed score tiles (lane holds index
// 16t + 4g + q of row lane%16): in-lane, then across the four lane groups.
// With RAGGED, entries at index >= n are left out.
template <int NT, bool RAGGED>
__device__ inline float tiles_max(const f32x4 *z, int n, int g)
{
    float mx = kMasked;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int q = 0; q < 4; ++q)
            if (!RAGGED || 16 * t + 4 * g + q < n) mx = max_nan(mx, z[t][q]);
    }
    mx = wave_xor_max<16>(mx);
    return wave_xor_max<32>(mx);
}

// 1 / x with the hardware reciprocal (at most 1 ulp from the rounded quotient).
__device__ inline float fast_rcp(float x) { return __builtin_amdgcn_rcpf(x); }

// Whether a softmax is normalised before it feeds a product (4 NT multiplies
// per lane) rather than after it (D / 16 * 4): whichever is fewer.
template <int NT, int D> struct NormFirst {
    static constexpr bool value = 16 * NT < D;
};

__device__ inline float lanegroup_sum(float x)
{
    x = wave_xor_sum<16>(x);
    return wave_xor_sum<32>(x);
}

// Store the 16 x D output tile held as D/16 transposed MFMA tiles (lane holds
// elements 16vt + 4g + q of row lane%16) to the row `row` (nullptr: skip).
// Lanes 16g and 16(g^1) swap halves so that every lane writes 16-byte
// chunks: each row receives 64 contiguous bytes per store instruction.
// Columns >= dcols (a multiple of 16 bytes' worth of elements) are not written.
template <typename T, int D>
__device__ inline void store_row(T *row, const f32x4 *acc, float scale, int lane, int dcols = D)
{
    const int g = lane >> 4;
    if constexpr (std::is_same<T, float>::value) {
        if (row) {
#pragma unroll
            for (int vt = 0; vt < D / 16; ++vt)
                if (16 * vt + 4 * g < dcols) *reinterpret_cast<f32x4 *>(row + 16 * vt + 4 * g) = acc[vt] * scale;
        }
    } else {
        const bool odd = g & 1;
#pragma unroll
        for (int i = 0; i < D / 32; ++i) {
            u32x2 pk[2];
#pragma unroll
            for (int h = 0; h < 2; ++h) {
                T e[4];
#pragma unroll
                for (int q = 0; q < 4; ++q) e[q] = to_elem<T>(acc[2 * i + h][q] * scale);
                __builtin_memcpy(&pk[h], e, 8);
            }
            const u32x2 give = odd ? pk[0] : pk[1];
            u32x2 got;
            got[0] = xor16_value(give[0], odd);
            got[1] = xor16_value(give[1], odd);
            const u32x4 chunk = odd ? u32x4{got[0], got[1], pk[1][0], pk[1][1]}
                                    : u32x4{pk[0][0], pk[0][1], got[0], got[1]};
            const int col = 16 * (2 * i + (odd ? 1 : 0)) + 8 * (g >> 1);
            if (row && col < dcols) *reinterpret_cast<u32x4 *>(row + col) = chunk;
        }
    }
}

// The same 16 x D tile to a row of an LDS matrix: 8 bytes per lane and MFMA
// tile, no exchange between lanes (LDS has no coalescing to serve).
template <typename T, int D> __device__ inline void store_row_lds(T *row, const f32x4 *acc, int lane)
{
    if (!row) return;
    const int g = lane >> 4;
#pragma unroll
    for (int vt = 0; vt < D / 16; ++vt) store4<T>(row + 16 * vt + 4 * g, acc[vt]);
}

struct HeadDims {
    int m, b;          // blocks and block size
    int n;             // rows of q, k, v, out per head, (m - 1) * b < n <= m * b
    int d;             // head dimension of q, k, v, out and of the state rows (<= the tile width D)
    float s_log2e;     // log2(e) / sqrt(d)
    int64_t units;     // work units of a half-step launch (grid size)
    int t = 0, T = 0;  // step of this L half-step (1..T) and the step count, for the objective
    // Per-sequence lengths (batch padding): head bh has lens[bh / H] real
    // rows (clamped to 0..n), or n when lens is null.
    const int *lens = nullptr;
    int H = 1;
    // fp32 L half-step: store alpha_R and c_R of every (k, j) divided by the
    // largest weight L[j][k][l] over l (see LHalf).  Off in the gradient's
    // recompute, whose reverse sweep takes the unscaled states.
    int colnorm = 0;
    // Pre-padded sequences: the kernels run the post-padded problem of the
    // row-reversed tensors, i.e. their row x is row n - 1 - x in memory (for
    // q, k, v and out alike).  The relabelling x -> m b - 1 - x of the padded
    // positions sends block l to m - 1 - l and row j to b - 1 - j: it keeps
    // L^(0) = I and the R and L softmaxes (a permutation of the keys within a
    // block, and of the blocks), and turns padding at the front into padding
    // at the end (Appendix "Padding and Masking").
    int rev = 0;
};

// Row of q, k, v, out in memory for row x (< n) of the kernels' problem.
__device__ inline int64_t mrow(const HeadDims &hd, int64_t x) { return hd.rev ? (int64_t)hd.n - 1 - x : x; }

// Memory rows of the kernels' rows x0 + i*step (i = 0, 1, ...) are
// mrow_u<RV>(x0) + i * rstep<RV>(step): the reversal folds into the first row
// and the sign of the step, so a row address stays one multiply-add.  The
// half-step kernels compile their unit loop with RV = false for calls without
// pre-padding (no reversal at all) and RV = true for the rest.
template <bool RV> __device__ inline int64_t mrow_u(const HeadDims &hd, int64_t x)
{
    return RV ? mrow(hd, x) : x;
}
template <bool RV> __device__ inline int64_t rstep(const HeadDims &hd, int64_t step)
{
    return RV && hd.rev ? -step : step;
}

// The head dimension as the unit code sees it: the compile-time constant DK
// when DK != 0 (the kernels run their unit loop with DK = D when d == D, the
// usual case), else the run-time d.  The row strides of q, k, v, out and of
// the states, and the column bound of their loads and stores, then fold into
// constants where the tile is full.
template <int DK> __device__ inline auto head_dim(int d)
{
    if constexpr (DK != 0)
        return std::integral_constant<int, DK>{};
    else
        return d;
}

// Real rows of head bh.  The kernels read it in fetch() but use it only from
// stage() on: their tile loads take the static bound n, so that they never
// wait for this load, and the rows beyond it are zeroed on their way to LDS.
__device__ inline int live_rows(const HeadDims &hd, int64_t bh)
{
    if (!hd.lens) return hd.n;
    const int len = hd.lens[(int)bh / hd.H];  // bh < 2^31: the grids are checked on the host
    return len < 0 ? 0 : len > hd.n ? hd.n : len;
}

// Real keys of block k of a head with nl real rows: b, fewer in a partly
// padded block, none (<= 0) in a block of padding only.
__device__ inline int block_keys(int b, int nl, int k) { return min(b, nl - k * b); }

// Key blocks holding at least one real key, ceil(nl / b) (m unless the head
// is batch-padded).
__device__ inline int live_blocks(int m, int b, int nl) { return min(m, (nl + b - 1) / b); }

// Tensors and states of one call.  When n < m * b the sequence is taken as
// post-padded with zero rows to N = m * b (Appendix "Padding and Masking"):
// rows >= n of q, k, v are never read (zero is loaded instead), keys >= n are
// masked out of every R softmax, rows >= n of out are never written, and the
// states cover all N rows.  With per-sequence lengths (HeadDims::lens) the
// real rows nl <= n of each head play the part of n: rows nl..n-1 of q, k, v
// may be loaded but are replaced by zero, whole key blocks can be padding
// (such a block gets R = 0, i.e. zero alpha_L, c_L, Y, and no weight in the
// L softmax, Z_L = -inf), and rows nl..n-1 of out are written as zero.
// Layouts (per head):
//   q, k, v, out [B*H][n][d], d <= D (columns d..D-1 of every tile are zero);
//   alpha_R [m][b][d] (row k*b + j), alpha_L and Y [b][m][d] (row j*m + k),
//   c_L [m][b] (written by the R half-step of block k for all j),
//   c_R [b][m] (written by the L half-step of class j for all k).
template <typename T> struct Bufs {
    const T *q, *k, *v;
    T *out;
    T *aR, *aL, *Y;
    float *cR, *cL;
    // Objective shares [B*H][T][b] (nullptr: not requested): after the L update
    // of step t, the sum over the query rows of class j of the logsumexp of the
    // L-update logits (natural units).  Their sum over j is f(M^(t); Q, K).
    float *obj_part = nullptr;
};

// Sum over the 16 rows of a wave (lanes 16g + c, c = 0..15, the four lane
// groups holding the same values): xor steps 8, 4, 2, 1; every lane ends with
// the sum, always in this order.
__device__ inline float rows16_sum(float x)
{
    x += __shfl_xor(x, 8);
    x += __shfl_xor(x, 4);
    x += __shfl_xor(x, 2);
    return x + __shfl_xor(x, 1);
}

// logsumexp (natural units) of a row held as log2-domain logits with maximum
// mx and sum of exp2(logit - mx) = sum.
__device__ inline float row_lse(float mx, float sum) { return kLn2 * (mx + __builtin_amdgcn_logf(sum)); }

// The work of one unit of each half-step, done by a workgroup of W waves in
// three parts: fetch() issues its global loads into registers, stage() moves
// the tiles into LDS, and compute() (after a barrier) does the rest.  RAGGED:
// the softmax index range (b for R, m for L) is shorter than the padded tile.

// ---------------------------------------------------------------------------------------
// R half-step for (head bh, key block k); each wave owns RT tiles of 16 rows j.
// NB = b rounded up to 16.  FIRST: alpha_R = the rows of Q (L^(0) = I) and
// c_R = 1.  FINAL: also Y.
// ---------------------------------------------------------------------------------------
template <typename T, int NB, int D, bool FIRST, bool FINAL, bool RAGGED, bool LENS = false> struct RHalf {
    static_assert(!LENS || RAGGED, "per-sequence lengths need the masked softmax");
    static constexpr int NT = NB / 16, RT = Split<NT>::RT, W = Split<NT>::W, NTH = 64 * W;
    static constexpr bool NF = NormFirst<NT, D>::value;
    static constexpr int LDK = Ld<T, D>::row;
    static constexpr int LDS_BYTES = (FINAL ? 2 : 1) * NB * LDK * (int)sizeof(T);

    // What a unit reads from global memory, held in registers until staged.
    struct Regs {
        TileChunks<T, NB, D, NTH> kt, vt;  // Kbar[k]; Vbar[k] (FINAL)
        RowFrags<T, D> bf[RT];             // rows j of alpha_R[k] (of Q when FIRST)
        float cr[RT];                      // c_R[k][j] (not FIRST)
        int nl, row0;                      // real rows of the head, first key row k*b (LENS)
    };

    template <int DK, bool RV>
    __device__ static void fetch(const Bufs<T> &p, const HeadDims &hd, int64_t bh, int k, int tid, Regs &gr)
    {
        if constexpr (LENS) {
            gr.nl = live_rows(hd, bh);
            gr.row0 = k * hd.b;
        }
        const int m = hd.m, b = hd.b, kv = block_keys(b, hd.n, k);  // rows in memory
        const auto dd = head_dim<DK>(hd.d);
        const int64_t N = (int64_t)m * b, hoff = bh * N * dd, toff = bh * (int64_t)hd.n * dd;  // states: rows of d
        const int lane = tid & 63, wave = tid >> 6;
        const int64_t r0 = (int64_t)k * b, first = mrow_u<RV>(hd, r0), step = rstep<RV>(hd, 1);
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            const int j = (wave * RT + r) * 16 + (lane & 15);
            const T *row = nullptr;  // alpha_R[k][j]; at t = 1 Q row k*b + j (zero if padding)
            if constexpr (FIRST) {
                if (j < kv) row = p.q + toff + (first + j * step) * dd;
            } else {
                if (j < b) row = p.aR + hoff + (r0 + j) * dd;
            }
            gr.bf[r].load(row, lane >> 4, dd);
            gr.cr[r] = 1.0f;
            if constexpr (!FIRST) {
                if (j < b) gr.cr[r] = p.cR[bh * N + (int64_t)j * m + k];
            }
        }
        // K and V after the alpha_R rows, V last: the scores wait for the rows
        // and K only, and V is staged just before the product that needs it
        const int64_t sd = step * dd;
        const T *kb = p.k + toff + first * dd;
        gr.kt.fetch([=](int r) { return kb + r * sd; }, kv, tid, dd);
        if constexpr (FINAL) {
            const T *vb = p.v + toff + first * dd;
            gr.vt.fetch([=](int r) { return vb + r * sd; }, kv, tid, dd);
        }
    }

    __device__ static void stage(const HeadDims &, const Regs &gr, char *lds, int tid)
    {
        T *Ks = reinterpret_cast<T *>(lds);
        if constexpr (LENS) {  // keys >= nl: zero (they are masked, zero keeps them finite)
            const int kv = gr.nl - gr.row0;
            gr.kt.template stage<LDK>(Ks, tid, kv);
        } else {
            gr.kt.template stage<LDK>(Ks, tid);
        }
    }

    // After stage() and a barrier.
    template <int DK, bool RV>
    __device__ static void compute(const Bufs<T> &p, const HeadDims &hd, int64_t bh, int k, const Regs &gr,
                                   char *lds, int tid)
    {
        T *Ks = reinterpret_cast<T *>(lds);
        T *Vs = Ks + NB * LDK;
        // keys >= kv: padding, masked (omega); kv <= 0: padding only, R = 0
        const int m = hd.m, b = hd.b, kv = block_keys(b, LENS ? gr.nl : hd.n, k);
        const int64_t N = (int64_t)m * b;
        const int lane = tid & 63, wave = tid >> 6;
        const int g = lane >> 4, c16 = lane & 15;
        int jr[RT];
        float rscale[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            jr[r] = (wave * RT + r) * 16 + c16;
            rscale[r] = (FIRST || jr[r] >= b) ? hd.s_log2e : hd.s_log2e * fast_rcp(fmaxf(gr.cr[r], kTiny));
        }

        RowFrags<T, D> bfq[RT];  // at t = 1 with per-sequence lengths: Q rows beyond the length zeroed
        if constexpr (FIRST && LENS) {
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                bfq[r] = gr.bf[r];
                bfq[r].clear_if(jr[r] >= kv);
            }
        }
        const RowFrags<T, D> *bf = (FIRST && LENS) ? bfq : gr.bf;
        f32x4 sc[RT][NT];  // lane holds S'[i = 16t + 4g + qq][j] of row tile r
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            f32x4 acc[RT];
            gemm_scores_rt<T, D, RT>(Ks + (16 * t + c16) * LDK, bf, acc, g);
#pragma unroll
            for (int r = 0; r < RT; ++r) sc[r][t] = acc[r];
        }
        ProbFrags<T, NT> pf[RT];
        float inv[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            // Z = s S / c_R in log2 units: u = Z - max Z = S * rs - max S * rs  (rs > 0)
            const float rs = rscale[r];
            const float nb = -tiles_max<NT, RAGGED>(sc[r], kv, g) * rs;
            float sum = 0.f, t2 = 0.f;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) {
                    const float u = __builtin_fmaf(sc[r][t][qq], rs, nb);
                    float e = __builtin_amdgcn_exp2f(u);
                    if (RAGGED && 16 * t + 4 * g + qq >= kv) e = 0.f;
                    const bool first = t == 0 && qq == 0;  // the sums start at their first term
                    sum = first ? e : sum + e;
                    t2 = first ? e * u : __builtin_fmaf(e, u, t2);
                    sc[r][t][qq] = e;
                }
            }
            sum = lanegroup_sum(sum);
            t2 = lanegroup_sum(t2);
            const bool live = !LENS || kv > 0;
            inv[r] = live ? fast_rcp(sum) : 0.f;
            // c_L = sum_i R log R = sum_i R (Z - max) - log(sum)   (natural-log units)
            if (g == 0 && jr[r] < b)
                p.cL[bh * N + (int64_t)k * b + jr[r]] =
                    live ? kLn2 * (t2 * inv[r] - __builtin_amdgcn_logf(sum)) : 0.f;
            if constexpr (NF) {
#pragma unroll
                for (int t = 0; t < NT; ++t) sc[r][t] *= inv[r];
                inv[r] = 1.0f;
            }
            pf[r].pack(sc[r]);  // !NF: unnormalised exp2 values, the row sum is divided out below
        }
        f32x4 out[RT][D / 16];
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) {
            f32x4 acc[RT];
            gemm_aggregate_rt<T, NT, RT>(Ks, LDK, 16 * vt, pf, acc, lane);
#pragma unroll
            for (int r = 0; r < RT; ++r) out[r][vt] = acc[r];
        }
        const auto dd = head_dim<DK>(hd.d);  // states: rows of d elements
#pragma unroll
        for (int r = 0; r < RT; ++r)  // alpha_L[j][k] (j-major)
            store_row<T, D>(jr[r] < b ? p.aL + bh * N * dd + ((int64_t)jr[r] * m + k) * dd : nullptr, out[r],
                            inv[r], lane, dd);
        if constexpr (FINAL) {
            // Vbar[k], staged here rather than with K: when a workgroup runs a
            // single unit, the scores and softmax overlap V's loads
            if constexpr (LENS)
                gr.vt.template stage<LDK>(Vs, tid, gr.nl - gr.row0);
            else
                gr.vt.template stage<LDK>(Vs, tid);
            __syncthreads();
#pragma unroll
            for (int vt = 0; vt < D / 16; ++vt) {
                f32x4 acc[RT];
                gemm_aggregate_rt<T, NT, RT>(Vs, LDK, 16 * vt, pf, acc, lane);
#pragma unroll
                for (int r = 0; r < RT; ++r) out[r][vt] = acc[r];
            }
#pragma unroll
            for (int r = 0; r < RT; ++r)
                store_row<T, D>(jr[r] < b ? p.Y + bh * N * dd + ((int64_t)jr[r] * m + k) * dd : nullptr, out[r],
                                inv[r], lane, dd);
        }
    }
};

// ---------------------------------------------------------------------------------------
// L half-step (not the last) for (head bh, residue class j).  NM = m rounded
// up to 16.  Wave w first owns RT tiles of 16 query rows l (scores and the
// softmax over k), then, after the probabilities have gone through LDS, RT
// tiles of 16 key-block columns k (c_R and alpha_R).
// ---------------------------------------------------------------------------------------
template <typename T, int NM, int D, bool RAGGED, bool LENS = false> struct LHalf {
    static_assert(!LENS || RAGGED, "per-sequence lengths need the masked softmax");
    static constexpr int NT = NM / 16, RT = Split<NT>::RT, W = Split<NT>::W, NTH = 64 * W;
    // P rows are padded by 8 elements, not the usual 32 bytes: with 16-bit
    // elements, the 16 rows that one P store instruction writes at one
    // column then fall on distinct LDS banks (at 128 rows the L half-step ran
    // 7% faster than with the 32-byte pad; pads of 4 and 24 measured the same).
    static constexpr int LDQ = Ld<T, D>::row, LDP = NM + 8;
    static constexpr int A_ELEMS = NM * LDQ, P_ELEMS = NM * LDP;
    static constexpr int AP_ELEMS = A_ELEMS > P_ELEMS ? A_ELEMS : P_ELEMS;
    static constexpr int LDS_BYTES = (NM * LDQ + AP_ELEMS) * (int)sizeof(T) + NM * 4 + W * 4;

    struct Regs {
        TileChunks<T, NM, D, NTH> qt, at;  // Qbar[j] (rows l), alpha_L[j] (rows k)
        float cl;                          // c_L[k = tid][j]
        int nl, j;                         // real rows of the head, the class (LENS)
    };

    template <int DK, bool RV>
    __device__ static void fetch(const Bufs<T> &p, const HeadDims &hd, int64_t bh, int j, int tid, Regs &gr)
    {
        const int m = hd.m, b = hd.b;
        const int64_t N = (int64_t)m * b;
        if constexpr (LENS) {
            gr.nl = live_rows(hd, bh);
            gr.j = j;
        }
        const int ml = (hd.n - j + b - 1) / b;  // rows l of class j in memory: l*b + j < n
        const auto dd = head_dim<DK>(hd.d);
        const int64_t hoff = bh * N * dd;  // states: rows of d elements
        const T *qb = p.q + bh * (int64_t)hd.n * dd + mrow_u<RV>(hd, j) * dd;  // Qbar[j][0]
        const int64_t sq = rstep<RV>(hd, b) * dd;                           // Qbar[j][l] -> Qbar[j][l + 1]
        const T *al = p.aL + hoff + (int64_t)j * m * dd;
        gr.qt.fetch([=](int l) { return qb + l * sq; }, ml, tid, dd);
        gr.at.fetch([=](int kk) { return al + (int64_t)kk * dd; }, m, tid, dd);
        gr.cl = tid < m ? p.cL[bh * N + (int64_t)tid * b + j] : 0.f;
    }

    __device__ static void stage(const HeadDims &hd, const Regs &gr, char *lds, int tid)
    {
        T *Qs = reinterpret_cast<T *>(lds);
        T *APs = Qs + NM * LDQ;
        if constexpr (LENS)  // real rows l of class j: l*b + j < nl
            gr.qt.template stage<LDQ>(Qs, tid, (gr.nl - gr.j + hd.b - 1) / hd.b);
        else
            gr.qt.template stage<LDQ>(Qs, tid);
        gr.at.template stage<LDQ>(APs, tid);
        if (tid < NM) reinterpret_cast<float *>(APs + AP_ELEMS)[tid] = gr.cl * kLog2e;
    }

    // After stage() and a barrier.
    template <int DK, bool RV>
    __device__ static void compute(const Bufs<T> &p, const HeadDims &hd, int64_t bh, int j, const Regs &gr,
                                   char *lds, int tid)
    {
        T *Qs = reinterpret_cast<T *>(lds);
        T *APs = Qs + NM * LDQ;  // alpha_L, then P
        float *cLs = reinterpret_cast<float *>(APs + AP_ELEMS);
        const int m = hd.m, b = hd.b;
        const int64_t N = (int64_t)m * b;
        const int lane = tid & 63, wave = tid >> 6;
        const int g = lane >> 4, c16 = lane & 15;
        const int mk = LENS ? live_blocks(m, b, gr.nl) : m;  // blocks k >= mk: no real key

        // scores and softmax over k for the query rows of this wave
        int lr[RT];
        float inv[RT], lse[RT];
        f32x4 sc[RT][NT];  // lane holds Z[k = 16t + 4g + qq][l] (log2 units) of row tile r
        RowFrags<T, D> bf[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            lr[r] = (wave * RT + r) * 16 + c16;
#pragma unroll
            for (int c = 0; c < D / Mma<T>::KC; ++c)
                bf[r].f[c] = *reinterpret_cast<const typename Mma<T>::frag *>(Qs + lr[r] * LDQ + c * Mma<T>::KC +
                                                                              g * Mma<T>::KPL);
        }
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            f32x4 acc[RT];
            gemm_scores_rt<T, D, RT>(APs + (16 * t + c16) * LDQ, bf, acc, g);
            const f32x4 bias = *reinterpret_cast<const f32x4 *>(cLs + 16 * t + 4 * g);
#pragma unroll
            for (int r = 0; r < RT; ++r) {
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) sc[r][t][qq] = __builtin_fmaf(acc[r][qq], hd.s_log2e, -bias[qq]);
            }
        }
        // fp32 with colnorm: the logits are kept, and P holds log2 L (below)
        constexpr bool F32 = std::is_same<T, float>::value;
        const bool logp = F32 && hd.colnorm;
        f32x4 zk[F32 ? RT : 1][F32 ? NT : 1];
        float lz[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            if constexpr (F32) {
#pragma unroll
                for (int t = 0; t < NT; ++t) zk[r][t] = sc[r][t];
            }
            const float mx = tiles_max<NT, RAGGED>(sc[r], mk, g);
            float sum = 0.f;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) {
                    float e = __builtin_amdgcn_exp2f(sc[r][t][qq] - mx);
                    if (RAGGED && 16 * t + 4 * g + qq >= mk) e = 0.f;
                    sum = (t == 0 && qq == 0) ? e : sum + e;
                    sc[r][t][qq] = e;
                }
            }
            sum = lanegroup_sum(sum);
            // tile rows l >= m carry no weight, nor does a head without a real key
            const bool live = lr[r] < m && (!LENS || mk > 0);
            inv[r] = live ? fast_rcp(sum) : 0.f;
            lse[r] = live ? row_lse(mx, sum) : 0.f;
            lz[r] = 0.f;  // log2 of the row normaliser (fp32)
            if constexpr (F32) lz[r] = live ? mx + __builtin_amdgcn_logf(sum) : 0.f;
        }
        float *objs = cLs + NM;  // one objective share per wave
        if (p.obj_part) {
            float part = 0.f;
#pragma unroll
            for (int r = 0; r < RT; ++r) part += lse[r];
            part = rows16_sum(part);
            if (lane == 0) objs[wave] = part;
        }
        __syncthreads();  // every wave is done reading alpha_L
        if (p.obj_part && tid == 0) {
            float f = 0.f;
            for (int w = 0; w < W; ++w) f += objs[w];
            p.obj_part[(bh * hd.T + hd.t - 1) * b + j] = f;
        }

        // P[l][k] (row-major, k contiguous) into the alpha_L space: L[j][k][l],
        // or with logp its log2 (kMasked where L is zero)
        using PT = typename std::conditional<std::is_same<T, float>::value, float, T>::type;
        PT *Ps = reinterpret_cast<PT *>(APs);
#pragma unroll
        for (int r = 0; r < RT; ++r) {
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                if constexpr (F32) {
                    if (logp) {
                        f32x4 y;
#pragma unroll
                        for (int qq = 0; qq < 4; ++qq) {
                            const bool on = inv[r] != 0.f && (!RAGGED || 16 * t + 4 * g + qq < mk);
                            y[qq] = on ? zk[r][t][qq] - lz[r] : kMasked;
                        }
                        store4<PT>(Ps + lr[r] * LDP + 16 * t + 4 * g, y);
                        continue;
                    }
                }
                store4<PT>(Ps + lr[r] * LDP + 16 * t + 4 * g, sc[r][t] * inv[r]);
            }
        }
        __syncthreads();

        // wave w: key-block columns k in tiles wave*RT + r
        int kr[RT];
        ProbFrags<T, NT> pf[RT];  // B operand: P[l-slots][k]
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            kr[r] = (wave * RT + r) * 16 + c16;
            pf[r].gather(Ps, LDP, (wave * RT + r) * 16, lane);
            if constexpr (F32) {
                // Column k of L divided by its largest entry: w[l] = 2^(log2 L[j][k][l] - max_l log2 L),
                // so c_R and alpha_R are the eq. beta_r sums times one positive factor per (k, j),
                // which eq. R_update (beta_R / c_R) does not see.  The largest weight is 1, so a
                // column whose weights all lie far below 1 keeps them instead of underflowing.
                if (logp) {
                    float mxc = kMasked;
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
#pragma unroll
                        for (int qq = 0; qq < 4; ++qq) mxc = max_nan(mxc, pf[r].p[t][qq]);
                    }
                    mxc = wave_xor_max<32>(wave_xor_max<16>(mxc));
                    const bool any = mxc > 0.5f * kMasked;
#pragma unroll
                    for (int t = 0; t < NT; ++t) {
#pragma unroll
                        for (int qq = 0; qq < 4; ++qq)
                            pf[r].p[t][qq] = any ? __builtin_amdgcn_exp2f(pf[r].p[t][qq] - mxc) : 0.f;
                    }
                }
            }
            const f32x4 cs = gemm_colsum<T, NT>(pf[r]);  // c_R[k][j] = sum_l L[j][k][l] (times the factor)
            if (g == 0 && kr[r] < m) p.cR[bh * N + (int64_t)j * m + kr[r]] = cs[0];
        }
        f32x4 out[RT][D / 16];
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) {
            f32x4 acc[RT];
            gemm_aggregate_rt<T, NT, RT>(Qs, LDQ, 16 * vt, pf, acc, lane);
#pragma unroll
            for (int r = 0; r < RT; ++r) out[r][vt] = acc[r];
        }
        const auto dd = head_dim<DK>(hd.d);  // states: rows of d elements
#pragma unroll
        for (int r = 0; r < RT; ++r)  // alpha_R[k][j] (k-major)
            store_row<T, D>(kr[r] < m ? p.aR + bh * N * dd + ((int64_t)kr[r] * b + j) * dd : nullptr, out[r],
                            1.0f, lane, dd);
    }
};

// ---------------------------------------------------------------------------------------
// Last L half-step fused with the second Monarch product and the store of O
// for (head bh, class j); each wave owns RT tiles of 16 query rows l.
// ---------------------------------------------------------------------------------------
template <typename T, int NM, int D, bool RAGGED, bool LENS = false> struct Apply {
    static_assert(!LENS || RAGGED, "per-sequence lengths need the masked softmax");
    static constexpr int NT = NM / 16, RT = Split<NT>::RT, W = Split<NT>::W, NTH = 64 * W;
    static constexpr bool NF = NormFirst<NT, D>::value;
    static constexpr int LDK = Ld<T, D>::row;
    static constexpr int LDS_BYTES = 2 * NM * LDK * (int)sizeof(T) + NM * 4 + W * 4;

    struct Regs {
        TileChunks<T, NM, D, NTH> at, yt;  // alpha_L[j], Y[j] (rows k)
        float cl;                          // c_L[k = tid][j]
        RowFrags<T, D> bf[RT];             // Qbar[j] rows l
        int nl;                            // real rows of the head (LENS)
    };

    template <int DK, bool RV>
    __device__ static void fetch(const Bufs<T> &p, const HeadDims &hd, int64_t bh, int j, int tid, Regs &gr)
    {
        const int m = hd.m, b = hd.b;
        const int64_t N = (int64_t)m * b;
        const int lane = tid & 63, wave = tid >> 6;
        const auto dd = head_dim<DK>(hd.d);
        const int64_t hoff = bh * N * dd;  // states: rows of d elements
        const T *al = p.aL + hoff + (int64_t)j * m * dd;
        const T *yj = p.Y + hoff + (int64_t)j * m * dd;
        gr.at.fetch([=](int kk) { return al + (int64_t)kk * dd; }, m, tid, dd);
        gr.yt.fetch([=](int kk) { return yj + (int64_t)kk * dd; }, m, tid, dd);
        const T *qb = p.q + bh * (int64_t)hd.n * dd + mrow_u<RV>(hd, j) * dd;  // Qbar[j][0]
        const int64_t sq = rstep<RV>(hd, b) * dd;
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            const int l = (wave * RT + r) * 16 + (lane & 15);
            gr.bf[r].load((int64_t)l * b + j < hd.n ? qb + l * sq : nullptr, lane >> 4, dd);  // Qbar[j][l]; zero if padded
        }
        gr.cl = tid < m ? p.cL[bh * N + (int64_t)tid * b + j] : 0.f;
        if constexpr (LENS) gr.nl = live_rows(hd, bh);
    }

    __device__ static void stage(const HeadDims &, const Regs &gr, char *lds, int tid)
    {
        T *As = reinterpret_cast<T *>(lds);
        T *Ys = As + NM * LDK;
        gr.at.template stage<LDK>(As, tid);
        gr.yt.template stage<LDK>(Ys, tid);
        if (tid < NM) reinterpret_cast<float *>(Ys + NM * LDK)[tid] = gr.cl * kLog2e;
    }

    // After stage() and a barrier.
    template <int DK, bool RV>
    __device__ static void compute(const Bufs<T> &p, const HeadDims &hd, int64_t bh, int j, const Regs &gr,
                                   char *lds, int tid)
    {
        T *As = reinterpret_cast<T *>(lds);
        T *Ys = As + NM * LDK;
        float *cLs = reinterpret_cast<float *>(Ys + NM * LDK);
        const int m = hd.m, b = hd.b;
        const int lane = tid & 63, wave = tid >> 6;
        const int g = lane >> 4, c16 = lane & 15;
        const int nl = LENS ? gr.nl : hd.n;
        const int mk = LENS ? live_blocks(m, b, nl) : m;  // blocks k >= mk: no real key
        int lr[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) lr[r] = (wave * RT + r) * 16 + c16;
        RowFrags<T, D> bfq[RT];  // with per-sequence lengths: query rows beyond the length zeroed
        if constexpr (LENS) {
#pragma unroll
            for (int r = 0; r < RT; ++r) {
                bfq[r] = gr.bf[r];
                bfq[r].clear_if((int64_t)lr[r] * b + j >= nl);
            }
        }
        const RowFrags<T, D> *bf = LENS ? bfq : gr.bf;

        f32x4 sc[RT][NT];  // lane holds Z[k = 16t + 4g + qq][l] (log2 units) of row tile r
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            f32x4 acc[RT];
            gemm_scores_rt<T, D, RT>(As + (16 * t + c16) * LDK, bf, acc, g);
            const f32x4 bias = *reinterpret_cast<const f32x4 *>(cLs + 16 * t + 4 * g);
#pragma unroll
            for (int r = 0; r < RT; ++r) {
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) sc[r][t][qq] = __builtin_fmaf(acc[r][qq], hd.s_log2e, -bias[qq]);
            }
        }
        ProbFrags<T, NT> pf[RT];
        float inv[RT], lse[RT];
#pragma unroll
        for (int r = 0; r < RT; ++r) {
            const float mx = tiles_max<NT, RAGGED>(sc[r], mk, g);
            float sum = 0.f;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) {
                    float e = __builtin_amdgcn_exp2f(sc[r][t][qq] - mx);
                    if (RAGGED && 16 * t + 4 * g + qq >= mk) e = 0.f;
                    sum = (t == 0 && qq == 0) ? e : sum + e;
                    sc[r][t][qq] = e;
                }
            }
            sum = lanegroup_sum(sum);
            const bool any = !LENS || mk > 0;  // a head without a real key has L = 0
            inv[r] = any ? fast_rcp(sum) : 0.f;
            lse[r] = (lr[r] < m && any) ? row_lse(mx, sum) : 0.f;
            if constexpr (NF) {
#pragma unroll
                for (int t = 0; t < NT; ++t) sc[r][t] *= inv[r];
                inv[r] = 1.0f;
            }
            pf[r].pack(sc[r]);  // !NF: unnormalised, the row sum is divided out of O below
        }
        if (p.obj_part) {  // objective share of class j at the last step (uniform branch)
            float *objs = cLs + NM;
            float part = 0.f;
#pragma unroll
            for (int r = 0; r < RT; ++r) part += lse[r];
            part = rows16_sum(part);
            if (lane == 0) objs[wave] = part;
            __syncthreads();
            if (tid == 0) {
                float f = 0.f;
                for (int w = 0; w < W; ++w) f += objs[w];
                p.obj_part[(bh * hd.T + hd.t - 1) * b + j] = f;
            }
        }
        f32x4 o[RT][D / 16];
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) {
            f32x4 acc[RT];
            gemm_aggregate_rt<T, NT, RT>(Ys, LDK, 16 * vt, pf, acc, lane);
#pragma unroll
            for (int r = 0; r < RT; ++r) o[r][vt] = acc[r];
        }
        const auto dd = head_dim<DK>(hd.d);
        T *ob = p.out + bh * (int64_t)hd.n * dd + mrow_u<RV>(hd, j) * dd;  // O[j], row 0 of class j
        const int64_t so = rstep<RV>(hd, b) * dd;
#pragma unroll
        for (int r = 0; r < RT; ++r) {  // rows nl..n-1 (batch padding) are written as zero
            const int64_t row = (int64_t)lr[r] * b + j;
            store_row<T, D>(row < hd.n ? ob + lr[r] * so : nullptr, o[r], (!LENS || row < nl) ? inv[r] : 0.f, lane,
                            dd);
        }
    }
};

// ---------------------------------------------------------------------------------------
// One launch per half-step.  The grid holds at most as many workgroups as
// are resident at once; workgroup i takes units i, i + gridDim.x, ... and
// issues the global loads of its next unit as soon as the current one is in
// LDS, so that they land while it computes.  `per` is the number of units
// per head (m for R, b for L).
// ---------------------------------------------------------------------------------------
template <typename U, int DK, bool RV, typename T>
__device__ inline void run_units_d(const Bufs<T> &p, const HeadDims &hd, int per, char *lds)
{
    const int tid = threadIdx.x;
    int64_t u = blockIdx.x;
    typename U::Regs cur, nxt;
    U::template fetch<DK, RV>(p, hd, u / per, (int)(u % per), tid, cur);
    while (true) {
        U::stage(hd, cur, lds, tid);
        __syncthreads();
        const int64_t un = u + gridDim.x;
        if (un < hd.units) U::template fetch<DK, RV>(p, hd, un / per, (int)(un % per), tid, nxt);
        U::template compute<DK, RV>(p, hd, u / per, (int)(u % per), cur, lds, tid);
        if (un >= hd.units) break;
        __syncthreads();  // LDS is restaged next
        cur = nxt;
        u = un;
    }
}

// The unit loop of the usual call (d fills the tile, no pre-padding), with
// the head dimension a constant and no row reversal, or of any other call
// (one uniform branch per workgroup; both loops are compiled into the kernel).
template <typename U, int D, typename T> __device__ inline void run_units(const Bufs<T> &p, const HeadDims &hd, int per, char *lds)
{
    if (hd.d == D && !hd.rev)
        run_units_d<U, D, false>(p, hd, per, lds);
    else
        run_units_d<U, 0, true>(p, hd, per, lds);
}

template <typename T, int NB, int D, bool FIRST, bool FINAL, bool RAGGED, bool LENS>
__global__ __launch_bounds__(64 * Split<NB / 16>::W) void r_half_step(Bufs<T> p, HeadDims hd)
{
    using U = RHalf<T, NB, D, FIRST, FINAL, RAGGED, LENS>;
    __shared__ __attribute__((aligned(16))) char lds[U::LDS_BYTES];
    run_units<U, D>(p, hd, hd.m, lds);
}

template <typename T, int NM, int D, bool RAGGED, bool LENS>
__global__ __launch_bounds__(64 * Split<NM / 16>::W) void l_half_step(Bufs<T> p, HeadDims hd)
{
    using U = LHalf<T, NM, D, RAGGED, LENS>;
    __shared__ __attribute__((aligned(16))) char lds[U::LDS_BYTES];
    run_units<U, D>(p, hd, hd.b, lds);
}

template <typename T, int NM, int D, bool RAGGED, bool LENS>
__global__ __launch_bounds__(64 * Split<NM / 16>::W) void monarch_apply(Bufs<T> p, HeadDims hd)
{
    using U = Apply<T, NM, D, RAGGED, LENS>;
    __shared__ __attribute__((aligned(16))) char lds[U::LDS_BYTES];
    run_units<U, D>(p, hd, hd.b, lds);
}

// ---------------------------------------------------------------------------------------
// Small heads (m, b <= 16, d = 64, 16-bit elements): the whole forward pass of
// one head in one workgroup of 16 waves (the fully fused one-head-per-block
// kernel for short sequences of Sec. 4, "Benchmarking"), with Q, K and every
// state resident in LDS, so that only Q, K, V and O cross global memory.  LDS regions, each 16
// blocks of 16 rows of LD elements, zero wherever there is no data:
//   Qs[j][l] = Qbar[j][l] = Q[l*b + j]
//   Ks[k][i] = Kbar[k][i] = K[k*b + i]; the last R half-step of block k
//              overwrites its own block with Y[k][j]
//   As[j][k] = alpha_L[j][k]; the L half-step of class j overwrites its own
//              block with its probabilities P[l][k] (rows l >= m zero)
//   Rs[k][j] = alpha_R[k][j]; the last R half-step of block k overwrites its
//              own block with Vbar[k]
// and c_R[k][j], c_L[j][k] in fp32.  In every half-step wave w does the unit
// w (block k or class j; one wave per unit at 16 rows): it overwrites only its
// own blocks, apart from the state it hands to the next half-step, and the
// half-steps are separated by workgroup barriers.  A wave's LDS accesses take
// effect in program order, so a unit may overwrite a block it has read.  The
// arithmetic of a unit is that of RHalf / LHalf / Apply at 16 rows.
// ---------------------------------------------------------------------------------------
template <typename T, bool RGB, bool RGM, bool LENS = false> struct FusedHead {
    static_assert(!LENS || (RGB && RGM), "per-sequence lengths need the masked softmaxes");
    static_assert(sizeof(T) == 2, "16-bit elements only");
    static constexpr int D = 64, NW = 16, LD = D + 8;  // 64 * NW threads (the launch bound below); rows + 16 bytes
    // Blocks are BS elements apart: 16 rows plus 16 bytes, so that the 16
    // lanes reading row r of 16 different blocks hit different LDS banks.
    static constexpr int BS = 16 * LD + 8;
    static constexpr int REGION = 16 * BS;  // elements
    static constexpr int CS = 17;  // row stride (floats) of c_R and c_L: writes along a column avoid bank conflicts
    static constexpr int LDS_BYTES = 4 * REGION * (int)sizeof(T) + 2 * 16 * CS * 4;

    struct Ctx {
        T *Qs, *Ks, *As, *Rs;
        float *cRs, *cLs;  // c_R[k][j] at k*CS + j, c_L[j][k] at j*CS + k
        int m, b, n, d, lane, g, c16;  // n: rows of a head in q, k, v, out; d <= D
        int rev;                       // pre-padded: row x in memory at n - 1 - x (HeadDims::rev)
        int nl, mk;        // with per-sequence lengths: real rows of the head being computed, live key blocks
        float s_log2e;
        int64_t bh;        // the head being computed
        int steps;         // T, the step count
        float *obj_part;   // objective shares [B*H][T][b], or nullptr
    };

    template <bool FIRST, bool FINAL>
    __device__ static void r_unit(const Ctx &c, int k, const u32x4 *vpre)
    {
        const int j = c.c16;
        const bool jv = j < c.b;
        RowFrags<T, D> bf;  // row j of alpha_R[k]; at t = 1 that is Q[k*b + j] = Qs[j][k]
        bf.load(FIRST ? c.Qs + j * BS + k * LD : c.Rs + k * BS + j * LD, c.g);
        float rs = c.s_log2e;
        if constexpr (!FIRST) {
            if (jv) rs = c.s_log2e * fast_rcp(fmaxf(c.cRs[k * CS + j], kTiny));
        }
        T *Kk = c.Ks + k * BS;
        const int kv = block_keys(c.b, LENS ? c.nl : c.n, k);  // keys >= kv: padding, masked (omega); none: R = 0
        f32x4 sc;  // lane holds S'[i = 4g + qq][j]
        gemm_scores_rt<T, D, 1>(Kk + c.c16 * LD, &bf, &sc, c.g);
        const float nb = -tiles_max<1, RGB>(&sc, kv, c.g) * rs;
        float sum = 0.f, t2 = 0.f;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const float u = __builtin_fmaf(sc[qq], rs, nb);
            float e = __builtin_amdgcn_exp2f(u);
            if (RGB && 4 * c.g + qq >= kv) e = 0.f;
            sum = qq == 0 ? e : sum + e;
            t2 = qq == 0 ? e * u : __builtin_fmaf(e, u, t2);
            sc[qq] = e;
        }
        sum = lanegroup_sum(sum);
        t2 = lanegroup_sum(t2);
        const bool live = !LENS || kv > 0;
        const float inv = live ? fast_rcp(sum) : 0.f;
        if (c.g == 0 && jv) c.cLs[j * CS + k] = live ? kLn2 * (t2 * inv - __builtin_amdgcn_logf(sum)) : 0.f;
        static_assert(NormFirst<1, D>::value, "probabilities normalised before the products, as in RHalf");
        sc *= inv;
        ProbFrags<T, 1> pf;
        pf.pack(&sc);
        f32x4 out[D / 16];
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) out[vt] = gemm_aggregate<T, 1>(Kk, LD, 16 * vt, pf, c.lane);
        store_row_lds<T, D>(jv ? c.As + j * BS + k * LD : nullptr, out, c.lane);  // alpha_L[j][k]
        if constexpr (FINAL) {
            T *Vk = c.Rs + k * BS;  // alpha_R[k] has been read: stage Vbar[k] in its place
#pragma unroll
            for (int h = 0; h < 2; ++h)
                *reinterpret_cast<u32x4 *>(Vk + ((c.lane >> 3) + 8 * h) * LD + (c.lane & 7) * 8) = vpre[h];
#pragma unroll
            for (int vt = 0; vt < D / 16; ++vt) out[vt] = gemm_aggregate<T, 1>(Vk, LD, 16 * vt, pf, c.lane);
            store_row_lds<T, D>(jv ? Kk + j * LD : nullptr, out, c.lane);  // Y[k][j] over Kbar[k]
        }
    }

    // Scores and softmax over k of class j, query row l = lane % 16 (lane
    // holds k = 4g + qq); returns exp2 values and sets inv = 1 / row sum and
    // lse = the row's logsumexp (natural units; 0 for tile rows l >= m).
    __device__ static f32x4 l_softmax(const Ctx &c, int j, float &inv, float &lse)
    {
        RowFrags<T, D> bf;
        bf.load(c.Qs + j * BS + c.c16 * LD, c.g);  // Qbar[j][l]
        f32x4 acc;
        gemm_scores_rt<T, D, 1>(c.As + j * BS + c.c16 * LD, &bf, &acc, c.g);
        f32x4 sc;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            // entries k >= m hold no c_L (their LDS words are never written);
            // the selects below leave them out of the maximum and the sum
            const float bias = c.cLs[j * CS + 4 * c.g + qq] * kLog2e;
            sc[qq] = __builtin_fmaf(acc[qq], c.s_log2e, -bias);
        }
        const int mk = LENS ? c.mk : c.m;  // blocks k >= mk: no real key
        const float mx = tiles_max<1, RGM>(&sc, mk, c.g);
        float sum = 0.f;
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            float e = __builtin_amdgcn_exp2f(sc[qq] - mx);
            if (RGM && 4 * c.g + qq >= mk) e = 0.f;
            sum = qq == 0 ? e : sum + e;
            sc[qq] = e;
        }
        sum = lanegroup_sum(sum);
        const bool any = !LENS || mk > 0;  // a head without a real key has L = 0
        inv = any ? fast_rcp(sum) : 0.f;
        lse = (c.c16 < c.m && any) ? row_lse(mx, sum) : 0.f;
        return sc;
    }

    // Objective share of class j after the L update of step t (as LHalf / Apply).
    __device__ static void objective_share(const Ctx &c, int j, int t, float lse)
    {
        if (!c.obj_part) return;
        const float part = rows16_sum(lse);
        if (c.lane == 0) c.obj_part[(c.bh * c.steps + t - 1) * c.b + j] = part;
    }

    __device__ static void l_unit(const Ctx &c, int j, int t)
    {
        const int l = c.c16;
        float inv, lse;
        const f32x4 e = l_softmax(c, j, inv, lse);
        objective_share(c, j, t, lse);
        T *Aj = c.As + j * BS;  // alpha_L[j] has been read: P[l][k] in its place
        const f32x4 pr = l < c.m ? e * inv : f32x4{0.f, 0.f, 0.f, 0.f};  // padded query rows carry no weight
        store4<T>(Aj + l * LD + 4 * c.g, pr);
        ProbFrags<T, 1> pf;  // B operand: P[l-slots][k = lane % 16]
        pf.gather(Aj, LD, 0, c.lane);
        const int k = c.c16;
        const f32x4 cs = gemm_colsum<T, 1>(pf);  // c_R[k][j] = sum_l L[j][k][l]
        if (c.g == 0 && k < c.m) c.cRs[k * CS + j] = cs[0];
        f32x4 out[D / 16];
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) out[vt] = gemm_aggregate<T, 1>(c.Qs + j * BS, LD, 16 * vt, pf, c.lane);
        store_row_lds<T, D>(k < c.m ? c.Rs + k * BS + j * LD : nullptr, out, c.lane);  // alpha_R[k][j]
    }

    __device__ static void apply_unit(const Ctx &c, int j, T *out_h)
    {
        const int l = c.c16;
        float inv, lse;
        const f32x4 e = l_softmax(c, j, inv, lse) * inv;  // normalised first, as in Apply at 16 rows
        objective_share(c, j, c.steps, lse);
        ProbFrags<T, 1> pf;
        pf.pack(&e);
        f32x4 o[D / 16];  // O[l*b + j] = sum_k L[j][k][l] Y[k][j]; Y[k][j] is row k of Ks + j*LD at stride BS
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) o[vt] = gemm_aggregate<T, 1>(c.Ks + j * LD, BS, 16 * vt, pf, c.lane);
        const int row = l * c.b + j;  // rows nl..n-1 (batch padding) are written as zero
        const int64_t mr = c.rev ? (int64_t)c.n - 1 - row : row;
        store_row<T, D>(row < c.n ? out_h + mr * c.d : nullptr, o, (!LENS || row < c.nl) ? 1.0f : 0.f,
                        c.lane, c.d);
    }

    static constexpr int PER = 2 * 256 * 8 / (64 * NW);  // 16-byte chunks of Qs and Ks per thread

    // Issue the loads of head bh: Qbar and Kbar chunks (zero where there is no
    // row) for the LDS regions, and Vbar[w] for wave w's last R half-step.
    // Rows >= n (padding) and columns >= d are zero and never read.
    __device__ static void load_head(const Bufs<T> &p, const HeadDims &hd, int64_t bh, int tid, u32x4 *raw, u32x4 *vb)
    {
        const int m = hd.m, b = hd.b, n = hd.n, d = hd.d;
        const int64_t hoff = bh * (int64_t)n * d;
        const T *qh = p.q + hoff, *kh = p.k + hoff, *vh = p.v + hoff;
        // Row x of the problem is memory row x0 + sx * x (mrow); offsets within
        // a head (at most 256 rows of 64 elements) are formed in 32 bits.
        const int x0 = hd.rev ? n - 1 : 0, sx = hd.rev ? -1 : 1;
#pragma unroll
        for (int h = 0; h < PER; ++h) {
            const int idx = tid + h * 64 * NW;
            const int reg = idx >> 11, blk = (idx >> 7) & 15, r = (idx >> 3) & 15, col = (idx & 7) * 8;
            raw[h] = u32x4{0u, 0u, 0u, 0u};
            if (reg == 0 && blk < b && r < m && r * b + blk < n && col < d)
                raw[h] = *reinterpret_cast<const u32x4 *>(qh + (x0 + sx * (r * b + blk)) * d + col);  // Qbar[blk][r]
            if (reg == 1 && blk < m && r < b && blk * b + r < n && col < d)
                raw[h] = *reinterpret_cast<const u32x4 *>(kh + (x0 + sx * (blk * b + r)) * d + col);  // Kbar[blk][r]
        }
        const int w = tid >> 6, lane = tid & 63;
#pragma unroll
        for (int h = 0; h < 2; ++h) {
            const int r = (lane >> 3) + 8 * h, col = (lane & 7) * 8;
            vb[h] = u32x4{0u, 0u, 0u, 0u};
            if (w < m && r < b && w * b + r < n && col < d)
                vb[h] = *reinterpret_cast<const u32x4 *>(vh + (x0 + sx * (w * b + r)) * d + col);
        }
    }

    // 16-byte chunk idx of two consecutive regions: region idx >> 11, block
    // (idx >> 7) & 15, row (idx >> 3) & 15.
    __device__ static u32x4 *chunk(T *base, int idx)
    {
        return reinterpret_cast<u32x4 *>(base + (idx >> 11) * REGION + ((idx >> 7) & 15) * BS + ((idx >> 3) & 15) * LD +
                                         (idx & 7) * 8);
    }

    // Heads blockIdx.x, blockIdx.x + gridDim.x, ... < BH.  The loads of the
    // next head are issued as soon as the current one is in LDS and land
    // while it is computed.  As and Rs are zeroed once: every head of a launch
    // leaves zero in their padding rows (see the units).
    __device__ static void run(const Bufs<T> &p, const HeadDims &hd, int64_t BH, int T_, char *lds)
    {
        Ctx c;
        c.Qs = reinterpret_cast<T *>(lds);
        c.Ks = c.Qs + REGION;
        c.As = c.Ks + REGION;
        c.Rs = c.As + REGION;
        c.cRs = reinterpret_cast<float *>(c.Rs + REGION);
        c.cLs = c.cRs + 16 * CS;
        c.m = hd.m;
        c.b = hd.b;
        c.n = hd.n;
        c.d = hd.d;
        c.rev = hd.rev;
        c.s_log2e = hd.s_log2e;
        c.steps = T_;
        c.obj_part = p.obj_part;
        const int tid = threadIdx.x, w = tid >> 6;
        c.lane = tid & 63;
        c.g = c.lane >> 4;
        c.c16 = c.lane & 15;
        const int m = hd.m, b = hd.b;

        u32x4 raw[PER], vcur[2], vnext[2];
        int64_t bh = blockIdx.x;
        load_head(p, hd, bh, tid, raw, vcur);
        for (int idx = tid; idx < 2 * 256 * 8; idx += 64 * NW) *chunk(c.As, idx) = u32x4{0u, 0u, 0u, 0u};
        for (; bh < BH; bh += gridDim.x) {
            c.bh = bh;
            if constexpr (LENS) {
                // the loads of this head were issued with the static bound n:
                // rows >= nl are zeroed here, on their way to LDS
                c.nl = live_rows(hd, bh);
                c.mk = live_blocks(m, b, c.nl);
#pragma unroll
                for (int h = 0; h < PER; ++h) {
                    const int idx = tid + h * 64 * NW, blk = (idx >> 7) & 15, r = (idx >> 3) & 15;
                    const int row = (idx >> 11) == 0 ? r * b + blk : blk * b + r;  // Qbar[blk][r] or Kbar[blk][r]
                    *chunk(c.Qs, idx) = row < c.nl ? raw[h] : u32x4{0u, 0u, 0u, 0u};
                }
#pragma unroll
                for (int h = 0; h < 2; ++h)
                    if (w * b + (c.lane >> 3) + 8 * h >= c.nl) vcur[h] = u32x4{0u, 0u, 0u, 0u};  // Vbar[w]
            } else {
#pragma unroll
                for (int h = 0; h < PER; ++h) *chunk(c.Qs, tid + h * 64 * NW) = raw[h];
            }
            __syncthreads();
            if (bh + gridDim.x < BH) load_head(p, hd, bh + gridDim.x, tid, raw, vnext);

            for (int t = 1; t <= T_; ++t) {
                const bool first = t == 1, last = t == T_;
                if (w < m) {
                    if (first && last)
                        r_unit<true, true>(c, w, vcur);
                    else if (first)
                        r_unit<true, false>(c, w, vcur);
                    else if (last)
                        r_unit<false, true>(c, w, vcur);
                    else
                        r_unit<false, false>(c, w, vcur);
                }
                __syncthreads();
                if (last) break;
                if (w < b) l_unit(c, w, t);
                __syncthreads();
            }
            if (w < b) apply_unit(c, w, p.out + bh * (int64_t)c.n * c.d);
            vcur[0] = vnext[0];
            vcur[1] = vnext[1];
            __syncthreads();  // the apply has read Qs, As and Ks
        }
    }
};

template <typename T, bool RGB, bool RGM, bool LENS>
__global__ __launch_bounds__(1024) void monarch_fused_head(Bufs<T> p, HeadDims hd, int64_t BH, int T_)
{
    using U = FusedHead<T, RGB, RGM, LENS>;
    __shared__ __attribute__((aligned(16))) char lds[U::LDS_BYTES];
    U::run(p, hd, BH, T_, lds);
}

// f(M^(t); Q, K) of every (head, step): the objective shares summed over the
// b classes, in class order.  One thread per (head, step).
static __global__ __launch_bounds__(256) void objective_sum(const float *part, float *obj, int64_t units, int b)
{
    const int64_t i = (int64_t)blockIdx.x * blockDim.x + threadIdx.x;
    if (i >= units) return;
    float f = 0.f;
    for (int j = 0; j < b; ++j) f += part[i * b + j];
    obj[i] = f;
}

// ---------------------------------------------------------------------------------------
// Exact softmax attention O = softmax(s Q K^T) V with the logsumexp of every
// row (eq. softmax_attention): the quality reference the Monarch output is
// measured against, and the upper bound of the objective (sum of the row
// logsumexps).  One workgroup of 4 waves per 64 query rows; wave w owns 16
// query rows (the B operand of the scores, in registers) and keeps an online
// softmax (running max, sum and output) over tiles of 64 keys.  Scores are
// transposed as in the half-steps (keys on the MFMA row axis), so the
// probabilities feed the V product straight from registers; the key and value
// tiles of the next step are fetched into registers while the current one is
// computed.
// ---------------------------------------------------------------------------------------
template <typename T, int D> struct ExactAttn {
    static constexpr int KT = 64, NT = KT / 16, W = 4, NTH = 64 * W;
    static constexpr int LDK = Ld<T, D>::row;
    static constexpr int LDS_BYTES = 2 * KT * LDK * (int)sizeof(T);

    struct Tiles {
        TileChunks<T, KT, D, NTH> kt, vt;
    };

    __device__ static void fetch(const T *kh, const T *vh, int n, int d, int key0, int tid, Tiles &g)
    {
        const int valid = n - key0 < KT ? n - key0 : KT;
        g.kt.fetch([=](int r) { return kh + (int64_t)(key0 + r) * d; }, valid, tid, d);
        g.vt.fetch([=](int r) { return vh + (int64_t)(key0 + r) * d; }, valid, tid, d);
    }

    __device__ static void run(const Bufs<T> &p, float *lse_out, int n, int d, float s_log2e, char *lds)
    {
        T *Ks = reinterpret_cast<T *>(lds);
        T *Vs = Ks + KT * LDK;
        const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6, g = lane >> 4, c16 = lane & 15;
        const int64_t qblocks = (n + 63) / 64;
        const int64_t bh = blockIdx.x / qblocks;
        const int row = (int)(blockIdx.x % qblocks) * 64 + wave * 16 + c16;  // this lane's query row
        const int64_t hoff = bh * (int64_t)n * d;
        const T *qh = p.q + hoff, *kh = p.k + hoff, *vh = p.v + hoff;

        RowFrags<T, D> bf;
        bf.load(row < n ? qh + (int64_t)row * d : nullptr, g, d);
        float mx = kMasked, sum = 0.f;  // running max (log2 units) and sum of this query row
        f32x4 o[D / 16];
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) o[vt] = f32x4{0.f, 0.f, 0.f, 0.f};

        Tiles cur, nxt;
        fetch(kh, vh, n, d, 0, tid, cur);
        for (int key0 = 0; key0 < n; key0 += KT) {
            cur.kt.template stage<LDK>(Ks, tid);
            cur.vt.template stage<LDK>(Vs, tid);
            __syncthreads();
            if (key0 + KT < n) fetch(kh, vh, n, d, key0 + KT, tid, nxt);
            const int kv = n - key0;  // keys >= kv of this tile are beyond N
            f32x4 sc[NT];             // lane holds u = s log2(e) q.k for keys 16t + 4g + qq
#pragma unroll
            for (int t = 0; t < NT; ++t) {
                f32x4 acc;
                gemm_scores_rt<T, D, 1>(Ks + (16 * t + c16) * LDK, &bf, &acc, g);
                sc[t] = acc * s_log2e;
            }
            const float tmax = tiles_max<NT, true>(sc, kv, g);
            const float mnew = max_nan(mx, tmax);
            const float corr = __builtin_amdgcn_exp2f(mx - mnew);
            float tsum = 0.f;
#pragma unroll
            for (int t = 0; t < NT; ++t) {
#pragma unroll
                for (int qq = 0; qq < 4; ++qq) {
                    float e = __builtin_amdgcn_exp2f(sc[t][qq] - mnew);
                    if (16 * t + 4 * g + qq >= kv) e = 0.f;
                    tsum += e;
                    sc[t][qq] = e;
                }
            }
            sum = sum * corr + lanegroup_sum(tsum);
            mx = mnew;
            ProbFrags<T, NT> pf;
            pf.pack(sc);
#pragma unroll
            for (int vt = 0; vt < D / 16; ++vt) o[vt] = o[vt] * corr + gemm_aggregate<T, NT>(Vs, LDK, 16 * vt, pf, lane);
            __syncthreads();  // the tiles are restaged next
            cur = nxt;
        }
        const float inv = fast_rcp(sum);
        store_row<T, D>(row < n ? p.out + hoff + (int64_t)row * d : nullptr, o, inv, lane, d);
        if (lse_out && g == 0 && row < n) lse_out[bh * n + row] = row_lse(mx, sum);
    }
};

template <typename T, int D>
__global__ __launch_bounds__(256) void exact_attention(Bufs<T> p, float *lse, int n, int d, float s_log2e)
{
    using U = ExactAttn<T, D>;
    __shared__ __attribute__((aligned(16))) char lds[U::LDS_BYTES];
    U::run(p, lse, n, d, s_log2e, lds);
}

}  // namespace ma
