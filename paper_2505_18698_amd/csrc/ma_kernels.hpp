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

// One wave per 16-row tile of the padded block (at most 8 waves).
template <int NT> struct Waves {
    static constexpr int value = NT < 8 ? NT : 8;
};

// Row stride (elements) of a row-major LDS tile with C columns: pad by 16 bytes.
template <typename T, int C> struct Ld {
    static constexpr int row = C + 16 / (int)sizeof(T);
};

__device__ inline float wave_xor_max(float x, int mask) { return fmaxf(x, __shfl_xor(x, mask)); }
__device__ inline float wave_xor_sum(float x, int mask) { return x + __shfl_xor(x, mask); }

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

// Cooperative load of a [NR][D] tile into row-major LDS (stride LDR); valid
// rows r < `valid` start at rowptr(r), the others are zero.
template <typename T, int NR, int D, int LDR, typename RowPtr>
__device__ inline void load_tile(RowPtr rowptr, int valid, T *sRow, int tid, int nthreads)
{
    constexpr int V = 16 / (int)sizeof(T);
    constexpr int CPR = D / V;
    for (int idx = tid; idx < NR * CPR; idx += nthreads) {
        const int r = idx / CPR, c = (idx % CPR) * V;
        u32x4 raw = {0u, 0u, 0u, 0u};
        if (r < valid) raw = *reinterpret_cast<const u32x4 *>(rowptr(r) + c);
        *reinterpret_cast<u32x4 *>(sRow + r * LDR + c) = raw;
    }
}

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
    __device__ inline void load(const T *row, int g)
    {
#pragma unroll
        for (int c = 0; c < D / M::KC; ++c) {
            if (row) {
                f[c] = *reinterpret_cast<const typename M::frag *>(row + c * M::KC + g * M::KPL);
            } else {
                f[c] = typename M::frag{};
            }
        }
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

// Row softmax of transposed score tiles: lane (c16, g) holds z for softmax
// index 16t + 4g + q of row c16.  Replaces z by exp2(z - max) and returns the
// row sum; also accumulates sum e*(z - max) into *t2 when t2 != nullptr.
template <int NT>
__device__ inline float softmax_cols(f32x4 *z, float *t2)
{
    float mx = kMasked;
#pragma unroll
    for (int t = 0; t < NT; ++t) mx = fmaxf(fmaxf(fmaxf(mx, z[t][0]), fmaxf(z[t][1], z[t][2])), z[t][3]);
    mx = wave_xor_max(mx, 16);
    mx = wave_xor_max(mx, 32);
    float sum = 0.f, acc2 = 0.f;
#pragma unroll
    for (int t = 0; t < NT; ++t) {
#pragma unroll
        for (int q = 0; q < 4; ++q) {
            const float u = z[t][q] - mx;
            const float e = __builtin_amdgcn_exp2f(u);
            sum += e;
            if (t2) acc2 += e * u;
            z[t][q] = e;
        }
    }
    sum = wave_xor_sum(sum, 16);
    sum = wave_xor_sum(sum, 32);
    if (t2) {
        acc2 = wave_xor_sum(acc2, 16);
        acc2 = wave_xor_sum(acc2, 32);
        *t2 = acc2;
    }
    return sum;
}

struct HeadDims {
    int m, b;          // blocks and block size, N = m * b
    float s_log2e;     // log2(e) / sqrt(d)
};

// ---------------------------------------------------------------------------------------
// R half-step: one workgroup per (head, key block k), one wave per 16 rows j.
// NB = b rounded up to 16.  FIRST: alpha_R = the rows of Q (L^(0) = I) and
// c_R = 1.  FINAL: also Y.
// ---------------------------------------------------------------------------------------
template <typename T, int NB, int D, bool FIRST, bool FINAL>
__global__ __launch_bounds__(64 * Waves<NB / 16>::value) void r_half_step(
    const T *__restrict__ q, const T *__restrict__ kmat, const T *__restrict__ vmat,
    const T *__restrict__ aR, const float *__restrict__ cR, T *__restrict__ aL,
    float *__restrict__ cL, T *__restrict__ Y, HeadDims hd)
{
    constexpr int NT = NB / 16, W = Waves<NT>::value;
    constexpr int LDK = Ld<T, D>::row;
    __shared__ __attribute__((aligned(16))) T Ks[NB * LDK];
    __shared__ __attribute__((aligned(16))) T Vs[FINAL ? NB * LDK : 8];

    const int m = hd.m, b = hd.b;
    const int64_t N = (int64_t)m * b;
    const int k = blockIdx.x % m;
    const int64_t bh = blockIdx.x / m;
    const int64_t hoff = bh * N * D;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;

    const T *kblk = kmat + hoff + (int64_t)k * b * D;
    load_tile<T, NB, D, LDK>([=](int r) { return kblk + (int64_t)r * D; }, b, Ks, tid, 64 * W);
    if constexpr (FINAL) {
        const T *vblk = vmat + hoff + (int64_t)k * b * D;
        load_tile<T, NB, D, LDK>([=](int r) { return vblk + (int64_t)r * D; }, b, Vs, tid, 64 * W);
    }

    static_assert(W == NT, "one wave per 16-row tile");
    {
        const int j = wave * 16 + c16;
        const bool jvalid = j < b;
        const int64_t arow = hoff + ((int64_t)k * b + j) * D;  // alpha_R[k][j] (k-major)
        RowFrags<T, D> bf;
        bf.load(jvalid ? (FIRST ? q : aR) + arow : nullptr, g);
        float rscale = hd.s_log2e;
        if constexpr (!FIRST) {
            if (jvalid) rscale = hd.s_log2e / fmaxf(cR[bh * N + (int64_t)k * b + j], kTiny);
        }
        __syncthreads();

        f32x4 sc[NT];  // lane holds S'[i = 16t + 4g + qq][j]
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            sc[t] = gemm_scores<T, D>(Ks + (16 * t + c16) * LDK, bf, g);
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) sc[t][qq] = (16 * t + 4 * g + qq < b) ? sc[t][qq] * rscale : kMasked;
        }
        float t2;
        const float sum = softmax_cols<NT>(sc, &t2);
        const float inv = 1.0f / sum;
        // c_L = sum_i R log R = sum_i R (Z - max) - log(sum)   (natural-log units)
        if (g == 0 && jvalid) cL[bh * N + (int64_t)j * m + k] = kLn2 * (t2 * inv - __builtin_amdgcn_logf(sum));
#pragma unroll
        for (int t = 0; t < NT; ++t) sc[t] *= inv;

        ProbFrags<T, NT> pf;
        pf.pack(sc);
        T *aL_row = aL + hoff + ((int64_t)j * m + k) * D;  // alpha_L[j][k] (j-major)
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) {
            const f32x4 acc = gemm_aggregate<T, NT>(Ks, LDK, 16 * vt, pf, lane);
            if (jvalid) store4<T>(aL_row + 16 * vt + 4 * g, acc);
        }
        if constexpr (FINAL) {
            T *y_row = Y + hoff + ((int64_t)j * m + k) * D;
#pragma unroll
            for (int vt = 0; vt < D / 16; ++vt) {
                const f32x4 acc = gemm_aggregate<T, NT>(Vs, LDK, 16 * vt, pf, lane);
                if (jvalid) store4<T>(y_row + 16 * vt + 4 * g, acc);
            }
        }
    }
}

// ---------------------------------------------------------------------------------------
// L half-step (not the last): one workgroup per (head, residue class j).
// NM = m rounded up to 16.  Wave w first owns query rows l in [16w, 16w+16)
// (scores and the softmax over k), then, after the probabilities have gone
// through LDS, key-block columns k in [16w, 16w+16) (c_R and alpha_R).
// ---------------------------------------------------------------------------------------
template <typename T, int NM, int D>
__global__ __launch_bounds__(64 * Waves<NM / 16>::value) void l_half_step(
    const T *__restrict__ q, const T *__restrict__ aL, const float *__restrict__ cL,
    T *__restrict__ aR, float *__restrict__ cR, HeadDims hd)
{
    constexpr int NT = NM / 16, W = Waves<NT>::value;
    constexpr int LDQ = Ld<T, D>::row, LDP = Ld<T, NM>::row;
    constexpr int A_ELEMS = NM * LDQ, P_ELEMS = NM * LDP;
    __shared__ __attribute__((aligned(16))) T Qs[NM * LDQ];
    __shared__ __attribute__((aligned(16))) T APs[A_ELEMS > P_ELEMS ? A_ELEMS : P_ELEMS];  // alpha_L, then P
    __shared__ __attribute__((aligned(16))) float cLs[NM];

    const int m = hd.m, b = hd.b;
    const int64_t N = (int64_t)m * b;
    const int j = blockIdx.x % b;
    const int64_t bh = blockIdx.x / b;
    const int64_t hoff = bh * N * D;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;

    const T *qh = q + hoff;
    const T *al = aL + hoff + (int64_t)j * m * D;
    load_tile<T, NM, D, LDQ>([=](int l) { return qh + ((int64_t)l * b + j) * D; }, m, Qs, tid, 64 * W);
    load_tile<T, NM, D, LDQ>([=](int kk) { return al + (int64_t)kk * D; }, m, APs, tid, 64 * W);
    for (int kk = tid; kk < NM; kk += 64 * W) cLs[kk] = kk < m ? cL[bh * N + (int64_t)j * m + kk] * kLog2e : 0.f;
    __syncthreads();

    // scores and softmax over k for the query rows of this wave
    static_assert(W == NT, "one wave per 16-row tile");
    const int l = wave * 16 + c16;
    RowFrags<T, D> bf;
#pragma unroll
    for (int c = 0; c < D / Mma<T>::KC; ++c)
        bf.f[c] = *reinterpret_cast<const typename Mma<T>::frag *>(Qs + l * LDQ + c * Mma<T>::KC + g * Mma<T>::KPL);
    f32x4 sc[NT];  // lane holds S'[k = 16t + 4g + qq][l]
#pragma unroll
    for (int t = 0; t < NT; ++t) {
        sc[t] = gemm_scores<T, D>(APs + (16 * t + c16) * LDQ, bf, g);
        const f32x4 bias = *reinterpret_cast<const f32x4 *>(cLs + 16 * t + 4 * g);
#pragma unroll
        for (int qq = 0; qq < 4; ++qq)
            sc[t][qq] = (16 * t + 4 * g + qq < m) ? sc[t][qq] * hd.s_log2e - bias[qq] : kMasked;
    }
    const float sum = softmax_cols<NT>(sc, nullptr);
    const float inv = (l < m) ? 1.0f / sum : 0.f;  // padded query rows carry no weight
    __syncthreads();  // every wave is done reading alpha_L

    // P[l][k] (row-major, k contiguous) into the alpha_L space
    using PT = typename std::conditional<std::is_same<T, float>::value, float, T>::type;
    PT *Ps = reinterpret_cast<PT *>(APs);
#pragma unroll
    for (int t = 0; t < NT; ++t) store4<PT>(Ps + l * LDP + 16 * t + 4 * g, sc[t] * inv);
    __syncthreads();

    // wave w: key-block columns k0 = 16w
    const int k0 = wave * 16;
    ProbFrags<T, NT> pf;  // B operand: P[l-slots][k0 + c16]
    pf.gather(Ps, LDP, k0, lane);
    const int kk = k0 + c16;
    const f32x4 cs = gemm_colsum<T, NT>(pf);  // c_R[k][j] = sum_l L[j][k][l]
    if (g == 0 && kk < m) cR[bh * N + (int64_t)kk * b + j] = cs[0];
    T *ar_row = aR + hoff + ((int64_t)kk * b + j) * D;  // alpha_R[k][j] (k-major)
#pragma unroll
    for (int vt = 0; vt < D / 16; ++vt) {
        const f32x4 acc = gemm_aggregate<T, NT>(Qs, LDQ, 16 * vt, pf, lane);
        if (kk < m) store4<T>(ar_row + 16 * vt + 4 * g, acc);
    }
}

// ---------------------------------------------------------------------------------------
// Last L half-step fused with the second Monarch product and the store of O:
// one workgroup per (head, j), one wave per 16 query rows l.
// ---------------------------------------------------------------------------------------
template <typename T, int NM, int D>
__global__ __launch_bounds__(64 * Waves<NM / 16>::value) void monarch_apply(
    const T *__restrict__ q, const T *__restrict__ aL, const float *__restrict__ cL,
    const T *__restrict__ Y, T *__restrict__ out, HeadDims hd)
{
    constexpr int NT = NM / 16, W = Waves<NT>::value;
    constexpr int LDK = Ld<T, D>::row;
    __shared__ __attribute__((aligned(16))) T As[NM * LDK];
    __shared__ __attribute__((aligned(16))) T Ys[NM * LDK];
    __shared__ __attribute__((aligned(16))) float cLs[NM];

    const int m = hd.m, b = hd.b;
    const int64_t N = (int64_t)m * b;
    const int j = blockIdx.x % b;
    const int64_t bh = blockIdx.x / b;
    const int64_t hoff = bh * N * D;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;

    const T *al = aL + hoff + (int64_t)j * m * D;
    const T *yj = Y + hoff + (int64_t)j * m * D;
    load_tile<T, NM, D, LDK>([=](int kk) { return al + (int64_t)kk * D; }, m, As, tid, 64 * W);
    load_tile<T, NM, D, LDK>([=](int kk) { return yj + (int64_t)kk * D; }, m, Ys, tid, 64 * W);
    for (int kk = tid; kk < NM; kk += 64 * W) cLs[kk] = kk < m ? cL[bh * N + (int64_t)j * m + kk] * kLog2e : 0.f;

    static_assert(W == NT, "one wave per 16-row tile");
    {
        const int l = wave * 16 + c16;
        const bool lvalid = l < m;
        const int64_t qrow = hoff + ((int64_t)l * b + j) * D;  // Qbar[j][l]
        RowFrags<T, D> bf;
        bf.load(lvalid ? q + qrow : nullptr, g);
        __syncthreads();

        f32x4 sc[NT];  // lane holds S'[k = 16t + 4g + qq][l]
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            sc[t] = gemm_scores<T, D>(As + (16 * t + c16) * LDK, bf, g);
            const f32x4 bias = *reinterpret_cast<const f32x4 *>(cLs + 16 * t + 4 * g);
#pragma unroll
            for (int qq = 0; qq < 4; ++qq)
                sc[t][qq] = (16 * t + 4 * g + qq < m) ? sc[t][qq] * hd.s_log2e - bias[qq] : kMasked;
        }
        const float inv = 1.0f / softmax_cols<NT>(sc, nullptr);
#pragma unroll
        for (int t = 0; t < NT; ++t) sc[t] *= inv;

        ProbFrags<T, NT> pf;
        pf.pack(sc);
        T *o_row = out + qrow;
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) {
            const f32x4 acc = gemm_aggregate<T, NT>(Ys, LDK, 16 * vt, pf, lane);
            if (lvalid) store4<T>(o_row + 16 * vt + 4 * g, acc);
        }
    }
}

}  // namespace ma
