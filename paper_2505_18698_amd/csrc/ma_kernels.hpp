// MonarchAttention forward kernels for CDNA4 (gfx950).
//
// One kernel per half-step of the alternating maximisation (Sec. 3 of the
// paper, eqs. R_update / L_update with beta_r / beta_l), organised as in the
// paper's Implementation paragraph: the factors L and R live only in
// registers; between launches only the states alpha_R, c_R, alpha_L, c_L and
// Y cross global memory.
//
//   r_half_step<FIRST, FINAL>  one workgroup per (head, key block k):
//        S'[i][j] = Kbar[k][i] . alpha_R[k][j]                (beta_R, MFMA)
//        R[k][j][:] = softmax_i(s * S'[:, j] / c_R[k][j])      (eq. R_update)
//        c_L[j][k] = sum_i R log R,  alpha_L[j][k] = R Kbar[k] (eq. beta_l, MFMA)
//        FINAL: Y[j][k] = R Vbar[k]                            (eq. monarch_multiply)
//   l_half_step                one workgroup per (head, residue class j):
//        S[l][k] = Qbar[j][l] . alpha_L[j][k]                  (beta_L, MFMA)
//        L[j][:][l] = softmax_k(s * S[l][:] - c_L[j][:])       (eq. L_update)
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
// output rows 4*(l/16)+q (q = 0..3) of column l%16.  The probability tile that
// a softmax leaves in registers is fed straight back as the B operand of the
// second product: for a chunk of 32 contraction indices made of two 16-wide
// score tiles, lane l's 8 operand slots are the 4 rows it holds of each tile,
// and the A operand (read from a transposed LDS copy) uses the same slot order.
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
typedef uint32_t u32x4 __attribute__((ext_vector_type(4)));
typedef uint32_t u32x2 __attribute__((ext_vector_type(2)));

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

template <int NT> struct Waves {
    static constexpr int value = NT < 4 ? NT : 4;
};

// Row strides (elements) of the LDS tiles: row-major [rows][D] and transposed [D][rows].
template <typename T, int D> struct Ld {
    static constexpr int row = D + 16 / (int)sizeof(T) * 1;  // keeps 16-byte row alignment
};
template <typename T, int NR> struct LdT {
    static constexpr int row = NR + (sizeof(T) == 4 ? 4 : 4);  // keeps 8/16-byte alignment
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

// Cooperative load of a [NR][D] tile whose valid rows r < valid start at
// rowptr(r); rows >= valid are zero.  Writes the row-major copy (stride LDR)
// when sRow != nullptr and the transposed copy (stride LDT) when sT != nullptr.
template <typename T, int NR, int D, int LDR, int LDT, typename RowPtr>
__device__ inline void load_tile(RowPtr rowptr, int valid, T *sRow, T *sT, int tid, int nthreads)
{
    constexpr int V = 16 / (int)sizeof(T);
    constexpr int CPR = D / V;
    for (int idx = tid; idx < NR * CPR; idx += nthreads) {
        const int r = idx / CPR, c = (idx % CPR) * V;
        u32x4 raw = {0u, 0u, 0u, 0u};
        if (r < valid) raw = *reinterpret_cast<const u32x4 *>(rowptr(r) + c);
        if (sRow) *reinterpret_cast<u32x4 *>(sRow + r * LDR + c) = raw;
        if (sT) {
            T e[V];
            __builtin_memcpy(e, &raw, 16);
#pragma unroll
            for (int q = 0; q < V; ++q) sT[(c + q) * LDT + r] = e[q];
        }
    }
}

// B-operand fragments of one 16-row block of a row-major [*, D] matrix held in
// global memory (row pointer `row`, nullptr for a zero row).
template <typename T, int D> struct RowFrags {
    using M = Mma<T>;
    typename M::frag f[D / M::KC];
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

// The probabilities of NT score tiles (4 values per lane per tile) packed as
// MFMA B-operand fragments, in the tile-pair slot order described above.
template <typename T, int NT, bool IS_F32 = std::is_same<T, float>::value> struct ProbFrags;

template <typename T, int NT> struct ProbFrags<T, NT, false> {
    using M = Mma<T>;
    static constexpr int NC = NT / 2;
    typename M::frag f[NC > 0 ? NC : 1];
    typename M::frag4 f4;
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
};

template <typename T, int NT> struct ProbFrags<T, NT, true> {
    f32x4 p[NT];
    __device__ inline void pack(const f32x4 *src)
    {
#pragma unroll
        for (int t = 0; t < NT; ++t) p[t] = src[t];
    }
};

// acc = A[r0 + 0..15][contraction] * P : one 16x16 tile of an aggregation
// product.  sT_row points to row (r0 + lane%16) of a transposed LDS copy, whose
// columns are the contraction index (the score tiles' row index).
template <typename T, int NT>
__device__ inline f32x4 gemm_aggregate(const T *sT_row, const ProbFrags<T, NT> &pf, int g)
{
    using M = Mma<T>;
    f32x4 acc = {0.f, 0.f, 0.f, 0.f};
    if constexpr (std::is_same<T, float>::value) {
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int q = 0; q < 4; ++q) acc = M::mma(sT_row[16 * t + 4 * g + q], pf.p[t][q], acc);
        }
    } else {
#pragma unroll
        for (int c = 0; c < NT / 2; ++c) {
            const typename M::frag4 lo = *reinterpret_cast<const typename M::frag4 *>(sT_row + 32 * c + 4 * g);
            const typename M::frag4 hi = *reinterpret_cast<const typename M::frag4 *>(sT_row + 32 * c + 16 + 4 * g);
            const typename M::frag a = __builtin_shufflevector(lo, hi, 0, 1, 2, 3, 4, 5, 6, 7);
            acc = M::mma(a, pf.f[c], acc);
        }
        if constexpr (NT % 2 == 1) {
            const typename M::frag4 a =
                *reinterpret_cast<const typename M::frag4 *>(sT_row + 16 * (NT - 1) + 4 * g);
            acc = M::mma4(a, pf.f4, acc);
        }
    }
    return acc;
}

struct HeadDims {
    int m, b;          // blocks and block size, N = m * b
    float s_log2e;     // log2(e) / sqrt(d)
};

// ---------------------------------------------------------------------------------------
// R half-step: one workgroup per (head, key block k).  NB = b rounded up to 16.
// FIRST: alpha_R = the rows of Q (L^(0) = I) and c_R = 1.  FINAL: also Y.
// ---------------------------------------------------------------------------------------
template <typename T, int NB, int D, bool FIRST, bool FINAL>
__global__ __launch_bounds__(64 * Waves<NB / 16>::value) void r_half_step(
    const T *__restrict__ q, const T *__restrict__ kmat, const T *__restrict__ vmat,
    const T *__restrict__ aR, const float *__restrict__ cR, T *__restrict__ aL,
    float *__restrict__ cL, T *__restrict__ Y, HeadDims hd)
{
    constexpr int NT = NB / 16, W = Waves<NT>::value;
    constexpr int LDK = Ld<T, D>::row, LDT = LdT<T, NB>::row;
    __shared__ __attribute__((aligned(16))) T Ks[NB * LDK];
    __shared__ __attribute__((aligned(16))) T KsT[D * LDT];
    __shared__ __attribute__((aligned(16))) T VsT[FINAL ? D * LDT : 8];

    const int m = hd.m, b = hd.b;
    const int64_t N = (int64_t)m * b;
    const int k = blockIdx.x % m;
    const int64_t bh = blockIdx.x / m;
    const int64_t hoff = bh * N * D;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;

    const T *kblk = kmat + hoff + (int64_t)k * b * D;
    load_tile<T, NB, D, LDK, LDT>([=](int r) { return kblk + (int64_t)r * D; }, b, Ks, KsT, tid, 64 * W);
    if constexpr (FINAL) {
        const T *vblk = vmat + hoff + (int64_t)k * b * D;
        load_tile<T, NB, D, LDK, LDT>([=](int r) { return vblk + (int64_t)r * D; }, b, (T *)nullptr, VsT,
                                      tid, 64 * W);
    }
    __syncthreads();

    for (int rt = wave; rt < NT; rt += W) {
        const int j = rt * 16 + c16;
        const bool jvalid = j < b;
        const int64_t arow = hoff + ((int64_t)k * b + j) * D;  // alpha_R[k][j] (k-major)
        RowFrags<T, D> bf;
        bf.load(jvalid ? (FIRST ? q : aR) + arow : nullptr, g);
        float rscale = hd.s_log2e;
        if constexpr (!FIRST) {
            if (jvalid) rscale = hd.s_log2e / fmaxf(cR[bh * N + (int64_t)k * b + j], kTiny);
        }

        f32x4 sc[NT];  // lane holds S'[i = 16t + 4g + qq][j]
#pragma unroll
        for (int t = 0; t < NT; ++t) sc[t] = gemm_scores<T, D>(Ks + (16 * t + c16) * LDK, bf, g);

        float mx = kMasked;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
                const int i = 16 * t + 4 * g + qq;
                const float z = (i < b) ? sc[t][qq] * rscale : kMasked;
                sc[t][qq] = z;
                mx = fmaxf(mx, z);
            }
        }
        mx = wave_xor_max(mx, 16);
        mx = wave_xor_max(mx, 32);
        float sum = 0.f, t2 = 0.f;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
                const float u = sc[t][qq] - mx;
                const float e = __builtin_amdgcn_exp2f(u);
                sum += e;
                t2 += e * u;
                sc[t][qq] = e;
            }
        }
        sum = wave_xor_sum(sum, 16);
        sum = wave_xor_sum(sum, 32);
        t2 = wave_xor_sum(t2, 16);
        t2 = wave_xor_sum(t2, 32);
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
            const f32x4 acc = gemm_aggregate<T, NT>(KsT + (16 * vt + c16) * LDT, pf, g);
            if (jvalid) store4<T>(aL_row + 16 * vt + 4 * g, acc);
        }
        if constexpr (FINAL) {
            T *y_row = Y + hoff + ((int64_t)j * m + k) * D;
#pragma unroll
            for (int vt = 0; vt < D / 16; ++vt) {
                const f32x4 acc = gemm_aggregate<T, NT>(VsT + (16 * vt + c16) * LDT, pf, g);
                if (jvalid) store4<T>(y_row + 16 * vt + 4 * g, acc);
            }
        }
    }
}

// ---------------------------------------------------------------------------------------
// L half-step (not the last): one workgroup per (head, residue class j).
// NM = m rounded up to 16.  Waves split the key-block columns k; each row's
// softmax statistics are combined across waves through LDS.
// ---------------------------------------------------------------------------------------
template <typename T, int NM, int D>
__global__ __launch_bounds__(64 * Waves<NM / 16>::value) void l_half_step(
    const T *__restrict__ q, const T *__restrict__ aL, const float *__restrict__ cL,
    T *__restrict__ aR, float *__restrict__ cR, HeadDims hd)
{
    constexpr int NT = NM / 16, W = Waves<NT>::value, KTW = NT / W;
    constexpr int LDK = Ld<T, D>::row, LDT = LdT<T, NM>::row;
    __shared__ __attribute__((aligned(16))) T Qs[NM * LDK];
    __shared__ __attribute__((aligned(16))) T QsT[D * LDT];
    __shared__ float rmax[W][NM];
    __shared__ float rsum[W][NM];

    const int m = hd.m, b = hd.b;
    const int64_t N = (int64_t)m * b;
    const int j = blockIdx.x % b;
    const int64_t bh = blockIdx.x / b;
    const int64_t hoff = bh * N * D;
    const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
    const int g = lane >> 4, c16 = lane & 15;

    const T *qh = q + hoff;
    load_tile<T, NM, D, LDK, LDT>([=](int l) { return qh + ((int64_t)l * b + j) * D; }, m, Qs, QsT, tid, 64 * W);

    RowFrags<T, D> bf[KTW];
    float bias[KTW];
#pragma unroll
    for (int e = 0; e < KTW; ++e) {
        const int kk = (wave * KTW + e) * 16 + c16;
        const bool kvalid = kk < m;
        bf[e].load(kvalid ? aL + hoff + ((int64_t)j * m + kk) * D : nullptr, g);
        bias[e] = kvalid ? cL[bh * N + (int64_t)j * m + kk] * kLog2e : 0.f;
    }
    __syncthreads();

    f32x4 sc[KTW][NT];  // lane holds S[l = 16 lt + 4g + qq][k = 16 (wave*KTW + e) + c16]
#pragma unroll
    for (int e = 0; e < KTW; ++e) {
        const int kk = (wave * KTW + e) * 16 + c16;
#pragma unroll
        for (int lt = 0; lt < NT; ++lt) {
            f32x4 s = gemm_scores<T, D>(Qs + (16 * lt + c16) * LDK, bf[e], g);
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) s[qq] = (kk < m) ? s[qq] * hd.s_log2e - bias[e] : kMasked;
            sc[e][lt] = s;
        }
    }
    // row maxima over k: in-lane over e, across the 16 lanes of a row group, across waves
#pragma unroll
    for (int lt = 0; lt < NT; ++lt) {
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            float mx = sc[0][lt][qq];
#pragma unroll
            for (int e = 1; e < KTW; ++e) mx = fmaxf(mx, sc[e][lt][qq]);
            mx = wave_xor_max(mx, 1);
            mx = wave_xor_max(mx, 2);
            mx = wave_xor_max(mx, 4);
            mx = wave_xor_max(mx, 8);
            if (c16 == 0) rmax[wave][16 * lt + 4 * g + qq] = mx;
        }
    }
    __syncthreads();
#pragma unroll
    for (int lt = 0; lt < NT; ++lt) {
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const int l = 16 * lt + 4 * g + qq;
            float mx = rmax[0][l];
#pragma unroll
            for (int w = 1; w < W; ++w) mx = fmaxf(mx, rmax[w][l]);
            float sm = 0.f;
#pragma unroll
            for (int e = 0; e < KTW; ++e) {
                const float ex = __builtin_amdgcn_exp2f(sc[e][lt][qq] - mx);
                sc[e][lt][qq] = ex;
                sm += ex;
            }
            sm = wave_xor_sum(sm, 1);
            sm = wave_xor_sum(sm, 2);
            sm = wave_xor_sum(sm, 4);
            sm = wave_xor_sum(sm, 8);
            if (c16 == 0) rsum[wave][l] = sm;
        }
    }
    __syncthreads();
#pragma unroll
    for (int lt = 0; lt < NT; ++lt) {
#pragma unroll
        for (int qq = 0; qq < 4; ++qq) {
            const int l = 16 * lt + 4 * g + qq;
            float sm = rsum[0][l];
#pragma unroll
            for (int w = 1; w < W; ++w) sm += rsum[w][l];
            const float inv = (l < m) ? 1.0f / sm : 0.f;  // padded query rows carry no weight
#pragma unroll
            for (int e = 0; e < KTW; ++e) sc[e][lt][qq] *= inv;
        }
    }

#pragma unroll
    for (int e = 0; e < KTW; ++e) {
        const int kk = (wave * KTW + e) * 16 + c16;
        // c_R[k][j] = sum_l L[j][k][l]
        float cs = 0.f;
#pragma unroll
        for (int lt = 0; lt < NT; ++lt) cs += sc[e][lt][0] + sc[e][lt][1] + sc[e][lt][2] + sc[e][lt][3];
        cs = wave_xor_sum(cs, 16);
        cs = wave_xor_sum(cs, 32);
        if (g == 0 && kk < m) cR[bh * N + (int64_t)kk * b + j] = cs;

        ProbFrags<T, NT> pf;
        pf.pack(sc[e]);
        T *ar_row = aR + hoff + ((int64_t)kk * b + j) * D;  // alpha_R[k][j] (k-major)
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) {
            const f32x4 acc = gemm_aggregate<T, NT>(QsT + (16 * vt + c16) * LDT, pf, g);
            if (kk < m) store4<T>(ar_row + 16 * vt + 4 * g, acc);
        }
    }
}

// ---------------------------------------------------------------------------------------
// Last L half-step fused with the second Monarch product and the store of O:
// one workgroup per (head, j).  Waves split the query rows l.
// ---------------------------------------------------------------------------------------
template <typename T, int NM, int D>
__global__ __launch_bounds__(64 * Waves<NM / 16>::value) void monarch_apply(
    const T *__restrict__ q, const T *__restrict__ aL, const float *__restrict__ cL,
    const T *__restrict__ Y, T *__restrict__ out, HeadDims hd)
{
    constexpr int NT = NM / 16, W = Waves<NT>::value;
    constexpr int LDK = Ld<T, D>::row, LDT = LdT<T, NM>::row;
    __shared__ __attribute__((aligned(16))) T As[NM * LDK];
    __shared__ __attribute__((aligned(16))) T YsT[D * LDT];
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
    load_tile<T, NM, D, LDK, LDT>([=](int kk) { return al + (int64_t)kk * D; }, m, As, (T *)nullptr, tid, 64 * W);
    load_tile<T, NM, D, LDK, LDT>([=](int kk) { return yj + (int64_t)kk * D; }, m, (T *)nullptr, YsT, tid, 64 * W);
    for (int kk = tid; kk < NM; kk += 64 * W) cLs[kk] = kk < m ? cL[bh * N + (int64_t)j * m + kk] * kLog2e : 0.f;
    __syncthreads();

    for (int rt = wave; rt < NT; rt += W) {
        const int l = rt * 16 + c16;
        const bool lvalid = l < m;
        const int64_t qrow = hoff + ((int64_t)l * b + j) * D;  // Qbar[j][l]
        RowFrags<T, D> bf;
        bf.load(lvalid ? q + qrow : nullptr, g);

        f32x4 sc[NT];  // lane holds S'[k = 16t + 4g + qq][l]
#pragma unroll
        for (int t = 0; t < NT; ++t) sc[t] = gemm_scores<T, D>(As + (16 * t + c16) * LDK, bf, g);
        float mx = kMasked;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
            const f32x4 bias = *reinterpret_cast<const f32x4 *>(cLs + 16 * t + 4 * g);
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
                const int kk = 16 * t + 4 * g + qq;
                const float z = (kk < m) ? sc[t][qq] * hd.s_log2e - bias[qq] : kMasked;
                sc[t][qq] = z;
                mx = fmaxf(mx, z);
            }
        }
        mx = wave_xor_max(mx, 16);
        mx = wave_xor_max(mx, 32);
        float sum = 0.f;
#pragma unroll
        for (int t = 0; t < NT; ++t) {
#pragma unroll
            for (int qq = 0; qq < 4; ++qq) {
                const float e = __builtin_amdgcn_exp2f(sc[t][qq] - mx);
                sc[t][qq] = e;
                sum += e;
            }
        }
        sum = wave_xor_sum(sum, 16);
        sum = wave_xor_sum(sum, 32);
        const float inv = 1.0f / sum;
#pragma unroll
        for (int t = 0; t < NT; ++t) sc[t] *= inv;

        ProbFrags<T, NT> pf;
        pf.pack(sc);
        T *o_row = out + qrow;
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) {
            const f32x4 acc = gemm_aggregate<T, NT>(YsT + (16 * vt + c16) * LDT, pf, g);
            if (lvalid) store4<T>(o_row + 16 * vt + 4 * g, acc);
        }
    }
}

}  // namespace ma
