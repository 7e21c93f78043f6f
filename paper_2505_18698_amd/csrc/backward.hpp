// Gradient of the MonarchAttention forward pass: reverse mode through the
// unrolled T steps of Sec. 3 (the paper gives no gradient; the sweep below is
// derived from the state form of its Implementation paragraph).
//
// Notation per head, with s = 1/sqrt(d), Qbar[j][l] = Q[l*b + j] (unscaled),
// Kbar[k][i] = K[k*b + i], and the states of step t as the forward stores
// them (alpha_R unscaled, the scale applied on the scores):
//   R update of block k:  Z_R[j][i] = s <alpha_R[k][j], Kbar[k][i]> / c_R[k][j]
//                         (keys i past the sequence masked), R = softmax_i Z_R,
//                         alpha_L[j][k] = sum_i R Kbar[k][i], c_L[j][k] = sum_i R log R,
//                         Y[j][k] = sum_i R Vbar[k][i] at the last step;
//   L update of class j:  Z_L[l][k] = s <Qbar[j][l], alpha_L[j][k]> - c_L[j][k],
//                         L = softmax_k Z_L, alpha_R'[k][j] = sum_l L Qbar[j][l],
//                         c_R'[k][j] = sum_l L (inputs of step t+1), and at the
//                         last step O[l*b + j] = sum_k L Y[j][k];
//   step 1 starts from L = I: alpha_R[k][j] = Q[k*b + j], c_R = 1.
// A softmax p = softmax(z) pulls dp back to dz = p (dp - <p, dp>).
//
// The sweep runs t = T .. 1, one launch per half-step:
//   l_bwd (class j of step t):  dL = dO . Y (t = T; also dY = L^T dO) or
//       dL = Qbar . d alpha_R' + d c_R' (t < T; also dQbar += L d alpha_R');
//       dW = s L (dL - <L, dL>) (the scale folded in);  dQbar += dW alpha_L,
//       d alpha_L = dW^T Qbar,  d c_L = -(1/s) sum_l dW.
//   r_bwd (block k of step t):  dR = d alpha_L . Kbar + d c_L (log R + 1)
//       (+ dY . Vbar at t = T, with dVbar = R^T dY);  dZ = R (dR - <R, dR>);
//       dKbar += R^T d alpha_L + (s dZ / c_R)^T alpha_R;
//       d alpha_R = (s dZ / c_R) Kbar;  d c_R = -sum_i dZ log R / c_R (the rows
//       of dZ sum to zero, so log R stands in for the logits);  at t = 1
//       d alpha_R is added to dQ (alpha_R = the rows of Q) and c_R is constant.
//
// Every unit keeps its matrices in LDS tiles, fp32 except the whole-unit tiles
// that are exact in a 16-bit element type at 64 and 128 rows (see Geo), and
// runs every product on v_mfma_f32_16x16x4f32.  A unit sizes its tiles by its
// own dimension (m for l_bwd, b for r_bwd).  When its tiles do not fit at
// once, it walks its own rows (j in r_bwd, l in l_bwd) in chunks, the sums
// over those rows (dK, dV, dY, d alpha_L, d c_L) accumulating in registers.  The gradients of the states and the dQ, dK
// accumulators are fp32 in the workspace.  Within a launch the units write
// disjoint rows, and launches that touch the same rows are ordered on the
// stream, so read-modify-writes need no atomics and the result is
// deterministic.  dq and dk are written in the element type by the step-1
// R launch (the last one to touch them), dv by the step-T R launch.
#pragma once

#include "ma_kernels.hpp"

namespace ma {

template <typename T> struct BwdBufs {
    const T *q, *k, *v, *dout;  // [B*H][n][d]
    const T *aR, *aL, *Y;       // states of the step being undone ([m][b][D], [b][m][D], [b][m][D], D the tile width)
    const float *cR, *cL;       // c_R [b][m] (j-major), c_L [m][b] (k-major), as the forward writes them
    float *dQ, *dK;             // fp32 accumulators [B*H][n][d]
    T *dq, *dk, *dv;            // results [B*H][n][d]
    float *daL, *dcL, *dY;      // [b][m][D], [b][m], [b][m][D]: written by l_bwd, read by r_bwd of the step
    float *daR, *dcR;           // [m][b][D], [m][b]: written by r_bwd of step t, read by l_bwd of step t-1
};

struct BwdDims {
    int m, b, n, d;  // as in the forward (the states have rows of d elements, the fp32 state gradients of D)
    float s;         // 1/sqrt(d)
    // Per-sequence lengths (batch padding): head bh has lens[bh / H] real
    // rows, clamped to 0..n, or n when lens is null.  Rows past them count as
    // zero in the forward, so their gradients are zero.
    const int *lens = nullptr;
    int H = 1;
};

namespace bwd {

// Real rows of head bh (bh < 2^31: the grids are checked on the host).
__device__ inline int live_rows(const BwdDims &dm, int64_t bh)
{
    if (!dm.lens) return dm.n;
    const int len = dm.lens[(int)bh / dm.H];
    return len < 0 ? 0 : len > dm.n ? dm.n : len;
}

// Row strides (floats) of the LDS tiles: 16-byte rows, 68 floats for tiles
// of up to 64 columns, 100 and 148 for 96 and 128.  The 64-column stride is
// the smallest measured: at 16-row units the smaller tiles let six workgroups
// share a CU instead of five (11% faster), and strides of 72 to 88 were no
// faster at 64 or 128 rows.
constexpr int row_stride(int cols) { return cols <= 64 ? 68 : cols <= 96 ? 100 : 148; }

constexpr int unit_waves(int S) { return S >= 64 ? 16 : S / 4; }

// Whether two workgroups of a unit kernel share a CU: 64-row units at D = 64
// with 16-bit elements, whose LDS (16-bit unit tiles) leaves room for two.
// Their kernels carry a waves-per-SIMD bound that keeps the registers of two.
constexpr bool two_per_cu(int S, int D, int elem_bytes) { return S == 64 && D == 64 && elem_bytes == 2; }

// With 16-bit elements (H16) the whole-unit tiles that are exact in the
// element type (alpha_L in l_bwd, K and V in r_bwd) can be held as 16-bit
// LDS tiles of row stride LD16, converted on every read (HALF):
// - at 128 rows and D = 128, where two fp32 128 x 128 tiles alone would fill
//   the LDS (the forward takes fp32 at D = 128 for blocks of up to 64 rows);
// - at 64 rows and D = 64, where with rows in chunks of 32 it brings a unit under half
//   the LDS, so that two workgroups share a CU and one's loads overlap the
//   other's compute.
template <int S, int D, bool H16 = false> struct Geo {
    static constexpr bool HALF = H16 && (S == 128 ? D == 128 : S == 64 && D == 64);
    static constexpr int BUDGET = (HALF && S == 64) ? 20480 : 40960;  // floats of LDS per workgroup
    static constexpr int LD16 = D + 8;  // row stride (elements) of a 16-bit tile: 16-byte rows
    static constexpr int W = unit_waves(S);
    static constexpr int NTH = 64 * W;
    static constexpr int LD = row_stride(D);
    static constexpr int LS = row_stride(S);
    // floats of the whole-unit tiles (the larger need, l_bwd's, when HALF)
    static constexpr int UNIT = HALF ? S * LD16 / 2 + S * LD : 2 * S * LD;
    static constexpr int lds_floats(int c) { return UNIT + 3 * c * LD + 2 * c * LS + 2 * S; }
    static constexpr int C = lds_floats(S) <= BUDGET ? S : lds_floats(32) <= BUDGET ? 32 : 16;
    static constexpr int NCH = S / C;
    // row passes: a row of S scores spans SPAN lanes (CPL columns each), a wave
    // instruction covers RPW rows
    static constexpr int SPAN = S < 64 ? S : 64, RPW = 64 / SPAN, CPL = S > 64 ? S / 64 : 1;
    static_assert(lds_floats(C) <= 40960, "tile shape exceeds the LDS of one CU");
};

// Cross-lane reductions with no LDS round trip.
template <int CTRL> __device__ inline float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E, kRowHalfMirror = 0x141, kRowMirror = 0x140;

// Sum and max over groups of G consecutive lanes (G = 16, 32 or 64): DPP
// within rows of 16 lanes, then the permlane swaps across rows as far as the
// group reaches.  Every lane of a group ends with the group's value.
template <int G> __device__ inline float group_sum(float x)
{
    x += dpp<kQuadXor1>(x);
    x += dpp<kQuadXor2>(x);
    x += dpp<kRowHalfMirror>(x);
    x += dpp<kRowMirror>(x);
    if constexpr (G >= 32) x = wave_xor_sum<16>(x);
    if constexpr (G >= 64) x = wave_xor_sum<32>(x);
    return x;
}

template <int G> __device__ inline float group_max(float x)
{
    x = max_nan(x, dpp<kQuadXor1>(x));
    x = max_nan(x, dpp<kQuadXor2>(x));
    x = max_nan(x, dpp<kRowHalfMirror>(x));
    x = max_nan(x, dpp<kRowMirror>(x));
    if constexpr (G >= 32) x = wave_xor_max<16>(x);
    if constexpr (G >= 64) x = wave_xor_max<32>(x);
    return x;
}

// Operands of a product, as LDS tiles with row strides LA, LB:
//   A(r, k) = TA ? A[k][r] : A[r][k],   B(k, n) = TB ? B[n][k] : B[k][n].
// MFMA step s of a 16-long chunk k0 hands lane group g = lane/16 the index
// k0 + 4g + s, so a lane reads four consecutive k at once: one 16-byte read
// where k is contiguous (A as stored, B transposed), four conflict-free
// scalar reads otherwise.  The contraction length is a compile-time constant:
// the loop unrolls, every read is the lane's base address plus an immediate
// offset, and all reads can be issued ahead of the MFMAs.
// Four consecutive elements of an LDS tile as floats: one 16-byte read of
// fp32, or one 8-byte read of 16-bit elements converted exactly.
template <typename E> __device__ inline void read4(const E *p, float *v)
{
    if constexpr (std::is_same<E, float>::value) {
        const f32x4 x = *reinterpret_cast<const f32x4 *>(p);
#pragma unroll
        for (int s = 0; s < 4; ++s) v[s] = x[s];
    } else {
        E e[4];
        *reinterpret_cast<u32x2 *>(e) = *reinterpret_cast<const u32x2 *>(p);
#pragma unroll
        for (int s = 0; s < 4; ++s) v[s] = static_cast<float>(e[s]);
    }
}

// Operands of a product, as LDS tiles (element types EA, EB: fp32, or the
// 16-bit element type for the whole-unit tiles of 128 x 128 units) with row
// strides LA, LB:
//   A(r, k) = TA ? A[k][r] : A[r][k],   B(k, n) = TB ? B[n][k] : B[k][n].
template <bool TA, bool TB, int LA, int LB, typename EA = float, typename EB = float> struct Pair {
    const EA *A;
    const EB *B;

    // acc += sum_{k < K} A(r, k) B(k, n)
    template <int K> __device__ void accumulate(f32x4 &acc, int r, int n, int g) const
    {
        const EA *pa = TA ? A + 4 * g * LA + r : A + r * LA + 4 * g;
        const EB *pb = TB ? B + n * LB + 4 * g : B + 4 * g * LB + n;
#pragma unroll
        for (int k0 = 0; k0 < K; k0 += 16) {
            float a[4], b[4];
            if constexpr (TA) {
#pragma unroll
                for (int s = 0; s < 4; ++s) a[s] = static_cast<float>(pa[(k0 + s) * LA]);
            } else {
                read4(pa + k0, a);
            }
            if constexpr (TB) {
                read4(pb + k0, b);
            } else {
#pragma unroll
                for (int s = 0; s < 4; ++s) b[s] = static_cast<float>(pb[(k0 + s) * LB]);
            }
#pragma unroll
            for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], acc, 0, 0, 0);
        }
    }
};

template <bool TA, bool TB, int LA, int LB, typename EA, typename EB>
__device__ inline Pair<TA, TB, LA, LB, EA, EB> pair(const EA *A, const EB *B)
{
    return Pair<TA, TB, LA, LB, EA, EB>{A, B};
}

// out(r, c) = sum over the pairs of A(r, :) B(:, c) for r < M, c < N, with
// contraction K (all multiples of 16, fixed at compile time: the tiles are
// zero beyond the live rows and columns).  The 16 x 16 output tiles are
// shared out over the W waves; lane (g, c) of v_mfma_f32_16x16x4f32 receives
// rows 4g + q, q = 0..3, of column c, and hands each element to
// st(r, c, value): every element is stored by exactly one lane.
template <int W, int M, int N, int K, typename Store, typename... P>
__device__ inline void gemm(int wave, int lane, Store &&st, const P &...pairs)
{
    constexpr int tn = N / 16, tiles = (M / 16) * tn;
    const int g = lane >> 4, c = lane & 15;
    for (int t = wave; t < tiles; t += W) {
        const int r0 = (t / tn) * 16, c0 = (t % tn) * 16;
        f32x4 acc = {0.f, 0.f, 0.f, 0.f};
        (pairs.template accumulate<K>(acc, r0 + c, c0 + c, g), ...);
#pragma unroll
        for (int q = 0; q < 4; ++q) st(r0 + 4 * g + q, c0 + c, acc[q]);
    }
}

// An M x N product accumulated over several calls (one per row chunk) in the
// registers of the waves that own its output tiles: the same tile-to-wave
// assignment as gemm, each wave holding SLOTS tiles.
template <int W, int M, int N> struct Acc {
    static constexpr int TN = N / 16, TILES = (M / 16) * TN, SLOTS = (TILES + W - 1) / W;
    f32x4 v[SLOTS];

    __device__ void zero()
    {
#pragma unroll
        for (int s = 0; s < SLOTS; ++s) v[s] = f32x4{0.f, 0.f, 0.f, 0.f};
    }

    template <int K, typename... P> __device__ void add(int wave, int lane, const P &...pairs)
    {
        const int g = lane >> 4, c = lane & 15;
#pragma unroll
        for (int s = 0; s < SLOTS; ++s) {
            const int t = wave + s * W;
            if (t < TILES) {
                const int r0 = (t / TN) * 16, c0 = (t % TN) * 16;
                (pairs.template accumulate<K>(v[s], r0 + c, c0 + c, g), ...);
            }
        }
    }

    template <typename Store> __device__ void store(int wave, int lane, Store &&st) const
    {
        const int g = lane >> 4, c = lane & 15;
#pragma unroll
        for (int s = 0; s < SLOTS; ++s) {
            const int t = wave + s * W;
            if (t < TILES) {
                const int r0 = (t / TN) * 16, c0 = (t % TN) * 16;
#pragma unroll
                for (int q = 0; q < 4; ++q) st(r0 + 4 * g + q, c0 + c, v[s][q]);
            }
        }
    }
};

template <int LD> __device__ inline auto to_lds(float *t)
{
    return [t](int r, int c, float v) { t[r * LD + c] = v; };
}

// Rows r < R and columns c < C (compile-time extents, C a multiple of 16;
// row stride LDT) of an LDS tile from a row-major global matrix of element type E whose
// row r starts at src(r) (16-byte aligned): element (r, c) is read while
// r < nr and c < nc (nc a multiple of 16 bytes' worth of elements), zero
// elsewhere.  One 16-byte global read per chunk.
template <typename E, int NTH, int R, int C, int LDT, typename Src>
__device__ inline void load_tile(float *dst, int nr, int nc, Src src, int tid)
{
    constexpr int V = 16 / (int)sizeof(E), CPR = C / V;  // elements per chunk, chunks per row
    for (int idx = tid; idx < R * CPR; idx += NTH) {
        const int r = idx / CPR, c = (idx % CPR) * V;
        float v[V];
        if (r < nr && c < nc) {
            E e[V];
            *reinterpret_cast<uint4 *>(e) = *reinterpret_cast<const uint4 *>(src(r) + c);
#pragma unroll
            for (int i = 0; i < V; ++i) v[i] = static_cast<float>(e[i]);
        } else {
#pragma unroll
            for (int i = 0; i < V; ++i) v[i] = 0.f;
        }
#pragma unroll
        for (int i = 0; i < V; i += 4)
            *reinterpret_cast<f32x4 *>(dst + r * LDT + c + i) = f32x4{v[i], v[i + 1], v[i + 2], v[i + 3]};
    }
}

// load_tile into a tile of the element type itself (no conversion): rows of
// C elements at row stride LDT, zero past nr rows and nc columns.
template <typename E, int NTH, int R, int C, int LDT, typename Src>
__device__ inline void load_tile_raw(E *dst, int nr, int nc, Src src, int tid)
{
    constexpr int V = 16 / (int)sizeof(E), CPR = C / V;
    static_assert(LDT % V == 0, "16-byte rows");
    for (int idx = tid; idx < R * CPR; idx += NTH) {
        const int r = idx / CPR, c = (idx % CPR) * V;
        uint4 x = {0u, 0u, 0u, 0u};
        if (r < nr && c < nc) x = *reinterpret_cast<const uint4 *>(src(r) + c);
        *reinterpret_cast<uint4 *>(dst + r * LDT + c) = x;
    }
}

// A whole-unit tile in the element type when HALF, else in fp32.
template <typename T, int NTH, int R, int C, int LDT, bool HALF, typename U, typename Src>
__device__ inline void load_unit(U *dst, int nr, int nc, Src src, int tid)
{
    if constexpr (HALF)
        load_tile_raw<T, NTH, R, C, LDT>(dst, nr, nc, src, tid);
    else
        load_tile<T, NTH, R, C, LDT>(dst, nr, nc, src, tid);
}

// ---------------------------------------------------------------------------------------
// The L update of class j of step t undone (LAST: t = T, the update that also
// produced O).  S >= m; query rows l in chunks of C.
// ---------------------------------------------------------------------------------------
template <typename T, int S, int D, bool LAST, bool LENS = false> struct LBwd {
    using G_ = Geo<S, D, sizeof(T) == 2>;
    static constexpr int W = G_::W, NTH = G_::NTH, C = G_::C, LS = G_::LS, CPL = G_::CPL, LD = G_::LD;
    static constexpr int SPAN = G_::SPAN, RPW = G_::RPW;
    static constexpr bool HALF = G_::HALF;
    static_assert(!HALF || sizeof(T) == 2, "16-bit unit tiles need 16-bit elements");
    using UT = typename std::conditional<HALF, T, float>::type;  // alpha_L tile
    static constexpr int LDU = HALF ? G_::LD16 : LD;
    static constexpr int UF = S * LDU * (int)sizeof(UT) / 4;  // its floats
    static constexpr int LDS_FLOATS = UF + S * LD + 2 * C * LD + 2 * C * LS + 2 * S;

    __device__ static void run(const BwdBufs<T> &p, const BwdDims &dm, float *lds)
    {
        const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
        const int m = dm.m, b = dm.b, n = dm.n, d = dm.d;
        const int64_t bh = blockIdx.x / b;
        const int j = blockIdx.x % b;
        const int nl = LENS ? live_rows(dm, bh) : n;
        const int ml = (nl - j + b - 1) / b;                 // real rows l: l*b + j < nl
        const int mk = LENS ? min(m, (nl + b - 1) / b) : m;  // key blocks k < mk hold a real key
        const int64_t Np = (int64_t)m * b, toff = bh * n * d, soff = bh * Np * D, coff = bh * Np;
        const int64_t xoff = bh * Np * d;  // the forward's states: rows of d elements
        // whole-unit tiles (rows k): alpha_L[j][k]; Y[j][k] (LAST) or d alpha_R'[k][j]
        UT *aL = reinterpret_cast<UT *>(lds);
        float *X = lds + UF;
        // chunk tiles (rows l of the chunk): Qbar, dO (LAST) or L d alpha_R', L, dL then dW
        float *Qb = X + S * LD, *G = Qb + C * LD, *Lm = G + C * LD, *dL = Lm + C * LS;
        float *cL = dL + C * LS, *dcR = cL + S;

        load_unit<T, NTH, S, D, LDU, HALF>(aL, m, d, [&](int k) { return p.aL + xoff + ((int64_t)j * m + k) * d; },
                                           tid);
        if constexpr (LAST) {
            load_tile<T, NTH, S, D, LD>(X, m, d, [&](int k) { return p.Y + xoff + ((int64_t)j * m + k) * d; }, tid);
        } else {
            load_tile<float, NTH, S, D, LD>(X, m, d, [&](int k) { return p.daR + soff + ((int64_t)k * b + j) * D; },
                                         tid);
        }
        for (int k = tid; k < S; k += NTH) {
            cL[k] = k < m ? p.cL[coff + (int64_t)k * b + j] : 0.f;
            dcR[k] = (!LAST && k < m) ? p.dcR[coff + (int64_t)k * b + j] : 0.f;
        }
        Acc<W, S, D> daL, dY;  // sums over all rows l
        daL.zero();
        if constexpr (LAST) dY.zero();
        float dcl = 0.f;  // thread k < S: sum over l of dW[l][k]
        float *dQ = p.dQ + toff + (int64_t)j * d;

        for (int ch = 0; ch < G_::NCH; ++ch) {
            const int l0 = ch * C, lc = min(max(ml - l0, 0), C);  // live rows of the chunk
            load_tile<T, NTH, C, D, LD>(Qb, lc, d, [&](int l) { return p.q + toff + ((int64_t)(l0 + l) * b + j) * d; },
                                     tid);
            if constexpr (LAST)
                load_tile<T, NTH, C, D, LD>(
                    G, lc, d, [&](int l) { return p.dout + toff + ((int64_t)(l0 + l) * b + j) * d; }, tid);
            __syncthreads();

            // unnormalised scores <Qbar[l], alpha_L[k]>
            gemm<W, C, S, D>(wave, lane, to_lds<LS>(Lm), pair<false, true, LD, LDU>(Qb, aL));
            __syncthreads();
            // L[l][k] = softmax_k (s score - c_L[k]): RPW rows l per wave instruction,
            // SPAN lanes and CPL columns k per lane for each
            for (int base = wave * RPW; base < C; base += W * RPW) {
                const int l = base + lane / SPAN, col = lane % SPAN;
                const bool live = l0 + l < m && (!LENS || mk > 0);  // no real key at all: L = 0
                float *row = Lm + l * LS;
                float z[CPL], mx = -INFINITY;
#pragma unroll
                for (int u = 0; u < CPL; ++u) {
                    const int k = col + 64 * u;
                    z[u] = live && k < mk ? dm.s * row[k] - cL[k] : -INFINITY;
                    mx = max_nan(mx, z[u]);
                }
                mx = group_max<SPAN>(mx);
                float sum = 0.f;
#pragma unroll
                for (int u = 0; u < CPL; ++u) {
                    z[u] = live && col + 64 * u < mk ? __expf(z[u] - mx) : 0.f;
                    sum += z[u];
                }
                sum = group_sum<SPAN>(sum);
                const float inv = live ? 1.f / sum : 0.f;  // rows past m: all zero
#pragma unroll
                for (int u = 0; u < CPL; ++u)
                    if (col + 64 * u < S) row[col + 64 * u] = z[u] * inv;
            }
            __syncthreads();

            if constexpr (LAST) {
                // dL = dO Y^T;  dY += L^T dO
                gemm<W, C, S, D>(wave, lane, to_lds<LS>(dL), pair<false, true, LD, LD>(G, X));
                dY.template add<C>(wave, lane, pair<true, false, LS, LD>(Lm, G));
            } else {
                // dL = Qbar d alpha_R'^T (+ d c_R' below);  G = L d alpha_R' (the alpha_R' term of dQbar)
                gemm<W, C, S, D>(wave, lane, to_lds<LS>(dL), pair<false, true, LD, LD>(Qb, X));
                gemm<W, C, D, S>(wave, lane, to_lds<LD>(G), pair<false, false, LS, LD>(Lm, X));
            }
            __syncthreads();
            // dW = s L (dL - <L, dL>), in place of dL
            for (int base = wave * RPW; base < C; base += W * RPW) {
                const int l = base + lane / SPAN, col = lane % SPAN;
                float *lr = Lm + l * LS, *wr = dL + l * LS;
                float pk[CPL], w[CPL], dot = 0.f;
#pragma unroll
                for (int u = 0; u < CPL; ++u) {
                    const int k = col + 64 * u;
                    pk[u] = k < S ? lr[k] : 0.f;
                    w[u] = k < S ? wr[k] + dcR[k] : 0.f;
                    dot += pk[u] * w[u];
                }
                dot = group_sum<SPAN>(dot);
#pragma unroll
                for (int u = 0; u < CPL; ++u)
                    if (col + 64 * u < S) wr[col + 64 * u] = dm.s * pk[u] * (w[u] - dot);
            }
            __syncthreads();

            // dQ rows (l0 + l)*b + j: dW alpha_L (+ L d alpha_R')
            gemm<W, C, D, S>(
                wave, lane,
                [&](int l, int e, float v) {
                    if (l < lc && e < d) {
                        float *o = dQ + (int64_t)(l0 + l) * b * d + e;
                        if constexpr (LAST) {
                            *o = v;
                        } else {
                            *o += v + G[l * LD + e];
                        }
                    }
                },
                pair<false, false, LS, LDU>(dL, aL));
            // d alpha_L[k] += dW^T Qbar;  d c_L[k] += sum_l dW[l][k]
            daL.template add<C>(wave, lane, pair<true, false, LS, LD>(dL, Qb));
            if (tid < S) {
                for (int l = 0; l < C; ++l) dcl += dL[l * LS + tid];
            }
            __syncthreads();  // the next chunk overwrites the chunk tiles
        }

        float *daLg = p.daL + soff + (int64_t)j * m * D;
        daL.store(wave, lane, [&](int k, int e, float v) {
            if (k < m && e < d) daLg[(int64_t)k * D + e] = v;
        });
        if constexpr (LAST) {
            float *dYg = p.dY + soff + (int64_t)j * m * D;
            dY.store(wave, lane, [&](int k, int e, float v) {
                if (k < m && e < d) dYg[(int64_t)k * D + e] = v;
            });
        }
        if (tid < m) p.dcL[coff + (int64_t)j * m + tid] = -dcl / dm.s;
    }
};

// ---------------------------------------------------------------------------------------
// The R update of block k of step t undone (FIRST: t = 1, LAST: t = T).
// S >= b; rows j in chunks of C.
// ---------------------------------------------------------------------------------------
template <typename T, int S, int D, bool FIRST, bool LAST, bool LENS = false> struct RBwd {
    using G_ = Geo<S, D, sizeof(T) == 2>;
    static constexpr int W = G_::W, NTH = G_::NTH, C = G_::C, LS = G_::LS, CPL = G_::CPL, LD = G_::LD;
    static constexpr int SPAN = G_::SPAN, RPW = G_::RPW;
    static constexpr bool HALF = G_::HALF;
    static_assert(!HALF || sizeof(T) == 2, "16-bit unit tiles need 16-bit elements");
    using UT = typename std::conditional<HALF, T, float>::type;  // K and V tiles
    static constexpr int LDU = HALF ? G_::LD16 : LD;
    static constexpr int UF = S * LDU * (int)sizeof(UT) / 4;  // floats of one
    static constexpr int LDS_FLOATS = (LAST ? 2 : 1) * UF + (LAST ? 3 : 2) * C * LD + 2 * C * LS + 2 * C;

    __device__ static void run(const BwdBufs<T> &p, const BwdDims &dm, float *lds)
    {
        const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
        const int m = dm.m, b = dm.b, n = dm.n, d = dm.d;
        const int64_t bh = blockIdx.x / m;
        const int k = blockIdx.x % m;
        const int kn = min(b, n - k * b);                                // rows of block k in memory
        const int kv = LENS ? min(b, live_rows(dm, bh) - k * b) : kn;  // real keys (and query rows); <= 0: none
        const int64_t Np = (int64_t)m * b, toff = bh * n * d, soff = bh * Np * D, coff = bh * Np;
        const int64_t xoff = bh * Np * d;     // the forward's states: rows of d elements
        const int64_t row0 = (int64_t)k * b;  // first row of block k
        // whole-unit tiles (rows i): Kbar, Vbar (LAST)
        UT *Kb = reinterpret_cast<UT *>(lds), *Vb = Kb + S * LDU;
        // chunk tiles (rows j of the chunk): alpha_R, d alpha_L, dY (LAST), R, dR then dZ s / c_R
        float *aR = lds + (LAST ? 2 : 1) * UF, *dA = aR + C * LD, *dYt = dA + C * LD;
        float *Rm = dA + (LAST ? 2 : 1) * C * LD, *dR = Rm + C * LS;
        float *cR = dR + C * LS, *dcL = cR + C;

        load_unit<T, NTH, S, D, LDU, HALF>(Kb, kv, d, [&](int i) { return p.k + toff + (row0 + i) * d; }, tid);
        if constexpr (LAST)
            load_unit<T, NTH, S, D, LDU, HALF>(Vb, kv, d, [&](int i) { return p.v + toff + (row0 + i) * d; }, tid);
        Acc<W, S, D> dK, dV;  // sums over all rows j
        dK.zero();
        if constexpr (LAST) dV.zero();

        for (int ch = 0; ch < G_::NCH; ++ch) {
            const int j0 = ch * C;
            const int jb = min(max(b - j0, 0), C), jq = min(max(kv - j0, 0), C);  // live rows; rows of Q (t = 1)
            const int jn = min(max(kn - j0, 0), C);                                // rows of dq in memory (t = 1)
            if constexpr (FIRST) {
                load_tile<T, NTH, C, D, LD>(aR, jq, d, [&](int jj) { return p.q + toff + (row0 + j0 + jj) * d; }, tid);
            } else {
                load_tile<T, NTH, C, D, LD>(aR, jb, d, [&](int jj) { return p.aR + xoff + (row0 + j0 + jj) * d; },
                                         tid);
            }
            load_tile<float, NTH, C, D, LD>(
                dA, jb, d, [&](int jj) { return p.daL + soff + ((int64_t)(j0 + jj) * m + k) * D; }, tid);
            if constexpr (LAST)
                load_tile<float, NTH, C, D, LD>(
                    dYt, jb, d, [&](int jj) { return p.dY + soff + ((int64_t)(j0 + jj) * m + k) * D; }, tid);
            for (int jj = tid; jj < C; jj += NTH) {
                cR[jj] = (FIRST || jj >= jb) ? 1.f : p.cR[coff + (int64_t)(j0 + jj) * m + k];
                dcL[jj] = jj < jb ? p.dcL[coff + (int64_t)(j0 + jj) * m + k] : 0.f;
            }
            __syncthreads();

            // unnormalised scores <alpha_R[j], Kbar[i]>;  dR = d alpha_L Kbar^T (+ dY Vbar^T)
            gemm<W, C, S, D>(wave, lane, to_lds<LS>(Rm), pair<false, true, LD, LDU>(aR, Kb));
            if constexpr (LAST) {
                gemm<W, C, S, D>(wave, lane, to_lds<LS>(dR), pair<false, true, LD, LDU>(dA, Kb),
                                 pair<false, true, LD, LDU>(dYt, Vb));
            } else {
                gemm<W, C, S, D>(wave, lane, to_lds<LS>(dR), pair<false, true, LD, LDU>(dA, Kb));
            }
            __syncthreads();
            // per row j (RPW rows per wave instruction, SPAN lanes and CPL keys i per
            // lane for each): R, then dZ scaled by s / c_R[j] in place of dR
            for (int base = wave * RPW; base < C; base += W * RPW) {
                const int jj = base + lane / SPAN, col = lane % SPAN;
                const bool live = jj < jb && (!LENS || kv > 0);  // a block of padding only has R = 0
                float *rr = Rm + jj * LS, *dr = dR + jj * LS;
                const float sc = (!LENS || live) ? dm.s / cR[jj] : 0.f;  // c_R = 1 past the rows j < b
                float z[CPL], mx = -INFINITY;
#pragma unroll
                for (int u = 0; u < CPL; ++u) {
                    const int i = col + 64 * u;
                    z[u] = live && i < kv ? sc * rr[i] : -INFINITY;
                    mx = max_nan(mx, z[u]);
                }
                mx = group_max<SPAN>(mx);
                if (!live) mx = 0.f;  // rows past b: every term below is zero
                float e[CPL], sum = 0.f;
#pragma unroll
                for (int u = 0; u < CPL; ++u) {
                    e[u] = live && col + 64 * u < kv ? __expf(z[u] - mx) : 0.f;
                    sum += e[u];
                }
                sum = group_sum<SPAN>(sum);
                const float lsum = live ? __logf(sum) : 0.f, inv = live ? 1.f / sum : 0.f;
                float r[CPL], logr[CPL], g[CPL], dot = 0.f;
#pragma unroll
                for (int u = 0; u < CPL; ++u) {
                    const int i = col + 64 * u;
                    const bool on = live && i < kv;
                    r[u] = e[u] * inv;
                    logr[u] = on ? z[u] - mx - lsum : 0.f;
                    g[u] = on ? dr[i] + dcL[jj] * (logr[u] + 1.f) : 0.f;
                    dot += r[u] * g[u];
                }
                dot = group_sum<SPAN>(dot);
                float dzlog = 0.f;
#pragma unroll
                for (int u = 0; u < CPL; ++u) {
                    const int i = col + 64 * u;
                    const float dz = r[u] * (g[u] - dot);
                    dzlog += dz * logr[u];
                    if (i < S) {
                        rr[i] = r[u];
                        dr[i] = dz * sc;
                    }
                }
                dzlog = group_sum<SPAN>(dzlog);
                if (!FIRST && jj < jb && col == 0)  // zero for a block of padding only (read by l_bwd)
                    p.dcR[coff + row0 + j0 + jj] = (!LENS || live) ? -dzlog / cR[jj] : 0.f;
            }
            __syncthreads();

            // d alpha_R[j] = sum_i dZs[j][i] Kbar[i]: to the workspace, or at step 1 into dq
            if constexpr (FIRST) {
                const float *dQ = p.dQ + toff + (row0 + j0) * d;
                T *dq = p.dq + toff + (row0 + j0) * d;
                gemm<W, C, D, S>(
                    wave, lane,
                    [&](int jj, int e, float v) {  // rows past the length: zero
                        if (jj < (LENS ? jn : jq) && e < d)
                            dq[(int64_t)jj * d + e] =
                                static_cast<T>((!LENS || jj < jq) ? dQ[(int64_t)jj * d + e] + v : 0.f);
                    },
                    pair<false, false, LS, LDU>(dR, Kb));
            } else {
                float *daR = p.daR + soff + (row0 + j0) * D;
                gemm<W, C, D, S>(
                    wave, lane,
                    [&](int jj, int e, float v) {
                        if (jj < jb && e < d) daR[(int64_t)jj * D + e] = v;
                    },
                    pair<false, false, LS, LDU>(dR, Kb));
            }
            // dKbar[i] += sum_j R[j][i] d alpha_L[j] + dZs[j][i] alpha_R[j];  dVbar[i] += sum_j R[j][i] dY[j]
            dK.template add<C>(wave, lane, pair<true, false, LS, LD>(Rm, dA), pair<true, false, LS, LD>(dR, aR));
            if constexpr (LAST) dV.template add<C>(wave, lane, pair<true, false, LS, LD>(Rm, dYt));
            __syncthreads();  // the next chunk overwrites the chunk tiles
        }

        {
            float *dKg = p.dK + toff + row0 * d;
            T *dk = p.dk + toff + row0 * d;
            dK.store(wave, lane, [&](int i, int e, float v) {
                if (i < (LENS && FIRST ? kn : kv) && e < d) {  // at t = 1 rows past the length get zero
                    const int64_t o = (int64_t)i * d + e;
                    const float acc = (LENS && i >= kv) ? 0.f : LAST ? v : v + dKg[o];
                    if constexpr (FIRST) {
                        dk[o] = static_cast<T>(acc);
                    } else {
                        dKg[o] = acc;
                    }
                }
            });
        }
        if constexpr (LAST) {
            T *dv = p.dv + toff + row0 * d;
            dV.store(wave, lane, [&](int i, int e, float v) {
                if (i < (LENS ? kn : kv) && e < d) dv[(int64_t)i * d + e] = static_cast<T>((!LENS || i < kv) ? v : 0.f);
            });
        }
    }
};

template <typename T, int S, int D, bool LAST, bool LENS>
__global__ __launch_bounds__(64 * unit_waves(S)) void l_bwd(BwdBufs<T> p, BwdDims dm)
{
    __shared__ __attribute__((aligned(16))) float lds[LBwd<T, S, D, LAST, LENS>::LDS_FLOATS];
    LBwd<T, S, D, LAST, LENS>::run(p, dm, lds);
}

template <typename T, int S, int D, bool FIRST, bool LAST, bool LENS>
__global__ __launch_bounds__(64 * unit_waves(S)) void r_bwd(BwdBufs<T> p, BwdDims dm)
{
    __shared__ __attribute__((aligned(16))) float lds[RBwd<T, S, D, FIRST, LAST, LENS>::LDS_FLOATS];
    RBwd<T, S, D, FIRST, LAST, LENS>::run(p, dm, lds);
}

// The same kernels with registers bounded for two workgroups per CU.
template <typename T, int S, int D, bool LAST, bool LENS>
__global__ __launch_bounds__(64 * unit_waves(S)) __attribute__((amdgpu_waves_per_eu(2 * unit_waves(S) / 4))) void l_bwd2(
    BwdBufs<T> p, BwdDims dm)
{
    __shared__ __attribute__((aligned(16))) float lds[LBwd<T, S, D, LAST, LENS>::LDS_FLOATS];
    LBwd<T, S, D, LAST, LENS>::run(p, dm, lds);
}

template <typename T, int S, int D, bool FIRST, bool LAST, bool LENS>
__global__ __launch_bounds__(64 * unit_waves(S)) __attribute__((amdgpu_waves_per_eu(2 * unit_waves(S) / 4))) void r_bwd2(
    BwdBufs<T> p, BwdDims dm)
{
    __shared__ __attribute__((aligned(16))) float lds[RBwd<T, S, D, FIRST, LAST, LENS>::LDS_FLOATS];
    RBwd<T, S, D, FIRST, LAST, LENS>::run(p, dm, lds);
}

}  // namespace bwd
}  // namespace ma
