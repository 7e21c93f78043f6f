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
// Every unit keeps its matrices in fp32 LDS tiles and runs every product on
// v_mfma_f32_16x16x4f32.  The gradients of the states and the dQ, dK
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
    const T *aR, *aL, *Y;       // states of the step being undone ([m][b][D], [b][m][D], [b][m][D])
    const float *cR, *cL;       // c_R [b][m] (j-major), c_L [m][b] (k-major), as the forward writes them
    float *dQ, *dK;             // fp32 accumulators [B*H][n][d]
    T *dq, *dk, *dv;            // results [B*H][n][d]
    float *daL, *dcL, *dY;      // [b][m][D], [b][m], [b][m][D]: written by l_bwd, read by r_bwd of the step
    float *daR, *dcR;           // [m][b][D], [m][b]: written by r_bwd of step t, read by l_bwd of step t-1
};

struct BwdDims {
    int m, b, n, d;  // as in the forward; here m, b <= 64 and d <= 64 (states of width 64)
    float s;         // 1/sqrt(d)
};

namespace bwd {

constexpr int kD = 64;   // row width of the states (the forward's tile width for d <= 64)
constexpr int kLd = 84;  // row stride (floats) of the LDS tiles: 16-byte rows, both access orders conflict-free

// Waves per workgroup for tiles of S rows: one 16 x 16 output tile of an
// S x S product per wave at S = 64.
template <int S> struct Waves {
    static constexpr int value = S / 4;
};

// Reductions over the 64 lanes with no LDS round trip: DPP within rows of 16
// lanes (xor 1, xor 2, then mirrors of 8 and 16 lanes), then the permlane
// swaps across rows.  Every lane ends with the same value.
template <int CTRL> __device__ inline float dpp(float x)
{
    return __int_as_float(__builtin_amdgcn_update_dpp(0, __float_as_int(x), CTRL, 0xf, 0xf, false));
}
constexpr int kQuadXor1 = 0xB1, kQuadXor2 = 0x4E, kRowHalfMirror = 0x141, kRowMirror = 0x140;

__device__ inline float wave_sum(float x)
{
    x += dpp<kQuadXor1>(x);
    x += dpp<kQuadXor2>(x);
    x += dpp<kRowHalfMirror>(x);
    x += dpp<kRowMirror>(x);
    x = wave_xor_sum<16>(x);
    return wave_xor_sum<32>(x);
}

__device__ inline float wave_max(float x)
{
    x = fmaxf(x, dpp<kQuadXor1>(x));
    x = fmaxf(x, dpp<kQuadXor2>(x));
    x = fmaxf(x, dpp<kRowHalfMirror>(x));
    x = fmaxf(x, dpp<kRowMirror>(x));
    x = wave_xor_max<16>(x);
    return wave_xor_max<32>(x);
}

// Operands of a product, as LDS tiles (row stride kLd):
//   A(r, k) = TA ? A[k][r] : A[r][k],   B(k, n) = TB ? B[n][k] : B[k][n].
// MFMA step s of a 16-long chunk k0 hands lane group g = lane/16 the index
// k0 + 4g + s, so a lane reads four consecutive k at once: one 16-byte read
// where k is contiguous (A as stored, B transposed), four conflict-free
// scalar reads otherwise.  The contraction length is a compile-time constant:
// the loop unrolls, every read is the lane's base address plus an immediate
// offset, and all reads can be issued ahead of the MFMAs.
template <bool TA, bool TB> struct Pair {
    const float *A, *B;

    // acc += sum_{k < K} A(r, k) B(k, n)
    template <int K> __device__ void accumulate(f32x4 &acc, int r, int n, int g) const
    {
        const float *pa = TA ? A + 4 * g * kLd + r : A + r * kLd + 4 * g;
        const float *pb = TB ? B + n * kLd + 4 * g : B + 4 * g * kLd + n;
#pragma unroll
        for (int k0 = 0; k0 < K; k0 += 16) {
            float a[4], b[4];
            if constexpr (TA) {
#pragma unroll
                for (int s = 0; s < 4; ++s) a[s] = pa[(k0 + s) * kLd];
            } else {
                const f32x4 v = *reinterpret_cast<const f32x4 *>(pa + k0);
#pragma unroll
                for (int s = 0; s < 4; ++s) a[s] = v[s];
            }
            if constexpr (TB) {
                const f32x4 v = *reinterpret_cast<const f32x4 *>(pb + k0);
#pragma unroll
                for (int s = 0; s < 4; ++s) b[s] = v[s];
            } else {
#pragma unroll
                for (int s = 0; s < 4; ++s) b[s] = pb[(k0 + s) * kLd];
            }
#pragma unroll
            for (int s = 0; s < 4; ++s) acc = __builtin_amdgcn_mfma_f32_16x16x4f32(a[s], b[s], acc, 0, 0, 0);
        }
    }
};

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

template <bool TA, bool TB> __device__ inline Pair<TA, TB> pair(const float *A, const float *B)
{
    return Pair<TA, TB>{A, B};
}

__device__ inline auto to_lds(float *t)
{
    return [t](int r, int c, float v) { t[r * kLd + c] = v; };
}

// Rows r < R and columns c < C (compile-time extents, C <= 64 a multiple of
// 16) of an LDS tile from a row-major global matrix of element type E whose
// row r starts at src(r) (16-byte aligned): element (r, c) is read while
// r < nr and c < nc (nc a multiple of 16 bytes' worth of elements), zero
// elsewhere.  One 16-byte global read per chunk.
template <typename E, int NTH, int R, int C, typename Src>
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
            *reinterpret_cast<f32x4 *>(dst + r * kLd + c + i) = f32x4{v[i], v[i + 1], v[i + 2], v[i + 3]};
    }
}

// ---------------------------------------------------------------------------------------
// The L update of class j of step t undone (LAST: t = T, the update that also
// produced O).  S: rows of the tiles (16, 32 or 64, >= m).
// ---------------------------------------------------------------------------------------
template <typename T, int S, bool LAST> struct LBwd {
    static constexpr int W = Waves<S>::value, NTH = 64 * W;
    static constexpr int LDS_FLOATS = 6 * S * kLd + 2 * S;

    __device__ static void run(const BwdBufs<T> &p, const BwdDims &dm, float *lds)
    {
        const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
        const int m = dm.m, b = dm.b, n = dm.n, d = dm.d;
        const int64_t bh = blockIdx.x / b;
        const int j = blockIdx.x % b;
        const int ml = (n - j + b - 1) / b;  // rows l with l*b + j < n
        const int64_t Np = (int64_t)m * b, toff = bh * n * d, soff = bh * Np * kD, coff = bh * Np;
        float *Qb = lds, *aL = Qb + S * kLd, *Lm = aL + S * kLd, *dL = Lm + S * kLd, *X = dL + S * kLd,
              *G = X + S * kLd;
        float *cL = G + S * kLd, *dcR = cL + S;

        load_tile<T, NTH, S, kD>(Qb, ml, d, [&](int l) { return p.q + toff + ((int64_t)l * b + j) * d; }, tid);
        load_tile<T, NTH, S, kD>(aL, m, d, [&](int k) { return p.aL + soff + ((int64_t)j * m + k) * kD; }, tid);
        if constexpr (LAST) {
            load_tile<T, NTH, S, kD>(X, m, d, [&](int k) { return p.Y + soff + ((int64_t)j * m + k) * kD; }, tid);
            load_tile<T, NTH, S, kD>(G, ml, d, [&](int l) { return p.dout + toff + ((int64_t)l * b + j) * d; }, tid);
        } else {
            load_tile<float, NTH, S, kD>(X, m, d, [&](int k) { return p.daR + soff + ((int64_t)k * b + j) * kD; }, tid);
        }
        for (int k = tid; k < S; k += NTH) {
            cL[k] = k < m ? p.cL[coff + (int64_t)k * b + j] : 0.f;
            dcR[k] = (!LAST && k < m) ? p.dcR[coff + (int64_t)k * b + j] : 0.f;
        }
        __syncthreads();

        // unnormalised scores <Qbar[l], alpha_L[k]>
        gemm<W, S, S, kD>(wave, lane, to_lds(Lm), pair<false, true>(Qb, aL));
        __syncthreads();
        // L[l][k] = softmax_k (s score - c_L[k]): one wave per row l, lane k
        for (int l = wave; l < S; l += W) {
            const int k = lane;
            if (l >= m) {
                if (k < S) Lm[l * kLd + k] = 0.f;
                continue;
            }
            const float z = k < m ? dm.s * Lm[l * kLd + k] - cL[k] : -INFINITY;
            const float mx = wave_max(z);
            const float e = k < m ? __expf(z - mx) : 0.f;
            const float sum = wave_sum(e);
            if (k < S) Lm[l * kLd + k] = e / sum;
        }
        __syncthreads();

        if constexpr (LAST) {
            // dL = dO Y^T;  dY = L^T dO (to the workspace, read by r_bwd of this step)
            gemm<W, S, S, kD>(wave, lane, to_lds(dL), pair<false, true>(G, X));
            float *dY = p.dY + soff + (int64_t)j * m * kD;
            gemm<W, S, kD, S>(
                wave, lane,
                [&](int k, int e, float v) {
                    if (k < m && e < d) dY[(int64_t)k * kD + e] = v;
                },
                pair<true, false>(Lm, G));
        } else {
            // dL = Qbar d alpha_R'^T (+ d c_R' below);  G = L d alpha_R' (the alpha_R' term of dQbar)
            gemm<W, S, S, kD>(wave, lane, to_lds(dL), pair<false, true>(Qb, X));
            gemm<W, S, kD, S>(wave, lane, to_lds(G), pair<false, false>(Lm, X));
        }
        __syncthreads();
        // dW = s L (dL - <L, dL>), in place of dL
        for (int l = wave; l < S; l += W) {
            const int k = lane;
            const float pk = k < S ? Lm[l * kLd + k] : 0.f;
            const float w = k < S ? dL[l * kLd + k] + dcR[k] : 0.f;
            const float dot = wave_sum(pk * w);
            if (k < S) dL[l * kLd + k] = dm.s * pk * (w - dot);
        }
        __syncthreads();

        // dQ rows l*b + j: dW alpha_L (+ L d alpha_R')
        float *dQ = p.dQ + toff + (int64_t)j * d;
        gemm<W, S, kD, S>(
            wave, lane,
            [&](int l, int e, float v) {
                if (l < ml && e < d) {
                    float *o = dQ + (int64_t)l * b * d + e;
                    if constexpr (LAST) {
                        *o = v;
                    } else {
                        *o += v + G[l * kLd + e];
                    }
                }
            },
            pair<false, false>(dL, aL));
        // d alpha_L[k] = dW^T Qbar
        float *daL = p.daL + soff + (int64_t)j * m * kD;
        gemm<W, S, kD, S>(
            wave, lane,
            [&](int k, int e, float v) {
                if (k < m && e < d) daL[(int64_t)k * kD + e] = v;
            },
            pair<true, false>(dL, Qb));
        // d c_L[k] = -(1/s) sum_l dW[l][k]
        for (int k = tid; k < m; k += NTH) {
            float cs = 0.f;
            for (int l = 0; l < S; ++l) cs += dL[l * kLd + k];
            p.dcL[coff + (int64_t)j * m + k] = -cs / dm.s;
        }
    }
};

// ---------------------------------------------------------------------------------------
// The R update of block k of step t undone (FIRST: t = 1, LAST: t = T).
// S: rows of the tiles (16, 32 or 64, >= b).
// ---------------------------------------------------------------------------------------
template <typename T, int S, bool FIRST, bool LAST> struct RBwd {
    static constexpr int W = Waves<S>::value, NTH = 64 * W;
    static constexpr int TILES = LAST ? 7 : 5;
    static constexpr int LDS_FLOATS = TILES * S * kLd + 2 * S;

    __device__ static void run(const BwdBufs<T> &p, const BwdDims &dm, float *lds)
    {
        const int tid = threadIdx.x, lane = tid & 63, wave = tid >> 6;
        const int m = dm.m, b = dm.b, n = dm.n, d = dm.d;
        const int64_t bh = blockIdx.x / m;
        const int k = blockIdx.x % m;
        const int kv = min(b, n - k * b);  // real keys (and query rows) of block k
        const int64_t Np = (int64_t)m * b, toff = bh * n * d, soff = bh * Np * kD, coff = bh * Np;
        const int64_t row0 = (int64_t)k * b;  // first row of block k
        float *Kb = lds, *aR = Kb + S * kLd, *dA = aR + S * kLd, *Rm = dA + S * kLd, *dR = Rm + S * kLd;
        float *Vb = dR + S * kLd, *dYt = Vb + S * kLd;  // LAST only
        float *cR = lds + TILES * S * kLd, *dcL = cR + S;

        load_tile<T, NTH, S, kD>(Kb, kv, d, [&](int i) { return p.k + toff + (row0 + i) * d; }, tid);
        if constexpr (FIRST) {
            load_tile<T, NTH, S, kD>(aR, kv, d, [&](int jj) { return p.q + toff + (row0 + jj) * d; }, tid);
        } else {
            load_tile<T, NTH, S, kD>(aR, b, d, [&](int jj) { return p.aR + soff + (row0 + jj) * kD; }, tid);
        }
        load_tile<float, NTH, S, kD>(dA, b, d, [&](int jj) { return p.daL + soff + ((int64_t)jj * m + k) * kD; }, tid);
        if constexpr (LAST) {
            load_tile<T, NTH, S, kD>(Vb, kv, d, [&](int i) { return p.v + toff + (row0 + i) * d; }, tid);
            load_tile<float, NTH, S, kD>(dYt, b, d, [&](int jj) { return p.dY + soff + ((int64_t)jj * m + k) * kD; },
                             tid);
        }
        for (int jj = tid; jj < S; jj += NTH) {
            cR[jj] = (FIRST || jj >= b) ? 1.f : p.cR[coff + (int64_t)jj * m + k];
            dcL[jj] = jj < b ? p.dcL[coff + (int64_t)jj * m + k] : 0.f;
        }
        __syncthreads();

        // unnormalised scores <alpha_R[j], Kbar[i]>;  dR = d alpha_L Kbar^T (+ dY Vbar^T)
        gemm<W, S, S, kD>(wave, lane, to_lds(Rm), pair<false, true>(aR, Kb));
        if constexpr (LAST) {
            gemm<W, S, S, kD>(wave, lane, to_lds(dR), pair<false, true>(dA, Kb), pair<false, true>(dYt, Vb));
        } else {
            gemm<W, S, S, kD>(wave, lane, to_lds(dR), pair<false, true>(dA, Kb));
        }
        __syncthreads();
        // per row j (one wave, lane i): R, then dZ scaled by s / c_R[j] in place of dR
        for (int jj = wave; jj < S; jj += W) {
            const int i = lane;
            if (jj >= b) {
                if (i < S) Rm[jj * kLd + i] = dR[jj * kLd + i] = 0.f;
                continue;
            }
            const float sc = dm.s / cR[jj];
            const bool live = i < kv;
            const float z = live ? sc * Rm[jj * kLd + i] : -INFINITY;
            const float mx = wave_max(z);
            const float e = live ? __expf(z - mx) : 0.f;
            const float sum = wave_sum(e);
            const float r = e / sum;
            const float logr = live ? z - mx - __logf(sum) : 0.f;
            const float dr = live ? dR[jj * kLd + i] + dcL[jj] * (logr + 1.f) : 0.f;
            const float dot = wave_sum(r * dr);
            const float dz = r * (dr - dot);
            const float dzlog = wave_sum(dz * logr);
            if (i < S) {
                Rm[jj * kLd + i] = r;
                dR[jj * kLd + i] = dz * sc;
            }
            if (!FIRST && i == 0) p.dcR[coff + row0 + jj] = -dzlog / cR[jj];
        }
        __syncthreads();

        // d alpha_R[j] = sum_i dZs[j][i] Kbar[i]: to the workspace, or at step 1 into dq
        if constexpr (FIRST) {
            const float *dQ = p.dQ + toff + row0 * d;
            T *dq = p.dq + toff + row0 * d;
            gemm<W, S, kD, S>(
                wave, lane,
                [&](int jj, int e, float v) {
                    if (jj < kv && e < d) dq[(int64_t)jj * d + e] = static_cast<T>(dQ[(int64_t)jj * d + e] + v);
                },
                pair<false, false>(dR, Kb));
        } else {
            float *daR = p.daR + soff + row0 * kD;
            gemm<W, S, kD, S>(
                wave, lane,
                [&](int jj, int e, float v) {
                    if (jj < b && e < d) daR[(int64_t)jj * kD + e] = v;
                },
                pair<false, false>(dR, Kb));
        }
        // dKbar[i] += sum_j R[j][i] d alpha_L[j] + sum_j dZs[j][i] alpha_R[j]
        {
            float *dK = p.dK + toff + row0 * d;
            T *dk = p.dk + toff + row0 * d;
            gemm<W, S, kD, S>(
                wave, lane,
                [&](int i, int e, float v) {
                    if (i < kv && e < d) {
                        const int64_t o = (int64_t)i * d + e;
                        const float acc = LAST ? v : v + dK[o];
                        if constexpr (FIRST) {
                            dk[o] = static_cast<T>(acc);
                        } else {
                            dK[o] = acc;
                        }
                    }
                },
                pair<true, false>(Rm, dA), pair<true, false>(dR, aR));
        }
        // dVbar[i] = sum_j R[j][i] dY[j]
        if constexpr (LAST) {
            T *dv = p.dv + toff + row0 * d;
            gemm<W, S, kD, S>(
                wave, lane,
                [&](int i, int e, float v) {
                    if (i < kv && e < d) dv[(int64_t)i * d + e] = static_cast<T>(v);
                },
                pair<true, false>(Rm, dYt));
        }
    }
};

template <typename T, int S, bool LAST>
__global__ __launch_bounds__(64 * Waves<S>::value) void l_bwd(BwdBufs<T> p, BwdDims dm)
{
    __shared__ __attribute__((aligned(16))) float lds[LBwd<T, S, LAST>::LDS_FLOATS];
    LBwd<T, S, LAST>::run(p, dm, lds);
}

template <typename T, int S, bool FIRST, bool LAST>
__global__ __launch_bounds__(64 * Waves<S>::value) void r_bwd(BwdBufs<T> p, BwdDims dm)
{
    __shared__ __attribute__((aligned(16))) float lds[RBwd<T, S, FIRST, LAST>::LDS_FLOATS];
    RBwd<T, S, FIRST, LAST>::run(p, dm, lds);
}

}  // namespace bwd
}  // namespace ma
