// The whole forward pass of one (batch, head, group of residue classes) in one
// workgroup, every step in a single launch.
//
// The residue classes j of a head are independent once all of K and V are
// at hand: class j's chain alpha_R[:][j] -> R[:][j][:] -> alpha_L[j] ->
// L[j] -> alpha_R[:][j] reads only the query rows l*b + j (Qbar[j]) and K,
// and at the end V (eqs. beta_r, beta_l, R_update, L_update read only these).
// A workgroup therefore takes G classes j0 .. j0+G-1 of one head and keeps
// their states in LDS through all T steps:
//
//   A[jj][k]  alpha_R[k][j0+jj] before an R half-step, alpha_L[j0+jj][k]
//             after it (the R half-step of block k reads slot (jj, k) and
//             writes it back; the L half-step of class j0+jj reads and writes
//             the slots (jj, *), so both update in place)
//   Y[jj][k]  Y[j0+jj][k] (last step; only where the tiles are ragged)
//   cR[jj][k], cL[jj][k] in fp32.
//
// With YG (full tiles only: n = m b, m and b the tile sizes), Y goes
// through the output tensor instead: Y[j][k] is stored at row k*b + j of O,
// a row of class j, and the last L half-step of class j stages its Y rows
// into the wave's staging area before it overwrites the same rows with O.
// That halves the LDS of a class, so up to twice as many classes share a
// workgroup, and K and V are streamed once per group and step.  It costs a
// round trip of Y through memory, so the host takes it only where it
// allows larger groups.
//
// Only Q, K, V and O touch global memory: K (and V) are streamed block by
// block in every R half-step, from the L2 that the other groups of the same
// head share (the grid puts the groups of a head on one XCD), and Qbar[j] is
// read in every L half-step.  The score tiles are those of the half-step
// kernels: an R half-step of block k is one 16-column tile (the G classes)
// against NB/16 tiles of keys, an L half-step of class j is the m x m tile of
// its query rows against its key blocks.  Each wave works on its own block k
// (R) or class j (L) with a staging area of its own, so waves meet only at
// the two barriers of each step.
#pragma once

#include "ma_kernels.hpp"

namespace ma {

template <typename T, int NB, int NM, int D, bool RG, bool YG> struct FusedGroup {
    static_assert(sizeof(T) == 2, "16-bit elements only");
    static_assert(!(RG && YG), "Y through O needs full tiles");
    static constexpr int W = 8, NTH = 64 * W;
    static constexpr int NTB = NB / 16, NTM = NM / 16;
    static constexpr int LDA = D + 8;                 // state rows: 16 bytes of padding
    static constexpr int LDK = Ld<T, D>::row;         // K, V and Qbar staging rows
    static constexpr int LDP = NM + 8;                // probability tile of the L half-step
    // Classes are CLS elements apart in A and Y, NM rows plus 16 bytes: the 16
    // lanes that read or write row k of 16 classes then start 16 bytes apart
    // modulo the 256 bytes of a bank row (NM * LDA elements alone are a
    // multiple of 256 bytes, which put all 16 on the same banks).  c_R and c_L
    // rows are CSF floats apart for the same reason.
    static constexpr int CLS = NM * LDA + 8, CSF = NM + 1;
    // staging: in an R half-step every wave holds Kbar[k], later Vbar[k] in
    // its place; in an L half-step each of the (at most G) busy waves holds
    // Qbar[j] and P.  The two phases are separated by barriers and share one
    // area.
    static constexpr int SW_R = NB * LDK, SW_L = NM * LDK + NM * LDP;
    __host__ __device__ static constexpr int stage_elems(int G)
    {
        return W * SW_R > (G < W ? G : W) * SW_L ? W * SW_R : (G < W ? G : W) * SW_L;
    }
    static constexpr bool NFR = NormFirst<NTB, D>::value, NFL = NormFirst<NTM, D>::value;
    static constexpr int NREG = YG ? 1 : 2;  // state regions: A, and Y unless it goes through O

    // LDS bytes for G classes per workgroup
    __host__ __device__ static constexpr int lds_bytes(int G)
    {
        return (NREG * G * CLS + stage_elems(G)) * (int)sizeof(T) + 2 * G * CSF * 4;
    }

    struct Ctx {
        T *A, *Yg, *S;        // states, Y, this wave's staging
        float *cR, *cL;       // [G][CSF]
        int m, b, n, d, G, gv, j0;
        int lane, g, c16, wave;
        float s_log2e;
        const T *qh, *kh, *vh;
        T *oh;
    };

    // Slot (jj, k) of a state region.
    __device__ static T *slot(T *base, int jj, int k) { return base + jj * CLS + k * LDA; }

    // R half-step of block k for the group (one wave).  FIRST: alpha_R[k][j] =
    // Q[k*b + j] and c_R = 1 (L^(0) = I).  FINAL: also Y.
    // kt (and vt) hold block k on entry; as soon as each is in LDS the same
    // registers take the loads of block kn (if kn < m), which land while this
    // block is computed.
    template <bool FIRST, bool FINAL>
    __device__ static void r_block(const Ctx &c, int k, int kn, TileChunks<T, NB, D, 64> &kt,
                                   TileChunks<T, NB, D, 64> &vt)
    {
        T *Ks = c.S + c.wave * SW_R, *Vs = Ks;  // Vbar[k] takes Kbar[k]'s place once alpha_L is formed
        kt.template stage<LDK>(Ks, c.lane);
        if (kn < c.m) fetch_rows(c, c.kh, kn, kt);
        const int jj = c.c16, j = c.j0 + jj;
        const bool jv = jj < c.gv;
        RowFrags<T, D> bf;  // row j of alpha_R[k]
        if constexpr (FIRST) {
            const int64_t row = (int64_t)k * c.b + j;
            bf.load(jv && row < c.n ? c.qh + row * c.d : nullptr, c.g, c.d);
        } else {
            const T *src = slot(c.A, jj, k);
#pragma unroll
            for (int cc = 0; cc < D / Mma<T>::KC; ++cc)
                bf.f[cc] = jv ? *reinterpret_cast<const typename Mma<T>::frag *>(src + cc * Mma<T>::KC + c.g * Mma<T>::KPL)
                              : typename Mma<T>::frag{};
        }
        float rs = c.s_log2e;
        if constexpr (!FIRST) {
            if (jv) rs = c.s_log2e * fast_rcp(fmaxf(c.cR[jj * CSF + k], kTiny));
        }
        const int kv = block_keys(c.b, c.n, k);  // keys >= kv: padding, masked (omega)
        f32x4 sc[NTB];                            // lane holds S'[i = 16t + 4g + q][j]
#pragma unroll
        for (int t = 0; t < NTB; ++t) gemm_scores_rt<T, D, 1>(Ks + (16 * t + c.c16) * LDK, &bf, &sc[t], c.g);
        const float nb = -tiles_max<NTB, RG>(sc, kv, c.g) * rs;
        float sum = 0.f, t2 = 0.f;
#pragma unroll
        for (int t = 0; t < NTB; ++t) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const float u = __builtin_fmaf(sc[t][q], rs, nb);
                float e = __builtin_amdgcn_exp2f(u);
                if (RG && 16 * t + 4 * c.g + q >= kv) e = 0.f;
                const bool first = t == 0 && q == 0;  // the sums start at their first term
                sum = first ? e : sum + e;
                t2 = first ? e * u : __builtin_fmaf(e, u, t2);
                sc[t][q] = e;
            }
        }
        sum = lanegroup_sum(sum);
        t2 = lanegroup_sum(t2);
        float inv = fast_rcp(sum);
        if (c.g == 0 && jv) c.cL[jj * CSF + k] = kLn2 * (t2 * inv - __builtin_amdgcn_logf(sum));
        if constexpr (NFR) {
#pragma unroll
            for (int t = 0; t < NTB; ++t) sc[t] *= inv;
            inv = 1.0f;
        }
        ProbFrags<T, NTB> pf;
        pf.pack(sc);
        // keep the compiler from hoisting the operand reads of the products
        // above this point (their registers would add to the scores' and the
        // prefetched blocks')
        asm volatile("" ::: "memory");
        f32x4 out[D / 16];
#pragma unroll
        for (int vt = 0; vt < D / 16; ++vt) out[vt] = gemm_aggregate<T, NTB>(Ks, LDK, 16 * vt, pf, c.lane) * inv;
        store_row_lds<T, D>(jv ? slot(c.A, jj, k) : nullptr, out, c.lane);  // alpha_L[j][k] over alpha_R[k][j]
        if constexpr (FINAL) {
            vt.template stage<LDK>(Vs, c.lane);
            if (kn < c.m) fetch_rows(c, c.vh, kn, vt);
            asm volatile("" ::: "memory");
#pragma unroll
            for (int q = 0; q < D / 16; ++q) out[q] = gemm_aggregate<T, NTB>(Vs, LDK, 16 * q, pf, c.lane) * inv;
            if constexpr (YG)  // Y[j][k] at row k*b + j of O
                store_row<T, D>(jv ? c.oh + ((int64_t)k * c.b + j) * c.d : nullptr, out, 1.0f, c.lane, c.d);
            else
                store_row_lds<T, D>(jv ? slot(c.Yg, jj, k) : nullptr, out, c.lane);  // Y[j][k]
        }
    }

    // Rows k*b + i < n of block k of K or V (base kh or vh) into registers, zero beyond.
    __device__ static void fetch_rows(const Ctx &c, const T *base, int k, TileChunks<T, NB, D, 64> &t)
    {
        const int kv = block_keys(c.b, c.n, k);
        const T *blk = base + (int64_t)k * c.b * c.d;
        const int d = c.d;
        t.fetch([=](int r) { return blk + (int64_t)r * d; }, kv, c.lane, d);
    }

    template <bool FIRST, bool FINAL> __device__ static void r_phase(const Ctx &c)
    {
        TileChunks<T, NB, D, 64> kt, vt;
        int k = c.wave;
        if (k < c.m) {
            fetch_rows(c, c.kh, k, kt);
            if constexpr (FINAL) fetch_rows(c, c.vh, k, vt);
        }
        for (; k < c.m; k += W) r_block<FIRST, FINAL>(c, k, k + W, kt, vt);
    }

    // Scores and softmax over k of class j0 + jj for the query rows
    // l = 16r + c16 of row tile r (B fragments bf): lane holds
    // Z[k = 16t + 4g + q][l] (log2 units) in sc[t]; on return sc holds
    // exp2(Z - max), and the result is 1 / row sum (0 for rows l >= m).
    __device__ static float l_row_scores(const Ctx &c, int jj, int r, const RowFrags<T, D> &bf, f32x4 *sc)
    {
        const T *Aj = slot(c.A, jj, 0);
#pragma unroll
        for (int t = 0; t < NTM; ++t) {
            f32x4 acc;
            gemm_scores_rt<T, D, 1>(Aj + (16 * t + c.c16) * LDA, &bf, &acc, c.g);
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                const int kk = 16 * t + 4 * c.g + q;
                const float bias = (!RG || kk < c.m) ? c.cL[jj * CSF + kk] * kLog2e : 0.f;
                sc[t][q] = __builtin_fmaf(acc[q], c.s_log2e, -bias);
            }
        }
        const float mx = tiles_max<NTM, RG>(sc, c.m, c.g);
        float sum = 0.f;
#pragma unroll
        for (int t = 0; t < NTM; ++t) {
#pragma unroll
            for (int q = 0; q < 4; ++q) {
                float e = __builtin_amdgcn_exp2f(sc[t][q] - mx);
                if (RG && 16 * t + 4 * c.g + q >= c.m) e = 0.f;
                sum = (t == 0 && q == 0) ? e : sum + e;
                sc[t][q] = e;
            }
        }
        sum = lanegroup_sum(sum);
        return 16 * r + c.c16 < c.m ? fast_rcp(sum) : 0.f;  // padded query rows carry no weight
    }

    // The rows l*b + j < n of class j of a [n][d] tensor (Qbar[j] of q; with
    // Y through O, Y[j] of out) into registers, zero beyond.
    __device__ static void fetch_class(const Ctx &c, const T *base, int j, TileChunks<T, NM, D, 64> &qt)
    {
        const int ml = (c.n - j + c.b - 1) / c.b;
        const int b = c.b, d = c.d;
        qt.fetch([=](int l) { return base + ((int64_t)l * b + j) * d; }, ml, c.lane, d);
    }
    __device__ static void fetch_qbar(const Ctx &c, int j, TileChunks<T, NM, D, 64> &qt) { fetch_class(c, c.qh, j, qt); }

    // L half-step of class j0 + jj (one wave): alpha_R[:][j] and c_R[:][j]
    // over the slots (jj, *).  qt holds Qbar[j] on entry; once it is in LDS
    // the same registers take the loads of class jn (if jn < gv).
    __device__ static void l_class(const Ctx &c, int jj, int jn, TileChunks<T, NM, D, 64> &qt)
    {
        T *Qs = c.S + c.wave * SW_L, *Ps = Qs + NM * LDK;
        qt.template stage<LDK>(Qs, c.lane);
        if (jn < c.gv) fetch_qbar(c, c.j0 + jn, qt);
        // P[l][k] = L[j][k][l], row-major (k contiguous), one row tile at a time
#pragma unroll 1
        for (int r = 0; r < NTM; ++r) {
            RowFrags<T, D> bf;  // Qbar[j][l] for l = 16r + c16
#pragma unroll
            for (int cc = 0; cc < D / Mma<T>::KC; ++cc)
                bf.f[cc] = *reinterpret_cast<const typename Mma<T>::frag *>(Qs + (16 * r + c.c16) * LDK +
                                                                            cc * Mma<T>::KC + c.g * Mma<T>::KPL);
            f32x4 sc[NTM];
            const float inv = l_row_scores(c, jj, r, bf, sc);
#pragma unroll
            for (int t = 0; t < NTM; ++t) store4<T>(Ps + (16 * r + c.c16) * LDP + 16 * t + 4 * c.g, sc[t] * inv);
        }
        // columns k: c_R[k][j] = sum_l L[j][k][l], alpha_R[k][j] = sum_l L[j][k][l] Qbar[j][l]
#pragma unroll 1
        for (int kt = 0; kt < NTM; ++kt) {
            const int k = 16 * kt + c.c16;
            ProbFrags<T, NTM> pf;
            pf.gather(Ps, LDP, 16 * kt, c.lane);
            const f32x4 cs = gemm_colsum<T, NTM>(pf);
            if (c.g == 0 && k < c.m) c.cR[jj * CSF + k] = cs[0];
            f32x4 out[D / 16];
#pragma unroll
            for (int vt = 0; vt < D / 16; ++vt) out[vt] = gemm_aggregate<T, NTM>(Qs, LDK, 16 * vt, pf, c.lane);
            store_row_lds<T, D>(k < c.m ? slot(c.A, jj, k) : nullptr, out, c.lane);
        }
    }

    __device__ static void l_phase(const Ctx &c)
    {
        TileChunks<T, NM, D, 64> qt;
        int jj = c.wave;
        if (jj < c.gv) fetch_qbar(c, c.j0 + jj, qt);
        for (; jj < c.gv; jj += W) l_class(c, jj, jj + W, qt);
    }

    // Last L half-step of class j0 + jj with O[l*b + j] = sum_k L[j][k][l] Y[j][k].
    __device__ static void apply_class(const Ctx &c, int jj)
    {
        const int j = c.j0 + jj;
        const T *Yj;
        int ldy;
        if constexpr (YG) {  // Y[j] from the rows of O that this class is about to overwrite
            T *Ys = c.S + c.wave * SW_L;
            TileChunks<T, NM, D, 64> yt;
            fetch_class(c, c.oh, j, yt);
            yt.template stage<LDK>(Ys, c.lane);  // (a wave's LDS accesses take effect in order)
            Yj = Ys;
            ldy = LDK;
        } else {
            Yj = slot(c.Yg, jj, 0);
            ldy = LDA;
        }
        RowFrags<T, D> bf;
        {
            const int64_t row = (int64_t)c.c16 * c.b + j;
            bf.load(row < c.n ? c.qh + row * c.d : nullptr, c.g, c.d);
        }
#pragma unroll 1
        for (int r = 0; r < NTM; ++r) {
            f32x4 sc[NTM];
            float inv = l_row_scores(c, jj, r, bf, sc);
            if (r + 1 < NTM) {  // the next row tile's query rows, while this one is finished
                const int64_t row = (int64_t)(16 * (r + 1) + c.c16) * c.b + j;
                bf.load(row < c.n ? c.qh + row * c.d : nullptr, c.g, c.d);
            }
            if constexpr (NFL) {
#pragma unroll
                for (int t = 0; t < NTM; ++t) sc[t] *= inv;
                inv = 1.0f;
            }
            ProbFrags<T, NTM> pf;
            pf.pack(sc);
            f32x4 o[D / 16];
#pragma unroll
            for (int vt = 0; vt < D / 16; ++vt) o[vt] = gemm_aggregate<T, NTM>(Yj, ldy, 16 * vt, pf, c.lane);
            const int64_t row = (int64_t)(16 * r + c.c16) * c.b + j;
            store_row<T, D>(row < c.n ? c.oh + row * c.d : nullptr, o, inv, c.lane, c.d);
        }
    }

    // Units u = blockIdx.x, blockIdx.x + gridDim.x, ... < units; unit u is
    // (head perm(u) / groups, group perm(u) % groups).
    __device__ static void run(const Bufs<T> &p, const HeadDims &hd, int G, int groups, int64_t units, int xcd_perm,
                               int T_, char *lds)
    {
        Ctx c;
        c.m = hd.m;
        c.b = hd.b;
        c.n = hd.n;
        c.d = hd.d;
        c.G = G;
        c.s_log2e = hd.s_log2e;
        const int tid = threadIdx.x;
        c.lane = tid & 63;
        c.wave = tid >> 6;
        c.g = c.lane >> 4;
        c.c16 = c.lane & 15;
        c.A = reinterpret_cast<T *>(lds);
        c.Yg = YG ? nullptr : c.A + G * CLS;
        c.S = c.A + NREG * G * CLS;
        c.cR = reinterpret_cast<float *>(c.S + stage_elems(G));
        c.cL = c.cR + G * CSF;
        // rows k >= m of the state regions are never written: zero them once
        // (they meet zero probabilities in the products, and 0 * NaN is NaN)
        if (NM > c.m) {
            for (int idx = tid; idx < NREG * G * (NM - c.m) * (D / 8); idx += NTH) {
                const int col = (idx % (D / 8)) * 8, rest = idx / (D / 8);
                const int k = c.m + rest % (NM - c.m), jr = rest / (NM - c.m);  // jr < NREG G: region jr / G
                T *base = jr < G ? c.A : c.Yg;
                *reinterpret_cast<u32x4 *>(slot(base, jr % G, k) + col) = u32x4{0u, 0u, 0u, 0u};
            }
            __syncthreads();
        }
        for (int64_t u = blockIdx.x; u < units; u += gridDim.x) {
            // the groups of one head on one XCD (workgroup i runs on XCD i % 8
            // when the grid is a multiple of 8): a placement, not a requirement
            int64_t v = u;
            if (xcd_perm) v = (u % 8) * (units / 8) + u / 8;
            const int64_t bh = v / groups;
            const int grp = (int)(v % groups);
            c.j0 = grp * G;
            c.gv = min(G, c.b - c.j0);
            const int64_t hoff = bh * (int64_t)c.n * c.d;
            c.qh = p.q + hoff;
            c.kh = p.k + hoff;
            c.vh = p.v + hoff;
            c.oh = p.out + hoff;
            for (int t = 1; t <= T_; ++t) {
                const bool first = t == 1, last = t == T_;
                if (first && last)
                    r_phase<true, true>(c);
                else if (first)
                    r_phase<true, false>(c);
                else if (last)
                    r_phase<false, true>(c);
                else
                    r_phase<false, false>(c);
                __syncthreads();  // alpha_L, c_L (and Y) of the group are complete
                if (last) break;
                l_phase(c);
                __syncthreads();  // alpha_R, c_R complete
            }
            for (int jj = c.wave; jj < c.gv; jj += W) apply_class(c, jj);
            __syncthreads();  // the next unit overwrites the states
        }
    }
};

template <typename T, int NB, int NM, int D, bool RG, bool YG>
__global__ __launch_bounds__(512) void monarch_fused_group(Bufs<T> p, HeadDims hd, int G, int groups, int64_t units,
                                                           int xcd_perm, int T_)
{
    extern __shared__ __attribute__((aligned(16))) char lds_dyn[];
    FusedGroup<T, NB, NM, D, RG, YG>::run(p, hd, G, groups, units, xcd_perm, T_, lds_dyn);
}

}  // namespace ma
