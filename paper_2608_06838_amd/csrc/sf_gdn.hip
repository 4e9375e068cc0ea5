// sf_gdn.hip -- gfx950 forward walk of the gated delta rule (Gated DeltaNet,
// the scalar-plus-low-rank transition of Sec. 2.1):
//
//   S_t = a_t (I - beta_t k_t k_t^T) S_{t-1} + beta_t k_t v_t^T,   o_t = S_t^T q_t,
//
// with S in R^{Dk x Dv} (the transpose of the paper's S) and a_t = exp(g_t).
//
// Chunkwise form (per chunk of C tokens, S the state entering it, b_t the
// chunk-local inclusive cumulative log-decay, gamma_t = e^{b_t}):
//   A[t][s]  = beta_t e^{b_t - b_s} (k_t . k_s)      for s < t   (strictly lower)
//   (I + A) [W | Ubar] = [diag(beta gamma) K | diag(beta) V]     (T = (I + A)^{-1} by blocks, then T R)
//   U        = Ubar - W S                                          (the corrected values, V^new)
//   O        = diag(gamma) Q S + (Q K^T o Gamma) U,  Gamma[t][s] = e^{b_t - b_s} (s <= t)
//   S_next   = gamma_C S + (K o e^{b_C - b})^T U
// This follows from writing u_t = beta_t (v_t - a_t S_{t-1}^T k_t), so that
// S_t = a_t S_{t-1} + k_t u_t^T is a plain gated linear recurrence in u, and
// solving the within-chunk dependence of u on the earlier u's.
//
// One workgroup walks the chunks of one (batch, head) superchunk with the state
// in registers: wave w owns the 16 state columns [16w, 16w+16) (D/16 waves).
// Per chunk: the q, k, v tiles are staged in LDS; the KK^T and QK^T scores run
// on MFMA (10 causal 16x16 tiles each); T = (I + A)^{-1} is formed in fp32 by
// 16 x 16 blocks (gdn_tinv) and [W | Ubar] = T R on MFMA (gdn_wu); U, the
// output and the state update are MFMA products whose computed operands
// (S, W, U) go in as bf16 hi/lo pairs, U straight from its accumulators (rows t,
// columns v), which two lane-row swaps make into operand fragments with the
// tokens as contraction.
//
// Superchunk parallelism (the Pre / ST / Out split of Sec. 2.2 with the delta
// rule's matrix-valued transition): the chunk map S -> gamma_C S + K~^T (Ubar - W S)
// is affine in S, so a superchunk of chunks maps S_J to S_{J+1} = M_J S_J + N_J
// with dense M_J, N_J in R^{Dk x Dk}, R^{Dk x Dv}.
//   k_gdn_walk<W_PREP>: walks the superchunk's chunks with the state [M | N]
//     (wave w owns columns [16w, 16w+16) of both; M from the identity with
//     Ubar = 0, N from zero) and writes M_J, N_J.  No outputs.
//   k_gdn_scan: S_{J+1} = M_J S_J + N_J in fp32, sequential over J, 16 state
//     columns per workgroup; writes every S_J and S_out.
//   k_gdn_walk<W_OUT>: the output walk above from S_J over superchunk J;
//   k_gdn_walk<W_STORE>: the same walk without outputs, writing the state that
//     enters every chunk (for the backward).
#include "sf_chunk.hpp"

namespace sf {

namespace {

// 16x16x16 bf16 MFMA: A lane (q, n) holds row n, k = 4q .. 4q+3; B lane (q, n)
// holds k = 4q .. 4q+3 of column n; the accumulator holds rows 4q .. 4q+3 of
// column n, the same slots as a B operand.
typedef short s4v __attribute__((ext_vector_type(4)));
__device__ __forceinline__ void mma16(f32x4 &c, s4v a, s4v b) {
    c = __builtin_amdgcn_mfma_f32_16x16x16bf16_1k(a, b, c, 0, 0, 0);
}
// hi = bf16(x), lo = bf16(x - hi), as the raw 16-bit patterns
__device__ __forceinline__ void split4(const f32x4 &x, s4v &hi, s4v &lo) {
#pragma unroll
    for (int j = 0; j < 4; ++j) {
        const __bf16 h = (__bf16)x[j];
        const __bf16 l = (__bf16)(x[j] - (float)h);
        hi[j] = __builtin_bit_cast(short, h);
        lo[j] = __builtin_bit_cast(short, l);
    }
}

// T = (I + A)^{-1} for the strictly lower 64 x 64 A = diag(rs) M with M in sA
// (pitch C + 4; rs == nullptr: A = M), into sT (fp32, pitch C + 4, zero above
// the diagonal), by 16 x 16 blocks: the four diagonal blocks by forward
// substitution in fp32 (64 threads, one column each); then level by level
// (i - j = 1, 2, 3) wave j forms T_ij = -T_ii sum_{k=j}^{i-1} A_ik T_kj on
// 16x16x16 MFMA with hi/lo operands, the inner sum staying in its
// accumulator, which is already the B operand of the T_ii product.  NT >= 256
// threads (four waves); ends with a barrier.
template <int NT>
__device__ __forceinline__ void gdn_tinv(int tid, const float *sA, float *sT, const float *rs = nullptr) {
    constexpr int LA = C + 4, LT = C + 4;
    if (tid < 64) {
        const int o = 16 * (tid >> 4), c = tid & 15;
        float x[16];
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            float acc = 0.f;
#pragma unroll
            for (int s2 = 0; s2 < r; ++s2) acc = fmaf(sA[(o + r) * LA + o + s2], x[s2], acc);
            x[r] = r == c ? 1.f : (r > c ? -(rs ? rs[o + r] : 1.f) * acc : 0.f);
        }
#pragma unroll
        for (int r = 0; r < 16; ++r) sT[(o + r) * LT + o + c] = x[r];
    }
    for (int e = tid; e < 6 * 256; e += NT) {  // blocks (0,1) (0,2) (0,3) (1,2) (1,3) (2,3)
        const int b = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
        const int bi = b < 3 ? 0 : (b < 5 ? 1 : 2), bj = b < 3 ? b + 1 : (b < 5 ? b - 1 : 3);
        sT[(16 * bi + rr) * LT + 16 * bj + cc] = 0.f;
    }
    __syncthreads();
    const int w = tid >> 6, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
#pragma unroll
    for (int d = 1; d < 4; ++d) {
        if (w < 4 - d) {  // block (i, j) = (d + w, w)
            const int i = d + w, j = w;
            f32x4 y = {0.f, 0.f, 0.f, 0.f};
            for (int k = j; k < i; ++k) {
                f32x4 av = *reinterpret_cast<const f32x4 *>(&sA[(16 * i + n16) * LA + 16 * k + 4 * q4]);
                if (rs) av *= rs[16 * i + n16];
                f32x4 tb;
#pragma unroll
                for (int u = 0; u < 4; ++u) tb[u] = sT[(16 * k + 4 * q4 + u) * LT + 16 * j + n16];
                s4v ah, al, bh, bl;
                split4(av, ah, al);
                split4(tb, bh, bl);
                mma16(y, ah, bh);
                mma16(y, ah, bl);
                mma16(y, al, bh);
            }
            const f32x4 tv = *reinterpret_cast<const f32x4 *>(&sT[(16 * i + n16) * LT + 16 * i + 4 * q4]);
            s4v th, tl, yh, yl;
            split4(tv, th, tl);
            split4(y, yh, yl);
            f32x4 t = {0.f, 0.f, 0.f, 0.f};
            mma16(t, th, yh);
            mma16(t, th, yl);
            mma16(t, tl, yh);
#pragma unroll
            for (int r = 0; r < 4; ++r) sT[(16 * i + 4 * q4 + r) * LT + 16 * j + n16] = -t[r];
        }
        __syncthreads();
    }
}

// [W | Ubar] = T [diag(beta gamma) K | diag(beta) V] on MFMA: wave w forms
// columns [16w, 16w+16) of W (and of Ubar when sU is given); T enters as a hi/lo
// pair, the scaled K and V columns too (K, V exact in bf16 times an fp32
// factor).  Results to sW / sU (fp32, pitch LDU).
template <typename T, int D, int LDN, int LDU, int SWX>
__device__ __forceinline__ void gdn_wu(int w, int lane, const LaneOff &tro, const float *sT, const T *sK, const T *sV,
                                       const float *sbeta, const float *sq, float *sW, float *sU) {
    constexpr int LT = C + 4;
    const int q4 = lane >> 4, n16 = lane & 15, c0 = 16 * w;
    f32x4 cw[4], cu[4];
#pragma unroll
    for (int tt = 0; tt < 4; ++tt) cw[tt] = cu[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
    for (int ks = 0; ks < C / 32; ++ks) {
        float fw[8], fu[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) {
            const int s2 = 32 * ks + 8 * q4 + j;
            fu[j] = sbeta[s2];
            fw[j] = sbeta[s2] * sq[s2];
        }
        frag_t<T> kh, kl, vh, vl;
        split_scaled<T, true>(ldfragTR<T, LDN, SWX>(sK, tro, 32 * ks, c0), fw, kh, kl);
        if (sU) split_scaled<T, true>(ldfragTR<T, LDN, SWX>(sV, tro, 32 * ks, c0), fu, vh, vl);
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) {
            if (32 * ks > 16 * tt + 15) continue;  // T is lower triangular
            const float *p = sT + (16 * tt + n16) * LT + 32 * ks + 8 * q4;
            const f32x4 x0 = *reinterpret_cast<const f32x4 *>(p), x1 = *reinterpret_cast<const f32x4 *>(p + 4);
            const float x[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
            frag_t<T> th, tl;
            split8<T, true>(x, th, tl);
            mma(cw[tt], th, kh);
            mma(cw[tt], th, kl);
            mma(cw[tt], tl, kh);
            if (sU) {
                mma(cu[tt], th, vh);
                mma(cu[tt], th, vl);
                mma(cu[tt], tl, vh);
            }
        }
    }
#pragma unroll
    for (int tt = 0; tt < 4; ++tt)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            sW[(16 * tt + 4 * q4 + r) * LDU + c0 + n16] = cw[tt][r];
            if (sU) sU[(16 * tt + 4 * q4 + r) * LDU + c0 + n16] = cu[tt][r];
        }
}

enum { W_OUT = 0, W_PREP = 1, W_STORE = 2 };

template <typename T, int D, int MODE>
__global__ void __launch_bounds__(64 * D / 16) k_gdn_walk(GdnArgs a) {
    constexpr bool PREP = MODE == W_PREP, OUTP = MODE == W_OUT;  // STORE: states only
    constexpr int NW = D / 16, NT = 64 * NW, NK = D / 16, NS = PREP ? 2 : 1;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr int LDA = C + 4, LDU = D + 4;  // 16-byte-odd pitches: conflict-free row-varying reads
    __shared__ __attribute__((aligned(16))) T sQ[OUTP ? C * LDN : 8];    // plain
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];               // plain, swizzled
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];               // plain
    // (Q K^T o Gamma)[t][s] hi, then lo; T = (I + A)^{-1} lives here before the P tiles
    __shared__ __attribute__((aligned(16))) T sPP[OUTP ? 2 * C * LDT : 8];
    __shared__ __attribute__((aligned(16))) float sTx[OUTP ? 4 : C * (C + 4)];
    static_assert(!OUTP || 2 * C * LDT * sizeof(T) >= C * (C + 4) * sizeof(float), "T does not fit the P tiles");
    T *sP = sPP, *sPl = sPP + (OUTP ? C * LDT : 0);
    float *sT = OUTP ? reinterpret_cast<float *>(sPP) : sTx;
    __shared__ __attribute__((aligned(16))) float sA[C * LDA];    // beta_t e^{b_t-b_s} k_t.k_s, s < t
    __shared__ __attribute__((aligned(16))) float sW[C * LDU];    // W [t][k], fp32
    __shared__ __attribute__((aligned(16))) float sU[C * LDU];    // Ubar [t][v], fp32
    __shared__ __attribute__((aligned(16))) float sb[C], sq[C], se[C], sbeta[C];

    const int tid = threadIdx.x, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c0 = 16 * w;
    // items: (b, h, J) with J < n_super (walk) or J < n_super - 1 (prep)
    const int nJ = PREP ? a.n_prep : a.n_super;
    const int item = blockIdx.x, bh = item / nJ, J = item % nJ;
    const int bb = bh / a.H, hh = bh % a.H;
    const int64_t tok0 = (int64_t)J * a.ts;
    const int64_t xo = bb * a.sx_b + hh * a.sx_h + tok0 * a.sx_l;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *V = (const T *)a.v + xo;
    T *Y = (T *)a.o + xo;
    T *VN = a.v_new ? (T *)a.v_new + xo : nullptr;
    const int64_t go = bb * a.sg_b + hh * a.sg_h + tok0 * a.sg_l;
    const float *gp = a.g + go;
    const float *bp = a.beta + go;
    const int64_t SS = (int64_t)D * D;
    const int nch = (int)((a.L - tok0 < a.ts ? a.L - tok0 : a.ts) / C);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    auto asw = [](int row) { return sizeof(T) == 2 ? 8 * ((row >> 2) & 1) : 0; };

    // S[m][16i + 4q4 + r][c0 + n16]: the walk's state starts from S_J (S_in for
    // one superchunk); the prep's M (m = 0) from I and its N (m = 1) from 0
    const float *src = a.n_super == 1 ? a.S_in + (a.S_in ? bh * SS : 0) : a.wsS + (int64_t)item * SS;
    f32x4 S[NS][NK];
#pragma unroll
    for (int i = 0; i < NK; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = 16 * i + 4 * q4 + r;
            if constexpr (PREP) {
                S[0][i][r] = row == c0 + n16 ? 1.f : 0.f;
                S[1][i][r] = 0.f;
            } else {
                S[0][i][r] = (a.n_super > 1 || a.S_in) ? src[(int64_t)row * D + c0 + n16] : 0.f;
            }
        }

    using TT = Tile<T, D, NT>;
    TT t1, t2, t3;
    float gl, bl;
    const int64_t cstep = (int64_t)C * a.sx_l;
    const uint32_t cspan = chunk_span<T, D>(a.sx_l), gspan = (uint32_t)(((C - 1) * a.sg_l + 1) * 4);
    uint32_t toff[TT::RPT];
    TT::offsets(toff, a.sx_l, tid);
    const uint32_t goff = (uint32_t)(lane * a.sg_l * 4);
    const uint32_t voff = (uint32_t)((n16 * a.sx_l + c0 + 4 * q4) * (int64_t)sizeof(T));
    const uint32_t tstep = (uint32_t)(16 * a.sx_l * (int64_t)sizeof(T));
    auto issue = [&](int c) {
        const int64_t nx = c * cstep;
        if constexpr (OUTP) t1.load_buf(buf_rsrc(Q + nx, cspan), toff, 0);
        t2.load_buf(buf_rsrc(K + nx, cspan), toff, 0);
        t3.load_buf(buf_rsrc(V + nx, cspan), toff, 0);
        gl = buf_ld<float>(buf_rsrc(gp + (int64_t)c * C * a.sg_l, gspan), goff, 0);
        bl = buf_ld<float>(buf_rsrc(bp + (int64_t)c * C * a.sg_l, gspan), goff, 0);
    };
    if (nch > 0) issue(0);

    for (int c = 0; c < nch; ++c) {
        if constexpr (MODE == W_STORE) {
            float *dst = a.wsSc + ((int64_t)bh * (a.L / C) + tok0 / C + c) * SS;
#pragma unroll
            for (int i = 0; i < NK; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) dst[(int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] = S[0][i][r];
        }
        const float b2 = wave_scan_dpp(gl * LOG2E);
        const float b63 = lane_value(b2, 63);
        const float betal = bl;
        __syncthreads();  // the previous chunk is done with every LDS tile
        if constexpr (OUTP) t1.store_swz(sQ, LDN, tid, 0);
        t2.store_swz(sK, LDN, tid, SWX);
        t3.store_swz(sV, LDN, tid, SWX);
        if (w == 0) {
            sb[lane] = b2;
            sq[lane] = fexp2(b2);
            se[lane] = fexp2(b63 - b2);
            sbeta[lane] = betal;
        }
        __syncthreads();
        if (c + 1 < nch) issue(c + 1);

        // scores on the causal tiles: k_s . k_t (A) first; k_s . q_t (P) after the
        // solve, whose T occupies the P tiles' LDS
        auto scores = [&](int i0) {
            for (int i = i0 + w; i < i0 + 10; i += NW) {
                const bool kk = i >= 10;
                int tt, st;
                tri_tile(kk ? i - 10 : i, tt, st);
                f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
                for (int ks = 0; ks < D / 32; ++ks) {
                    const frag_t<T> kf = ldfrag_swz<T, LDN, SWX>(sK, swo, 16 * st, 32 * ks);
                    const frag_t<T> xf = kk ? ldfrag_swz<T, LDN, SWX>(sK, swo, 16 * tt, 32 * ks)
                                            : ldfrag(sQ, LDN, 16 * tt, 32 * ks, lane);
                    mma(p, kf, xf);
                }
                const int t = 16 * tt + n16;
                const float bt = sb[t];
                const f32x4 bs = *reinterpret_cast<const f32x4 *>(&sb[16 * st + 4 * q4]);
                float v4[4];
                if (!kk) {
                    if constexpr (OUTP) {
#pragma unroll
                        for (int r = 0; r < 4; ++r) {
                            const int s = 16 * st + 4 * q4 + r;
                            v4[r] = s <= t ? p[r] * fexp2(bt - bs[r]) : 0.f;
                        }
                        const int o = t * LDT + ((16 * st + 4 * q4) ^ asw(t));
                        st4_split<T, true>(&sP[o], &sPl[o], v4);
                    }
                } else {
                    const float be = sbeta[t];
#pragma unroll
                    for (int r = 0; r < 4; ++r) {
                        const int s = 16 * st + 4 * q4 + r;
                        v4[r] = s < t ? be * p[r] * fexp2(bt - bs[r]) : 0.f;
                    }
                    *reinterpret_cast<f32x4 *>(&sA[t * LDA + 16 * st + 4 * q4]) = f32x4{v4[0], v4[1], v4[2], v4[3]};
                }
            }
        };
        scores(10);
        __syncthreads();
        gdn_tinv<NT>(tid, sA, sT);
        gdn_wu<T, D, LDN, LDU, SWX>(w, lane, tro, sT, sK, sV, sbeta, sq, sW, sU);
        __syncthreads();
        if constexpr (OUTP) {
            scores(0);
            // P tiles above the diagonal that the output product reads are zero
            for (int e = tid; e < (OUTP ? 512 : 0); e += NT) {
                const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
                const int row = tile ? 32 + rr : rr, col = tile ? 48 + cc : 16 + cc;
                sP[row * LDT + (col ^ asw(row))] = cvt<T>(0.f);
                sPl[row * LDT + (col ^ asw(row))] = cvt<T>(0.f);
            }
        }
        __syncthreads();

        // U[t][v] = Ubar[t][v] - sum_k W[t][k] S[k][v]  (rows t = 16tt + 4q4 + r, column v = c0 + n16);
        // the prep's M columns take Ubar = 0
        f32x4 U[NS][4];
#pragma unroll
        for (int m = 0; m < NS; ++m)
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    U[m][tt][r] = PREP && m == 0 ? 0.f : sU[(16 * tt + 4 * q4 + r) * LDU + c0 + n16];
        // O^T[v][t] = gamma_t sum_k S[k][v] Q[t][k] + sum_s U[s][v] P[t][s]
        f32x4 O[4];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) O[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            frag_t<T> fh[NS], fl[NS];
#pragma unroll
            for (int m = 0; m < NS; ++m) split_acc_plain<T, true>(S[m][2 * ks], S[m][2 * ks + 1], fh[m], fl[m]);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                // -W[t][32ks + 8q4 .. +7], split hi/lo (fp32 in LDS)
                const float *wp = &sW[(16 * tt + n16) * LDU + 32 * ks + 8 * q4];
                const f32x4 w0 = *reinterpret_cast<const f32x4 *>(wp), w1 = *reinterpret_cast<const f32x4 *>(wp + 4);
                const float wn[8] = {-w0[0], -w0[1], -w0[2], -w0[3], -w1[0], -w1[1], -w1[2], -w1[3]};
                frag_t<T> wh, wl;
                split8<T, true>(wn, wh, wl);
#pragma unroll
                for (int m = 0; m < NS; ++m) {
                    mma(U[m][tt], wh, fh[m]);
                    mma(U[m][tt], wh, fl[m]);
                    mma(U[m][tt], wl, fh[m]);
                }
                if constexpr (OUTP) mma2<T, true>(O[tt], fh[0], fl[0], ldfrag(sQ, LDN, 16 * tt, 32 * ks, lane));
            }
        }
        if constexpr (OUTP) {
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) O[tt] *= sq[16 * tt + n16];
#pragma unroll
            for (int ks = 0; ks < C / 32; ++ks) {
                frag_t<T> uh, ul;
                split_acc_plain<T, true>(U[0][2 * ks], U[0][2 * ks + 1], uh, ul);
#pragma unroll
                for (int tt = 0; tt < 4; ++tt) {
                    if (32 * ks > 16 * tt + 15) continue;
                    const int aw = asw(lane & 15);
                    const frag_t<T> ph = *reinterpret_cast<const frag_t<T> *>(sP + (16 * tt + (lane & 15)) * LDT + ((32 * ks + 8 * (lane >> 4)) ^ aw));
                    const frag_t<T> pl = *reinterpret_cast<const frag_t<T> *>(sPl + (16 * tt + (lane & 15)) * LDT + ((32 * ks + 8 * (lane >> 4)) ^ aw));
                    mma(O[tt], uh, ph);
                    mma(O[tt], uh, pl);
                    mma(O[tt], ul, ph);
                }
            }
            const rsrc_t ro = buf_rsrc(Y + c * cstep, cspan);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) st4_buf<T>(ro, voff, tt * tstep, O[tt]);
        }

        // V^new (optional): U[16tt + 4q4 + r][c0 + n16]
        if (OUTP && VN) {
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    VN[(int64_t)(c * C + 16 * tt + 4 * q4 + r) * a.sx_l + c0 + n16] = cvt<T>(U[0][tt][r]);
        }

        // S = gamma_C S + K^T (e^{b_C - b} o U)
        const float gam = fexp2(b63);
#pragma unroll
        for (int m = 0; m < NS; ++m) {
#pragma unroll
            for (int i = 0; i < NK; ++i) S[m][i] *= gam;
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int r = 0; r < 4; ++r) U[m][tt][r] *= se[16 * tt + 4 * q4 + r];
        }
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            frag_t<T> uh[NS], ul[NS];
#pragma unroll
            for (int m = 0; m < NS; ++m) split_acc_plain<T, true>(U[m][2 * ks], U[m][2 * ks + 1], uh[m], ul[m]);
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const frag_t<T> kf = ldfragTR<T, LDN, SWX>(sK, tro, 32 * ks, 16 * i);
#pragma unroll
                for (int m = 0; m < NS; ++m) mma2b<T, true>(S[m][i], kf, uh[m], ul[m]);
            }
        }
    }
    // prep: M_J, N_J; walk: S_out after the last superchunk
    if (PREP || (OUTP && J == a.n_super - 1 && !(a.scan_out && a.n_super > 1))) {
#pragma unroll
        for (int m = 0; m < NS; ++m) {
            float *dst = PREP ? (m == 0 ? a.wsM : a.wsN) + (int64_t)item * SS : a.S_out + bh * SS;
#pragma unroll
            for (int i = 0; i < NK; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) dst[(int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] = S[m][i][r];
        }
    }
}

// S_{J+1} = M_J S_J + N_J for J = 0 .. n_super - 2 in fp32, S_0 = S_in (or 0);
// writes S_J (J < n_super) to wsS; with scan_out (maps of every superchunk)
// one more step gives S_out.  Workgroup (b, h, 16-column block); thread
// row k = tid % D owns CPT consecutive columns of the block.  M_J is staged
// in LDS (row pitch D + 4 floats) with the next one prefetched in registers.
template <int D>
__global__ void __launch_bounds__(256) k_gdn_scan(GdnArgs a) {
    constexpr int NT = 256, RPT = NT / D, CPT = 16 / RPT, LDM = D + 4, MV = D * D / 4 / NT;
    __shared__ __attribute__((aligned(16))) float sM[D * LDM];
    __shared__ __attribute__((aligned(16))) float sS[D * 16];
    const int tid = threadIdx.x, k = tid % D, cg = tid / D;
    const int bh = blockIdx.x / (D / 16), col0 = 16 * (blockIdx.x % (D / 16)) + CPT * cg;
    const int64_t SS = (int64_t)D * D;
    const int nJ = a.n_super;
    float *wsS = a.wsS + (int64_t)bh * nJ * SS;
    const float *wsM = a.wsM + (int64_t)bh * a.n_prep * SS;
    const float *wsN = a.wsN + (int64_t)bh * a.n_prep * SS;
    float acc[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) acc[j] = a.S_in ? a.S_in[bh * SS + (int64_t)k * D + col0 + j] : 0.f;
    f32x4 mreg[MV];
    auto fetch = [&](int J) {
        const f32x4 *m = reinterpret_cast<const f32x4 *>(wsM + (int64_t)J * SS);
#pragma unroll
        for (int i = 0; i < MV; ++i) mreg[i] = m[tid + NT * i];
    };
    const int last = a.scan_out ? nJ : nJ - 1;  // steps taken
    // S_J and S_out go out through buffer stores (32-bit lane offsets)
    constexpr int NV = CPT / 4;
    const rsrc_t rS = buf_rsrc(wsS, (uint32_t)(nJ * SS * 4));
    const uint32_t vo = (uint32_t)(((int64_t)k * D + col0) * 4);
    if (last > 0) fetch(0);
    for (int J = 0; J < nJ; ++J) {
#pragma unroll
        for (int u = 0; u < NV; ++u) {
            const f32x4 x = {acc[4 * u], acc[4 * u + 1], acc[4 * u + 2], acc[4 * u + 3]};
            *reinterpret_cast<f32x4 *>(&sS[k * 16 + col0 % 16 + 4 * u]) = x;
            buf_st(rS, vo + 16 * u, (uint32_t)(J * SS * 4), x);
        }
        if (J == last) break;
        float nv[CPT];
#pragma unroll
        for (int j = 0; j < CPT; ++j) nv[j] = wsN[(int64_t)J * SS + (int64_t)k * D + col0 + j];
#pragma unroll
        for (int i = 0; i < MV; ++i) {
            const int e = 4 * (tid + NT * i);
            *reinterpret_cast<f32x4 *>(&sM[(e / D) * LDM + e % D]) = mreg[i];
        }
        __syncthreads();
        if (J + 1 < last) fetch(J + 1);
#pragma unroll
        for (int j = 0; j < CPT; ++j) acc[j] = nv[j];
#pragma unroll 4
        for (int c = 0; c < D; c += 4) {
            const f32x4 m4 = *reinterpret_cast<const f32x4 *>(&sM[k * LDM + c]);
#pragma unroll
            for (int u = 0; u < 4; ++u)
#pragma unroll
                for (int j = 0; j < CPT; ++j) acc[j] = fmaf(m4[u], sS[(c + u) * 16 + col0 % 16 + j], acc[j]);
        }
        __syncthreads();  // every read of sM and sS is done
    }
    if (a.scan_out) {  // the state after the last superchunk
        const rsrc_t rO = buf_rsrc(a.S_out + bh * SS, (uint32_t)(SS * 4));
#pragma unroll
        for (int u = 0; u < NV; ++u)
            buf_st(rO, vo + 16 * u, 0u, f32x4{acc[4 * u], acc[4 * u + 1], acc[4 * u + 2], acc[4 * u + 3]});
    }
}


// ------------------------------------------------------------------ backward
//
// Per chunk, with S the state entering it, dS' the gradient of the state leaving
// it and the forward quantities above (b, gamma, Gamma, A, W, Ubar, U, P):
//   dU  = diag(e^{b_C - b}) K dS' + P^T dO
//   dS  = gamma_C dS' + Q^T diag(gamma) dO - W^T dU          (the state gradient entering)
//   dq  = diag(gamma) dO S^T + (dO U^T o Gamma) K
//   dk  = diag(e^{b_C - b}) U dS'^T + (dO U^T o Gamma)^T Q + diag(beta gamma) G_W + Ah K + Ah^T K
//   dv  = diag(beta) G_U,   [G_W | G_U] = (I + A)^{-T} [-dU S^T | dU]
//   dA  = -(G_W W^T + G_U Ubar^T) on s < t,   Ah = dA o beta_t e^{b_t - b_s}
//   dbeta_t = gamma_t <G_W_t, k_t> + <G_U_t, v_t> + sum_s dA[t][s] e^{b_t - b_s} k_t.k_s
// and the log-decay gradient collects, per token, every term through b_t
// (gamma_t, Gamma, A, e^{b_C - b_t}, gamma_C), summed in reverse over the chunk.
// dS runs backwards over the chunks; it is the chunk map's transpose, so a
// superchunk maps dS_end to dS_start = M_J^T dS_end + E_J, with M_J the forward
// prep's and E_J the walk from dS_end = 0.
//   k_gdn_dwalk<true>:  E_J for J >= 1;
//   k_gdn_dscan:        dS_end(J) for every J (M_{J+1}^T, fp32, in reverse);
//   k_gdn_dwalk<false>: from dS_end(J), writes dS' of every chunk and dS_in;
//   k_gdn_dchunk:       the parameter gradients of every chunk, all chunks in
//                       parallel, from the stored S and dS' (fp32 arithmetic).

template <typename T, int D, bool PREP>
__global__ void __launch_bounds__(64 * D / 16) k_gdn_dwalk(GdnArgs a) {
    constexpr int NW = D / 16, NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr int LDA = C + 4, LDU = D + 4;
    __shared__ __attribute__((aligned(16))) T sQ[C * LDN];   // swizzled
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];   // swizzled
    __shared__ __attribute__((aligned(16))) T sO[C * LDN];   // dO, swizzled
    // P^T[s][t] = e^{b_t-b_s} k_s.q_t (s <= t) hi, then lo; T = (I + A)^{-1} lives here first
    __shared__ __attribute__((aligned(16))) T sPP[2 * C * LDT];
    static_assert(2 * C * LDT * sizeof(T) >= C * (C + 4) * sizeof(float), "T does not fit the P tiles");
    T *sP = sPP, *sPl = sPP + C * LDT;
    float *sT = reinterpret_cast<float *>(sPP);
    __shared__ __attribute__((aligned(16))) float sA[C * LDA];
    __shared__ __attribute__((aligned(16))) float sW[C * LDU];
    __shared__ __attribute__((aligned(16))) float sb[C], sq[C], se[C], sbeta[C];

    const int tid = threadIdx.x, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c0 = 16 * w;
    const int nJ = PREP ? a.n_super - 1 : a.n_super;
    const int item = blockIdx.x, bh = item / nJ, J = (PREP ? 1 : 0) + item % nJ;
    const int bb = bh / a.H, hh = bh % a.H;
    const int64_t tok0 = (int64_t)J * a.ts;
    const int64_t xo = bb * a.sx_b + hh * a.sx_h + tok0 * a.sx_l;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *DO = (const T *)a.dO + xo;
    const int64_t go = bb * a.sg_b + hh * a.sg_h + tok0 * a.sg_l;
    const float *gp = a.g + go;
    const float *bp = a.beta + go;
    const int64_t SS = (int64_t)D * D;
    const int nch = (int)((a.L - tok0 < a.ts ? a.L - tok0 : a.ts) / C);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    auto asw = [](int row) { return sizeof(T) == 2 ? 8 * ((row >> 2) & 1) : 0; };

    // dS[16i + 4q4 + r][c0 + n16]: from dS_end(J) (dS_out for one superchunk), or 0 (prep)
    f32x4 dS[NK];
    {
        const float *src = a.n_super == 1 ? (a.dS_out ? a.dS_out + bh * SS : nullptr)
                                          : a.wsDe + ((int64_t)bh * a.n_super + J) * SS;
#pragma unroll
        for (int i = 0; i < NK; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                dS[i][r] = (!PREP && src) ? src[(int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] : 0.f;
    }

    using TT = Tile<T, D, NT>;
    TT t1, t2, t3;
    float gl, bl;
    const int64_t cstep = (int64_t)C * a.sx_l;
    const uint32_t cspan = chunk_span<T, D>(a.sx_l), gspan = (uint32_t)(((C - 1) * a.sg_l + 1) * 4);
    uint32_t toff[TT::RPT];
    TT::offsets(toff, a.sx_l, tid);
    const uint32_t goff = (uint32_t)(lane * a.sg_l * 4);
    auto issue = [&](int c) {
        const int64_t nx = c * cstep;
        t1.load_buf(buf_rsrc(Q + nx, cspan), toff, 0);
        t2.load_buf(buf_rsrc(K + nx, cspan), toff, 0);
        t3.load_buf(buf_rsrc(DO + nx, cspan), toff, 0);
        gl = buf_ld<float>(buf_rsrc(gp + (int64_t)c * C * a.sg_l, gspan), goff, 0);
        bl = buf_ld<float>(buf_rsrc(bp + (int64_t)c * C * a.sg_l, gspan), goff, 0);
    };
    if (nch > 0) issue(nch - 1);

    for (int c = nch - 1; c >= 0; --c) {
        if constexpr (!PREP) {  // dS' of chunk c: the gradient of the state leaving it
            float *dst = a.wsDc + ((int64_t)bh * (a.L / C) + tok0 / C + c) * SS;
#pragma unroll
            for (int i = 0; i < NK; ++i)
#pragma unroll
                for (int r = 0; r < 4; ++r) dst[(int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] = dS[i][r];
        }
        const float b2 = wave_scan_dpp(gl * LOG2E);
        const float b63 = lane_value(b2, 63);
        const float betal = bl;
        __syncthreads();  // the previous chunk is done with every LDS tile
        t1.store_swz(sQ, LDN, tid, SWX);
        t2.store_swz(sK, LDN, tid, SWX);
        t3.store_swz(sO, LDN, tid, SWX);
        if (w == 0) {
            sb[lane] = b2;
            sq[lane] = fexp2(b2);
            se[lane] = fexp2(b63 - b2);
            sbeta[lane] = betal;
        }
        __syncthreads();
        if (c > 0) issue(c - 1);

        // scores on the causal tiles: k_s . k_t -> A first; k_s . q_t -> P^T after the
        // solve, whose T occupies the P tiles' LDS
        auto scores = [&](int i0) {
        for (int i = i0 + w; i < i0 + 10; i += NW) {
            const bool kk = i >= 10;
            int tt, st;
            tri_tile(kk ? i - 10 : i, tt, st);
            f32x4 p = {0.f, 0.f, 0.f, 0.f};
#pragma unroll
            for (int ks = 0; ks < D / 32; ++ks) {
                const frag_t<T> kf = ldfrag_swz<T, LDN, SWX>(sK, swo, 16 * st, 32 * ks);
                const frag_t<T> xf = ldfrag_swz<T, LDN, SWX>(kk ? sK : sQ, swo, 16 * tt, 32 * ks);
                mma(p, kf, xf);
            }
            const int t = 16 * tt + n16;
            const float bt = sb[t];
            const f32x4 bs = *reinterpret_cast<const f32x4 *>(&sb[16 * st + 4 * q4]);
            if (!kk) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int s = 16 * st + 4 * q4 + r;
                    const float v = s <= t ? p[r] * fexp2(bt - bs[r]) : 0.f;
                    const T h = cvt<T>(v);
                    sP[s * LDT + (t ^ asw(s))] = h;
                    sPl[s * LDT + (t ^ asw(s))] = cvt<T>(v - tof<T>(h));
                }
            } else {
                const float be = sbeta[t];
                float v4[4];
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int s = 16 * st + 4 * q4 + r;
                    v4[r] = s < t ? be * p[r] * fexp2(bt - bs[r]) : 0.f;
                }
                *reinterpret_cast<f32x4 *>(&sA[t * LDA + 16 * st + 4 * q4]) = f32x4{v4[0], v4[1], v4[2], v4[3]};
            }
        }
        };
        scores(10);
        __syncthreads();
        gdn_tinv<NT>(tid, sA, sT);
        gdn_wu<T, D, LDN, LDU, SWX>(w, lane, tro, sT, sK, (const T *)nullptr, sbeta, sq, sW, nullptr);
        __syncthreads();
        scores(0);
        // P^T tiles below the diagonal that the dU product reads are zero
        for (int e = tid; e < 512; e += NT) {
            const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
            const int row = tile ? 48 + rr : 16 + rr, col = tile ? 32 + cc : cc;
            sP[row * LDT + (col ^ asw(row))] = cvt<T>(0.f);
            sPl[row * LDT + (col ^ asw(row))] = cvt<T>(0.f);
        }
        __syncthreads();

        // dU[t][v] = e^{b_C - b_t} sum_k K[t][k] dS[k][v] + sum_{t' >= t} P^T[t][t'] dO[t'][v]
        // (rows t = 16tt + 4q4 + r, column v = c0 + n16)
        f32x4 dU[4];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) dU[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            frag_t<T> fh, fl;
            split_acc_plain<T, true>(dS[2 * ks], dS[2 * ks + 1], fh, fl);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                const frag_t<T> kf = ldfrag_swz<T, LDN, SWX>(sK, swo, 16 * tt, 32 * ks);
                mma(dU[tt], kf, fh);
                mma(dU[tt], kf, fl);
            }
        }
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) dU[tt][r] *= se[16 * tt + 4 * q4 + r];
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            const frag_t<T> of = ldfragTR<T, LDN, SWX>(sO, tro, 32 * ks, c0);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                if (32 * ks + 31 < 16 * tt) continue;
                const int aw = asw(lane & 15);
                const int o = (16 * tt + (lane & 15)) * LDT + ((32 * ks + 8 * (lane >> 4)) ^ aw);
                mma(dU[tt], *reinterpret_cast<const frag_t<T> *>(sP + o), of);
                mma(dU[tt], *reinterpret_cast<const frag_t<T> *>(sPl + o), of);
            }
        }

        // dS = gamma_C dS + Q^T diag(gamma) dO - W^T dU
        const float gam = fexp2(b63);
#pragma unroll
        for (int i = 0; i < NK; ++i) dS[i] *= gam;
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            f32x4 g0, g1;  // gamma_t dO[t][c0 + n16], t = 32ks + 16h + 4q4 + r
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ta = 32 * ks + 4 * q4 + r, tb = ta + 16;
                g0[r] = sq[ta] * tof<T>(sO[ta * LDN + swz_col(ta, c0 + n16, SWX)]);
                g1[r] = sq[tb] * tof<T>(sO[tb * LDN + swz_col(tb, c0 + n16, SWX)]);
            }
            frag_t<T> gh, glo, uh, ul;
            split_acc_plain<T, true>(g0, g1, gh, glo);
            split_acc_plain<T, true>(dU[2 * ks], dU[2 * ks + 1], uh, ul);
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                mma2b<T, true>(dS[i], ldfragTR<T, LDN, SWX>(sQ, tro, 32 * ks, 16 * i), gh, glo);
                float wn[8];  // -W[t][k], k = 16i + lane % 16, t = 32ks + 8 (lane / 16) + j
#pragma unroll
                for (int j = 0; j < 8; ++j) wn[j] = -sW[(32 * ks + 8 * q4 + j) * LDU + 16 * i + n16];
                frag_t<T> wh, wl;
                split8<T, true>(wn, wh, wl);
                mma(dS[i], wh, uh);
                mma(dS[i], wh, ul);
                mma(dS[i], wl, uh);
            }
        }
    }
    float *dst = PREP ? a.wsE + ((int64_t)bh * (a.n_super - 1) + J - 1) * SS : (J == 0 ? a.dS_in + bh * SS : nullptr);
    if (dst) {
#pragma unroll
        for (int i = 0; i < NK; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] = dS[i][r];
    }
}

// dS_end(n-1) = dS_out (or 0); dS_end(J-1) = M_J^T dS_end(J) + E_J, written to
// wsDe for every J.  Same shape of work as k_gdn_scan, with M_J read transposed.
template <int D>
__global__ void __launch_bounds__(256) k_gdn_dscan(GdnArgs a) {
    constexpr int NT = 256, RPT = NT / D, CPT = 16 / RPT, LDM = D + 4, MV = D * D / 4 / NT;
    __shared__ __attribute__((aligned(16))) float sM[D * LDM];
    __shared__ __attribute__((aligned(16))) float sS[D * 16];
    const int tid = threadIdx.x, k = tid % D, cg = tid / D;
    const int bh = blockIdx.x / (D / 16), col0 = 16 * (blockIdx.x % (D / 16)) + CPT * cg;
    const int64_t SS = (int64_t)D * D;
    const int nJ = a.n_super;
    float *wsDe = a.wsDe + (int64_t)bh * nJ * SS;
    const float *wsM = a.wsM + (int64_t)bh * a.n_prep * SS;
    const float *wsE = a.wsE + (int64_t)bh * (nJ - 1) * SS;
    float acc[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) acc[j] = a.dS_out ? a.dS_out[bh * SS + (int64_t)k * D + col0 + j] : 0.f;
    f32x4 mreg[MV];
    auto fetch = [&](int J) {
        const f32x4 *m = reinterpret_cast<const f32x4 *>(wsM + (int64_t)J * SS);
#pragma unroll
        for (int i = 0; i < MV; ++i) mreg[i] = m[tid + NT * i];
    };
    if (nJ > 1) fetch(nJ - 1);
    for (int J = nJ - 1;; --J) {
#pragma unroll
        for (int j = 0; j < CPT; ++j) {
            sS[k * 16 + col0 % 16 + j] = acc[j];
            wsDe[(int64_t)J * SS + (int64_t)k * D + col0 + j] = acc[j];
        }
        if (J == 0) break;
        float nv[CPT];
#pragma unroll
        for (int j = 0; j < CPT; ++j) nv[j] = wsE[(int64_t)(J - 1) * SS + (int64_t)k * D + col0 + j];
#pragma unroll
        for (int i = 0; i < MV; ++i) {
            const int e = 4 * (tid + NT * i);
            *reinterpret_cast<f32x4 *>(&sM[(e / D) * LDM + e % D]) = mreg[i];
        }
        __syncthreads();
        if (J - 1 >= 1) fetch(J - 1);
#pragma unroll
        for (int j = 0; j < CPT; ++j) acc[j] = nv[j];
#pragma unroll 4
        for (int c = 0; c < D; ++c) {
            const float m = sM[c * LDM + k];  // M_J^T[k][c]
#pragma unroll
            for (int j = 0; j < CPT; ++j) acc[j] = fmaf(m, sS[c * 16 + col0 % 16 + j], acc[j]);
        }
        __syncthreads();
    }
}

// Parameter gradients of one chunk per item (b, h, chunk), items in a
// grid-stride loop.  Every product runs on MFMA: 8 waves, wave w owns rows
// [16 (w % 4), +16) and half the column tiles (half w / 4) of each 64-row
// result, so two waves share each SIMD.  Operands enter as bf16 fragments,
// computed fp32 operands as hi/lo pairs (three products, the lo x lo term
// dropped), q, k, v, dO exactly.  q, k, v, dO and the 64 x 64 matrices sit in
// LDS; the 64 x D intermediates in a per-workgroup scratch slab of wsX (eight
// 64 x D fp32 matrices, addressed through one buffer resource); S and dS' come
// from the stored per-chunk states.  T = (I + A)^{-1} comes from gdn_tinv
// with beta applied per row.
template <typename T, int D>
__global__ void __launch_bounds__(512) k_gdn_dchunk(GdnArgs a) {
    constexpr int LDX = D + 8, LD6 = C + 4, NT2 = D / 32, NTH = 512;
    __shared__ __attribute__((aligned(16))) T xq[C * LDX], xk[C * LDX], xo[C * LDX], xv[C * LDX];
    __shared__ __attribute__((aligned(16))) float sKK[C * LD6];  // e^{b_t-b_s} k_t.k_s, s < t (later Ah + Ah^T)
    __shared__ __attribute__((aligned(16))) float sT[C * LD6];   // (I + A)^{-1}
    __shared__ __attribute__((aligned(16))) float sPt[C * LD6];  // e^{b_t-b_s} q_t.k_s, s <= t
    __shared__ __attribute__((aligned(16))) float sdP[C * LD6];  // (dO U^T o Gamma)[t][s], s <= t
    __shared__ float sb[C], sg[C], se[C], sbe[C], sRb[2 * C], sRd[2 * C], sCol[4 * C], s63[8];

    const int tid = threadIdx.x, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6), r0 = 16 * (w & 3), hf = w >> 2;
    const int64_t SS = (int64_t)D * D, SX = (int64_t)C * D;
    const int nc = (int)(a.L / C);
    const int64_t items = (int64_t)a.B * a.H * nc;
    const rsrc_t rX = buf_rsrc(a.wsX + (int64_t)blockIdx.x * 8 * SX, (uint32_t)(8 * SX * 4));
    constexpr uint32_t MB = (uint32_t)(C * D * 4);  // bytes of one slab matrix
    constexpr uint32_t mW = 0, mUb = MB, mU = 2 * MB, mdU = 3 * MB, mGW = 4 * MB, mGU = 5 * MB, mQ = 6 * MB, mK = 7 * MB;
    // lane offsets: row-major fragment (row n16, k 8q4..), transposed fragment
    // (k 8q4 + j, row n16), accumulator element (row 4q4 + r, column n16)
    const uint32_t v_rm = (uint32_t)((n16 * D + 8 * q4) * 4), v_tr = (uint32_t)((8 * q4 * D + n16) * 4);
    const uint32_t v_acc = (uint32_t)((4 * q4 * D + n16) * 4);

    auto g_rm = [&](rsrc_t rs, uint32_t base, int rr, int kk, frag_t<T> &h, frag_t<T> &l) {
        const uint32_t so = base + (uint32_t)((rr * D + kk) * 4);
        const f32x4 x0 = buf_ld<f32x4>(rs, v_rm, so), x1 = buf_ld<f32x4>(rs, v_rm + 16, so);
        const float x[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
        split8<T, true>(x, h, l);
    };
    auto g_tr = [&](rsrc_t rs, uint32_t base, int rr, int kk, frag_t<T> &h, frag_t<T> &l) {
        const uint32_t so = base + (uint32_t)((kk * D + rr) * 4);
        float x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = buf_ld<float>(rs, v_tr + j * D * 4, so);
        split8<T, true>(x, h, l);
    };
    auto g_acc_ld = [&](rsrc_t rs, uint32_t base, int ct, f32x4 &c) {
#pragma unroll
        for (int r = 0; r < 4; ++r) c[r] = buf_ld<float>(rs, v_acc + r * D * 4, base + (uint32_t)((r0 * D + 16 * ct) * 4));
    };
    auto g_acc_st = [&](rsrc_t rs, uint32_t base, int ct, const f32x4 &c) {
#pragma unroll
        for (int r = 0; r < 4; ++r) buf_st<float>(rs, v_acc + r * D * 4, base + (uint32_t)((r0 * D + 16 * ct) * 4), c[r]);
    };
    // the same at an explicit row base (row tile rt: rows 16 rt + 4 q4 + r)
    auto g_acc_ld_rt = [&](rsrc_t rs, uint32_t base, int rt, int ct, f32x4 &c) {
#pragma unroll
        for (int r = 0; r < 4; ++r) c[r] = buf_ld<float>(rs, v_acc + r * D * 4, base + (uint32_t)((16 * rt * D + 16 * ct) * 4));
    };
    auto g_acc_st_rt = [&](rsrc_t rs, uint32_t base, int rt, int ct, const f32x4 &c) {
#pragma unroll
        for (int r = 0; r < 4; ++r) buf_st<float>(rs, v_acc + r * D * 4, base + (uint32_t)((16 * rt * D + 16 * ct) * 4), c[r]);
    };
    auto l_rm = [&](const float *M, int rr, int kk, frag_t<T> &h, frag_t<T> &l) {  // LDS 64 x 64, M[row][k]
        const float *p = M + (rr + n16) * LD6 + kk + 8 * q4;
        const f32x4 x0 = *reinterpret_cast<const f32x4 *>(p), x1 = *reinterpret_cast<const f32x4 *>(p + 4);
        const float x[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
        split8<T, true>(x, h, l);
    };
    auto l_tr = [&](const float *M, int rr, int kk, frag_t<T> &h, frag_t<T> &l) {  // LDS 64 x 64, M[k][row]
        float x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = M[(kk + 8 * q4 + j) * LD6 + rr + n16];
        split8<T, true>(x, h, l);
    };
    auto x_rm = [&](const T *M, int rr, int kk) {  // exact, M[row][k]
        return *reinterpret_cast<const frag_t<T> *>(M + (rr + n16) * LDX + kk + 8 * q4);
    };
    auto x_tr = [&](const T *M, int rr, int kk) {  // exact, M[k][row]
        frag_t<T> f = {};
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = M[(kk + 8 * q4 + j) * LDX + rr + n16];
        return f;
    };
    auto mma3 = [](f32x4 &c, const frag_t<T> &ah, const frag_t<T> &al, const frag_t<T> &bh, const frag_t<T> &bl) {
        mma(c, ah, bh);
        mma(c, ah, bl);
        mma(c, al, bh);
    };
    auto zeroN = [](f32x4 (&c)[NT2]) {
#pragma unroll
        for (int i = 0; i < NT2; ++i) c[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    auto zero2 = [](f32x4 (&c)[2]) {
#pragma unroll
        for (int i = 0; i < 2; ++i) c[i] = f32x4{0.f, 0.f, 0.f, 0.f};
    };
    // accumulator c[nt][r] <-> row r0 + 4 q4 + r, column 16 (hf NT2 + nt) + n16 (64 x D results)
    // or 16 (2 hf + nt) + n16 (64 x 64 results)

    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        const int bh = (int)(it / nc), ch = (int)(it % nc), bb = bh / a.H, hh = bh % a.H;
        const int64_t xo0 = bb * a.sx_b + hh * a.sx_h + (int64_t)ch * C * a.sx_l;
        const int64_t go0 = bb * a.sg_b + hh * a.sg_h + (int64_t)ch * C * a.sg_l;
        const float *S = a.wsSc + ((int64_t)bh * nc + ch) * SS;
        const float *dS = a.wsDc + ((int64_t)bh * nc + ch) * SS;
        const rsrc_t rS = buf_rsrc(S, (uint32_t)(SS * 4)), rD = buf_rsrc(dS, (uint32_t)(SS * 4));
        __syncthreads();  // the previous item is done with LDS and the slab
        for (int e = tid; e < C * D / 8; e += NTH) {
            const int t = e / (D / 8), c8 = 8 * (e % (D / 8));
            const int64_t off = xo0 + (int64_t)t * a.sx_l + c8;
            *reinterpret_cast<frag_t<T> *>(&xq[t * LDX + c8]) = *reinterpret_cast<const frag_t<T> *>((const T *)a.q + off);
            *reinterpret_cast<frag_t<T> *>(&xk[t * LDX + c8]) = *reinterpret_cast<const frag_t<T> *>((const T *)a.k + off);
            *reinterpret_cast<frag_t<T> *>(&xo[t * LDX + c8]) = *reinterpret_cast<const frag_t<T> *>((const T *)a.dO + off);
            *reinterpret_cast<frag_t<T> *>(&xv[t * LDX + c8]) = *reinterpret_cast<const frag_t<T> *>((const T *)a.v + off);
        }
        if (tid < 64) {
            const float b = wave_scan_dpp(a.g[go0 + (int64_t)tid * a.sg_l]);
            const float bC = lane_value(b, 63);
            sb[tid] = b;
            sg[tid] = expf(b);
            se[tid] = expf(bC - b);
            sbe[tid] = a.beta[go0 + (int64_t)tid * a.sg_l];
        }
        __syncthreads();

        float rowb[4] = {0.f, 0.f, 0.f, 0.f}, rowd[4] = {0.f, 0.f, 0.f, 0.f}, colb[4] = {0.f, 0.f, 0.f, 0.f};
        float tot63 = 0.f;
        // scores: k_t.k_s and q_t.k_s
        {
            f32x4 pk[2], pq[2];
            zero2(pk);
            zero2(pq);
#pragma unroll
            for (int kk = 0; kk < D; kk += 32) {
                const frag_t<T> ak = x_rm(xk, r0, kk), aq = x_rm(xq, r0, kk);
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) {
                    const frag_t<T> bk = x_rm(xk, 16 * (2 * hf + nt), kk);
                    mma(pk[nt], ak, bk);
                    mma(pq[nt], aq, bk);
                }
            }
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = r0 + 4 * q4 + r, s2 = 16 * (2 * hf + nt) + n16;
                    const float ga = expf(sb[t] - sb[s2]);
                    sKK[t * LD6 + s2] = s2 < t ? ga * pk[nt][r] : 0.f;
                    sPt[t * LD6 + s2] = s2 <= t ? ga * pq[nt][r] : 0.f;
                }
        }
        __syncthreads();
        // T = (I + A)^{-1}, A = diag(beta) KK
        gdn_tinv<NTH>(tid, sKK, sT, sbe);
        // W = T diag(beta gamma) K, Ubar = T diag(beta) V
        {
            f32x4 cw[NT2], cu[NT2];
            zeroN(cw);
            zeroN(cu);
#pragma unroll
            for (int kk = 0; kk < C; kk += 32) {
                frag_t<T> th, tl;
                l_rm(sT, r0, kk, th, tl);
#pragma unroll
                for (int nt = 0; nt < NT2; ++nt) {
                    const int col = 16 * (NT2 * hf + nt) + n16;
                    float xw[8], xu[8];
#pragma unroll
                    for (int j = 0; j < 8; ++j) {
                        const int s2 = kk + 8 * q4 + j;
                        xw[j] = sbe[s2] * sg[s2] * tof<T>(xk[s2 * LDX + col]);
                        xu[j] = sbe[s2] * tof<T>(xv[s2 * LDX + col]);
                    }
                    frag_t<T> bh, bl;
                    split8<T, true>(xw, bh, bl);
                    mma3(cw[nt], th, tl, bh, bl);
                    split8<T, true>(xu, bh, bl);
                    mma3(cu[nt], th, tl, bh, bl);
                }
            }
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt) {
                g_acc_st(rX, mW, NT2 * hf + nt, cw[nt]);
                g_acc_st(rX, mUb, NT2 * hf + nt, cu[nt]);
            }
        }
        __syncthreads();
        // U = Ubar - W S;  dU = diag(e^{b_C - b}) K dS' + P^T dO.  Here wave w
        // owns row tiles 2 (w % 2) + i (i < 2) and column tiles CT (w / 2) + j
        // (j < CT), so no two waves load the same S or dS' fragment.
        {
            constexpr int CT = NT2 / 2 > 0 ? NT2 / 2 : 1;
            static_assert(2 * CT * 8 == 4 * (D / 16), "eight waves cover the 4 x D/16 tiles once");
            const int rp = w & 1, cg = w >> 1;
            f32x4 cu[2][CT], cd[2][CT];
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < CT; ++j) {
                    g_acc_ld_rt(rX, mUb, 2 * rp + i, CT * cg + j, cu[i][j]);
                    cd[i][j] = f32x4{0.f, 0.f, 0.f, 0.f};
                }
#pragma unroll 1
            for (int kk = 0; kk < D; kk += 32) {
                frag_t<T> wh[2], wl[2], ak[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) {
                    g_rm(rX, mW, 16 * (2 * rp + i), kk, wh[i], wl[i]);
                    wh[i] = -wh[i];
                    wl[i] = -wl[i];
                    ak[i] = x_rm(xk, 16 * (2 * rp + i), kk);
                }
#pragma unroll
                for (int j = 0; j < CT; ++j) {
                    frag_t<T> sh, sl;
                    g_tr(rS, 0, 16 * (CT * cg + j), kk, sh, sl);
#pragma unroll
                    for (int i = 0; i < 2; ++i) mma3(cu[i][j], wh[i], wl[i], sh, sl);
                    g_tr(rD, 0, 16 * (CT * cg + j), kk, sh, sl);
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        mma(cd[i][j], ak[i], sh);
                        mma(cd[i][j], ak[i], sl);
                    }
                }
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < CT; ++j)
#pragma unroll
                    for (int r = 0; r < 4; ++r) cd[i][j][r] *= se[16 * (2 * rp + i) + 4 * q4 + r];
#pragma unroll
            for (int kk = 0; kk < C; kk += 32) {
                frag_t<T> ph[2], pl[2];
#pragma unroll
                for (int i = 0; i < 2; ++i) l_tr(sPt, 16 * (2 * rp + i), kk, ph[i], pl[i]);  // P^T[t][t'] = P[t'][t]
#pragma unroll
                for (int j = 0; j < CT; ++j) {
                    const frag_t<T> bo = x_tr(xo, 16 * (CT * cg + j), kk);
#pragma unroll
                    for (int i = 0; i < 2; ++i) {
                        mma(cd[i][j], ph[i], bo);
                        mma(cd[i][j], pl[i], bo);
                    }
                }
            }
#pragma unroll
            for (int i = 0; i < 2; ++i)
#pragma unroll
                for (int j = 0; j < CT; ++j) {
                    g_acc_st_rt(rX, mU, 2 * rp + i, CT * cg + j, cu[i][j]);
                    g_acc_st_rt(rX, mdU, 2 * rp + i, CT * cg + j, cd[i][j]);
                }
        }
        __syncthreads();
        // G_U = T^T dU (dv, dbeta)
        {
            f32x4 cg[NT2];
            zeroN(cg);
#pragma unroll
            for (int kk = 0; kk < C; kk += 32) {
                frag_t<T> th, tl;
                l_tr(sT, r0, kk, th, tl);
#pragma unroll
                for (int nt = 0; nt < NT2; ++nt) {
                    frag_t<T> bh, bl;
                    g_tr(rX, mdU, 16 * (NT2 * hf + nt), kk, bh, bl);
                    mma3(cg[nt], th, tl, bh, bl);
                }
            }
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt) {
                g_acc_st(rX, mGU, NT2 * hf + nt, cg[nt]);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = r0 + 4 * q4 + r, c = 16 * (NT2 * hf + nt) + n16;
                    ((T *)a.dv)[xo0 + (int64_t)t * a.sx_l + c] = cvt<T>(sbe[t] * cg[nt][r]);
                    rowd[r] = fmaf(cg[nt][r], tof<T>(xv[t * LDX + c]), rowd[r]);
                }
            }
        }
        // dW = -dU S^T and diag(gamma) dO S^T
        {
            f32x4 cw[NT2], cq[NT2];
            zeroN(cw);
            zeroN(cq);
#pragma unroll 1
            for (int kk = 0; kk < D; kk += 32) {
                frag_t<T> uh, ul;
                g_rm(rX, mdU, r0, kk, uh, ul);
                uh = -uh;
                ul = -ul;
                const frag_t<T> ao = x_rm(xo, r0, kk);
#pragma unroll
                for (int nt = 0; nt < NT2; ++nt) {
                    frag_t<T> sh, sl;
                    g_rm(rS, 0, 16 * (NT2 * hf + nt), kk, sh, sl);  // B[k'][v] = S[k'][v]
                    mma3(cw[nt], uh, ul, sh, sl);
                    mma(cq[nt], ao, sh);
                    mma(cq[nt], ao, sl);
                }
            }
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = r0 + 4 * q4 + r, c = 16 * (NT2 * hf + nt) + n16;
                    cq[nt][r] *= sg[t];
                    rowb[r] = fmaf(tof<T>(xq[t * LDX + c]), cq[nt][r], rowb[r]);
                }
                g_acc_st(rX, mGW, NT2 * hf + nt, cw[nt]);
                g_acc_st(rX, mQ, NT2 * hf + nt, cq[nt]);
            }
        }
        __syncthreads();
        // G_W = T^T dW, held until every wave has read dW; dk starts as diag(beta gamma) G_W
        {
            f32x4 cg[NT2];
            zeroN(cg);
#pragma unroll
            for (int kk = 0; kk < C; kk += 32) {
                frag_t<T> th, tl;
                l_tr(sT, r0, kk, th, tl);
#pragma unroll
                for (int nt = 0; nt < NT2; ++nt) {
                    frag_t<T> bh, bl;
                    g_tr(rX, mGW, 16 * (NT2 * hf + nt), kk, bh, bl);
                    mma3(cg[nt], th, tl, bh, bl);
                }
            }
            __syncthreads();  // every read of dW is done
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt) {
                f32x4 kg4;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = r0 + 4 * q4 + r, c = 16 * (NT2 * hf + nt) + n16;
                    const float kg = cg[nt][r] * tof<T>(xk[t * LDX + c]);
                    rowd[r] = fmaf(sg[t], kg, rowd[r]);
                    rowb[r] = fmaf(sbe[t] * sg[t], kg, rowb[r]);
                    kg4[r] = sbe[t] * sg[t] * cg[nt][r];
                }
                g_acc_st(rX, mGW, NT2 * hf + nt, cg[nt]);
                g_acc_st(rX, mK, NT2 * hf + nt, kg4);
            }
        }
        __syncthreads();
        // dA = -(G_W W^T + G_U Ubar^T) on s < t;  dP = dO U^T on s <= t
        {
            f32x4 ca[2], cp[2];
            zero2(ca);
            zero2(cp);
#pragma unroll 1
            for (int kk = 0; kk < D; kk += 32) {
                frag_t<T> gh, gl, uh, ul;
                g_rm(rX, mGW, r0, kk, gh, gl);
                g_rm(rX, mGU, r0, kk, uh, ul);
                gh = -gh;
                gl = -gl;
                uh = -uh;
                ul = -ul;
                const frag_t<T> ao = x_rm(xo, r0, kk);
#pragma unroll
                for (int nt = 0; nt < 2; ++nt) {
                    frag_t<T> bh, bl;
                    g_rm(rX, mW, 16 * (2 * hf + nt), kk, bh, bl);
                    mma3(ca[nt], gh, gl, bh, bl);
                    g_rm(rX, mUb, 16 * (2 * hf + nt), kk, bh, bl);
                    mma3(ca[nt], uh, ul, bh, bl);
                    g_rm(rX, mU, 16 * (2 * hf + nt), kk, bh, bl);
                    mma(cp[nt], ao, bh);
                    mma(cp[nt], ao, bl);
                }
            }
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = r0 + 4 * q4 + r, s2 = 16 * (2 * hf + nt) + n16;
                    const float kk = sKK[t * LD6 + s2];  // 0 unless s < t
                    const float dA = s2 < t ? ca[nt][r] : 0.f;
                    rowd[r] = fmaf(dA, kk, rowd[r]);
                    const float ea = dA * sbe[t] * kk;  // dA o A
                    const float pt = sPt[t * LD6 + s2];  // 0 unless s <= t
                    const float ep = s2 <= t ? cp[nt][r] * pt : 0.f;  // dP o P
                    rowb[r] += ea + ep;
                    colb[nt] -= ea + ep;
                    const float ga = s2 <= t ? expf(sb[t] - sb[s2]) : 0.f;
                    sdP[t * LD6 + s2] = cp[nt][r] * ga;
                    ca[nt][r] = dA * sbe[t] * ga;  // Ah
                }
#pragma unroll
            for (int nt = 0; nt < 2; ++nt) {  // column sums over this wave's rows
                float v = colb[nt];
                v += __shfl_xor(v, 16);
                v += __shfl_xor(v, 32);
                if (q4 == 0) sCol[(w & 3) * C + 16 * (2 * hf + nt) + n16] = v;
            }
            __syncthreads();  // every read of the scores in sKK is done
#pragma unroll
            for (int nt = 0; nt < 2; ++nt)
#pragma unroll
                for (int r = 0; r < 4; ++r) sKK[(r0 + 4 * q4 + r) * LD6 + 16 * (2 * hf + nt) + n16] = ca[nt][r];
        }
        __syncthreads();
        // symmetrise: sKK = Ah + Ah^T (Ah strictly lower)
        for (int e = tid; e < C * C; e += NTH) {
            const int t = e / C, s2 = e % C;
            if (s2 < t) sKK[s2 * LD6 + t] = sKK[t * LD6 + s2];
            else if (s2 == t) sKK[t * LD6 + t] = 0.f;
        }
        __syncthreads();
        // dq = diag(gamma) dO S^T + dP K
        {
            f32x4 cq[NT2];
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt) g_acc_ld(rX, mQ, NT2 * hf + nt, cq[nt]);
#pragma unroll
            for (int kk = 0; kk < C; kk += 32) {
                frag_t<T> ph, pl;
                l_rm(sdP, r0, kk, ph, pl);
#pragma unroll
                for (int nt = 0; nt < NT2; ++nt) {
                    const frag_t<T> bk = x_tr(xk, 16 * (NT2 * hf + nt), kk);  // B[k'][s] = K[s][k']
                    mma(cq[nt], ph, bk);
                    mma(cq[nt], pl, bk);
                }
            }
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    ((T *)a.dq)[xo0 + (int64_t)(r0 + 4 * q4 + r) * a.sx_l + 16 * (NT2 * hf + nt) + n16] = cvt<T>(cq[nt][r]);
        }
        // dk = diag(beta gamma) G_W + diag(e^{b_C - b}) U dS'^T + dP^T Q + (Ah + Ah^T) K
        {
            f32x4 ck[NT2];
            zeroN(ck);
#pragma unroll 1
            for (int kk = 0; kk < D; kk += 32) {
                frag_t<T> uh, ul;
                g_rm(rX, mU, r0, kk, uh, ul);
#pragma unroll
                for (int nt = 0; nt < NT2; ++nt) {
                    frag_t<T> bh, bl;
                    g_rm(rD, 0, 16 * (NT2 * hf + nt), kk, bh, bl);  // B[k'][v] = dS'[k'][v]
                    mma3(ck[nt], uh, ul, bh, bl);
                }
            }
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt) {
                f32x4 gk;
                g_acc_ld(rX, mK, NT2 * hf + nt, gk);
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = r0 + 4 * q4 + r, c = 16 * (NT2 * hf + nt) + n16;
                    const float rk = ck[nt][r] * tof<T>(xk[t * LDX + c]);
                    rowb[r] -= se[t] * rk;
                    tot63 += se[t] * rk;
                    ck[nt][r] = fmaf(se[t], ck[nt][r], gk[r]);
                }
            }
#pragma unroll
            for (int kk = 0; kk < C; kk += 32) {
                frag_t<T> ph, pl, ah, al;
                l_tr(sdP, r0, kk, ph, pl);  // dP^T[t][t'] = dP[t'][t]
                l_rm(sKK, r0, kk, ah, al);
#pragma unroll
                for (int nt = 0; nt < NT2; ++nt) {
                    const frag_t<T> bq = x_tr(xq, 16 * (NT2 * hf + nt), kk), bk = x_tr(xk, 16 * (NT2 * hf + nt), kk);
                    mma(ck[nt], ph, bq);
                    mma(ck[nt], pl, bq);
                    mma(ck[nt], ah, bk);
                    mma(ck[nt], al, bk);
                }
            }
#pragma unroll
            for (int nt = 0; nt < NT2; ++nt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    ((T *)a.dk)[xo0 + (int64_t)(r0 + 4 * q4 + r) * a.sx_l + 16 * (NT2 * hf + nt) + n16] = cvt<T>(ck[nt][r]);
        }
        // gamma_C <dS', S> for b_C
        {
            float sd = 0.f;
            for (int e = 4 * tid; e < D * D; e += 4 * NTH) {
                const f32x4 x = buf_ld<f32x4>(rD, (uint32_t)(e * 4), 0), y = buf_ld<f32x4>(rS, (uint32_t)(e * 4), 0);
                sd = fmaf(x[0], y[0], fmaf(x[1], y[1], fmaf(x[2], y[2], fmaf(x[3], y[3], sd))));
            }
            tot63 = fmaf(sg[C - 1], sd, tot63);
        }
        // row sums over the 16 lanes of each row; tot63 over the workgroup
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            float vb = rowb[r], vd = rowd[r];
#pragma unroll
            for (int m = 1; m < 16; m <<= 1) {
                vb += __shfl_xor(vb, m);
                vd += __shfl_xor(vd, m);
            }
            if (n16 == 0) {
                sRb[hf * C + r0 + 4 * q4 + r] = vb;
                sRd[hf * C + r0 + 4 * q4 + r] = vd;
            }
        }
#pragma unroll
        for (int m = 1; m < 64; m <<= 1) tot63 += __shfl_xor(tot63, m);
        if (lane == 0) s63[w] = tot63;
        __syncthreads();
        if (tid < C) {
            float db = sRb[tid] + sRb[C + tid];
            for (int u = 0; u < 4; ++u) db += sCol[u * C + tid];
            if (tid == C - 1)
                for (int u = 0; u < 8; ++u) db += s63[u];
            sb[tid] = db;  // b no longer needed
            a.dbeta[go0 + (int64_t)tid * a.sg_l] = sRd[tid] + sRd[C + tid];
        }
        __syncthreads();
        if (tid == 0) {  // dg_i = sum_{t >= i} db_t
            float acc = 0.f;
            for (int t = C - 1; t >= 0; --t) {
                acc += sb[t];
                a.dg[go0 + (int64_t)t * a.sg_l] = acc;
            }
        }
    }
}

template <int D>
hipError_t gdn_phase_d(int phase, const GdnArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    const unsigned bh = (unsigned)(a.B * a.H);
    const dim3 wblk(64 * D / 16);
    switch (phase) {
    case GDN_PREP:
        hipExtLaunchKernelGGL((k_gdn_walk<__bf16, D, W_PREP>), dim3(bh * a.n_prep), wblk, 0, s, e0, e1, 0, a);
        break;
    case GDN_SCAN: hipExtLaunchKernelGGL((k_gdn_scan<D>), dim3(bh * (D / 16)), dim3(256), 0, s, e0, e1, 0, a); break;
    case GDN_OUT:
        hipExtLaunchKernelGGL((k_gdn_walk<__bf16, D, W_OUT>), dim3(bh * a.n_super), wblk, 0, s, e0, e1, 0, a);
        break;
    case GDN_STORE:
        hipExtLaunchKernelGGL((k_gdn_walk<__bf16, D, W_STORE>), dim3(bh * a.n_super), wblk, 0, s, e0, e1, 0, a);
        break;
    case GDN_DPREP:
        hipExtLaunchKernelGGL((k_gdn_dwalk<__bf16, D, true>), dim3(bh * (a.n_super - 1)), wblk, 0, s, e0, e1, 0, a);
        break;
    case GDN_DSCAN: hipExtLaunchKernelGGL((k_gdn_dscan<D>), dim3(bh * (D / 16)), dim3(256), 0, s, e0, e1, 0, a); break;
    case GDN_DWALK:
        hipExtLaunchKernelGGL((k_gdn_dwalk<__bf16, D, false>), dim3(bh * a.n_super), wblk, 0, s, e0, e1, 0, a);
        break;
    case GDN_DCHUNK: {
        const int64_t items = (int64_t)bh * (a.L / C);
        if (items > 0)
            hipExtLaunchKernelGGL((k_gdn_dchunk<__bf16, D>), dim3((unsigned)std::min<int64_t>(items, a.n_x)),
                                  dim3(512), 0, s, e0, e1, 0, a);
        break;
    }
    default: return hipErrorInvalidValue;
    }
    return hipGetLastError();
}

}  // namespace

// Argument checks shared by every phase: the superchunk buffers a phase reads
// or writes must be there.
hipError_t launch_gdn_phase(int phase, const GdnArgs &a, int D, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (a.n_super < 1) return hipErrorInvalidValue;
    const bool multi = a.n_super > 1;
    switch (phase) {
    case GDN_PREP:
    case GDN_SCAN:
        if (!multi || !a.wsS || !a.wsM || !a.wsN || a.n_prep < a.n_super - 1) return hipErrorInvalidValue;
        if (a.scan_out && (a.n_prep != a.n_super || !a.S_out)) return hipErrorInvalidValue;
        break;
    case GDN_DPREP:
    case GDN_DSCAN:
        if (!multi || !a.wsM || !a.wsE || !a.wsDe || a.n_prep != a.n_super) return hipErrorInvalidValue;
        break;
    case GDN_OUT:
        if (multi && !a.wsS) return hipErrorInvalidValue;
        break;
    case GDN_STORE:
        if (!a.wsSc || (multi && !a.wsS)) return hipErrorInvalidValue;
        break;
    case GDN_DWALK:
        if (!a.wsDc || (multi && !a.wsDe)) return hipErrorInvalidValue;
        break;
    case GDN_DCHUNK:
        if (!a.wsSc || !a.wsDc || !a.wsX || a.n_x < 1) return hipErrorInvalidValue;
        break;
    default: return hipErrorInvalidValue;
    }
    if (D == 128) return gdn_phase_d<128>(phase, a, s, e0, e1);
    if (D == 64) return gdn_phase_d<64>(phase, a, s, e0, e1);
    return hipErrorInvalidValue;
}

}  // namespace sf
