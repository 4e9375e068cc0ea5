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
//   (I + A) [W | Ubar] = [diag(beta gamma) K | diag(beta) V]     (forward substitution)
//   U        = Ubar - W S                                          (the corrected values, V^new)
//   O        = diag(gamma) Q S + (Q K^T o Gamma) U,  Gamma[t][s] = e^{b_t - b_s} (s <= t)
//   S_next   = gamma_C S + (K o e^{b_C - b})^T U
// This follows from writing u_t = beta_t (v_t - a_t S_{t-1}^T k_t), so that
// S_t = a_t S_{t-1} + k_t u_t^T is a plain gated linear recurrence in u, and
// solving the within-chunk dependence of u on the earlier u's.
//
// One workgroup walks all chunks of one (batch, head) segment with the state in
// registers: wave w owns the 16 state columns [16w, 16w+16) (D/16 waves).  Per
// chunk: the q, k, v tiles are staged in LDS; the QK^T and KK^T scores run on
// MFMA (10 causal 16x16 tiles each); the triangular system is solved in fp32,
// one thread per right-hand-side column; U, the output and the state update are
// MFMA products whose computed operands (S, W, U) go in as bf16 hi/lo pairs,
// U straight from its accumulators (rows t, columns v), which two lane-row
// swaps make into operand fragments with the tokens as contraction.
//
// Superchunk parallelism (the Pre / ST / Out split of Sec. 2.2 with the delta
// rule's matrix-valued transition): the chunk map S -> gamma_C S + K~^T (Ubar - W S)
// is affine in S, so a superchunk of chunks maps S_J to S_{J+1} = M_J S_J + N_J
// with dense M_J, N_J in R^{Dk x Dk}, R^{Dk x Dv}.
//   k_gdn_walk<PREP>: walks the superchunk's chunks with the state [M | N]
//     (wave w owns columns [16w, 16w+16) of both; M from the identity with
//     Ubar = 0, N from zero) and writes M_J, N_J.  No outputs.
//   k_gdn_scan: S_{J+1} = M_J S_J + N_J in fp32, sequential over J, 16 state
//     columns per workgroup; writes every S_J and S_out.
//   k_gdn_walk<!PREP>: the output walk above from S_J over superchunk J.
#include "sf_chunk.hpp"

namespace sf {

namespace {

template <typename T, int D, bool PREP>
__global__ void __launch_bounds__(64 * D / 16) k_gdn_walk(GdnArgs a) {
    constexpr int NW = D / 16, NT = 64 * NW, NK = D / 16, NS = PREP ? 2 : 1;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr int LDA = C + 4, LDU = D + 4;  // 16-byte-odd pitches: conflict-free row-varying reads
    __shared__ __attribute__((aligned(16))) T sQ[PREP ? 8 : C * LDN];    // plain
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];               // plain, swizzled
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];               // plain
    __shared__ __attribute__((aligned(16))) T sP[PREP ? 8 : C * LDT];    // (Q K^T o Gamma)[t][s] hi
    __shared__ __attribute__((aligned(16))) T sPl[PREP ? 8 : C * LDT];   // lo
    __shared__ __attribute__((aligned(16))) float sA[C * LDA];    // beta_t e^{b_t-b_s} k_t.k_s, s < t
    __shared__ __attribute__((aligned(16))) float sW[C * LDU];    // W [t][k], fp32
    __shared__ __attribute__((aligned(16))) float sU[C * LDU];    // Ubar [t][v], fp32
    __shared__ __attribute__((aligned(16))) float sb[C], sq[C], se[C], sbeta[C];

    const int tid = threadIdx.x, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c0 = 16 * w;
    // items: (b, h, J) with J < n_super (walk) or J < n_super - 1 (prep)
    const int nJ = PREP ? a.n_super - 1 : a.n_super;
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
        if constexpr (!PREP) t1.load_buf(buf_rsrc(Q + nx, cspan), toff, 0);
        t2.load_buf(buf_rsrc(K + nx, cspan), toff, 0);
        t3.load_buf(buf_rsrc(V + nx, cspan), toff, 0);
        gl = buf_ld<float>(buf_rsrc(gp + (int64_t)c * C * a.sg_l, gspan), goff, 0);
        bl = buf_ld<float>(buf_rsrc(bp + (int64_t)c * C * a.sg_l, gspan), goff, 0);
    };
    if (nch > 0) issue(0);

    for (int c = 0; c < nch; ++c) {
        const float b2 = wave_scan_dpp(gl * LOG2E);
        const float b63 = lane_value(b2, 63);
        const float betal = bl;
        __syncthreads();  // the previous chunk is done with every LDS tile
        if constexpr (!PREP) t1.store_swz(sQ, LDN, tid, 0);
        t2.store_swz(sK, LDN, tid, SWX);
        t3.store_swz(sV, LDN, tid, 0);
        if (w == 0) {
            sb[lane] = b2;
            sq[lane] = fexp2(b2);
            se[lane] = fexp2(b63 - b2);
            sbeta[lane] = betal;
        }
        __syncthreads();
        if (c + 1 < nch) issue(c + 1);

        // scores on the causal tiles: P^T[s][t] = k_s . q_t and k_s . k_t
        for (int i = PREP ? 10 + w : w; i < 20; i += NW) {
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
                if constexpr (!PREP) {
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
        // P tiles above the diagonal that the output product reads are zero
        for (int e = tid; e < (PREP ? 0 : 512); e += NT) {
            const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
            const int row = tile ? 32 + rr : rr, col = tile ? 48 + cc : 16 + cc;
            sP[row * LDT + (col ^ asw(row))] = cvt<T>(0.f);
            sPl[row * LDT + (col ^ asw(row))] = cvt<T>(0.f);
        }
        __syncthreads();

        // (I + A) X = R, forward substitution in fp32, one thread per column of
        // R = [diag(beta gamma) K | diag(beta) V]; X = [W | Ubar] is written to
        // sW / sU, whose column of this thread doubles as its working store.
        // Blocks of 16 rows: the earlier blocks' contribution is a 16 x 16
        // block update from LDS, the diagonal block a 16-row triangular solve in
        // registers (every register index a compile-time constant).
        if (tid < 2 * D) {
            const bool wcol = tid < D;
            const int j = wcol ? tid : tid - D;
            float *xc = (wcol ? sW : sU) + j;  // column j, row stride LDU
            for (int tb = 0; tb < C / 16; ++tb) {
                float xb[16];
#pragma unroll
                for (int tl = 0; tl < 16; ++tl) {
                    const int t = 16 * tb + tl;
                    xb[tl] = wcol ? tof<T>(sK[t * LDN + swz_col(t, j, SWX)]) * sbeta[t] * sq[t]
                                  : tof<T>(sV[t * LDN + j]) * sbeta[t];
                }
                for (int sb = 0; sb < tb; ++sb) {
                    float xs[16];
#pragma unroll
                    for (int e = 0; e < 16; ++e) xs[e] = xc[(16 * sb + e) * LDU];
#pragma unroll
                    for (int tl = 0; tl < 16; ++tl) {
                        const float *ar = &sA[(16 * tb + tl) * LDA + 16 * sb];
#pragma unroll
                        for (int e4 = 0; e4 < 4; ++e4) {
                            const f32x4 av = *reinterpret_cast<const f32x4 *>(ar + 4 * e4);
#pragma unroll
                            for (int u = 0; u < 4; ++u) xb[tl] = fmaf(-av[u], xs[4 * e4 + u], xb[tl]);
                        }
                    }
                }
#pragma unroll
                for (int tl = 1; tl < 16; ++tl) {
                    const float *ar = &sA[(16 * tb + tl) * LDA + 16 * tb];
#pragma unroll
                    for (int e = 0; e < 16; ++e)
                        if (e < tl) xb[tl] = fmaf(-ar[e], xb[e], xb[tl]);
                }
#pragma unroll
                for (int tl = 0; tl < 16; ++tl) xc[(16 * tb + tl) * LDU] = xb[tl];
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
                if constexpr (!PREP) mma2<T, true>(O[tt], fh[0], fl[0], ldfrag(sQ, LDN, 16 * tt, 32 * ks, lane));
            }
        }
        if constexpr (!PREP) {
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
        if (!PREP && VN) {
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
    if (PREP || J == a.n_super - 1) {
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
// writes S_J (J < n_super) to wsS.  Workgroup (b, h, 16-column block); thread
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
    const float *wsM = a.wsM + (int64_t)bh * (nJ - 1) * SS;
    const float *wsN = a.wsN + (int64_t)bh * (nJ - 1) * SS;
    float acc[CPT];
#pragma unroll
    for (int j = 0; j < CPT; ++j) acc[j] = a.S_in ? a.S_in[bh * SS + (int64_t)k * D + col0 + j] : 0.f;
    f32x4 mreg[MV];
    auto fetch = [&](int J) {
        const f32x4 *m = reinterpret_cast<const f32x4 *>(wsM + (int64_t)J * SS);
#pragma unroll
        for (int i = 0; i < MV; ++i) mreg[i] = m[tid + NT * i];
    };
    if (nJ > 1) fetch(0);
    for (int J = 0;; ++J) {
#pragma unroll
        for (int j = 0; j < CPT; ++j) {
            sS[k * 16 + col0 % 16 + j] = acc[j];
            wsS[(int64_t)J * SS + (int64_t)k * D + col0 + j] = acc[j];
        }
        if (J == nJ - 1) break;
        float nv[CPT];
#pragma unroll
        for (int j = 0; j < CPT; ++j) nv[j] = wsN[(int64_t)J * SS + (int64_t)k * D + col0 + j];
#pragma unroll
        for (int i = 0; i < MV; ++i) {
            const int e = 4 * (tid + NT * i);
            *reinterpret_cast<f32x4 *>(&sM[(e / D) * LDM + e % D]) = mreg[i];
        }
        __syncthreads();
        if (J + 2 < nJ) fetch(J + 1);
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
}


template <int D>
hipError_t gdn_fwd_d(const GdnArgs &a, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    const unsigned bh = (unsigned)(a.B * a.H);
    if (a.n_super > 1) {
        hipExtLaunchKernelGGL((k_gdn_walk<__bf16, D, true>), dim3(bh * (a.n_super - 1)), dim3(64 * D / 16), 0, s,
                              e0, nullptr, 0, a);
        hipExtLaunchKernelGGL((k_gdn_scan<D>), dim3(bh * (D / 16)), dim3(256), 0, s, nullptr, nullptr, 0, a);
    }
    hipExtLaunchKernelGGL((k_gdn_walk<__bf16, D, false>), dim3(bh * a.n_super), dim3(64 * D / 16), 0, s,
                          a.n_super > 1 ? nullptr : e0, e1, 0, a);
    return hipGetLastError();
}

}  // namespace

hipError_t launch_gdn_fwd(const GdnArgs &a, int D, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    if (a.n_super < 1 || (a.n_super > 1 && (!a.wsS || !a.wsM || !a.wsN))) return hipErrorInvalidValue;
    if (D == 128) return gdn_fwd_d<128>(a, s, e0, e1);
    if (D == 64) return gdn_fwd_d<64>(a, s, e0, e1);
    return hipErrorInvalidValue;
}

}  // namespace sf
