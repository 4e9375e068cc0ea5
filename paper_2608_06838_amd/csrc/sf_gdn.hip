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
#include "sf_chunk.hpp"

namespace sf {

namespace {

template <typename T, int D>
__global__ void __launch_bounds__(64 * D / 16) k_gdn_walk(GdnArgs a) {
    constexpr int NW = D / 16, NT = 64 * NW, NK = D / 16;
    constexpr int LDN = D + pad<T>(), LDT = C + pad<T>(), SWX = swx<T, D>();
    constexpr int LDA = C, LDU = D;  // unpadded: the LDS budget is 160 KB
    __shared__ __attribute__((aligned(16))) T sQ[C * LDN];    // plain
    __shared__ __attribute__((aligned(16))) T sK[C * LDN];    // plain, swizzled
    __shared__ __attribute__((aligned(16))) T sV[C * LDN];    // plain
    __shared__ __attribute__((aligned(16))) T sP[C * LDT];    // (Q K^T o Gamma)[t][s] hi
    __shared__ __attribute__((aligned(16))) T sPl[C * LDT];   // lo
    __shared__ __attribute__((aligned(16))) float sA[C * LDA];    // beta_t e^{b_t-b_s} k_t.k_s, s < t
    __shared__ __attribute__((aligned(16))) T sW[C * LDN];    // -W hi  [t][k]
    __shared__ __attribute__((aligned(16))) T sWl[C * LDN];   // -W lo
    __shared__ __attribute__((aligned(16))) float sU[C * LDU];    // Ubar [t][v]
    __shared__ __attribute__((aligned(16))) float sb[C], sq[C], se[C], sbeta[C];

    const int tid = threadIdx.x, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    const int c0 = 16 * w;
    const int bh = blockIdx.x, bb = bh / a.H, hh = bh % a.H;
    const int64_t xo = bb * a.sx_b + hh * a.sx_h;
    const T *Q = (const T *)a.q + xo;
    const T *K = (const T *)a.k + xo;
    const T *V = (const T *)a.v + xo;
    T *Y = (T *)a.o + xo;
    const int64_t go = bb * a.sg_b + hh * a.sg_h;
    const float *gp = a.g + go;
    const float *bp = a.beta + go;
    const int64_t SS = (int64_t)D * D;
    const int nch = (int)(a.L / C);
    const LaneOff tro = tr_off<T, LDN, SWX>(lane), swo = swz_off<T, LDN, SWX>(lane);
    auto asw = [](int row) { return sizeof(T) == 2 ? 8 * ((row >> 2) & 1) : 0; };

    f32x4 S[NK];  // S[16i + 4q4 + r][c0 + n16]
#pragma unroll
    for (int i = 0; i < NK; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) S[i][r] = a.S_in ? a.S_in[bh * SS + (int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] : 0.f;

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
        t1.load_buf(buf_rsrc(Q + nx, cspan), toff, 0);
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
        t1.store_swz(sQ, LDN, tid, 0);
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
        for (int i = w; i < 20; i += NW) {
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
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int s = 16 * st + 4 * q4 + r;
                    v4[r] = s <= t ? p[r] * fexp2(bt - bs[r]) : 0.f;
                }
                const int o = t * LDT + ((16 * st + 4 * q4) ^ asw(t));
                st4_split<T, true>(&sP[o], &sPl[o], v4);
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
        for (int e = tid; e < 512; e += NT) {
            const int tile = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
            const int row = tile ? 32 + rr : rr, col = tile ? 48 + cc : 16 + cc;
            sP[row * LDT + (col ^ asw(row))] = cvt<T>(0.f);
            sPl[row * LDT + (col ^ asw(row))] = cvt<T>(0.f);
        }
        __syncthreads();

        // (I + A) X = R, forward substitution in fp32, one thread per column of
        // R = [diag(beta gamma) K | diag(beta) V]; X = [W | Ubar]
        if (tid < 2 * D) {
            const int j = tid < D ? tid : tid - D;
            float x[C];
#pragma unroll
            for (int t = 0; t < C; ++t) {
                const float r = tid < D ? tof<T>(sK[t * LDN + swz_col(t, j, SWX)]) * sbeta[t] * sq[t]
                                        : tof<T>(sV[t * LDN + j]) * sbeta[t];
                float acc = r;
                // constant trip counts (the guards fold once t is unrolled), so
                // x stays in registers
#pragma unroll
                for (int s4 = 0; s4 < C / 4; ++s4) {
                    if (4 * s4 < t) {
                        const f32x4 av = *reinterpret_cast<const f32x4 *>(&sA[t * LDA + 4 * s4]);
#pragma unroll
                        for (int e = 0; e < 4; ++e)
                            if (4 * s4 + e < t) acc = fmaf(-av[e], x[4 * s4 + e], acc);
                    }
                }
                x[t] = acc;
                sched_fence();  // keep each row's A loads next to its arithmetic (no hoisting of all 64 rows)
            }
            if (tid < D) {
#pragma unroll
                for (int t = 0; t < C; ++t) {
                    const float nw = -x[t];
                    const T h = cvt<T>(nw);
                    sW[t * LDN + j] = h;
                    sWl[t * LDN + j] = cvt<T>(nw - tof<T>(h));
                }
            } else {
#pragma unroll
                for (int t = 0; t < C; ++t) sU[t * LDU + j] = x[t];
            }
        }
        __syncthreads();

        // U[t][v] = Ubar[t][v] - sum_k W[t][k] S[k][v]  (rows t = 16tt + 4q4 + r, column v = c0 + n16)
        f32x4 U[4];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) U[tt][r] = sU[(16 * tt + 4 * q4 + r) * LDU + c0 + n16];
        // O^T[v][t] = gamma_t sum_k S[k][v] Q[t][k] + sum_s U[s][v] P[t][s]
        f32x4 O[4];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) O[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            frag_t<T> fh, fl;
            split_acc_plain<T, true>(S[2 * ks], S[2 * ks + 1], fh, fl);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                const frag_t<T> wh = ldfrag(sW, LDN, 16 * tt, 32 * ks, lane);
                const frag_t<T> wl = ldfrag(sWl, LDN, 16 * tt, 32 * ks, lane);
                mma(U[tt], wh, fh);
                mma(U[tt], wh, fl);
                mma(U[tt], wl, fh);
                mma2<T, true>(O[tt], fh, fl, ldfrag(sQ, LDN, 16 * tt, 32 * ks, lane));
            }
        }
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) O[tt] *= sq[16 * tt + n16];
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            frag_t<T> uh, ul;
            split_acc_plain<T, true>(U[2 * ks], U[2 * ks + 1], uh, ul);
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

        // S = gamma_C S + K^T (e^{b_C - b} o U)
        const float gam = fexp2(b63);
#pragma unroll
        for (int i = 0; i < NK; ++i) S[i] *= gam;
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) U[tt][r] *= se[16 * tt + 4 * q4 + r];
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            frag_t<T> uh, ul;
            split_acc_plain<T, true>(U[2 * ks], U[2 * ks + 1], uh, ul);
#pragma unroll
            for (int i = 0; i < NK; ++i) mma2b<T, true>(S[i], ldfragTR<T, LDN, SWX>(sK, tro, 32 * ks, 16 * i), uh, ul);
        }
    }
    if (a.S_out) {
        float *dst = a.S_out + bh * SS;
#pragma unroll
        for (int i = 0; i < NK; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) dst[(int64_t)(16 * i + 4 * q4 + r) * D + c0 + n16] = S[i][r];
    }
}

}  // namespace

hipError_t launch_gdn_fwd(const GdnArgs &a, int D, hipStream_t s, hipEvent_t e0, hipEvent_t e1) {
    const dim3 grid((unsigned)(a.B * a.H));
    if (D == 128) hipExtLaunchKernelGGL((k_gdn_walk<__bf16, 128>), grid, dim3(64 * 128 / 16), 0, s, e0, e1, 0, a);
    else if (D == 64) hipExtLaunchKernelGGL((k_gdn_walk<__bf16, 64>), grid, dim3(64 * 64 / 16), 0, s, e0, e1, 0, a);
    else return hipErrorInvalidValue;
    return hipGetLastError();
}

}  // namespace sf
