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

// Column c of (I + diag(rs) M)^{-1} for a strictly lower 16 x 16 block M
// (row pitch ld; rs == nullptr: rs = 1) by forward substitution in fp32:
// x[r] = [r == c] - rs[r] sum_{s < r} M[r][s] x[s].  Right-looking: once x[s]
// is final, every later row takes its term, so the 120 products form 16
// dependent steps of independent updates instead of one chain.  Each row's sum
// still runs over s in increasing order.
__device__ __forceinline__ void gdn_diag_column(const float *M, int ld, int c, const float *rs, float (&x)[16]) {
    float acc[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) acc[r] = 0.f;
#pragma unroll
    for (int s2 = 0; s2 < 16; ++s2) {
        x[s2] = s2 == c ? 1.f : (s2 > c ? -(rs ? rs[s2] : 1.f) * acc[s2] : 0.f);
#pragma unroll
        for (int r = s2 + 1; r < 16; ++r) acc[r] = fmaf(M[r * ld + s2], x[s2], acc[r]);
    }
}
// The same column, the same sums in the same order (so the same bits), row by
// row for a kernel short of registers (ld a multiple of 4, M 16-byte aligned):
// row r's part left of the diagonal is read with 16-byte loads that do not
// depend on x, and the row scales are read up front, so the rows are selected
// arithmetically (a load under the per-lane condition r > c made every row a
// branch with its own wait).
__device__ __forceinline__ void gdn_diag_column_rows(const float *M, int ld, int c, const float *rs, float (&x)[16]) {
    float rv[16];
#pragma unroll
    for (int r = 0; r < 16; ++r) rv[r] = rs ? rs[r] : 1.f;
#pragma unroll
    for (int r = 0; r < 16; ++r) {
        float acc = 0.f;
#pragma unroll
        for (int m = 0; 4 * m < r; ++m) {
            const f32x4 mv = *reinterpret_cast<const f32x4 *>(M + r * ld + 4 * m);
#pragma unroll
            for (int u = 0; u < 4; ++u)
                if (4 * m + u < r) acc = fmaf(mv[u], x[4 * m + u], acc);
        }
        const float y = -rv[r] * acc;
        x[r] = r > c ? y : (r == c ? 1.f : 0.f);
    }
}

// T = (I + A)^{-1} for the strictly lower 64 x 64 A = diag(rs) M with M in sA
// (pitch C + 4; rs == nullptr: A = M), into sT (fp32, pitch C + 4, zero above
// the diagonal), by 16 x 16 blocks: the four diagonal blocks by forward
// substitution in fp32 (64 threads, one column each); then level by level
// (i - j = 1, 2, 3) wave j forms T_ij = -T_ii sum_{k=j}^{i-1} A_ik T_kj on
// 16x16x16 MFMA with hi/lo operands, the inner sum staying in its
// accumulator, which is already the B operand of the T_ii product.  NT >= 256
// threads (four waves); ends with a barrier.  (The per-chunk gradient kernel's
// form; the walks use gdn_tinv_hl below.)
template <int NT>
__device__ __forceinline__ void gdn_tinv(int tid, const float *sA, float *sT, const float *rs = nullptr) {
    constexpr int LA = C + 4, LT = C + 4;
    if (tid < 64) {
        const int o = 16 * (tid >> 4), c = tid & 15;
        float x[16];
        gdn_diag_column_rows(sA + o * LA + o, LA, c, rs ? rs + o : nullptr, x);
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

// The walks' T = (I + A)^{-1} (A = M in sA, pitch C + 4), stored as the bf16
// hi/lo pair that every consumer splits it into (sTh, sTl: raw 16-bit
// patterns, pitch C + 16, zero above the diagonal): the four diagonal blocks
// by forward substitution in fp32 (64 threads, one column each), the
// off-diagonal blocks level by level as in gdn_tinv, reading the stored pairs.
// (A diagonal block N is nilpotent, and (I + N)^{-1} = (I + N^8)(I + N^4)
// (I + N^2)(I - N) on MFMA ran the walks 4% faster; but the series' partial
// sums grow like binomial coefficients when neighbouring keys are nearly
// parallel with little decay, and the outputs then lost up to 1e-1 (bf16
// hi/lo operands) or 1e-3 (fp32 MFMA) against the oracle, where substitution
// keeps them at output rounding.)  NT >= 256 threads; ends with a barrier.
template <int NT>
__device__ __forceinline__ void gdn_tinv_hl(int tid, const float *sA, short *sTh, short *sTl) {
    constexpr int LA = C + 4, LTB = C + 16;
    const int w = tid >> 6, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    // rows row0 .. row0+3 of column col (the B layout), as hi/lo
    auto put = [&](int row0, int col, const f32x4 &x) {
        s4v h, l;
        split4(x, h, l);
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            sTh[(row0 + r) * LTB + col] = h[r];
            sTl[(row0 + r) * LTB + col] = l[r];
        }
    };
    if (tid < 64) {  // one column of a diagonal block per thread
        const int o = 16 * (tid >> 4), c = tid & 15;
        float x[16];
        gdn_diag_column(sA + o * LA + o, LA, c, nullptr, x);
#pragma unroll
        for (int r = 0; r < 16; ++r) {
            const __bf16 h = (__bf16)x[r];
            sTh[(o + r) * LTB + o + c] = __builtin_bit_cast(short, h);
            sTl[(o + r) * LTB + o + c] = __builtin_bit_cast(short, (__bf16)(x[r] - (float)h));
        }
    }
    for (int e = tid; e < 6 * 256; e += NT) {  // blocks (0,1) (0,2) (0,3) (1,2) (1,3) (2,3)
        const int b = e >> 8, rr = (e >> 4) & 15, cc = e & 15;
        const int bi = b < 3 ? 0 : (b < 5 ? 1 : 2), bj = b < 3 ? b + 1 : (b < 5 ? b - 1 : 3);
        sTh[(16 * bi + rr) * LTB + 16 * bj + cc] = 0;
        sTl[(16 * bi + rr) * LTB + 16 * bj + cc] = 0;
    }
    __syncthreads();
#pragma unroll
    for (int d = 1; d < 4; ++d) {
        if (w < 4 - d) {  // block (i, j) = (d + w, w)
            const int i = d + w, j = w;
            f32x4 y = {0.f, 0.f, 0.f, 0.f};
            for (int k = j; k < i; ++k) {
                const f32x4 av = *reinterpret_cast<const f32x4 *>(&sA[(16 * i + n16) * LA + 16 * k + 4 * q4]);
                s4v ah, al, bh = {0, 0, 0, 0}, bl = bh;
                split4(av, ah, al);
#pragma unroll
                for (int u = 0; u < 4; ++u) {
                    bh[u] = sTh[(16 * k + 4 * q4 + u) * LTB + 16 * j + n16];
                    bl[u] = sTl[(16 * k + 4 * q4 + u) * LTB + 16 * j + n16];
                }
                mma16(y, ah, bh);
                mma16(y, ah, bl);
                mma16(y, al, bh);
            }
            const s4v th = *reinterpret_cast<const s4v *>(&sTh[(16 * i + n16) * LTB + 16 * i + 4 * q4]);
            const s4v tl = *reinterpret_cast<const s4v *>(&sTl[(16 * i + n16) * LTB + 16 * i + 4 * q4]);
            s4v yh, yl;
            split4(y, yh, yl);
            f32x4 t = {0.f, 0.f, 0.f, 0.f};
            mma16(t, th, yh);
            mma16(t, th, yl);
            mma16(t, tl, yh);
            put(16 * i + 4 * q4, 16 * j + n16, -t);
        }
        __syncthreads();
    }
}

// [W | Ubar] = T [diag(beta gamma) K | diag(beta) V] on MFMA: wave w forms
// columns [16w, 16w+16) of W (and of Ubar when sU is given); T enters as its
// stored hi/lo pair (gdn_tinv_hl), the scaled K and V columns as hi/lo pairs too (K, V exact in bf16 times an fp32
// factor).  Results: -W as a bf16 hi/lo pair (sWh, sWl: natural [t][k] tiles,
// pitch LDN, channel blocks of rows with bit 3 set XOR-swizzled by SWX, the
// layout of the staged q/k tiles), split once here for every wave that reads
// it; Ubar to sU (fp32, pitch LDU).
template <typename T, int D, int LDN, int LDU, int SWX>
__device__ __forceinline__ void gdn_wu(int w, int lane, const LaneOff &tro, const short *sTh, const short *sTl,
                                       const T *sK, const T *sV,
                                       const float *sbeta, const float *sq, T *sWh, T *sWl, float *sU) {
    constexpr int LTB = C + 16;
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
            const int pt = (16 * tt + n16) * LTB + 32 * ks + 8 * q4;
            const frag_t<T> th = *reinterpret_cast<const frag_t<T> *>(sTh + pt);
            const frag_t<T> tl = *reinterpret_cast<const frag_t<T> *>(sTl + pt);
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
            const int t = 16 * tt + 4 * q4 + r, pw = t * LDN + swz_col(t, c0 + n16, SWX);
            const float x = -cw[tt][r];
            const T h = cvt<T>(x);
            sWh[pw] = h;
            sWl[pw] = cvt<T>(x - tof<T>(h));
            if (sU) sU[t * LDU + c0 + n16] = cu[tt][r];
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
    __shared__ __attribute__((aligned(16))) T sTx[OUTP ? 8 : 2 * C * LDT];
    static_assert(LDT == C + 16, "T's hi/lo pair has the P tiles' pitch");
    T *sP = sPP, *sPl = sPP + (OUTP ? C * LDT : 0);
    short *const sTh = reinterpret_cast<short *>(OUTP ? sPP : sTx), *const sTl = sTh + C * LDT;
    // A = beta_t e^{b_t-b_s} k_t.k_s (s < t, fp32) until the inverse is formed; then -W
    // as a hi/lo pair of bf16 tiles in the same bytes
    constexpr int AWB = C * LDA * 4 > 2 * C * LDN * (int)sizeof(T) ? C * LDA * 4 : 2 * C * LDN * (int)sizeof(T);
    __shared__ __attribute__((aligned(16))) char sAW[AWB];
    float *const sA = reinterpret_cast<float *>(sAW);
    T *const sWh = reinterpret_cast<T *>(sAW), *const sWl = sWh + C * LDN;
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
    const LaneOff tro8 = tr_off8<T, LDN, SWX>(lane);
    auto asw = [](int row) { return sizeof(T) == 2 ? 8 * ((row >> 2) & 1) : 0; };
    // Accumulator pairs (2m, 2m+1) of the state (rows: key channels) and of U
    // (rows: tokens) hold, in lane row q4, indices 32m + 8 q4 .. +7 (slot r of
    // tile i: prow(i, r)), so each pair splits into an operand fragment in plain
    // order with no lane swaps.  The products that build them read their A rows
    // in that order: fragment row n of tile i is prow(i, n / 4, n % 4).
    auto prow = [&](int i, int r) { return 32 * (i >> 1) + 8 * q4 + 4 * (i & 1) + r; };
    auto arow = [](int i, int n) { return 32 * (i >> 1) + 8 * (n >> 2) + 4 * (i & 1) + (n & 3); };
    auto roff = [](int i) { return 32 * (i >> 1) + 4 * (i & 1); };  // ldfragTR column for tro8

    // S[m][prow(i, r)][c0 + n16]: the walk's state starts from S_J (S_in for
    // one superchunk); the prep's M (m = 0) from I and its N (m = 1) from 0
    const float *src = a.n_super == 1 ? a.S_in + (a.S_in ? bh * SS : 0) : a.wsS + (int64_t)item * SS;
    f32x4 S[NS][NK];
#pragma unroll
    for (int i = 0; i < NK; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int row = prow(i, r);
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
                for (int r = 0; r < 4; ++r) dst[(int64_t)prow(i, r) * D + c0 + n16] = S[0][i][r];
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
        gdn_tinv_hl<NT>(tid, sA, sTh, sTl);
        gdn_wu<T, D, LDN, LDU, SWX>(w, lane, tro, sTh, sTl, sK, sV, sbeta, sq, sWh, sWl, sU);
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

        // U[t][v] = Ubar[t][v] - sum_k W[t][k] S[k][v]  (rows t = prow(tt, r), column v = c0 + n16);
        // the prep's M columns take Ubar = 0
        f32x4 U[NS][4];
#pragma unroll
        for (int m = 0; m < NS; ++m)
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    U[m][tt][r] = PREP && m == 0 ? 0.f : sU[prow(tt, r) * LDU + c0 + n16];
        // O^T[v][t] = gamma_t sum_k S[k][v] Q[t][k] + sum_s U[s][v] P[t][s]
        f32x4 O[4];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) O[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            frag_t<T> fh[NS], fl[NS];
#pragma unroll
            for (int m = 0; m < NS; ++m) split_acc<T, true>(S[m][2 * ks], S[m][2 * ks + 1], fh[m], fl[m]);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                // -W[t][32ks + 8q4 .. +7], t = arow(tt, n16), as its hi/lo pair
                const int t = arow(tt, n16), pw = t * LDN + swz_col(t, 32 * ks + 8 * q4, SWX);
                const frag_t<T> wh = *reinterpret_cast<const frag_t<T> *>(&sWh[pw]);
                const frag_t<T> wl = *reinterpret_cast<const frag_t<T> *>(&sWl[pw]);
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
                split_acc<T, true>(U[0][2 * ks], U[0][2 * ks + 1], uh, ul);
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

        // V^new (optional): U[prow(tt, r)][c0 + n16]
        if (OUTP && VN) {
#pragma unroll
            for (int tt = 0; tt < 4; ++tt)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    VN[(int64_t)(c * C + prow(tt, r)) * a.sx_l + c0 + n16] = cvt<T>(U[0][tt][r]);
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
                for (int r = 0; r < 4; ++r) U[m][tt][r] *= se[prow(tt, r)];
        }
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            frag_t<T> uh[NS], ul[NS];
#pragma unroll
            for (int m = 0; m < NS; ++m) split_acc<T, true>(U[m][2 * ks], U[m][2 * ks + 1], uh[m], ul[m]);
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                const frag_t<T> kf = ldfragTR<T, LDN, SWX>(sK, tro8, 32 * ks, roff(i));
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
                for (int r = 0; r < 4; ++r) dst[(int64_t)prow(i, r) * D + c0 + n16] = S[m][i][r];
        }
    }
}

// S_{J+1} = M_J S_J + N_J for J = 0 .. n_super - 2 in fp32, S_0 = S_in (or 0);
// writes S_J (J < n_super) to wsS; with scan_out (maps of every superchunk)
// one more step gives S_out.  Workgroup (b, h, 16-column block), four waves;
// wave w owns the row tiles RTW w .. RTW w + RTW - 1 of the block, and the
// product runs on the fp32 MFMA (16x16x4, fp32 products and sums): in step m
// of the contraction lane (q4, n16) supplies M[row n16][KQ q4 + m] and
// S[KQ q4 + m][col n16], the same order on both sides, so a lane's M operands
// are KQ consecutive floats of its row.  M_J is staged in LDS (row pitch
// D + 4 floats) with the next one prefetched in registers; S_J sits in LDS
// (pitch 17) for the B operands.
template <int D>
__global__ void __launch_bounds__(256) k_gdn_scan(GdnArgs a) {
    constexpr int NT = 256, LDM = D + 4, MV = D * D / 4 / NT, RTW = D / 64, KQ = D / 4, LS = 17;
    __shared__ __attribute__((aligned(16))) float sM[D * LDM];
    __shared__ float sS[D * LS];
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int bh = blockIdx.x / (D / 16), col0 = 16 * (blockIdx.x % (D / 16));
    const int64_t SS = (int64_t)D * D;
    const int nJ = a.n_super;
    float *wsS = a.wsS + (int64_t)bh * nJ * SS;
    const float *wsM = a.wsM + (int64_t)bh * a.n_prep * SS;
    const float *wsN = a.wsN + (int64_t)bh * a.n_prep * SS;
    auto row = [&](int i, int r) { return 16 * (RTW * w + i) + 4 * q4 + r; };
    f32x4 acc[RTW];  // S[row(i, r)][col0 + n16]
#pragma unroll
    for (int i = 0; i < RTW; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][r] = a.S_in ? a.S_in[bh * SS + (int64_t)row(i, r) * D + col0 + n16] : 0.f;
    // M_J and N_J two steps ahead, in two register sets used alternately
    f32x4 mA[MV], mB[MV];
    float nA[RTW][4], nB[RTW][4];
    auto fetch = [&](f32x4 (&mr)[MV], float (&nr)[RTW][4], int J) {
        const f32x4 *m = reinterpret_cast<const f32x4 *>(wsM + (int64_t)J * SS);
#pragma unroll
        for (int i = 0; i < MV; ++i) mr[i] = m[tid + NT * i];
#pragma unroll
        for (int i = 0; i < RTW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) nr[i][r] = wsN[(int64_t)J * SS + (int64_t)row(i, r) * D + col0 + n16];
    };
    const int last = a.scan_out ? nJ : nJ - 1;  // steps taken
    // S_J and S_out go out through buffer stores (32-bit lane offsets)
    const rsrc_t rS = buf_rsrc(wsS, (uint32_t)(nJ * SS * 4));
    // step J: store S_J; unless J is the last, S_{J+1} = M_J S_J + N_J from
    // (mr, nr), which then take the maps of J + 2; false after the last store
    auto step = [&](int J, f32x4 (&mr)[MV], float (&nr)[RTW][4]) {
#pragma unroll
        for (int i = 0; i < RTW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                sS[row(i, r) * LS + n16] = acc[i][r];
                buf_st(rS, (uint32_t)((row(i, r) * D + col0 + n16) * 4), (uint32_t)(J * SS * 4), acc[i][r]);
            }
        if (J == last) return false;
#pragma unroll
        for (int i = 0; i < MV; ++i) {
            const int e = 4 * (tid + NT * i);
            *reinterpret_cast<f32x4 *>(&sM[(e / D) * LDM + e % D]) = mr[i];
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < RTW; ++i) acc[i] = f32x4{nr[i][0], nr[i][1], nr[i][2], nr[i][3]};
        if (J + 2 < last) fetch(mr, nr, J + 2);
#pragma unroll 2
        for (int m = 0; m < KQ; m += 4) {
            float bv[4];
#pragma unroll
            for (int u = 0; u < 4; ++u) bv[u] = sS[(KQ * q4 + m + u) * LS + n16];
#pragma unroll
            for (int i = 0; i < RTW; ++i) {
                const f32x4 av = *reinterpret_cast<const f32x4 *>(&sM[(16 * (RTW * w + i) + n16) * LDM + KQ * q4 + m]);
#pragma unroll
                for (int u = 0; u < 4; ++u) acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(av[u], bv[u], acc[i], 0, 0, 0);
            }
        }
        __syncthreads();  // every read of sM and sS is done
        return true;
    };
    if (last > 0) fetch(mA, nA, 0);
    if (last > 1) fetch(mB, nB, 1);
    for (int J = 0;; J += 2)
        if (!step(J, mA, nA) || !step(J + 1, mB, nB)) break;
    if (a.scan_out) {  // the state after the last superchunk
        const rsrc_t rO = buf_rsrc(a.S_out + bh * SS, (uint32_t)(SS * 4));
#pragma unroll
        for (int i = 0; i < RTW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) buf_st(rO, (uint32_t)((row(i, r) * D + col0 + n16) * 4), 0u, acc[i][r]);
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
    static_assert(LDT == C + 16, "T's hi/lo pair has the P tiles' pitch");
    T *sP = sPP, *sPl = sPP + C * LDT;
    short *const sTh = reinterpret_cast<short *>(sPP), *const sTl = sTh + C * LDT;
    // A until the inverse is formed, then -W as a hi/lo pair of bf16 tiles (see the walk)
    constexpr int AWB = C * LDA * 4 > 2 * C * LDN * (int)sizeof(T) ? C * LDA * 4 : 2 * C * LDN * (int)sizeof(T);
    __shared__ __attribute__((aligned(16))) char sAW[AWB];
    float *const sA = reinterpret_cast<float *>(sAW);
    T *const sWh = reinterpret_cast<T *>(sAW), *const sWl = sWh + C * LDN;
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
    const LaneOff tro8 = tr_off8<T, LDN, SWX>(lane);
    auto asw = [](int row) { return sizeof(T) == 2 ? 8 * ((row >> 2) & 1) : 0; };
    // Accumulator pairs (2m, 2m+1) of dS (rows: key channels) and of dU (rows:
    // tokens) hold, in lane row q4, indices 32m + 8 q4 .. +7 (slot r of tile i:
    // prow(i, r)), so each pair splits into an operand fragment in plain order
    // with no lane swaps; the products that build them read their A rows in that
    // order (fragment row n of tile i: arow(i, n)).
    auto prow = [&](int i, int r) { return 32 * (i >> 1) + 8 * q4 + 4 * (i & 1) + r; };
    auto arow = [](int i, int n) { return 32 * (i >> 1) + 8 * (n >> 2) + 4 * (i & 1) + (n & 3); };
    auto roff = [](int i) { return 32 * (i >> 1) + 4 * (i & 1); };  // ldfragTR column for tro8

    // dS[prow(i, r)][c0 + n16]: from dS_end(J) (dS_out for one superchunk), or 0 (prep)
    f32x4 dS[NK];
    {
        const float *src = a.n_super == 1 ? (a.dS_out ? a.dS_out + bh * SS : nullptr)
                                          : a.wsDe + ((int64_t)bh * a.n_super + J) * SS;
#pragma unroll
        for (int i = 0; i < NK; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r)
                dS[i][r] = (!PREP && src) ? src[(int64_t)prow(i, r) * D + c0 + n16] : 0.f;
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
                for (int r = 0; r < 4; ++r) dst[(int64_t)prow(i, r) * D + c0 + n16] = dS[i][r];
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
        gdn_tinv_hl<NT>(tid, sA, sTh, sTl);
        gdn_wu<T, D, LDN, LDU, SWX>(w, lane, tro, sTh, sTl, sK, (const T *)nullptr, sbeta, sq, sWh, sWl, nullptr);
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
        // (rows t = prow(tt, r), column v = c0 + n16)
        f32x4 dU[4];
#pragma unroll
        for (int tt = 0; tt < 4; ++tt) dU[tt] = f32x4{0.f, 0.f, 0.f, 0.f};
#pragma unroll
        for (int ks = 0; ks < D / 32; ++ks) {
            frag_t<T> fh, fl;
            split_acc<T, true>(dS[2 * ks], dS[2 * ks + 1], fh, fl);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                const int t = arow(tt, n16);  // K[t][32ks + 8q4 ..] (swizzled rows)
                const frag_t<T> kf =
                    *reinterpret_cast<const frag_t<T> *>(&sK[t * LDN + swz_col(t, 32 * ks + 8 * q4, SWX)]);
                mma(dU[tt], kf, fh);
                mma(dU[tt], kf, fl);
            }
        }
#pragma unroll
        for (int tt = 0; tt < 4; ++tt)
#pragma unroll
            for (int r = 0; r < 4; ++r) dU[tt][r] *= se[prow(tt, r)];
#pragma unroll
        for (int ks = 0; ks < C / 32; ++ks) {
            const frag_t<T> of = ldfragTR<T, LDN, SWX>(sO, tro, 32 * ks, c0);
#pragma unroll
            for (int tt = 0; tt < 4; ++tt) {
                if (32 * ks + 31 < 16 * tt) continue;
                const int row = arow(tt, n16);
                const int o = row * LDT + ((32 * ks + 8 * (lane >> 4)) ^ asw(row));
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
            f32x4 g0, g1;  // gamma_t dO[t][c0 + n16], t = 32ks + 8q4 + 4h + r
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int ta = 32 * ks + 8 * q4 + r, tb = ta + 4;
                g0[r] = sq[ta] * tof<T>(sO[ta * LDN + swz_col(ta, c0 + n16, SWX)]);
                g1[r] = sq[tb] * tof<T>(sO[tb * LDN + swz_col(tb, c0 + n16, SWX)]);
            }
            frag_t<T> gh, glo, uh, ul;
            split_acc<T, true>(g0, g1, gh, glo);
            split_acc<T, true>(dU[2 * ks], dU[2 * ks + 1], uh, ul);
#pragma unroll
            for (int i = 0; i < NK; ++i) {
                mma2b<T, true>(dS[i], ldfragTR<T, LDN, SWX>(sQ, tro8, 32 * ks, roff(i)), gh, glo);
                // -W[t][k] hi/lo, k = arow(i, lane % 16), t = 32ks + 8 (lane / 16) + j
                const frag_t<T> wh = ldfragTR<T, LDN, SWX>(sWh, tro8, 32 * ks, roff(i));
                const frag_t<T> wl = ldfragTR<T, LDN, SWX>(sWl, tro8, 32 * ks, roff(i));
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
            for (int r = 0; r < 4; ++r) dst[(int64_t)prow(i, r) * D + c0 + n16] = dS[i][r];
    }
}

// dS_end(n-1) = dS_out (or 0); dS_end(J-1) = M_J^T dS_end(J) + E_J, written to
// wsDe for every J.  Same shape of work as k_gdn_scan, with M_J read
// transposed: in step m lane (q4, n16) supplies M[4 m + q4][row n16] (the
// pitch D + 16 spreads the four q4 rows over the banks) and dS[4 m + q4][col].
template <int D>
__global__ void __launch_bounds__(256) k_gdn_dscan(GdnArgs a) {
    constexpr int NT = 256, LDM = D + 16, MV = D * D / 4 / NT, RTW = D / 64, LS = 17;
    __shared__ __attribute__((aligned(16))) float sM[D * LDM];
    __shared__ float sS[D * LS];
    const int tid = threadIdx.x, w = tid >> 6, lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const int bh = blockIdx.x / (D / 16), col0 = 16 * (blockIdx.x % (D / 16));
    const int64_t SS = (int64_t)D * D;
    const int nJ = a.n_super;
    float *wsDe = a.wsDe + (int64_t)bh * nJ * SS;
    const float *wsM = a.wsM + (int64_t)bh * a.n_prep * SS;
    const float *wsE = a.wsE + (int64_t)bh * (nJ - 1) * SS;
    auto row = [&](int i, int r) { return 16 * (RTW * w + i) + 4 * q4 + r; };
    f32x4 acc[RTW];  // dS[row(i, r)][col0 + n16]
#pragma unroll
    for (int i = 0; i < RTW; ++i)
#pragma unroll
        for (int r = 0; r < 4; ++r) acc[i][r] = a.dS_out ? a.dS_out[bh * SS + (int64_t)row(i, r) * D + col0 + n16] : 0.f;
    // M_J and E_{J-1} two steps ahead, in two register sets used alternately
    f32x4 mA[MV], mB[MV];
    float nA[RTW][4], nB[RTW][4];
    auto fetch = [&](f32x4 (&mr)[MV], float (&nr)[RTW][4], int J) {
        const f32x4 *m = reinterpret_cast<const f32x4 *>(wsM + (int64_t)J * SS);
#pragma unroll
        for (int i = 0; i < MV; ++i) mr[i] = m[tid + NT * i];
#pragma unroll
        for (int i = 0; i < RTW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) nr[i][r] = wsE[(int64_t)(J - 1) * SS + (int64_t)row(i, r) * D + col0 + n16];
    };
    // step J: store dS_end(J); unless J = 0, dS_end(J-1) = M_J^T dS_end(J) +
    // E_{J-1} from (mr, nr), which then take the maps of J - 2; false after J = 0
    auto step = [&](int J, f32x4 (&mr)[MV], float (&nr)[RTW][4]) {
#pragma unroll
        for (int i = 0; i < RTW; ++i)
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                sS[row(i, r) * LS + n16] = acc[i][r];
                wsDe[(int64_t)J * SS + (int64_t)row(i, r) * D + col0 + n16] = acc[i][r];
            }
        if (J == 0) return false;
#pragma unroll
        for (int i = 0; i < MV; ++i) {
            const int e = 4 * (tid + NT * i);
            *reinterpret_cast<f32x4 *>(&sM[(e / D) * LDM + e % D]) = mr[i];
        }
        __syncthreads();
#pragma unroll
        for (int i = 0; i < RTW; ++i) acc[i] = f32x4{nr[i][0], nr[i][1], nr[i][2], nr[i][3]};
        if (J - 2 >= 1) fetch(mr, nr, J - 2);
#pragma unroll 4
        for (int m = 0; m < D / 4; ++m) {
            const float bv = sS[(4 * m + q4) * LS + n16];
#pragma unroll
            for (int i = 0; i < RTW; ++i)
                acc[i] = __builtin_amdgcn_mfma_f32_16x16x4f32(sM[(4 * m + q4) * LDM + 16 * (RTW * w + i) + n16], bv, acc[i],
                                                              0, 0, 0);
        }
        __syncthreads();
        return true;
    };
    if (nJ > 1) fetch(mA, nA, nJ - 1);
    if (nJ > 2) fetch(mB, nB, nJ - 2);
    for (int J = nJ - 1;; J -= 2)
        if (!step(J, mA, nA) || !step(J - 1, mB, nB)) break;
}

// Parameter gradients of one chunk per item (b, h, chunk), items in a
// grid-stride loop, one workgroup of 16 waves per CU.  S is the state entering
// the chunk and dS' the gradient of the state leaving it (both stored per chunk
// by the walks).  The value channels go in blocks of VB = 32 columns: each
// block of S and dS' is read from memory once and staged in LDS, and every
// contraction over the value channels accumulates in registers across the
// blocks.  Two identities keep W = T diag(beta gamma) K and Ubar out of the
// kernel (and out of memory):
//   U_J = Ubar_J - W S_J = T diag(beta) (V_J - diag(gamma) K S_J),
//   G_W = T^T (-dU S^T) = -G_U S^T,   dA = -(G_W W^T + G_U Ubar^T) = -G_U U^T.
// Per block J, waves 0-7 (group A) and 8-15 (group B):
//   A: Y = K S_J, R = diag(beta) (V_J - diag(gamma) Y), U_J = T R;
//   B: dU_J = diag(e) K dS'_J + P^T dO_J, G_U,J = T^T dU_J (dv_J = beta G_U,J);
//   A: G_W -= G_U,J S_J^T, dK_S += U_J dS'_J^T;
//   B: dQ_S += dO_J S_J^T, dA -= G_U,J U_J^T, dP += dO_J U_J^T.
// After the blocks (Gamma[t][s] = e^{b_t - b_s}, Ah = dA o beta_t Gamma):
//   dq = diag(gamma) dQ_S + (dP o Gamma) K                                (B)
//   dk = diag(e) dK_S + (dP o Gamma)^T Q + diag(beta gamma) G_W + (Ah + Ah^T) K   (A)
// and dbeta and the log-decay gradient from row and column sums in a fixed
// order (no atomics).  q, k, v, dO enter the products exactly (bf16); the
// computed fp32 operands (S, dS', T, P, R, U, dU, G_U, dP o Gamma, Ah) as
// hi/lo bf16 pairs (three products, lo x lo dropped).
template <typename T, int D>
__global__ void __launch_bounds__(1024) k_gdn_dchunk(GdnArgs a) {
    constexpr int NTH = 1024, VB = 32, NBLK = D / VB, NTW = D / 32;
    constexpr int LDX = D + 8, LD6 = C + 4, LDB = VB + 4, LDV = VB + 8, LDOT = C + 8, LDU = VB + 4, LDR = VB + 1;
    constexpr int NBLKF = 2 * D * LDB > 2 * C * LD6 ? 2 * D * LDB : 2 * C * LD6;
    static_assert(2 * C * LDR <= C * LD6, "R and dU fit in the scores' buffer");
    __shared__ __attribute__((aligned(16))) T xq[C * LDX], xk[C * LDX];
    __shared__ __attribute__((aligned(16))) float sT[C * LD6];  // T = (I + A)^{-1}
    __shared__ __attribute__((aligned(16))) float sP[C * LD6];  // P[t][s] = e^{b_t - b_s} q_t.k_s, s <= t
    __shared__ __attribute__((aligned(16))) float sX[C * LD6];  // KK o Gamma (s < t) for the inverse; then R, dU
    __shared__ __attribute__((aligned(16))) float sBlk[NBLKF];  // S_J, dS'_J; after the blocks dP o Gamma, Ah + Ah^T
    __shared__ __attribute__((aligned(16))) T sV[C * LDV], sO[C * LDV], sOt[VB * LDOT];
    __shared__ __attribute__((aligned(16))) float sU[C * LDU], sGU[C * LDU];
    __shared__ float sb[C], sg[C], se[C], sbe[C];
    __shared__ float sRow[6][2][C];  // row-sum partials, two waves per row tile
    __shared__ float sCol[4][C];     // column-sum partials, one per row tile
    __shared__ float sWav[16];

    // S_J and dS'_J of the block as hi/lo bf16 pairs, split once when staged:
    // [k'][v] tiles of VB = 32 channels (64-byte rows), the 16-byte channel blocks
    // of row r XOR-swizzled by (r / 4) % 4
    static_assert(VB == 32 && 4 * D * VB * (int)sizeof(T) <= NBLKF * 4, "block tiles fit sBlk");
    T *const sSh = reinterpret_cast<T *>(sBlk), *const sSl = sSh + D * VB;
    T *const sDh = sSl + D * VB, *const sDl = sDh + D * VB;
    auto bpos = [](int r, int ch) { return r * VB + ((((ch >> 3) ^ (r >> 2)) & 3) << 3) + (ch & 7); };
    // T, once formed, as a hi/lo pair of C x C bf16 tiles in its own bytes (128-byte
    // rows, the 16-byte blocks of row r XOR-swizzled by r % 8)
    static_assert(2 * C * C * (int)sizeof(T) <= C * LD6 * 4, "T's pair fits its fp32 bytes");
    T *const sTh = reinterpret_cast<T *>(sT), *const sTl = sTh + C * C;
    auto tpos = [](int r, int c) { return r * C + ((((c >> 3) ^ r) & 7) << 3) + (c & 7); };
    float *const sE1 = sBlk, *const sE2 = sBlk + C * LD6;      // dP o Gamma, Ah + Ah^T
    float *const sR = sX, *const sdU = sX + C * LDR;           // [t][v] of the block

    const int tid = threadIdx.x;
    const int w = __builtin_amdgcn_readfirstlane(tid >> 6);
    int lane = tid & 63, q4 = lane >> 4, n16 = lane & 15;
    const bool grpB = w >= 8;
    const int wg = w & 7, mt = wg & 3, half = wg >> 2;  // row tile; which half of the column tiles
    const int64_t SS = (int64_t)D * D;
    const int nc = (int)(a.L / C);
    const int64_t items = (int64_t)a.B * a.H * nc;

    // fragments: rows row0 + n16, contraction k0 + 8 q4 + j (j < 8)
    auto x_rm = [&](const T *M, int ld, int row0, int k0) {  // exact, M[row][k]
        return *reinterpret_cast<const frag_t<T> *>(M + (row0 + n16) * ld + k0 + 8 * q4);
    };
    auto x_tr = [&](const T *M, int ld, int row0, int k0) {  // exact, M[k][row]
        frag_t<T> f = {};
#pragma unroll
        for (int j = 0; j < 8; ++j) f[j] = M[(k0 + 8 * q4 + j) * ld + row0 + n16];
        return f;
    };
    auto f_rm = [&](const float *M, int ld, int row0, int k0, frag_t<T> &h, frag_t<T> &l) {  // M[row][k], split
        const float *p = M + (row0 + n16) * ld + k0 + 8 * q4;
        const f32x4 x0 = *reinterpret_cast<const f32x4 *>(p), x1 = *reinterpret_cast<const f32x4 *>(p + 4);
        const float x[8] = {x0[0], x0[1], x0[2], x0[3], x1[0], x1[1], x1[2], x1[3]};
        split8<T, true>(x, h, l);
    };
    auto f_tr = [&](const float *M, int ld, int row0, int k0, frag_t<T> &h, frag_t<T> &l) {  // M[k][row], split
        float x[8];
#pragma unroll
        for (int j = 0; j < 8; ++j) x[j] = M[(k0 + 8 * q4 + j) * ld + row0 + n16];
        split8<T, true>(x, h, l);
    };
    // from a block tile [k'][v] (bpos layout): rows row0 + n16 over channels
    // 8 q4 .. +7 (b_rm), or rows = channels c0 + n16 over k0 + 8 q4 + j through
    // two transposing reads (b_tr; the lane map of ldfragTR)
    auto b_rm = [&](const T *M, int row0) {
        return *reinterpret_cast<const frag_t<T> *>(M + bpos(row0 + n16, 8 * q4));
    };
    auto b_tr = [&](const T *M, int k0, int c0) {
        typedef short s4 __attribute__((ext_vector_type(4)));
        typedef short s8 __attribute__((ext_vector_type(8)));
        const int ch = c0 + 4 * (lane & 3), r0 = k0 + 8 * q4 + ((lane & 15) >> 2);
        const s4 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)(M + bpos(r0, ch)));
        const s4 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)(M + bpos(r0 + 4, ch)));
        const s8 v = __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(frag_t<T>, v);
    };
    // the same two forms from T's tiles (tpos layout)
    auto t_rm = [&](const T *M, int row0, int k0) {
        return *reinterpret_cast<const frag_t<T> *>(M + tpos(row0 + n16, k0 + 8 * q4));
    };
    auto t_tr = [&](const T *M, int k0, int c0) {
        typedef short s4 __attribute__((ext_vector_type(4)));
        typedef short s8 __attribute__((ext_vector_type(8)));
        const int ch = c0 + 4 * (lane & 3), r0 = k0 + 8 * q4 + ((lane & 15) >> 2);
        const s4 x0 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)(M + tpos(r0, ch)));
        const s4 x1 = __builtin_amdgcn_ds_read_tr16_b64_v4i16((__attribute__((address_space(3))) s4 *)(M + tpos(r0 + 4, ch)));
        const s8 v = __builtin_shufflevector(x0, x1, 0, 1, 2, 3, 4, 5, 6, 7);
        return __builtin_bit_cast(frag_t<T>, v);
    };
    auto mma3 = [](f32x4 &c, const frag_t<T> &ah, const frag_t<T> &al, const frag_t<T> &bh, const frag_t<T> &bl) {
        mma(c, ah, bh);
        mma(c, ah, bl);
        mma(c, al, bh);
    };
    auto rowsum16 = [](float v) {  // sum over the 16 lanes of a row group
#pragma unroll
        for (int m = 1; m < 16; m <<= 1) v += __shfl_xor(v, m);
        return v;
    };
    const f32x4 z4 = {0.f, 0.f, 0.f, 0.f};

    for (int64_t it = blockIdx.x; it < items; it += gridDim.x) {
        // the lane index, opaque per item: the many per-lane LDS addresses are
        // recomputed where they are used instead of being hoisted out of the
        // item loop (where they would not fit the 128 registers of 16 waves)
        asm volatile("" : "+v"(lane));
        q4 = lane >> 4;
        n16 = lane & 15;
        const int bh = (int)(it / nc), ch = (int)(it % nc), bb = bh / a.H, hh = bh % a.H;
        const int64_t xo0 = bb * a.sx_b + hh * a.sx_h + (int64_t)ch * C * a.sx_l;
        const int64_t go0 = bb * a.sg_b + hh * a.sg_h + (int64_t)ch * C * a.sg_l;
        const float *Sg = a.wsSc + ((int64_t)bh * nc + ch) * SS;
        const float *dSg = a.wsDc + ((int64_t)bh * nc + ch) * SS;
        const T *Vg = (const T *)a.v + xo0, *Og = (const T *)a.dO + xo0;

        // block staging: S_J and dS'_J as D x VB floats (one 16-byte unit of
        // each per thread), V_J and dO_J as C x VB bf16 (threads 0-255 and 256-511)
        constexpr int NSU = D * VB / 4;
        int tidv = tid;
        asm volatile("" : "+v"(tidv));
        const int su_r = tidv / (VB / 4), su_c = 4 * (tidv % (VB / 4));
        const int vu = tidv & 255, vu_t = vu / (VB / 8), vu_c = 8 * (vu % (VB / 8));
        f32x4 pS = z4, pD = z4;
        frag_t<T> pX = {};
        auto fetch = [&](int jb) {
            const int v0 = jb * VB;
            if (tid < NSU) {
                pS = *reinterpret_cast<const f32x4 *>(Sg + (int64_t)su_r * D + v0 + su_c);
                pD = *reinterpret_cast<const f32x4 *>(dSg + (int64_t)su_r * D + v0 + su_c);
            }
            if (tid < 512) {
                const T *src = (tid < 256 ? Vg : Og) + (int64_t)vu_t * a.sx_l + v0 + vu_c;
                pX = *reinterpret_cast<const frag_t<T> *>(src);
            }
        };
        float sd = 0.f;  // <dS', S> over this thread's units
        auto stage = [&]() {
            if (tid < NSU) {
                typedef T t4 __attribute__((ext_vector_type(4)));
                t4 sh = {}, sl = {}, dh = {}, dl = {};
#pragma unroll
                for (int j = 0; j < 4; ++j) {
                    sh[j] = cvt<T>(pS[j]);
                    sl[j] = cvt<T>(pS[j] - tof<T>(sh[j]));
                    dh[j] = cvt<T>(pD[j]);
                    dl[j] = cvt<T>(pD[j] - tof<T>(dh[j]));
                }
                const int pb = bpos(su_r, su_c);
                *reinterpret_cast<t4 *>(&sSh[pb]) = sh;
                *reinterpret_cast<t4 *>(&sSl[pb]) = sl;
                *reinterpret_cast<t4 *>(&sDh[pb]) = dh;
                *reinterpret_cast<t4 *>(&sDl[pb]) = dl;
                sd = fmaf(pS[0], pD[0], fmaf(pS[1], pD[1], fmaf(pS[2], pD[2], fmaf(pS[3], pD[3], sd))));
            }
            if (tid < 256) {
                *reinterpret_cast<frag_t<T> *>(&sV[vu_t * LDV + vu_c]) = pX;
            } else if (tid < 512) {
                *reinterpret_cast<frag_t<T> *>(&sO[vu_t * LDV + vu_c]) = pX;
#pragma unroll
                for (int j = 0; j < 8; ++j) sOt[(vu_c + j) * LDOT + vu_t] = pX[j];
            }
        };

        __syncthreads();  // the previous item is done with LDS
        for (int e = tid; e < C * D / 8; e += NTH) {
            const int t = e / (D / 8), c8 = 8 * (e % (D / 8));
            const int64_t off = xo0 + (int64_t)t * a.sx_l + c8;
            *reinterpret_cast<frag_t<T> *>(&xq[t * LDX + c8]) = *reinterpret_cast<const frag_t<T> *>((const T *)a.q + off);
            *reinterpret_cast<frag_t<T> *>(&xk[t * LDX + c8]) = *reinterpret_cast<const frag_t<T> *>((const T *)a.k + off);
        }
        fetch(0);
        if (tid < 64) {
            const float b = wave_scan_dpp(a.g[go0 + (int64_t)tid * a.sg_l]);
            const float bC = lane_value(b, 63);
            sb[tid] = b;
            sg[tid] = expf(b);
            se[tid] = expf(bC - b);
            sbe[tid] = a.beta[go0 + (int64_t)tid * a.sg_l];
        }
        __syncthreads();

        // scores: wave w forms tile (w % 4, w / 4) of K K^T and of Q K^T
        {
            const int st = w >> 2;
            f32x4 pk = z4, pq = z4;
#pragma unroll 1
            for (int kk = 0; kk < D; kk += 32) {
                const frag_t<T> bk = x_rm(xk, LDX, 16 * st, kk);
                mma(pk, x_rm(xk, LDX, 16 * mt, kk), bk);
                mma(pq, x_rm(xq, LDX, 16 * mt, kk), bk);
            }
#pragma unroll
            for (int r = 0; r < 4; ++r) {
                const int t = 16 * mt + 4 * q4 + r, s2 = 16 * st + n16;
                const float ga = expf(sb[t] - sb[s2]);
                sX[t * LD6 + s2] = s2 < t ? ga * pk[r] : 0.f;
                sP[t * LD6 + s2] = s2 <= t ? ga * pq[r] : 0.f;
            }
        }
        __syncthreads();
        gdn_tinv<NTH>(tid, sX, sT, sbe);  // T = (I + diag(beta) KK o Gamma)^{-1}; ends with a barrier
        {  // T -> its hi/lo pair, split once for every wave that reads it
            static_assert(4 * NTH == C * C, "four elements of T per thread");
            typedef T t4 __attribute__((ext_vector_type(4)));
            const int r = (4 * tid) / C, c = (4 * tid) % C;
            const f32x4 x = *reinterpret_cast<const f32x4 *>(&sT[r * LD6 + c]);
            t4 h = {}, l = {};
#pragma unroll
            for (int j = 0; j < 4; ++j) {
                h[j] = cvt<T>(x[j]);
                l[j] = cvt<T>(x[j] - tof<T>(h[j]));
            }
            __syncthreads();  // every fp32 read of T is done
            *reinterpret_cast<t4 *>(&sTh[tpos(r, c)]) = h;
            *reinterpret_cast<t4 *>(&sTl[tpos(r, c)]) = l;
        }

        // one accumulator array, overlaid by role (both roles run the same code,
        // so separate arrays would all stay live on every wave):
        //   A: G_W = acc[0, NTW), dK_S = acc[NTW, 2 NTW)
        //   B: dQ_S = acc[0, NTW), dA = acc[NTW, NTW + 2), dP = acc[NTW + 2, NTW + 4)
        constexpr int NACC = 2 * NTW > NTW + 4 ? 2 * NTW : NTW + 4;
        f32x4 acc[NACC];
#pragma unroll
        for (int j = 0; j < NACC; ++j) acc[j] = z4;
        f32x4 *const accA = acc, *const accB = acc + NTW, *const dA2 = acc + NTW, *const dP2 = acc + NTW + 2;
        float rGUv[4] = {0.f, 0.f, 0.f, 0.f};  // B: sum_v G_U v over the blocks

        for (int jb = 0; jb < NBLK; ++jb) {
            const int v0 = jb * VB, nb = half;  // the wave's 16 columns of the block
            asm volatile("" : "+v"(lane));      // (as at the top of the item loop)
            q4 = lane >> 4;
            n16 = lane & 15;
            if (jb > 0) __syncthreads();     // every read of the previous block is done
            stage();
            if (jb + 1 < NBLK) fetch(jb + 1);
            __syncthreads();
            if (!grpB) {  // Y = K S_J;  R = beta (V_J - gamma Y)
                f32x4 y = z4;
#pragma unroll 1
                for (int kk = 0; kk < D; kk += 32) {
                    const frag_t<T> bh = b_tr(sSh, kk, 16 * nb), bl = b_tr(sSl, kk, 16 * nb);  // B[v][k'] = S_J[k'][v]
                    const frag_t<T> ak = x_rm(xk, LDX, 16 * mt, kk);
                    mma(y, ak, bh);
                    mma(y, ak, bl);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * mt + 4 * q4 + r, v = 16 * nb + n16;
                    sR[t * LDR + v] = sbe[t] * (tof<T>(sV[t * LDV + v]) - sg[t] * y[r]);
                }
            } else {  // dU_J = e o K dS'_J + P^T dO_J
                f32x4 u = z4;
#pragma unroll 1
                for (int kk = 0; kk < D; kk += 32) {
                    const frag_t<T> bh = b_tr(sDh, kk, 16 * nb), bl = b_tr(sDl, kk, 16 * nb);  // B[v][k'] = dS'_J[k'][v]
                    const frag_t<T> ak = x_rm(xk, LDX, 16 * mt, kk);
                    mma(u, ak, bh);
                    mma(u, ak, bl);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) u[r] *= se[16 * mt + 4 * q4 + r];
#pragma unroll 1
                for (int kk = 0; kk < C; kk += 32) {
                    frag_t<T> ph, pl;
                    f_tr(sP, LD6, 16 * mt, kk, ph, pl);                 // A[t][s] = P[s][t]
                    const frag_t<T> bo = x_rm(sOt, LDOT, 16 * nb, kk);  // B[v][s] = dO_J[s][v]
                    mma(u, ph, bo);
                    mma(u, pl, bo);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) sdU[(16 * mt + 4 * q4 + r) * LDR + 16 * nb + n16] = u[r];
            }
            __syncthreads();
            if (!grpB) {  // U_J = T R
                f32x4 u = z4;
#pragma unroll 1
                for (int kk = 0; kk < C; kk += 32) {
                    frag_t<T> th, tl, rh, rl;
                    th = t_rm(sTh, 16 * mt, kk);
                    tl = t_rm(sTl, 16 * mt, kk);
                    f_tr(sR, LDR, 16 * nb, kk, rh, rl);  // B[v][s] = R[s][v]
                    mma3(u, th, tl, rh, rl);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) sU[(16 * mt + 4 * q4 + r) * LDU + 16 * nb + n16] = u[r];
            } else {  // G_U,J = T^T dU_J;  dv_J = beta G_U,J
                f32x4 gu = z4;
#pragma unroll 1
                for (int kk = 0; kk < C; kk += 32) {
                    frag_t<T> th, tl, dh, dl;
                    th = t_tr(sTh, kk, 16 * mt);  // A[t][s] = T[s][t]
                    tl = t_tr(sTl, kk, 16 * mt);
                    f_tr(sdU, LDR, 16 * nb, kk, dh, dl);  // B[v][s] = dU[s][v]
                    mma3(gu, th, tl, dh, dl);
                }
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * mt + 4 * q4 + r, v = 16 * nb + n16;
                    sGU[t * LDU + v] = gu[r];
                    ((T *)a.dv)[xo0 + (int64_t)t * a.sx_l + v0 + v] = cvt<T>(sbe[t] * gu[r]);
                    rGUv[r] = fmaf(gu[r], tof<T>(sV[t * LDV + v]), rGUv[r]);
                }
            }
            __syncthreads();
            if (!grpB) {  // G_W -= G_U,J S_J^T;  dK_S += U_J dS'_J^T  (contraction over the block's 32 v)
                frag_t<T> gh, gl, uh, ul;
                f_rm(sGU, LDU, 16 * mt, 0, gh, gl);
                f_rm(sU, LDU, 16 * mt, 0, uh, ul);
                gh = -gh;
                gl = -gl;
#pragma unroll
                for (int j = 0; j < NTW; ++j) {
                    const int nt = NTW * half + j;
                    mma3(accA[j], gh, gl, b_rm(sSh, 16 * nt), b_rm(sSl, 16 * nt));  // B[k'][v] = S_J[k'][v]
                    mma3(accB[j], uh, ul, b_rm(sDh, 16 * nt), b_rm(sDl, 16 * nt));
                    sched_fence();  // one tile's operands live at a time
                }
            } else {  // dQ_S += dO_J S_J^T;  dA -= G_U,J U_J^T;  dP += dO_J U_J^T
                const frag_t<T> ao = x_rm(sO, LDV, 16 * mt, 0);
#pragma unroll
                for (int j = 0; j < NTW; ++j) {
                    mma(accA[j], ao, b_rm(sSh, 16 * (NTW * half + j)));
                    mma(accA[j], ao, b_rm(sSl, 16 * (NTW * half + j)));
                    sched_fence();
                }
                frag_t<T> gh, gl;
                f_rm(sGU, LDU, 16 * mt, 0, gh, gl);
                gh = -gh;
                gl = -gl;
#pragma unroll
                for (int j = 0; j < 2; ++j) {
                    frag_t<T> uh, ul;
                    f_rm(sU, LDU, 16 * (2 * half + j), 0, uh, ul);  // B[s][v] = U_J[s][v]
                    mma3(dA2[j], gh, gl, uh, ul);
                    mma(dP2[j], ao, uh);
                    mma(dP2[j], ao, ul);
                    sched_fence();
                }
            }
        }
        __syncthreads();  // the blocks are done: sBlk, sX are free
        asm volatile("" : "+v"(lane));
        q4 = lane >> 4;
        n16 = lane & 15;

        // B: dA and dP terms.  KK of the wave's two C x C tiles again (exact
        // bf16 operands), dbeta and decay-gradient sums, dP o Gamma and
        // Ah + Ah^T (Ah strictly lower, mirrored) to LDS.
        float rowX[4] = {0.f, 0.f, 0.f, 0.f}, rowY[4] = {0.f, 0.f, 0.f, 0.f};
        if (grpB) {
#pragma unroll
            for (int j = 0; j < 2; ++j) {
                const int ns = 2 * half + j;
                f32x4 kk4 = z4;
#pragma unroll 1
                for (int kk = 0; kk < D; kk += 32) mma(kk4, x_rm(xk, LDX, 16 * mt, kk), x_rm(xk, LDX, 16 * ns, kk));
                float col = 0.f;
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * mt + 4 * q4 + r, s2 = 16 * ns + n16;
                    const float ge = expf(sb[t] - sb[s2]);
                    const float dAv = s2 < t ? dA2[j][r] : 0.f;
                    const float kkm = s2 < t ? ge * kk4[r] : 0.f;
                    const float dPv = s2 <= t ? dP2[j][r] : 0.f;
                    rowX[r] = fmaf(dAv, kkm, rowX[r]);                           // sum_s dA KK o Gamma (dbeta)
                    const float ex = dAv * sbe[t] * kkm + dPv * sP[t * LD6 + s2];  // dA o A + dP o P
                    rowY[r] += ex;
                    col -= ex;
                    sE1[t * LD6 + s2] = s2 <= t ? dPv * ge : 0.f;
                    const float ah = dAv * sbe[t] * ge;
                    if (s2 < t) {
                        sE2[t * LD6 + s2] = ah;
                        sE2[s2 * LD6 + t] = ah;
                    } else if (s2 == t) {
                        sE2[t * LD6 + t] = 0.f;
                    }
                }
                col += __shfl_xor(col, 16);
                col += __shfl_xor(col, 32);
                if (q4 == 0) sCol[mt][16 * ns + n16] = col;
            }
        }
        __syncthreads();
        float rowZ[4] = {0.f, 0.f, 0.f, 0.f};  // A: sum G_W k;  B: gamma sum q dQ_S
        float rowW[4] = {0.f, 0.f, 0.f, 0.f};  // A: sum dK_S k
        if (!grpB) {  // dk
            f32x4 dk[NTW];
#pragma unroll
            for (int j = 0; j < NTW; ++j) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * mt + 4 * q4 + r, c = 16 * (NTW * half + j) + n16;
                    const float kv = tof<T>(xk[t * LDX + c]);
                    rowZ[r] = fmaf(accA[j][r], kv, rowZ[r]);
                    rowW[r] = fmaf(accB[j][r], kv, rowW[r]);
                    dk[j][r] = se[t] * accB[j][r] + sbe[t] * sg[t] * accA[j][r];
                }
            }
#pragma unroll 1
            for (int kk = 0; kk < C; kk += 32) {
                frag_t<T> eh, el, ah, al;
                f_tr(sE1, LD6, 16 * mt, kk, eh, el);  // A[t][s] = (dP o Gamma)[s][t]
                f_rm(sE2, LD6, 16 * mt, kk, ah, al);  // A[t][s] = (Ah + Ah^T)[t][s]
#pragma unroll
                for (int j = 0; j < NTW; ++j) {
                    const int c0 = 16 * (NTW * half + j);
                    const frag_t<T> bq = x_tr(xq, LDX, c0, kk), bk = x_tr(xk, LDX, c0, kk);  // B[c][s] = X[s][c]
                    mma(dk[j], eh, bq);
                    mma(dk[j], el, bq);
                    mma(dk[j], ah, bk);
                    mma(dk[j], al, bk);
                    sched_fence();
                }
            }
#pragma unroll
            for (int j = 0; j < NTW; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    ((T *)a.dk)[xo0 + (int64_t)(16 * mt + 4 * q4 + r) * a.sx_l + 16 * (NTW * half + j) + n16] =
                        cvt<T>(dk[j][r]);
        } else {  // dq
            f32x4 dq[NTW];
#pragma unroll
            for (int j = 0; j < NTW; ++j) {
#pragma unroll
                for (int r = 0; r < 4; ++r) {
                    const int t = 16 * mt + 4 * q4 + r, c = 16 * (NTW * half + j) + n16;
                    dq[j][r] = sg[t] * accA[j][r];
                    rowZ[r] = fmaf(tof<T>(xq[t * LDX + c]), dq[j][r], rowZ[r]);
                }
            }
#pragma unroll 1
            for (int kk = 0; kk < C; kk += 32) {
                frag_t<T> eh, el;
                f_rm(sE1, LD6, 16 * mt, kk, eh, el);  // A[t][s] = (dP o Gamma)[t][s]
#pragma unroll
                for (int j = 0; j < NTW; ++j) {
                    const frag_t<T> bk = x_tr(xk, LDX, 16 * (NTW * half + j), kk);
                    mma(dq[j], eh, bk);
                    mma(dq[j], el, bk);
                    sched_fence();
                }
            }
#pragma unroll
            for (int j = 0; j < NTW; ++j)
#pragma unroll
                for (int r = 0; r < 4; ++r)
                    ((T *)a.dq)[xo0 + (int64_t)(16 * mt + 4 * q4 + r) * a.sx_l + 16 * (NTW * half + j) + n16] =
                        cvt<T>(dq[j][r]);
        }
        // row sums over the 16 lanes of each row, two waves (halves) per row tile
        //   sRow[0]: A sum G_W k        [1]: A sum dK_S k       [2]: B gamma sum q dQ_S
        //   sRow[3]: B sum_v G_U v      [4]: B sum dA KK o Gamma [5]: B rows of dA o A + dP o P
#pragma unroll
        for (int r = 0; r < 4; ++r) {
            const int t = 16 * mt + 4 * q4 + r;
            const float z = rowsum16(rowZ[r]), wv = rowsum16(rowW[r]);
            const float x = rowsum16(rowX[r]), y = rowsum16(rowY[r]), u = rowsum16(rGUv[r]);
            if (n16 == 0) {
                if (!grpB) {
                    sRow[0][half][t] = z;
                    sRow[1][half][t] = wv;
                } else {
                    sRow[2][half][t] = z;
                    sRow[3][half][t] = u;
                    sRow[4][half][t] = x;
                    sRow[5][half][t] = y;
                }
            }
        }
        sd = wave_sum(sd);
        if (lane == 0) sWav[w] = sd;
        __syncthreads();
        if (tid < 64) {  // per token, then dg_t = sum_{t' >= t} db_t' (one wave)
            const int t = tid;
            auto R = [&](int k) { return sRow[k][0][t] + sRow[k][1][t]; };
            const float gwk = R(0), rt = se[t] * R(1);
            a.dbeta[go0 + (int64_t)t * a.sg_l] = sg[t] * gwk + R(3) + R(4);
            // sCol holds the column sums negated (rows minus columns of dA o A + dP o P)
            float db = R(2) + R(5) + (sCol[0][t] + sCol[1][t] + sCol[2][t] + sCol[3][t]) + sbe[t] * sg[t] * gwk - rt;
            float tot = 0.f;
            for (int u = 0; u < 16; ++u) tot += sWav[u];
            const float rsum = wave_sum(rt);
            if (t == C - 1) db += rsum + sg[C - 1] * tot;
            a.dg[go0 + (int64_t)t * a.sg_l] = wave_incl_suffix(db, lane);
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
                                  dim3(1024), 0, s, e0, e1, 0, a);
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
        if (!a.wsSc || !a.wsDc || a.n_x < 1) return hipErrorInvalidValue;
        break;
    default: return hipErrorInvalidValue;
    }
    if (D == 128) return gdn_phase_d<128>(phase, a, s, e0, e1);
    if (D == 64) return gdn_phase_d<64>(phase, a, s, e0, e1);
    return hipErrorInvalidValue;
}

}  // namespace sf
